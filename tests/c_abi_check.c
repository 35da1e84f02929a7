/* The C ABI from plain C99: the header needs nothing but the C library,
 * and the host-only calls work without a GPU.  Built and run by
 * test_abi_host.py against the in-tree library. */
#include <stdio.h>
#include <string.h>

#include "sparseserve.h"

#define CHECK(c)                                                      \
    do {                                                              \
        if (!(c)) {                                                   \
            fprintf(stderr, "failed at line %d: %s\n", __LINE__, #c); \
            return 1;                                                 \
        }                                                             \
    } while (0)

int main(void)
{
    int64_t ws[4] = {30, 50, 10, 40};
    int32_t admit[4];
    int64_t used = -1, n_items = -1;
    int32_t items[16 * 4];

    CHECK(ss_abi_version() == SS_ABI_VERSION);
    CHECK(strlen(ss_status_string(SS_OK)) > 0);
    CHECK(strcmp(ss_status_string(SS_ERR_TIMEOUT), "unknown status") != 0);
    CHECK(ss_set_host_wait_timeout(250) == SS_OK && ss_set_host_wait_timeout(0) == SS_OK);
    /* the multi-layer step: no layers is no work; bad counts and null arrays are errors */
    CHECK(ss_decode_step_dev(NULL, NULL, 0, 0, NULL, NULL, NULL, NULL, NULL, NULL) == SS_OK);
    CHECK(ss_decode_step_dev(NULL, NULL, 1, 0, NULL, NULL, NULL, NULL, NULL, NULL) == SS_ERR_INVALID_ARG);
    CHECK(ss_decode_step_dev(NULL, NULL, -1, 0, NULL, NULL, NULL, NULL, NULL, NULL) == SS_ERR_INVALID_ARG);
    CHECK(ss_decode_step(NULL, 0, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == SS_OK);
    CHECK(ss_decode_step(NULL, 1, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == SS_ERR_INVALID_ARG);

    /* Algorithm 1 over 100 bytes: 30 fits, 50 fits (80), 10 fits (90), 40 does not */
    CHECK(ss_schedule_batch(ws, 4, 100, admit, &used) == SS_OK);
    CHECK(admit[0] == 1 && admit[1] == 1 && admit[2] == 1 && admit[3] == 0 && used == 90);

    /* a 1000-token prompt of 4 layers, 2500 tokens per batch: 2 layers per batch */
    CHECK(ss_prefill_plan(1000, 4, 2500, items, 16, &n_items) == SS_OK);
    CHECK(n_items == 4);
    CHECK(items[0] == 0 && items[1] == 0 && items[2] == 0 && items[3] == 1000);
    CHECK(items[4 * 3 + 0] == 1 && items[4 * 3 + 1] == 3);

    /* errors come back as codes with a message, never as a crash */
    CHECK(ss_schedule_batch(ws, -1, 100, admit, &used) != SS_OK);
    CHECK(strlen(ss_last_error()) > 0);
    printf("c abi ok\n");
    return 0;
}

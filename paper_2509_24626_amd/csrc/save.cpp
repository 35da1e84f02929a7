// FlashD2H, CPU-assisted saving of new KV to the DRAM pool (Section 3.2.2).
//
// The new tokens of a layer form one contiguous tensor on the GPU.  Saving
// them is split in two, as the paper does: one device-to-host copy of the
// whole tensor into a pinned staging buffer on the caller's (save) stream,
// then host threads place every token into its block record in the pool.
// The GPU spends no compute on it: the copy runs on a copy engine, and the
// scatter on this library's own threads, so it overlaps the next layers'
// work.  Staging buffers form a ring; a save whose buffer is still being
// scattered waits for it.
//
// Record layout: K tile [blk][d] row-major, then V tile channel-major
// [d][blk] (bf16), so a token is one 256-byte K row and d strided V values.
#include <atomic>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <mutex>
#include <thread>
#include <vector>

#include "internal.hpp"

namespace {

struct job {
    int slot;
    int n_new;
    std::vector<int32_t> len;
    std::atomic<int> parts_left{0};
};

}  // namespace

struct ss_kv_saver {
    int B = 0, Hkv = 0, blk = 0, d = 0, max_new = 0;
    size_t record_bytes = 0, slot_bytes = 0;
    uint8_t *pool = nullptr;
    std::vector<int64_t> pool_off;
    std::vector<int32_t> pool_blocks;
    std::vector<void *> staging;
    std::vector<hipEvent_t> copied;
    std::vector<bool> busy;
    int next = 0;
    int threads = 1;

    std::mutex mu;
    std::condition_variable cv_work, cv_done;
    std::deque<std::pair<job *, int>> queue;  // (job, part)
    int in_flight = 0;                        // jobs queued or running
    bool quit = false;
    ss_status error = SS_OK;
    std::string error_msg;
    std::vector<std::thread> workers;

    ~ss_kv_saver()
    {
        {
            std::lock_guard<std::mutex> g(mu);
            quit = true;
        }
        cv_work.notify_all();
        for (auto &t : workers) t.join();
        for (hipEvent_t e : copied)
            if (e) (void)hipEventDestroy(e);
        for (void *p : staging)
            if (p) (void)hipHostFree(p);
    }

    // the units [u0, u1) of a job: every token of every (sequence, head)
    void scatter(const job &jb, int part)
    {
        const int units = B * Hkv;
        const int u0 = (int)((int64_t)units * part / threads), u1 = (int)((int64_t)units * (part + 1) / threads);
        const uint16_t *src = static_cast<const uint16_t *>(staging[jb.slot]);
        for (int u = u0; u < u1; ++u) {
            const int b = u / Hkv, g = u - b * Hkv;
            for (int i = 0; i < jb.n_new; ++i) {
                const int T = jb.len[b] + i;
                const int j = T / blk, p = T - j * blk;
                const uint16_t *kv = src + (((int64_t)b * jb.n_new + i) * Hkv + g) * 2 * d;
                uint8_t *rec = pool + pool_off[u] + (int64_t)j * (int64_t)record_bytes;
                std::memcpy(rec + (size_t)p * d * 2, kv, (size_t)d * 2);
                uint16_t *vt = reinterpret_cast<uint16_t *>(rec + (size_t)blk * d * 2);
                for (int c = 0; c < d; ++c) vt[c * blk + p] = kv[d + c];
            }
        }
    }

    void worker()
    {
        for (;;) {
            std::pair<job *, int> w;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv_work.wait(lk, [&] { return quit || !queue.empty(); });
                if (queue.empty()) return;  // quit with nothing left
                w = queue.front();
                queue.pop_front();
            }
            job *jb = w.first;
            hipError_t e = hipEventSynchronize(copied[jb->slot]);
            if (e == hipSuccess) scatter(*jb, w.second);
            if (jb->parts_left.fetch_sub(1) == 1 || e != hipSuccess) {
                std::lock_guard<std::mutex> g(mu);
                if (e != hipSuccess && error == SS_OK) {
                    error = SS_ERR_HIP;
                    error_msg = std::string("ss_kv_save: wait for the copy: ") + hipGetErrorString(e);
                }
                if (jb->parts_left.load() == 0) {
                    busy[jb->slot] = false;
                    --in_flight;
                    delete jb;
                    cv_done.notify_all();
                }
            }
        }
    }

    // with mu held: wait until `slot` is free (or everything, slot < 0)
    void wait_locked(std::unique_lock<std::mutex> &lk, int slot)
    {
        cv_done.wait(lk, [&] { return slot < 0 ? in_flight == 0 : !busy[slot]; });
    }
};

extern "C" {

ss_status ss_kv_saver_create(int B, int Hkv, int blk, int d, void *pool_host, const int64_t *pool_off,
                             const int32_t *pool_blocks, int max_new_tokens, int staging_slots, int threads,
                             ss_kv_saver **out)
{
    SS_CHECK_ARG(out, "ss_kv_saver_create: null output");
    *out = nullptr;
    SS_CHECK_ARG(B > 0 && Hkv > 0 && max_new_tokens > 0, "ss_kv_saver_create: bad shape B=%d Hkv=%d max_new=%d", B,
                 Hkv, max_new_tokens);
    SS_CHECK_SUPPORTED(d == ss::kHeadDim, "ss_kv_saver_create: d=%d (only 128)", d);
    SS_CHECK_SUPPORTED(ss::supported_blk(blk), "ss_kv_saver_create: blk=%d (8, 16 or 32)", blk);
    SS_CHECK_ARG(pool_host && pool_off && pool_blocks, "ss_kv_saver_create: null pointer");
    SS_CHECK_ARG(staging_slots >= 1 && staging_slots <= 64, "ss_kv_saver_create: staging_slots=%d (1..64)",
                 staging_slots);
    SS_CHECK_ARG(threads >= 1 && threads <= 64, "ss_kv_saver_create: threads=%d (1..64)", threads);
    for (int b = 0; b < B; ++b) SS_CHECK_ARG(pool_blocks[b] >= 0, "ss_kv_saver_create: pool_blocks[%d] < 0", b);
    auto *sv = new ss_kv_saver;
    sv->B = B;
    sv->Hkv = Hkv;
    sv->blk = blk;
    sv->d = d;
    sv->max_new = max_new_tokens;
    sv->record_bytes = (size_t)2 * blk * d * 2;
    sv->slot_bytes = (size_t)B * max_new_tokens * Hkv * 2 * d * 2;
    sv->pool = static_cast<uint8_t *>(pool_host);
    sv->pool_off.assign(pool_off, pool_off + (size_t)B * Hkv);
    sv->pool_blocks.assign(pool_blocks, pool_blocks + B);
    sv->threads = threads;
    sv->staging.assign(staging_slots, nullptr);
    sv->copied.assign(staging_slots, nullptr);
    sv->busy.assign(staging_slots, false);
    for (int i = 0; i < staging_slots; ++i) {
        hipError_t e = hipHostMalloc(&sv->staging[i], sv->slot_bytes, hipHostMallocDefault);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&sv->copied[i], hipEventDisableTiming | hipEventBlockingSync);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            delete sv;
            return ss::fail(SS_ERR_OOM, "ss_kv_saver_create: staging buffer or event: %s", hipGetErrorString(e));
        }
    }
    for (int i = 0; i < threads; ++i) sv->workers.emplace_back([sv] { sv->worker(); });
    *out = sv;
    ss::clear_error();
    return SS_OK;
}

void ss_kv_saver_destroy(ss_kv_saver *sv)
{
    if (!sv) return;
    {
        std::unique_lock<std::mutex> lk(sv->mu);
        sv->wait_locked(lk, -1);
    }
    delete sv;
}

ss_status ss_kv_save(ss_kv_saver *sv, const void *new_kv, int n_new, const int32_t *len, void *stream)
{
    SS_CHECK_ARG(sv && len, "ss_kv_save: null argument");
    SS_CHECK_ARG(n_new >= 0 && n_new <= sv->max_new, "ss_kv_save: n_new=%d (0..%d)", n_new, sv->max_new);
    if (n_new == 0) return SS_OK;
    SS_CHECK_ARG(new_kv, "ss_kv_save: null new_kv");
    for (int b = 0; b < sv->B; ++b) {
        SS_CHECK_ARG(len[b] >= 0, "ss_kv_save: len[%d] < 0", b);
        SS_CHECK_ARG((int64_t)(len[b] + n_new - 1) / sv->blk < sv->pool_blocks[b],
                     "ss_kv_save: sequence %d: token %d lies past its %d pool blocks", b, len[b] + n_new - 1,
                     sv->pool_blocks[b]);
    }
    const hipStream_t s = ss::as_stream(stream);
    std::unique_lock<std::mutex> lk(sv->mu);
    if (sv->error != SS_OK) return ss::fail(sv->error, "%s", sv->error_msg.c_str());
    const int slot = sv->next;
    sv->wait_locked(lk, slot);  // its previous scatter must be finished
    const size_t bytes = (size_t)sv->B * n_new * sv->Hkv * 2 * sv->d * 2;
    hipError_t e = hipMemcpyAsync(sv->staging[slot], new_kv, bytes, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipEventRecord(sv->copied[slot], s);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return ss::fail(SS_ERR_HIP, "ss_kv_save: copy to staging: %s", hipGetErrorString(e));
    }
    job *jb = new job;
    jb->slot = slot;
    jb->n_new = n_new;
    jb->len.assign(len, len + sv->B);
    jb->parts_left.store(sv->threads);
    sv->busy[slot] = true;
    ++sv->in_flight;
    for (int part = 0; part < sv->threads; ++part) sv->queue.emplace_back(jb, part);
    sv->next = (slot + 1) % (int)sv->staging.size();
    lk.unlock();
    sv->cv_work.notify_all();
    return SS_OK;
}

ss_status ss_kv_save_wait(ss_kv_saver *sv)
{
    SS_CHECK_ARG(sv, "ss_kv_save_wait: null saver");
    std::unique_lock<std::mutex> lk(sv->mu);
    sv->wait_locked(lk, -1);
    if (sv->error != SS_OK) return ss::fail(sv->error, "%s", sv->error_msg.c_str());
    return SS_OK;
}

}  // extern "C"

/*
 * CPU oracle for the decode-step hot path of SparseServe (arXiv 2509.24626):
 * block metadata, block criticality scoring, top-k block selection, the LRU
 * HBM block cache, the miss gather and sparse attention over the selected
 * blocks; on the saving side, appending new tokens to the open blocks
 * (with metadata when a block fills) and saving them to the DRAM pool; and
 * the working-set estimates and batch control of the scheduler; and the
 * mean-key metadata and score variants the paper names; and the plan of a
 * layer-segmented prefill.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library calls, links or
 * loads this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do.  It shares no header, helper or constant with the GPU path.
 *
 * Style: plain loops in the order the definitions are written, fp64 for all
 * floating-point arithmetic, no blocking, fusion or reordering.  Each
 * function names the passage of the paper it follows.
 *
 * Data formats (the input contract shared with the GPU path, restated here):
 *   bf16 values are passed as their uint16 bit patterns.
 *   A KV block record of one (sequence, KV head, block) holds blk tokens:
 *     K tile  : blk rows of d channels, element (t, c) at word t*d + c
 *     V tile  : stored channel-major, element (t, c) at word blk*d + c*blk + t
 *   Records of one (sequence b, KV head g) unit are consecutive: block j
 *   starts at byte  unit_off[b*Hkv + g] + j * record_bytes  from the base.
 *   Metadata of block j of unit u: lo[d] then hi[d] (bf16) at
 *     meta + ((u * nblk_max) + j) * 2 * d.
 *
 * Parity pins: every function here is checked against closed forms,
 * invariants, special cases and brute force in tests/test_oracle_pins.py,
 * and tests/test_oracle_mutants.py shows that planted mistakes fail them.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* exact widening of a bf16 bit pattern to double */
static double bf(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int sign_bit(uint16_t h) { return (h & 0x8000u) != 0; }

/* ------------------------------------------------------------------------
 * O0  Block metadata: the bounding cuboid of the keys of a block, i.e. the
 * channel-wise minimum and maximum of K over the block's tokens (Section 2.2,
 * "Dynamic Sparse Attention": metadata that bounds the token keys; created
 * when a block fills, Section 3.1 "KV Cache Manager").
 * Ties between +0 and -0 are broken as IEEE-754 totalOrder does: -0 < +0,
 * so the result is one of the input values and does not depend on the
 * order the tokens are visited in.
 * Blocks j >= nblk[b] are not written.
 * ---------------------------------------------------------------------- */
int oracle_build_metadata(const void *base, const int64_t *unit_off,
                          const int32_t *nblk, int B, int Hkv, int nblk_max,
                          int blk, int d, size_t record_bytes, uint16_t *meta)
{
    if (B < 0 || Hkv <= 0 || nblk_max < 0 || blk <= 0 || d <= 0)
        return 1;
    for (int b = 0; b < B; ++b) {
        int n = nblk[b] < nblk_max ? nblk[b] : nblk_max;
        for (int g = 0; g < Hkv; ++g) {
            int u = b * Hkv + g;
            for (int j = 0; j < n; ++j) {
                const uint16_t *rec = (const uint16_t *)((const char *)base + unit_off[u]
                                                         + (int64_t)j * (int64_t)record_bytes);
                uint16_t *lo = meta + ((int64_t)u * nblk_max + j) * 2 * d;
                uint16_t *hi = lo + d;
                for (int c = 0; c < d; ++c) {
                    uint16_t mn = rec[0 * d + c], mx = rec[0 * d + c];
                    for (int t = 1; t < blk; ++t) {
                        uint16_t x = rec[t * d + c];
                        double vx = bf(x), vmn = bf(mn), vmx = bf(mx);
                        if (vx < vmn || (vx == vmn && sign_bit(x) && !sign_bit(mn)))
                            mn = x;
                        if (vx > vmx || (vx == vmx && !sign_bit(x) && sign_bit(mx)))
                            mx = x;
                    }
                    lo[c] = mn;
                    hi[c] = mx;
                }
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * O1  Block criticality (Section 2.2: a dot product between the query and
 * the block metadata approximates the attention score of the block).
 * With cuboid metadata the score is the largest value q.k can take for any
 * key k inside the cuboid [lo, hi]:
 *     s_h(j) = sum_c max(q_h[c] * lo_j[c], q_h[c] * hi_j[c]).
 * A KV head g serves the query heads h = g*G .. g*G+G-1 (G = Hq / Hkv);
 * the block score of the head is the largest of their bounds:
 *     S(b, g, j) = max_h s_h(j).
 * S has layout [B][Hkv][nblk_max]; entries j >= nblk[b] are set to -inf.
 * ---------------------------------------------------------------------- */
int oracle_score(const uint16_t *q, const uint16_t *meta, const int32_t *nblk,
                 int B, int Hq, int Hkv, int nblk_max, int d, double *S)
{
    if (B < 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || nblk_max < 0 || d <= 0)
        return 1;
    int G = Hq / Hkv;
    for (int b = 0; b < B; ++b) {
        int n = nblk[b] < nblk_max ? nblk[b] : nblk_max;
        for (int g = 0; g < Hkv; ++g) {
            int u = b * Hkv + g;
            for (int j = 0; j < nblk_max; ++j) {
                double best = -INFINITY;
                if (j < n) {
                    const uint16_t *lo = meta + ((int64_t)u * nblk_max + j) * 2 * d;
                    const uint16_t *hi = lo + d;
                    for (int i = 0; i < G; ++i) {
                        int h = g * G + i;
                        const uint16_t *qh = q + ((int64_t)b * Hq + h) * d;
                        double s = 0.0;
                        for (int c = 0; c < d; ++c) {
                            double a = bf(qh[c]) * bf(lo[c]);
                            double e = bf(qh[c]) * bf(hi[c]);
                            s += (a > e ? a : e);
                        }
                        if (s > best)
                            best = s;
                    }
                }
                S[(int64_t)u * nblk_max + j] = best;
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * O2  Top-k block selection per (sequence, KV head) (Section 2.2: select the
 * k most critical blocks; selection is per head, Section 3.2).
 * Order: larger score first; equal scores -> lower block index first.
 * The first min(k, nblk[b]) blocks in that order are returned sorted by
 * ascending block index; remaining entries are -1.  sel: [B][Hkv][k].
 * ---------------------------------------------------------------------- */
static __thread const double *g_sort_scores; /* per-thread: qsort has no context argument */

static int by_score_then_index(const void *pa, const void *pb)
{
    int a = *(const int *)pa, b = *(const int *)pb;
    double sa = g_sort_scores[a], sb = g_sort_scores[b];
    if (sa > sb) return -1;
    if (sa < sb) return 1;
    return (a > b) - (a < b);
}

static int ascending_int(const void *pa, const void *pb)
{
    int a = *(const int *)pa, b = *(const int *)pb;
    return (a > b) - (a < b);
}

int oracle_select(const double *S, const int32_t *nblk, int B, int Hkv,
                  int nblk_max, int k, int32_t *sel)
{
    if (B < 0 || Hkv <= 0 || nblk_max < 0 || k <= 0)
        return 1;
    int *order = (int *)malloc(sizeof(int) * (size_t)(nblk_max > 0 ? nblk_max : 1));
    if (!order)
        return 4;
    for (int b = 0; b < B; ++b) {
        int n = nblk[b] < nblk_max ? nblk[b] : nblk_max;
        if (n < 0) n = 0;
        for (int g = 0; g < Hkv; ++g) {
            int u = b * Hkv + g;
            for (int j = 0; j < n; ++j)
                order[j] = j;
            g_sort_scores = S + (int64_t)u * nblk_max;
            qsort(order, (size_t)n, sizeof(int), by_score_then_index);
            int m = k < n ? k : n;
            qsort(order, (size_t)m, sizeof(int), ascending_int);
            int32_t *out = sel + (int64_t)u * k;
            for (int i = 0; i < k; ++i)
                out[i] = i < m ? order[i] : -1;
        }
    }
    free(order);
    return 0;
}

/* ------------------------------------------------------------------------
 * O3  The HBM block cache of the KV cache manager (Section 3.1): HBM holds
 * fixed-size block slots managed independently per (sequence, KV head);
 * blocks that miss are loaded from DRAM into free slots, and when no slot is
 * free the least recently used block is evicted.
 * Per unit u: C[u] slots numbered 0..C-1, each empty or holding one block
 * together with the step it was last used in.  At step t, with the unit's
 * selection (ascending, -1 entries ignored):
 *   1. every selected block already cached (a hit) has last_use := t;
 *   2. every selected block not cached (a miss), in ascending block order,
 *      goes to the lowest-numbered empty slot if there is one, otherwise to
 *      the slot whose block is not selected at step t and has the smallest
 *      last_use (equal last_use: lowest slot number), evicting that block;
 *      the slot gets last_use := t and the miss is reported as
 *      (b, g, block, slot).
 * slots_out[u][i] is the slot of the i-th selected block (-1 for -1 entries).
 * A selection larger than C[u] is a capacity error (return 3).
 * ---------------------------------------------------------------------- */
typedef struct {
    int units, Hkv;
    int32_t *cap;        /* [units] */
    int64_t *first_slot; /* [units] start of the unit's slots in the arrays below */
    int32_t *slot_block; /* [total] block held, -1 = empty */
    int64_t *slot_last;  /* [total] step of last use */
    int32_t *nblk;       /* [units] blocks of the unit */
} oracle_lru;

void oracle_lru_destroy(oracle_lru *c)
{
    if (!c) return;
    free(c->cap); free(c->first_slot); free(c->slot_block); free(c->slot_last); free(c->nblk);
    free(c);
}

oracle_lru *oracle_lru_create(int B, int Hkv, const int32_t *nblk_per_seq, const int32_t *cap_per_unit)
{
    if (B < 0 || Hkv <= 0) return NULL;
    oracle_lru *c = (oracle_lru *)calloc(1, sizeof *c);
    if (!c) return NULL;
    int units = B * Hkv;
    c->units = units;
    c->Hkv = Hkv;
    c->cap = (int32_t *)malloc(sizeof(int32_t) * (size_t)(units + 1));
    c->first_slot = (int64_t *)malloc(sizeof(int64_t) * (size_t)(units + 1));
    c->nblk = (int32_t *)malloc(sizeof(int32_t) * (size_t)(units + 1));
    int64_t total = 0;
    if (!c->cap || !c->first_slot || !c->nblk) { oracle_lru_destroy(c); return NULL; }
    for (int u = 0; u < units; ++u) {
        c->cap[u] = cap_per_unit[u];
        c->nblk[u] = nblk_per_seq[u / Hkv];
        c->first_slot[u] = total;
        total += cap_per_unit[u] > 0 ? cap_per_unit[u] : 0;
    }
    c->slot_block = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total + 1));
    c->slot_last = (int64_t *)malloc(sizeof(int64_t) * (size_t)(total + 1));
    if (!c->slot_block || !c->slot_last) { oracle_lru_destroy(c); return NULL; }
    for (int64_t s = 0; s < total; ++s) {
        c->slot_block[s] = -1;
        c->slot_last[s] = 0;
    }
    return c;
}

static int is_selected(const int32_t *sel_u, int k, int32_t block)
{
    for (int i = 0; i < k; ++i)
        if (sel_u[i] == block)
            return 1;
    return 0;
}

/* miss_out has room for miss_cap rows of 4 int32; returns 3 on capacity
 * error, 1 on bad arguments, 4 if miss_out is too small. */
int oracle_lru_step(oracle_lru *c, int64_t step, const int32_t *sel, int k,
                    int32_t *slots_out, int32_t *miss_out, int64_t miss_cap,
                    int64_t *n_miss)
{
    if (!c || k <= 0) return 1;
    int64_t nm = 0;
    for (int u = 0; u < c->units; ++u) {
        const int32_t *sel_u = sel + (int64_t)u * k;
        int32_t *out_u = slots_out + (int64_t)u * k;
        int32_t *blocks = c->slot_block + c->first_slot[u];
        int64_t *last = c->slot_last + c->first_slot[u];
        int C = c->cap[u];
        /* the selection must be strictly ascending, then -1 padding */
        int count = 0;
        for (int i = 0; i < k; ++i) {
            if (sel_u[i] < 0) {
                if (sel_u[i] != -1) return 1;
                continue;
            }
            if (i > 0 && (sel_u[i - 1] < 0 || sel_u[i - 1] >= sel_u[i])) return 1;
            if (sel_u[i] >= c->nblk[u]) return 1;
            ++count;
        }
        if (count > C) return 3;
        /* 1. hits */
        for (int i = 0; i < k; ++i) {
            out_u[i] = -1;
            if (sel_u[i] < 0) continue;
            for (int s = 0; s < C; ++s)
                if (blocks[s] == sel_u[i]) {
                    last[s] = step;
                    out_u[i] = s;
                }
        }
        /* 2. misses in ascending block order (the selection is ascending) */
        for (int i = 0; i < k; ++i) {
            if (sel_u[i] < 0 || out_u[i] >= 0) continue;
            int chosen = -1;
            for (int s = 0; s < C; ++s)
                if (blocks[s] < 0) { chosen = s; break; }
            if (chosen < 0) {
                for (int s = 0; s < C; ++s) {
                    if (is_selected(sel_u, k, blocks[s])) continue;
                    if (chosen < 0 || last[s] < last[chosen])
                        chosen = s;
                }
            }
            if (chosen < 0) return 3;
            blocks[chosen] = sel_u[i];
            last[chosen] = step;
            out_u[i] = chosen;
            if (nm >= miss_cap) return 4;
            miss_out[nm * 4 + 0] = u / c->Hkv;
            miss_out[nm * 4 + 1] = u % c->Hkv;
            miss_out[nm * 4 + 2] = sel_u[i];
            miss_out[nm * 4 + 3] = chosen;
            ++nm;
        }
    }
    *n_miss = nm;
    return 0;
}

/* state export: block held by each slot and its last use, units in order */
int64_t oracle_lru_total_slots(const oracle_lru *c)
{
    return c->units ? c->first_slot[c->units - 1] + c->cap[c->units - 1] : 0;
}

void oracle_lru_export(const oracle_lru *c, int32_t *slot_block, int64_t *slot_last)
{
    int64_t total = oracle_lru_total_slots(c);
    for (int64_t s = 0; s < total; ++s) {
        slot_block[s] = c->slot_block[s];
        slot_last[s] = c->slot_last[s];
    }
}

/* ------------------------------------------------------------------------
 * O4  Loading missed blocks from DRAM into their HBM slots (Section 3.2.1):
 * each reported miss (b, g, block, slot) copies the whole block record from
 * the unit's DRAM blocks into the unit's cache slot.
 * ---------------------------------------------------------------------- */
int oracle_gather(const int32_t *miss, int64_t n_miss, const void *pool,
                  const int64_t *pool_off, void *cache, const int64_t *cache_off,
                  size_t record_bytes, int Hkv)
{
    for (int64_t m = 0; m < n_miss; ++m) {
        int b = miss[m * 4 + 0], g = miss[m * 4 + 1];
        int32_t j = miss[m * 4 + 2], s = miss[m * 4 + 3];
        int u = b * Hkv + g;
        const char *src = (const char *)pool + pool_off[u] + (int64_t)j * (int64_t)record_bytes;
        char *dst = (char *)cache + cache_off[u] + (int64_t)s * (int64_t)record_bytes;
        memcpy(dst, src, record_bytes);
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * O5  Attention of one decode query over the selected blocks (Section 2.1,
 * the attention equations S = Q K^T / sqrt(d), P = softmax(S), O = P V,
 * restricted to the tokens of the selected blocks, Section 2.2).
 * For query head h of sequence b (KV head g = h / G), over the tokens t of
 * the blocks listed in slots[b][g][*] (-1 entries skipped), in list order:
 *     z_t = scale * sum_c q[b][h][c] * K[t][c]
 *     p_t = exp(z_t - max z) / sum_t' exp(z_t' - max z)
 *     out[b][h][c] = sum_t p_t * V[t][c]
 * The block of list entry i lives at base + region_off[b*Hkv+g]
 * + slots[b][g][i] * record_bytes.  With no token selected the output is 0.
 * out: fp32 [B][Hq][d].
 * ---------------------------------------------------------------------- */
int oracle_attention(const uint16_t *q, const void *base, const int64_t *region_off,
                     const int32_t *slots, int B, int Hq, int Hkv, int d, int blk,
                     int k, double scale, float *out)
{
    if (B < 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || d <= 0 || blk <= 0 || k <= 0)
        return 1;
    int G = Hq / Hkv;
    size_t record_bytes = (size_t)2 * blk * d * sizeof(uint16_t);
    int64_t ntok_max = (int64_t)k * blk;
    double *z = (double *)malloc(sizeof(double) * (size_t)ntok_max);
    const uint16_t **kv_of = (const uint16_t **)malloc(sizeof(uint16_t *) * (size_t)ntok_max);
    int *t_of = (int *)malloc(sizeof(int) * (size_t)ntok_max);
    double *acc = (double *)malloc(sizeof(double) * (size_t)d);
    if (!z || !kv_of || !t_of || !acc) { free(z); free(kv_of); free(t_of); free(acc); return 4; }
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < Hq; ++h) {
            int g = h / G;
            int u = b * Hkv + g;
            const uint16_t *qh = q + ((int64_t)b * Hq + h) * d;
            /* the selected tokens in order */
            int64_t n = 0;
            for (int i = 0; i < k; ++i) {
                int32_t s = slots[(int64_t)u * k + i];
                if (s < 0) continue;
                const uint16_t *rec = (const uint16_t *)((const char *)base + region_off[u]
                                                         + (int64_t)s * (int64_t)record_bytes);
                for (int t = 0; t < blk; ++t) {
                    kv_of[n] = rec;
                    t_of[n] = t;
                    ++n;
                }
            }
            float *o = out + ((int64_t)b * Hq + h) * d;
            if (n == 0) {
                for (int c = 0; c < d; ++c) o[c] = 0.0f;
                continue;
            }
            double zmax = -INFINITY;
            for (int64_t i = 0; i < n; ++i) {
                const uint16_t *K = kv_of[i];
                int t = t_of[i];
                double dot = 0.0;
                for (int c = 0; c < d; ++c)
                    dot += bf(qh[c]) * bf(K[t * d + c]);
                z[i] = scale * dot;
                if (z[i] > zmax) zmax = z[i];
            }
            double denom = 0.0;
            for (int64_t i = 0; i < n; ++i) {
                z[i] = exp(z[i] - zmax);
                denom += z[i];
            }
            for (int c = 0; c < d; ++c) acc[c] = 0.0;
            for (int64_t i = 0; i < n; ++i) {
                const uint16_t *Vt = kv_of[i] + (int64_t)blk * d; /* channel-major V tile */
                int t = t_of[i];
                double p = z[i] / denom;
                for (int c = 0; c < d; ++c)
                    acc[c] += p * bf(Vt[c * blk + t]);
            }
            for (int c = 0; c < d; ++c) o[c] = (float)acc[c];
        }
    free(z); free(kv_of); free(t_of); free(acc);
    return 0;
}

/* ------------------------------------------------------------------------
 * Writing one token into a block record: the K row at position p and the V
 * column at position p (V tiles are channel-major), in the record layout
 * stated at the top of this file.  kv holds the token's K (d values) then
 * its V (d values).
 * ---------------------------------------------------------------------- */
static void put_token(uint16_t *rec, int blk, int d, int p, const uint16_t *kv)
{
    for (int c = 0; c < d; ++c)
        rec[p * d + c] = kv[c];
    for (int c = 0; c < d; ++c)
        rec[blk * d + c * blk + p] = kv[d + c];
}

/* ------------------------------------------------------------------------
 * O6  Appending a decode step's new tokens in HBM (Section 3.2.2: the
 * layer's new KV tensor, one token per sequence and head, goes into the
 * free slot of the sequence's open block; Section 3.1: a block's metadata
 * is created when the block fills).
 *   new_kv : [B][Hkv][2][d] bf16, K then V of sequence b's new token
 *   len    : [B] tokens of sequence b before this token (updated: +1)
 *   nblk   : [B] full blocks of sequence b (set to j + 1 when block j fills)
 *   open   : [B][Hkv] block records, the open block of each (b, g)
 *   meta   : [B][Hkv][nblk_max][2][d], written for the block that fills
 * The token goes to block j = len / blk at position p = len % blk.  When
 * p == blk - 1 the open record is complete: its metadata (O0 on that one
 * record) is stored as block j of the unit.  Returns 2 if a block that
 * fills has j >= nblk_max; nothing is changed then.
 * ---------------------------------------------------------------------- */
int oracle_append(const uint16_t *new_kv, int32_t *len, int32_t *nblk, int B, int Hkv,
                  int blk, int d, int nblk_max, void *open, uint16_t *meta)
{
    if (B < 0 || Hkv <= 0 || blk <= 0 || d <= 0 || nblk_max < 0)
        return 1;
    size_t record_bytes = (size_t)2 * blk * d * 2;
    for (int b = 0; b < B; ++b)
        if (len[b] < 0 || (len[b] % blk == blk - 1 && len[b] / blk >= nblk_max))
            return 2;
    for (int b = 0; b < B; ++b) {
        int j = len[b] / blk, p = len[b] % blk;
        for (int g = 0; g < Hkv; ++g) {
            int u = b * Hkv + g;
            uint16_t *rec = (uint16_t *)((char *)open + (int64_t)u * (int64_t)record_bytes);
            put_token(rec, blk, d, p, new_kv + (int64_t)u * 2 * d);
            if (p == blk - 1) {
                int64_t zero = 0;
                int32_t one = 1;
                oracle_build_metadata(rec, &zero, &one, 1, 1, 1, blk, d, record_bytes,
                                      meta + ((int64_t)u * nblk_max + j) * 2 * d);
            }
        }
        len[b] += 1;
        if (p == blk - 1)
            nblk[b] = j + 1;
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * O7  Saving new tokens to the DRAM pool (Section 3.2.2, FlashD2H: the new
 * KV tensor is contiguous; it is copied to host memory in one transfer and
 * host threads then place each token into its KV block in DRAM).  What the
 * pool holds afterwards is defined here, token by token:
 *   new_kv      : [B][n_new][Hkv][2][d] bf16, the n_new new tokens of each
 *                 sequence in order
 *   len         : [B] tokens of sequence b before the first new token
 *   pool        : DRAM pool; block j of unit u = b*Hkv + g is the record at
 *                 pool + pool_off[u] + j * record_bytes
 *   pool_blocks : [B] blocks the pool holds per unit of sequence b
 * Token i of sequence b is token T = len[b] + i of the sequence: block
 * j = T / blk, position p = T % blk.  Returns 2 (nothing written) if some
 * j >= pool_blocks[b].
 * ---------------------------------------------------------------------- */
int oracle_save(const uint16_t *new_kv, int n_new, const int32_t *len, int B, int Hkv,
                int blk, int d, void *pool, const int64_t *pool_off, const int32_t *pool_blocks)
{
    if (B < 0 || n_new < 0 || Hkv <= 0 || blk <= 0 || d <= 0)
        return 1;
    size_t record_bytes = (size_t)2 * blk * d * 2;
    for (int b = 0; b < B; ++b)
        if (n_new > 0 && (len[b] < 0 || (len[b] + n_new - 1) / blk >= pool_blocks[b]))
            return 2;
    for (int b = 0; b < B; ++b)
        for (int i = 0; i < n_new; ++i) {
            int T = len[b] + i;
            int j = T / blk, p = T % blk;
            for (int g = 0; g < Hkv; ++g) {
                int u = b * Hkv + g;
                uint16_t *rec = (uint16_t *)((char *)pool + pool_off[u] + (int64_t)j * (int64_t)record_bytes);
                put_token(rec, blk, d, p, new_kv + (((int64_t)b * n_new + i) * Hkv + g) * 2 * d);
            }
        }
    return 0;
}

/* ------------------------------------------------------------------------
 * O8  Working set of a decoding request (Section 3.3, decoding working
 * set): per (layer, KV head), the union of the blocks selected in the last
 * w decoding steps; the request's working set is the HBM the union takes,
 *     record_bytes * sum over (layer, head) of |union|.
 *   sel_hist : [m][layers][Hkv][k] the request's selections of its m
 *              observed steps, oldest first; -1 entries are padding
 *   fallback : blocks per (layer, head) counted when m == 0 (no history)
 * Steps taken: the last min(w, m) steps, all their entries per (layer,
 * head) collected, sorted, and the distinct non-negative values counted.
 * ---------------------------------------------------------------------- */
static int ascending_i32(const void *pa, const void *pb)
{
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

int64_t oracle_ws_decode(const int32_t *sel_hist, int m, int layers, int Hkv, int k, int w,
                         int fallback, size_t record_bytes)
{
    if (m < 0 || layers <= 0 || Hkv <= 0 || k <= 0 || w <= 0)
        return -1;
    if (m == 0)
        return (int64_t)fallback * layers * Hkv * (int64_t)record_bytes;
    int n_steps = m < w ? m : w;
    int32_t *all = malloc(sizeof(int32_t) * (size_t)n_steps * k);
    if (!all)
        return -1;
    int64_t blocks = 0;
    for (int l = 0; l < layers; ++l)
        for (int g = 0; g < Hkv; ++g) {
            int n = 0;
            for (int s = m - n_steps; s < m; ++s)
                for (int i = 0; i < k; ++i) {
                    int32_t j = sel_hist[(((int64_t)s * layers + l) * Hkv + g) * k + i];
                    if (j >= 0)
                        all[n++] = j;
                }
            qsort(all, (size_t)n, sizeof(int32_t), ascending_i32);
            for (int i = 0; i < n; ++i)
                if (i == 0 || all[i] != all[i - 1])
                    ++blocks;
        }
    free(all);
    return blocks * (int64_t)record_bytes;
}

/* ------------------------------------------------------------------------
 * O9  Working set of a prefill request (Section 3.3, prefill working set):
 * the HBM its KV needs in the current iteration, which is exact.
 *   layer-segmented prefill: one layer of KV of the whole prompt,
 *       ceil(prompt / blk) blocks per KV head;
 *   chunked prefill: the KV of every chunk so far, this one included, in
 *       every layer, ceil(min(prompt, done + chunk) / blk) blocks per KV head
 *       per layer.
 * ---------------------------------------------------------------------- */
int64_t oracle_ws_prefill(int64_t prompt, int64_t done, int64_t chunk, int layers, int Hkv, int blk,
                          size_t record_bytes, int layer_segmented)
{
    if (prompt < 0 || done < 0 || chunk < 0 || layers <= 0 || Hkv <= 0 || blk <= 0)
        return -1;
    int64_t tokens, layer_count;
    if (layer_segmented) {
        tokens = prompt;
        layer_count = 1;
    } else {
        tokens = done + chunk < prompt ? done + chunk : prompt;
        layer_count = layers;
    }
    int64_t blocks = (tokens + blk - 1) / blk;
    return blocks * Hkv * layer_count * (int64_t)record_bytes;
}

/* ------------------------------------------------------------------------
 * O10  Working-set-aware batch control (Section 3.3, Algorithm 1): walk the
 * initial batch in its order; a request joins the batch if the HBM used so
 * far plus its working set stays within m_avl, otherwise it is reset
 * (rejected for this iteration).
 *   ws     : [n] working-set bytes of the initial batch's requests, in order
 *   admit  : [n] 1 if the request joins the batch, 0 if it is reset
 *   m_used : the HBM the admitted requests take
 * ---------------------------------------------------------------------- */
int oracle_schedule(const int64_t *ws, int n, int64_t m_avl, int32_t *admit, int64_t *m_used)
{
    if (n < 0)
        return 1;
    int64_t used = 0;
    for (int i = 0; i < n; ++i) {
        if (ws[i] < 0)
            return 1;
        if (used + ws[i] <= m_avl) {
            admit[i] = 1;
            used += ws[i];
        } else {
            admit[i] = 0;
        }
    }
    *m_used = used;
    return 0;
}

/* ------------------------------------------------------------------------
 * O11  Mean-key block metadata (Section 2.2: the simplest metadata of the
 * DSAs the paper cites is the mean of the block's token keys).  One d-vector
 * per block, bf16: per channel, the exact mean of the blk keys, rounded once
 * to the nearest bf16 (ties to even).
 * The keys are summed in fp64 in token order.  Each key is a bf16 value (8
 * significant bits), so the sum is exact whenever the keys' magnitudes span
 * less than about 2^40; every addition is checked with an error-free
 * transformation, and a block whose sum would be rounded is refused (return
 * 2) rather than given an inexact mean.  Dividing by blk is exact for any
 * blk that is a power of two; otherwise the quotient is rounded to fp64
 * first.
 * meta layout [B*Hkv][nblk_max][d]; blocks j >= nblk[b] are not written.
 * ---------------------------------------------------------------------- */

/* The bf16 value nearest to x, ties to the even significand, from the
 * definition: bf16 carries 8 significant bits down to its smallest normal
 * 2^-126 and a fixed quantum of 2^-133 below it, with the same exponent
 * range as fp32.  x is scaled to that quantum (a power of two, so exactly),
 * rounded to an integer with ties to even (nearbyint in the default
 * rounding mode), and scaled back; the result is exactly representable in
 * fp32, whose upper 16 bits are the bf16 pattern. */
static uint16_t bf16_nearest(double x)
{
    if (x == 0.0)
        return signbit(x) ? 0x8000u : 0u;
    int e;
    (void)frexp(x, &e);          /* |x| in [2^(e-1), 2^e) */
    int qexp = e - 8;            /* quantum of an 8-bit significand */
    if (qexp < -133)
        qexp = -133;             /* subnormal range */
    double r = ldexp(nearbyint(ldexp(x, -qexp)), qexp);
    if (fabs(r) >= ldexp(1.0, 128))
        return x > 0 ? 0x7F80u : 0xFF80u;  /* beyond the largest finite value */
    float f = (float)r;          /* exact */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if (r == 0.0)                /* rounded to zero: keep the sign of x */
        return signbit(x) ? 0x8000u : 0u;
    return (uint16_t)(u >> 16);
}

int oracle_build_metadata_mean(const void *base, const int64_t *unit_off, const int32_t *nblk, int B, int Hkv,
                               int nblk_max, int blk, int d, size_t record_bytes, uint16_t *meta)
{
    if (B < 0 || Hkv <= 0 || nblk_max < 0 || blk <= 0 || d <= 0)
        return 1;
    for (int b = 0; b < B; ++b) {
        int n = nblk[b] < nblk_max ? nblk[b] : nblk_max;
        for (int g = 0; g < Hkv; ++g) {
            int u = b * Hkv + g;
            for (int j = 0; j < n; ++j) {
                const char *unit_base = (const char *)base + unit_off[u];
                const uint16_t *rec = (const uint16_t *)(unit_base + (int64_t)j * (int64_t)record_bytes);
                uint16_t *m = meta + ((int64_t)u * nblk_max + j) * d;
                for (int c = 0; c < d; ++c) {
                    double s = 0.0;
                    for (int t = 0; t < blk; ++t) {
                        double v = bf(rec[t * d + c]);
                        double sum = s + v;
                        /* error of this addition (Knuth's two-sum); 0 iff exact */
                        double vv = sum - s;
                        double err = (s - (sum - vv)) + (v - vv);
                        if (err != 0.0)
                            return 2;
                        s = sum;
                    }
                    m[c] = bf16_nearest(s / (double)blk);
                }
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * O12  Block scores for the metadata kinds and GQA aggregations (Section
 * 2.2: a dot product of the block metadata with the query estimates the
 * block's attention score; the paper's DSAs differ in the metadata).
 *   kind 0 (cuboid, [lo, hi]): s_h(j) = sum_c max(q_h[c]*lo[c], q_h[c]*hi[c])
 *   kind 1 (mean key m):       s_h(j) = sum_c q_h[c] * m[c]
 *   agg 0: S = max over the group's query heads of s_h
 *   agg 1: S = sum over the group's query heads of s_h (the mean over the
 *          heads ranks the blocks the same way)
 * meta layout: kind 0 [B*Hkv][nblk_max][2][d], kind 1 [B*Hkv][nblk_max][d].
 * fp64 arithmetic; entries j >= nblk[b] are -inf.
 * ---------------------------------------------------------------------- */
int oracle_score_variant(const uint16_t *q, const uint16_t *meta, int kind, int agg, const int32_t *nblk, int B,
                         int Hq, int Hkv, int nblk_max, int d, double *S)
{
    if (B < 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv != 0 || nblk_max < 0 || d <= 0 || kind < 0 || kind > 1 ||
        agg < 0 || agg > 1)
        return 1;
    int G = Hq / Hkv;
    int row = kind == 0 ? 2 * d : d;
    for (int b = 0; b < B; ++b) {
        int n = nblk[b] < nblk_max ? nblk[b] : nblk_max;
        for (int g = 0; g < Hkv; ++g) {
            int u = b * Hkv + g;
            for (int j = 0; j < nblk_max; ++j) {
                if (j >= n) {
                    S[(int64_t)u * nblk_max + j] = -INFINITY;
                    continue;
                }
                const uint16_t *mj = meta + ((int64_t)u * nblk_max + j) * row;
                double best = -INFINITY, total = 0.0;
                for (int i = 0; i < G; ++i) {
                    const uint16_t *qh = q + ((int64_t)b * Hq + g * G + i) * d;
                    double s = 0.0;
                    for (int c = 0; c < d; ++c) {
                        if (kind == 0) {
                            double at_lo = bf(qh[c]) * bf(mj[c]);
                            double at_hi = bf(qh[c]) * bf(mj[d + c]);
                            s += at_lo > at_hi ? at_lo : at_hi;
                        } else {
                            s += bf(qh[c]) * bf(mj[c]);
                        }
                    }
                    best = s > best ? s : best;
                    total += s;
                }
                S[(int64_t)u * nblk_max + j] = agg == 0 ? best : total;
            }
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * O13  Layer-segmented prefill plan (Section 3.4): the prompt's layers are
 * run in consecutive batches, each injecting at most max_inject prompt
 * tokens (the maxInjectToken bound; a layer over T prompt tokens injects T).
 *   T <= max_inject: a batch runs s = floor(max_inject / T) whole layers
 *       (the last batch the remaining ones);
 *   T > max_inject: each layer is split into chunks of max_inject tokens
 *       (the last chunk shorter), one chunk per batch, layer after layer
 *       (the combination with chunked prefill).
 * Output: one item per (batch, layer, token range), in execution order:
 *   items[i] = {batch, layer, tok_begin, tok_end}.
 * Returns the number of items, or -1 for invalid arguments or when more
 * than cap items would be needed.
 * ---------------------------------------------------------------------- */
int64_t oracle_prefill_plan(int64_t T, int layers, int64_t max_inject, int32_t *items, int64_t cap)
{
    if (T <= 0 || layers <= 0 || max_inject <= 0)
        return -1;
    int64_t n = 0;
    if (T <= max_inject) {
        int64_t s = max_inject / T;
        for (int l = 0; l < layers; ++l) {
            if (n >= cap)
                return -1;
            items[4 * n + 0] = (int32_t)(l / s);
            items[4 * n + 1] = l;
            items[4 * n + 2] = 0;
            items[4 * n + 3] = (int32_t)T;
            ++n;
        }
    } else {
        int64_t chunks = (T + max_inject - 1) / max_inject;
        for (int l = 0; l < layers; ++l)
            for (int64_t c = 0; c < chunks; ++c) {
                if (n >= cap)
                    return -1;
                int64_t b = c * max_inject;
                int64_t e = b + max_inject < T ? b + max_inject : T;
                items[4 * n + 0] = (int32_t)(l * chunks + c);
                items[4 * n + 1] = l;
                items[4 * n + 2] = (int32_t)b;
                items[4 * n + 3] = (int32_t)e;
                ++n;
            }
    }
    return n;
}

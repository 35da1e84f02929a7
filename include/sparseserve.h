/*
 * sparseserve.h -- C ABI of the MI355X (gfx950) decode-step hot path of
 * SparseServe's dynamic sparse attention over a hierarchical HBM/DRAM KV
 * cache (arXiv 2509.24626).
 *
 * One decode step of one layer is:
 *   ss_score_topk        criticality of every KV block from its metadata and
 *                        top-k block selection per (sequence, KV head)
 *   ss_cache_resolve     the KV cache manager maps the selected blocks to
 *                        HBM cache slots and lists the misses (host side)
 *   ss_gather_blocks     one fused kernel loads every missed block record
 *                        from pinned, device-mapped DRAM into its slot
 *   ss_sparse_attention  attention of the decode query over the selected
 *                        blocks only
 * plus ss_build_metadata, run when blocks fill.
 *
 * Conventions for every call
 *   - Plain C types only.  `stream` is a hipStream_t passed as void*; NULL
 *     means the null stream.  GPU calls only enqueue work on `stream` and
 *     return without synchronising; host calls (ss_cache_*) are synchronous.
 *   - "device" pointers are GPU-accessible addresses: HBM allocations or the
 *     device address of pinned, mapped host memory (ss_host_alloc_mapped).
 *     "host" pointers are ordinary CPU memory.
 *   - The caller owns every buffer it passes.  The library owns only
 *     ss_cache handles and memory from ss_host_alloc_mapped.  No GPU call
 *     allocates memory; workspaces are passed in by the caller.
 *   - Arguments are validated before anything is enqueued; on failure the
 *     call returns a non-zero ss_status, enqueues nothing and sets a
 *     per-thread message readable with ss_last_error().  HIP launch errors
 *     return SS_ERR_HIP.  Nothing throws across this boundary.
 *   - Values read by a kernel from device arrays (lengths, selections,
 *     slots, miss entries) are range-checked by the kernel; out-of-range
 *     entries are skipped, never dereferenced.
 *
 * Shapes and notation: B sequences, Hq query heads, Hkv KV heads with
 * G = Hq / Hkv query heads per KV head (query head h uses KV head h / G),
 * d = head dim, blk = tokens per block, nblk_max = block capacity per
 * sequence in the metadata and score arrays, nblk[b] = blocks of sequence b,
 * k = blocks selected per (sequence, KV head).  A (sequence b, KV head g)
 * pair is a "unit" u = b * Hkv + g.
 * Supported: d == 128, blk in {8, 16, 32}, 1 <= G <= 16, 1 <= k,
 * nblk_max <= 65536; other values return SS_ERR_UNSUPPORTED.
 *
 * Block record (bf16, 2*blk*d*2 bytes; the KV cache block of one KV head,
 * Section 3.2's (H,N,D) layout: the tokens of one head are contiguous):
 *     K tile: blk rows of d channels, element (t, c) at bf16 index t*d + c
 *     V tile: channel-major, element (t, c) at bf16 index blk*d + c*blk + t
 * The channel-major V tile lets the attention kernel load V^T operand
 * fragments as 16-byte vectors.
 */
#ifndef SPARSESERVE_H
#define SPARSESERVE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int ss_status;
#define SS_OK 0
#define SS_ERR_INVALID_ARG 1 /* null pointer, negative size, inconsistent shape */
#define SS_ERR_UNSUPPORTED 2 /* outside the supported set above */
#define SS_ERR_CAPACITY 3    /* a unit selects more blocks than it has cache slots */
#define SS_ERR_OOM 4         /* host allocation failed, or a caller buffer is too small */
#define SS_ERR_HIP 5         /* a HIP runtime call or kernel launch failed */
#define SS_ERR_TIMEOUT 6     /* the host waited longer than its deadline for GPU work */

#define SS_ABI_VERSION 5

int ss_abi_version(void);
const char *ss_status_string(ss_status status);
/* Message of the last failing call on this thread ("" if none). */
const char *ss_last_error(void);

/* ---------------------------------------------------------------- memory
 * Pinned host memory mapped into the GPU's address space: the DRAM tier of
 * the KV cache that GPU kernels read directly over the host link
 * (Section 3.2.1, GPU-direct loading).
 * flags: 0 = coherent (fine-grained), 1 = non-coherent (coarse-grained).
 * On success *host_ptr is the CPU address and *dev_ptr the GPU address of
 * the same bytes.  Free with ss_host_free(host_ptr). */
ss_status ss_host_alloc_mapped(size_t bytes, unsigned flags, void **host_ptr, void **dev_ptr);
ss_status ss_host_free(void *host_ptr);

/* Measurement hook (not part of the method).  The next kernel that the
 * calling thread launches through this library -- the scoring, top-k,
 * gather, attention or metadata kernel of the next call that launches one;
 * for a split attention, its first kernel only -- records `start_event`
 * (may be NULL) when it starts executing and `stop_event` (may be NULL)
 * when it finishes, as hipExtLaunchKernel does: kernel execution time
 * without the queue's dispatch latency.  Events are hipEvent_t created by
 * the caller.  The setting is per thread and is consumed by that one
 * launch; ss_time_next_kernel(NULL, NULL) cancels it.  ss_decode_layer
 * attaches its gather timing events (see below) the same way.  Always
 * returns SS_OK. */
ss_status ss_time_next_kernel(void *start_event, void *stop_event);

/* --------------------------------------------------------------- metadata
 * Block metadata is the bounding cuboid of the block's keys: the
 * channel-wise minimum (lo) and maximum (hi) of K over the blk tokens
 * (Section 2.2; created when a block fills, Section 3.1).  Minimum and
 * maximum follow IEEE-754 totalOrder (-0 < +0), so every entry is one of the
 * input values.
 *   kv_base, unit_off: device; block j of unit u is the record at
 *       kv_base + unit_off[u] + j * record_bytes (unit_off: device int64
 *       [B*Hkv], byte offsets; kv_base may be HBM or mapped host memory)
 *   nblk: device int32 [B], clamped to [0, nblk_max]
 *   meta: device bf16 [B][Hkv][nblk_max][2][d]: lo[d] then hi[d]; entries
 *       with j >= nblk[b] are not written. */
ss_status ss_build_metadata(const void *kv_base, const int64_t *unit_off, const int32_t *nblk,
                            int B, int Hkv, int nblk_max, int blk, int d, void *meta, void *stream);

/* Metadata kinds and GQA aggregations of the scoring variants. */
#define SS_META_CUBOID 0 /* [lo, hi] per block, 2*d bf16 (ss_build_metadata) */
#define SS_META_MEAN 1   /* mean key per block, d bf16 (ss_build_metadata_mean) */
#define SS_AGG_MAX 0     /* a KV head's score: the largest of its query heads' scores */
#define SS_AGG_SUM 1     /* ... their sum (ranks as their mean does) */

/* Mean-key metadata, the variant the paper cites first in Section 2.2: per
 * block and channel, the mean of K over the blk tokens rounded once to the
 * nearest bf16 (ties to even).  The keys are summed in fp64 in token order,
 * which is exact unless a block's keys span more than about 2^40 in
 * magnitude, and scaled by 1/blk (exact).
 * Arguments as ss_build_metadata, except meta: device bf16
 * [B][Hkv][nblk_max][d] (4-byte aligned). */
ss_status ss_build_metadata_mean(const void *kv_base, const int64_t *unit_off, const int32_t *nblk, int B, int Hkv,
                                 int nblk_max, int blk, int d, void *meta, void *stream);

/* Metadata of either kind from keys in any layout: block j of unit u
 * starts at kv_base + unit_off[u] + j*block_stride, and its token t's d
 * keys at + t*row_stride (the V part is not read).  Block records are
 * block_stride = 2*blk*d*2, row_stride = d*2 (ss_build_metadata and
 * ss_build_metadata_mean call this); a token-major KV tensor [tokens][Hkv]
 * [2][d], e.g. a prompt's new KV during prefill, is block_stride =
 * blk*Hkv*2*d*2, row_stride = Hkv*2*d*2, unit_off[g] = g*2*d*2.  Strides
 * positive multiples of 16; kv_base, unit_off values and meta 16-byte
 * aligned.  meta layout as for meta_kind. */
ss_status ss_build_metadata_strided(const void *kv_base, const int64_t *unit_off, const int32_t *nblk, int B,
                                    int Hkv, int nblk_max, int blk, int d, int64_t block_stride, int64_t row_stride,
                                    int meta_kind, void *meta, void *stream);

/* ------------------------------------------------------ scoring, selection
 * Criticality of block j for KV head g of sequence b (Section 2.2, the dot
 * product of the query with the block metadata, taken as the largest value
 * q.k can reach inside the cuboid), maximised over the G query heads that
 * share g:
 *     S(b,g,j) = max_{h in group g} sum_c max(q[b,h,c]*lo[c], q[b,h,c]*hi[c])
 * computed with exact bf16 products and fp32 accumulation.
 *   q: device bf16 [B][Hq][d]; meta as produced by ss_build_metadata;
 *   nblk: device int32 [B]
 *   scores: device fp32 [B][Hkv][nblk_max]; entries j >= nblk[b] are not
 *       written. */
ss_status ss_score_blocks(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                          int nblk_max, int d, float *scores, void *stream);

/* Scoring variants (Section 2.2: the DSAs the paper cites differ in their
 * metadata; the dot product with the query is common to them):
 *   meta_kind SS_META_CUBOID: s_h(j) = sum_c max(q_h[c]*lo[c], q_h[c]*hi[c])
 *   meta_kind SS_META_MEAN:   s_h(j) = sum_c q_h[c] * m[c]  (mean key m)
 *   agg SS_AGG_MAX: S = max over the group's heads; SS_AGG_SUM: their sum.
 * meta in the layout of its kind; other arguments as ss_score_blocks, which
 * is the (SS_META_CUBOID, SS_AGG_MAX) case.  SS_ERR_INVALID_ARG for an
 * unknown kind or aggregation. */
ss_status ss_score_blocks_variant(const void *q, const void *meta, int meta_kind, int agg, const int32_t *nblk,
                                  int B, int Hq, int Hkv, int nblk_max, int d, float *scores, void *stream);

/* Top-k block selection per unit (Section 2.2: the k most critical blocks,
 * chosen per head).  Order: higher score first, equal scores -> lower block
 * index first (-0.0 and +0.0 are equal).  Output per unit: the first
 * min(k, nblk[b]) blocks in that order, listed in ascending block index,
 * then -1 padding.  Scores must not be NaN.
 *   scores: device fp32 [B][Hkv][nblk_max]; sel: device int32 [B][Hkv][k]. */
ss_status ss_select_topk(const float *scores, const int32_t *nblk, int B, int Hkv, int nblk_max, int k,
                         int32_t *sel, void *stream);

/* ss_score_blocks followed by ss_select_topk; `scores` is the caller's
 * fp32 [B][Hkv][nblk_max] buffer and holds the scores afterwards. */
ss_status ss_score_topk(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                        int nblk_max, int d, int k, float *scores, int32_t *sel, void *stream);
/* Bytes of the `scores` buffer ss_score_topk needs (B*Hkv*nblk_max fp32);
 * 0 for invalid shapes.  Host-only. */
size_t ss_score_topk_workspace(int B, int Hq, int Hkv, int nblk_max, int d, int k);

/* ------------------------------------------------------------ block cache
 * The HBM tier of the KV cache manager (Section 3.1): per unit, a region of
 * capacity[u] fixed-size block slots, managed per head; least-recently-used
 * eviction.  Host-side state only; the slots' bytes live in the caller's
 * HBM cache buffer at cache_base + region_off[u] + slot * record_bytes.
 * Not thread-safe per handle; use one handle per layer.
 *   nblk: host int32 [B] blocks per sequence; capacity: host int32 [B*Hkv]
 *   (>= 0).  Regions are laid out unit after unit. */
typedef struct ss_cache ss_cache;
ss_status ss_cache_create(int B, int Hkv, const int32_t *nblk, const int32_t *capacity, size_t record_bytes,
                          ss_cache **out);
void ss_cache_destroy(ss_cache *cache);
/* total slots over all units (the HBM cache holds total * record_bytes) */
int64_t ss_cache_total_slots(const ss_cache *cache);
/* off: host int64 [B*Hkv], byte offset of each unit's region */
ss_status ss_cache_region_offsets(const ss_cache *cache, int64_t *off);
/* Host threads used by ss_cache_resolve (default: half the CPUs the process may run on, at most 8). */
ss_status ss_cache_set_threads(ss_cache *cache, int n_threads);
/* New block counts after sequences grew (a block fills when its last token
 * is appended, Section 3.1): nblk host int32 [B], each >= the current
 * count (SS_ERR_INVALID_ARG otherwise).  Capacities and cached blocks are
 * unchanged; the new blocks start uncached.  Each unit's host block table
 * keeps room for max(16, nblk/8) more blocks; within it the call costs
 * O(B*Hkv), beyond it the table is laid out again (O(total blocks), once
 * per such growth). */
ss_status ss_cache_set_blocks(ss_cache *cache, const int32_t *nblk);

/* Resolve one step's selection.  Per unit, with sel[u][*] strictly
 * ascending then -1 padded:
 *   1. every selected block already cached (a hit) gets last_use = step;
 *   2. every other selected block (a miss), in ascending block order, takes
 *      the lowest-numbered empty slot, else the slot whose block is not
 *      selected in this call and has the smallest last_use (ties: lowest
 *      slot), evicting that block; the slot gets last_use = step.
 *   sel: host int32 [B][Hkv][k]
 *   slots: host int32 [B][Hkv][k], the slot of each selected block (-1 for
 *       -1 entries)
 *   miss: host int32 [miss_cap][4] rows (b, g, block, slot), units in order,
 *       ascending block within a unit; *n_miss rows are written.
 * Errors (state unchanged): SS_ERR_INVALID_ARG for a malformed selection,
 * SS_ERR_CAPACITY if a unit selects more blocks than it has slots,
 * SS_ERR_OOM if miss_cap rows are not enough. */
ss_status ss_cache_resolve(ss_cache *cache, int64_t step, const int32_t *sel, int k, int32_t *slots,
                           int32_t *miss, int64_t miss_cap, int64_t *n_miss);
/* ss_cache_resolve restricted to sequences [b_begin, b_end): sel and slots
 * point at the rows of sequence b_begin ([b_end-b_begin][Hkv][k]); miss rows
 * carry absolute (b, g).  Other sequences are untouched, so a step can be
 * resolved in several calls over disjoint ranges with the same step number. */
ss_status ss_cache_resolve_range(ss_cache *cache, int64_t step, int b_begin, int b_end, const int32_t *sel, int k,
                                 int32_t *slots, int32_t *miss, int64_t miss_cap, int64_t *n_miss);
/* State dump for tests: per slot (units in order) the block it holds (-1
 * empty) and its last use.  Arrays hold ss_cache_total_slots entries. */
ss_status ss_cache_export(const ss_cache *cache, int32_t *slot_block, int64_t *slot_last);

/* ------------------------------------------------ block cache on the GPU
 * The same per-unit LRU as ss_cache (identical slots and misses for the
 * same selections), with its state in HBM and its resolve a kernel, so that
 * a decode step needs no host round trip (ss_decode_layer_dev).  Supported:
 * capacities up to 8192 slots per unit, k up to 512, steps in [0, 2^31)
 * and not decreasing.
 *   table_room: host int32 [B], the most blocks each sequence can reach
 *       (block indices below it); capacity: host int32 [B*Hkv]
 * Creation allocates the state in device memory (one hipMalloc) and waits
 * for its initialisation on `stream`; the resolve allocates nothing. */
typedef struct ss_dev_cache ss_dev_cache;
ss_status ss_dev_cache_create(int B, int Hkv, const int32_t *table_room, const int32_t *capacity, void *stream,
                              ss_dev_cache **out);
void ss_dev_cache_destroy(ss_dev_cache *cache);
int64_t ss_dev_cache_total_slots(const ss_dev_cache *cache);
/* Resolves sequences [b_begin, b_end) on `stream` with the rules of
 * ss_cache_resolve.  sel: device int32 [b_end-b_begin][Hkv][k] (the rows of
 * sequence b_begin on); nblk: device int32 [B]; slots: device int32, same
 * shape as sel; miss: device int32 [B*Hkv][k][4]: unit u's miss rows (b, g,
 * block, slot), ascending by block, at row u*k, their number kept in the
 * cache (ss_dev_cache_miss_counts).  A malformed selection or one larger
 * than the unit's capacity leaves that unit unchanged, writes -1 slots and
 * no misses, and raises a flag that ss_dev_cache_miss_counts reports (1:
 * malformed, 2: capacity). */
ss_status ss_dev_cache_resolve(ss_dev_cache *cache, int64_t step, int b_begin, int b_end, const int32_t *sel, int k,
                               const int32_t *nblk, int32_t *slots, int32_t *miss, void *stream);
/* Waits for the device, then copies the last resolve's miss count per unit
 * (host int32 [B*Hkv]) and, if error_flags is not NULL, the error flags
 * raised so far. */
ss_status ss_dev_cache_miss_counts(const ss_dev_cache *cache, int32_t *counts, int32_t *error_flags);
/* State dump for tests, as ss_cache_export (waits for the device). */
ss_status ss_dev_cache_export(const ss_dev_cache *cache, int32_t *slot_block, int64_t *slot_last);
/* Waits for the device; *total = misses over every resolve so far. */
ss_status ss_dev_cache_total_misses(const ss_dev_cache *cache, int64_t *total);

/* ----------------------------------------------------------------- gather
 * FlashH2D-style loading (Section 3.2.1): one kernel copies every missed
 * block record from the DRAM pool into its HBM cache slot:
 *     cache_base + cache_off[u] + slot*record_bytes
 *         <- pool_base + pool_off[u] + block*record_bytes,   u = b*Hkv + g
 * for each row (b, g, block, slot) of `miss`.
 *   miss: device (or mapped host) int32 [n_miss][4]
 *   pool_base: device address of the pool (mapped host memory or HBM)
 *   pool_off, cache_off: device int64 [B*Hkv] byte offsets
 *   nblk: device int32 [B]; capacity: device int32 [B*Hkv]
 * Rows with b, g, block or slot out of range are skipped. */
ss_status ss_gather_blocks(const int32_t *miss, int64_t n_miss, const void *pool_base, const int64_t *pool_off,
                           void *cache_base, const int64_t *cache_off, const int32_t *nblk,
                           const int32_t *capacity, int B, int Hkv, size_t record_bytes, void *stream);

/* ------------------------------------------------------ sparse attention
 * Attention of each sequence's decode query over the tokens of its selected
 * blocks only (Section 2.1's S = QK^T/sqrt(d), P = softmax(S), O = PV,
 * restricted as in Section 2.2):
 *     z_t = scale * q[b,h] . K_t,  p = softmax(z),  out[b,h] = sum_t p_t V_t
 * over the tokens t of the records at kv_base + region_off[u] +
 * slots[u][i]*record_bytes, i < k.  An entry is skipped (never read) if it
 * is < 0, >= slot_limit, or >= capacity[u] when `capacity` is given, so a
 * unit reads only its own region even when the units' slot counts differ.
 * With no token the output is 0.  fp32 accumulation; the probabilities
 * enter the PV product as a bf16 hi/lo pair, so they are carried to about
 * 16 significant bits.
 *   q: device bf16 [B][Hq][d]; region_off: device int64 [B*Hkv];
 *   slots: device int32 [B][Hkv][k]; out: device fp32 [B][Hq][d]
 *   capacity: device int32 [B*Hkv], the slots of each unit's region (the
 *   block cache's capacities), or NULL to bound every unit by slot_limit
 *   slot_limit: the largest slot count of any unit (slot_limit records
 *   must span less than 2 GiB; SS_ERR_UNSUPPORTED otherwise)
 *   workspace: device, at least ss_sparse_attention_workspace(...) bytes
 *   (the call fails with SS_ERR_OOM if ws_bytes is smaller).
 * All-HBM layouts pass slots = the selection, region_off = the units'
 * block arrays, capacity = NULL and slot_limit = nblk_max. */
size_t ss_sparse_attention_workspace(int B, int Hq, int Hkv, int d, int blk, int k);
ss_status ss_sparse_attention(const void *q, const void *kv_base, const int64_t *region_off, const int32_t *slots,
                              const int32_t *capacity, int32_t slot_limit, int B, int Hq, int Hkv, int d, int blk,
                              int k, float scale, float *out, void *workspace, size_t ws_bytes, void *stream);

/* ss_sparse_attention without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The split partials go to a static
 * device array of 9 MiB that the library holds on each GPU it runs on until
 * the process ends; every supported shape fits it (SS_ERR_OOM otherwise).
 * The first call on a device looks the array up (hipGetSymbolAddress);
 * no call allocates or frees memory.  All calls on one GPU share the array,
 * so calls that overlap on one GPU (on different streams, or from several
 * threads) race and must be serialised by the caller; every partial a call
 * reads is written by that call first, so nothing carries over between
 * calls.  Arguments and results as ss_sparse_attention. */
ss_status ss_sparse_attention_static(const void *q, const void *kv_base, const int64_t *region_off,
                                     const int32_t *slots, const int32_t *capacity, int32_t slot_limit, int B,
                                     int Hq, int Hkv, int d, int blk, int k, float scale, float *out, void *stream);

/* ------------------------------------------------------ appending tokens
 * The decode step's new KV (Section 3.2.2: each layer's new KV tensor, one
 * token per sequence and KV head, goes into the free slot of the
 * sequence's open block in HBM) and the metadata of a block that fills
 * (Section 3.1).  Sequence b's token is token len[b] of the sequence: block
 * j = len[b] / blk, row p = len[b] % blk of the open record.
 *   new_kv: device bf16 [B][Hkv][2][d], K then V of each (sequence, head)
 *   len_dev: device int32 [B] tokens before the append; advanced by 1
 *   nblk_dev: device int32 [B] full blocks; set to j + 1 when block j fills
 *   open_blocks: device [B][Hkv] block records (2*blk*d bf16 each: K tile
 *       row-major, V tile channel-major); row / column p is written
 *   meta, meta_kind: on a fill, block j's metadata of that kind:
 *       SS_META_CUBOID, meta bf16 [B][Hkv][nblk_max][2][d]: lo/hi
 *       (channel-wise min/max of the record's K rows, IEEE totalOrder);
 *       SS_META_MEAN, meta bf16 [B][Hkv][nblk_max][d]: the mean key, as
 *       ss_build_metadata_mean computes it
 *   overflow: device int32 or NULL; set to 1 if a block fills at
 *       j >= nblk_max (its metadata is then not written and nblk_dev not
 *       advanced; the token is still written and len_dev advanced)
 * Buffers 4-byte aligned.  d must be 128, blk 8, 16 or 32.  One kernel on
 * `stream`, one workgroup per sequence. */
ss_status ss_append_kv(const void *new_kv, int32_t *len_dev, int32_t *nblk_dev, int B, int Hkv, int blk, int d,
                       int nblk_max, void *open_blocks, void *meta, int meta_kind, int32_t *overflow,
                       void *stream);

/* ------------------------------------------------------ FlashD2H saving
 * CPU-assisted saving of new tokens to the DRAM pool (Section 3.2.2): the
 * contiguous new-KV tensor is copied to pinned host staging memory on the
 * caller's stream (in chunks of consecutive token rows when it is large),
 * and this library's host threads place each token in its block record in
 * the pool (the same record layout), each chunk as soon as its copy has
 * landed.  The GPU's compute units take no part.
 *   pool_host: host address of the pool; block j of unit u = b*Hkv + g is
 *       the record at pool_host + pool_off[u] + j*record_bytes
 *   pool_off: host int64 [B*Hkv]; pool_blocks: host int32 [B] records the
 *       pool holds per unit of sequence b (both copied)
 *   max_new_tokens: largest n_new of ss_kv_save
 *   staging_slots: pinned staging buffers, used in turn (1..64); a save
 *       whose buffer is still being scattered waits for it
 *   threads: host threads that scatter (1..64); they start now
 * The saver owns its staging memory, events and threads. */
typedef struct ss_kv_saver ss_kv_saver;
ss_status ss_kv_saver_create(int B, int Hkv, int blk, int d, void *pool_host, const int64_t *pool_off,
                             const int32_t *pool_blocks, int max_new_tokens, int staging_slots, int threads,
                             ss_kv_saver **out);
/* Waits for the saves in flight, then frees everything. */
void ss_kv_saver_destroy(ss_kv_saver *saver);
/* Saves n_new tokens per sequence: new_kv device bf16
 * [B][n_new][Hkv][2][d]; token i of sequence b is token len[b] + i of the
 * sequence (len: host int32 [B], copied).  Enqueues the copy on `stream`
 * and returns; the scatter runs when the copy has finished.  new_kv must
 * stay unchanged until the copy has run (stream order).  SS_ERR_INVALID_ARG
 * if a token lies past its unit's pool blocks.  Not thread-safe per saver. */
ss_status ss_kv_save(ss_kv_saver *saver, const void *new_kv, int n_new, const int32_t *len, void *stream);
/* Points the saver at other records of the pool (e.g. the next layer's
 * during a layer-segmented prefill): pool_off host int64 [B*Hkv],
 * pool_blocks host int32 [B], copied.  Saves already issued keep the
 * records they were issued for; the staging memory and threads are kept. */
ss_status ss_kv_saver_retarget(ss_kv_saver *saver, const int64_t *pool_off, const int32_t *pool_blocks);
/* Blocks until every save so far is in the pool; returns the first error
 * met by the asynchronous part (SS_ERR_HIP). */
ss_status ss_kv_save_wait(ss_kv_saver *saver);

/* ------------------------------------------- working sets, batch control
 * Working-set-aware batch size control (Section 3.3).  A decoding
 * request's working set is, per (layer, KV head), the union of the blocks
 * selected over its last `window` observed decoding steps (Section 3.3
 * uses 12), times record_bytes; the tracker follows it incrementally.
 * Requests are named by caller-chosen int64 ids.  Host-only; not
 * thread-safe per tracker. */
typedef struct ss_ws ss_ws;
/* window: 1..255 observations */
ss_status ss_ws_create(int layers, int Hkv, int window, size_t record_bytes, ss_ws **out);
void ss_ws_destroy(ss_ws *ws);
/* One decoding step of one layer for a batch: req_ids host int64 [B]
 * (distinct); sel host int32 [B][Hkv][k] (-1 entries ignored; block
 * indices below 2^24).  k must be the same in every call.  Steps of a
 * (request, layer) must increase (SS_ERR_INVALID_ARG otherwise, nothing
 * recorded).  Unknown ids start a history. */
ss_status ss_ws_observe(ss_ws *ws, int layer, int64_t step, const int64_t *req_ids, int B, const int32_t *sel,
                        int k);
/* bytes[i] = working set of request req_ids[i]: record_bytes times the sum
 * over (layer, head) of its union size; a (layer, head) with no
 * observation yet counts fallback_blocks[i] blocks (NULL: 0), e.g. one
 * step's selection, min(k, blocks), for a request that just left
 * prefill. */
ss_status ss_ws_decode_bytes(const ss_ws *ws, const int64_t *req_ids, int n, const int32_t *fallback_blocks,
                             int64_t *bytes);
/* Drops a request's history (finished or reset). */
ss_status ss_ws_forget(ss_ws *ws, int64_t req_id);
/* A prefill request's working set (exact): layer-segmented prefill needs
 * one layer of the prompt's KV, ceil(prompt/blk) blocks per KV head;
 * chunked prefill the KV of every chunk so far in every layer,
 * ceil(min(prompt, done + chunk)/blk) blocks per KV head and layer.
 * Returns bytes, or -1 for invalid arguments. */
int64_t ss_ws_prefill_bytes(int64_t prompt_tokens, int64_t done_tokens, int64_t chunk_tokens, int layers, int Hkv,
                            int blk, size_t record_bytes, int layer_segmented);
/* Algorithm 1 (Section 3.3): walks the initial batch in its order and
 * admits request i (admit[i] = 1) if the working sets admitted so far plus
 * ws_bytes[i] stay within m_avl, else resets it (admit[i] = 0).
 * ws_bytes host int64 [n] (>= 0); *m_used = bytes admitted. */
ss_status ss_schedule_batch(const int64_t *ws_bytes, int n, int64_t m_avl, int32_t *admit, int64_t *m_used);

/* ------------------------------------------------ layer-segmented prefill
 * The plan of a layer-segmented prefill (Section 3.4): a prompt of T
 * tokens runs its `layers` layers in consecutive batches, each injecting at
 * most max_inject prompt tokens (maxInjectToken; a layer over the prompt
 * injects T).  If T <= max_inject a batch runs floor(max_inject / T) whole
 * layers; otherwise every layer is split into chunks of max_inject tokens
 * (the last shorter), one chunk per batch (the combination with chunked
 * prefill).  items: host int32 [cap][4] rows (batch, layer, tok_begin,
 * tok_end) in execution order; *n_items rows written.  SS_ERR_OOM if cap
 * rows are not enough, SS_ERR_INVALID_ARG for non-positive arguments. */
ss_status ss_prefill_plan(int64_t T, int layers, int64_t max_inject, int32_t *items, int64_t cap, int64_t *n_items);

/* ------------------------------------------------------- one layer's step
 * The decode step of one layer over the HBM/DRAM hierarchy (Section 3.1's
 * executor / cache-manager exchange): score and select on the GPU, copy the
 * selection to the host, resolve it in the block cache, copy slots and the
 * miss list back, gather the misses, attend.
 * The batch is processed in `parts` consecutive sequence groups (1 <= parts
 * <= B; 0 means 1) -- equal groups, or group p = sequences
 * [part_end[p-1], part_end[p]) when part_end (host int32 [parts], strictly
 * increasing, last = B) is given -- so that the host-link gather of one
 * group overlaps the
 * scoring and the host resolve of the next: scoring, selection and
 * attention run on `stream`; the gathers run on two transfer streams the
 * library creates once per device (default priority; groups alternate
 * between them) and orders against `stream` with events.  Calls of
 * ss_decode_layer take turns on a process-wide lock (they share those
 * streams).  Selections reach the host, and
 * slots and miss rows reach the GPU, through the mapped host buffers (no
 * copy-engine transfers).  The host waits only for each group's selection;
 * everything after the last resolve is enqueued and the call returns
 * without waiting.  Work enqueued later on `stream` is ordered after the
 * whole step.
 * All pointers below are caller-owned.  Device buffers: scores fp32
 * [B][Hkv][nblk_max]; sel_dev and slots_dev int32 [B][Hkv][k]; miss_dev
 * int32 [miss_cap][4] (16-byte aligned); attn_ws of attn_ws_bytes >= the
 * largest ss_sparse_attention_workspace(...) of a group.  Host buffers
 * (pinned, mapped, coherent: ss_host_alloc_mapped with flags 0): sel_host,
 * slots_host int32 [B][Hkv][k]; miss_host int32 [miss_cap][4];
 * miss_cap >= B*Hkv*k; SS_ERR_INVALID_ARG if they are not mapped.
 * slot_limit: the largest per-unit capacity; attention reads no slot at or
 * above a unit's own capacity_dev entry.  cache_off_dev = ss_cache_region_offsets, copied to the device.
 * After the call, miss_host rows [0, *n_miss) hold the step's misses in
 * unit order (as one ss_cache_resolve would list them).
 * events: NULL, or 7*parts hipEvent_t (any entry may be NULL); for group p,
 * events[7p+0..2] are recorded on `stream` before scoring, after scoring
 * and after selection, events[7p+3..4] are attached to the gather kernel
 * itself (its start and end of execution, as ss_time_next_kernel does), and
 * events[7p+5..6] are recorded on `stream` before and after attention.
 * Streams and events are created for the device current at the call.
 * On error nothing further is enqueued; a resolve error or a wait past the
 * deadline (ss_set_host_wait_timeout) leaves the cache unchanged for the
 * groups not yet resolved. */
typedef struct ss_layer_buffers {
    int B, Hq, Hkv, d, blk, nblk_max, k;
    float scale;
    const void *meta;           /* device bf16 metadata in meta_kind's layout */
    const int32_t *nblk_dev;    /* device int32 [B] */
    const void *pool;           /* device address of the DRAM pool */
    const int64_t *pool_off_dev; /* device int64 [B*Hkv] */
    ss_cache *cache;
    void *cache_base;           /* HBM cache, ss_cache_total_slots records */
    const int64_t *cache_off_dev; /* device int64 [B*Hkv] */
    const int32_t *capacity_dev;  /* device int32 [B*Hkv] */
    int32_t slot_limit;
    float *scores;
    int32_t *sel_dev, *slots_dev, *miss_dev;
    int32_t *sel_host, *slots_host, *miss_host;
    int64_t miss_cap;
    void *attn_ws;
    size_t attn_ws_bytes;
    int parts;
    const int32_t *part_end;    /* host int32 [parts] or NULL */
    int meta_kind;              /* SS_META_CUBOID or SS_META_MEAN (layout of meta) */
    int agg;                    /* SS_AGG_MAX or SS_AGG_SUM */
} ss_layer_buffers;

ss_status ss_decode_layer(const ss_layer_buffers *L, int64_t step, const void *q, float *out, void *stream,
                          void *const *events, int64_t *n_miss);

/* Deadline of ss_decode_layer's host waits for a group's selection, in
 * milliseconds, for every thread of the process (default 10000; ms <= 0
 * restores it).  When a wait passes it, the call returns SS_ERR_TIMEOUT
 * with the group and step in ss_last_error(): the work already enqueued
 * stays enqueued and the block cache is unchanged for the groups not yet
 * resolved, so the caller synchronises the device before going on. */
ss_status ss_set_host_wait_timeout(int64_t ms);

/* The decode step with the resolve on the GPU (ss_dev_cache, which takes
 * the place of L->cache; the host buffers sel_host, slots_host and
 * miss_host are not used).  The first group's scoring, top-k, resolve,
 * gather and attention run in order on `stream`.  Each later group's
 * scoring, top-k and resolve run on a compute stream the library creates
 * once per device (default priority).  A middle group's gather runs on a
 * transfer stream behind its resolve and its attention on the compute
 * stream behind the gather; the last group's gather runs on `stream`, with
 * its attention right behind it.  Everything is ordered after the work
 * already on `stream`, and `stream` waits for the compute stream at the end,
 * so work enqueued on `stream` afterwards sees the whole step.  The host
 * enqueues the step and returns without waiting; the misses are counted in
 * the cache (ss_dev_cache_miss_counts).  L->miss_dev holds each unit's miss
 * rows at row u*k.  Attentions of two groups run at once, so with three
 * groups or more L->attn_ws_bytes must hold two regions, each the largest
 * ss_sparse_attention_workspace of a group rounded up to 256 bytes
 * (SS_ERR_OOM otherwise).  events as for ss_decode_layer, except that
 * events[7p+0..2] are recorded on the stream that runs group p's scoring
 * (events[7p+2] after the resolve), events[7p+5..6] on the stream that runs
 * its attention, and the last group's events[7p+6] on `stream` once the
 * whole step is done.  The block cache's regions must be laid out as
 * ss_cache_region_offsets gives them for the same capacities. */
ss_status ss_decode_layer_dev(const ss_layer_buffers *L, ss_dev_cache *cache, int64_t step, const void *q,
                              float *out, void *stream, void *const *events);

/* The decode step of n_layers layers with the resolve on the GPU, the
 * sequence groups pipelined across layers (Section 3.1's executor / cache
 * manager exchange, layer after layer).  A sequence's attention reads only
 * its own blocks, and its next layer depends only on its own output of this
 * one, so group p (the groups of layers[0], the same in every layer) runs
 * score, top-k, resolve, gather and attention of layer 0, then of layer 1,
 * ..., in order on one stream: group 0 on `stream`, groups 1..3 on streams
 * the library creates once per device (default priority), group p > 3
 * behind group p mod 4 on its stream.  Group p's layer l+1 therefore starts
 * as soon as its layer l is attended, beside the other groups' gathers of
 * layer l.  Everything is ordered after the work already on `stream`, and
 * `stream` waits for every group stream at the end (also after an error, so
 * that a synchronisation sees all that was enqueued).  The host enqueues the
 * whole step and returns without waiting.
 *   layers, caches, q, out: host arrays [n_layers]; layer l is decoded with
 *       layers[l] and caches[l] (as ss_decode_layer_dev), its queries q[l]
 *       (device bf16 [B][Hq][d]) and its output out[l] (device fp32
 *       [B][Hq][d]).  Every layer has the same B, Hq, Hkv, d and k; each
 *       layers[l]->attn_ws_bytes must hold min(groups, 4) regions of the
 *       largest ss_sparse_attention_workspace of a group, each rounded up to
 *       256 bytes (SS_ERR_OOM otherwise).
 *   between: NULL, or a callback the call makes on the calling thread,
 *       while enqueueing, for every layer l < n_layers-1 and group p: after
 *       group p's layer-l attention is enqueued and before its layer-(l+1)
 *       scoring, with the group's sequences [b_begin, b_end) and its stream.
 *       The caller enqueues on that stream the work that turns the group's
 *       rows of out[l] into its rows of q[l+1] (the rest of the model's layer)
 *       and returns SS_OK; any other value stops the call with that status.
 *       It must not call ss_decode_layer, ss_decode_layer_dev,
 *       ss_decode_step_dev or ss_decode_step (they return SS_ERR_INVALID_ARG
 *       there: the step holds their lock).  With NULL the queries are taken as they are.
 *   events: NULL, or 2*n_layers*groups hipEvent_t (any entry may be NULL):
 *       events[2*(l*groups+p)+0..1] are attached to group p's layer-l gather
 *       kernel itself (start and end of its execution).
 * On error the calls already enqueued stay enqueued. */
typedef ss_status (*ss_between_fn)(void *ctx, int layer, int b_begin, int b_end, void *stream);
ss_status ss_decode_step_dev(const ss_layer_buffers *const *layers, ss_dev_cache *const *caches, int n_layers,
                             int64_t step, const void *const *q, float *const *out, void *stream,
                             ss_between_fn between, void *ctx, void *const *events);

/* The step of n_layers layers with the groups pipelined across layers as in
 * ss_decode_step_dev, with each layer's slot table resolved on host threads
 * (layers[l]->cache, as ss_decode_layer; Section 3.1's cache manager on the
 * CPU).  Each group's scoring and top-k run on the group's stream and leave
 * the selection in the layer's mapped sel_host rows as well; the host takes
 * the (layer, group) pairs in order, waits for the pair's selection (with
 * the deadline of ss_set_host_wait_timeout), resolves it into the layer's
 * mapped slots_host and miss_host rows (the layer's miss rows kept compact
 * in group order), and enqueues on the group's stream the gather (in the
 * link order of ss_decode_step_dev; it also copies the group's slots to
 * slots_dev), the attention, the between-layer callback and the next
 * layer's scoring and top-k.  The call returns once everything is enqueued;
 * `stream` waits for every group stream at the end.
 *   layers, q, out, between, ctx, events: as ss_decode_step_dev; each layer
 *       needs the buffers ss_decode_layer needs and an attention workspace of
 *       min(groups, 4) regions as ss_decode_step_dev.
 *   n_miss: NULL or host int64 [n_layers], each layer's missed blocks.
 * On error the calls already enqueued stay enqueued; the slot tables of the
 * (layer, group) pairs not yet resolved are unchanged. */
ss_status ss_decode_step(const ss_layer_buffers *const *layers, int n_layers, int64_t step, const void *const *q,
                         float *const *out, void *stream, ss_between_fn between, void *ctx, void *const *events,
                         int64_t *n_miss);

#ifdef __cplusplus
}
#endif
#endif /* SPARSESERVE_H */

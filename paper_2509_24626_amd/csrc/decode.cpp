// One layer's decode step over the HBM/DRAM hierarchy: the model executor
// selects blocks on the GPU and hands the indices to the KV cache manager,
// which resolves them against the HBM block cache and loads the misses
// from DRAM in one fused gather (Section 3.1, Section 3.2.1); attention
// then reads only HBM.
//
// The batch runs as a pipeline over sequence groups.  Scoring and
// selection of every group are enqueued up front on the caller's stream;
// the top-k kernel writes each selection both to HBM and straight into
// pinned, mapped host memory.  The host then takes the groups in order:
// wait for the group's selection, resolve it, and enqueue its gather on the
// transfer stream (the kernel reads the miss rows from mapped host memory
// and also copies the group's slot table to HBM) and its attention on the
// caller's stream behind that gather.  So the host-link transfer of group p
// overlaps the resolve of group p+1 and the scoring still in flight, and
// attention of group p overlaps the gather of group p+1.  Groups alternate
// between two transfer streams, so a group's gather starts while the
// previous one drains (no launch gap, no idle tail on the link).  Every hand-off is
// a kernel on a compute queue: no copy-engine transfer, whose cross-engine
// synchronisation costs tens of microseconds per hand-off, is on the path.
#include <atomic>
#include <chrono>
#include <mutex>
#include <new>
#include <thread>
#include <unordered_map>
#include <vector>

#include "internal.hpp"

namespace ss {
ss_status launch_topk(const float *scores, const int32_t *nblk, int B, int Hkv, int nblk_max, int k, int32_t *sel,
                      int32_t *mirror, hipStream_t s);
ss_status launch_gather(const int32_t *miss, int64_t n_miss, const void *pool_base, const int64_t *pool_off,
                        void *cache_base, const int64_t *cache_off, const int32_t *nblk, const int32_t *capacity,
                        int B, int Hkv, size_t record_bytes, const int32_t *copy_src, int32_t *copy_dst,
                        int64_t copy_n, hipStream_t s);
int cache_batch(const ss_cache *c);
int cache_kv_heads(const ss_cache *c);
int dev_cache_batch(const ss_dev_cache *c);
int dev_cache_kv_heads(const ss_dev_cache *c);
int32_t *dev_cache_counts(ss_dev_cache *c);
ss_status dev_cache_check_step(ss_dev_cache *c, int64_t step, int k);
ss_status dev_cache_launch(ss_dev_cache *c, int64_t step, int b_begin, int b_end, const int32_t *sel, int k,
                           const int32_t *nblk, int32_t *slots, int32_t *miss, hipStream_t s);
ss_status launch_gather_units(const int32_t *rows, const int32_t *counts, int u0, int u1, int k,
                              const void *pool_base, const int64_t *pool_off, void *cache_base,
                              const int64_t *cache_off, const int32_t *nblk, const int32_t *capacity, int B, int Hkv,
                              size_t record_bytes, hipStream_t s);
}  // namespace ss

namespace {

// Transfer streams and synchronisation events, one set per device for the
// whole process (every layer's cache handle shares them; decode-step calls
// take turns under g_exec_mu).  A set per handle would multiply streams over
// the few hardware queues, and a transfer stream sharing a queue with the
// caller's stream would serialise the pipeline.
struct exec_state {
    hipStream_t xfer[2] = {nullptr, nullptr};  // groups alternate between them
    hipStream_t comp = nullptr;                // device resolve: scoring chain of groups after the first
    hipEvent_t start = nullptr;
    hipEvent_t comp_done = nullptr;  // device resolve: the attentions on the compute stream are done
    std::vector<hipEvent_t> sel_ready, gathered;
    std::vector<hipEvent_t> link_order;  // multi-layer steps: one per (layer, group) gather
    std::vector<hipEvent_t> step_sel;    // multi-layer step, host resolve: one per (layer, group) selection
};

// Grows `v` to n events (disable-timing).
ss_status grow_events(std::vector<hipEvent_t> &v, int64_t n, const char *who)
{
    while ((int64_t)v.size() < n) {
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess)
            return ss::fail(SS_ERR_HIP, "%s: create event", who);
        try {
            v.push_back(e);
        } catch (const std::bad_alloc &) {
            (void)hipEventDestroy(e);
            return ss::fail(SS_ERR_OOM, "%s: out of memory", who);
        }
    }
    return SS_OK;
}

std::mutex g_exec_mu;
// set on the thread running ss_decode_step_dev's between-layer callback: the
// step calls hold g_exec_mu, so a step call from inside the callback is refused
thread_local bool t_in_callback = false;
std::unordered_map<int, exec_state *> g_exec;  // by device

ss_status hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "ss_decode_layer: %s: %s", what, hipGetErrorString(e));
    return SS_OK;
}

// called with g_exec_mu held
ss_status get_exec(int parts, exec_state **out)
{
    int dev = 0;
    ss_status st;
    if ((st = hip_check(hipGetDevice(&dev), "hipGetDevice"))) return st;
    exec_state *&e = g_exec[dev];
    if (!e) {
        exec_state *n = new (std::nothrow) exec_state;
        if (!n) return ss::fail(SS_ERR_OOM, "ss_decode_layer: out of memory");
        if ((st = hip_check(hipStreamCreateWithFlags(&n->xfer[0], hipStreamNonBlocking), "create transfer stream")) ||
            (st = hip_check(hipStreamCreateWithFlags(&n->xfer[1], hipStreamNonBlocking), "create transfer stream")) ||
            (st = hip_check(hipEventCreateWithFlags(&n->start, hipEventDisableTiming), "create event"))) {
            for (hipStream_t x : n->xfer)
                if (x) (void)hipStreamDestroy(x);
            if (n->start) (void)hipEventDestroy(n->start);
            delete n;
            return st;
        }
        e = n;
    }
    while ((int)e->sel_ready.size() < parts) {
        hipEvent_t a = nullptr, b = nullptr;
        if ((st = hip_check(hipEventCreateWithFlags(&a, hipEventDisableTiming), "create event"))) return st;
        if ((st = hip_check(hipEventCreateWithFlags(&b, hipEventDisableTiming), "create event"))) {
            (void)hipEventDestroy(a);
            return st;
        }
        try {
            e->sel_ready.reserve(e->sel_ready.size() + 1);
            e->gathered.reserve(e->gathered.size() + 1);
        } catch (const std::bad_alloc &) {
            (void)hipEventDestroy(a);
            (void)hipEventDestroy(b);
            return ss::fail(SS_ERR_OOM, "ss_decode_layer: out of memory");
        }
        e->sel_ready.push_back(a);
        e->gathered.push_back(b);
    }
    *out = e;
    return SS_OK;
}

// Looked up on every call (cheap): a cached translation could outlive the
// host buffer it was taken for.
ss_status device_address(void *host, void **dev)
{
    void *d = nullptr;
    if (hipHostGetDevicePointer(&d, host, 0) != hipSuccess || !d) {
        (void)hipGetLastError();
        return ss::fail(SS_ERR_INVALID_ARG, "ss_decode_layer: a host buffer is not pinned, mapped memory");
    }
    *dev = d;
    return SS_OK;
}

constexpr int64_t kDefaultWaitMs = 10000;
std::atomic<int64_t> g_wait_ms{kDefaultWaitMs};

// Polls until group p's selection is in host memory; a kernel that never
// finishes makes the call fail after the deadline instead of spinning (and
// holding g_exec_mu) for ever.
ss_status wait_host(hipEvent_t ev, int p, int64_t step)
{
    const int64_t ms = g_wait_ms.load(std::memory_order_relaxed);
    const auto deadline = std::chrono::steady_clock::now() + std::chrono::milliseconds(ms);
    for (;;) {
        hipError_t r = hipEventQuery(ev);
        if (r == hipSuccess) return SS_OK;
        if (r != hipErrorNotReady) return hip_check(r, "wait for a selection");
        if (std::chrono::steady_clock::now() > deadline)
            return ss::fail(SS_ERR_TIMEOUT, "ss_decode_layer: the selection of group %d at step %lld was not ready "
                            "after %lld ms", p, (long long)step, (long long)ms);
        std::this_thread::yield();
    }
}

ss_status record(void *const *events, int i, hipStream_t s)
{
    if (!events || !events[i]) return SS_OK;
    return hip_check(hipEventRecord(reinterpret_cast<hipEvent_t>(events[i]), s), "record timing event");
}

}  // namespace

extern "C" ss_status ss_decode_layer(const ss_layer_buffers *L, int64_t step, const void *q, float *out, void *stream,
                                     void *const *events, int64_t *n_miss)
{
    SS_CHECK_ARG(!t_in_callback, "ss_decode_layer: called from a between-layer callback of ss_decode_step_dev");
    SS_CHECK_ARG(L && q && out && n_miss, "ss_decode_layer: null argument");
    SS_CHECK_ARG(L->cache && L->sel_host && L->slots_host && L->miss_host && L->sel_dev && L->slots_dev &&
                     L->miss_dev && L->scores && L->meta && L->nblk_dev,
                 "ss_decode_layer: null buffer");
    SS_CHECK_ARG(L->B == ss::cache_batch(L->cache) && L->Hkv == ss::cache_kv_heads(L->cache),
                 "ss_decode_layer: shape differs from the cache handle's");
    *n_miss = 0;
    const int B = L->B, Hkv = L->Hkv, Hq = L->Hq, k = L->k, d = L->d;
    if (B == 0) return SS_OK;
    SS_CHECK_ARG(k > 0, "ss_decode_layer: k=%d", k);
    const int64_t rows_per_seq = (int64_t)Hkv * k;
    SS_CHECK_ARG(L->miss_cap >= (int64_t)B * rows_per_seq, "ss_decode_layer: miss_cap %lld < B*Hkv*k",
                 (long long)L->miss_cap);
    int P = L->parts < 1 ? 1 : (L->parts > B ? B : L->parts);
    if (L->part_end) {
        P = L->parts;
        SS_CHECK_ARG(P >= 1 && L->part_end[P - 1] == B, "ss_decode_layer: part_end must end at B=%d", B);
        for (int p = 0; p < P; ++p)
            SS_CHECK_ARG(L->part_end[p] > (p ? L->part_end[p - 1] : 0),
                         "ss_decode_layer: part_end must be strictly increasing");
    }
    std::lock_guard<std::mutex> lock(g_exec_mu);
    exec_state *ex = nullptr;
    ss_status st = get_exec(P, &ex);
    if (st) return st;
    hipStream_t s = ss::as_stream(stream);
    const size_t rec = (size_t)2 * L->blk * d * 2;
    const char *q8 = static_cast<const char *>(q);
    const char *meta8 = static_cast<const char *>(L->meta);
    SS_CHECK_ARG(L->meta_kind == SS_META_CUBOID || L->meta_kind == SS_META_MEAN, "ss_decode_layer: metadata kind %d",
                 L->meta_kind);
    const size_t meta_row = (size_t)(L->meta_kind == SS_META_MEAN ? 1 : 2) * d * 2;  // bytes per block
    const int32_t *pe = L->part_end;
    auto b_of = [&](int p) { return p == 0 ? 0 : (pe ? pe[p - 1] : (int)((int64_t)B * p / P)); };

    int32_t *sel_hd = nullptr, *slots_hd = nullptr, *miss_hd = nullptr;  // device views of the host buffers
    if ((st = device_address(L->sel_host, (void **)&sel_hd)) ||
        (st = device_address(L->slots_host, (void **)&slots_hd)) ||
        (st = device_address(L->miss_host, (void **)&miss_hd)))
        return st;

    // the transfer streams start after everything already on `stream`
    if ((st = hip_check(hipEventRecord(ex->start, s), "record")) ||
        (st = hip_check(hipStreamWaitEvent(ex->xfer[0], ex->start, 0), "order transfer stream")) ||
        (st = hip_check(hipStreamWaitEvent(ex->xfer[1], ex->start, 0), "order transfer stream")))
        return st;

    // scoring and selection of every group; selections land in HBM and host memory
    for (int p = 0; p < P; ++p) {
        const int b0 = b_of(p), Bp = b_of(p + 1) - b0;
        if ((st = record(events, 7 * p + 0, s))) return st;
        st = ss_score_blocks_variant(q8 + (size_t)b0 * Hq * d * 2, meta8 + (size_t)b0 * Hkv * L->nblk_max * meta_row,
                                     L->meta_kind, L->agg, L->nblk_dev + b0, Bp, Hq, Hkv, L->nblk_max, d,
                                     L->scores + (size_t)b0 * Hkv * L->nblk_max, stream);
        if (st) return st;
        if ((st = record(events, 7 * p + 1, s))) return st;
        st = ss::launch_topk(L->scores + (size_t)b0 * Hkv * L->nblk_max, L->nblk_dev + b0, Bp, Hkv, L->nblk_max, k,
                             L->sel_dev + b0 * rows_per_seq, sel_hd + b0 * rows_per_seq, s);
        if (st) return st;
        if ((st = record(events, 7 * p + 2, s))) return st;
        if ((st = hip_check(hipEventRecord(ex->sel_ready[p], s), "record"))) return st;
    }

    // resolve group by group; gather on the transfer stream, attend behind it
    int64_t total = 0;
    for (int p = 0; p < P; ++p) {
        const int b0 = b_of(p), b1 = b_of(p + 1), Bp = b1 - b0;
        const int64_t row0 = b0 * rows_per_seq;
        // consecutive groups' gathers run on alternate transfer streams, so the
        // next gather is already streaming while the previous one drains
        hipStream_t x = ex->xfer[p & 1];
        if ((st = wait_host(ex->sel_ready[p], p, step))) return st;
        // miss rows of the step are kept compact: this group appends at `total`
        int64_t np = 0;
        st = ss_cache_resolve_range(L->cache, step, b0, b1, L->sel_host + row0, k, L->slots_host + row0,
                                    L->miss_host + 4 * total, L->miss_cap - total, &np);
        if (st) return st;
        // the gather's timing events ride on its dispatch (kernel execution only)
        hipEvent_t g0 = events ? reinterpret_cast<hipEvent_t>(events[7 * p + 3]) : nullptr;
        hipEvent_t g1 = events ? reinterpret_cast<hipEvent_t>(events[7 * p + 4]) : nullptr;
        ss::set_kernel_timing(g0, g1);
        st = ss::launch_gather(miss_hd + 4 * total, np, L->pool, L->pool_off_dev, L->cache_base, L->cache_off_dev,
                               L->nblk_dev, L->capacity_dev, B, Hkv, rec, slots_hd + row0, L->slots_dev + row0,
                               (int64_t)Bp * rows_per_seq, x);
        const ss::kernel_timing unused = ss::take_kernel_timing();  // set if nothing was launched
        if (st) return st;
        if ((unused.start && (st = hip_check(hipEventRecord(unused.start, x), "record timing event"))) ||
            (unused.stop && (st = hip_check(hipEventRecord(unused.stop, x), "record timing event"))))
            return st;
        if ((st = hip_check(hipEventRecord(ex->gathered[p], x), "record")) ||
            (st = hip_check(hipStreamWaitEvent(s, ex->gathered[p], 0), "order attention after gather")))
            return st;
        if ((st = record(events, 7 * p + 5, s))) return st;
        st = ss_sparse_attention(q8 + (size_t)b0 * Hq * d * 2, L->cache_base, L->cache_off_dev + b0 * Hkv,
                                 L->slots_dev + row0, L->capacity_dev ? L->capacity_dev + b0 * Hkv : nullptr,
                                 L->slot_limit, Bp, Hq, Hkv, d, L->blk, k, L->scale,
                                 out + (size_t)b0 * Hq * d, L->attn_ws, L->attn_ws_bytes, stream);
        if (st) return st;
        if ((st = record(events, 7 * p + 6, s))) return st;
        total += np;
    }
    *n_miss = total;
    return SS_OK;
}

// The same step with the slot table resolved on the GPU (ss_dev_cache).  The
// first group's scoring, top-k, resolve, gather and attention run in order
// on `stream`, so the link starts with no cross-queue hand-off (each costs
// 10-30 us in the traces).  The later groups' scoring, top-k and resolve run
// on a compute stream of the library's, in parallel with the first group's.
// A middle group's gather runs on a transfer stream (the two alternate)
// behind an event recorded after its resolve, and its attention on the
// compute stream behind the gather, after every group's resolve so that no
// resolve waits for a gather.  The last group's gather runs on `stream`
// (still beside the previous group's gather on its transfer stream) with its
// attention right behind it, so no hand-off between queues lies between the
// link's last byte and the end of the step when that gather ends last, as
// with groups that grow to the end.  `stream` then waits for the compute
// stream.  The host enqueues the whole step and returns without
// waiting for any of it.
extern "C" ss_status ss_decode_layer_dev(const ss_layer_buffers *L, ss_dev_cache *dc, int64_t step, const void *q,
                                         float *out, void *stream, void *const *events)
{
    SS_CHECK_ARG(!t_in_callback, "ss_decode_layer_dev: called from a between-layer callback of ss_decode_step_dev");
    SS_CHECK_ARG(L && dc && q && out, "ss_decode_layer_dev: null argument");
    SS_CHECK_ARG(L->sel_dev && L->slots_dev && L->miss_dev && L->scores && L->meta && L->nblk_dev,
                 "ss_decode_layer_dev: null buffer");
    SS_CHECK_ARG(L->B == ss::dev_cache_batch(dc) && L->Hkv == ss::dev_cache_kv_heads(dc),
                 "ss_decode_layer_dev: shape differs from the cache's");
    const int B = L->B, Hkv = L->Hkv, Hq = L->Hq, k = L->k, d = L->d;
    if (B == 0) return SS_OK;
    const int64_t rows_per_seq = (int64_t)Hkv * k;
    SS_CHECK_ARG(L->miss_cap >= (int64_t)B * rows_per_seq, "ss_decode_layer_dev: miss_cap %lld < B*Hkv*k",
                 (long long)L->miss_cap);
    SS_CHECK_ARG(L->meta_kind == SS_META_CUBOID || L->meta_kind == SS_META_MEAN,
                 "ss_decode_layer_dev: metadata kind %d", L->meta_kind);
    int P = L->parts < 1 ? 1 : (L->parts > B ? B : L->parts);
    if (L->part_end) {
        P = L->parts;
        SS_CHECK_ARG(P >= 1 && L->part_end[P - 1] == B, "ss_decode_layer_dev: part_end must end at B=%d", B);
        for (int p = 0; p < P; ++p)
            SS_CHECK_ARG(L->part_end[p] > (p ? L->part_end[p - 1] : 0),
                         "ss_decode_layer_dev: part_end must be strictly increasing");
    }
    const int32_t *pe = L->part_end;
    auto b_of = [&](int p) { return p == 0 ? 0 : (pe ? pe[p - 1] : (int)((int64_t)B * p / P)); };
    // attention workspace: one region for the attentions on `stream`, one for
    // those on the compute stream (the two run at the same time)
    size_t ws_one = 0;
    for (int p = 0; p < P; ++p) {
        const size_t w = ss_sparse_attention_workspace(b_of(p + 1) - b_of(p), Hq, Hkv, d, L->blk, k);
        ws_one = w > ws_one ? w : ws_one;
    }
    ws_one = (ws_one + 255) & ~(size_t)255;
    const bool comp_attn = P > 2;  // the middle groups attend on the compute stream
    const size_t ws_need = ws_one * (comp_attn ? 2 : 1);
    if (L->attn_ws_bytes < ws_need || (ws_need && !L->attn_ws))
        return ss::fail(SS_ERR_OOM, "ss_decode_layer_dev: attention workspace %zu bytes < %zu", L->attn_ws_bytes,
                        ws_need);
    char *ws_s = static_cast<char *>(L->attn_ws);
    char *ws_c = ws_s ? ws_s + ws_one : nullptr;
    ss_status st = ss::dev_cache_check_step(dc, step, k);
    if (st) return st;
    std::lock_guard<std::mutex> lock(g_exec_mu);
    exec_state *ex = nullptr;
    if ((st = get_exec(P, &ex))) return st;
    const hipStream_t s = ss::as_stream(stream);
    const size_t rec = (size_t)2 * L->blk * d * 2;
    const size_t meta_row = (size_t)(L->meta_kind == SS_META_MEAN ? 1 : 2) * d * 2;
    const char *q8 = static_cast<const char *>(q);
    const char *meta8 = static_cast<const char *>(L->meta);
    int32_t *counts = ss::dev_cache_counts(dc);

    if (P > 1 && !ex->comp &&
        (st = hip_check(hipStreamCreateWithFlags(&ex->comp, hipStreamNonBlocking), "create compute stream")))
        return st;
    if (comp_attn && !ex->comp_done &&
        (st = hip_check(hipEventCreateWithFlags(&ex->comp_done, hipEventDisableTiming), "create event")))
        return st;
    if ((st = hip_check(hipEventRecord(ex->start, s), "record")) ||
        (st = hip_check(hipStreamWaitEvent(ex->xfer[0], ex->start, 0), "order transfer stream")) ||
        (st = hip_check(hipStreamWaitEvent(ex->xfer[1], ex->start, 0), "order transfer stream")) ||
        (P > 1 && (st = hip_check(hipStreamWaitEvent(ex->comp, ex->start, 0), "order compute stream"))))
        return st;
    auto attend = [&](int p, hipStream_t on, char *ws) {
        const int b0 = b_of(p), Bp = b_of(p + 1) - b0;
        return ss_sparse_attention(q8 + (size_t)b0 * Hq * d * 2, L->cache_base, L->cache_off_dev + b0 * Hkv,
                                   L->slots_dev + b0 * rows_per_seq,
                                   L->capacity_dev ? L->capacity_dev + b0 * Hkv : nullptr, L->slot_limit, Bp, Hq,
                                   Hkv, d, L->blk, k, L->scale, out + (size_t)b0 * Hq * d, ws, ws_one, on);
    };
    for (int p = 0; p < P; ++p) {
        const int b0 = b_of(p), b1 = b_of(p + 1), Bp = b1 - b0;
        const int64_t row0 = b0 * rows_per_seq;
        const bool last = p == P - 1;
        // the first group's chain on `stream`; later groups' chains on the compute stream
        const hipStream_t c = p == 0 ? s : ex->comp;
        if ((st = record(events, 7 * p + 0, c))) return st;
        st = ss_score_blocks_variant(q8 + (size_t)b0 * Hq * d * 2, meta8 + (size_t)b0 * Hkv * L->nblk_max * meta_row,
                                     L->meta_kind, L->agg, L->nblk_dev + b0, Bp, Hq, Hkv, L->nblk_max, d,
                                     L->scores + (size_t)b0 * Hkv * L->nblk_max, c);
        if (st) return st;
        if ((st = record(events, 7 * p + 1, c))) return st;
        st = ss::launch_topk(L->scores + (size_t)b0 * Hkv * L->nblk_max, L->nblk_dev + b0, Bp, Hkv, L->nblk_max, k,
                             L->sel_dev + row0, nullptr, c);
        if (st) return st;
        st = ss::dev_cache_launch(dc, step, b0, b1, L->sel_dev + row0, k, L->nblk_dev, L->slots_dev + row0,
                                  L->miss_dev, c);
        if (st) return st;
        if ((st = record(events, 7 * p + 2, c))) return st;
        // the group's transfer: the first and the last group's on `stream`, the
        // middle groups' on alternate transfer streams
        const hipStream_t x = (p == 0 || last) ? s : ex->xfer[p & 1];
        if (p > 0 && ((st = hip_check(hipEventRecord(ex->sel_ready[p], c), "record")) ||
                      (st = hip_check(hipStreamWaitEvent(x, ex->sel_ready[p], 0), "order transfer after resolve"))))
            return st;
        hipEvent_t g0 = events ? reinterpret_cast<hipEvent_t>(events[7 * p + 3]) : nullptr;
        hipEvent_t g1 = events ? reinterpret_cast<hipEvent_t>(events[7 * p + 4]) : nullptr;
        ss::set_kernel_timing(g0, g1);
        st = ss::launch_gather_units(L->miss_dev, counts, b0 * Hkv, b1 * Hkv, k, L->pool, L->pool_off_dev,
                                     L->cache_base, L->cache_off_dev, L->nblk_dev, L->capacity_dev, B, Hkv, rec, x);
        const ss::kernel_timing unused = ss::take_kernel_timing();
        if (st) return st;
        if ((unused.start && (st = hip_check(hipEventRecord(unused.start, x), "record timing event"))) ||
            (unused.stop && (st = hip_check(hipEventRecord(unused.stop, x), "record timing event"))))
            return st;
        if (p == 0 || last) {
            // the first and the last group attend right behind their gathers, on `stream`
            if ((st = record(events, 7 * p + 5, s))) return st;
            if ((st = attend(p, s, ws_s))) return st;
            if (!last && (st = record(events, 7 * p + 6, s))) return st;
        }
        if (p > 0 && !last && (st = hip_check(hipEventRecord(ex->gathered[p], x), "record"))) return st;
    }
    // the middle groups' attentions on the compute stream, each behind its gather
    for (int p = 1; p < P - 1; ++p) {
        if ((st = hip_check(hipStreamWaitEvent(ex->comp, ex->gathered[p], 0), "order attention after gather")))
            return st;
        if ((st = record(events, 7 * p + 5, ex->comp))) return st;
        if ((st = attend(p, ex->comp, ws_c))) return st;
        if ((st = record(events, 7 * p + 6, ex->comp))) return st;
    }
    if (comp_attn && ((st = hip_check(hipEventRecord(ex->comp_done, ex->comp), "record")) ||
                      (st = hip_check(hipStreamWaitEvent(s, ex->comp_done, 0), "order stream after attention"))))
        return st;
    // the last group's end event, once everything of the step is done on `stream`
    if ((st = record(events, 7 * (P - 1) + 6, s))) return st;
    return SS_OK;
}

extern "C" ss_status ss_set_host_wait_timeout(int64_t ms)
{
    g_wait_ms.store(ms > 0 ? ms : kDefaultWaitMs, std::memory_order_relaxed);
    return SS_OK;
}

// The decode step over many layers with the resolve on the GPU, the sequence
// groups pipelined across layers.  Within a layer the groups are independent
// (each sequence's attention reads only its own blocks), and a group's next
// layer depends only on its own output of this layer.  So group p runs its
// whole chain -- score, top-k, resolve, gather, attention -- layer after
// layer on one stream of its own: its layer l+1 starts as soon as its layer l
// is attended, while the other groups' gathers of layer l still hold the
// link.  The link then fills and drains once per step instead of once per
// layer.  Inside a group's chain nothing waits for another queue; the only
// waits between queues order the gathers on the link (below).  Group 0 runs
// on `stream`, groups 1..3 on the library's compute and transfer streams
// (the hardware queues a process has); with more than four groups, group p
// shares the stream of group p mod 4 and runs behind it.
extern "C" ss_status ss_decode_step_dev(const ss_layer_buffers *const *layers, ss_dev_cache *const *caches,
                                        int n_layers, int64_t step, const void *const *q, float *const *out,
                                        void *stream, ss_between_fn between, void *ctx, void *const *events)
{
    SS_CHECK_ARG(!t_in_callback, "ss_decode_step_dev: called from its own between-layer callback");
    SS_CHECK_ARG(n_layers >= 0, "ss_decode_step_dev: n_layers=%d", n_layers);
    if (n_layers == 0) return SS_OK;
    SS_CHECK_ARG(layers && caches && q && out, "ss_decode_step_dev: null argument");
    const ss_layer_buffers *L0 = layers[0];
    SS_CHECK_ARG(L0, "ss_decode_step_dev: null layer 0");
    const int B = L0->B, Hkv = L0->Hkv, Hq = L0->Hq, k = L0->k, d = L0->d;
    int P = L0->parts < 1 ? 1 : (L0->parts > B ? B : L0->parts);
    if (L0->part_end) P = L0->parts;
    SS_CHECK_ARG(B >= 0 && P >= 1, "ss_decode_step_dev: B=%d parts=%d", B, L0->parts);
    if (B == 0) return SS_OK;
    const int32_t *pe = L0->part_end;
    if (pe) {
        SS_CHECK_ARG(pe[P - 1] == B, "ss_decode_step_dev: part_end must end at B=%d", B);
        for (int p = 0; p < P; ++p)
            SS_CHECK_ARG(pe[p] > (p ? pe[p - 1] : 0), "ss_decode_step_dev: part_end must be strictly increasing");
    }
    auto b_of = [&](int p) { return p == 0 ? 0 : (pe ? pe[p - 1] : (int)((int64_t)B * p / P)); };
    const int NS = P < 4 ? P : 4;  // group streams
    const int64_t rows_per_seq = (int64_t)Hkv * k;
    std::vector<size_t> ws_one(n_layers);
    for (int l = 0; l < n_layers; ++l) {
        const ss_layer_buffers *L = layers[l];
        ss_dev_cache *dc = caches[l];
        SS_CHECK_ARG(L && dc && q[l] && out[l], "ss_decode_step_dev: null argument for layer %d", l);
        SS_CHECK_ARG(L->sel_dev && L->slots_dev && L->miss_dev && L->scores && L->meta && L->nblk_dev,
                     "ss_decode_step_dev: null buffer in layer %d", l);
        SS_CHECK_ARG(L->B == B && L->Hkv == Hkv && L->Hq == Hq && L->k == k && L->d == d,
                     "ss_decode_step_dev: layer %d's shape differs from layer 0's", l);
        SS_CHECK_ARG(L->B == ss::dev_cache_batch(dc) && L->Hkv == ss::dev_cache_kv_heads(dc),
                     "ss_decode_step_dev: layer %d's shape differs from its cache's", l);
        SS_CHECK_ARG(L->miss_cap >= (int64_t)B * rows_per_seq, "ss_decode_step_dev: layer %d: miss_cap %lld < B*Hkv*k",
                     l, (long long)L->miss_cap);
        SS_CHECK_ARG(L->meta_kind == SS_META_CUBOID || L->meta_kind == SS_META_MEAN,
                     "ss_decode_step_dev: layer %d: metadata kind %d", l, L->meta_kind);
        size_t w1 = 0;
        for (int p = 0; p < P; ++p) {
            const size_t w = ss_sparse_attention_workspace(b_of(p + 1) - b_of(p), Hq, Hkv, d, L->blk, k);
            w1 = w > w1 ? w : w1;
        }
        w1 = (w1 + 255) & ~(size_t)255;
        ws_one[l] = w1;
        if (L->attn_ws_bytes < w1 * NS || (w1 && !L->attn_ws))
            return ss::fail(SS_ERR_OOM, "ss_decode_step_dev: layer %d: attention workspace %zu bytes < %zu", l,
                            L->attn_ws_bytes, w1 * NS);
    }
    ss_status st;
    for (int l = 0; l < n_layers; ++l)
        if ((st = ss::dev_cache_check_step(caches[l], step, k))) return st;
    std::lock_guard<std::mutex> lock(g_exec_mu);
    exec_state *ex = nullptr;
    if ((st = get_exec(P, &ex))) return st;
    const hipStream_t s = ss::as_stream(stream);
    if (NS > 1 && !ex->comp &&
        (st = hip_check(hipStreamCreateWithFlags(&ex->comp, hipStreamNonBlocking), "create compute stream")))
        return st;
    const hipStream_t gs[4] = {s, ex->comp, ex->xfer[0], ex->xfer[1]};
    if ((st = grow_events(ex->link_order, (int64_t)n_layers * P, "ss_decode_step_dev"))) return st;
    if ((st = hip_check(hipEventRecord(ex->start, s), "record"))) return st;
    for (int i = 1; i < NS; ++i)
        if ((st = hip_check(hipStreamWaitEvent(gs[i], ex->start, 0), "order group stream"))) return st;

    auto enqueue = [&]() -> ss_status {
        ss_status e;
        for (int l = 0; l < n_layers; ++l) {
            const ss_layer_buffers *L = layers[l];
            ss_dev_cache *dc = caches[l];
            const size_t rec = (size_t)2 * L->blk * d * 2;
            const size_t meta_row = (size_t)(L->meta_kind == SS_META_MEAN ? 1 : 2) * d * 2;
            const char *q8 = static_cast<const char *>(q[l]);
            const char *meta8 = static_cast<const char *>(L->meta);
            int32_t *counts = ss::dev_cache_counts(dc);
            for (int p = 0; p < P; ++p) {
                const int i = p % NS;
                const hipStream_t g = gs[i];
                const int b0 = b_of(p), b1 = b_of(p + 1), Bp = b1 - b0;
                const int64_t row0 = b0 * rows_per_seq;
                if (l > 0 && between) {
                    // the caller's work that turns the group's layer l-1 output into its layer l queries
                    t_in_callback = true;
                    const ss_status r = between(ctx, l - 1, b0, b1, g);
                    t_in_callback = false;
                    if (r != SS_OK)
                        return ss::fail(r, "ss_decode_step_dev: the between-layer callback returned %d for layer %d, "
                                        "sequences [%d, %d)", (int)r, l - 1, b0, b1);
                }
                e = ss_score_blocks_variant(q8 + (size_t)b0 * Hq * d * 2,
                                            meta8 + (size_t)b0 * Hkv * L->nblk_max * meta_row, L->meta_kind, L->agg,
                                            L->nblk_dev + b0, Bp, Hq, Hkv, L->nblk_max, d,
                                            L->scores + (size_t)b0 * Hkv * L->nblk_max, g);
                if (e) return e;
                e = ss::launch_topk(L->scores + (size_t)b0 * Hkv * L->nblk_max, L->nblk_dev + b0, Bp, Hkv,
                                    L->nblk_max, k, L->sel_dev + row0, nullptr, g);
                if (e) return e;
                e = ss::dev_cache_launch(dc, step, b0, b1, L->sel_dev + row0, k, L->nblk_dev, L->slots_dev + row0,
                                         L->miss_dev, g);
                if (e) return e;
                // The link takes the gathers in (layer, group) order: gather j starts
                // once gather j-(NS-1) has ended, so group p's gather of layer l waits
                // for group p+1's of layer l-1 and at most NS-1 share the link.
                // Equal groups left to share the link freely fall into step with each
                // other (all gather, then all score and select while the link idles);
                // in this order each group scores, selects and resolves under the
                // other groups' transfers.
                const int64_t j = (int64_t)l * P + p;
                const int depth = NS - 1;
                if (depth > 0 && j >= depth) {
                    const int pj = (int)((j - depth) % P);
                    if (gs[pj % NS] != g &&
                        (e = hip_check(hipStreamWaitEvent(g, ex->link_order[j - depth], 0), "order the gathers")))
                        return e;
                }
                const int ev = 2 * (l * P + p);
                hipEvent_t g0 = events ? reinterpret_cast<hipEvent_t>(events[ev]) : nullptr;
                hipEvent_t g1 = events ? reinterpret_cast<hipEvent_t>(events[ev + 1]) : nullptr;
                ss::set_kernel_timing(g0, g1);
                e = ss::launch_gather_units(L->miss_dev, counts, b0 * Hkv, b1 * Hkv, k, L->pool, L->pool_off_dev,
                                            L->cache_base, L->cache_off_dev, L->nblk_dev, L->capacity_dev, B, Hkv,
                                            rec, g);
                const ss::kernel_timing unused = ss::take_kernel_timing();
                if (e) return e;
                if ((unused.start && (e = hip_check(hipEventRecord(unused.start, g), "record timing event"))) ||
                    (unused.stop && (e = hip_check(hipEventRecord(unused.stop, g), "record timing event"))))
                    return e;
                if ((e = hip_check(hipEventRecord(ex->link_order[j], g), "record"))) return e;
                e = ss_sparse_attention(q8 + (size_t)b0 * Hq * d * 2, L->cache_base, L->cache_off_dev + b0 * Hkv,
                                        L->slots_dev + row0, L->capacity_dev ? L->capacity_dev + b0 * Hkv : nullptr,
                                        L->slot_limit, Bp, Hq, Hkv, d, L->blk, k, L->scale,
                                        out[l] + (size_t)b0 * Hq * d, static_cast<char *>(L->attn_ws) + i * ws_one[l],
                                        ws_one[l], g);
                if (e) return e;
            }
        }
        return SS_OK;
    };
    st = enqueue();
    // `stream` waits for every group stream, also after an error, so that work
    // enqueued on it later (or a synchronisation) sees whatever was enqueued
    for (int i = 1; i < NS; ++i) {
        ss_status j = hip_check(hipEventRecord(ex->gathered[i], gs[i]), "record");
        if (!j) j = hip_check(hipStreamWaitEvent(s, ex->gathered[i], 0), "order stream after the group streams");
        if (j && !st) st = j;
    }
    return st;
}

// The same schedule with the slot table resolved on host threads (the
// paper's cache manager): each group's score and top-k run on its stream and
// leave the selection in mapped host memory; the host takes the (layer,
// group) pairs in order, waits for the pair's selection, resolves it, and
// enqueues on the group's stream the gather (in the link order above), the
// attention, the caller's between-layer work and the next layer's score and
// top-k.  A group's host resolve is hidden under the other groups' gathers.
extern "C" ss_status ss_decode_step(const ss_layer_buffers *const *layers, int n_layers, int64_t step,
                                    const void *const *q, float *const *out, void *stream, ss_between_fn between,
                                    void *ctx, void *const *events, int64_t *n_miss)
{
    SS_CHECK_ARG(!t_in_callback, "ss_decode_step: called from a between-layer callback");
    SS_CHECK_ARG(n_layers >= 0, "ss_decode_step: n_layers=%d", n_layers);
    if (n_layers == 0) return SS_OK;
    SS_CHECK_ARG(layers && q && out, "ss_decode_step: null argument");
    const ss_layer_buffers *L0 = layers[0];
    SS_CHECK_ARG(L0, "ss_decode_step: null layer 0");
    const int B = L0->B, Hkv = L0->Hkv, Hq = L0->Hq, k = L0->k, d = L0->d;
    int P = L0->parts < 1 ? 1 : (L0->parts > B ? B : L0->parts);
    if (L0->part_end) P = L0->parts;
    SS_CHECK_ARG(B >= 0 && P >= 1 && k > 0, "ss_decode_step: B=%d parts=%d k=%d", B, L0->parts, k);
    if (n_miss)
        for (int l = 0; l < n_layers; ++l) n_miss[l] = 0;
    if (B == 0) return SS_OK;
    const int32_t *pe = L0->part_end;
    if (pe) {
        SS_CHECK_ARG(pe[P - 1] == B, "ss_decode_step: part_end must end at B=%d", B);
        for (int p = 0; p < P; ++p)
            SS_CHECK_ARG(pe[p] > (p ? pe[p - 1] : 0), "ss_decode_step: part_end must be strictly increasing");
    }
    auto b_of = [&](int p) { return p == 0 ? 0 : (pe ? pe[p - 1] : (int)((int64_t)B * p / P)); };
    const int NS = P < 4 ? P : 4;  // group streams
    const int64_t rows_per_seq = (int64_t)Hkv * k;
    std::vector<size_t> ws_one(n_layers);
    std::vector<int32_t *> sel_hd(n_layers), slots_hd(n_layers), miss_hd(n_layers);  // device views
    ss_status st;
    for (int l = 0; l < n_layers; ++l) {
        const ss_layer_buffers *L = layers[l];
        SS_CHECK_ARG(L && q[l] && out[l], "ss_decode_step: null argument for layer %d", l);
        SS_CHECK_ARG(L->cache && L->sel_host && L->slots_host && L->miss_host && L->sel_dev && L->slots_dev &&
                         L->scores && L->meta && L->nblk_dev,
                     "ss_decode_step: null buffer in layer %d", l);
        SS_CHECK_ARG(L->B == B && L->Hkv == Hkv && L->Hq == Hq && L->k == k && L->d == d,
                     "ss_decode_step: layer %d's shape differs from layer 0's", l);
        SS_CHECK_ARG(L->B == ss::cache_batch(L->cache) && L->Hkv == ss::cache_kv_heads(L->cache),
                     "ss_decode_step: layer %d's shape differs from its cache handle's", l);
        SS_CHECK_ARG(L->miss_cap >= (int64_t)B * rows_per_seq, "ss_decode_step: layer %d: miss_cap %lld < B*Hkv*k",
                     l, (long long)L->miss_cap);
        SS_CHECK_ARG(L->meta_kind == SS_META_CUBOID || L->meta_kind == SS_META_MEAN,
                     "ss_decode_step: layer %d: metadata kind %d", l, L->meta_kind);
        size_t w1 = 0;
        for (int p = 0; p < P; ++p) {
            const size_t w = ss_sparse_attention_workspace(b_of(p + 1) - b_of(p), Hq, Hkv, d, L->blk, k);
            w1 = w > w1 ? w : w1;
        }
        w1 = (w1 + 255) & ~(size_t)255;
        ws_one[l] = w1;
        if (L->attn_ws_bytes < w1 * NS || (w1 && !L->attn_ws))
            return ss::fail(SS_ERR_OOM, "ss_decode_step: layer %d: attention workspace %zu bytes < %zu", l,
                            L->attn_ws_bytes, w1 * NS);
        if ((st = device_address(L->sel_host, (void **)&sel_hd[l])) ||
            (st = device_address(L->slots_host, (void **)&slots_hd[l])) ||
            (st = device_address(L->miss_host, (void **)&miss_hd[l])))
            return st;
    }
    std::lock_guard<std::mutex> lock(g_exec_mu);
    exec_state *ex = nullptr;
    if ((st = get_exec(P, &ex))) return st;
    const hipStream_t s = ss::as_stream(stream);
    if (NS > 1 && !ex->comp &&
        (st = hip_check(hipStreamCreateWithFlags(&ex->comp, hipStreamNonBlocking), "create compute stream")))
        return st;
    if ((st = grow_events(ex->link_order, (int64_t)n_layers * P, "ss_decode_step")) ||
        (st = grow_events(ex->step_sel, (int64_t)n_layers * P, "ss_decode_step")))
        return st;
    const hipStream_t gs[4] = {s, ex->comp, ex->xfer[0], ex->xfer[1]};
    if ((st = hip_check(hipEventRecord(ex->start, s), "record"))) return st;
    for (int i = 1; i < NS; ++i)
        if ((st = hip_check(hipStreamWaitEvent(gs[i], ex->start, 0), "order group stream"))) return st;

    // score and top-k of (layer l, group p) on the group's stream; the
    // selection lands in HBM and in mapped host memory
    auto select = [&](int l, int p) -> ss_status {
        const ss_layer_buffers *L = layers[l];
        const hipStream_t g = gs[p % NS];
        const int b0 = b_of(p), Bp = b_of(p + 1) - b0;
        const int64_t row0 = b0 * rows_per_seq;
        const size_t meta_row = (size_t)(L->meta_kind == SS_META_MEAN ? 1 : 2) * d * 2;
        ss_status e = ss_score_blocks_variant(static_cast<const char *>(q[l]) + (size_t)b0 * Hq * d * 2,
                                              static_cast<const char *>(L->meta) +
                                                  (size_t)b0 * Hkv * L->nblk_max * meta_row,
                                              L->meta_kind, L->agg, L->nblk_dev + b0, Bp, Hq, Hkv, L->nblk_max, d,
                                              L->scores + (size_t)b0 * Hkv * L->nblk_max, g);
        if (e) return e;
        e = ss::launch_topk(L->scores + (size_t)b0 * Hkv * L->nblk_max, L->nblk_dev + b0, Bp, Hkv, L->nblk_max, k,
                            L->sel_dev + row0, sel_hd[l] + row0, g);
        if (e) return e;
        return hip_check(hipEventRecord(ex->step_sel[(size_t)l * P + p], g), "record");
    };
    std::vector<int64_t> total(n_layers, 0);  // each layer's miss rows so far (kept compact)
    auto run = [&]() -> ss_status {
        ss_status e;
        for (int p = 0; p < P; ++p)
            if ((e = select(0, p))) return e;
        for (int l = 0; l < n_layers; ++l) {
            const ss_layer_buffers *L = layers[l];
            const size_t rec = (size_t)2 * L->blk * d * 2;
            for (int p = 0; p < P; ++p) {
                const int i = p % NS;
                const hipStream_t g = gs[i];
                const int b0 = b_of(p), b1 = b_of(p + 1), Bp = b1 - b0;
                const int64_t row0 = b0 * rows_per_seq;
                const int64_t j = (int64_t)l * P + p;
                if ((e = wait_host(ex->step_sel[j], p, step))) return e;
                int64_t np = 0;
                e = ss_cache_resolve_range(L->cache, step, b0, b1, L->sel_host + row0, k, L->slots_host + row0,
                                           L->miss_host + 4 * total[l], L->miss_cap - total[l], &np);
                if (e) return e;
                // the link order of ss_decode_step_dev
                const int depth = NS - 1;
                if (depth > 0 && j >= depth) {
                    const int pj = (int)((j - depth) % P);
                    if (gs[pj % NS] != g &&
                        (e = hip_check(hipStreamWaitEvent(g, ex->link_order[j - depth], 0), "order the gathers")))
                        return e;
                }
                const int ev = 2 * (int)j;
                hipEvent_t g0 = events ? reinterpret_cast<hipEvent_t>(events[ev]) : nullptr;
                hipEvent_t g1 = events ? reinterpret_cast<hipEvent_t>(events[ev + 1]) : nullptr;
                ss::set_kernel_timing(g0, g1);
                e = ss::launch_gather(miss_hd[l] + 4 * total[l], np, L->pool, L->pool_off_dev, L->cache_base,
                                      L->cache_off_dev, L->nblk_dev, L->capacity_dev, B, Hkv, rec,
                                      slots_hd[l] + row0, L->slots_dev + row0, (int64_t)Bp * rows_per_seq, g);
                const ss::kernel_timing unused = ss::take_kernel_timing();
                if (e) return e;
                if ((unused.start && (e = hip_check(hipEventRecord(unused.start, g), "record timing event"))) ||
                    (unused.stop && (e = hip_check(hipEventRecord(unused.stop, g), "record timing event"))) ||
                    (e = hip_check(hipEventRecord(ex->link_order[j], g), "record")))
                    return e;
                total[l] += np;
                e = ss_sparse_attention(static_cast<const char *>(q[l]) + (size_t)b0 * Hq * d * 2, L->cache_base,
                                        L->cache_off_dev + b0 * Hkv, L->slots_dev + row0,
                                        L->capacity_dev ? L->capacity_dev + b0 * Hkv : nullptr, L->slot_limit, Bp, Hq,
                                        Hkv, d, L->blk, k, L->scale, out[l] + (size_t)b0 * Hq * d,
                                        static_cast<char *>(L->attn_ws) + i * ws_one[l], ws_one[l], g);
                if (e) return e;
                if (l + 1 < n_layers) {
                    if (between) {
                        t_in_callback = true;
                        const ss_status r = between(ctx, l, b0, b1, g);
                        t_in_callback = false;
                        if (r != SS_OK)
                            return ss::fail(r, "ss_decode_step: the between-layer callback returned %d for layer %d, "
                                            "sequences [%d, %d)", (int)r, l, b0, b1);
                    }
                    if ((e = select(l + 1, p))) return e;
                }
            }
        }
        return SS_OK;
    };
    st = run();
    for (int i = 1; i < NS; ++i) {
        ss_status j = hip_check(hipEventRecord(ex->gathered[i], gs[i]), "record");
        if (!j) j = hip_check(hipStreamWaitEvent(s, ex->gathered[i], 0), "order stream after the group streams");
        if (j && !st) st = j;
    }
    if (n_miss)
        for (int l = 0; l < n_layers; ++l) n_miss[l] = total[l];
    return st;
}

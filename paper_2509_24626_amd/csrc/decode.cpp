// One layer's decode step over the HBM/DRAM hierarchy: the model executor
// selects blocks on the GPU and hands the indices to the KV cache manager,
// which resolves them against the HBM block cache and loads the misses
// from DRAM in one fused gather (Section 3.1, Section 3.2.1); attention
// then reads only HBM.
#include "internal.hpp"

namespace {

ss_status hip_check(hipError_t e, const char *what)
{
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "ss_decode_layer: %s: %s", what, hipGetErrorString(e));
    return SS_OK;
}

ss_status record(void *const *events, int i, hipStream_t s)
{
    if (!events || !events[i]) return SS_OK;
    return hip_check(hipEventRecord(reinterpret_cast<hipEvent_t>(events[i]), s), "hipEventRecord");
}

}  // namespace

extern "C" ss_status ss_decode_layer(const ss_layer_buffers *L, int64_t step, const void *q, float *out, void *stream,
                                     void *const *events, int64_t *n_miss)
{
    SS_CHECK_ARG(L && q && out && n_miss, "ss_decode_layer: null argument");
    SS_CHECK_ARG(L->cache && L->sel_host && L->slots_host && L->miss_host && L->sel_dev && L->slots_dev &&
                     L->miss_dev,
                 "ss_decode_layer: null buffer");
    *n_miss = 0;
    hipStream_t s = ss::as_stream(stream);
    const size_t sel_bytes = (size_t)L->B * L->Hkv * L->k * sizeof(int32_t);
    ss_status st;

    if ((st = record(events, 0, s))) return st;
    st = ss_score_blocks(q, L->meta, L->nblk_dev, L->B, L->Hq, L->Hkv, L->nblk_max, L->d, L->scores, stream);
    if (st) return st;
    if ((st = record(events, 1, s))) return st;
    st = ss_select_topk(L->scores, L->nblk_dev, L->B, L->Hkv, L->nblk_max, L->k, L->sel_dev, stream);
    if (st) return st;
    if ((st = record(events, 2, s))) return st;
    if ((st = hip_check(hipMemcpyAsync(L->sel_host, L->sel_dev, sel_bytes, hipMemcpyDeviceToHost, s), "copy sel")))
        return st;
    if ((st = hip_check(hipStreamSynchronize(s), "wait for the selection"))) return st;

    int64_t nm = 0;
    st = ss_cache_resolve(L->cache, step, L->sel_host, L->k, L->slots_host, L->miss_host, L->miss_cap, &nm);
    if (st) return st;

    if ((st = hip_check(hipMemcpyAsync(L->slots_dev, L->slots_host, sel_bytes, hipMemcpyHostToDevice, s),
                        "copy slots")))
        return st;
    if (nm > 0 && (st = hip_check(hipMemcpyAsync(L->miss_dev, L->miss_host, (size_t)nm * 4 * sizeof(int32_t),
                                                 hipMemcpyHostToDevice, s),
                                  "copy miss list")))
        return st;
    if ((st = record(events, 3, s))) return st;
    st = ss_gather_blocks(L->miss_dev, nm, L->pool, L->pool_off_dev, L->cache_base, L->cache_off_dev, L->nblk_dev,
                          L->capacity_dev, L->B, L->Hkv, (size_t)2 * L->blk * L->d * 2, stream);
    if (st) return st;
    if ((st = record(events, 4, s))) return st;
    st = ss_sparse_attention(q, L->cache_base, L->cache_off_dev, L->slots_dev, L->slot_limit, L->B, L->Hq, L->Hkv,
                             L->d, L->blk, L->k, L->scale, out, L->attn_ws, L->attn_ws_bytes, stream);
    if (st) return st;
    if ((st = record(events, 5, s))) return st;
    *n_miss = nm;
    return SS_OK;
}

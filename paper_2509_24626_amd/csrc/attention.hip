// Sparse decode attention over the selected KV blocks (Section 2.1's
// softmax(q K^T / sqrt(d)) V, restricted to the tokens of the top-k blocks
// chosen in Section 2.2).
//
// The G query heads that share a KV head make both products small dense
// contractions, run on MFMA with heads as the 16-wide N dimension (padded
// with zero queries).  A wave consumes 16 tokens (8 KiB of K and V) per
// step:
//   S^T[16 tok x 16 heads]  = K[16 tok x 128] * Q^T     4 x v_mfma_f32_16x16x32_bf16
//   O^T[128 ch x 16 heads] += V^T[128 x 16 tok] * P^T   8 x v_mfma_f32_16x16x16_bf16 (x2, hi/lo)
// The S^T accumulator leaves lane (L = lane/16, col = lane%16) holding head
// `col` for tokens 4L .. 4L+3, which is exactly the lane's B fragment of the
// 16x16x16 PV product, so P never moves between lanes.  The step's K rows
// are read as four contiguous 1 KiB loads and staged in the wave's LDS tile,
// from which the A fragments (channels m*32 + 8L .. +7 of row `col`) are
// read; loading the fragments directly (each instruction a 64-byte piece of
// 16 rows) measured 0.805 of the HBM peak on the 128k batch against 0.825.
// The V tile of a block record is stored channel-major, so each V^T
// fragment is one 8-byte load and each V load instruction reads 512
// contiguous bytes.
// Each wave keeps two steps in flight (the next step's loads are issued
// before the current step is computed).  K and V are read with raw buffer
// loads over the unit's cache region: a skipped entry gets an offset past
// the region's end, which the hardware answers with zeros, so the loads
// are unconditional and the compiler can wait for exactly one step's loads
// (a conditional load forces a wait for all outstanding loads).
//
// Softmax runs online in the exp2 domain with fp32 state per head; the
// accumulator rescale is skipped while no head's running maximum changes.
// P enters the PV product as a bf16 hi + lo pair, which keeps about 16
// significant bits of every probability.
//
// Work split: grid (unit, split); a workgroup of 4 waves owns a contiguous
// range of 16-token steps, waves take steps round-robin, the 4 wave partials
// are merged in LDS in wave order, and with several splits a second kernel
// merges the split partials in split order.  All merges run in a fixed
// order, so results do not depend on scheduling.
#include <mutex>
#include <unordered_map>

#include "internal.hpp"

namespace {

constexpr int D = ss::kHeadDim;
constexpr int WAVES = 4;
constexpr int TOK = 16;  // tokens per wave step
constexpr int KPITCH = D * 2 / 16 + 1;  // LDS row pitch of a staged K tile, in 16-byte units

typedef short s16x4_t __attribute__((ext_vector_type(4)));
constexpr int kBufferFlags = 0x00020000;  // raw buffer descriptor word 3 for gfx9 (32-bit data)
// cache policy of the K/V loads: non-temporal (each record is read once per
// launch); measured 0.81 of the HBM peak for the 128k batch against 0.72
// with the default policy
constexpr int kStream = 2;

union frag8_t {  // 8 x bf16: A/B fragment of the 16x16x32 MFMA
    bf16x8_t v;
    uint4 u;
};

union frag4_t {  // 4 x bf16: A/B fragment of the 16x16x16 MFMA
    s16x4_t v;
    uint2 u;
    uint16_t h[4];
};

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

struct split_plan {
    int splits, steps_per_split;
};

template <int BLK>
__global__ __launch_bounds__(256, 3) void attn_kernel(const uint16_t *__restrict__ q, const uint8_t *__restrict__ kv,
                                                      const int64_t *__restrict__ region_off,
                                                      const int32_t *__restrict__ slots,
                                                      const int32_t *__restrict__ capacity, int slot_limit, int Hq,
                                                      int Hkv, int G, int k, float scale_log2, int steps_per_split,
                                                      float *__restrict__ out, float *__restrict__ ws)
{
    constexpr int64_t REC = 2LL * BLK * D * 2;
    __shared__ float sm_m[WAVES][16], sm_l[WAVES][16];
    __shared__ float sm_o[WAVES][16][D + 4];
    __shared__ uint4 kst[WAVES][TOK * KPITCH];  // each wave's K tile of the current step

    const int u = blockIdx.x, split = blockIdx.y, splits = gridDim.y;
    const int b = u / Hkv, g = u - b * Hkv;
    const int lane = threadIdx.x & 63;
    // wave-uniform, so per-step slot indices are scalar loads: a vector load
    // would make every step wait for the previous step's K/V loads (the
    // vector-memory counter completes in order)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int L = lane >> 4, col = lane & 15;
    const int nsteps = (int)(((int64_t)k * BLK + TOK - 1) / TOK);
    const int s_begin = split * steps_per_split;
    const int s_end = min(s_begin + steps_per_split, nsteps);

    // B fragments of S^T = K Q^T: head `col`, channels m*32 + 8L .. +7
    frag8_t qf[4];
    {
        const bool live = col < G;
        const uint16_t *qh = q + ((int64_t)b * Hq + g * G + (live ? col : 0)) * D + L * 8;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            uint4 x = *reinterpret_cast<const uint4 *>(qh + m * 32);
            qf[m].u = live ? x : make_uint4(0, 0, 0, 0);
        }
    }

    const uint8_t *ubase = kv + region_off[u];
    const int32_t *us = slots + (int64_t)u * k;
    // the unit's own slot count bounds its entries, so a slot past it can
    // never reach into the next unit's region (or past the cache)
    int nslot = slot_limit;
    if (capacity) {
        const int c = capacity[u];
        nslot = c < 0 ? 0 : (c < slot_limit ? c : slot_limit);
    }
    const uint32_t lim = (uint32_t)nslot * (uint32_t)REC;  // bytes of the region (< 2^31, host-checked)
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc((void *)ubase, (short)0, (int)lim,
                                                                          kBufferFlags);

    float mrun = -INFINITY, lrun = 0.f;
    f32x4_t o[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    struct step_t {
        uint4 kr[4];  // K rows 4i + L, channels 8col .. 8col+7
        frag4_t vf[8];
        bool vz;  // the lane's accumulator tokens 4L .. 4L+3 are selected
    };
    // token t of the unit's selected-token sequence -> (entry t / BLK, position t % BLK)
    auto load_step = [&](int st, step_t &x) {
        const int tv = st * TOK + L * 4;  // this lane's V^T / accumulator tokens
        // entries of the step (uniform): one, or two when BLK = 8
        const int e0 = (st * TOK) / BLK;
        const int s0 = e0 < k ? us[e0] : -1;
        const int s1 = (BLK == 8 && e0 + 1 < k) ? us[e0 + 1] : -1;
        const int sv = (BLK == 8 && L >= 2) ? s1 : s0;
        const bool live = st < s_end;  // steps past the range load zeros
        const bool vv = live && sv >= 0 && sv < nslot;
        // skipped entries read at `lim`, past the region: the loads return zeros.
        // K: load i reads token rows 4i .. 4i+3 of the step, 1 KiB contiguous
        // (whole 128-byte lines, so the non-temporal policy pays)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = 4 * i + L;
            const int sr = (BLK == 8 && r >= 8) ? s1 : s0;
            const bool vr = live && sr >= 0 && sr < nslot;
            const uint32_t ko = vr ? (uint32_t)sr * (uint32_t)REC + ((st * TOK + r) % BLK) * (D * 2) + col * 16 : lim;
            x.kr[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, ko, 0, kStream));
        }
        const uint32_t vo = vv ? (uint32_t)sv * (uint32_t)REC + BLK * D * 2 + (col * BLK + tv % BLK) * 2 : lim;
#pragma unroll
        for (int t = 0; t < 8; ++t)
            x.vf[t].v = __builtin_bit_cast(s16x4_t, __builtin_amdgcn_raw_buffer_load_b64(rsrc, vo + t * 16 * BLK * 2, 0, kStream));
        x.vz = vv;
    };
    auto compute_step = [&](const step_t &x) {
        // K rows through the wave's LDS tile into A fragments: row `col`,
        // channels m*32 + 8L .. +7 (the padded pitch keeps each 16-lane group
        // of a fragment read on 64 distinct banks)
        uint4 *kt = kst[wave];
#pragma unroll
        for (int i = 0; i < 4; ++i) kt[(4 * i + L) * KPITCH + col] = x.kr[i];
        f32x4_t sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < 4; ++m)
            sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kt[col * KPITCH + 4 * m + L]),
                                                           qf[m].v, sacc, 0, 0, 0);
        float z[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) z[i] = x.vz ? sacc[i] * scale_log2 : -INFINITY;
        float cm = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
        cm = fmaxf(cm, __shfl_xor(cm, 16));
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        const float mnew = fmaxf(mrun, cm);
        float p[4], alpha = 1.f;
        if (mnew == -INFINITY) {
#pragma unroll
            for (int i = 0; i < 4; ++i) p[i] = 0.f;
        } else {
            alpha = __builtin_amdgcn_exp2f(mrun - mnew);
#pragma unroll
            for (int i = 0; i < 4; ++i) p[i] = __builtin_amdgcn_exp2f(z[i] - mnew);
        }
        if (__any(mnew != mrun)) {
#pragma unroll
            for (int t = 0; t < 8; ++t) o[t] *= alpha;
        }
        mrun = mnew;
        frag4_t ph, pl;
        float psum = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            psum += p[i];
            const uint16_t hi = f32_to_bf16_rne(p[i]);
            ph.h[i] = hi;
            pl.h[i] = f32_to_bf16_rne(p[i] - bf16_to_f32(hi));
        }
        lrun = lrun * alpha + psum;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.vf[t].v, ph.v, o[t], 0, 0, 0);
            o[t] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(x.vf[t].v, pl.v, o[t], 0, 0, 0);
        }
    };

    // the prefetches are unconditional (a step past the end loads zeros) so
    // that every path has the same loads in flight and each compute waits
    // only for its own step
    step_t bufA, bufB;
    int st = s_begin + wave;
    load_step(st, bufA);
    for (; st < s_end; st += 2 * WAVES) {
        load_step(st + WAVES, bufB);
        compute_step(bufA);
        if (st + WAVES >= s_end) break;
        load_step(st + 2 * WAVES, bufA);
        compute_step(bufB);
    }
    lrun += __shfl_xor(lrun, 16);
    lrun += __shfl_xor(lrun, 32);

    // wave partials -> LDS; lane holds O^T[16t + 4L + i][col]
    if (L == 0) {
        sm_m[wave][col] = mrun;
        sm_l[wave][col] = lrun;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) sm_o[wave][col][16 * t + L * 4 + i] = o[t][i];
    __syncthreads();

    for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
        const int h = idx / D, ch = idx - h * D;
        float M = sm_m[0][h];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) M = fmaxf(M, sm_m[w][h]);
        float lsum = 0.f, osum = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < WAVES; ++w) {
                const float sc = __builtin_amdgcn_exp2f(sm_m[w][h] - M);
                lsum += sc * sm_l[w][h];
                osum += sc * sm_o[w][h][ch];
            }
        }
        if (splits == 1) {
            out[((int64_t)b * Hq + g * G + h) * D + ch] = lsum > 0.f ? osum / lsum : 0.f;
        } else {
            float *pp = ws + (((int64_t)u * splits + split) * G + h) * (D + 2);
            if (ch == 0) {
                pp[0] = M;
                pp[1] = lsum;
            }
            pp[2 + ch] = osum;
        }
    }
}

__global__ __launch_bounds__(D) void combine_kernel(const float *__restrict__ ws, int Hq, int Hkv, int G, int splits,
                                                    float *__restrict__ out)
{
    const int u = blockIdx.x, h = blockIdx.y, ch = threadIdx.x;
    const int b = u / Hkv, g = u - b * Hkv;
    const float *p = ws + ((int64_t)u * splits * G + h) * (D + 2);
    const int64_t stride = (int64_t)G * (D + 2);
    float M = -INFINITY;
    for (int s = 0; s < splits; ++s) M = fmaxf(M, p[s * stride]);
    float lsum = 0.f, osum = 0.f;
    if (M != -INFINITY)
        for (int s = 0; s < splits; ++s) {
            const float *ps = p + s * stride;
            const float sc = __builtin_amdgcn_exp2f(ps[0] - M);
            lsum += sc * ps[1];
            osum += sc * ps[2 + ch];
        }
    out[((int64_t)b * Hq + g * G + h) * D + ch] = lsum > 0.f ? osum / lsum : 0.f;
}

split_plan plan(int units, int k, int blk)
{
    const int steps = (int)(((int64_t)k * blk + TOK - 1) / TOK);
    const int target_wg = 512;  // two 4-wave workgroups per CU
    int splits = units > 0 ? (target_wg + units - 1) / units : 1;
    int max_splits = steps / (WAVES * 4);  // keep >= 4 steps per wave
    if (max_splits < 1) max_splits = 1;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    int sps = (steps + splits - 1) / splits;
    splits = (steps + sps - 1) / sps;
    return {splits, sps};
}

}  // namespace

extern "C" size_t ss_sparse_attention_workspace(int B, int Hq, int Hkv, int d, int blk, int k)
{
    if (B <= 0 || Hkv <= 0 || Hq <= 0 || Hq % Hkv || d != D || !ss::supported_blk(blk) || k <= 0) return 0;
    const int units = B * Hkv;
    split_plan sp = plan(units, k, blk);
    if (sp.splits <= 1) return 0;
    return (size_t)units * sp.splits * (Hq / Hkv) * (D + 2) * sizeof(float);
}

extern "C" ss_status ss_sparse_attention(const void *q, const void *kv_base, const int64_t *region_off,
                                         const int32_t *slots, const int32_t *capacity, int32_t slot_limit, int B,
                                         int Hq, int Hkv, int d,
                                         int blk, int k, float scale, float *out, void *workspace, size_t ws_bytes,
                                         void *stream)
{
    SS_CHECK_ARG(B >= 0 && Hq > 0 && Hkv > 0 && k > 0, "ss_sparse_attention: bad shape B=%d Hq=%d Hkv=%d k=%d", B, Hq,
                 Hkv, k);
    SS_CHECK_ARG(Hq % Hkv == 0, "ss_sparse_attention: Hq=%d not a multiple of Hkv=%d", Hq, Hkv);
    SS_CHECK_SUPPORTED(Hq / Hkv <= ss::kMaxGroup, "ss_sparse_attention: group size %d > %d", Hq / Hkv, ss::kMaxGroup);
    SS_CHECK_SUPPORTED(d == D, "ss_sparse_attention: d=%d (only 128)", d);
    SS_CHECK_SUPPORTED(ss::supported_blk(blk), "ss_sparse_attention: blk=%d (8, 16 or 32)", blk);
    SS_CHECK_ARG(std::isfinite(scale), "ss_sparse_attention: scale not finite");
    if (B == 0) return SS_OK;
    SS_CHECK_ARG(q && kv_base && region_off && slots && out, "ss_sparse_attention: null pointer");
    SS_CHECK_SUPPORTED(slot_limit >= 0 && (int64_t)slot_limit * 2 * blk * D * 2 <= 0x7FFFFFFF,
                       "ss_sparse_attention: slot_limit=%d records exceed a 2 GiB region", slot_limit);
    const int units = B * Hkv;
    split_plan sp = plan(units, k, blk);
    const size_t need = ss_sparse_attention_workspace(B, Hq, Hkv, d, blk, k);
    if (ws_bytes < need || (need && !workspace))
        return ss::fail(SS_ERR_OOM, "ss_sparse_attention: workspace %zu bytes < %zu", ws_bytes, need);
    hipStream_t s = ss::as_stream(stream);
    const float scale_log2 = scale * 1.4426950408889634f;
    const dim3 grid(units, sp.splits);
    const int G = Hq / Hkv;
    const uint16_t *qq = static_cast<const uint16_t *>(q);
    const uint8_t *kv = static_cast<const uint8_t *>(kv_base);
    float *ws = static_cast<float *>(workspace);
    switch (blk) {
    case 8: ss::launch(attn_kernel<8>, grid, dim3(256), s, qq, kv, region_off, slots, capacity, slot_limit, Hq, Hkv, G, k, scale_log2, sp.steps_per_split, out, ws); break;
    case 16: ss::launch(attn_kernel<16>, grid, dim3(256), s, qq, kv, region_off, slots, capacity, slot_limit, Hq, Hkv, G, k, scale_log2, sp.steps_per_split, out, ws); break;
    default: ss::launch(attn_kernel<32>, grid, dim3(256), s, qq, kv, region_off, slots, capacity, slot_limit, Hq, Hkv, G, k, scale_log2, sp.steps_per_split, out, ws); break;
    }
    ss_status st = ss::check_launch("ss_sparse_attention");
    if (st != SS_OK || sp.splits == 1) return st;
    combine_kernel<<<dim3(units, G), dim3(D), 0, s>>>(ws, Hq, Hkv, G, sp.splits, out);
    return ss::check_launch("ss_sparse_attention(combine)");
}

// ------------------------------------------------- allocation-free variant
// The split partials of ss_sparse_attention_static live in this file-scope
// device array instead of a caller workspace.  Every supported shape fits:
// with more than one split, units * splits < units + 512 <= 1023 and
// G <= 16, so the partials take at most 1023 * 16 * (128 + 2) * 4 bytes.
// Host code never uses the array's name as an address: each device's copy
// is looked up once with hipGetSymbolAddress and that pointer is passed on.
namespace {
constexpr size_t kStaticScratchBytes = 9u << 20;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

std::mutex g_scratch_mu;
std::unordered_map<int, void *> g_scratch_addr;  // by device

ss_status scratch_address(void **out)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "ss_sparse_attention_static: hipGetDevice: %s", hipGetErrorString(e));
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    auto it = g_scratch_addr.find(dev);
    if (it != g_scratch_addr.end()) {
        *out = it->second;
        return SS_OK;
    }
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
        return ss::fail(SS_ERR_HIP, "ss_sparse_attention_static: hipGetSymbolAddress of the scratch array: %s",
                        hipGetErrorString(e));
    g_scratch_addr[dev] = p;
    *out = p;
    return SS_OK;
}
}  // namespace

extern "C" ss_status ss_sparse_attention_static(const void *q, const void *kv_base, const int64_t *region_off,
                                                const int32_t *slots, const int32_t *capacity, int32_t slot_limit,
                                                int B, int Hq, int Hkv, int d, int blk, int k, float scale,
                                                float *out, void *stream)
{
    // shapes the main entry point rejects are rejected there; this only sizes the partials
    const size_t need = ss_sparse_attention_workspace(B, Hq, Hkv, d, blk, k);
    if (need > kStaticScratchBytes)
        return ss::fail(SS_ERR_OOM, "ss_sparse_attention_static: %zu bytes of split partials exceed the %zu-byte "
                        "static scratch", need, kStaticScratchBytes);
    void *ws = nullptr;
    if (need) {
        ss_status st = scratch_address(&ws);
        if (st) return st;
    }
    return ss_sparse_attention(q, kv_base, region_off, slots, capacity, slot_limit, B, Hq, Hkv, d, blk, k, scale,
                               out, ws, need, stream);
}

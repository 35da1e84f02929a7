// Sparse decode attention over the selected KV blocks (Section 2.1's
// softmax(q K^T / sqrt(d)) V, restricted to the tokens of the top-k blocks
// chosen in Section 2.2).
//
// The G query heads that share a KV head make both products small dense
// contractions, run on v_mfma_f32_16x16x32_bf16 with heads as the 16-wide
// N dimension (padded with zero queries):
//   S^T[32 tok x 16 heads] = K[32 tok x 128] * Q^T         (2 row tiles x 4 k-steps)
//   O^T[128 ch x 16 heads] += V^T[128 x 32 tok] * P^T      (8 row tiles, K = 32 tokens)
// A wave consumes 32 tokens (16 KiB of K and V) per step.  The K rows of
// the two S^T tiles are permuted (tile T, row r -> token (r/4)*8 + T*4 + r%4)
// so that the accumulator lane holding head `col` ends up with exactly the
// 8 consecutive tokens (lane/16)*8 .. +7, which is the B-operand fragment
// the PV product needs: P never moves between lanes.  The V tile of a
// block record is stored channel-major, so each V^T fragment is one
// 16-byte load.
//
// Softmax runs online in the exp2 domain with fp32 state per head.  P is
// split into bf16 hi + lo parts (two PV MFMAs), which keeps about 16
// significant bits of every probability.
//
// Work split: grid (unit, split); a workgroup of 4 waves owns a contiguous
// range of 32-token chunks, waves take chunks round-robin, the 4 wave
// partials are merged in LDS in wave order, and with several splits a
// second kernel merges the split partials in split order.  All merges run
// in a fixed order, so results do not depend on scheduling.
#include "internal.hpp"

namespace {

constexpr int D = ss::kHeadDim;
constexpr int WAVES = 4;

union frag_t {
    bf16x8_t v;
    uint4 u;
    uint16_t h[8];
};

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

struct split_plan {
    int splits, chunks_per_split;
};

template <int BLK>
__global__ __launch_bounds__(256) void attn_kernel(const uint16_t *__restrict__ q, const uint8_t *__restrict__ kv,
                                                   const int64_t *__restrict__ region_off,
                                                   const int32_t *__restrict__ slots, int slot_limit, int Hq,
                                                   int Hkv, int G, int k, float scale_log2, int chunks_per_split,
                                                   float *__restrict__ out, float *__restrict__ ws)
{
    constexpr int64_t REC = 2LL * BLK * D * 2;
    constexpr int EPC = 32 / BLK;  // block records per 32-token chunk
    __shared__ float sm_m[WAVES][16], sm_l[WAVES][16];
    __shared__ float sm_o[WAVES][16][D + 4];

    const int u = blockIdx.x, split = blockIdx.y, splits = gridDim.y;
    const int b = u / Hkv, g = u - b * Hkv;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int L = lane >> 4, col = lane & 15;
    const int nchunks = (k + EPC - 1) / EPC;
    const int c0 = split * chunks_per_split;
    const int c1 = min(c0 + chunks_per_split, nchunks);

    // B fragments of S^T = K Q^T: head `col`, channels m*32 + L*8 .. +7 (so
    // each K load instruction reads a contiguous 64-byte piece of every row)
    frag_t qf[4];
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
    // token handled by this lane's A rows in the two S^T tiles, and its record
    const int tokA0 = (col >> 2) * 8 + (col & 3);  // tile 0; tile 1 adds 4
    const int eK0 = tokA0 / BLK, eK1 = (tokA0 + 4) / BLK;
    const int posK0 = tokA0 % BLK, posK1 = (tokA0 + 4) % BLK;
    const int eV = (L * 8) / BLK, posV = (L * 8) % BLK;  // V^T fragment: tokens L*8 .. +7
    const int eZ0 = (L * 8) / BLK, eZ1 = (L * 8 + 4) / BLK;  // records of accumulator tokens

    float mrun = -INFINITY, lrun = 0.f;
    f32x4_t o[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // One 32-token chunk: its K and V^T operand fragments and the validity of
    // the accumulator tokens.  Waves prefetch their next chunk while the
    // current one is computed (two buffers, loop unrolled by two).
    struct chunk_t {
        frag_t kf[2][4], vf[8];
        bool vz0, vz1;
    };
    auto load_chunk = [&](int c, chunk_t &ch) {
        const uint8_t *rec[EPC];
        bool valid[EPC];
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
            const int idx = c * EPC + e;
            const int s = idx < k ? us[idx] : -1;
            valid[e] = s >= 0 && s < slot_limit;
            rec[e] = ubase + (int64_t)(valid[e] ? s : 0) * REC;
        }
        const bool vk0 = valid[eK0], vk1 = valid[eK1], vv = valid[eV];
        const uint8_t *pk0 = rec[eK0] + posK0 * (D * 2) + L * 16;
        const uint8_t *pk1 = rec[eK1] + posK1 * (D * 2) + L * 16;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            ch.kf[0][m].u = vk0 ? *reinterpret_cast<const uint4 *>(pk0 + m * 64) : make_uint4(0, 0, 0, 0);
            ch.kf[1][m].u = vk1 ? *reinterpret_cast<const uint4 *>(pk1 + m * 64) : make_uint4(0, 0, 0, 0);
        }
        const uint8_t *pv = rec[eV] + BLK * D * 2 + (col * BLK + posV) * 2;
#pragma unroll
        for (int t = 0; t < 8; ++t)
            ch.vf[t].u = vv ? *reinterpret_cast<const uint4 *>(pv + t * 16 * BLK * 2) : make_uint4(0, 0, 0, 0);
        ch.vz0 = valid[eZ0];
        ch.vz1 = valid[eZ1];
    };
    auto compute_chunk = [&](const chunk_t &ch) {
        f32x4_t s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ch.kf[0][m].v, qf[m].v, s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ch.kf[1][m].v, qf[m].v, s1, 0, 0, 0);
        }
        // lane holds z for head `col`, tokens L*8 + v (v = T*4 + i)
        float z[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            z[i] = ch.vz0 ? s0[i] * scale_log2 : -INFINITY;
            z[4 + i] = ch.vz1 ? s1[i] * scale_log2 : -INFINITY;
        }
        float cm = z[0];
#pragma unroll
        for (int v = 1; v < 8; ++v) cm = fmaxf(cm, z[v]);
        cm = fmaxf(cm, __shfl_xor(cm, 16));
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        const float mnew = fmaxf(mrun, cm);
        float p[8], alpha;
        if (mnew == -INFINITY) {
            alpha = 1.f;
#pragma unroll
            for (int v = 0; v < 8; ++v) p[v] = 0.f;
        } else {
            alpha = __builtin_amdgcn_exp2f(mrun - mnew);
#pragma unroll
            for (int v = 0; v < 8; ++v) p[v] = __builtin_amdgcn_exp2f(z[v] - mnew);
        }
        mrun = mnew;
        float psum = 0.f;
        frag_t ph, pl;
#pragma unroll
        for (int v = 0; v < 8; ++v) {
            psum += p[v];
            const uint16_t hi = f32_to_bf16_rne(p[v]);
            ph.h[v] = hi;
            pl.h[v] = f32_to_bf16_rne(p[v] - bf16_to_f32(hi));
        }
        lrun = lrun * alpha + psum;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            o[t] *= alpha;
            o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ch.vf[t].v, ph.v, o[t], 0, 0, 0);
            o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ch.vf[t].v, pl.v, o[t], 0, 0, 0);
        }
    };

    for (int c = c0 + wave; c < c1; c += WAVES) {
        chunk_t buf;
        load_chunk(c, buf);
        compute_chunk(buf);
    }
    lrun += __shfl_xor(lrun, 16);
    lrun += __shfl_xor(lrun, 32);

    // wave partials -> LDS; lane holds O^T[16t + L*4 + i][col]
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
            float *p = ws + (((int64_t)u * splits + split) * G + h) * (D + 2);
            if (ch == 0) {
                p[0] = M;
                p[1] = lsum;
            }
            p[2 + ch] = osum;
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
    const int epc = 32 / blk;
    const int chunks = (k + epc - 1) / epc;
    const int target_wg = 1024;
    int splits = units > 0 ? (target_wg + units - 1) / units : 1;
    int max_splits = chunks / (WAVES * 2);  // keep >= 2 chunks per wave
    if (max_splits < 1) max_splits = 1;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    int cps = (chunks + splits - 1) / splits;
    splits = (chunks + cps - 1) / cps;
    return {splits, cps};
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
                                         const int32_t *slots, int32_t slot_limit, int B, int Hq, int Hkv, int d,
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
    case 8: attn_kernel<8><<<grid, dim3(256), 0, s>>>(qq, kv, region_off, slots, slot_limit, Hq, Hkv, G, k, scale_log2, sp.chunks_per_split, out, ws); break;
    case 16: attn_kernel<16><<<grid, dim3(256), 0, s>>>(qq, kv, region_off, slots, slot_limit, Hq, Hkv, G, k, scale_log2, sp.chunks_per_split, out, ws); break;
    default: attn_kernel<32><<<grid, dim3(256), 0, s>>>(qq, kv, region_off, slots, slot_limit, Hq, Hkv, G, k, scale_log2, sp.chunks_per_split, out, ws); break;
    }
    ss_status st = ss::check_launch("ss_sparse_attention");
    if (st != SS_OK || sp.splits == 1) return st;
    combine_kernel<<<dim3(units, G), dim3(D), 0, s>>>(ws, Hq, Hkv, G, sp.splits, out);
    return ss::check_launch("ss_sparse_attention(combine)");
}

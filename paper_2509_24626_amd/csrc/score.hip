// Block criticality scores (Section 2.2): for block j of KV head g and each
// query head h of the group, the largest q_h.k over the block's key cuboid
// [lo, hi], then the maximum over the group's heads.
//
// Since hi >= lo channel-wise,
//     max(q*lo, q*hi) = max(q,0)*hi + min(q,0)*lo     (exactly, per channel),
// so with the metadata row m_j = [lo_j, hi_j] (256 bf16) and the query
// weights w_h = [min(q_h,0), max(q_h,0)] the per-head bound is the plain dot
// product w_h . m_j.  For one unit this is the small dense contraction
//     S^T[heads x blocks] = W^T[G x 256] * M^T[256 x nblk],
// done with v_mfma_f32_16x16x32_bf16: bf16 x bf16 products are exact in
// fp32 and accumulate in fp32.  The GQA heads fill the MFMA rows (padded to
// 16 with zero weights); each column is one block.
//
// Every MFMA B fragment is a direct 16-byte load of one metadata row, so the
// 512-byte rows stream from HBM with no LDS staging and no cross-lane
// reduction; the head maximum is taken over accumulator registers.
#include "internal.hpp"

namespace {

constexpr int D = ss::kHeadDim;
constexpr int ROW_BYTES = 2 * D * 2;  // lo + hi, bf16
constexpr int TILE = 16;              // blocks per MFMA tile
constexpr int WAVES = 4;
constexpr int TILES_PER_WAVE = 4;
constexpr int BLOCKS_PER_WG = TILE * WAVES * TILES_PER_WAVE;  // 256

union frag_t {
    bf16x8_t v;
    uint4 u;
    uint16_t h[8];
};

// Lane (L = lane/16, col = lane%16) takes 16-byte chunks c = L*8 + m of a
// metadata row for the 8 MFMAs m of a tile (chunks 0..15 are lo, 16..31
// hi): each lane streams 128 contiguous bytes of its row.  (A mapping where
// each load instruction covers a contiguous 64-byte piece of every row
// instead measured 6% slower on MI355X.)  The A fragments hold the matching
// weights of head `col`.
__global__ __launch_bounds__(256) void score_kernel(const uint16_t *__restrict__ q,
                                                    const uint8_t *__restrict__ meta,
                                                    const int32_t *__restrict__ nblk, int Hq, int Hkv, int G,
                                                    int nblk_max, int chunks_per_unit, float *__restrict__ scores)
{
    const int u = blockIdx.x / chunks_per_unit;
    const int chunk = blockIdx.x - u * chunks_per_unit;
    const int b = u / Hkv, g = u - b * Hkv;
    int n = nblk[b];
    n = n < 0 ? 0 : (n > nblk_max ? nblk_max : n);
    const int j0 = chunk * BLOCKS_PER_WG;
    if (j0 >= n) return;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int L = lane >> 4;
    const int col = lane & 15;

    // weights of head g*G + col for chunks L*8 .. L*8+7
    frag_t w[8];
    {
        const bool live = col < G;
        const uint16_t *qh = q + ((int64_t)b * Hq + g * G + (live ? col : 0)) * D;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const bool hi_half = L >= 2;            // chunks 16..31 multiply hi
            const int c = ((L * 8 + m) & 15) * 8;  // channel of the chunk
            frag_t x;
            x.u = *reinterpret_cast<const uint4 *>(qh + c);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const bool neg = (x.h[e] & 0x8000u) != 0;
                // hi half keeps the non-negative part, lo half the negative part
                w[m].h[e] = (live && (neg != hi_half)) ? x.h[e] : (uint16_t)0;
            }
        }
    }

    const uint8_t *mu = meta + (int64_t)u * nblk_max * ROW_BYTES;
    float *su = scores + (int64_t)u * nblk_max;
    const int lane_off = L * 128;  // byte offset of chunk L*8

    // interleave waves over tiles so the WG walks memory front to back
    frag_t cur[8], nxt[8];
    auto load_tile = [&](int t, frag_t *f) {
        int j = j0 + (t * WAVES + wave) * TILE + col;
        j = j < n ? j : n - 1;  // rows past the end are loaded in range and not stored
        const uint8_t *row = mu + (int64_t)j * ROW_BYTES + lane_off;
#pragma unroll
        for (int m = 0; m < 8; ++m) f[m].u = *reinterpret_cast<const uint4 *>(row + m * 16);
    };

    int ntiles = 0;
    for (int t = 0; t < TILES_PER_WAVE; ++t)
        if (j0 + (t * WAVES + wave) * TILE < n) ntiles = t + 1;
    if (ntiles == 0) return;

    load_tile(0, cur);
    for (int t = 0; t < ntiles; ++t) {
        if (t + 1 < ntiles) load_tile(t + 1, nxt);
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < 8; ++m) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[m].v, cur[m].v, acc, 0, 0, 0);
        // lane holds heads L*4 .. L*4+3 of block column `col`
        float s = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (L * 4 + i < G) s = fmaxf(s, acc[i]);
        s = fmaxf(s, __shfl_xor(s, 16));
        s = fmaxf(s, __shfl_xor(s, 32));
        const int j = j0 + (t * WAVES + wave) * TILE + col;
        if (L == 0 && j < n) su[j] = s;
        if (t + 1 < ntiles) {
#pragma unroll
            for (int m = 0; m < 8; ++m) cur[m] = nxt[m];
        }
    }
}

}  // namespace

namespace ss {

ss_status launch_score(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv, int nblk_max,
                       float *scores, hipStream_t s)
{
    const int chunks = (nblk_max + BLOCKS_PER_WG - 1) / BLOCKS_PER_WG;
    const int64_t grid = (int64_t)B * Hkv * chunks;
    if (grid == 0) return SS_OK;
    SS_CHECK_SUPPORTED(grid <= 0x7FFFFFFF, "score: grid too large");
    ss::launch(score_kernel, dim3((unsigned)grid), dim3(256), s, static_cast<const uint16_t *>(q),
               static_cast<const uint8_t *>(meta), nblk, Hq, Hkv, Hq / Hkv, nblk_max, chunks, scores);
    return check_launch("ss_score_blocks");
}

ss_status check_score_args(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                           int nblk_max, int d, const void *scores, const char *who)
{
    SS_CHECK_ARG(B >= 0 && Hq > 0 && Hkv > 0 && nblk_max >= 0, "%s: bad shape B=%d Hq=%d Hkv=%d nblk_max=%d", who, B,
                 Hq, Hkv, nblk_max);
    SS_CHECK_ARG(Hq % Hkv == 0, "%s: Hq=%d not a multiple of Hkv=%d", who, Hq, Hkv);
    SS_CHECK_SUPPORTED(Hq / Hkv <= kMaxGroup, "%s: group size %d > %d", who, Hq / Hkv, kMaxGroup);
    SS_CHECK_SUPPORTED(d == kHeadDim, "%s: d=%d (only 128)", who, d);
    SS_CHECK_SUPPORTED(nblk_max <= kMaxBlocks, "%s: nblk_max=%d > %d", who, nblk_max, kMaxBlocks);
    if ((int64_t)B * nblk_max > 0) SS_CHECK_ARG(q && meta && nblk && scores, "%s: null pointer", who);
    return SS_OK;
}

}  // namespace ss

extern "C" ss_status ss_score_blocks(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                                     int nblk_max, int d, float *scores, void *stream)
{
    ss_status st = ss::check_score_args(q, meta, nblk, B, Hq, Hkv, nblk_max, d, scores, "ss_score_blocks");
    if (st != SS_OK) return st;
    return ss::launch_score(q, meta, nblk, B, Hq, Hkv, nblk_max, scores, ss::as_stream(stream));
}

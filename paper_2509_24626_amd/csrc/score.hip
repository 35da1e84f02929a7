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
//
// For cuboid rows the launch reserves LDS that the kernel never touches
// (kResidencyLds), so that at most two workgroups (8 waves) share a CU: on
// MI355X the 128k-token batch streams at 0.765 of the 8 TB/s peak that way,
// against 0.73 with the eight workgroups per CU the registers allow, 0.75
// with three and 0.69 with one.  Mean-key rows are half as long, so each
// workgroup streams half the bytes; they run fastest with no reservation
// (0.186 ms for the batch, against 0.183-0.205 with four, three or two
// workgroups per CU).
#include "internal.hpp"

namespace {

constexpr int D = ss::kHeadDim;
constexpr int TILE = 16;              // blocks per MFMA tile
constexpr int WAVES = 4;
constexpr int TILES_PER_WAVE = 4;
constexpr int BLOCKS_PER_WG = TILE * WAVES * TILES_PER_WAVE;  // 256
// 2 x 60 KiB fit in a CU's 160 KiB of LDS and 3 do not; the 40 KiB left over
// still take one attention workgroup (34 KiB) beside two scoring workgroups
constexpr size_t kResidencyLds = 60 * 1024;
constexpr int kBufferFlags = 0x00020000;  // raw buffer descriptor word 3 for gfx9 (32-bit data)

union frag_t {
    bf16x8_t v;
    uint4 u;
    uint16_t h[8];
};

// Lane (L = lane/16, col = lane%16) takes 16-byte chunk c = 4*m + L of a
// metadata row for MFMA m of a tile, so each load instruction covers one
// contiguous 64-byte piece of each of the tile's 16 rows.  (Each lane
// streaming NCH*16 contiguous bytes of its row instead measured 1.5% slower
// through buffer loads.)  The A fragments hold the matching weights of head
// `col`.
//
// KIND 0, cuboid rows [lo, hi] (512 B, NCH = 8): chunks 0..15 are lo and
// multiply min(q, 0), chunks 16..31 (m >= 4) are hi and multiply max(q, 0).
// KIND 1, mean-key rows (256 B, NCH = 4): each chunk multiplies q itself.
// AGG 0 takes the maximum over the group's heads, AGG 1 their sum.
template <int KIND, int AGG>
__global__ __launch_bounds__(256) void score_kernel(const uint16_t *__restrict__ q,
                                                    const uint8_t *__restrict__ meta,
                                                    const int32_t *__restrict__ nblk, int Hq, int Hkv, int G,
                                                    int nblk_max, int chunks_per_unit, float *__restrict__ scores)
{
    constexpr int NCH = KIND == 0 ? 8 : 4;
    constexpr int ROW = NCH * 4 * 16;  // 512 or 256 bytes
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

    // weights of head g*G + col for chunks L*NCH .. L*NCH+NCH-1, selected
    // branch-free with masks on the 32-bit words (two bf16 each)
    frag_t w[NCH];
    {
        const bool live = col < G;
        const uint16_t *qh = q + ((int64_t)b * Hq + g * G + (live ? col : 0)) * D;
        const uint32_t live_mask = live ? 0xFFFFFFFFu : 0u;
#pragma unroll
        for (int m = 0; m < NCH; ++m) {
            const bool hi_half = KIND == 0 && m >= 4;  // cuboid chunks 16..31 multiply hi
            const int c = (4 * m + L) & 15;            // q channels c*8 .. c*8+7
            const uint4 x = *reinterpret_cast<const uint4 *>(qh + c * 8);
            uint32_t v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                uint32_t keep = live_mask;
                if (KIND == 0) {
                    const uint32_t neg = ((v[i] >> 15) & 0x00010001u) * 0xFFFFu;  // 0xFFFF per negative half
                    keep &= hi_half ? ~neg : neg;  // hi keeps max(q, 0), lo keeps min(q, 0)
                }
                v[i] &= keep;
            }
            w[m].u = make_uint4(v[0], v[1], v[2], v[3]);
        }
    }

    const uint8_t *mu = meta + (int64_t)u * nblk_max * ROW;
    float *su = scores + (int64_t)u * nblk_max;
    // n * ROW <= kMaxBlocks * 512 bytes < 2^31
    const __amdgpu_buffer_rsrc_t mrs = __builtin_amdgcn_make_buffer_rsrc((void *)mu, (short)0, n * ROW, kBufferFlags);

    // interleave waves over tiles so the WG walks memory front to back
    frag_t cur[NCH], nxt[NCH];
    auto load_tile = [&](int t, frag_t *f) {
        int j = j0 + (t * WAVES + wave) * TILE + col;
        j = j < n ? j : n - 1;  // rows past the end are loaded in range and not stored
        const uint32_t off = (uint32_t)j * ROW + L * 16;
#pragma unroll
        for (int m = 0; m < NCH; ++m)
            f[m].v = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(mrs, off + m * 64, 0, 0));
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
        for (int m = 0; m < NCH; ++m) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[m].v, cur[m].v, acc, 0, 0, 0);
        // lane holds heads L*4 .. L*4+3 of block column `col`
        float s;
        if (AGG == 0) {
            s = -INFINITY;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (L * 4 + i < G) s = fmaxf(s, acc[i]);
            s = fmaxf(s, __shfl_xor(s, 16));
            s = fmaxf(s, __shfl_xor(s, 32));
        } else {
            s = (acc[0] + acc[1]) + (acc[2] + acc[3]);  // padded heads hold exact zeros
            s += __shfl_xor(s, 16);
            s += __shfl_xor(s, 32);
        }
        const int j = j0 + (t * WAVES + wave) * TILE + col;
        if (L == 0 && j < n) su[j] = s;
        if (t + 1 < ntiles) {
#pragma unroll
            for (int m = 0; m < NCH; ++m) cur[m] = nxt[m];
        }
    }
}

}  // namespace

namespace ss {

ss_status launch_score(const void *q, const void *meta, int meta_kind, int agg, const int32_t *nblk, int B, int Hq,
                       int Hkv, int nblk_max, float *scores, hipStream_t s)
{
    const int chunks = (nblk_max + BLOCKS_PER_WG - 1) / BLOCKS_PER_WG;
    const int64_t grid = (int64_t)B * Hkv * chunks;
    if (grid == 0) return SS_OK;
    SS_CHECK_SUPPORTED(grid <= 0x7FFFFFFF, "score: grid too large");
    const auto *qq = static_cast<const uint16_t *>(q);
    const auto *mm = static_cast<const uint8_t *>(meta);
    const dim3 gr((unsigned)grid), bl(256);
    const int G = Hq / Hkv;
    if (meta_kind == SS_META_CUBOID && agg == SS_AGG_MAX)
        ss::launch_lds(score_kernel<0, 0>, gr, bl, kResidencyLds, s, qq, mm, nblk, Hq, Hkv, G, nblk_max, chunks, scores);
    else if (meta_kind == SS_META_CUBOID)
        ss::launch_lds(score_kernel<0, 1>, gr, bl, kResidencyLds, s, qq, mm, nblk, Hq, Hkv, G, nblk_max, chunks, scores);
    else if (agg == SS_AGG_MAX)
        ss::launch_lds(score_kernel<1, 0>, gr, bl, 0, s, qq, mm, nblk, Hq, Hkv, G, nblk_max, chunks, scores);
    else
        ss::launch_lds(score_kernel<1, 1>, gr, bl, 0, s, qq, mm, nblk, Hq, Hkv, G, nblk_max, chunks, scores);
    return check_launch("ss_score_blocks");
}

ss_status check_score_args(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                           int nblk_max, int d, const void *scores, const char *who, int meta_kind, int agg)
{
    SS_CHECK_ARG(meta_kind == SS_META_CUBOID || meta_kind == SS_META_MEAN, "%s: metadata kind %d", who, meta_kind);
    SS_CHECK_ARG(agg == SS_AGG_MAX || agg == SS_AGG_SUM, "%s: aggregation %d", who, agg);
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
    return ss_score_blocks_variant(q, meta, SS_META_CUBOID, SS_AGG_MAX, nblk, B, Hq, Hkv, nblk_max, d, scores,
                                   stream);
}

extern "C" ss_status ss_score_blocks_variant(const void *q, const void *meta, int meta_kind, int agg,
                                             const int32_t *nblk, int B, int Hq, int Hkv, int nblk_max, int d,
                                             float *scores, void *stream)
{
    ss_status st = ss::check_score_args(q, meta, nblk, B, Hq, Hkv, nblk_max, d, scores, "ss_score_blocks", meta_kind,
                                        agg);
    if (st != SS_OK) return st;
    return ss::launch_score(q, meta, meta_kind, agg, nblk, B, Hq, Hkv, nblk_max, scores, ss::as_stream(stream));
}

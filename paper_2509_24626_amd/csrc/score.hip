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
// Each wave reads a tile of 16 consecutive metadata rows as whole contiguous
// 1 KiB pieces with the non-temporal cache policy, stages it in LDS and reads
// its MFMA B fragments from there; there is no cross-lane reduction, the head
// maximum is taken over accumulator registers.  On MI355X the 128k-token
// batch streams at 0.82 of the 8 TB/s peak this way.  Fragments loaded
// straight from HBM (each instruction covering 64-byte pieces of 16 rows)
// reached 0.765 and got slower with the non-temporal policy, since a
// 128-byte line was then requested by two instructions; staged through LDS
// with the default policy they reached 0.765 too.
//
// For cuboid rows the launch reserves LDS up to kResidencyLds per workgroup,
// so that at most two workgroups (8 waves) share a CU: 0.82 that way against
// 0.81 with four.  (With direct fragment loads, before the staging: 0.765
// with two, 0.73 with the eight the registers allow, 0.75 with three, 0.69
// with one.)  Mean-key rows are half as long and launch with no reservation.
#include "internal.hpp"

namespace {

constexpr int D = ss::kHeadDim;
constexpr int TILE = 16;              // blocks per MFMA tile
constexpr int WAVES = 4;
constexpr int TILES_PER_WAVE = 4;
constexpr int BLOCKS_PER_WG = TILE * WAVES * TILES_PER_WAVE;  // 256
// 2 x 54 KiB fit in a CU's 160 KiB of LDS and 3 do not; the 52 KiB left over
// still take one attention workgroup (50.5 KiB) beside two scoring workgroups
constexpr size_t kResidencyLds = 54 * 1024;
// static LDS of the staging buffers for `row` bytes per metadata row
constexpr size_t stage_bytes(int row) { return (size_t)WAVES * TILE * (row / 16 + 1) * 16; }
static_assert(stage_bytes(512) <= kResidencyLds, "staging exceeds the residency budget");
constexpr int kBufferFlags = 0x00020000;  // raw buffer descriptor word 3 for gfx9 (32-bit data)
constexpr int kStream = 2;                // cache policy of the metadata loads: non-temporal

union frag_t {
    bf16x8_t v;
    uint4 u;
    uint16_t h[8];
};

// Lane (L = lane/16, col = lane%16) reads 16-byte chunk c = 4*m + L of
// metadata row `col` of the staged tile for MFMA m.  The A fragments hold
// the matching weights of head `col`.
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

    // each wave stages its 16-row tile through its own LDS region: eight (cuboid)
    // or four (mean key) contiguous 1 KiB non-temporal loads, then the MFMA
    // fragments are read back (row pitch padded by 16 B, so each 16-lane group
    // of a fragment read touches 64 distinct banks); the waves interleave over
    // tiles, so the workgroup walks its rows front to back
    constexpr int NLD = TILE * ROW / 1024;
    constexpr int RU = ROW / 16;  // 16-byte units per row
    constexpr int LR = RU + 1;    // LDS row pitch in 16-byte units
    __shared__ uint4 stage[WAVES][TILE * LR];
    uint4 *my = stage[wave];
    const int lane_id = threadIdx.x & 63;
    uint4 buf[2][NLD];
    auto load_tile = [&](int t, uint4 *r) {
        const uint32_t base = (uint32_t)(j0 + (t * WAVES + wave) * TILE) * ROW + lane_id * 16;
#pragma unroll
        for (int i = 0; i < NLD; ++i)  // rows at or past n read as zero (buffer bounds) and are not stored
            r[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(mrs, base + i * 1024, 0, kStream));
    };

    int ntiles = 0;
    for (int t = 0; t < TILES_PER_WAVE; ++t)
        if (j0 + (t * WAVES + wave) * TILE < n) ntiles = t + 1;
    if (ntiles == 0) return;

    load_tile(0, buf[0]);
#pragma unroll
    for (int t = 0; t < TILES_PER_WAVE; ++t) {
        if (t >= ntiles) break;
        if (t + 1 < ntiles) load_tile(t + 1, buf[(t + 1) & 1]);
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
            const int e = i * 64 + lane_id;
            my[(e / RU) * LR + e % RU] = buf[t & 1][i];
        }
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int m = 0; m < NCH; ++m) {
            frag_t f;
            f.u = my[col * LR + 4 * m + L];
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[m].v, f.v, acc, 0, 0, 0);
        }
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
        ss::launch_lds(score_kernel<0, 0>, gr, bl, kResidencyLds - stage_bytes(512), s, qq, mm, nblk, Hq, Hkv, G, nblk_max, chunks, scores);
    else if (meta_kind == SS_META_CUBOID)
        ss::launch_lds(score_kernel<0, 1>, gr, bl, kResidencyLds - stage_bytes(512), s, qq, mm, nblk, Hq, Hkv, G, nblk_max, chunks, scores);
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

// Appending the decode step's new tokens in HBM (Section 3.2.2: the layer's
// new KV tensor goes into the free slot of each sequence's open block) and
// building a block's metadata when it fills (Section 3.1).
//
// One workgroup per sequence; its four waves take the KV heads in turn.
// For head g the token's K row (256 B) lands in row p of the open record
// and its V values in column p of the channel-major V tile.  When p is the
// block's last row, the wave takes the channel-wise min/max of the tile's K
// rows (rows written by earlier launches, plus the new row from registers)
// and writes the block's metadata row; for mean-key metadata it sums the
// rows in fp64 in token order instead and rounds the mean once to bf16.  After all heads, one thread
// advances the sequence's token count and, on a fill, its block count; only
// this workgroup touches them, so there is no race.  The work is a few
// hundred bytes per head: the kernel is latency-bound by design and runs on
// the caller's stream between the layer's decode and its save.
#include "internal.hpp"

namespace {

constexpr int D = ss::kHeadDim;
constexpr int WAVES = 4;

// order-preserving 16-bit key of a bf16 value under IEEE totalOrder (-0 < +0)
__device__ __forceinline__ uint32_t key16(uint32_t h) { return (h & 0x8000u) ? (~h & 0xFFFFu) : (h | 0x8000u); }
__device__ __forceinline__ uint32_t unkey16(uint32_t k) { return (k & 0x8000u) ? (k & 0x7FFFu) : (~k & 0xFFFFu); }

template <int BLK, int KIND>
__global__ __launch_bounds__(WAVES * 64) void append_kernel(const uint32_t *__restrict__ new_kv, int32_t *len,
                                                            int32_t *nblk, int Hkv, int nblk_max,
                                                            uint8_t *__restrict__ open, uint8_t *__restrict__ meta,
                                                            int32_t *overflow)
{
    constexpr int REC = 2 * BLK * D * 2;
    const int b = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int T = len[b];
    const int j = T / BLK, p = T - j * BLK;
    const bool fills = p == BLK - 1;
    const bool record_meta = fills && j < nblk_max;

    for (int g = wave; g < Hkv; g += WAVES) {
        const int64_t u = (int64_t)b * Hkv + g;
        // lane holds channels 2*lane and 2*lane+1 of K and of V
        const uint32_t *src = new_kv + u * D;  // 2*D bf16 = D words: K words then V words
        const uint32_t k2 = src[lane];
        const uint32_t v2 = src[D / 2 + lane];
        uint8_t *rec = open + u * REC;
        reinterpret_cast<uint32_t *>(rec + (size_t)p * D * 2)[lane] = k2;
        uint16_t *vt = reinterpret_cast<uint16_t *>(rec + (size_t)BLK * D * 2);
        vt[(2 * lane) * BLK + p] = (uint16_t)(v2 & 0xFFFFu);
        vt[(2 * lane + 1) * BLK + p] = (uint16_t)(v2 >> 16);
        if (record_meta && KIND == SS_META_MEAN) {
            // the block's keys summed in fp64 in token order (the new token is the last row)
            const uint32_t *rows = reinterpret_cast<const uint32_t *>(rec);
            double s0 = 0.0, s1 = 0.0;
#pragma unroll 4
            for (int t = 0; t < BLK - 1; ++t) {
                const uint32_t w = rows[t * (D / 2) + lane];
                s0 = s0 + (double)__uint_as_float(w << 16);
                s1 = s1 + (double)__uint_as_float(w & 0xFFFF0000u);
            }
            s0 = s0 + (double)__uint_as_float(k2 << 16);
            s1 = s1 + (double)__uint_as_float(k2 & 0xFFFF0000u);
            uint32_t *m = reinterpret_cast<uint32_t *>(meta + (u * nblk_max + j) * (size_t)(D * 2));
            m[lane] = ss::pack_bf16_rne_f64(s0 * (1.0 / BLK), s1 * (1.0 / BLK));
        } else if (record_meta) {
            uint32_t lo0 = key16(k2 & 0xFFFFu), lo1 = key16(k2 >> 16);
            uint32_t hi0 = lo0, hi1 = lo1;
            const uint32_t *rows = reinterpret_cast<const uint32_t *>(rec);
#pragma unroll 4
            for (int t = 0; t < BLK - 1; ++t) {
                const uint32_t w = rows[t * (D / 2) + lane];
                const uint32_t a = key16(w & 0xFFFFu), c = key16(w >> 16);
                lo0 = min(lo0, a);
                hi0 = max(hi0, a);
                lo1 = min(lo1, c);
                hi1 = max(hi1, c);
            }
            uint32_t *m = reinterpret_cast<uint32_t *>(meta + (u * nblk_max + j) * (size_t)(2 * D * 2));
            m[lane] = unkey16(lo0) | (unkey16(lo1) << 16);
            m[D / 2 + lane] = unkey16(hi0) | (unkey16(hi1) << 16);
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        len[b] = T + 1;
        if (record_meta) nblk[b] = j + 1;
        if (fills && !record_meta && overflow) *overflow = 1;
    }
}

template <int KIND>
void launch_append(int blk, dim3 grid, dim3 block, hipStream_t s, const uint32_t *kv, int32_t *len, int32_t *nblk,
                   int Hkv, int nblk_max, uint8_t *o, uint8_t *m, int32_t *overflow)
{
    switch (blk) {
    case 8: ss::launch(append_kernel<8, KIND>, grid, block, s, kv, len, nblk, Hkv, nblk_max, o, m, overflow); break;
    case 16: ss::launch(append_kernel<16, KIND>, grid, block, s, kv, len, nblk, Hkv, nblk_max, o, m, overflow); break;
    default: ss::launch(append_kernel<32, KIND>, grid, block, s, kv, len, nblk, Hkv, nblk_max, o, m, overflow); break;
    }
}

}  // namespace

extern "C" ss_status ss_append_kv(const void *new_kv, int32_t *len_dev, int32_t *nblk_dev, int B, int Hkv, int blk,
                                  int d, int nblk_max, void *open_blocks, void *meta, int meta_kind, int32_t *overflow,
                                  void *stream)
{
    SS_CHECK_ARG(meta_kind == SS_META_CUBOID || meta_kind == SS_META_MEAN, "ss_append_kv: metadata kind %d",
                 meta_kind);
    SS_CHECK_ARG(B >= 0 && Hkv > 0 && nblk_max >= 0, "ss_append_kv: bad shape B=%d Hkv=%d nblk_max=%d", B, Hkv,
                 nblk_max);
    SS_CHECK_SUPPORTED(d == ss::kHeadDim, "ss_append_kv: d=%d (only 128)", d);
    SS_CHECK_SUPPORTED(ss::supported_blk(blk), "ss_append_kv: blk=%d (8, 16 or 32)", blk);
    if (B == 0) return SS_OK;
    SS_CHECK_ARG(new_kv && len_dev && nblk_dev && open_blocks && meta, "ss_append_kv: null pointer");
    SS_CHECK_ARG(((uintptr_t)new_kv & 3) == 0 && ((uintptr_t)open_blocks & 3) == 0 && ((uintptr_t)meta & 3) == 0,
                 "ss_append_kv: buffers must be 4-byte aligned");
    const hipStream_t s = ss::as_stream(stream);
    const auto *kv = static_cast<const uint32_t *>(new_kv);
    auto *o = static_cast<uint8_t *>(open_blocks);
    auto *m = static_cast<uint8_t *>(meta);
    const dim3 grid(B), block(WAVES * 64);
    if (meta_kind == SS_META_MEAN)
        launch_append<SS_META_MEAN>(blk, grid, block, s, kv, len_dev, nblk_dev, Hkv, nblk_max, o, m, overflow);
    else
        launch_append<SS_META_CUBOID>(blk, grid, block, s, kv, len_dev, nblk_dev, Hkv, nblk_max, o, m, overflow);
    return ss::check_launch("ss_append_kv");
}

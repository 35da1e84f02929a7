// Block metadata (Section 2.2; built when a block fills, Section 3.1): the
// bounding cuboid (channel-wise min and max) of the keys of each KV block,
// or, as the mean-key variant, the mean of the block's keys.
//
// Cuboids: one wave per 64/blk consecutive block records.  A K tile is blk
// rows of 128 bf16 channels (256 B per row); each lane loads 16 B (8
// channels) of one row per step, so one wave-wide load covers 4 rows, and
// all 16 loads of the wave's records are issued before any is reduced (a
// wave per single record kept too few bytes in flight).  Min and max run on
// 16-bit totalOrder keys, two channels per 32-bit word, then across the four
// row groups of the wave.  Lanes 0..15 write lo and hi.
#include "internal.hpp"

namespace {

// bf16 bits -> 16-bit key with unsigned order equal to IEEE totalOrder,
// two lanes per word: negative values flip all bits, others set the sign.
__device__ __forceinline__ uint32_t to_key2(uint32_t w)
{
    uint32_t s = (w >> 15) & 0x00010001u;
    return w ^ (0x80008000u | (s * 0x7FFFu));
}

__device__ __forceinline__ uint32_t from_key2(uint32_t k)
{
    uint32_t s = (k >> 15) & 0x00010001u;  // set for non-negative values
    return k ^ (0xFFFFFFFFu ^ (s * 0x7FFFu));
}

typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t min2(uint32_t a, uint32_t b)
{
    u16x2_t r = __builtin_elementwise_min(__builtin_bit_cast(u16x2_t, a), __builtin_bit_cast(u16x2_t, b));
    return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ uint32_t max2(uint32_t a, uint32_t b)
{
    u16x2_t r = __builtin_elementwise_max(__builtin_bit_cast(u16x2_t, a), __builtin_bit_cast(u16x2_t, b));
    return __builtin_bit_cast(uint32_t, r);
}

template <int BLK>
__global__ __launch_bounds__(256) void meta_kernel(const uint8_t *__restrict__ kv_base,
                                                   const int64_t *__restrict__ unit_off,
                                                   const int32_t *__restrict__ nblk, int Hkv, int nblk_max,
                                                   int64_t total_blocks, int64_t block_stride, int64_t row_stride,
                                                   uint16_t *__restrict__ meta)
{
    constexpr int D = ss::kHeadDim;
    constexpr int BPW = 64 / BLK;  // block records per wave: 16 loads of 16 B per lane in flight
    constexpr int LPB = BLK / 4;   // wave-wide loads per K tile (4 rows each)
    const int lane = threadIdx.x & 63;
    const int64_t id0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * BPW;
    const int row0 = lane >> 4;          // 0..3
    const int cbyte = (lane & 15) * 16;  // 8 channels

    // issue every load of the wave's records before reducing any of them
    uint4 v[BPW][LPB];
    bool live[BPW];
    int64_t u_of[BPW];
    int j_of[BPW];
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
        const int64_t id = id0 + b;  // wave-uniform
        live[b] = id < total_blocks;
        u_of[b] = 0;
        j_of[b] = 0;
        if (live[b]) {
            const int64_t u = id / nblk_max;
            const int j = (int)(id - u * nblk_max);
            int n = nblk[u / Hkv];
            n = n < 0 ? 0 : (n > nblk_max ? nblk_max : n);
            live[b] = j < n;
            u_of[b] = u;
            j_of[b] = j;
        }
        if (live[b]) {
            const uint8_t *rec = kv_base + unit_off[u_of[b]] + (int64_t)j_of[b] * block_stride;
#pragma unroll
            for (int r = 0; r < LPB; ++r)
                v[b][r] = *reinterpret_cast<const uint4 *>(rec + (4 * r + row0) * row_stride + cbyte);
        }
    }
#pragma unroll
    for (int b = 0; b < BPW; ++b) {
        if (!live[b]) continue;
        uint32_t lo[4], hi[4];
        lo[0] = hi[0] = to_key2(v[b][0].x);
        lo[1] = hi[1] = to_key2(v[b][0].y);
        lo[2] = hi[2] = to_key2(v[b][0].z);
        lo[3] = hi[3] = to_key2(v[b][0].w);
#pragma unroll
        for (int r = 1; r < LPB; ++r) {
            const uint32_t k0 = to_key2(v[b][r].x), k1 = to_key2(v[b][r].y), k2 = to_key2(v[b][r].z),
                           k3 = to_key2(v[b][r].w);
            lo[0] = min2(lo[0], k0); hi[0] = max2(hi[0], k0);
            lo[1] = min2(lo[1], k1); hi[1] = max2(hi[1], k1);
            lo[2] = min2(lo[2], k2); hi[2] = max2(hi[2], k2);
            lo[3] = min2(lo[3], k3); hi[3] = max2(hi[3], k3);
        }
#pragma unroll
        for (int x = 16; x <= 32; x <<= 1) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                lo[i] = min2(lo[i], (uint32_t)__shfl_xor((int)lo[i], x));
                hi[i] = max2(hi[i], (uint32_t)__shfl_xor((int)hi[i], x));
            }
        }
        if (lane < 16) {
            uint16_t *m = meta + ((int64_t)u_of[b] * nblk_max + j_of[b]) * (2 * D);
            const uint4 l4 = make_uint4(from_key2(lo[0]), from_key2(lo[1]), from_key2(lo[2]), from_key2(lo[3]));
            const uint4 h4 = make_uint4(from_key2(hi[0]), from_key2(hi[1]), from_key2(hi[2]), from_key2(hi[3]));
            *reinterpret_cast<uint4 *>(m + lane * 8) = l4;
            *reinterpret_cast<uint4 *>(m + D + lane * 8) = h4;
        }
    }
}

// Mean key of each block: one wave per block record, each lane two
// channels; rows are summed in fp64 in token order (each wave-wide load is
// one contiguous 256-byte row; the sum of blk bf16 keys is exact unless
// their magnitudes span more than about 2^40), scaled by 1/blk (exact) and
// rounded once to bf16, ties to even.
template <int BLK>
__global__ __launch_bounds__(256) void meta_mean_kernel(const uint8_t *__restrict__ kv_base,
                                                        const int64_t *__restrict__ unit_off,
                                                        const int32_t *__restrict__ nblk, int Hkv, int nblk_max,
                                                        int64_t total_blocks, int64_t block_stride,
                                                        int64_t row_stride, uint32_t *__restrict__ meta)
{
    constexpr int D = ss::kHeadDim;
    const int lane = threadIdx.x & 63;
    const int64_t id = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (id >= total_blocks) return;
    const int64_t u = id / nblk_max;
    const int j = (int)(id - u * nblk_max);
    int n = nblk[u / Hkv];
    n = n < 0 ? 0 : (n > nblk_max ? nblk_max : n);
    if (j >= n) return;
    const uint8_t *rec = kv_base + unit_off[u] + (int64_t)j * block_stride;
    uint32_t w[BLK];
#pragma unroll
    for (int t = 0; t < BLK; ++t) w[t] = reinterpret_cast<const uint32_t *>(rec + t * row_stride)[lane];
    double s0 = 0.0, s1 = 0.0;
#pragma unroll
    for (int t = 0; t < BLK; ++t) {
        s0 = s0 + (double)__uint_as_float(w[t] << 16);
        s1 = s1 + (double)__uint_as_float(w[t] & 0xFFFF0000u);
    }
    meta[(u * nblk_max + j) * (D / 2) + lane] = ss::pack_bf16_rne_f64(s0 * (1.0 / BLK), s1 * (1.0 / BLK));
}

}  // namespace

extern "C" ss_status ss_build_metadata_strided(const void *kv_base, const int64_t *unit_off, const int32_t *nblk,
                                               int B, int Hkv, int nblk_max, int blk, int d, int64_t block_stride,
                                               int64_t row_stride, int meta_kind, void *meta, void *stream)
{
    SS_CHECK_ARG(B >= 0 && Hkv > 0 && nblk_max >= 0, "ss_build_metadata: bad shape B=%d Hkv=%d nblk_max=%d", B,
                 Hkv, nblk_max);
    SS_CHECK_ARG(meta_kind == SS_META_CUBOID || meta_kind == SS_META_MEAN, "ss_build_metadata: metadata kind %d",
                 meta_kind);
    SS_CHECK_SUPPORTED(d == ss::kHeadDim, "ss_build_metadata: d=%d (only 128)", d);
    SS_CHECK_SUPPORTED(ss::supported_blk(blk), "ss_build_metadata: blk=%d (8, 16 or 32)", blk);
    SS_CHECK_SUPPORTED(nblk_max <= ss::kMaxBlocks, "ss_build_metadata: nblk_max=%d > %d", nblk_max, ss::kMaxBlocks);
    SS_CHECK_ARG(block_stride > 0 && row_stride > 0 && block_stride % 16 == 0 && row_stride % 16 == 0,
                 "ss_build_metadata: strides %lld, %lld must be positive multiples of 16", (long long)block_stride,
                 (long long)row_stride);
    const int64_t total = (int64_t)B * Hkv * nblk_max;
    if (total == 0) return SS_OK;
    SS_CHECK_ARG(kv_base && unit_off && nblk && meta, "ss_build_metadata: null pointer");
    SS_CHECK_ARG(((uintptr_t)kv_base & 15) == 0 && ((uintptr_t)meta & 15) == 0,
                 "ss_build_metadata: kv_base and meta must be 16-byte aligned");
    // cuboids: 4 waves of 64/blk records per workgroup; mean keys: 4 records
    const int64_t per_wg = meta_kind == SS_META_CUBOID ? 4 * (64 / blk) : 4;
    const int64_t grid = (total + per_wg - 1) / per_wg;
    SS_CHECK_SUPPORTED(grid <= 0x7FFFFFFF, "ss_build_metadata: too many blocks");
    hipStream_t s = ss::as_stream(stream);
    const uint8_t *kv = static_cast<const uint8_t *>(kv_base);
    const dim3 gr((unsigned)grid), bl(256);
    const int64_t bs = block_stride, rs = row_stride;
    if (meta_kind == SS_META_CUBOID) {
        uint16_t *m = static_cast<uint16_t *>(meta);
        switch (blk) {
        case 8: ss::launch(meta_kernel<8>, gr, bl, s, kv, unit_off, nblk, Hkv, nblk_max, total, bs, rs, m); break;
        case 16: ss::launch(meta_kernel<16>, gr, bl, s, kv, unit_off, nblk, Hkv, nblk_max, total, bs, rs, m); break;
        default: ss::launch(meta_kernel<32>, gr, bl, s, kv, unit_off, nblk, Hkv, nblk_max, total, bs, rs, m); break;
        }
    } else {
        uint32_t *m = static_cast<uint32_t *>(meta);
        switch (blk) {
        case 8: ss::launch(meta_mean_kernel<8>, gr, bl, s, kv, unit_off, nblk, Hkv, nblk_max, total, bs, rs, m); break;
        case 16: ss::launch(meta_mean_kernel<16>, gr, bl, s, kv, unit_off, nblk, Hkv, nblk_max, total, bs, rs, m); break;
        default: ss::launch(meta_mean_kernel<32>, gr, bl, s, kv, unit_off, nblk, Hkv, nblk_max, total, bs, rs, m); break;
        }
    }
    return ss::check_launch("ss_build_metadata");
}

extern "C" ss_status ss_build_metadata(const void *kv_base, const int64_t *unit_off, const int32_t *nblk, int B,
                                       int Hkv, int nblk_max, int blk, int d, void *meta, void *stream)
{
    const int64_t rec = 2LL * blk * d * 2;  // block records: K rows of d bf16 each
    return ss_build_metadata_strided(kv_base, unit_off, nblk, B, Hkv, nblk_max, blk, d, rec, (int64_t)d * 2,
                                     SS_META_CUBOID, meta, stream);
}

extern "C" ss_status ss_build_metadata_mean(const void *kv_base, const int64_t *unit_off, const int32_t *nblk,
                                            int B, int Hkv, int nblk_max, int blk, int d, void *meta, void *stream)
{
    const int64_t rec = 2LL * blk * d * 2;
    return ss_build_metadata_strided(kv_base, unit_off, nblk, B, Hkv, nblk_max, blk, d, rec, (int64_t)d * 2,
                                     SS_META_MEAN, meta, stream);
}

// GPU-direct loading of missed KV blocks (Section 3.2.1, FlashH2D): a single
// kernel copies every missed block record from the pinned, device-mapped
// DRAM pool into its HBM cache slot, instead of one memcpy per block.
//
// Each workgroup copies whole records (4, 8 or 16 KiB).  Every thread issues
// all of its 16-byte loads for RPI records before the first store, so each
// wave keeps RPI*CH KiB of host-link reads in flight; workgroups stride over
// the miss list.  The grid is small on purpose: a launch-shape sweep on
// MI355X (8 GiB pinned pool, 16384 random 8 KiB records) measured 57.1-57.5
// GB/s with 16-128 workgroups alone (a contiguous hipMemcpy reaches 57.0)
// but only 54.5 GB/s with 2048.  Inside the pipelined decode step, where two
// gathers overlap beside the scoring and attention kernels, 32 workgroups
// per launch of 8 KiB records gave the shortest step (2.50 ms on the 128k
// workload, against 2.58-2.63 with 64, 2.70 with 128, 2.55-2.64 with 16-24
// and 3.0 with 8); the grid scales inversely with the record size so that
// each launch keeps the same bytes in flight.
// Loads and stores both carry the non-temporal cache policy: each record
// passes through once (inside the decode step the stores measured 0.3-0.5%
// more tokens/s than with the default policy, on the 128k and the 32-layer
// workloads alike).
// The decode step also hands the kernel a small side copy (the group's slot
// table, from mapped host memory to HBM) so that no copy-engine transfer,
// and no cross-engine synchronisation, sits between resolve and attention.
#include <climits>

#include "internal.hpp"

namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <int CH, int RPI>  // 16-byte chunks per thread per record; records per iteration
__global__ __launch_bounds__(256) void gather_kernel(const int4 *__restrict__ miss, int64_t n_miss,
                                                     const uint8_t *__restrict__ pool,
                                                     const int64_t *__restrict__ pool_off,
                                                     uint8_t *__restrict__ cache,
                                                     const int64_t *__restrict__ cache_off,
                                                     const int32_t *__restrict__ nblk,
                                                     const int32_t *__restrict__ capacity, int B, int Hkv,
                                                     const int32_t *__restrict__ copy_src,
                                                     int32_t *__restrict__ copy_dst, int64_t copy_n)
{
    constexpr int64_t REC = 4096LL * CH;
    const int t = threadIdx.x;
    for (int64_t i = (int64_t)blockIdx.x * 256 + t; i < copy_n; i += (int64_t)gridDim.x * 256) copy_dst[i] = copy_src[i];
    for (int64_t m0 = (int64_t)blockIdx.x * RPI; m0 < n_miss; m0 += (int64_t)gridDim.x * RPI) {
        const u32x4_t *src[RPI];
        u32x4_t *dst[RPI];
        bool ok[RPI];
#pragma unroll
        for (int r = 0; r < RPI; ++r) {
            ok[r] = false;
            src[r] = nullptr;
            dst[r] = nullptr;
            const int64_t mi = m0 + r;
            if (mi < n_miss) {
                const int4 e = miss[mi];  // (b, g, block, slot)
                if (e.x >= 0 && e.x < B && e.y >= 0 && e.y < Hkv) {
                    const int64_t u = (int64_t)e.x * Hkv + e.y;
                    if (e.z >= 0 && e.z < nblk[e.x] && e.w >= 0 && e.w < capacity[u]) {
                        ok[r] = true;
                        src[r] = reinterpret_cast<const u32x4_t *>(pool + pool_off[u] + (int64_t)e.z * REC);
                        dst[r] = reinterpret_cast<u32x4_t *>(cache + cache_off[u] + (int64_t)e.w * REC);
                    }
                }
            }
        }
        u32x4_t v[RPI][CH];
#pragma unroll
        for (int r = 0; r < RPI; ++r)
            if (ok[r]) {
#pragma unroll
                for (int c = 0; c < CH; ++c) v[r][c] = __builtin_nontemporal_load(src[r] + c * 256 + t);
            }
#pragma unroll
        for (int r = 0; r < RPI; ++r)
            if (ok[r]) {
#pragma unroll
                for (int c = 0; c < CH; ++c) __builtin_nontemporal_store(v[r][c], &dst[r][c * 256 + t]);
            }
    }
}

// The same copy for miss rows kept per unit: unit u's counts[u] rows start at
// rows + u * k * 4 (the device resolve writes them so).  The units' counts
// are summed into a prefix in LDS, UCH units at a time; the workgroups then
// stride over the flat miss index as gather_kernel does (RPI records each,
// neighbouring workgroups on neighbouring records, so the load is balanced
// whatever the spread of misses over units) and find each index's unit with a
// cursor that only moves forward, 64 prefix entries per wave ballot.
template <int CH, int RPI>
__global__ __launch_bounds__(256) void gather_units_kernel(const int4 *__restrict__ rows_base,
                                                           const int32_t *__restrict__ counts, int u0, int u1, int k,
                                                           const uint8_t *__restrict__ pool,
                                                           const int64_t *__restrict__ pool_off,
                                                           uint8_t *__restrict__ cache,
                                                           const int64_t *__restrict__ cache_off,
                                                           const int32_t *__restrict__ nblk,
                                                           const int32_t *__restrict__ capacity, int B, int Hkv)
{
    constexpr int64_t REC = 4096LL * CH;
    constexpr int UCH = 1024, PER = UCH / 256;
    __shared__ int s_pre[UCH + 1];  // s_pre[i]: misses of the chunk's units before unit i
    __shared__ int s_wave[4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    for (int c0 = u0; c0 < u1; c0 += UCH) {
        const int n = min(UCH, u1 - c0);
        int c[PER], sum = 0;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int i = t * PER + j;
            int v = i < n ? counts[c0 + i] : 0;
            v = v < 0 ? 0 : (v > k ? k : v);
            c[j] = v;
            sum += v;
        }
        int incl = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o);
            if (lane >= o) incl += y;
        }
        if (lane == 63) s_wave[wave] = incl;
        __syncthreads();
        int run = incl - sum;
        for (int w = 0; w < wave; ++w) run += s_wave[w];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            s_pre[t * PER + j] = run;
            run += c[j];
        }
        if (t == 255) s_pre[UCH] = run;  // the chunk's total: units past n count 0
        __syncthreads();
        const int total = s_pre[UCH];
        int cur = 0;  // s_pre[cur] <= m < s_pre[cur + 1] for the last index m placed
        for (int m0 = blockIdx.x * RPI; m0 < total; m0 += gridDim.x * RPI) {
            const u32x4_t *src[RPI];
            u32x4_t *dst[RPI];
            bool ok[RPI];
#pragma unroll
            for (int r = 0; r < RPI; ++r) {
                ok[r] = false;
                src[r] = nullptr;
                dst[r] = nullptr;
                const int m = m0 + r;
                if (m < total) {  // the same m in every lane: the ballots below are uniform
                    for (;;) {
                        const int j = cur + 1 + lane;
                        const int v = j <= UCH ? s_pre[j] : INT_MAX;
                        const unsigned long long hit = __ballot(v > m);
                        if (hit) {
                            cur += __builtin_ctzll(hit);
                            break;
                        }
                        cur += 64;
                    }
                    const int4 e = rows_base[(int64_t)(c0 + cur) * k + (m - s_pre[cur])];  // (b, g, block, slot)
                    if (e.x >= 0 && e.x < B && e.y >= 0 && e.y < Hkv) {
                        const int64_t u = (int64_t)e.x * Hkv + e.y;
                        if (e.z >= 0 && e.z < nblk[e.x] && e.w >= 0 && e.w < capacity[u]) {
                            ok[r] = true;
                            src[r] = reinterpret_cast<const u32x4_t *>(pool + pool_off[u] + (int64_t)e.z * REC);
                            dst[r] = reinterpret_cast<u32x4_t *>(cache + cache_off[u] + (int64_t)e.w * REC);
                        }
                    }
                }
            }
            u32x4_t v[RPI][CH];
#pragma unroll
            for (int r = 0; r < RPI; ++r)
                if (ok[r]) {
#pragma unroll
                    for (int c2 = 0; c2 < CH; ++c2) v[r][c2] = __builtin_nontemporal_load(src[r] + c2 * 256 + t);
                }
#pragma unroll
            for (int r = 0; r < RPI; ++r)
                if (ok[r]) {
#pragma unroll
                    for (int c2 = 0; c2 < CH; ++c2) __builtin_nontemporal_store(v[r][c2], &dst[r][c2 * 256 + t]);
                }
        }
        __syncthreads();  // every wave is done with s_pre before the next chunk overwrites it
    }
}

template <int CH>
void launch_variant(const int4 *miss, int64_t n_miss, const uint8_t *pool, const int64_t *pool_off, uint8_t *cache,
            const int64_t *cache_off, const int32_t *nblk, const int32_t *cap, int B, int Hkv,
            const int32_t *copy_src, int32_t *copy_dst, int64_t copy_n, hipStream_t s)
{
    constexpr int RPI = 2;
    int64_t blocks = (n_miss + RPI - 1) / RPI;
    // about 512 KiB of records in flight per launch: 32 workgroups of two 8 KiB
    // records, 64 of 4 KiB, 16 of 16 KiB
    const int64_t max_blocks = 32 * 2 / CH;
    if (blocks > max_blocks) blocks = max_blocks;
    if (blocks < 1) blocks = 1;
    ss::launch(gather_kernel<CH, RPI>, dim3((unsigned)blocks), dim3(256), s, miss, n_miss, pool, pool_off, cache,
               cache_off, nblk, cap, B, Hkv, copy_src, copy_dst, copy_n);
}

template <int CH>
void launch_units_variant(const int4 *rows, const int32_t *counts, int u0, int u1, int k, const uint8_t *pool,
                          const int64_t *pool_off, uint8_t *cache, const int64_t *cache_off, const int32_t *nblk,
                          const int32_t *cap, int B, int Hkv, hipStream_t s)
{
    constexpr int RPI = 2;
    // as launch_variant: about 512 KiB in flight (the miss total is known only on the GPU)
    const int64_t blocks = 32 * 2 / CH;
    ss::launch(gather_units_kernel<CH, RPI>, dim3((unsigned)blocks), dim3(256), s, rows, counts, u0, u1, k, pool,
               pool_off, cache, cache_off, nblk, cap, B, Hkv);
}

}  // namespace

namespace ss {

// Gather of the miss rows a device resolve left per unit, for units [u0, u1).
ss_status launch_gather_units(const int32_t *rows, const int32_t *counts, int u0, int u1, int k,
                              const void *pool_base, const int64_t *pool_off, void *cache_base,
                              const int64_t *cache_off, const int32_t *nblk, const int32_t *capacity, int B, int Hkv,
                              size_t record_bytes, hipStream_t s)
{
    if (u1 <= u0) return SS_OK;
    const int4 *r = reinterpret_cast<const int4 *>(rows);
    const uint8_t *p = static_cast<const uint8_t *>(pool_base);
    uint8_t *c = static_cast<uint8_t *>(cache_base);
    switch (record_bytes) {
    case 4096: launch_units_variant<1>(r, counts, u0, u1, k, p, pool_off, c, cache_off, nblk, capacity, B, Hkv, s); break;
    case 8192: launch_units_variant<2>(r, counts, u0, u1, k, p, pool_off, c, cache_off, nblk, capacity, B, Hkv, s); break;
    default: launch_units_variant<4>(r, counts, u0, u1, k, p, pool_off, c, cache_off, nblk, capacity, B, Hkv, s); break;
    }
    return check_launch("ss_decode_layer_dev (gather)");
}

// Gather plus an optional word copy copy_src[0, copy_n) -> copy_dst (both
// device-accessible); launches only if there is work.
ss_status launch_gather(const int32_t *miss, int64_t n_miss, const void *pool_base, const int64_t *pool_off,
                        void *cache_base, const int64_t *cache_off, const int32_t *nblk, const int32_t *capacity,
                        int B, int Hkv, size_t record_bytes, const int32_t *copy_src, int32_t *copy_dst,
                        int64_t copy_n, hipStream_t s)
{
    if (n_miss == 0 && copy_n == 0) return SS_OK;
    const int4 *m = reinterpret_cast<const int4 *>(miss);
    const uint8_t *p = static_cast<const uint8_t *>(pool_base);
    uint8_t *c = static_cast<uint8_t *>(cache_base);
    switch (record_bytes) {
    case 4096: launch_variant<1>(m, n_miss, p, pool_off, c, cache_off, nblk, capacity, B, Hkv, copy_src, copy_dst, copy_n, s); break;
    case 8192: launch_variant<2>(m, n_miss, p, pool_off, c, cache_off, nblk, capacity, B, Hkv, copy_src, copy_dst, copy_n, s); break;
    default: launch_variant<4>(m, n_miss, p, pool_off, c, cache_off, nblk, capacity, B, Hkv, copy_src, copy_dst, copy_n, s); break;
    }
    return check_launch("ss_gather_blocks");
}

}  // namespace ss

extern "C" ss_status ss_gather_blocks(const int32_t *miss, int64_t n_miss, const void *pool_base,
                                      const int64_t *pool_off, void *cache_base, const int64_t *cache_off,
                                      const int32_t *nblk, const int32_t *capacity, int B, int Hkv,
                                      size_t record_bytes, void *stream)
{
    SS_CHECK_ARG(n_miss >= 0 && B >= 0 && Hkv > 0, "ss_gather_blocks: bad shape n_miss=%lld B=%d Hkv=%d",
                 (long long)n_miss, B, Hkv);
    SS_CHECK_SUPPORTED(record_bytes == 4096 || record_bytes == 8192 || record_bytes == 16384,
                       "ss_gather_blocks: record_bytes=%zu (blk 8/16/32 at d=128)", record_bytes);
    if (n_miss == 0) return SS_OK;
    SS_CHECK_ARG(miss && pool_base && pool_off && cache_base && cache_off && nblk && capacity,
                 "ss_gather_blocks: null pointer");
    SS_CHECK_ARG((reinterpret_cast<uintptr_t>(miss) & 15) == 0, "ss_gather_blocks: miss list not 16-byte aligned");
    return ss::launch_gather(miss, n_miss, pool_base, pool_off, cache_base, cache_off, nblk, capacity, B, Hkv,
                             record_bytes, nullptr, nullptr, 0, ss::as_stream(stream));
}

// Top-k block selection per (sequence, KV head) (Section 2.2), ties to the
// lower block index, output in ascending block order.
//
// One workgroup per unit.  Thread t owns the R consecutive scores
// [t*R, t*R+R) in registers as 32-bit keys whose unsigned order is the
// float order (-0 folded onto +0; padding gets key 0, below every float).
// A radix select finds the m-th largest key T (m = min(k, n)) 8 bits at a
// time, starting below the bits shared by the smallest and largest key so
// that the LDS histogram is spread from the first pass.  The selection is
// then {key > T} plus the first (m - #{key > T}) keys equal to T in index
// order; because threads own consecutive indices, two block-wide exclusive
// scans give every thread its output position in ascending block order.
#include "internal.hpp"

namespace {

__device__ __forceinline__ uint32_t score_key(float f)
{
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7FFFFFFFu) == 0) b = 0;  // -0 == +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

template <int NT>
struct block_scan {
    static constexpr int NW = NT / 64;
    int *wave_tot;  // LDS [NW]

    // exclusive prefix sum over the block in thread order; *total = sum
    __device__ int exclusive(int v, int *total)
    {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        int x = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            int y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (lane == 63) wave_tot[wave] = x;
        __syncthreads();
        int before = 0, all = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            int t = wave_tot[w];
            before += (w < wave) ? t : 0;
            all += t;
        }
        __syncthreads();
        *total = all;
        return before + x - v;
    }
};

template <int NT, int R>
__global__ __launch_bounds__(NT) void topk_kernel(const float *__restrict__ scores, const int32_t *__restrict__ nblk,
                                                  int Hkv, int nblk_max, int k, int32_t *__restrict__ sel,
                                                  int32_t *__restrict__ mirror)
{
    __shared__ int hist[256];
    __shared__ int wave_tot[NT / 64];
    __shared__ uint32_t red_min[NT / 64], red_max[NT / 64];
    __shared__ int pick[2];

    const int u = blockIdx.x;
    const int b = u / Hkv;
    int n = nblk[b];
    n = n < 0 ? 0 : (n > nblk_max ? nblk_max : n);
    const int m = k < n ? k : n;
    int32_t *out = sel + (int64_t)u * k;
    int32_t *out2 = mirror ? mirror + (int64_t)u * k : nullptr;  // copy in mapped host memory
    const float *s = scores + (int64_t)u * nblk_max;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;

    for (int i = m + t; i < k; i += NT) {
        out[i] = -1;
        if (out2) out2[i] = -1;
    }
    if (m == 0) return;

    uint32_t key[R];
    const int base = t * R;
#pragma unroll
    for (int r = 0; r < R; ++r) key[r] = (base + r < n) ? score_key(s[base + r]) : 0u;

    // smallest and largest valid key
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (base + r < n) {
            kmin = min(kmin, key[r]);
            kmax = max(kmax, key[r]);
        }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o));
        kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o));
    }
    if (lane == 0) {
        red_min[wave] = kmin;
        red_max[wave] = kmax;
    }
    __syncthreads();
    kmin = red_min[0];
    kmax = red_max[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) {
        kmin = min(kmin, red_min[w]);
        kmax = max(kmax, red_max[w]);
    }

    // radix select of the m-th largest key below the shared prefix
    uint32_t prefix = kmin & kmax, pmask = 0;
    int krem = m;
    if (kmin != kmax) {
        const int top = 31 - __clz(kmin ^ kmax);  // highest differing bit
        pmask = ~((2u << top) - 1u);              // bits above it are shared
        if (top == 31) pmask = 0;
        prefix = kmax & pmask;
        for (int hi_bit = top; hi_bit >= 0; hi_bit -= 8) {
            const int lo_bit = hi_bit >= 7 ? hi_bit - 7 : 0;
            const int width = hi_bit - lo_bit + 1;
            const uint32_t dmask = (1u << width) - 1u;
            for (int i = t; i < 256; i += NT) hist[i] = 0;
            __syncthreads();
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (base + r < n && (key[r] & pmask) == prefix) atomicAdd(&hist[(key[r] >> lo_bit) & dmask], 1);
            __syncthreads();
            if (wave == 0) {
                // lane l holds digits 255-4l .. 252-4l (descending order)
                int c[4], sum = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    c[i] = hist[255 - 4 * lane - i];
                    sum += c[i];
                }
                int incl = sum;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    int y = __shfl_up(incl, o);
                    if (lane >= o) incl += y;
                }
                int above = incl - sum;  // keys in higher digits than this lane's
                // the digit where the krem-th largest falls
                if (above < krem && krem <= incl) {
                    int acc = above;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        if (acc < krem && krem <= acc + c[i]) {
                            pick[0] = 255 - 4 * lane - i;
                            pick[1] = krem - acc;
                        }
                        acc += c[i];
                    }
                }
            }
            __syncthreads();
            const uint32_t digit = (uint32_t)pick[0];
            krem = pick[1];
            prefix |= digit << lo_bit;
            pmask |= dmask << lo_bit;
            __syncthreads();
        }
    }
    const uint32_t T = prefix;  // the m-th largest key; take krem keys equal to T

    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        n_gt += (key[r] > T) ? 1 : 0;
        n_eq += (key[r] == T && base + r < n) ? 1 : 0;
    }
    block_scan<NT> scan{wave_tot};
    int tot;
    const int eq_before = scan.exclusive(n_eq, &tot);
    int eq_quota = krem - eq_before;
    eq_quota = eq_quota < 0 ? 0 : (eq_quota > n_eq ? n_eq : eq_quota);
    int pos = scan.exclusive(n_gt + eq_quota, &tot);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool eq = key[r] == T && base + r < n;
        const bool take = key[r] > T || (eq && eq_quota > 0);
        if (eq && eq_quota > 0) --eq_quota;
        if (take && pos < m) {  // pos < m always holds; the guard keeps writes in range
            out[pos] = base + r;
            if (out2) out2[pos] = base + r;
            ++pos;
        }
    }
}

template <int NT, int R>
void launch_variant(const float *scores, const int32_t *nblk, int units, int Hkv, int nblk_max, int k, int32_t *sel,
            int32_t *mirror, hipStream_t s)
{
    ss::launch(topk_kernel<NT, R>, dim3(units), dim3(NT), s, scores, nblk, Hkv, nblk_max, k, sel, mirror);
}

}  // namespace

namespace ss {

// `mirror` (nullable): a second copy of the selection, e.g. in mapped host memory
ss_status launch_topk(const float *scores, const int32_t *nblk, int B, int Hkv, int nblk_max, int k, int32_t *sel,
                      int32_t *mirror, hipStream_t s)
{
    const int units = B * Hkv;
    if (units == 0) return SS_OK;
    // Workgroup width per size class: 512 threads from 2048 blocks up, so that
    // each thread holds at most 16 keys.  On MI355X (k = 128) this took a
    // 16-unit launch over 8192 blocks from 14.2 to 11.0 us and the 512-unit
    // one from 26.3 to 18.0 us against 256 threads of 32 keys, and 1024
    // threads of 8 keys measured 11.4 and 22.9 us.
    if (nblk_max <= 256 * 4) launch_variant<256, 4>(scores, nblk, units, Hkv, nblk_max, k, sel, mirror, s);
    else if (nblk_max <= 512 * 4) launch_variant<512, 4>(scores, nblk, units, Hkv, nblk_max, k, sel, mirror, s);
    else if (nblk_max <= 512 * 8) launch_variant<512, 8>(scores, nblk, units, Hkv, nblk_max, k, sel, mirror, s);
    else if (nblk_max <= 512 * 16) launch_variant<512, 16>(scores, nblk, units, Hkv, nblk_max, k, sel, mirror, s);
    else if (nblk_max <= 1024 * 16) launch_variant<1024, 16>(scores, nblk, units, Hkv, nblk_max, k, sel, mirror, s);
    else launch_variant<1024, 64>(scores, nblk, units, Hkv, nblk_max, k, sel, mirror, s);
    return check_launch("ss_select_topk");
}

}  // namespace ss

extern "C" ss_status ss_select_topk(const float *scores, const int32_t *nblk, int B, int Hkv, int nblk_max, int k,
                                    int32_t *sel, void *stream)
{
    SS_CHECK_ARG(B >= 0 && Hkv > 0 && nblk_max >= 0 && k > 0, "ss_select_topk: bad shape B=%d Hkv=%d nblk_max=%d k=%d",
                 B, Hkv, nblk_max, k);
    SS_CHECK_SUPPORTED(nblk_max <= ss::kMaxBlocks, "ss_select_topk: nblk_max=%d > %d", nblk_max, ss::kMaxBlocks);
    if (B == 0) return SS_OK;
    SS_CHECK_ARG(nblk && sel && (scores || nblk_max == 0), "ss_select_topk: null pointer");
    return ss::launch_topk(scores, nblk, B, Hkv, nblk_max, k, sel, nullptr, ss::as_stream(stream));
}

extern "C" size_t ss_score_topk_workspace(int B, int Hq, int Hkv, int nblk_max, int d, int k)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || d != ss::kHeadDim || nblk_max < 0 || k <= 0) return 0;
    return (size_t)B * Hkv * nblk_max * sizeof(float);
}

extern "C" ss_status ss_score_topk(const void *q, const void *meta, const int32_t *nblk, int B, int Hq, int Hkv,
                                   int nblk_max, int d, int k, float *scores, int32_t *sel, void *stream)
{
    ss_status st = ss::check_score_args(q, meta, nblk, B, Hq, Hkv, nblk_max, d, scores, "ss_score_topk",
                                        SS_META_CUBOID, SS_AGG_MAX);
    if (st != SS_OK) return st;
    SS_CHECK_ARG(k > 0, "ss_score_topk: k=%d", k);
    if (B == 0) return SS_OK;
    SS_CHECK_ARG(sel, "ss_score_topk: null sel");
    hipStream_t s = ss::as_stream(stream);
    st = ss::launch_score(q, meta, SS_META_CUBOID, SS_AGG_MAX, nblk, B, Hq, Hkv, nblk_max, scores, s);
    if (st != SS_OK) return st;
    return ss::launch_topk(scores, nblk, B, Hkv, nblk_max, k, sel, nullptr, s);
}

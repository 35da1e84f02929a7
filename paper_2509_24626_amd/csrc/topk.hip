// Top-k block selection per (sequence, KV head) (Section 2.2), ties to the
// lower block index, output in ascending block order.
//
// One workgroup per unit.  Thread t owns the R consecutive scores
// [t*R, t*R+R) in registers as 32-bit keys whose unsigned order is the
// float order (-0 folded onto +0; padding gets key 0, below every float).
// The row is read with coalesced loads (each wave instruction 256
// consecutive bytes) and handed to its owners through LDS; the loads are
// issued before the unit's block count arrives (the row holds nblk_max
// scores, so every load is in bounds).  A radix select finds the m-th
// largest key (m = min(k, n)) 8 bits at a time, starting below the bits
// shared by the smallest and largest key.  The first pass counts every key,
// and its digits are often a handful of values (the sign and exponent bits
// of similar scores); LDS atomics from one wave instruction to the same
// address are processed one lane at a time, so that pass counts into 16
// interleaved copies of the histogram (lane l adds to copy l mod 16; the
// copies of a bin are adjacent words, so the lanes spread over banks too)
// and sums them afterwards.  The select stops as soon as the bucket it
// lands in is needed whole.  The selection is then {key above the bucket}
// plus the first (m - #{above}) keys in the bucket in index order; because
// threads own consecutive indices, one block-wide exclusive scan of two
// counts gives every thread its output positions in ascending block order.
// On MI355X this took the kernel from 26.2 to 14.2 us for 512 units of
// 8192 blocks (k = 128), from 15.7 to 10.3 us for 16 units and from 27.1
// to 15.2 us for 192 units of 16384 blocks.
#include "internal.hpp"

namespace {

constexpr int kCopies = 16;  // histogram copies of the first radix pass

__device__ __forceinline__ uint32_t score_key(float f)
{
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7FFFFFFFu) == 0) b = 0;  // -0 == +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

template <int NT, int R>
__global__ __launch_bounds__(NT) void topk_kernel(const float *__restrict__ scores, const int32_t *__restrict__ nblk,
                                                  int Hkv, int nblk_max, int k, int32_t *__restrict__ sel,
                                                  int32_t *__restrict__ mirror)
{
    constexpr int NW = NT / 64;
    constexpr bool kStaged = NT * R <= 16384;  // the row staged through LDS (up to 64 KiB)
    static_assert(R % 4 == 0 && (R & (R - 1)) == 0, "R: a power of two, at least 4");
    __shared__ __align__(16) int stage[kStaged ? NT * R : 4];
    __shared__ __align__(16) int rep[256 * kCopies];  // the first pass's histogram copies, bin-major
    __shared__ int hist[2][256];                       // later passes, alternating
    __shared__ int wave_tot[2][NW];
    __shared__ uint32_t red_min[NW], red_max[NW];
    __shared__ int pick[2][3];

    const int u = blockIdx.x;
    const int b = u / Hkv;
    const float *s = scores + (int64_t)u * nblk_max;
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int base = t * R;

    {
        int4 *z = reinterpret_cast<int4 *>(rep);
        for (int i = t; i < 256 * kCopies / 4; i += NT) z[i] = make_int4(0, 0, 0, 0);
    }

    // the whole row's loads first; the block count masks them afterwards
    uint32_t key[R];
    if constexpr (kStaged) {
        // each wave instruction reads 64 consecutive scores; LDS turns them
        // into each thread's R consecutive ones.  Float e goes to the word
        // R*o + 4*((q + rot) mod G) + i of its owner o = e / R (q = e mod R / 4,
        // i = e mod 4, G = R/4 chunks per thread, rot = o*G/16 mod G), so the
        // owners' 16-byte reads of one instruction fall on distinct banks.
        constexpr int G = R / 4;
#pragma unroll
        for (int j = 0; j < R; ++j) {
            const int e = j * NT + t;
            const uint32_t v = e < nblk_max ? __float_as_uint(s[e]) : 0u;
            const int o = e / R, q = (e % R) >> 2;
            stage[o * R + 4 * ((q + ((o * G) >> 4)) % G) + (e & 3)] = (int)v;
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < G; ++q) {
            const int4 v = *reinterpret_cast<const int4 *>(stage + base + 4 * ((q + ((t * G) >> 4)) % G));
            key[4 * q + 0] = score_key(__int_as_float(v.x));
            key[4 * q + 1] = score_key(__int_as_float(v.y));
            key[4 * q + 2] = score_key(__int_as_float(v.z));
            key[4 * q + 3] = score_key(__int_as_float(v.w));
        }
    } else {
#pragma unroll
        for (int r = 0; r < R; ++r) key[r] = (base + r < nblk_max) ? score_key(s[base + r]) : 0u;
    }

    int n = nblk[b];
    n = n < 0 ? 0 : (n > nblk_max ? nblk_max : n);
    const int m = k < n ? k : n;
    int32_t *out = sel + (int64_t)u * k;
    int32_t *out2 = mirror ? mirror + (int64_t)u * k : nullptr;  // copy in mapped host memory

    for (int i = m + t; i < k; i += NT) {
        out[i] = -1;
        if (out2) out2[i] = -1;
    }
    if (m == 0) return;
    auto valid = [&](int r) { return base + r < n; };
#pragma unroll
    for (int r = 0; r < R; ++r) key[r] = valid(r) ? key[r] : 0u;

    // smallest and largest valid key
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (valid(r)) {
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
    for (int w = 1; w < NW; ++w) {
        kmin = min(kmin, red_min[w]);
        kmax = max(kmax, red_max[w]);
    }

    // Radix select below the shared prefix.  Afterwards the keys with
    // (key & pmask) == prefix form the bucket that holds the m-th largest key,
    // and krem of them are selected.  Pass p counts into hist[p & 1] (the
    // first into the copies, summed into hist[0]); while wave 0 scans it, the
    // other waves clear the other buffer for the next pass, so a pass takes
    // two barriers.
    uint32_t prefix = kmin, pmask = 0xFFFFFFFFu;
    int krem = m;
    if (kmin != kmax) {
        const int top = 31 - __clz(kmin ^ kmax);  // highest differing bit
        pmask = top == 31 ? 0u : ~((2u << top) - 1u);  // bits above it are shared
        prefix = kmax & pmask;
        for (int hi_bit = top, p = 0;; hi_bit -= 8, ++p) {
            const int lo_bit = hi_bit >= 7 ? hi_bit - 7 : 0;
            const int width = hi_bit - lo_bit + 1;
            const uint32_t dmask = (1u << width) - 1u;
            const int cur = p & 1;
            if (p == 0) {
                // every valid key shares the prefix: no test
                const int c = lane & (kCopies - 1);
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (valid(r)) atomicAdd(&rep[((key[r] >> lo_bit) & dmask) * kCopies + c], 1);
                __syncthreads();
                for (int i = t; i < 256; i += NT) {
                    const int4 *row = reinterpret_cast<const int4 *>(rep + i * kCopies);
                    int sum = 0;
#pragma unroll
                    for (int j = 0; j < kCopies / 4; ++j) {
                        const int4 v = row[j];
                        sum += v.x + v.y + v.z + v.w;
                    }
                    hist[0][i] = sum;
                }
            } else {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (valid(r) && (key[r] & pmask) == prefix)
                        atomicAdd(&hist[cur][(key[r] >> lo_bit) & dmask], 1);
            }
            __syncthreads();
            if (wave == 0) {
                // lane l holds digits 255-4l .. 252-4l (descending order)
                int c[4], sum = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    c[i] = hist[cur][255 - 4 * lane - i];
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
                            pick[cur][0] = 255 - 4 * lane - i;
                            pick[cur][1] = krem - acc;
                            pick[cur][2] = c[i];
                        }
                        acc += c[i];
                    }
                }
            } else {
                for (int i = t - 64; i < 256; i += NT - 64) hist[cur ^ 1][i] = 0;
            }
            __syncthreads();
            const uint32_t digit = (uint32_t)pick[cur][0];
            krem = pick[cur][1];
            const int in_bucket = pick[cur][2];
            prefix |= digit << lo_bit;
            pmask |= dmask << lo_bit;
            if (krem == in_bucket || lo_bit == 0) break;  // the whole bucket is selected, or single keys
        }
    }

    // Output positions in block order: with gt_before and eq_before the counts
    // of keys above the bucket and in it over the threads before this one, the
    // bucket's first krem keys are taken in order, so this thread takes
    // min(n_eq, krem - eq_before) of its bucket keys and its first output goes
    // to gt_before + min(krem, eq_before).
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const uint32_t kk = key[r] & pmask;
        n_gt += (valid(r) && kk > prefix) ? 1 : 0;
        n_eq += (valid(r) && kk == prefix) ? 1 : 0;
    }
    int x_gt = n_gt, x_eq = n_eq;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y_gt = __shfl_up(x_gt, o), y_eq = __shfl_up(x_eq, o);
        if (lane >= o) {
            x_gt += y_gt;
            x_eq += y_eq;
        }
    }
    if (lane == 63) {
        wave_tot[0][wave] = x_gt;
        wave_tot[1][wave] = x_eq;
    }
    __syncthreads();
    int gt_before = x_gt - n_gt, eq_before = x_eq - n_eq;
#pragma unroll
    for (int w = 0; w < NW; ++w)
        if (w < wave) {
            gt_before += wave_tot[0][w];
            eq_before += wave_tot[1][w];
        }
    int eq_quota = krem - eq_before;
    eq_quota = eq_quota < 0 ? 0 : (eq_quota > n_eq ? n_eq : eq_quota);
    int pos = gt_before + (eq_before < krem ? eq_before : krem);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const uint32_t kk = key[r] & pmask;
        const bool eq = valid(r) && kk == prefix;
        const bool take = (valid(r) && kk > prefix) || (eq && eq_quota > 0);
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

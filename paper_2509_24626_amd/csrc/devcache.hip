// The HBM block cache's slot table resolved on the GPU: the same LRU as the
// host-side ss_cache (Section 3.1 names LRU; the replacement details are
// the ones stated for ss_cache_resolve), with its state in HBM, so a
// decode step needs no host round trip between selection and gather.
//
// One workgroup per (sequence, KV head) unit:
//   1. the selection is checked (ascending, -1 padding, blocks below the
//      sequence's count, no more than the unit's capacity); a malformed one
//      raises the error flag and leaves the unit untouched;
//   2. hits are looked up in the unit's block table and refresh their last
//      use; the hit slots are marked in an LDS bitmap;
//   3. misses, ranked in ascending block order by a workgroup scan, take the
//      unit's empty slots first (in slot order);
//   4. the remaining r victims are the r smallest keys (last use, slot) among
//      the occupied, unmarked slots.  A binary search over last-use values
//      (slot last uses staged in LDS) finds the threshold T with at least r
//      keys at or below it; the victims are all keys below T and the lowest
//      slots at T; each victim's rank among them orders the assignment;
//   5. miss q takes empty slot q, or the victim of rank q - empties; the
//      evicted blocks leave the block table; the unit's miss rows (b, g,
//      block, slot), in ascending block order, go to the unit's own region
//      of the miss buffer, with their count.
#include <vector>

#include "internal.hpp"

namespace {

constexpr int NT = 256;
constexpr int KMAX = 512;         // selections per unit
constexpr int CMAX = 8192;        // slots per unit
constexpr int ERR_SELECTION = 1;  // error flag bits
constexpr int ERR_CAPACITY = 2;

// exclusive scan of one int per thread over the workgroup; returns the prefix, *total gets the sum
__device__ int block_scan(int v, int *total, int *sm)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) sm[wave] = x;
    __syncthreads();
    int base = 0, sum = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
        const int s = sm[w];
        base += w < wave ? s : 0;
        sum += s;
    }
    __syncthreads();
    *total = sum;
    return base + x - v;
}

__device__ int block_sum(int v, int *sm)
{
    int t;
    (void)block_scan(v, &t, sm);
    return t;
}

__device__ int block_min(int v, int *sm)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
    if (lane == 0) sm[wave] = v;
    __syncthreads();
    int r = sm[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) r = min(r, sm[w]);
    __syncthreads();
    return r;
}

__device__ int block_max(int v, int *sm)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
    if (lane == 0) sm[wave] = v;
    __syncthreads();
    int r = sm[0];
#pragma unroll
    for (int w = 1; w < NT / 64; ++w) r = max(r, sm[w]);
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(NT) void resolve_kernel(const int32_t *__restrict__ sel, int k, int32_t step, int u0,
                                                     int Hkv, const int32_t *__restrict__ nblk,
                                                     const int64_t *__restrict__ slot_base,
                                                     const int64_t *__restrict__ block_base,
                                                     const int32_t *__restrict__ cap,
                                                     const int32_t *__restrict__ table_room, int32_t *used,
                                                     int32_t *slot_block, int32_t *slot_last, int32_t *block_slot,
                                                     int32_t *__restrict__ slots_out, int32_t *__restrict__ miss_out,
                                                     int32_t *__restrict__ counts, int32_t *err,
                                                     unsigned long long *total_misses)
{
    __shared__ int32_t s_sel[KMAX], s_hit[KMAX];
    __shared__ uint32_t s_mark[CMAX / 32];
    __shared__ int32_t s_last[CMAX];
    __shared__ int32_t s_vic[KMAX], s_vsorted[KMAX];
    __shared__ int s_red[NT / 64];

    const int t = threadIdx.x;
    const int u = u0 + blockIdx.x;  // absolute unit
    const int b = u / Hkv, g = u - b * Hkv;
    const int C = cap[u];
    const int n = min(nblk[b], table_room[b]);
    const int used_old = used[u];  // read before any barrier: thread 0 rewrites it at the end
    const int32_t *su = sel + (int64_t)blockIdx.x * k;  // rows of this call's units
    int32_t *out = slots_out + (int64_t)blockIdx.x * k;
    int32_t *rows = miss_out + (int64_t)u * k * 4;
    int32_t *bs = block_slot + block_base[u];
    int32_t *sb = slot_block + slot_base[u];
    int32_t *sl = slot_last + slot_base[u];

    // 1. check the selection
    int bad = 0, valid = 0;
    for (int i = t; i < k; i += NT) {
        const int32_t j = su[i];
        s_sel[i] = j;
        if (j < 0) {
            bad |= j != -1;
        } else {
            const int32_t p = i > 0 ? su[i - 1] : -1;
            bad |= (i > 0 && (p < 0 || p >= j)) || j >= n;
            ++valid;
        }
    }
    for (int i = t; i < CMAX / 32; i += NT) s_mark[i] = 0u;
    bad = block_sum(bad, s_red);
    valid = block_sum(valid, s_red);
    if (bad || valid > C) {
        for (int i = t; i < k; i += NT) out[i] = -1;
        if (t == 0) {
            counts[u] = 0;
            atomicOr(err, bad ? ERR_SELECTION : ERR_CAPACITY);
        }
        return;
    }

    // 2. hits
    for (int i = t; i < k; i += NT) {
        const int32_t j = s_sel[i];
        int32_t s = -1;
        if (j >= 0) {
            s = bs[j];
            if (s >= 0) atomicOr(&s_mark[s >> 5], 1u << (s & 31));
        }
        s_hit[i] = s;
    }
    __syncthreads();

    // 3. miss ranks in selection (ascending block) order: each thread owns a
    //    contiguous run of entries so the scan keeps that order
    constexpr int PER = KMAX / NT;  // 2
    int flags[PER], local = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int i = t * PER + e;
        flags[e] = (i < k && s_sel[i] >= 0 && s_hit[i] < 0) ? 1 : 0;
        local += flags[e];
    }
    int m;
    const int base = block_scan(local, &m, s_red);
    const int empties = min(m, C - used_old);
    const int r = m - empties;  // evictions

    // 4. victims: the r smallest (last use, slot) among occupied, unmarked slots
    if (r > 0) {
        for (int s = t; s < used_old; s += NT) s_last[s] = sl[s];
        __syncthreads();
        auto cand = [&](int s) { return ((s_mark[s >> 5] >> (s & 31)) & 1u) == 0u; };
        int lo = INT32_MAX, hi = -1;  // occupied slots have last uses >= 0
        for (int s = t; s < used_old; s += NT)
            if (cand(s)) {
                lo = min(lo, s_last[s]);
                hi = max(hi, s_last[s]);
            }
        lo = block_min(lo, s_red);
        hi = block_max(hi, s_red);
        // smallest T in [lo, hi] with count(last <= T) >= r
        while (lo < hi) {
            const int mid = lo + (int)(((int64_t)hi - lo) >> 1);
            int c = 0;
            for (int s = t; s < used_old; s += NT) c += (cand(s) && s_last[s] <= mid) ? 1 : 0;
            c = block_sum(c, s_red);
            if (c >= r) hi = mid;
            else lo = mid + 1;
        }
        const int T = lo;
        int below = 0;
        for (int s = t; s < used_old; s += NT) below += (cand(s) && s_last[s] < T) ? 1 : 0;
        below = block_sum(below, s_red);
        const int need_at = r - below;  // lowest slots with last use T
        // victims in slot order: each thread owns a contiguous run of slots
        const int per = (used_old + NT - 1) / NT;
        const int s0 = t * per, s1 = min(used_old, s0 + per);
        int at = 0, vic = 0;
        for (int s = s0; s < s1; ++s)
            if (cand(s) && s_last[s] == T) ++at;
        int at_total;
        int at_rank = block_scan(at, &at_total, s_red);
        for (int s = s0; s < s1; ++s)
            if (cand(s)) {
                if (s_last[s] < T) ++vic;
                else if (s_last[s] == T && at_rank++ < need_at) ++vic;
            }
        int vic_total;
        int vpos = block_scan(vic, &vic_total, s_red);
        at_rank = block_scan(at, &at_total, s_red);  // recount for the second pass
        for (int s = s0; s < s1; ++s)
            if (cand(s)) {
                bool take = false;
                if (s_last[s] < T) take = true;
                else if (s_last[s] == T && at_rank++ < need_at) take = true;
                if (take) s_vic[vpos++] = s;
            }
        __syncthreads();
        // rank of each victim by (last use, slot)
        for (int i = t; i < r; i += NT) {
            const int v = s_vic[i];
            const int lv = s_last[v];
            int rank = 0;
            for (int w = 0; w < r; ++w) {
                const int x = s_vic[w];
                const int lx = s_last[x];
                rank += (lx < lv || (lx == lv && x < v)) ? 1 : 0;
            }
            s_vsorted[rank] = v;
        }
        __syncthreads();
    }

    // 5. assignment and state updates
    int q = base;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int i = t * PER + e;
        if (i >= k) continue;
        const int32_t j = s_sel[i];
        if (j < 0) {
            out[i] = -1;
        } else if (s_hit[i] >= 0) {
            out[i] = s_hit[i];
            sl[s_hit[i]] = step;
        } else {
            int32_t s;
            if (q < empties) {
                s = used_old + q;
            } else {
                s = s_vsorted[q - empties];
                bs[sb[s]] = -1;  // the evicted block leaves the table
            }
            sb[s] = j;
            bs[j] = s;
            sl[s] = step;
            out[i] = s;
            int32_t *row = rows + 4 * q;
            row[0] = b;
            row[1] = g;
            row[2] = j;
            row[3] = s;
            ++q;
        }
    }
    if (t == 0) {
        used[u] = used_old + empties;
        counts[u] = m;
        atomicAdd(total_misses, (unsigned long long)m);
    }
}

}  // namespace

struct ss_dev_cache {
    int B = 0, Hkv = 0, units = 0;
    int64_t total_slots = 0, total_table = 0;
    int64_t last_step = INT64_MIN;
    std::vector<int32_t> cap_host;
    void *mem = nullptr;  // one device allocation holding every array below
    int64_t *slot_base = nullptr, *block_base = nullptr;
    int32_t *cap = nullptr, *room = nullptr, *used = nullptr, *counts = nullptr, *err = nullptr;
    int32_t *slot_block = nullptr, *slot_last = nullptr, *block_slot = nullptr;
    unsigned long long *total = nullptr;  // misses over all resolves
};

namespace ss {
int32_t *dev_cache_counts(ss_dev_cache *c) { return c->counts; }
int dev_cache_batch(const ss_dev_cache *c) { return c->B; }
int dev_cache_kv_heads(const ss_dev_cache *c) { return c->Hkv; }

ss_status dev_cache_launch(ss_dev_cache *c, int64_t step, int b_begin, int b_end, const int32_t *sel, int k,
                           const int32_t *nblk, int32_t *slots, int32_t *miss, hipStream_t s)
{
    const int units = (b_end - b_begin) * c->Hkv;
    if (units == 0) return SS_OK;
    ss::launch(resolve_kernel, dim3(units), dim3(NT), s, sel, k, (int32_t)step, b_begin * c->Hkv, c->Hkv, nblk,
               c->slot_base, c->block_base, c->cap, c->room, c->used, c->slot_block, c->slot_last, c->block_slot,
               slots, miss, c->counts, c->err, c->total);
    return check_launch("ss_dev_cache_resolve");
}

ss_status dev_cache_check_step(ss_dev_cache *c, int64_t step, int k)
{
    SS_CHECK_ARG(k > 0 && k <= KMAX, "ss_dev_cache_resolve: k=%d (1..%d)", k, KMAX);
    SS_CHECK_ARG(step >= 0 && step <= INT32_MAX, "ss_dev_cache_resolve: step %lld outside [0, 2^31)",
                 (long long)step);
    SS_CHECK_ARG(step >= c->last_step, "ss_dev_cache_resolve: step %lld before %lld", (long long)step,
                 (long long)c->last_step);
    c->last_step = step;
    return SS_OK;
}
}  // namespace ss

extern "C" {

ss_status ss_dev_cache_create(int B, int Hkv, const int32_t *table_room, const int32_t *capacity, void *stream,
                              ss_dev_cache **out)
{
    SS_CHECK_ARG(out, "ss_dev_cache_create: null out");
    *out = nullptr;
    SS_CHECK_ARG(B > 0 && Hkv > 0, "ss_dev_cache_create: bad shape B=%d Hkv=%d", B, Hkv);
    SS_CHECK_ARG(table_room && capacity, "ss_dev_cache_create: null pointer");
    const int units = B * Hkv;
    std::vector<int64_t> sbase(units), bbase(units);
    int64_t slots = 0, table = 0;
    for (int u = 0; u < units; ++u) {
        SS_CHECK_ARG(capacity[u] >= 0, "ss_dev_cache_create: capacity[%d] < 0", u);
        SS_CHECK_SUPPORTED(capacity[u] <= CMAX, "ss_dev_cache_create: capacity[%d]=%d > %d", u, capacity[u], CMAX);
        SS_CHECK_ARG(table_room[u / Hkv] >= 0, "ss_dev_cache_create: table_room[%d] < 0", u / Hkv);
        sbase[u] = slots;
        bbase[u] = table;
        slots += capacity[u];
        table += table_room[u / Hkv];
    }
    auto *c = new (std::nothrow) ss_dev_cache;
    if (!c) return ss::fail(SS_ERR_OOM, "ss_dev_cache_create: out of memory");
    c->B = B;
    c->Hkv = Hkv;
    c->units = units;
    c->total_slots = slots;
    c->total_table = table;
    c->cap_host.assign(capacity, capacity + units);
    // layout: 2 int64 arrays [units]; int32 arrays cap, used, counts [units], room [B], err [1];
    // slot_block, slot_last [slots]; block_slot [table]
    const size_t bytes = 8 + 16 * (size_t)units + 4 * (3 * (size_t)units + B + 1) + 8 * (size_t)slots +
                         4 * (size_t)table + 64;
    hipError_t e = hipMalloc(&c->mem, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        delete c;
        return ss::fail(SS_ERR_OOM, "ss_dev_cache_create: hipMalloc(%zu): %s", bytes, hipGetErrorString(e));
    }
    char *p = static_cast<char *>(c->mem);
    c->total = reinterpret_cast<unsigned long long *>(p);
    p += 8;
    c->slot_base = reinterpret_cast<int64_t *>(p);
    c->block_base = c->slot_base + units;
    c->cap = reinterpret_cast<int32_t *>(c->block_base + units);
    c->used = c->cap + units;
    c->counts = c->used + units;
    c->room = c->counts + units;
    c->err = c->room + B;
    c->slot_block = c->err + 1;
    c->slot_last = c->slot_block + slots;
    c->block_slot = c->slot_last + slots;
    const hipStream_t s = ss::as_stream(stream);
    std::vector<int32_t> zeros(units, 0), room(table_room, table_room + B);
    ss_status st = SS_OK;
    e = hipMemcpyAsync(c->slot_base, sbase.data(), 8 * (size_t)units, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(c->block_base, bbase.data(), 8 * (size_t)units, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(c->cap, capacity, 4 * (size_t)units, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(c->used, zeros.data(), 4 * (size_t)units, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(c->counts, zeros.data(), 4 * (size_t)units, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemcpyAsync(c->room, room.data(), 4 * (size_t)B, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipMemsetAsync(c->err, 0, 4, s);
    if (e == hipSuccess) e = hipMemsetAsync(c->total, 0, 8, s);
    if (e == hipSuccess) e = hipMemsetAsync(c->slot_block, 0xFF, 4 * (size_t)slots, s);  // -1: empty
    if (e == hipSuccess) e = hipMemsetAsync(c->slot_last, 0xFF, 4 * (size_t)slots, s);
    if (e == hipSuccess) e = hipMemsetAsync(c->block_slot, 0xFF, 4 * (size_t)table, s);  // -1: not cached
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // the host vectors above go out of scope
    if (e != hipSuccess) {
        (void)hipGetLastError();
        st = ss::fail(SS_ERR_HIP, "ss_dev_cache_create: initialising the state: %s", hipGetErrorString(e));
        (void)hipFree(c->mem);
        delete c;
        return st;
    }
    *out = c;
    return SS_OK;
}

void ss_dev_cache_destroy(ss_dev_cache *c)
{
    if (!c) return;
    if (c->mem) (void)hipFree(c->mem);
    delete c;
}

ss_status ss_dev_cache_resolve(ss_dev_cache *c, int64_t step, int b_begin, int b_end, const int32_t *sel, int k,
                               const int32_t *nblk, int32_t *slots, int32_t *miss, void *stream)
{
    SS_CHECK_ARG(c, "ss_dev_cache_resolve: null cache");
    SS_CHECK_ARG(0 <= b_begin && b_begin <= b_end && b_end <= c->B, "ss_dev_cache_resolve: range [%d, %d) of %d",
                 b_begin, b_end, c->B);
    if (b_begin == b_end) return SS_OK;
    SS_CHECK_ARG(sel && nblk && slots && miss, "ss_dev_cache_resolve: null pointer");
    ss_status st = ss::dev_cache_check_step(c, step, k);
    if (st) return st;
    return ss::dev_cache_launch(c, step, b_begin, b_end, sel, k, nblk, slots, miss, ss::as_stream(stream));
}

ss_status ss_dev_cache_miss_counts(const ss_dev_cache *c, int32_t *counts_host, int32_t *error_flags)
{
    SS_CHECK_ARG(c && counts_host, "ss_dev_cache_miss_counts: null pointer");
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(counts_host, c->counts, 4 * (size_t)c->units, hipMemcpyDeviceToHost);
    if (e == hipSuccess && error_flags) e = hipMemcpy(error_flags, c->err, 4, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "ss_dev_cache_miss_counts: %s", hipGetErrorString(e));
    return SS_OK;
}

ss_status ss_dev_cache_export(const ss_dev_cache *c, int32_t *slot_block, int64_t *slot_last)
{
    SS_CHECK_ARG(c && slot_block && slot_last, "ss_dev_cache_export: null pointer");
    std::vector<int32_t> last(c->total_slots);
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(slot_block, c->slot_block, 4 * (size_t)c->total_slots, hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(last.data(), c->slot_last, 4 * (size_t)c->total_slots, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "ss_dev_cache_export: %s", hipGetErrorString(e));
    for (int64_t i = 0; i < c->total_slots; ++i) slot_last[i] = slot_block[i] >= 0 ? last[i] : 0;
    return SS_OK;
}

int64_t ss_dev_cache_total_slots(const ss_dev_cache *c) { return c ? c->total_slots : 0; }

ss_status ss_dev_cache_total_misses(const ss_dev_cache *c, int64_t *total)
{
    SS_CHECK_ARG(c && total, "ss_dev_cache_total_misses: null pointer");
    unsigned long long v = 0;
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipMemcpy(&v, c->total, 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return ss::fail(SS_ERR_HIP, "ss_dev_cache_total_misses: %s", hipGetErrorString(e));
    *total = (int64_t)v;
    return SS_OK;
}

}  // extern "C"

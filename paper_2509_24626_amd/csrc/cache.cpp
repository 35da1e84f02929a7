// Host side of the KV cache manager's HBM tier (Section 3.1): per
// (sequence, KV head) unit, a region of fixed-size block slots with
// least-recently-used replacement.  The selected blocks of a step are
// resolved to slots here; the misses go to the GPU gather.
//
// Per unit: block -> slot map (O(1) hit test) and one 32-byte record per
// slot (block held, last use, links of an intrusive doubly linked list of the
// cached slots in (last_use, slot) order), so the eviction victim is always
// the list head and a hit touches one cache line of slot state.  A unit's
// state is cold at every step (all units together hold tens of MB), so the
// block lookups of a unit are all issued before any update.  Hits and misses of
// a call are unlinked while they are processed (a block selected in this
// call can never be the victim) and re-appended at the tail in slot order,
// merged with any tail entries already stamped with the same step.  Empty
// slots are only ever the top range [used, capacity): slots never empty
// again, so "lowest empty slot" is a counter.
//
// Units are independent; ss_cache_resolve validates every unit, sizes the
// miss list with a prefix sum, then updates the units in parallel on a
// small persistent thread pool (both passes in one dispatch, with a barrier
// between them).  Output order does not depend on threading.
#include <sched.h>

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstring>
#include <functional>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "internal.hpp"

namespace {

class pool {
  public:
    explicit pool(int n) { resize(n); }
    ~pool() { stop(); }

    void resize(int n)
    {
        stop();
        n = std::max(1, std::min(n, 64));
        quit_.store(false);
        const uint64_t start = gen_.load(std::memory_order_acquire);  // no job is pending now
        for (int i = 1; i < n; ++i) workers_.emplace_back([this, i, start] { loop(i, start); });
        size_ = n;
    }
    int size() const { return size_; }

    // run f(worker_index) on every worker (the caller is worker 0), wait for all
    void run(const std::function<void(int)> &f)
    {
        if (size_ == 1) {
            f(0);
            return;
        }
        {
            std::lock_guard<std::mutex> g(mu_);
            job_ = &f;
            pending_.store(size_ - 1, std::memory_order_relaxed);
            gen_.fetch_add(1, std::memory_order_release);
        }
        cv_.notify_all();
        f(0);
        while (pending_.load(std::memory_order_acquire) != 0) std::this_thread::yield();
        job_ = nullptr;
    }

  private:
    void loop(int idx, uint64_t seen)
    {
        for (;;) {
            // spin briefly (a decode step resolves every layer), then sleep
            uint64_t g = gen_.load(std::memory_order_acquire);
            for (int spin = 0; g == seen && spin < 20000; ++spin) {
                std::this_thread::yield();
                g = gen_.load(std::memory_order_acquire);
            }
            if (g == seen) {
                std::unique_lock<std::mutex> lk(mu_);
                cv_.wait(lk, [&] { return quit_.load() || gen_.load(std::memory_order_acquire) != seen; });
                if (quit_.load()) return;
                g = gen_.load(std::memory_order_acquire);
            }
            if (quit_.load()) return;
            seen = g;
            (*job_)(idx);
            pending_.fetch_sub(1, std::memory_order_acq_rel);
        }
    }
    void stop()
    {
        {
            std::lock_guard<std::mutex> g(mu_);
            quit_.store(true);
        }
        cv_.notify_all();
        for (auto &t : workers_) t.join();
        workers_.clear();
        size_ = 1;
    }

    std::vector<std::thread> workers_;
    std::mutex mu_;
    std::condition_variable cv_;
    std::atomic<uint64_t> gen_{0};
    std::atomic<int> pending_{0};
    const std::function<void(int)> *job_ = nullptr;
    std::atomic<bool> quit_{false};
    int size_ = 1;
};

struct unit_state {
    int32_t cap = 0, nblk = 0, used = 0;
    int32_t head = -1, tail = -1;  // LRU list of cached slots
    int64_t slot_base = 0;         // first slot of this unit in the slot arrays
    int64_t block_base = 0;        // first entry of this unit in block_slot
    int32_t block_cap = 0;         // entries reserved there (>= nblk)
};

// host block-table entries a unit reserves beyond its blocks (sequences grow)
int32_t block_slack(int32_t n) { return std::max<int32_t>(16, n / 8); }

// Half the CPUs this process may run on, at most 8: idle workers spin
// (yielding) between the groups of a step, and a pool as wide as the
// process's CPU share, with the caller also polling, can exhaust a CPU quota
// and get the whole process throttled for a scheduling period.
int default_threads()
{
    int n = 0;
    cpu_set_t set;
    if (sched_getaffinity(0, sizeof(set), &set) == 0) n = CPU_COUNT(&set);
    if (n <= 0) n = (int)std::thread::hardware_concurrency();
    return std::max(1, std::min(8, n / 2));
}

// One pool for the process: resolves on different handles take turns.
std::mutex g_pool_mu;
pool &shared_pool()
{
    static pool p(default_threads());
    return p;
}

}  // namespace

namespace ss {
// Runs f(begin, end) over [0, n) split across the process's resolve
// workers (at most max_threads of them); returns when all parts are done.
void parallel_for(int64_t n, int max_threads, const std::function<void(int64_t, int64_t)> &f)
{
    if (n <= 0) return;
    std::lock_guard<std::mutex> lock(g_pool_mu);
    pool &workers = shared_pool();
    const int T = (int)std::max<int64_t>(1, std::min<int64_t>({(int64_t)workers.size(), (int64_t)max_threads, n}));
    if (T == 1) {
        f(0, n);
        return;
    }
    workers.run([&](int w) {
        if (w < T) f(n * w / T, n * (w + 1) / T);
    });
}
}  // namespace ss

// one slot's state; 32 bytes, so a record never straddles a cache line
struct alignas(32) slot_rec {
    int64_t last = 0;              // step of the last use
    int32_t block = -1;            // block held, -1 empty
    int32_t prev = -1, next = -1;  // LRU list links (slots local to the unit), -1 none
};

struct ss_cache {
    int B = 0, Hkv = 0;
    size_t record_bytes = 0;
    int64_t total_slots = 0;
    int64_t last_step = INT64_MIN;
    std::vector<unit_state> units;
    std::vector<int32_t> block_slot;  // [sum block_cap] slot holding the block, -1
    std::vector<slot_rec> rec;        // [total]
    std::vector<int64_t> miss_count;  // [units] scratch
    int threads = 1;                          // workers used by resolve
    std::vector<std::vector<uint64_t>> mark;  // per worker: slot bitmap for ordering
    std::vector<std::vector<int32_t>> touched;  // per worker
    std::vector<std::vector<int32_t>> found;    // per worker: slot of each selected block, -1
    std::vector<int64_t> part_misses;           // per worker: misses of its units
};

namespace ss {
int cache_batch(const ss_cache *c) { return c->B; }
int cache_kv_heads(const ss_cache *c) { return c->Hkv; }
}  // namespace ss

namespace {

// validates one unit's selection; returns count of valid entries or -1 / -2
int check_unit(const unit_state &st, const int32_t *sel, int k)
{
    int count = 0;
    int32_t prev = -1;
    bool padding = false;
    for (int i = 0; i < k; ++i) {
        const int32_t j = sel[i];
        if (j < 0) {
            if (j != -1) return -1;
            padding = true;
            continue;
        }
        if (padding || j <= prev || j >= st.nblk) return -1;
        prev = j;
        ++count;
    }
    if (count > st.cap) return -2;
    return count;
}

inline void unlink(slot_rec *r, unit_state &st, int32_t s)
{
    const int32_t p = r[s].prev, n = r[s].next;
    if (p >= 0) r[p].next = n; else st.head = n;
    if (n >= 0) r[n].prev = p; else st.tail = p;
    r[s].prev = r[s].next = -1;
}

void resolve_unit(ss_cache *c, int worker, int u, int64_t step, const int32_t *sel, int k, int32_t *slots,
                  int32_t *miss_rows, int b, int g)
{
    unit_state &st = c->units[u];
    int32_t *bs = c->block_slot.data() + st.block_base;
    slot_rec *r = c->rec.data() + st.slot_base;
    std::vector<int32_t> &touched = c->touched[worker];
    int32_t *found = c->found[worker].data();
    touched.clear();

    // 1. hits: every lookup first (independent loads, prefetching the hit
    //    slots' records), then the updates
    for (int i = 0; i < k; ++i) {
        const int32_t j = sel[i];
        const int32_t s = j >= 0 ? bs[j] : -1;
        found[i] = s;
        if (s >= 0) __builtin_prefetch(r + s, 1);
    }
    for (int i = 0; i < k; ++i) {
        const int32_t s = found[i];
        slots[i] = s;
        if (s < 0) continue;
        r[s].last = step;
        unlink(r, st, s);
        touched.push_back(s);
    }
    // 2. misses, ascending block order
    int64_t nm = 0;
    for (int i = 0; i < k; ++i) {
        const int32_t j = sel[i];
        if (j < 0 || found[i] >= 0) continue;
        int32_t s;
        if (st.used < st.cap) {
            s = st.used++;
        } else {
            s = st.head;  // least recently used, lowest slot among equals
            unlink(r, st, s);
            bs[r[s].block] = -1;
        }
        r[s].block = j;
        bs[j] = s;
        r[s].last = step;
        touched.push_back(s);
        slots[i] = s;
        int32_t *row = miss_rows + 4 * nm++;
        row[0] = b;
        row[1] = g;
        row[2] = j;
        row[3] = s;
    }
    if (touched.empty()) return;
    // 3. re-append the touched slots in slot order, merged with the tail run
    //    already stamped with this step
    while (st.tail >= 0 && r[st.tail].last == step) {
        const int32_t s = st.tail;
        unlink(r, st, s);
        touched.push_back(s);
    }
    std::vector<uint64_t> &bits = c->mark[worker];
    const size_t words = ((size_t)st.cap + 63) / 64;
    if (bits.size() < words) bits.resize(words);
    std::fill(bits.begin(), bits.begin() + words, 0ull);
    for (int32_t s : touched) bits[s >> 6] |= 1ull << (s & 63);
    for (size_t w = 0; w < words; ++w) {
        uint64_t x = bits[w];
        while (x) {
            const int32_t s = (int32_t)(w * 64 + __builtin_ctzll(x));
            x &= x - 1;
            r[s].prev = st.tail;
            r[s].next = -1;
            if (st.tail >= 0) r[st.tail].next = s; else st.head = s;
            st.tail = s;
        }
    }
}

}  // namespace

extern "C" {

ss_status ss_cache_create(int B, int Hkv, const int32_t *nblk, const int32_t *capacity, size_t record_bytes,
                          ss_cache **out)
{
    SS_CHECK_ARG(out, "ss_cache_create: null out");
    *out = nullptr;
    SS_CHECK_ARG(B >= 0 && Hkv > 0, "ss_cache_create: bad shape B=%d Hkv=%d", B, Hkv);
    SS_CHECK_ARG(record_bytes > 0, "ss_cache_create: record_bytes=0");
    if (B > 0) SS_CHECK_ARG(nblk && capacity, "ss_cache_create: null pointer");
    ss_cache *c = new (std::nothrow) ss_cache;
    if (!c) return ss::fail(SS_ERR_OOM, "ss_cache_create: out of memory");
    try {
        c->B = B;
        c->Hkv = Hkv;
        c->record_bytes = record_bytes;
        const int units = B * Hkv;
        c->units.resize(units);
        int64_t slots = 0, blocks = 0;
        for (int u = 0; u < units; ++u) {
            const int32_t n = nblk[u / Hkv], cap = capacity[u];
            if (n < 0 || cap < 0) {
                delete c;
                return ss::fail(SS_ERR_INVALID_ARG, "ss_cache_create: negative nblk or capacity at unit %d", u);
            }
            unit_state &st = c->units[u];
            st.cap = cap;
            st.nblk = n;
            st.block_cap = n + block_slack(n);  // room to grow without laying the table out again
            st.slot_base = slots;
            st.block_base = blocks;
            slots += cap;
            blocks += st.block_cap;
        }
        c->total_slots = slots;
        c->block_slot.assign(blocks, -1);
        c->rec.assign(slots, slot_rec{});
        c->miss_count.assign(units, 0);
        c->threads = default_threads();
        c->mark.resize(64);
        c->touched.resize(64);
        c->found.resize(64);
        c->part_misses.assign(64, 0);
    } catch (const std::bad_alloc &) {
        delete c;
        return ss::fail(SS_ERR_OOM, "ss_cache_create: out of memory");
    }
    *out = c;
    return SS_OK;
}

void ss_cache_destroy(ss_cache *c) { delete c; }

int64_t ss_cache_total_slots(const ss_cache *c) { return c ? c->total_slots : 0; }

ss_status ss_cache_region_offsets(const ss_cache *c, int64_t *off)
{
    SS_CHECK_ARG(c && off, "ss_cache_region_offsets: null pointer");
    for (size_t u = 0; u < c->units.size(); ++u) off[u] = c->units[u].slot_base * (int64_t)c->record_bytes;
    return SS_OK;
}

ss_status ss_cache_set_blocks(ss_cache *c, const int32_t *nblk)
{
    SS_CHECK_ARG(c && (c->B == 0 || nblk), "ss_cache_set_blocks: null pointer");
    bool grow = false;
    for (int b = 0; b < c->B; ++b) {
        const unit_state &st = c->units[(size_t)b * c->Hkv];
        SS_CHECK_ARG(nblk[b] >= st.nblk, "ss_cache_set_blocks: sequence %d shrinks from %d to %d blocks", b, st.nblk,
                     nblk[b]);
        grow |= nblk[b] > st.block_cap;
    }
    if (grow) {
        // lay the block table out again with room to grow (amortised)
        try {
            std::vector<int32_t> bs;
            std::vector<int64_t> base(c->units.size());
            std::vector<int32_t> cap(c->units.size());
            int64_t total = 0;
            for (size_t u = 0; u < c->units.size(); ++u) {
                const int32_t n = nblk[u / c->Hkv];
                const unit_state &st = c->units[u];
                cap[u] = n > st.block_cap ? n + block_slack(n) : st.block_cap;
                base[u] = total;
                total += cap[u];
            }
            bs.assign(total, -1);
            for (size_t u = 0; u < c->units.size(); ++u) {
                const unit_state &st = c->units[u];
                std::copy(c->block_slot.begin() + st.block_base, c->block_slot.begin() + st.block_base + st.nblk,
                          bs.begin() + base[u]);
            }
            c->block_slot.swap(bs);
            for (size_t u = 0; u < c->units.size(); ++u) {
                c->units[u].block_base = base[u];
                c->units[u].block_cap = cap[u];
            }
        } catch (const std::bad_alloc &) {
            return ss::fail(SS_ERR_OOM, "ss_cache_set_blocks: out of memory");
        }
    }
    for (size_t u = 0; u < c->units.size(); ++u) c->units[u].nblk = nblk[u / c->Hkv];
    return SS_OK;
}

ss_status ss_cache_set_threads(ss_cache *c, int n)
{
    SS_CHECK_ARG(c && n > 0, "ss_cache_set_threads: bad argument");
    c->threads = std::min(n, 64);
    return SS_OK;
}

ss_status ss_cache_resolve(ss_cache *c, int64_t step, const int32_t *sel, int k, int32_t *slots, int32_t *miss,
                           int64_t miss_cap, int64_t *n_miss)
{
    SS_CHECK_ARG(c, "ss_cache_resolve: null cache");
    return ss_cache_resolve_range(c, step, 0, c->B, sel, k, slots, miss, miss_cap, n_miss);
}

ss_status ss_cache_resolve_range(ss_cache *c, int64_t step, int b_begin, int b_end, const int32_t *sel, int k,
                                 int32_t *slots, int32_t *miss, int64_t miss_cap, int64_t *n_miss)
{
    SS_CHECK_ARG(c && n_miss && k > 0 && miss_cap >= 0, "ss_cache_resolve: bad argument");
    SS_CHECK_ARG(0 <= b_begin && b_begin <= b_end && b_end <= c->B, "ss_cache_resolve: sequence range [%d, %d) "
                 "outside [0, %d)", b_begin, b_end, c->B);
    *n_miss = 0;
    const int u0 = b_begin * c->Hkv;
    const int units = (b_end - b_begin) * c->Hkv;
    if (units == 0) return SS_OK;
    SS_CHECK_ARG(sel && slots && (miss || miss_cap == 0), "ss_cache_resolve: null pointer");
    SS_CHECK_ARG(step >= c->last_step, "ss_cache_resolve: step %lld precedes the previous step %lld",
                 (long long)step, (long long)c->last_step);

    std::lock_guard<std::mutex> pool_lock(g_pool_mu);
    pool &workers = shared_pool();
    if (workers.size() < c->threads) {
        try {
            workers.resize(c->threads);
        } catch (const std::exception &) {
            return ss::fail(SS_ERR_OOM, "ss_cache_resolve: could not start %d threads", c->threads);
        }
    }
    const int nt = std::min(c->threads, workers.size());
    // the workers' scratch (touched slots, slot bitmap) at full size up front:
    // nothing may allocate, and so throw, inside a worker thread
    try {
        int32_t cap_max = 0;
        for (int u = u0; u < u0 + units; ++u) cap_max = std::max(cap_max, c->units[u].cap);
        const size_t words = ((size_t)cap_max + 63) / 64;
        for (int w = 0; w < nt; ++w) {
            c->touched[w].reserve((size_t)k + (size_t)cap_max);
            if (c->mark[w].size() < words) c->mark[w].resize(words);
            if (c->found[w].size() < (size_t)k) c->found[w].resize(k);
        }
    } catch (const std::bad_alloc &) {
        return ss::fail(SS_ERR_OOM, "ss_cache_resolve: out of memory");
    }
    // one dispatch: pass 1 (read-only) validates the units and counts their
    // misses; after a barrier every worker sees all counts and either stops
    // (an invalid unit, too many misses: no state changed) or, in pass 2,
    // updates its units, writing their miss rows at their prefix offsets
    std::atomic<int> bad_unit{-1}, bad_kind{0}, arrived{0};
    int64_t *part = c->part_misses.data();
    workers.run([&](int w) {
        if (w >= nt) return;
        const int lo = (int)((int64_t)units * w / nt), hi = (int)((int64_t)units * (w + 1) / nt);
        int64_t mine = 0;
        for (int i = lo; i < hi; ++i) {
            const int u = u0 + i;
            const unit_state &st = c->units[u];
            const int32_t *su = sel + (int64_t)i * k;
            const int cnt = check_unit(st, su, k);
            if (cnt < 0) {
                int expect = -1;
                if (bad_unit.compare_exchange_strong(expect, u)) bad_kind.store(cnt);
                c->miss_count[u] = 0;
                continue;
            }
            const int32_t *bs = c->block_slot.data() + st.block_base;
            int64_t m = 0;
            for (int e = 0; e < k; ++e)
                if (su[e] >= 0 && bs[su[e]] < 0) ++m;
            c->miss_count[u] = m;
            mine += m;
        }
        part[w] = mine;
        arrived.fetch_add(1, std::memory_order_acq_rel);
        while (arrived.load(std::memory_order_acquire) < nt) std::this_thread::yield();
        if (bad_unit.load() >= 0) return;
        int64_t before = 0, all = 0;
        for (int v = 0; v < nt; ++v) {
            if (v < w) before += part[v];
            all += part[v];
        }
        if (all > miss_cap) return;
        for (int i = lo; i < hi; ++i) {
            const int u = u0 + i;
            int32_t *rows = miss + 4 * before;
            before += c->miss_count[u];
            resolve_unit(c, w, u, step, sel + (int64_t)i * k, k, slots + (int64_t)i * k, rows, u / c->Hkv,
                         u % c->Hkv);
        }
    });
    if (bad_unit.load() >= 0) {
        const int u = bad_unit.load();
        if (bad_kind.load() == -2)
            return ss::fail(SS_ERR_CAPACITY, "ss_cache_resolve: unit %d selects more blocks than its %d slots", u,
                            c->units[u].cap);
        return ss::fail(SS_ERR_INVALID_ARG,
                        "ss_cache_resolve: unit %d selection is not strictly ascending in [0, nblk) then -1", u);
    }
    int64_t total = 0;
    for (int w = 0; w < nt; ++w) total += part[w];
    if (total > miss_cap)
        return ss::fail(SS_ERR_OOM, "ss_cache_resolve: %lld misses > miss_cap %lld", (long long)total,
                        (long long)miss_cap);
    c->last_step = step;
    *n_miss = total;
    return SS_OK;
}

ss_status ss_cache_export(const ss_cache *c, int32_t *slot_block, int64_t *slot_last)
{
    SS_CHECK_ARG(c && slot_block && slot_last, "ss_cache_export: null pointer");
    for (int64_t s = 0; s < c->total_slots; ++s) {
        slot_block[s] = c->rec[s].block;
        slot_last[s] = c->rec[s].last;
    }
    return SS_OK;
}

}  // extern "C"

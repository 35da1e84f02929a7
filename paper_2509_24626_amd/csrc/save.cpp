// FlashD2H, CPU-assisted saving of new KV to the DRAM pool (Section 3.2.2).
//
// The new tokens of a layer form one contiguous tensor on the GPU.  Saving
// them is split in two, as the paper does: device-to-host copies of the
// contiguous tensor into a pinned staging buffer on the caller's (save)
// stream, then host threads place every token into its block record in the
// pool.  The GPU spends no compute on it: the copies run on a copy engine,
// and the scatter on this library's own threads, so it overlaps the next
// layers' work.  A large save is copied in chunks of consecutive token rows
// (at least 1 MiB, about four per thread), each with its own event, so the
// scatter of one chunk overlaps the copy of the next.  Staging buffers form
// a ring; a save whose buffer is still being scattered waits for it.
//
// Record layout: K tile [blk][d] row-major, then V tile channel-major
// [d][blk] (bf16), so a token is one 256-byte K row and d strided V values.
#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <memory>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "internal.hpp"

namespace {

constexpr int kMaxChunks = 64;            // copies (and events) per save
constexpr size_t kMinChunkBytes = 1 << 20;

// where a save's tokens go: per unit the byte offset of its block array in
// the pool, per sequence the blocks that array holds
struct target {
    std::vector<int64_t> pool_off;
    std::vector<int32_t> pool_blocks;
};

struct job {
    int slot;
    int n_new;
    std::vector<int32_t> len;
    std::shared_ptr<const target> to;  // fixed when the save is issued
    std::atomic<int> chunks_left{0};
};

struct chunk {
    job *jb;
    int ev;          // event index within the slot
    int64_t r0, r1;  // token rows [r0, r1) of the [B][n_new] order
};

}  // namespace

struct ss_kv_saver {
    int B = 0, Hkv = 0, blk = 0, d = 0, max_new = 0;
    size_t record_bytes = 0, row_bytes = 0, slot_bytes = 0;
    uint8_t *pool = nullptr;
    std::shared_ptr<const target> to;
    std::vector<void *> staging;
    std::vector<std::vector<hipEvent_t>> copied;  // [slot][chunk]
    std::vector<bool> busy;
    int next = 0;
    int threads = 1;

    std::mutex mu;
    std::condition_variable cv_work, cv_done;
    std::deque<chunk> queue;
    int in_flight = 0;  // saves queued or running
    bool quit = false;
    ss_status error = SS_OK;
    std::string error_msg;
    std::vector<std::thread> workers;

    ~ss_kv_saver()
    {
        {
            std::lock_guard<std::mutex> g(mu);
            quit = true;
        }
        cv_work.notify_all();
        for (auto &t : workers) t.join();
        for (auto &evs : copied)
            for (hipEvent_t e : evs)
                if (e) (void)hipEventDestroy(e);
        for (void *p : staging)
            if (p) (void)hipHostFree(p);
    }

    // every (sequence, head) of the token rows [r0, r1)
    void scatter(const job &jb, int64_t r0, int64_t r1)
    {
        const uint16_t *src = static_cast<const uint16_t *>(staging[jb.slot]);
        for (int64_t r = r0; r < r1; ++r) {
            const int b = (int)(r / jb.n_new), i = (int)(r - (int64_t)b * jb.n_new);
            const int T = jb.len[b] + i;
            const int j = T / blk, p = T - j * blk;
            for (int g = 0; g < Hkv; ++g) {
                const uint16_t *kv = src + (r * Hkv + g) * 2 * d;
                uint8_t *rec = pool + jb.to->pool_off[(size_t)b * Hkv + g] + (int64_t)j * (int64_t)record_bytes;
                std::memcpy(rec + (size_t)p * d * 2, kv, (size_t)d * 2);
                uint16_t *vt = reinterpret_cast<uint16_t *>(rec + (size_t)blk * d * 2);
                for (int c = 0; c < d; ++c) vt[c * blk + p] = kv[d + c];
            }
        }
    }

    void worker()
    {
        for (;;) {
            chunk w;
            {
                std::unique_lock<std::mutex> lk(mu);
                cv_work.wait(lk, [&] { return quit || !queue.empty(); });
                if (queue.empty()) return;  // quit with nothing left
                w = queue.front();
                queue.pop_front();
            }
            job *jb = w.jb;
            hipError_t e = hipEventSynchronize(copied[jb->slot][w.ev]);
            if (e == hipSuccess) scatter(*jb, w.r0, w.r1);
            const bool last = jb->chunks_left.fetch_sub(1) == 1;
            if (last || e != hipSuccess) {
                std::lock_guard<std::mutex> g(mu);
                if (e != hipSuccess && error == SS_OK) {
                    error = SS_ERR_HIP;
                    error_msg = std::string("ss_kv_save: wait for the copy: ") + hipGetErrorString(e);
                }
                if (last) {
                    busy[jb->slot] = false;
                    --in_flight;
                    delete jb;
                    cv_done.notify_all();
                }
            }
        }
    }

    // with mu held: wait until `slot` is free (or everything, slot < 0)
    void wait_locked(std::unique_lock<std::mutex> &lk, int slot)
    {
        cv_done.wait(lk, [&] { return slot < 0 ? in_flight == 0 : !busy[slot]; });
    }
};

extern "C" {

ss_status ss_kv_saver_create(int B, int Hkv, int blk, int d, void *pool_host, const int64_t *pool_off,
                             const int32_t *pool_blocks, int max_new_tokens, int staging_slots, int threads,
                             ss_kv_saver **out)
{
    SS_CHECK_ARG(out, "ss_kv_saver_create: null output");
    *out = nullptr;
    SS_CHECK_ARG(B > 0 && Hkv > 0 && max_new_tokens > 0, "ss_kv_saver_create: bad shape B=%d Hkv=%d max_new=%d", B,
                 Hkv, max_new_tokens);
    SS_CHECK_SUPPORTED(d == ss::kHeadDim, "ss_kv_saver_create: d=%d (only 128)", d);
    SS_CHECK_SUPPORTED(ss::supported_blk(blk), "ss_kv_saver_create: blk=%d (8, 16 or 32)", blk);
    SS_CHECK_ARG(pool_host && pool_off && pool_blocks, "ss_kv_saver_create: null pointer");
    SS_CHECK_ARG(staging_slots >= 1 && staging_slots <= 64, "ss_kv_saver_create: staging_slots=%d (1..64)",
                 staging_slots);
    SS_CHECK_ARG(threads >= 1 && threads <= 64, "ss_kv_saver_create: threads=%d (1..64)", threads);
    for (int b = 0; b < B; ++b) SS_CHECK_ARG(pool_blocks[b] >= 0, "ss_kv_saver_create: pool_blocks[%d] < 0", b);
    auto *sv = new (std::nothrow) ss_kv_saver;
    if (!sv) return ss::fail(SS_ERR_OOM, "ss_kv_saver_create: out of memory");
    try {
    sv->B = B;
    sv->Hkv = Hkv;
    sv->blk = blk;
    sv->d = d;
    sv->max_new = max_new_tokens;
    sv->record_bytes = (size_t)2 * blk * d * 2;
    sv->slot_bytes = (size_t)B * max_new_tokens * Hkv * 2 * d * 2;
    sv->pool = static_cast<uint8_t *>(pool_host);
    {
        auto t = std::make_shared<target>();
        t->pool_off.assign(pool_off, pool_off + (size_t)B * Hkv);
        t->pool_blocks.assign(pool_blocks, pool_blocks + B);
        sv->to = std::move(t);
    }
    sv->threads = threads;
    sv->row_bytes = (size_t)Hkv * 2 * d * 2;
    sv->staging.assign(staging_slots, nullptr);
    sv->copied.assign(staging_slots, std::vector<hipEvent_t>(kMaxChunks, nullptr));
    sv->busy.assign(staging_slots, false);
    } catch (const std::bad_alloc &) {
        delete sv;
        return ss::fail(SS_ERR_OOM, "ss_kv_saver_create: out of memory");
    }
    for (int i = 0; i < staging_slots; ++i) {
        hipError_t e = hipHostMalloc(&sv->staging[i], sv->slot_bytes, hipHostMallocDefault);
        for (int c = 0; c < kMaxChunks && e == hipSuccess; ++c)
            e = hipEventCreateWithFlags(&sv->copied[i][c], hipEventDisableTiming | hipEventBlockingSync);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            delete sv;
            return ss::fail(SS_ERR_OOM, "ss_kv_saver_create: staging buffer or event: %s", hipGetErrorString(e));
        }
    }
    try {
        for (int i = 0; i < threads; ++i) sv->workers.emplace_back([sv] { sv->worker(); });
    } catch (const std::exception &) {
        delete sv;  // joins the workers already started
        return ss::fail(SS_ERR_OOM, "ss_kv_saver_create: could not start %d threads", threads);
    }
    *out = sv;
    ss::clear_error();
    return SS_OK;
}

void ss_kv_saver_destroy(ss_kv_saver *sv)
{
    if (!sv) return;
    {
        std::unique_lock<std::mutex> lk(sv->mu);
        sv->wait_locked(lk, -1);
    }
    delete sv;
}

ss_status ss_kv_save(ss_kv_saver *sv, const void *new_kv, int n_new, const int32_t *len, void *stream)
{
    SS_CHECK_ARG(sv && len, "ss_kv_save: null argument");
    SS_CHECK_ARG(n_new >= 0 && n_new <= sv->max_new, "ss_kv_save: n_new=%d (0..%d)", n_new, sv->max_new);
    if (n_new == 0) return SS_OK;
    SS_CHECK_ARG(new_kv, "ss_kv_save: null new_kv");
    const hipStream_t s = ss::as_stream(stream);
    std::unique_lock<std::mutex> lk(sv->mu);
    const std::shared_ptr<const target> to = sv->to;  // ss_kv_saver_retarget swaps it under the lock
    for (int b = 0; b < sv->B; ++b) {
        SS_CHECK_ARG(len[b] >= 0, "ss_kv_save: len[%d] < 0", b);
        SS_CHECK_ARG((int64_t)(len[b] + n_new - 1) / sv->blk < to->pool_blocks[b],
                     "ss_kv_save: sequence %d: token %d lies past its %d pool blocks", b, len[b] + n_new - 1,
                     to->pool_blocks[b]);
    }
    if (sv->error != SS_OK) return ss::fail(sv->error, "%s", sv->error_msg.c_str());
    const int slot = sv->next;
    sv->wait_locked(lk, slot);  // its previous scatter must be finished
    // chunks of whole token rows, copied one after another on `stream`; each
    // is scattered as soon as its own copy has landed, so scattering overlaps
    // the copies still running
    const int64_t rows = (int64_t)sv->B * n_new;
    const size_t total = (size_t)rows * sv->row_bytes;
    size_t target = std::max(kMinChunkBytes, total / (size_t)(4 * sv->threads));
    int64_t per = std::max<int64_t>(1, (int64_t)((target + sv->row_bytes - 1) / sv->row_bytes));
    if ((rows + per - 1) / per > kMaxChunks) per = (rows + kMaxChunks - 1) / kMaxChunks;
    const int n_chunks = (int)((rows + per - 1) / per);
    const uint8_t *src = static_cast<const uint8_t *>(new_kv);
    uint8_t *dst = static_cast<uint8_t *>(sv->staging[slot]);
    for (int c = 0; c < n_chunks; ++c) {
        const int64_t r0 = c * per, r1 = std::min(rows, r0 + per);
        hipError_t e = hipMemcpyAsync(dst + r0 * sv->row_bytes, src + r0 * sv->row_bytes,
                                      (size_t)(r1 - r0) * sv->row_bytes, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipEventRecord(sv->copied[slot][c], s);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            // copies enqueued so far are harmless: the slot is not marked busy
            return ss::fail(SS_ERR_HIP, "ss_kv_save: copy to staging: %s", hipGetErrorString(e));
        }
    }
    job *jb = new (std::nothrow) job;
    if (!jb) return ss::fail(SS_ERR_OOM, "ss_kv_save: out of memory");
    try {
        jb->len.assign(len, len + sv->B);
    } catch (const std::bad_alloc &) {
        delete jb;
        return ss::fail(SS_ERR_OOM, "ss_kv_save: out of memory");
    }
    jb->slot = slot;
    jb->n_new = n_new;
    jb->to = to;
    jb->chunks_left.store(n_chunks);
    sv->busy[slot] = true;
    ++sv->in_flight;
    for (int c = 0; c < n_chunks; ++c) {
        const int64_t r0 = c * per, r1 = std::min(rows, r0 + per);
        sv->queue.push_back(chunk{jb, c, r0, r1});
    }
    sv->next = (slot + 1) % (int)sv->staging.size();
    lk.unlock();
    sv->cv_work.notify_all();
    return SS_OK;
}

ss_status ss_kv_saver_retarget(ss_kv_saver *sv, const int64_t *pool_off, const int32_t *pool_blocks)
{
    SS_CHECK_ARG(sv && pool_off && pool_blocks, "ss_kv_saver_retarget: null pointer");
    for (int b = 0; b < sv->B; ++b) SS_CHECK_ARG(pool_blocks[b] >= 0, "ss_kv_saver_retarget: pool_blocks[%d] < 0", b);
    try {
        auto t = std::make_shared<target>();
        t->pool_off.assign(pool_off, pool_off + (size_t)sv->B * sv->Hkv);
        t->pool_blocks.assign(pool_blocks, pool_blocks + sv->B);
        std::lock_guard<std::mutex> g(sv->mu);
        sv->to = std::move(t);  // saves in flight keep the targets they were issued with
    } catch (const std::bad_alloc &) {
        return ss::fail(SS_ERR_OOM, "ss_kv_saver_retarget: out of memory");
    }
    return SS_OK;
}

ss_status ss_kv_save_wait(ss_kv_saver *sv)
{
    SS_CHECK_ARG(sv, "ss_kv_save_wait: null saver");
    std::unique_lock<std::mutex> lk(sv->mu);
    sv->wait_locked(lk, -1);
    if (sv->error != SS_OK) return ss::fail(sv->error, "%s", sv->error_msg.c_str());
    return SS_OK;
}

}  // extern "C"

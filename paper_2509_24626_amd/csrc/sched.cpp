// Working-set-aware batch size control (Section 3.3).
//
// Decoding working set: per (request, layer, KV head), the union of the
// blocks selected over the last w decoding steps.  The tracker keeps, per
// such unit, a ring of the last w selections and a per-block count of how
// often the block occurs in the ring, so the union's size moves with each
// observation: entries leaving the window decrement (a count reaching 0
// leaves the union), entries joining increment (a count leaving 0 joins).
// An observation of one layer for a batch costs O(B * Hkv * k), spread over
// the library's host threads; the estimate of a request is a sum over its
// units.
//
// Prefill working sets are exact (closed forms), and the batch control of
// Algorithm 1 walks the initial batch in order, admitting a request while
// the admitted working sets fit the available HBM.  The plan of a
// layer-segmented prefill (Section 3.4) assigns a prompt's layers, or
// chunks of them, to batches under the maxInjectToken bound.
#include <algorithm>
#include <unordered_map>
#include <vector>

#include "internal.hpp"

namespace {

constexpr int32_t kMaxBlockIndex = 1 << 24;

struct unit_ws {
    std::vector<int32_t> ring;   // [w][k] the last w selections
    std::vector<uint8_t> count;  // per block: occurrences in the ring (<= w <= 255)
    int32_t size = 0;            // blocks with count > 0
    int32_t head = 0, held = 0;  // next ring row; rows holding an observation
};

struct request_ws {
    std::vector<unit_ws> units;     // [layers][Hkv]
    std::vector<int64_t> last_step; // [layers]
};

}  // namespace

struct ss_ws {
    int layers = 0, Hkv = 0, w = 0, k = 0;
    size_t record_bytes = 0;
    std::unordered_map<int64_t, request_ws> reqs;
};

extern "C" {

ss_status ss_ws_create(int layers, int Hkv, int window, size_t record_bytes, ss_ws **out)
{
    SS_CHECK_ARG(out, "ss_ws_create: null output");
    *out = nullptr;
    SS_CHECK_ARG(layers > 0 && Hkv > 0, "ss_ws_create: layers=%d Hkv=%d", layers, Hkv);
    SS_CHECK_ARG(window >= 1 && window <= 255, "ss_ws_create: window=%d (1..255)", window);
    SS_CHECK_ARG(record_bytes > 0, "ss_ws_create: record_bytes=0");
    auto *t = new (std::nothrow) ss_ws;
    if (!t) return ss::fail(SS_ERR_OOM, "ss_ws_create: out of memory");
    t->layers = layers;
    t->Hkv = Hkv;
    t->w = window;
    t->record_bytes = record_bytes;
    *out = t;
    return SS_OK;
}

void ss_ws_destroy(ss_ws *t) { delete t; }

ss_status ss_ws_observe(ss_ws *t, int layer, int64_t step, const int64_t *req_ids, int B, const int32_t *sel, int k)
{
    SS_CHECK_ARG(t, "ss_ws_observe: null tracker");
    SS_CHECK_ARG(layer >= 0 && layer < t->layers, "ss_ws_observe: layer %d of %d", layer, t->layers);
    SS_CHECK_ARG(B >= 0 && k > 0, "ss_ws_observe: B=%d k=%d", B, k);
    if (B == 0) return SS_OK;
    SS_CHECK_ARG(req_ids && sel, "ss_ws_observe: null pointer");
    SS_CHECK_ARG(t->k == 0 || t->k == k, "ss_ws_observe: k=%d differs from the tracker's %d", k, t->k);
    const int64_t n_sel = (int64_t)B * t->Hkv * k;
    for (int64_t i = 0; i < n_sel; ++i)
        SS_CHECK_ARG(sel[i] < kMaxBlockIndex, "ss_ws_observe: block index %d out of range", sel[i]);
    std::vector<request_ws *> rq(B);
    for (int b = 0; b < B; ++b) {
        auto it = t->reqs.find(req_ids[b]);
        if (it != t->reqs.end()) {
            SS_CHECK_ARG(step > it->second.last_step[layer], "ss_ws_observe: request %lld, layer %d: step %lld "
                         "after %lld", (long long)req_ids[b], layer, (long long)step,
                         (long long)it->second.last_step[layer]);
        }
        for (int c = 0; c < b; ++c)
            SS_CHECK_ARG(req_ids[c] != req_ids[b], "ss_ws_observe: request %lld twice", (long long)req_ids[b]);
    }
    try {
        for (int b = 0; b < B; ++b) {
            request_ws &r = t->reqs[req_ids[b]];
            if (r.units.empty()) {
                r.units.resize((size_t)t->layers * t->Hkv);
                r.last_step.assign(t->layers, INT64_MIN);
            }
            r.last_step[layer] = step;
            rq[b] = &r;
        }
        t->k = k;
        const int w = t->w, Hkv = t->Hkv;
        // every allocation on this thread (a worker thread must not throw):
        // the workers find each unit's largest block index, then the rings and
        // counts that need room get it here
        std::vector<int32_t> hi((size_t)B * Hkv);
        ss::parallel_for((int64_t)B * Hkv, 16, [&](int64_t u0, int64_t u1) {
            for (int64_t u = u0; u < u1; ++u) {
                int32_t m = -1;
                for (int i = 0; i < k; ++i) m = std::max(m, sel[u * k + i]);
                hi[u] = m;
            }
        });
        for (int64_t u = 0; u < (int64_t)B * Hkv; ++u) {
            const int b = (int)(u / Hkv), g = (int)(u - (int64_t)b * Hkv);
            unit_ws &st = rq[b]->units[(size_t)layer * Hkv + g];
            if (st.ring.empty()) st.ring.assign((size_t)w * k, -1);
            if (hi[u] >= 0 && (size_t)hi[u] >= st.count.size())
                st.count.resize(std::max<size_t>((size_t)hi[u] + 1, st.count.size() * 2), 0);
        }
        ss::parallel_for((int64_t)B * Hkv, 16, [&](int64_t u0, int64_t u1) {
            for (int64_t u = u0; u < u1; ++u) {
                const int b = (int)(u / Hkv), g = (int)(u - (int64_t)b * Hkv);
                unit_ws &st = rq[b]->units[(size_t)layer * Hkv + g];
                int32_t *row = st.ring.data() + (size_t)st.head * k;
                if (st.held == w)  // the oldest observation leaves the window
                    for (int i = 0; i < k; ++i)
                        if (row[i] >= 0 && --st.count[row[i]] == 0) --st.size;
                const int32_t *s = sel + u * k;
                for (int i = 0; i < k; ++i) {
                    const int32_t j = s[i];
                    row[i] = j;
                    if (j < 0) continue;
                    if (st.count[j]++ == 0) ++st.size;
                }
                st.head = (st.head + 1) % w;
                st.held = std::min(st.held + 1, w);
            }
        });
    } catch (const std::bad_alloc &) {
        return ss::fail(SS_ERR_OOM, "ss_ws_observe: out of memory");
    }
    return SS_OK;
}

ss_status ss_ws_decode_bytes(const ss_ws *t, const int64_t *req_ids, int n, const int32_t *fallback_blocks,
                             int64_t *bytes)
{
    SS_CHECK_ARG(t && (n == 0 || (req_ids && bytes)), "ss_ws_decode_bytes: null pointer");
    SS_CHECK_ARG(n >= 0, "ss_ws_decode_bytes: n=%d", n);
    for (int i = 0; i < n; ++i) {
        const int64_t fb = fallback_blocks ? fallback_blocks[i] : 0;
        SS_CHECK_ARG(fb >= 0, "ss_ws_decode_bytes: fallback_blocks[%d] < 0", i);
        auto it = t->reqs.find(req_ids[i]);
        int64_t blocks = 0;
        if (it == t->reqs.end()) {
            blocks = fb * t->layers * t->Hkv;
        } else {
            for (const unit_ws &st : it->second.units) blocks += st.held ? st.size : fb;
        }
        bytes[i] = blocks * (int64_t)t->record_bytes;
    }
    return SS_OK;
}

ss_status ss_ws_forget(ss_ws *t, int64_t req_id)
{
    SS_CHECK_ARG(t, "ss_ws_forget: null tracker");
    t->reqs.erase(req_id);
    return SS_OK;
}

int64_t ss_ws_prefill_bytes(int64_t prompt_tokens, int64_t done_tokens, int64_t chunk_tokens, int layers, int Hkv,
                            int blk, size_t record_bytes, int layer_segmented)
{
    if (prompt_tokens < 0 || done_tokens < 0 || chunk_tokens < 0 || layers <= 0 || Hkv <= 0 || blk <= 0) return -1;
    const int64_t tokens = layer_segmented ? prompt_tokens : std::min(prompt_tokens, done_tokens + chunk_tokens);
    const int64_t blocks = (tokens + blk - 1) / blk;
    return blocks * Hkv * (layer_segmented ? 1 : layers) * (int64_t)record_bytes;
}

ss_status ss_schedule_batch(const int64_t *ws_bytes, int n, int64_t m_avl, int32_t *admit, int64_t *m_used)
{
    SS_CHECK_ARG(n >= 0 && m_used && (n == 0 || (ws_bytes && admit)), "ss_schedule_batch: bad argument");
    for (int i = 0; i < n; ++i) SS_CHECK_ARG(ws_bytes[i] >= 0, "ss_schedule_batch: ws_bytes[%d] < 0", i);
    int64_t used = 0;
    for (int i = 0; i < n; ++i) {
        const bool fits = ws_bytes[i] <= m_avl - used;
        admit[i] = fits ? 1 : 0;
        if (fits) used += ws_bytes[i];
    }
    *m_used = used;
    return SS_OK;
}

ss_status ss_prefill_plan(int64_t T, int layers, int64_t max_inject, int32_t *items, int64_t cap, int64_t *n_items)
{
    SS_CHECK_ARG(n_items && (cap == 0 || items), "ss_prefill_plan: null pointer");
    *n_items = 0;
    SS_CHECK_ARG(T > 0 && layers > 0 && max_inject > 0, "ss_prefill_plan: T=%lld layers=%d max_inject=%lld",
                 (long long)T, layers, (long long)max_inject);
    SS_CHECK_ARG(T <= INT32_MAX, "ss_prefill_plan: T=%lld too large", (long long)T);
    const bool whole = T <= max_inject;
    const int64_t per_layer = whole ? 1 : (T + max_inject - 1) / max_inject;
    const int64_t n = per_layer * layers;
    if (n > cap) return ss::fail(SS_ERR_OOM, "ss_prefill_plan: %lld items > cap %lld", (long long)n, (long long)cap);
    const int64_t seg = whole ? max_inject / T : 1;  // whole layers per batch
    int64_t i = 0;
    for (int l = 0; l < layers; ++l)
        for (int64_t c = 0; c < per_layer; ++c, ++i) {
            const int64_t t0 = whole ? 0 : c * max_inject;
            const int64_t t1 = whole ? T : std::min(T, t0 + max_inject);
            items[4 * i + 0] = (int32_t)(whole ? l / seg : l * per_layer + c);
            items[4 * i + 1] = l;
            items[4 * i + 2] = (int32_t)t0;
            items[4 * i + 3] = (int32_t)t1;
        }
    *n_items = n;
    return SS_OK;
}

}  // extern "C"

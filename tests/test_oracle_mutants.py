"""Planted mistakes in the oracle must fail its pins.

Each case copies oracle/oracle.c, applies one small edit of the kind a
mistake would make (a dropped term, a wrong sign, index or tie-break, a
transposed operand), compiles the copy on the CPU and runs the pins of the
affected group against it: at least one pin must fail.  The real oracle is
never modified.
"""
import multiprocessing
import os
import tempfile

import pytest

import oracle
import oracle.build as obuild
import pins

MUTANTS = [
    # (id, group, pattern, replacement)
    ("meta-min-is-max", "meta", "if (vx < vmn ||", "if (vx > vmn ||"),
    ("meta-drops-last-token", "meta", "for (int t = 1; t < blk; ++t)", "for (int t = 1; t < blk - 1; ++t)"),
    ("meta-zero-tie-reversed", "meta", "(vx == vmn && sign_bit(x) && !sign_bit(mn))",
     "(vx == vmn && !sign_bit(x) && sign_bit(mn))"),
    ("meta-k-transposed", "meta", "uint16_t x = rec[t * d + c];", "uint16_t x = rec[c * blk + t];"),
    ("meta-ignores-offsets", "meta", "((const char *)base + unit_off[u]\n",
     "((const char *)base + (int64_t)u * nblk_max * (int64_t)record_bytes\n"),
    ("score-min-corner", "score", "s += (a > e ? a : e);", "s += (a < e ? a : e);"),
    ("score-drops-lo", "score", "s += (a > e ? a : e);", "s += e;"),
    ("score-first-head-only", "score", "if (s > best)", "if (i == 0)"),
    ("score-sum-of-heads", "score", "double best = -INFINITY;\n                if (j < n) {",
     "double best = 0.0;\n                if (j < n) {"),
    ("score-interleaved-heads", "score", "int h = g * G + i;\n                        const uint16_t *qh",
     "int h = g + i * Hkv;\n                        const uint16_t *qh"),
    ("score-ragged-ignored", "score", "if (j < n) {", "if (j < nblk_max) {"),
    ("select-tie-to-higher", "select", "    if (sa < sb) return 1;\n    return (a > b) - (a < b);",
     "    if (sa < sb) return 1;\n    return (a < b) - (a > b);"),
    ("select-unsorted-output", "select", "qsort(order, (size_t)m, sizeof(int), ascending_int);", ""),
    ("select-smallest", "select", "if (sa > sb) return -1;\n    if (sa < sb) return 1;",
     "if (sa < sb) return -1;\n    if (sa > sb) return 1;"),
    ("lru-highest-free-slot", "lru", "if (blocks[s] < 0) { chosen = s; break; }", "if (blocks[s] < 0) { chosen = s; }"),
    ("lru-evicts-mru", "lru", "last[s] < last[chosen]", "last[s] > last[chosen]"),
    ("lru-tie-to-higher-slot", "lru", "last[s] < last[chosen]", "last[s] <= last[chosen]"),
    ("lru-evicts-selected", "lru", "if (is_selected(sel_u, k, blocks[s])) continue;", ""),
    ("lru-hit-no-refresh", "lru", "                    last[s] = step;\n                    out_u[i] = s;",
     "                    out_u[i] = s;"),
    ("gather-slot-as-source", "gather", "pool_off[u] + (int64_t)j * (int64_t)record_bytes;",
     "pool_off[u] + (int64_t)s * (int64_t)record_bytes;"),
    ("gather-unit-swap", "gather", "int u = b * Hkv + g;\n        const char *src",
     "int u = g * Hkv + b;\n        const char *src"),
    ("attn-no-scale", "attention", "z[i] = scale * dot;", "z[i] = dot;"),
    ("attn-v-row-major", "attention", "acc[c] += p * bf(Vt[c * blk + t]);", "acc[c] += p * bf(Vt[t * d + c]);"),
    ("attn-head-mod", "attention", "int g = h / G;\n            int u = b * Hkv + g;\n            const uint16_t *qh",
     "int g = h % Hkv;\n            int u = b * Hkv + g;\n            const uint16_t *qh"),
    ("attn-unnormalised", "attention", "double p = z[i] / denom;", "double p = z[i];"),
    ("attn-drops-last-entry", "attention", "for (int i = 0; i < k; ++i) {\n                int32_t s = slots",
     "for (int i = 0; i < k - 1; ++i) {\n                int32_t s = slots"),
    ("attn-drops-first-token", "attention", "for (int t = 0; t < blk; ++t) {\n                    kv_of[n] = rec;",
     "for (int t = 1; t < blk; ++t) {\n                    kv_of[n] = rec;"),
    ("append-v-row-major", "append", "rec[blk * d + c * blk + p] = kv[d + c];", "rec[blk * d + p * d + c] = kv[d + c];"),
    ("append-position-off-by-one", "append", "int j = len[b] / blk, p = len[b] % blk;",
     "int j = len[b] / blk, p = (len[b] + 1) % blk;"),
    ("append-meta-next-block", "append", "meta + ((int64_t)u * nblk_max + j) * 2 * d);",
     "meta + ((int64_t)u * nblk_max + j + 1) * 2 * d);"),
    ("append-nblk-not-updated", "append", "            nblk[b] = j + 1;\n", "            nblk[b] += 0;\n"),
    ("append-k-and-v-swapped", "append", "put_token(rec, blk, d, p, new_kv + (int64_t)u * 2 * d);",
     "put_token(rec, blk, d, p, new_kv + (int64_t)u * 2 * d + d);"),
    ("save-v-row-major", "save", "rec[blk * d + c * blk + p] = kv[d + c];", "rec[blk * d + p * d + c] = kv[d + c];"),
    ("save-ignores-len", "save", "int T = len[b] + i;", "int T = i;"),
    ("save-token-major-input", "save", "new_kv + (((int64_t)b * n_new + i) * Hkv + g) * 2 * d",
     "new_kv + (((int64_t)i * B + b) * Hkv + g) * 2 * d"),
    ("ws-whole-history", "ws", "int n_steps = m < w ? m : w;", "int n_steps = m;"),
    ("ws-counts-duplicates", "ws", "if (i == 0 || all[i] != all[i - 1])", "if (1)"),
    ("ws-counts-padding", "ws", "                    if (j >= 0)\n                        all[n++] = j;",
     "                    all[n++] = j;"),
    ("ws-oldest-steps", "ws", "for (int s = m - n_steps; s < m; ++s)", "for (int s = 0; s < n_steps; ++s)"),
    ("ws-chunked-one-layer", "ws", "        layer_count = layers;", "        layer_count = 1;"),
    ("ws-prefill-floor", "ws", "int64_t blocks = (tokens + blk - 1) / blk;", "int64_t blocks = tokens / blk;"),
    ("schedule-strict", "schedule", "if (used + ws[i] <= m_avl) {", "if (used + ws[i] < m_avl) {"),
    ("schedule-stops-at-first-reject", "schedule", "            admit[i] = 0;\n",
     "            admit[i] = 0;\n            m_avl = -1;\n"),
    ("mean-divides-by-blk-minus-1", "meta_mean", "m[c] = bf16_nearest(s / (double)blk);",
     "m[c] = bf16_nearest(s / (double)(blk > 1 ? blk - 1 : 1));"),
    ("mean-skips-first-token", "meta_mean", "for (int t = 0; t < blk; ++t) {\n                        double v = bf(",
     "for (int t = 1; t < blk; ++t) {\n                        double v = bf("),
    ("mean-truncates", "meta_mean", "double r = ldexp(nearbyint(ldexp(x, -qexp)), qexp);",
     "double r = ldexp(trunc(ldexp(x, -qexp)), qexp);"),
    ("mean-ties-away-from-zero", "meta_mean", "double r = ldexp(nearbyint(ldexp(x, -qexp)), qexp);",
     "double r = ldexp(round(ldexp(x, -qexp)), qexp);"),
    ("mean-rounds-through-fp32", "meta_mean", "m[c] = bf16_nearest(s / (double)blk);",
     "m[c] = bf16_nearest((double)(float)(s / (double)blk));"),
    ("mean-nine-bit-significand", "meta_mean", "int qexp = e - 8;", "int qexp = e - 9;"),
    ("mean-accepts-inexact-sums", "meta_mean", "                        if (err != 0.0)\n                            return 2;\n",
     ""),
    ("mean-reads-v", "meta_mean", "double v = bf(rec[t * d + c]);", "double v = bf(rec[blk * d + c * blk + t]);"),
    ("variant-mean-reads-hi", "score_variant", "s += bf(qh[c]) * bf(mj[c]);", "s += bf(qh[c]) * bf(mj[d + c]);"),
    ("variant-sum-is-max", "score_variant", "= agg == 0 ? best : total;", "= best;"),
    ("variant-sum-drops-last-head", "score_variant", "                    total += s;\n",
     "                    if (i < G - 1) total += s;\n"),
    ("variant-cuboid-min-corner", "score_variant", "s += at_lo > at_hi ? at_lo : at_hi;",
     "s += at_lo < at_hi ? at_lo : at_hi;"),
    ("variant-ragged-ignored", "score_variant", "if (j >= n) {", "if (j >= nblk_max) {"),
    ("variant-mean-row-stride", "score_variant", "int row = kind == 0 ? 2 * d : d;", "int row = 2 * d;"),
    ("plan-one-layer-per-batch", "prefill_plan", "int64_t s = max_inject / T;", "int64_t s = 1;"),
    ("plan-chunk-floor", "prefill_plan", "int64_t chunks = (T + max_inject - 1) / max_inject;",
     "int64_t chunks = T / max_inject;"),
    ("plan-chunk-overruns", "prefill_plan", "int64_t e = b + max_inject < T ? b + max_inject : T;",
     "int64_t e = b + max_inject;"),
    ("plan-segment-off-by-one", "prefill_plan", "int64_t s = max_inject / T;", "int64_t s = max_inject / T + 1;"),
    ("save-ignores-offsets", "save", "(char *)pool + pool_off[u] + (int64_t)j",
     "(char *)pool + (int64_t)u * pool_blocks[b] * (int64_t)record_bytes + (int64_t)j"),
]


@pytest.fixture(scope="module")
def src():
    return open(obuild.SRC).read()


@pytest.mark.parametrize("mid,group,pattern,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(mid, group, pattern, repl, src):
    assert src.count(pattern) == 1, f"mutation pattern for {mid} must occur exactly once"
    mutated = src.replace(pattern, repl)
    with tempfile.TemporaryDirectory() as tmp:
        path = os.path.join(tmp, f"oracle_{mid}.c")
        open(path, "w").write(mutated)
        lib = obuild.build(path, os.path.join(tmp, f"liboracle_{mid}.so"), extra=("-Wno-unused-function",
                                                                                 "-Wno-unused-variable",
                                                                                 "-Wno-unused-parameter"))
        # run the pins in a forked child so that a mutant that crashes
        # (an out-of-bounds index) counts as caught instead of ending pytest
        ctx = multiprocessing.get_context("fork")
        child = ctx.Process(target=_run_group, args=(lib, group))
        child.start()
        child.join(120)
        hung = child.is_alive()
        if hung:
            child.kill()
            child.join()
        # a child that hangs has not shown anything: only a pin failure or a
        # crash counts as catching the mistake
        assert not hung, f"pins of {group} did not finish for planted mistake {mid}"
        assert child.exitcode != 0, f"planted mistake {mid} passed every {group} pin"


def _run_group(lib, group):
    import faulthandler
    faulthandler.disable()  # a crashing mutant is an expected outcome here
    # the parent's intra-op thread pool does not survive fork(): run torch's
    # CPU ops of the pins on this thread only
    import torch
    torch.set_num_threads(1)
    O = oracle.Oracle(oracle.load(lib))
    for pin in pins.GROUPS[group]:
        try:
            pin(O)
        except (AssertionError, RuntimeError, OverflowError, ValueError):
            os._exit(1)
    os._exit(0)

"""The library's host-side block cache (ss_cache_*) against the oracle's
LRU on seeded selection streams: slots, miss lists and the whole slot state
must match exactly, step after step.  Runs on the CPU (no GPU involved)."""
import numpy as np
import pytest

import synth
from paper_2509_24626_amd import binding as ss


class LibCache:
    def __init__(self, B, Hkv, nblk, cap, rec=8192, threads=None):
        self.B, self.Hkv = B, Hkv
        self.h = ss.ss_cache_create(B, Hkv, np.ascontiguousarray(nblk, np.int32), np.ascontiguousarray(cap, np.int32),
                                    rec)
        if threads:
            ss.ss_cache_set_threads(self.h, threads)

    def __del__(self):
        ss.ss_cache_destroy(self.h)

    def step(self, t, sel):
        sel = np.ascontiguousarray(sel, np.int32)
        k = sel.shape[-1]
        slots = np.empty_like(sel)
        cap = self.B * self.Hkv * k
        miss = np.empty((cap, 4), np.int32)
        n = ss.ss_cache_resolve(self.h, t, sel, k, slots, miss, cap)
        return slots, miss[:n].copy()

    def export(self):
        n = ss.ss_cache_total_slots(self.h)
        blocks = np.empty(n, np.int32)
        last = np.empty(n, np.int64)
        ss.ss_cache_export(self.h, blocks, last)
        return blocks, last


def run_stream(oracle_impl, nblk, Hkv, k, cap, steps, churn, seed, threads=None, step_ids=None):
    B = len(nblk)
    stream = synth.gen.selection_stream(nblk, Hkv, k, steps, churn, seed)
    lib = LibCache(B, Hkv, nblk, cap, threads=threads)
    ora = oracle_impl.lru(B, Hkv, nblk, cap)
    total_miss = 0
    for s in range(steps):
        t = s if step_ids is None else step_ids[s]
        ls, lm = lib.step(t, stream[s])
        os_, om = ora.step(t, stream[s])
        np.testing.assert_array_equal(ls, os_, err_msg=f"slots differ at step {s}")
        np.testing.assert_array_equal(lm, om, err_msg=f"miss list differs at step {s}")
        total_miss += len(lm)
    lb, ll = lib.export()
    ob, ol = ora.export()
    np.testing.assert_array_equal(lb, ob)
    np.testing.assert_array_equal(ll, ol)
    return total_miss


@pytest.mark.parametrize("churn", [0.0, 0.2, 0.6, 1.0])
def test_stream_matches_oracle(oracle_impl, churn):
    nblk = [64, 40, 97]
    Hkv, k = 3, 12
    cap = np.array([[16, 12, 30], [13, 20, 12], [25, 14, 40]], np.int32)
    run_stream(oracle_impl, nblk, Hkv, k, cap, steps=20, churn=churn, seed=7)


def test_ragged_and_short_sequences(oracle_impl):
    # sequences shorter than k (-1 padding), capacity == k, a zero-length sequence
    nblk = [5, 0, 300, 17]
    Hkv, k = 2, 8
    cap = np.array([[8, 8], [0, 3], [60, 8], [9, 12]], np.int32)
    run_stream(oracle_impl, nblk, Hkv, k, cap, steps=15, churn=0.5, seed=11)


@pytest.mark.parametrize("threads", [1, 3, 16])
def test_thread_count_does_not_change_results(oracle_impl, threads):
    nblk = [200] * 12
    Hkv, k = 4, 16
    cap = np.full((12, 4), 40, np.int32)
    run_stream(oracle_impl, nblk, Hkv, k, cap, steps=10, churn=0.3, seed=13, threads=threads)


def test_caches_resolved_from_several_threads(oracle_impl):
    """The resolve workers are one pool per process, shared by every cache,
    and one call validates and updates in a single dispatch with a barrier
    between the passes.  Four caches (different shapes and thread counts)
    resolved at the same time from four Python threads (the C call releases
    the interpreter lock) must each match the oracle step for step."""
    import threading
    shapes = [([120] * 9, 3, 10, 30, 2), ([64, 7, 200], 4, 12, 25, 5), ([300] * 4, 2, 16, 48, 16), ([90] * 6, 1, 8, 8, 1)]
    errors = []

    def run(i, nblk, Hkv, k, capv, threads):
        try:
            cap = np.full((len(nblk), Hkv), capv, np.int32)
            run_stream(oracle_impl, nblk, Hkv, k, cap, steps=25, churn=0.4, seed=100 + i, threads=threads)
        except BaseException as e:  # reported on the main thread
            errors.append((i, e))

    workers = [threading.Thread(target=run, args=(i, *sh)) for i, sh in enumerate(shapes)]
    for w in workers:
        w.start()
    for w in workers:
        w.join(timeout=120)
    assert not any(w.is_alive() for w in workers), "a resolve did not return"
    assert not errors, errors


def test_repeated_step_numbers(oracle_impl):
    nblk = [50, 50]
    cap = np.full((2, 2), 10, np.int32)
    ids = [0, 0, 1, 1, 1, 2, 5, 5, 9, 9]
    run_stream(oracle_impl, nblk, 2, 6, cap, steps=10, churn=0.7, seed=17, step_ids=ids)


def test_config_shaped_stream(oracle_impl):
    # the hierarchical 128k-context workload's cache shape at reduced batch:
    # 8192 blocks per unit, 25% capacity, k = 128
    nblk = [8192] * 2
    cap = np.full((2, 8), 2048, np.int32)
    m = run_stream(oracle_impl, nblk, 8, 128, cap, steps=6, churn=0.25, seed=19)
    assert m > 0


def test_capacity_error_leaves_state_unchanged():
    c = LibCache(1, 2, [10], [[4, 2]])
    c.step(0, np.array([[[0, 1, -1], [3, 4, -1]]], np.int32))
    before = c.export()
    with pytest.raises(ss.SparseServeError) as e:
        c.step(1, np.array([[[5, 6, 7], [1, 2, 3]]], np.int32))  # unit 1 has 2 slots
    assert e.value.status == ss.SS_ERR_CAPACITY
    after = c.export()
    np.testing.assert_array_equal(before[0], after[0])
    np.testing.assert_array_equal(before[1], after[1])


@pytest.mark.parametrize("bad", [[3, 1, -1], [1, 1, 2], [-1, 2, 3], [1, 10, -1], [1, -2, -1]])
def test_malformed_selection_rejected(bad):
    c = LibCache(1, 1, [10], [[8]])
    with pytest.raises(ss.SparseServeError) as e:
        c.step(0, np.array([[bad]], np.int32))
    assert e.value.status == ss.SS_ERR_INVALID_ARG


def test_step_must_not_decrease():
    c = LibCache(1, 1, [10], [[8]])
    c.step(5, np.array([[[1, 2]]], np.int32))
    with pytest.raises(ss.SparseServeError) as e:
        c.step(4, np.array([[[1, 2]]], np.int32))
    assert e.value.status == ss.SS_ERR_INVALID_ARG


def test_miss_capacity_too_small():
    c = LibCache(1, 1, [10], [[8]])
    sel = np.array([[[1, 2, 3]]], np.int32)
    slots = np.empty_like(sel)
    miss = np.empty((2, 4), np.int32)
    with pytest.raises(ss.SparseServeError) as e:
        ss.ss_cache_resolve(c.h, 0, sel, 3, slots, miss, 2)
    assert e.value.status == ss.SS_ERR_OOM


def test_region_offsets():
    c = LibCache(2, 2, [10, 10], [[3, 0], [5, 1]], rec=4096)
    off = np.empty(4, np.int64)
    ss.ss_cache_region_offsets(c.h, off)
    assert off.tolist() == [0, 3 * 4096, 3 * 4096, 8 * 4096]
    assert ss.ss_cache_total_slots(c.h) == 9


@pytest.mark.parametrize("cuts", [[0, 3], [0, 1, 3], [0, 1, 2, 3], [0, 0, 2, 3]])
def test_resolve_in_ranges_equals_whole(oracle_impl, cuts):
    """A step resolved as several disjoint sequence ranges (same step
    number) gives exactly the whole-batch result, step after step."""
    nblk = [64, 40, 97]
    Hkv, k = 2, 10
    cap = np.array([[16, 12], [13, 20], [25, 14]], np.int32)
    stream = synth.gen.selection_stream(nblk, Hkv, k, 12, 0.4, 23)
    lib = LibCache(3, Hkv, nblk, cap)
    ora = oracle_impl.lru(3, Hkv, nblk, cap)
    for t in range(12):
        sel = stream[t]
        slots = np.empty_like(sel)
        miss_all = []
        for b0, b1 in zip(cuts[:-1], cuts[1:]):
            rows = (b1 - b0) * Hkv * k
            miss = np.empty((max(rows, 1), 4), np.int32)
            n = ss.ss_cache_resolve_range(lib.h, t, b0, b1, np.ascontiguousarray(sel[b0:b1]), k,
                                          slots[b0:b1], miss, rows)
            miss_all.append(miss[:n])
        os_, om = ora.step(t, sel)
        np.testing.assert_array_equal(slots, os_)
        np.testing.assert_array_equal(np.concatenate(miss_all), om)


def test_resolve_range_rejects_bad_range():
    c = LibCache(2, 1, [10, 10], [[4], [4]])
    sel = np.zeros((1, 1, 2), np.int32)
    for b0, b1 in [(-1, 1), (1, 0), (0, 3)]:
        with pytest.raises(ss.SparseServeError) as e:
            ss.ss_cache_resolve_range(c.h, 0, b0, b1, sel, 2, np.empty_like(sel), np.empty((4, 4), np.int32), 4)
        assert e.value.status == ss.SS_ERR_INVALID_ARG


def test_growing_sequences_match_oracle(oracle_impl):
    """Sequences gain blocks between steps (ss_cache_set_blocks, several
    times past the reserved room): with selections drawn from the blocks
    that exist at each step, slots and misses equal the oracle's LRU, which
    knows the final block counts from the start (block counts only bound
    which indices are valid)."""
    rng = np.random.default_rng(21)
    B, Hkv, k = 3, 2, 6
    n0 = np.array([8, 20, 30], np.int32)
    steps = 40
    grow = rng.integers(0, 3, size=(steps, B)).astype(np.int32)
    grow[5] = [40, 0, 0]  # one jump well past the slack
    nb = [n0.copy()]
    for s in range(steps):
        nb.append(nb[-1] + grow[s])
    final = nb[-1]
    cap = np.repeat([8, 10, 12], Hkv).astype(np.int32)
    lib = LibCache(B, Hkv, n0, cap)
    ora = oracle_impl.lru(B, Hkv, final, cap)
    for s in range(steps):
        cur = nb[s]
        if s:
            ss.ss_cache_set_blocks(lib.h, cur)
        sel = np.full((B, Hkv, k), -1, np.int32)
        for b in range(B):
            for g in range(Hkv):
                # favour the newest blocks, as a growing context would
                pick = np.unique(np.concatenate([rng.integers(max(0, cur[b] - 12), cur[b], size=k - 2),
                                                 rng.integers(0, cur[b], size=2)]))[:k]
                sel[b, g, :len(pick)] = pick
        ls, lm = lib.step(s, sel)
        os_, om = ora.step(s, sel)
        np.testing.assert_array_equal(ls, os_, err_msg=f"slots differ at step {s}")
        np.testing.assert_array_equal(lm, om, err_msg=f"misses differ at step {s}")
    lb, ll = lib.export()
    ob, ol = ora.export()
    np.testing.assert_array_equal(lb, ob)
    np.testing.assert_array_equal(ll, ol)


def test_set_blocks_rejects_shrinking_and_guards_new_blocks():
    lib = LibCache(2, 1, [4, 4], [4, 4])
    with pytest.raises(ss.SparseServeError):
        ss.ss_cache_set_blocks(lib.h, [3, 4])
    sel = np.array([[[4, -1]], [[0, -1]]], np.int32)
    with pytest.raises(ss.SparseServeError):  # block 4 does not exist yet
        lib.step(0, sel)
    ss.ss_cache_set_blocks(lib.h, [5, 4])
    slots, miss = lib.step(0, sel)
    assert slots[0, 0, 0] == 0 and len(miss) == 2

"""The block cache resolved on the GPU (ss_dev_cache_*) against the oracle's
LRU on seeded selection streams: slots, each unit's miss rows and the whole
slot state must match exactly, step after step.  Streams with low and high
churn, ragged and short sequences, caches that fill in the middle of a
step, repeated step numbers, resolves split over sequence ranges, the
128k-workload and GQA-7 shapes, and the error flags."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ss():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2509_24626_amd import binding
    binding.lib()
    return binding


class DevCache:
    def __init__(self, ss, B, Hkv, nblk, cap, k):
        self.ss, self.B, self.Hkv, self.k = ss, B, Hkv, k
        self.units = B * Hkv
        self.h = ss.ss_dev_cache_create(B, Hkv, np.asarray(nblk, np.int32), np.asarray(cap, np.int32))
        self.nblk = torch.from_numpy(np.asarray(nblk, np.int32)).cuda()
        self.slots = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
        self.miss = torch.full((self.units, k, 4), -7, dtype=torch.int32, device="cuda")
        self.cap = np.asarray(cap, np.int32)

    def close(self):
        self.ss.ss_dev_cache_destroy(self.h)

    def step(self, t, sel, ranges=None):
        sel_d = torch.from_numpy(np.ascontiguousarray(sel, np.int32)).cuda()
        for b0, b1 in (ranges or [(0, self.B)]):
            self.ss.ss_dev_cache_resolve(self.h, t, b0, b1, sel_d[b0:b1], self.k, self.nblk, self.slots[b0:b1],
                                         self.miss)
        counts, err = self.ss.ss_dev_cache_miss_counts(self.h, self.units)
        rows = self.miss.cpu().numpy()
        miss = np.concatenate([rows[u, :counts[u]] for u in range(self.units)] + [np.zeros((0, 4), np.int32)])
        return self.slots.cpu().numpy(), miss, err

    def export(self):
        n = self.ss.ss_dev_cache_total_slots(self.h)
        blocks = np.empty(n, np.int32)
        last = np.empty(n, np.int64)
        self.ss.ss_dev_cache_export(self.h, blocks, last)
        return blocks, last


def run_stream(ss, oracle_impl, nblk, Hkv, k, cap, steps, churn, seed, step_ids=None, ranges=None):
    B = len(nblk)
    stream = synth.gen.selection_stream(nblk, Hkv, k, steps, churn, seed)
    dev = DevCache(ss, B, Hkv, nblk, cap, k)
    ora = oracle_impl.lru(B, Hkv, nblk, cap)
    total = 0
    try:
        for s in range(steps):
            t = s if step_ids is None else step_ids[s]
            ds, dm, err = dev.step(t, stream[s], ranges)
            assert err == 0
            os_, om = ora.step(t, stream[s])
            np.testing.assert_array_equal(ds, os_, err_msg=f"slots differ at step {s}")
            np.testing.assert_array_equal(dm, om, err_msg=f"miss rows differ at step {s}")
            total += len(dm)
        db, dl = dev.export()
        ob, ol = ora.export()
        np.testing.assert_array_equal(db, ob)
        np.testing.assert_array_equal(dl[ob >= 0], ol[ob >= 0])
        assert ss.ss_dev_cache_total_misses(dev.h) == total
    finally:
        dev.close()
    return total


@pytest.mark.parametrize("churn", [0.0, 0.2, 0.6, 1.0])
def test_stream_matches_oracle(ss, oracle_impl, churn):
    nblk = np.array([300, 120, 64], np.int32)
    cap = np.repeat([40, 24, 32], 2).astype(np.int32)
    print(f"[gpu] device resolve, churn {churn}", flush=True)
    run_stream(ss, oracle_impl, nblk, 2, 16, cap, 25, churn, seed=int(churn * 10) + 1)


def test_ragged_short_and_empty_sequences(ss, oracle_impl):
    nblk = np.array([50, 7, 0, 33], np.int32)
    cap = np.repeat([20, 8, 0, 16], 3).astype(np.int32)
    run_stream(ss, oracle_impl, nblk, 3, 12, cap, 20, 0.5, seed=11)


def test_repeated_step_numbers_and_ranges(ss, oracle_impl):
    nblk = np.array([200, 150, 90, 60], np.int32)
    cap = np.repeat([30, 30, 20, 20], 2).astype(np.int32)
    ids = [0, 1, 1, 2, 5, 5, 5, 6, 9, 10, 10, 11]
    run_stream(ss, oracle_impl, nblk, 2, 16, cap, len(ids), 0.4, seed=12, step_ids=ids, ranges=[(0, 1), (1, 3), (3, 4)])


def test_hier128k_shape(ss, oracle_impl):
    """64 sequences x 8 KV heads, 8192 blocks, k = 128, 2048 slots: the shape
    of the 128k workload, with drifting selections."""
    nblk = np.full(64, 8192, np.int32)
    cap = np.full(64 * 8, 2048, np.int32)
    run_stream(ss, oracle_impl, nblk, 8, 128, cap, 18, 0.25, seed=13)


def test_gqa7_shape_k512(ss, oracle_impl):
    """k = 512 and 2457 slots per unit (the GQA-7 workload's shape)."""
    nblk = np.full(6, 16384, np.int32)
    cap = np.full(6 * 4, 2457, np.int32)
    run_stream(ss, oracle_impl, nblk, 4, 512, cap, 10, 0.5, seed=14)


def test_largest_capacity_and_k(ss, oracle_impl):
    """8192 slots (the largest supported region, every LDS array full) and
    k = 512 with full churn: the cache fills after 16 steps, then every step
    evicts 512 of 8192 candidates."""
    nblk = np.array([16384, 12000], np.int32)
    cap = np.full(2 * 2, 8192, np.int32)
    run_stream(ss, oracle_impl, nblk, 2, 512, cap, 24, 1.0, seed=15)


def test_error_flags_leave_units_unchanged(ss, oracle_impl):
    B, Hkv, k = 2, 1, 4
    nblk = np.array([20, 20], np.int32)
    cap = np.array([3, 4], np.int32)
    dev = DevCache(ss, B, Hkv, nblk, cap, k)
    try:
        ok = np.array([[[1, 2, 3, -1]], [[4, 5, -1, -1]]], np.int32)
        s1, m1, err = dev.step(0, ok)
        assert err == 0 and len(m1) == 5
        before = dev.export()
        bad = np.array([[[1, 2, 3, 4]], [[5, 4, -1, -1]]], np.int32)  # too many for 3 slots; not ascending
        s2, m2, err = dev.step(1, bad)
        assert err == 3 and len(m2) == 0 and np.all(s2 == -1)
        after = dev.export()
        np.testing.assert_array_equal(before[0], after[0])
        np.testing.assert_array_equal(before[1], after[1])
        with pytest.raises(ss.SparseServeError):  # steps must not decrease
            dev.step(0, ok)
    finally:
        dev.close()


def test_rejects_unsupported_sizes(ss):
    with pytest.raises(ss.SparseServeError):
        ss.ss_dev_cache_create(1, 1, np.array([10], np.int32), np.array([8193], np.int32))
    h = ss.ss_dev_cache_create(1, 1, np.array([10], np.int32), np.array([4], np.int32))
    try:
        z = torch.zeros(1024, dtype=torch.int32, device="cuda")
        with pytest.raises(ss.SparseServeError):
            ss.ss_dev_cache_resolve(h, 0, 0, 1, z, 513, z, z, z)
    finally:
        ss.ss_dev_cache_destroy(h)

"""Pins for the CPU oracle: checks that tie it to the paper's definitions
through something other than itself (hand-worked fixtures, closed forms,
invariants, special cases that reduce to a library routine, brute force on
tiny inputs).

Every pin takes an `oracle.Oracle` instance so the same checks run on the
real oracle (tests/test_oracle_pins.py) and on copies of it with planted
mistakes (tests/test_oracle_mutants.py), where at least one pin of the
group must fail.  Each pin raises AssertionError on failure.
"""
import itertools
import math
import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ------------------------------------------------------------- test helpers
def bits_to_f64(u16):
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bits(x):
    """Exact bf16 values -> bit patterns (asserts exactness)."""
    x32 = np.asarray(x, dtype=np.float32)
    u = x32.view(np.uint32)
    assert np.all((u & 0xFFFF) == 0), "value not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def rand_bf16(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(*shape, generator=g) * scale
    return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def make_records(Kbits, Vbits):
    """Kbits, Vbits: uint16 [..., nblk, blk, d] -> records uint16 [..., nblk, 2*blk*d]
    (K tile row-major, V tile channel-major)."""
    Kbits = np.asarray(Kbits, dtype=np.uint16)
    Vbits = np.asarray(Vbits, dtype=np.uint16)
    *lead, blk, d = Kbits.shape
    kpart = Kbits.reshape(*lead, blk * d)
    vpart = np.swapaxes(Vbits, -1, -2).reshape(*lead, d * blk)
    return np.ascontiguousarray(np.concatenate([kpart, vpart], axis=-1))


def dense_offsets(units, nblk_max, blk, d):
    return (np.arange(units, dtype=np.int64) * nblk_max * 2 * blk * d * 2)


def read_fixture(name):
    rows = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        rows[key] = vals
    return rows


# ------------------------------------------------------------------ O0 meta
def pin_meta_bruteforce(O):
    """lo/hi equal numpy's channel-wise min/max over each block's tokens,
    and lo <= K <= hi for every token (the cuboid bounds every key)."""
    B, Hkv, nblk, blk, d = 2, 3, 5, 4, 8
    K = rand_bf16((B, Hkv, nblk, blk, d), 11)
    V = rand_bf16((B, Hkv, nblk, blk, d), 12)
    rec = make_records(K, V)
    meta = O.build_metadata(rec, dense_offsets(B * Hkv, nblk, blk, d), np.full(B, nblk, np.int32),
                            B, Hkv, nblk, blk, d)
    Kf = bits_to_f64(K)
    lo = bits_to_f64(meta[..., 0, :])
    hi = bits_to_f64(meta[..., 1, :])
    assert np.array_equal(lo, Kf.min(axis=3)), "lo is not the channel-wise minimum"
    assert np.array_equal(hi, Kf.max(axis=3)), "hi is not the channel-wise maximum"
    assert np.all(lo[:, :, :, None, :] <= Kf) and np.all(Kf <= hi[:, :, :, None, :])


def pin_meta_ragged_untouched(O):
    """Blocks past a sequence's length are not written; shorter sequences
    still get the right metadata."""
    B, Hkv, nblk_max, blk, d = 3, 2, 6, 2, 4
    nblk = np.array([6, 2, 0], np.int32)
    K = rand_bf16((B, Hkv, nblk_max, blk, d), 21)
    rec = make_records(K, K)
    sentinel = np.full((B, Hkv, nblk_max, 2, d), 0x7777, np.uint16)
    meta = O.build_metadata(rec, dense_offsets(B * Hkv, nblk_max, blk, d), nblk, B, Hkv, nblk_max, blk, d,
                            meta=sentinel.copy())
    Kf = bits_to_f64(K)
    for b in range(B):
        n = nblk[b]
        assert np.all(meta[b, :, n:] == 0x7777), "wrote past the sequence's blocks"
        assert np.array_equal(bits_to_f64(meta[b, :, :n, 0]), Kf[b, :, :n].min(axis=2))
        assert np.array_equal(bits_to_f64(meta[b, :, :n, 1]), Kf[b, :, :n].max(axis=2))


def pin_meta_signed_zero(O):
    """Hand-worked fixture: -0 < +0 in the min/max (totalOrder reading)."""
    fx = read_fixture("metadata_signed_zero.txt")
    K = np.array([[int(x, 16) for x in fx[f"key_t{t}"]] for t in range(3)], np.uint16)
    rec = make_records(K[None, None, None], K[None, None, None])
    meta = O.build_metadata(rec, np.zeros(1, np.int64), np.array([1], np.int32), 1, 1, 1, 3, 3)
    assert [int(x) for x in meta[0, 0, 0, 0]] == [int(x, 16) for x in fx["lo"]]
    assert [int(x) for x in meta[0, 0, 0, 1]] == [int(x, 16) for x in fx["hi"]]


def pin_meta_record_offsets(O):
    """Units placed at arbitrary (non-dense, reversed) byte offsets."""
    Hkv, nblk, blk, d = 3, 4, 2, 4
    K = rand_bf16((1, Hkv, nblk, blk, d), 31)
    rec = make_records(K, K)[0]  # [Hkv][nblk][rec]
    rb = rec.shape[-1] * 2
    buf = np.zeros((Hkv + 1) * nblk * rec.shape[-1], np.uint16)
    offs = np.array([(Hkv - g) * nblk * rb for g in range(Hkv)], np.int64)
    for g in range(Hkv):
        w = offs[g] // 2
        buf[w:w + nblk * rec.shape[-1]] = rec[g].reshape(-1)
    meta = O.build_metadata(buf, offs, np.array([nblk], np.int32), 1, Hkv, nblk, blk, d)
    Kf = bits_to_f64(K)
    assert np.array_equal(bits_to_f64(meta[0, :, :, 0]), Kf[0].min(axis=2))
    assert np.array_equal(bits_to_f64(meta[0, :, :, 1]), Kf[0].max(axis=2))


# ----------------------------------------------------------------- O1 score
def _meta_from_keys(Kf):
    """[..., blk, d] exact bf16 values -> metadata bits [..., 2, d] via numpy min/max."""
    return np.stack([f64_to_bits(Kf.min(axis=-2)), f64_to_bits(Kf.max(axis=-2))], axis=-2)


def pin_score_fixture(O):
    """Hand-worked fixture (golden/score_box.txt)."""
    fx = read_fixture("score_box.txt")
    K = np.array([[float(x) for x in fx["key_t0"]], [float(x) for x in fx["key_t1"]]])
    q = np.array([[float(x) for x in fx["q_h0"]], [float(x) for x in fx["q_h1"]]])
    meta = _meta_from_keys(K)[None, None, None]
    S = O.score(f64_to_bits(q)[None], meta, np.array([1], np.int32), 2, 1, 1, 4)
    assert S[0, 0, 0] == float(fx["score"][0]), S
    # each head alone (G = 1 views of the same data)
    for h in range(2):
        S1 = O.score(f64_to_bits(q[h:h + 1])[None], meta, np.array([1], np.int32), 1, 1, 1, 4)
        assert S1[0, 0, 0] == float(fx[f"s_h{h}"][0]), (h, S1)


def pin_score_upper_bound(O):
    """Every token's q_h.k_t is <= the block score, for every head of the
    group (the cuboid contains all keys of the block)."""
    B, Hq, Hkv, nblk, blk, d = 2, 6, 2, 7, 5, 16
    K = rand_bf16((B, Hkv, nblk, blk, d), 41, 1.5)
    q = rand_bf16((B, Hq, d), 42)
    meta = _meta_from_keys(bits_to_f64(K))
    S = O.score(q, meta, np.full(B, nblk, np.int32), Hq, Hkv, nblk, d)
    qf, Kf = bits_to_f64(q), bits_to_f64(K)
    G = Hq // Hkv
    for b, g in itertools.product(range(B), range(Hkv)):
        dots = np.einsum("hc,jtc->hjt", qf[b, g * G:(g + 1) * G], Kf[b, g])
        assert np.all(dots.max(axis=(0, 2)) <= S[b, g] + 1e-12 * np.abs(S[b, g])), "not an upper bound"


def pin_score_point_block(O):
    """blk = 1: the cuboid is a point, so the score equals max_h q_h.k exactly
    (up to fp64 rounding of a 32-term sum)."""
    B, Hq, Hkv, nblk, d = 2, 8, 2, 9, 32
    K = rand_bf16((B, Hkv, nblk, 1, d), 51)
    q = rand_bf16((B, Hq, d), 52)
    meta = _meta_from_keys(bits_to_f64(K))
    S = O.score(q, meta, np.full(B, nblk, np.int32), Hq, Hkv, nblk, d)
    qf, Kf = bits_to_f64(q), bits_to_f64(K)
    G = Hq // Hkv
    for b, g in itertools.product(range(B), range(Hkv)):
        ref = (qf[b, g * G:(g + 1) * G] @ Kf[b, g, :, 0].T).max(axis=0)
        assert np.allclose(S[b, g], ref, rtol=1e-13, atol=1e-13), (S[b, g], ref)


def pin_score_corner_tight(O):
    """A block that contains the cuboid corner favoured by q (hi where q >= 0,
    lo where q < 0) has score exactly q.corner: the bound is attained."""
    d, blk, nblk = 16, 6, 5
    rng = np.random.default_rng(61)
    q = rand_bf16((1, 1, d), 62)
    qf = bits_to_f64(q)[0, 0]
    K = bits_to_f64(rand_bf16((1, 1, nblk, blk, d), 63))
    lo, hi = K.min(axis=3), K.max(axis=3)
    corner = np.where(qf >= 0, hi, lo)  # [1,1,nblk,d]
    for j in range(nblk):
        K[0, 0, j, rng.integers(blk)] = corner[0, 0, j]
    meta = _meta_from_keys(K)
    S = O.score(q, meta, np.array([nblk], np.int32), 1, 1, nblk, d)
    ref = corner[0, 0] @ qf
    assert np.allclose(S[0, 0], ref, rtol=1e-13, atol=1e-13), (S[0, 0], ref)


def pin_score_ragged(O):
    """Blocks past a sequence's length score -inf; earlier blocks unaffected."""
    B, Hq, Hkv, nblk_max, d = 2, 2, 1, 5, 8
    K = bits_to_f64(rand_bf16((B, Hkv, nblk_max, 1, d), 71))
    q = rand_bf16((B, Hq, d), 72)
    meta = _meta_from_keys(K)
    S = O.score(q, meta, np.array([5, 3], np.int32), Hq, Hkv, nblk_max, d)
    assert np.all(np.isneginf(S[1, 0, 3:])) and np.all(np.isfinite(S[1, 0, :3]))
    ref = (bits_to_f64(q)[1] @ K[1, 0, :3, 0].T).max(axis=0)
    assert np.allclose(S[1, 0, :3], ref, rtol=1e-13)


# ---------------------------------------------------------------- O2 select
def _brute_select(S_row, n, k):
    order = sorted(range(n), key=lambda j: (-S_row[j], j))[:k]
    out = sorted(order)
    return out + [-1] * (k - len(out))


def pin_select_fixture(O):
    fx = read_fixture("select_ties.txt")
    s = np.array([float(x) for x in fx["scores"]])
    for k in (1, 2, 3, 4, 6, 8):
        sel = O.select(s[None, None], np.array([6], np.int32), k)
        assert sel[0, 0].tolist() == [int(x) for x in fx[f"k{k}"]], (k, sel)


def pin_select_bruteforce(O):
    """Random scores with many exact ties vs a full stable sort."""
    rng = np.random.default_rng(81)
    B, Hkv, nblk_max = 3, 2, 40
    nblk = np.array([40, 17, 3], np.int32)
    for trial in range(20):
        S = rng.integers(0, 6, size=(B, Hkv, nblk_max)).astype(np.float64) * 0.5 - 1.0
        k = int(rng.integers(1, 45))
        sel = O.select(S, nblk, k)
        for b, g in itertools.product(range(B), range(Hkv)):
            assert sel[b, g].tolist() == _brute_select(S[b, g], int(nblk[b]), k), (trial, b, g, k)


def pin_select_all_when_k_large(O):
    """k >= number of blocks selects every block, in order."""
    S = np.random.default_rng(91).standard_normal((1, 1, 10))
    sel = O.select(S, np.array([10], np.int32), 10)
    assert sel[0, 0].tolist() == list(range(10))


# ------------------------------------------------------------------ O3 LRU
class ListLRU:
    """Brute-force reference for one unit: an explicit recency list of
    (last_use, slot) entries scanned in order."""

    def __init__(self, cap):
        self.cap = cap
        self.block = [-1] * cap
        self.last = [0] * cap

    def step(self, t, sel):
        sel = [j for j in sel if j >= 0]
        slots = {}
        for j in sel:
            if j in self.block:
                s = self.block.index(j)
                self.last[s] = t
                slots[j] = s
        misses = []
        for j in sel:
            if j in slots:
                continue
            empty = [s for s in range(self.cap) if self.block[s] < 0]
            if empty:
                s = empty[0]
            else:
                recency = sorted((self.last[s], s) for s in range(self.cap) if self.block[s] not in sel)
                s = recency[0][1]
            self.block[s] = j
            self.last[s] = t
            slots[j] = s
            misses.append((j, s))
        return [slots[j] for j in sel], misses


def pin_lru_fixture(O):
    rows = []
    final = None
    for line in open(os.path.join(GOLDEN, "lru_trace.txt")):
        line = line.strip()
        if line.startswith("step"):
            parts = [p.strip() for p in line.split("|")]
            t = int(parts[0].split()[1])
            sel = [int(x) for x in parts[1].split()]
            slots = [int(x) for x in parts[2].split()]
            miss = [tuple(int(y) for y in x.split(":")) for x in parts[3].split()] if len(parts) > 3 else []
            rows.append((t, sel, slots, miss))
        elif line.startswith("final"):
            final = [tuple(int(y) for y in x.split(":")) for x in line.split()[1:]]
    c = O.lru(1, 1, np.array([8], np.int32), np.array([3], np.int32))
    for t, sel, slots, miss in rows:
        got_slots, got_miss = c.step(t, np.array(sel, np.int32)[None, None])
        assert got_slots[0, 0].tolist() == slots, (t, got_slots)
        assert [(int(m[2]), int(m[3])) for m in got_miss] == miss, (t, got_miss)
        assert all(int(m[0]) == 0 and int(m[1]) == 0 for m in got_miss)
    blocks, last = c.export()
    assert [(s, int(blocks[s]), int(last[s])) for s in range(3)] == final


def pin_lru_bruteforce(O):
    """Random selection streams with locality vs the recency-list reference,
    plus the cache invariants."""
    rng = np.random.default_rng(101)
    for trial in range(6):
        B, Hkv = 2, 2
        nblk = rng.integers(6, 30, size=B).astype(np.int32)
        k = int(rng.integers(1, 6))
        cap = np.array([[int(rng.integers(k, k + 6)) for _ in range(Hkv)] for _ in range(B)], np.int32)
        c = O.lru(B, Hkv, nblk, cap)
        refs = [[ListLRU(int(cap[b, g])) for g in range(Hkv)] for b in range(B)]
        prev = [[None] * Hkv for _ in range(B)]
        cached = [[set() for _ in range(Hkv)] for _ in range(B)]
        for t in range(25):
            sel = np.full((B, Hkv, k), -1, np.int32)
            for b, g in itertools.product(range(B), range(Hkv)):
                m = min(k, int(nblk[b])) - (1 if rng.random() < 0.2 and k > 1 else 0)
                base = prev[b][g] if prev[b][g] is not None and rng.random() < 0.7 else []
                keep = [j for j in base if rng.random() < 0.6][:m]
                rest = [j for j in rng.permutation(int(nblk[b])).tolist() if j not in keep]
                chosen = sorted(keep + rest[: m - len(keep)])
                sel[b, g, :len(chosen)] = chosen
                prev[b][g] = chosen
            slots, miss = c.step(t, sel)
            by_unit = {}
            for mb, mg, j, s in miss.tolist():
                by_unit.setdefault((mb, mg), []).append((j, s))
            for b, g in itertools.product(range(B), range(Hkv)):
                chosen = [j for j in sel[b, g] if j >= 0]
                rslots, rmiss = refs[b][g].step(t, chosen)
                assert slots[b, g, :len(chosen)].tolist() == rslots, (trial, t, b, g)
                assert by_unit.get((b, g), []) == rmiss, (trial, t, b, g)
                # invariants
                assert len(set(rslots)) == len(rslots)
                assert len(rmiss) == len(set(chosen) - cached[b][g])
                cached[b][g] = set(j for j in refs[b][g].block if j >= 0)
                assert set(chosen) <= cached[b][g]


def pin_lru_repeated_step(O):
    """Two resolves with the same step number (e.g. a second pass in one
    decode step): blocks selected by the second call are never evicted by it,
    even when their last use ties with unselected blocks."""
    rng = np.random.default_rng(105)
    for trial in range(10):
        nblk, cap, k = 12, 4, 3
        c = O.lru(1, 1, np.array([nblk], np.int32), np.array([cap], np.int32))
        ref = ListLRU(cap)
        t = 0
        for call in range(12):
            t += int(rng.integers(0, 2))  # nondecreasing, often repeated
            chosen = sorted(rng.choice(nblk, size=k, replace=False).tolist())
            slots, miss = c.step(t, np.array(chosen, np.int32)[None, None])
            rslots, rmiss = ref.step(t, chosen)
            assert slots[0, 0].tolist() == rslots, (trial, call)
            assert [(int(m[2]), int(m[3])) for m in miss] == rmiss, (trial, call)


def pin_lru_capacity_error(O):
    c = O.lru(1, 1, np.array([10], np.int32), np.array([2], np.int32))
    try:
        c.step(0, np.array([[[1, 2, 3]]], np.int32))
    except OverflowError:
        return
    raise AssertionError("capacity error not raised")


# ---------------------------------------------------------------- O4 gather
def pin_gather_bytes(O):
    """Each reported miss copies exactly its source record into its slot;
    nothing else in the cache image changes."""
    rng = np.random.default_rng(111)
    B, Hkv, nblk, rb = 2, 3, 7, 64
    pool = rng.integers(0, 256, size=B * Hkv * nblk * rb, dtype=np.uint8)
    pool_off = np.arange(B * Hkv, dtype=np.int64) * nblk * rb
    cap = 4
    cache = rng.integers(0, 256, size=B * Hkv * cap * rb, dtype=np.uint8)
    before = cache.copy()
    cache_off = np.arange(B * Hkv, dtype=np.int64)[::-1].copy() * cap * rb
    miss = np.array([[0, 0, 3, 1], [1, 2, 6, 0], [1, 0, 0, 3], [0, 2, 5, 2]], np.int32)
    O.gather(miss, pool, pool_off, cache, cache_off, rb, Hkv)
    touched = np.zeros_like(cache, dtype=bool)
    for b, g, j, s in miss.tolist():
        u = b * Hkv + g
        dst = slice(cache_off[u] + s * rb, cache_off[u] + (s + 1) * rb)
        src = slice(pool_off[u] + j * rb, pool_off[u] + (j + 1) * rb)
        assert np.array_equal(cache[dst], pool[src]), (b, g, j, s)
        touched[dst] = True
    assert np.array_equal(cache[~touched], before[~touched])


# ------------------------------------------------------------- O5 attention
def _torch_attention(q, Ksel, Vsel, scale):
    """Library-routine reference in fp64: softmax(q K^T * scale) V."""
    qt = torch.from_numpy(q)
    p = torch.softmax(torch.from_numpy(Ksel) @ qt * scale, dim=0)
    return (p @ torch.from_numpy(Vsel)).numpy()


def pin_attention_fixture(O):
    fx = read_fixture("attention_two_tokens.txt")
    q = np.array([[[float(x) for x in fx["q"]]]])
    K = np.array([[float(x) for x in fx["k0"]], [float(x) for x in fx["k1"]]])
    V = np.array([[float(x) for x in fx["v0"]], [float(x) for x in fx["v1"]]])
    rec = make_records(f64_to_bits(K)[None], f64_to_bits(V)[None])
    out = O.attention(f64_to_bits(q), rec, np.zeros(1, np.int64), np.array([[[0]]], np.int32), 1, 2)
    ref = np.array([float(x) for x in fx["out"]])
    assert np.allclose(out[0, 0], ref, rtol=0, atol=1e-6), (out, ref)


def pin_attention_dense(O):
    """Selecting every block reproduces dense softmax attention (torch fp64)."""
    B, Hq, Hkv, nblk, blk, d = 2, 8, 2, 6, 4, 16
    K = rand_bf16((B, Hkv, nblk, blk, d), 121, 1.5)
    V = rand_bf16((B, Hkv, nblk, blk, d), 122)
    q = rand_bf16((B, Hq, d), 123)
    rec = make_records(K, V)
    slots = np.broadcast_to(np.arange(nblk, dtype=np.int32), (B, Hkv, nblk)).copy()
    out = O.attention(q, rec, dense_offsets(B * Hkv, nblk, blk, d), slots, Hkv, blk)
    G = Hq // Hkv
    qf, Kf, Vf = bits_to_f64(q), bits_to_f64(K), bits_to_f64(V)
    for b, h in itertools.product(range(B), range(Hq)):
        g = h // G
        ref = _torch_attention(qf[b, h], Kf[b, g].reshape(-1, d), Vf[b, g].reshape(-1, d), 1 / math.sqrt(d))
        assert np.allclose(out[b, h], ref, rtol=1e-6, atol=1e-6), (b, h)


def pin_attention_subset(O):
    """Attention over selected slots equals dense attention over just the
    tokens of those blocks; -1 entries are skipped; slot order is the
    order listed."""
    B, Hq, Hkv, nblk, blk, d = 1, 4, 2, 9, 3, 8
    K = rand_bf16((B, Hkv, nblk, blk, d), 131, 2.0)
    V = rand_bf16((B, Hkv, nblk, blk, d), 132)
    q = rand_bf16((B, Hq, d), 133)
    rec = make_records(K, V)
    slots = np.array([[[7, 1, 4, -1], [0, 8, -1, -1]]], np.int32)
    out = O.attention(q, rec, dense_offsets(B * Hkv, nblk, blk, d), slots, Hkv, blk)
    qf, Kf, Vf = bits_to_f64(q), bits_to_f64(K), bits_to_f64(V)
    for h in range(Hq):
        g = h // 2
        js = [j for j in slots[0, g] if j >= 0]
        ref = _torch_attention(qf[0, h], Kf[0, g, js].reshape(-1, d), Vf[0, g, js].reshape(-1, d), 1 / math.sqrt(d))
        assert np.allclose(out[0, h], ref, rtol=1e-6, atol=1e-6), h
        lo = Vf[0, g, js].reshape(-1, d).min(axis=0)
        hi = Vf[0, g, js].reshape(-1, d).max(axis=0)
        assert np.all(out[0, h] >= lo - 1e-6) and np.all(out[0, h] <= hi + 1e-6), "outside the convex hull of V"


def pin_attention_empty(O):
    """No selected token -> zero output."""
    q = rand_bf16((1, 2, 4), 141)
    rec = make_records(rand_bf16((1, 2, 2, 4), 142), rand_bf16((1, 2, 2, 4), 143))
    out = O.attention(q, rec, np.zeros(1, np.int64), np.full((1, 1, 2), -1, np.int32), 1, 2)
    assert np.all(out == 0)


# ------------------------------------------------------ O6 append, O7 save
def record_tokens(rec, blk, d):
    """Inverse of make_records for one record: uint16 [2*blk*d] -> (K [blk][d], V [blk][d])."""
    rec = np.asarray(rec, dtype=np.uint16)
    K = rec[:blk * d].reshape(blk, d)
    V = rec[blk * d:].reshape(d, blk).T
    return K, V


def _nonzero_bf16(shape, seed):
    x = rand_bf16(shape, seed)
    x[(x & 0x7FFF) == 0] = 0x3F80  # no signed zeros: numpy's min/max then agrees with totalOrder
    return x


def pin_append_record_layout(O):
    """blk appends starting on a block boundary leave the open record equal
    to the record assembled from the tokens (numpy layout), and the block's
    metadata equal to numpy's channel-wise min/max of its keys."""
    B, Hkv, blk, d, nmax = 2, 3, 4, 8, 3
    tok = _nonzero_bf16((blk, B, Hkv, 2, d), 11)
    len_ = np.array([0, 4], np.int32)
    nblk = np.array([0, 1], np.int32)
    open_rec = np.zeros((B, Hkv, 2 * blk * d), np.uint16)
    meta = np.zeros((B, Hkv, nmax, 2, d), np.uint16)
    for t in range(blk):
        if t < blk - 1:
            assert list(nblk) == [0, 1]
        O.append(tok[t], len_, nblk, blk, nmax, open_rec, meta)
    assert list(len_) == [blk, 2 * blk] and list(nblk) == [1, 2]
    for b in range(B):
        j = b  # block filled by these appends
        for g in range(Hkv):
            K = tok[:, b, g, 0]
            V = tok[:, b, g, 1]
            want = make_records(K[None], V[None])[0]
            assert np.array_equal(open_rec[b, g], want), (b, g)
            np.testing.assert_array_equal(meta[b, g, j], _meta_from_keys(bits_to_f64(K)))
            others = [x for x in range(nmax) if x != j]
            assert np.all(meta[b, g, others] == 0)


def pin_append_ragged_positions(O):
    """Sequences at different offsets: after each append, positions below the
    fill level of the open record hold the current block's tokens; blocks
    fill (nblk, metadata) exactly when their last token arrives."""
    B, Hkv, blk, d, nmax = 3, 2, 4, 8, 6
    start = np.array([1, 6, 11], np.int32)
    steps = 9
    tok = _nonzero_bf16((steps, B, Hkv, 2, d), 12)
    len_ = start.copy()
    nblk = (start // blk).astype(np.int32)
    open_rec = np.zeros((B, Hkv, 2 * blk * d), np.uint16)
    meta = np.zeros((B, Hkv, nmax, 2, d), np.uint16)
    hist = {b: {} for b in range(B)}  # token index -> step
    for t in range(steps):
        O.append(tok[t], len_, nblk, blk, nmax, open_rec, meta)
        for b in range(B):
            T = start[b] + t
            hist[b][T] = t
            assert len_[b] == T + 1 and nblk[b] == (T + 1) // blk
            j0 = T // blk * blk
            for g in range(Hkv):
                K, V = record_tokens(open_rec[b, g], blk, d)
                for T2 in range(max(j0, start[b]), T + 1):
                    assert np.array_equal(K[T2 - j0], tok[hist[b][T2], b, g, 0]), (t, b, g, T2)
                    assert np.array_equal(V[T2 - j0], tok[hist[b][T2], b, g, 1]), (t, b, g, T2)
                if (T + 1) % blk == 0:  # block T // blk just filled from tokens j0 .. T
                    if j0 >= start[b]:
                        Kb = np.stack([tok[hist[b][x], b, g, 0] for x in range(j0, T + 1)])
                        np.testing.assert_array_equal(meta[b, g, T // blk], _meta_from_keys(bits_to_f64(Kb)))
    # blocks that were already full before the first append are never written
    for b in range(B):
        for j in range(start[b] // blk):
            assert np.all(meta[b, :, j] == 0)


def pin_append_capacity_error(O):
    """Filling a block at index >= nblk_max is an error and changes nothing."""
    B, Hkv, blk, d, nmax = 1, 1, 4, 8, 2
    len_ = np.array([2 * blk - 1], np.int32)
    nblk = np.array([1], np.int32)
    open_rec = np.zeros((1, 1, 2 * blk * d), np.uint16)
    meta = np.zeros((1, 1, nmax, 2, d), np.uint16)
    O.append(_nonzero_bf16((1, 1, 2, d), 13), len_, nblk, blk, nmax, open_rec, meta)  # fills block 1: fine
    assert nblk[0] == 2 and len_[0] == 2 * blk
    len_[0] = 3 * blk - 1
    before = open_rec.copy()
    try:
        O.append(_nonzero_bf16((1, 1, 2, d), 14), len_, nblk, blk, nmax, open_rec, meta)
    except OverflowError:
        assert np.array_equal(open_rec, before) and len_[0] == 3 * blk - 1 and nblk[0] == 2
        return
    raise AssertionError("filling block nblk_max did not fail")


def pin_save_spans_blocks(O):
    """Saving several tokens per sequence that span block boundaries writes
    each token at its (block, position) and leaves every other byte of the
    pool as it was; units sit at arbitrary pool offsets."""
    B, Hkv, blk, d, n_new = 2, 2, 4, 8, 7
    rb = 2 * blk * d * 2
    nb = 4
    units = B * Hkv
    off = (np.arange(units, dtype=np.int64)[::-1] * (nb + 1) * rb).copy()  # reversed, with a gap record
    pool = np.frombuffer(np.random.default_rng(15).bytes((units * (nb + 1)) * rb), np.uint8).copy()
    before = pool.copy()
    len_ = np.array([3, 9], np.int32)
    tok = _nonzero_bf16((B, n_new, Hkv, 2, d), 16)
    O.save(tok, len_, blk, pool, off, np.full(B, nb, np.int32))
    touched = np.zeros(pool.size, bool)
    for b in range(B):
        for g in range(Hkv):
            u = b * Hkv + g
            for j in range(nb):
                lo = off[u] + j * rb
                rec = pool[lo:lo + rb].view(np.uint16)
                K, V = record_tokens(rec, blk, d)
                K0, V0 = record_tokens(before[lo:lo + rb].view(np.uint16), blk, d)
                for p in range(blk):
                    i = j * blk + p - len_[b]
                    if 0 <= i < n_new:
                        assert np.array_equal(K[p], tok[b, i, g, 0]) and np.array_equal(V[p], tok[b, i, g, 1]), \
                            (b, g, j, p)
                    else:
                        assert np.array_equal(K[p], K0[p]) and np.array_equal(V[p], V0[p]), (b, g, j, p)
                touched[lo:lo + rb] = True
    assert np.array_equal(pool[~touched], before[~touched])


def pin_save_full_block_record(O):
    """Saving exactly one block's tokens from a block boundary writes the
    record that numpy assembles from those tokens."""
    B, Hkv, blk, d = 1, 2, 8, 16
    rb = 2 * blk * d * 2
    pool = np.zeros(Hkv * 3 * rb, np.uint8)
    off = np.arange(Hkv, dtype=np.int64) * 3 * rb
    tok = _nonzero_bf16((B, blk, Hkv, 2, d), 17)
    O.save(tok, np.array([blk], np.int32), blk, pool, off, np.array([3], np.int32))
    for g in range(Hkv):
        rec = pool[off[g] + rb:off[g] + 2 * rb].view(np.uint16)
        assert np.array_equal(rec, make_records(tok[0, :, g, 0][None], tok[0, :, g, 1][None])[0]), g
        assert np.all(pool[off[g]:off[g] + rb] == 0) and np.all(pool[off[g] + 2 * rb:off[g] + 3 * rb] == 0)


def pin_save_capacity_error(O):
    """A token past the unit's pool blocks is an error and writes nothing."""
    blk, d = 4, 8
    rb = 2 * blk * d * 2
    pool = np.zeros(2 * rb, np.uint8)
    try:
        O.save(_nonzero_bf16((1, 3, 1, 2, d), 18), np.array([6], np.int32), blk, pool, np.zeros(1, np.int64),
               np.array([2], np.int32))
    except OverflowError:
        assert np.all(pool == 0)
        return
    raise AssertionError("saving past the pool did not fail")


# ------------------------------------------- O8-O10 working sets, Alg. 1
def pin_ws_fixture(O):
    """Hand-worked fixture (golden/working_set.txt): a 4-step history with
    w = 2, and the prefill working sets of both prefill strategies."""
    fx = read_fixture("working_set.txt")
    hist = np.array([[int(x) for x in fx[f"dec_sel{s}"]] for s in range(4)], np.int32).reshape(4, 1, 1, 3)
    want = [int(x) for x in fx["dec_bytes"]]
    got = [O.ws_decode(hist[:m + 1], 2, 8192) for m in range(4)]
    assert got == want, (got, want)
    assert O.ws_prefill(1000, 512, 256, 32, 8, 16, 8192, True) == int(fx["pre_seg"][0])
    assert O.ws_prefill(1000, 512, 256, 32, 8, 16, 8192, False) == int(fx["pre_chunk"][0])
    assert O.ws_prefill(1000, 768, 512, 32, 8, 16, 8192, False) == int(fx["pre_chunk_last"][0])


def pin_ws_bruteforce(O):
    """Random histories vs Python sets: per (layer, head) the union of the
    last w steps' non-negative entries."""
    rng = np.random.default_rng(31)
    for trial in range(20):
        m, layers, Hkv, k, w = int(rng.integers(1, 9)), int(rng.integers(1, 4)), int(rng.integers(1, 4)), \
            int(rng.integers(1, 6)), int(rng.integers(1, 6))
        hist = rng.integers(-1, 12, size=(m, layers, Hkv, k)).astype(np.int32)
        want = 0
        for l in range(layers):
            for g in range(Hkv):
                u = set()
                for s in range(max(0, m - w), m):
                    u |= {int(x) for x in hist[s, l, g] if x >= 0}
                want += len(u)
        assert O.ws_decode(hist, w, 4096) == want * 4096, trial


def pin_ws_closed_forms(O):
    """The same selection every step gives k blocks per (layer, head);
    disjoint selections give min(w, m) * k; no history uses the fallback."""
    layers, Hkv, k, rb = 2, 3, 4, 8192
    same = np.tile(np.arange(k, dtype=np.int32), (7, layers, Hkv, 1))
    assert O.ws_decode(same, 12, rb) == k * layers * Hkv * rb
    disj = (np.arange(7 * k, dtype=np.int32).reshape(7, 1, 1, k) + np.zeros((1, layers, Hkv, 1), np.int32))
    for w in (1, 3, 7, 12):
        assert O.ws_decode(disj, w, rb) == min(w, 7) * k * layers * Hkv * rb, w
    assert O.ws_decode(np.zeros((0, layers, Hkv, k), np.int32), 12, rb, fallback=5) == 5 * layers * Hkv * rb


def pin_schedule_fixture(O):
    """Hand-worked fixture (golden/schedule_alg1.txt)."""
    fx = read_fixture("schedule_alg1.txt")
    for case in "abc":
        admit, used = O.schedule([int(x) for x in fx[f"{case}_ws"]], int(fx[f"{case}_avl"][0]))
        assert admit.tolist() == [int(x) for x in fx[f"{case}_admit"]], case
        assert used == int(fx[f"{case}_used"][0]), case


def pin_schedule_invariants(O):
    """Random batches: the admitted requests fit M_avl; every reset request
    would not have fitted at its turn (greedy in the given order)."""
    rng = np.random.default_rng(32)
    for _ in range(50):
        ws = rng.integers(0, 100, size=int(rng.integers(0, 20)))
        avl = int(rng.integers(0, 600))
        admit, used = O.schedule(ws, avl)
        assert used == int(ws[admit == 1].sum()) <= avl
        run = 0
        for x, a in zip(ws, admit):
            if a:
                run += x
            else:
                assert run + x > avl


# ------------------------------------------- O11/O12 metadata and score variants
def _bf16_rne_from_f64(x):
    """Library routine: torch's float64 -> bfloat16 conversion (round to nearest even)."""
    return torch.tensor(np.asarray(x, np.float64)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def pin_meta_mean_exact_cases(O):
    """Inputs whose fp32 token sums are exact (small integers times 1/8):
    the mean key equals the exact mean rounded by torch's bf16 conversion;
    a block of identical tokens has exactly that token as its mean."""
    rng = np.random.default_rng(41)
    B, Hkv, nmax, d = 2, 2, 5, 16
    for blk in (1, 4, 16, 32):
        Kf = rng.integers(-40, 41, size=(B, Hkv, nmax, blk, d)) / 8.0
        Kf[1, 1, 2] = Kf[1, 1, 2, :1]  # identical tokens
        Kb = f64_to_bits(Kf)
        rec = make_records(Kb, rand_bf16(Kb.shape, 49 + blk))  # V differs from K
        off = dense_offsets(B * Hkv, nmax, blk, d)
        nblk = np.array([nmax, 3], np.int32)
        meta = O.build_metadata_mean(rec, off, nblk, B, Hkv, nmax, blk, d)
        want = _bf16_rne_from_f64(Kf.mean(axis=3))
        for b in range(B):
            np.testing.assert_array_equal(meta[b, :, :nblk[b]], want[b, :, :nblk[b]])
            assert np.all(meta[b, :, nblk[b]:] == 0)
        np.testing.assert_array_equal(meta[1, 1, 2], Kb[1, 1, 2, 0])


def _bf16_nearest_exact(x):
    """bf16 bits of the rational x rounded to the nearest bf16, ties to the
    even significand, in exact rational arithmetic (fractions): 8
    significant bits above 2^-126, a fixed quantum of 2^-133 below."""
    from fractions import Fraction
    x = Fraction(x)
    if x == 0:
        return 0
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()  # floor(log2 a) is e or e - 1
    if Fraction(2) ** e > a:
        e -= 1
    q = Fraction(2) ** max(e - 7, -133)
    r = round(a / q) * q  # Fraction rounding: half to even
    bits = int(np.array(float(r), np.float32).view(np.uint32)) >> 16
    return bits | (0x8000 if x < 0 else 0)


def pin_meta_mean_rounding(O):
    """Random keys: every mean key equals the exact mean (a rational sum of
    the bf16 keys over blk) rounded once to the nearest bf16, computed here
    in exact rational arithmetic; no entry may differ."""
    from fractions import Fraction
    B, Hkv, nmax, blk, d = 1, 2, 16, 16, 128
    Kb = rand_bf16((B, Hkv, nmax, blk, d), 42)
    Kb[0, 1, 3] = rand_bf16((blk, d), 43, scale=1e-4)  # small keys: other exponents
    rec = make_records(Kb, rand_bf16((B, Hkv, nmax, blk, d), 50))
    meta = O.build_metadata_mean(rec, dense_offsets(B * Hkv, nmax, blk, d), np.array([nmax], np.int32), B, Hkv,
                                 nmax, blk, d)
    Kf = bits_to_f64(Kb)
    for g in range(Hkv):
        for j in range(nmax):
            for c in range(d):
                exact = sum((Fraction(float(v)) for v in Kf[0, g, j, :, c]), Fraction(0)) / blk
                assert int(meta[0, g, j, c]) == _bf16_nearest_exact(exact), (g, j, c)


def pin_meta_mean_fixture(O):
    """Hand-worked fixture (golden/mean_key_rounding.txt): a mean just above
    a rounding midpoint (where rounding through fp32 first would tie the
    other way), exact midpoints tying to even both ways, and a negative
    mean."""
    fx = read_fixture("mean_key_rounding.txt")
    blk = int(fx["blk"][0])
    rows = [[float(x) for x in fx["token_0_to_29"]]] * 30 + [[float(x) for x in fx["token_30"]],
                                                              [float(x) for x in fx["token_31"]]]
    assert len(rows) == blk
    Kb = f64_to_bits(np.array(rows))[None, None, None]  # [1][1][1][blk][d]
    assert np.array_equal(bits_to_f64(Kb)[0, 0, 0], np.array(rows))  # every input is a bf16 value
    d = Kb.shape[-1]
    meta = O.build_metadata_mean(make_records(Kb, Kb), np.zeros(1, np.int64), np.array([1], np.int32), 1, 1, 1, blk,
                                 d)
    np.testing.assert_array_equal(bits_to_f64(meta[0, 0, 0]), [float(x) for x in fx["mean_key"]])


def pin_meta_mean_refuses_inexact(O):
    """Keys whose magnitudes are too far apart for an exact fp64 sum (2^100
    and 2^-100) are refused instead of given a rounded mean."""
    Kf = np.zeros((1, 1, 1, 2, 2))
    Kf[0, 0, 0, :, 0] = [2.0 ** 100, 2.0 ** -100]
    Kb = f64_to_bits(Kf)
    try:
        O.build_metadata_mean(make_records(Kb, Kb), np.zeros(1, np.int64), np.array([1], np.int32), 1, 1, 1, 2, 2)
    except RuntimeError:
        return
    raise AssertionError("an inexact fp64 sum was accepted")


def pin_score_variant_fixture(O):
    """Hand-worked fixture (golden/score_box.txt): both kinds, both
    aggregations, and the mean-key metadata of the two tokens."""
    fx = read_fixture("score_box.txt")
    K = np.array([[float(x) for x in fx["key_t0"]], [float(x) for x in fx["key_t1"]]])
    q = f64_to_bits(np.array([[float(x) for x in fx["q_h0"]], [float(x) for x in fx["q_h1"]]]))[None]
    cub = _meta_from_keys(K)[None, None, None]
    Kb = f64_to_bits(K)[None, None, None]
    mean = O.build_metadata_mean(make_records(Kb, Kb), np.zeros(1, np.int64), np.array([1], np.int32), 1, 1, 1, 2, 4)
    np.testing.assert_array_equal(bits_to_f64(mean[0, 0, 0]), [float(x) for x in fx["mean_key"]])
    one = np.array([1], np.int32)
    for meta, kind, agg, key in ((cub, 0, 0, "score"), (cub, 0, 1, "cuboid_sum"), (mean, 1, 0, "mean_max"),
                                 (mean, 1, 1, "mean_sum")):
        S = O.score_variant(q, meta, kind, agg, one, 2, 1, 1, 4)
        assert S[0, 0, 0] == float(fx[key][0]), (key, S)


def pin_score_mean_is_mean_of_dots(O):
    """With exact mean keys the mean-key score is the average of the token
    scores q.k_t (linearity), computed here with numpy's matmul."""
    rng = np.random.default_rng(43)
    Hq, Hkv, nmax, blk, d = 4, 2, 6, 8, 32
    Kf = rng.integers(-16, 17, size=(1, Hkv, nmax, blk, d)) / 4.0
    qf = rng.integers(-8, 9, size=(1, Hq, d)) / 4.0
    meta = f64_to_bits(Kf.mean(axis=3))  # exact: sums of quarters over 8 tokens
    S = O.score_variant(f64_to_bits(qf), meta, 1, 0, np.array([nmax], np.int32), Hq, Hkv, nmax, d)
    G = Hq // Hkv
    for g in range(Hkv):
        dots = np.einsum("hc,jtc->hjt", qf[0, g * G:(g + 1) * G], Kf[0, g])  # [G][nblk][blk]
        np.testing.assert_allclose(S[0, g], dots.mean(axis=2).max(axis=0), rtol=0, atol=1e-12)


def pin_score_aggregations_reduce_to_heads(O):
    """max and sum over the group equal numpy's max and sum of the per-head
    scores obtained with groups of one head (G = 1), for both kinds."""
    rng = np.random.default_rng(44)
    Hq, Hkv, nmax, d = 6, 2, 9, 16
    G = Hq // Hkv
    q = rand_bf16((2, Hq, d), 45)
    nblk = np.array([nmax, 4], np.int32)
    for kind in (0, 1):
        if kind == 0:
            a, b2 = rand_bf16((2, Hkv, nmax, d), 46), rand_bf16((2, Hkv, nmax, d), 47)
            lo = np.where(bits_to_f64(a) <= bits_to_f64(b2), a, b2)
            hi = np.where(bits_to_f64(a) <= bits_to_f64(b2), b2, a)
            meta = np.stack([lo, hi], axis=3)
        else:
            meta = rand_bf16((2, Hkv, nmax, d), 48)
        per_head_meta = np.repeat(meta, G, axis=1)  # head h uses its group's metadata
        per = O.score_variant(q, per_head_meta, kind, 0, nblk, Hq, Hq, nmax, d)  # [2][Hq][nmax]
        for agg, fn in ((0, np.max), (1, np.sum)):
            S = O.score_variant(q, meta, kind, agg, nblk, Hq, Hkv, nmax, d)
            for b in range(2):
                n = nblk[b]
                want = fn(per[b, :, :n].reshape(Hkv, G, n), axis=1)
                np.testing.assert_allclose(S[b, :, :n], want, rtol=1e-13, atol=1e-12)
                assert np.all(np.isneginf(S[b, :, n:]))


# ----------------------------------------------- O13 layer-segmented prefill
def pin_prefill_plan_fixture(O):
    """Hand-worked fixture (golden/prefill_plan.txt)."""
    fx = read_fixture("prefill_plan.txt")
    for case, (T, layers, M) in {"a": (1000, 5, 2500), "b": (1000, 2, 400), "c": (3, 4, 3)}.items():
        want = [[int(x) for x in fx[k]] for k in sorted((k for k in fx if k.startswith(case + "_item")),
                                                       key=lambda k: int(k.split("item")[1]))]
        assert O.prefill_plan(T, layers, M).tolist() == want, case


def pin_prefill_plan_invariants(O):
    """Every (layer, token) is covered exactly once, layers run in order, a
    batch injects at most maxInjectToken tokens, and batches are as full as
    the rule allows: whole layers when the prompt fits, else chunks."""
    rng = np.random.default_rng(51)
    for _ in range(60):
        T, layers, M = int(rng.integers(1, 3000)), int(rng.integers(1, 9)), int(rng.integers(1, 5000))
        it = O.prefill_plan(T, layers, M)
        cover = np.zeros((layers, T), np.int32)
        for b, l, t0, t1 in it:
            cover[l, t0:t1] += 1
        assert np.all(cover == 1), (T, layers, M)
        assert np.all(np.diff(it[:, 1]) >= 0) and np.all(np.diff(it[:, 0]) >= 0)
        per_batch = np.bincount(it[:, 0], weights=it[:, 3] - it[:, 2])
        assert per_batch.max() <= M
        n_batches = it[-1, 0] + 1
        if T <= M:
            assert n_batches == -(-layers // (M // T))
        else:
            assert n_batches == layers * -(-T // M)


GROUPS = {
    "meta": [pin_meta_bruteforce, pin_meta_ragged_untouched, pin_meta_signed_zero, pin_meta_record_offsets],
    "score": [pin_score_fixture, pin_score_upper_bound, pin_score_point_block, pin_score_corner_tight,
              pin_score_ragged],
    "select": [pin_select_fixture, pin_select_bruteforce, pin_select_all_when_k_large],
    "lru": [pin_lru_fixture, pin_lru_bruteforce, pin_lru_repeated_step, pin_lru_capacity_error],
    "gather": [pin_gather_bytes],
    "attention": [pin_attention_fixture, pin_attention_dense, pin_attention_subset, pin_attention_empty],
    "append": [pin_append_record_layout, pin_append_ragged_positions, pin_append_capacity_error],
    "save": [pin_save_spans_blocks, pin_save_full_block_record, pin_save_capacity_error],
    "ws": [pin_ws_fixture, pin_ws_bruteforce, pin_ws_closed_forms],
    "meta_mean": [pin_meta_mean_exact_cases, pin_meta_mean_rounding, pin_meta_mean_fixture,
                  pin_meta_mean_refuses_inexact],
    "prefill_plan": [pin_prefill_plan_fixture, pin_prefill_plan_invariants],
    "score_variant": [pin_score_variant_fixture, pin_score_mean_is_mean_of_dots, pin_score_aggregations_reduce_to_heads],
    "schedule": [pin_schedule_fixture, pin_schedule_invariants],
}
ALL_PINS = [p for ps in GROUPS.values() for p in ps]

"""The library's working-set tracker and batch control (ss_ws_*,
ss_schedule_batch, ss_ws_prefill_bytes; Section 3.3) against the oracle:
requests that join and leave, several layers, windows of 1 to 16 steps,
padded selections, growing block indices, fallbacks for layers without
history.  Host-only, runs on the CPU."""
import numpy as np
import pytest

import synth
from paper_2509_24626_amd import binding as ss


class Tracker:
    def __init__(self, layers, Hkv, w, rb=8192):
        self.h = ss.ss_ws_create(layers, Hkv, w, rb)

    def __del__(self):
        ss.ss_ws_destroy(self.h)


def random_sel(rng, B, Hkv, k, hi, pad_frac=0.1):
    """Ascending selections with -1 padding, as top-k emits them."""
    out = np.full((B, Hkv, k), -1, np.int32)
    for b in range(B):
        for g in range(Hkv):
            m = k - int(rng.random() < pad_frac) * int(rng.integers(1, k + 1))
            pick = np.sort(rng.choice(hi, size=min(m, hi), replace=False))
            out[b, g, :len(pick)] = pick
    return out


@pytest.mark.parametrize("w", [1, 3, 12, 16])
def test_requests_joining_and_leaving(oracle_impl, w):
    rng = np.random.default_rng(w)
    layers, Hkv, k, rb = 3, 2, 5, 8192
    T = Tracker(layers, Hkv, w, rb)
    hist = {}  # request id -> list of [layers][Hkv][k]
    live = [10, 11, 12]
    next_id = 13
    for step in range(30):
        if step % 7 == 3:  # one request finishes, another joins
            gone = live.pop(int(rng.integers(0, len(live))))
            ss.ss_ws_forget(T.h, gone)
            hist.pop(gone, None)
            live.append(next_id)
            next_id += 1
        B = len(live)
        hi = 20 + step  # sequences grow: newer, larger block indices appear
        sels = np.stack([random_sel(rng, B, Hkv, k, hi) for _ in range(layers)])  # [layers][B][Hkv][k]
        order = rng.permutation(B)  # batch order differs from id order
        for l in range(layers):
            ss.ss_ws_observe(T.h, l, step, np.array(live)[order], sels[l][order])
        for i, r in enumerate(live):
            hist.setdefault(r, []).append(sels[:, i])
        got = ss.ss_ws_decode_bytes(T.h, live)
        for i, r in enumerate(live):
            want = oracle_impl.ws_decode(np.stack(hist[r]), w, rb)
            assert got[i] == want, (step, r)


def test_config_shaped_selection_stream(oracle_impl):
    """Selection streams with the locality of a drifting decode (synth),
    64 sequences x 8 heads x 128 blocks, window 12, 20 steps."""
    nblk = np.full(64, 8192, np.int32)
    B, Hkv, k, w, steps = 64, 8, 128, 12, 20
    stream = synth.gen.selection_stream(nblk, Hkv, k, steps, 0.25, seed=5)
    T = Tracker(1, Hkv, w)
    ids = np.arange(1000, 1000 + B, dtype=np.int64)
    for s in range(steps):
        ss.ss_ws_observe(T.h, 0, s, ids, stream[s])
    got = ss.ss_ws_decode_bytes(T.h, ids)
    hist = np.stack(stream)[:, None]  # [steps][layers=1][B][Hkv][k] -> per request below
    for b in range(0, B, 7):
        want = oracle_impl.ws_decode(hist[:, :, b], w, 8192)
        assert got[b] == want, b
    # the union of 12 steps of a slowly drifting selection is well below 12 * k
    assert 128 * 8192 * Hkv < got.mean() < 12 * 128 * 8192 * Hkv


def test_fallback_for_missing_history(oracle_impl):
    layers, Hkv, k, rb = 4, 2, 3, 4096
    T = Tracker(layers, Hkv, 5, rb)
    fb = np.array([7, 2], np.int32)
    got = ss.ss_ws_decode_bytes(T.h, [1, 2], fb)  # unknown requests
    assert got.tolist() == [oracle_impl.ws_decode(np.zeros((0, layers, Hkv, k), np.int32), 5, rb, fallback=7),
                            oracle_impl.ws_decode(np.zeros((0, layers, Hkv, k), np.int32), 5, rb, fallback=2)]
    # request 1 observed in layers 0 and 2 only: the other layers count the fallback
    rng = np.random.default_rng(3)
    s0, s2 = random_sel(rng, 1, Hkv, k, 10), random_sel(rng, 1, Hkv, k, 10)
    ss.ss_ws_observe(T.h, 0, 0, [1], s0)
    ss.ss_ws_observe(T.h, 2, 0, [1], s2)
    got = ss.ss_ws_decode_bytes(T.h, [1], fb[:1])
    want = oracle_impl.ws_decode(s0[None, :1], 5, rb) + oracle_impl.ws_decode(s2[None, :1], 5, rb) + \
        2 * Hkv * 7 * rb
    assert got[0] == want


def test_observe_errors_leave_state_unchanged(oracle_impl):
    T = Tracker(2, 1, 4, 8192)
    sel = np.array([[[1, 2]]], np.int32)
    ss.ss_ws_observe(T.h, 0, 5, [9], sel)
    before = ss.ss_ws_decode_bytes(T.h, [9]).tolist()
    for bad in [dict(layer=0, step=5, ids=[9], sel=sel),                      # step not increasing
                dict(layer=2, step=6, ids=[9], sel=sel),                      # no such layer
                dict(layer=0, step=6, ids=[9, 9], sel=np.concatenate([sel, sel])),  # id twice
                dict(layer=0, step=6, ids=[9], sel=np.array([[[1, 2, 3]]], np.int32)),  # k changed
                dict(layer=0, step=6, ids=[9], sel=np.array([[[1, 1 << 24]]], np.int32))]:  # index too large
        with pytest.raises(ss.SparseServeError):
            ss.ss_ws_observe(T.h, bad["layer"], bad["step"], bad["ids"], bad["sel"])
        assert ss.ss_ws_decode_bytes(T.h, [9]).tolist() == before
    with pytest.raises(ss.SparseServeError):
        ss.ss_ws_create(1, 1, 0, 8192)
    with pytest.raises(ss.SparseServeError):
        ss.ss_ws_create(1, 1, 256, 8192)


def test_schedule_matches_oracle(oracle_impl):
    rng = np.random.default_rng(4)
    for _ in range(200):
        n = int(rng.integers(0, 40))
        ws = rng.integers(0, 1 << 30, size=n) * int(rng.integers(1, 64))
        avl = int(rng.integers(-5, 1 << 34))
        a_lib, u_lib = ss.ss_schedule_batch(ws, avl)
        a_o, u_o = oracle_impl.schedule(ws, avl)
        assert a_lib.tolist() == a_o.tolist() and u_lib == u_o
    with pytest.raises(ss.SparseServeError):
        ss.ss_schedule_batch([1, -1], 10)


def test_prefill_bytes_match_oracle(oracle_impl):
    for prompt in (0, 1, 15, 16, 17, 1000, 131072):
        for done in (0, 7, 512, 131072):
            for chunk in (0, 1, 256, 4096):
                for seg in (False, True):
                    for blk in (8, 16, 32):
                        args = (prompt, done, chunk, 32, 8, blk, 2 * blk * 128 * 2, seg)
                        assert ss.ss_ws_prefill_bytes(*args) == oracle_impl.ws_prefill(*args), args
    with pytest.raises(ss.SparseServeError):
        ss.ss_ws_prefill_bytes(-1, 0, 0, 32, 8, 16, 8192, True)


def test_prefill_plan_matches_oracle(oracle_impl):
    rng = np.random.default_rng(52)
    for _ in range(100):
        T, layers, M = int(rng.integers(1, 200000)), int(rng.integers(1, 40)), int(rng.integers(1, 300000))
        np.testing.assert_array_equal(ss.ss_prefill_plan(T, layers, M), oracle_impl.prefill_plan(T, layers, M))
    with pytest.raises(ss.SparseServeError):
        ss.ss_prefill_plan(0, 2, 10)

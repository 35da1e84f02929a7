"""GPU parity, all KV resident in HBM: metadata, block scores, top-k
selection and sparse attention against the CPU oracle, through the C ABI.

Cases span several tiles with ragged tails, sequences shorter than k, an
empty sequence, GQA groups of 1, 4, 7 and 16, blocks of 8, 16 and 32
tokens, k equal to and above the block count (dense attention), exact score
ties, and the tiny and Llama-3-8B-shaped workloads at their full sizes.
"""
import math
import zlib

import numpy as np
import pytest
import torch

import gpu_util as gu
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ss():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2509_24626_amd import binding
    binding.lib()
    return binding


CASES = {
    # name: B, Hq, Hkv, blk, nblk_max, k, n_plant, nblk
    "tiny-b2-h8kv2-ctx4k": (2, 8, 2, 16, 256, 16, 8, None),
    "ragged-short-empty": (3, 8, 2, 16, 40, 16, 0, [40, 7, 0]),
    "gqa7-blk8-ragged": (2, 28, 4, 8, 300, 24, 0, [300, 123]),
    "gqa1-blk32": (2, 4, 4, 32, 64, 8, 0, None),
    "gqa16-blk16": (1, 32, 2, 16, 100, 10, 0, None),
    "k-equals-blocks": (2, 8, 2, 16, 20, 20, 0, None),
    "k-above-blocks": (2, 8, 2, 16, 20, 32, 0, [20, 13]),
}



def _random_cases(n, seed):
    """Seeded extra shapes: heads and group size (1 to 16), block size,
    nblk_max, k (1 to 200, often above some sequences' block counts) and
    ragged block counts, empty sequences included."""
    rng = np.random.default_rng(seed)
    out = {}
    for i in range(n):
        Hkv = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.choice([1, 2, 4, 7, 16]))
        blk = int(rng.choice([8, 16, 32]))
        nmax = int(rng.integers(1, 700))
        k = int(rng.choice([1, 5, 16, 64, 200]))
        B = int(rng.integers(1, 6))
        nblk = [int(x) for x in rng.integers(0, nmax + 1, size=B)]
        out[f"random-{seed}-{i}"] = (B, Hkv * G, Hkv, blk, nmax, k, 0, nblk)
    return out


CASES.update(_random_cases(8, 17))

_cache = {}


def workload(name):
    if name not in _cache:
        B, Hq, Hkv, blk, nmax, k, npl, nblk = CASES[name]
        print(f"[gpu] workload {name}: B={B} Hq={Hq} Hkv={Hkv} blk={blk} nblk_max={nmax} k={k}", flush=True)
        _cache[name] = gu.HbmWorkload(B, Hq, Hkv, blk, nmax, k, seed=zlib.crc32(name.encode()) % 1000, n_plant=npl, nblk=nblk)
    return _cache[name]


def oracle_meta(oracle_impl, w):
    return oracle_impl.build_metadata(w.kv_host, w.unit_off_host, w.nblk_host, w.B, w.Hkv, w.nblk_max, w.blk, w.d)


def valid_rows_equal(a, b, nblk):
    for bb in range(a.shape[0]):
        n = int(nblk[bb])
        np.testing.assert_array_equal(a[bb, :, :n], b[bb, :, :n])


@pytest.mark.parametrize("name", list(CASES))
def test_metadata_bitexact(ss, oracle_impl, name):
    w = workload(name)
    meta = gu.run_metadata(ss, w)
    torch.cuda.synchronize()
    valid_rows_equal(gu.u16(meta), oracle_meta(oracle_impl, w), w.nblk_host)


@pytest.mark.parametrize("name", list(CASES))
def test_scores_and_selection(ss, oracle_impl, name):
    w = workload(name)
    meta = gu.run_metadata(ss, w)
    scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
    sel = torch.empty(w.B, w.Hkv, w.k, dtype=torch.int32, device="cuda")
    ss.ss_score_topk(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, w.k, scores, sel)
    torch.cuda.synchronize()
    om = oracle_meta(oracle_impl, w)
    S = oracle_impl.score(w.q_host, om, w.nblk_host, w.Hq, w.Hkv, w.nblk_max, w.d)
    osel = oracle_impl.select(S, w.nblk_host, w.k)
    worst = gu.check_scores(scores.cpu().numpy(), S, w.q_host, om, w.nblk_host, w.Hq // w.Hkv)
    diff = gu.check_selection(sel.cpu().numpy(), osel, S, w.nblk_host, w.k)
    print(f"[gpu] {name}: worst relative score error {worst:.2e}; units with tie-band differences {len(diff)}")


@pytest.mark.parametrize("name", list(CASES))
def test_metadata_mean_bitexact(ss, oracle_impl, name):
    """Mean-key metadata: the exact mean of each block's keys rounded once to bf16, bit-exact."""
    w = workload(name)
    meta = torch.empty(w.B, w.Hkv, w.nblk_max, w.d, dtype=torch.int16, device="cuda")
    ss.ss_build_metadata_mean(w.kv, w.unit_off, w.nblk, w.B, w.Hkv, w.nblk_max, w.blk, w.d, meta)
    torch.cuda.synchronize()
    om = oracle_impl.build_metadata_mean(w.kv_host, w.unit_off_host, w.nblk_host, w.B, w.Hkv, w.nblk_max, w.blk, w.d)
    valid_rows_equal(gu.u16(meta), om, w.nblk_host)


def test_metadata_mean_rounds_once(ss):
    """The hand-worked mean-key fixture (golden/mean_key_rounding.txt) on the
    GPU, through ss_build_metadata_mean and through the fill path of
    ss_append_kv: a mean 2^-25 above a rounding midpoint (which a rounding
    through fp32 would tie the other way), exact midpoints tying to even
    both ways, and a negative mean.  The fixture's 4 channels repeat over
    the 128."""
    import pins
    fx = pins.read_fixture("mean_key_rounding.txt")
    blk, d = int(fx["blk"][0]), 128
    rows = [[float(x) for x in fx["token_0_to_29"]]] * 30 + [[float(x) for x in fx["token_30"]],
                                                              [float(x) for x in fx["token_31"]]]
    K = torch.tensor(np.tile(np.array(rows), (1, d // 4)), dtype=torch.float32).to(torch.bfloat16)  # [blk][d]
    assert torch.equal(K.float(), torch.tensor(np.tile(np.array(rows), (1, d // 4)), dtype=torch.float32))
    want = np.tile(np.array([float(x) for x in fx["mean_key"]]), d // 4)
    rec = torch.zeros(2 * blk * d, dtype=torch.bfloat16)
    rec[:blk * d] = K.reshape(-1)
    rec = rec.cuda()
    one = torch.ones(1, dtype=torch.int32, device="cuda")
    meta = torch.zeros(1, 1, 1, d, dtype=torch.int16, device="cuda")
    ss.ss_build_metadata_mean(rec, torch.zeros(1, dtype=torch.int64, device="cuda"), one, 1, 1, 1, blk, d, meta)
    got = meta.view(torch.bfloat16).float().cpu().numpy().reshape(-1)
    np.testing.assert_array_equal(got, want)
    # the same block filled token by token: its metadata row is written by the append of token 31
    length = torch.zeros(1, dtype=torch.int32, device="cuda")
    nblk = torch.zeros(1, dtype=torch.int32, device="cuda")
    open_rec = torch.zeros(1, 1, 2 * blk * d, dtype=torch.int16, device="cuda")
    meta2 = torch.zeros(1, 1, 1, d, dtype=torch.int16, device="cuda")
    for t in range(blk):
        kv = torch.zeros(1, 1, 2, d, dtype=torch.bfloat16)
        kv[0, 0, 0] = K[t]
        ss.ss_append_kv(kv.cuda(), length, nblk, 1, 1, blk, d, 1, open_rec, meta2, None, meta_kind=ss.SS_META_MEAN)
    torch.cuda.synchronize()
    assert int(nblk.item()) == 1 and int(length.item()) == blk
    got2 = meta2.view(torch.bfloat16).float().cpu().numpy().reshape(-1)
    np.testing.assert_array_equal(got2, want)


@pytest.mark.parametrize("kind,agg", [(0, 1), (1, 0), (1, 1)], ids=["cuboid-sum", "mean-max", "mean-sum"])
@pytest.mark.parametrize("name", list(CASES))
def test_score_variants_and_selection(ss, oracle_impl, name, kind, agg):
    w = workload(name)
    if kind == 0:
        meta = gu.run_metadata(ss, w)
        om = oracle_meta(oracle_impl, w)
    else:
        meta = torch.empty(w.B, w.Hkv, w.nblk_max, w.d, dtype=torch.int16, device="cuda")
        ss.ss_build_metadata_mean(w.kv, w.unit_off, w.nblk, w.B, w.Hkv, w.nblk_max, w.blk, w.d, meta)
        om = oracle_impl.build_metadata_mean(w.kv_host, w.unit_off_host, w.nblk_host, w.B, w.Hkv, w.nblk_max, w.blk,
                                             w.d)
    scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
    sel = torch.empty(w.B, w.Hkv, w.k, dtype=torch.int32, device="cuda")
    ss.ss_score_blocks_variant(w.q, meta, kind, agg, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, scores)
    ss.ss_select_topk(scores, w.nblk, w.B, w.Hkv, w.nblk_max, w.k, sel)
    torch.cuda.synchronize()
    S = oracle_impl.score_variant(w.q_host, om, kind, agg, w.nblk_host, w.Hq, w.Hkv, w.nblk_max, w.d)
    osel = oracle_impl.select(S, w.nblk_host, w.k)
    worst = gu.check_scores_variant(scores.cpu().numpy(), S, w.q_host, om, w.nblk_host, w.Hq // w.Hkv, kind, agg)
    diff = gu.check_selection(sel.cpu().numpy(), osel, S, w.nblk_host, w.k)
    print(f"[gpu] {name} kind={kind} agg={agg}: worst relative score error {worst:.2e}; tie-band units {len(diff)}")


def test_score_variant_rejects_unknown_kind(ss):
    w = workload("tiny-b2-h8kv2-ctx4k")
    scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
    for kind, agg in ((2, 0), (0, 2), (-1, 0)):
        with pytest.raises(ss.SparseServeError):
            ss.ss_score_blocks_variant(w.q, scores, kind, agg, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, scores)


@pytest.mark.parametrize("name", list(CASES))
def test_attention_on_oracle_selection(ss, oracle_impl, name):
    w = workload(name)
    om = oracle_meta(oracle_impl, w)
    S = oracle_impl.score(w.q_host, om, w.nblk_host, w.Hq, w.Hkv, w.nblk_max, w.d)
    osel = oracle_impl.select(S, w.nblk_host, w.k)
    out = gu.run_attention(ss, w, torch.from_numpy(osel).cuda())
    torch.cuda.synchronize()
    ref = oracle_impl.attention(w.q_host, w.kv_host, w.unit_off_host, osel, w.Hkv, w.blk)
    err = np.abs(out.cpu().numpy() - ref).max()
    print(f"[gpu] {name}: attention max abs error {err:.2e}")
    assert err <= gu.ATTN_TOL


@pytest.mark.parametrize("name", ["tiny-b2-h8kv2-ctx4k", "gqa7-blk8-ragged", "ragged-short-empty"])
def test_end_to_end_step(ss, oracle_impl, name):
    """GPU selection feeds GPU attention; units whose selection equals the
    oracle's must match the oracle's attention."""
    w = workload(name)
    meta = gu.run_metadata(ss, w)
    scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
    sel = torch.empty(w.B, w.Hkv, w.k, dtype=torch.int32, device="cuda")
    ss.ss_score_topk(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, w.k, scores, sel)
    out = gu.run_attention(ss, w, sel).cpu().numpy()
    om = oracle_meta(oracle_impl, w)
    S = oracle_impl.score(w.q_host, om, w.nblk_host, w.Hq, w.Hkv, w.nblk_max, w.d)
    osel = oracle_impl.select(S, w.nblk_host, w.k)
    ref = oracle_impl.attention(w.q_host, w.kv_host, w.unit_off_host, osel, w.Hkv, w.blk)
    gsel = sel.cpu().numpy()
    G = w.Hq // w.Hkv
    compared = 0
    for b in range(w.B):
        for g in range(w.Hkv):
            if np.array_equal(gsel[b, g], osel[b, g]):
                compared += 1
                assert np.abs(out[b, g * G:(g + 1) * G] - ref[b, g * G:(g + 1) * G]).max() <= gu.ATTN_TOL
    assert compared >= w.units - 1


def test_planted_blocks_are_selected(ss):
    """Sanity (not parity): on the tiny workload every planted block is
    among the selected blocks of its KV head."""
    B, Hq, Hkv, blk, nmax, k, npl, _ = CASES["tiny-b2-h8kv2-ctx4k"]
    seed = zlib.crc32(b"tiny-b2-h8kv2-ctx4k") % 1000
    w = workload("tiny-b2-h8kv2-ctx4k")
    meta = gu.run_metadata(ss, w)
    scores = torch.empty(B, Hkv, nmax, dtype=torch.float32, device="cuda")
    sel = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
    ss.ss_score_topk(w.q, meta, w.nblk, B, Hq, Hkv, nmax, 128, k, scores, sel)
    gsel = sel.cpu().numpy()
    for b in range(B):
        for g in range(Hkv):
            planted = synth.gen.planted_blocks(nmax, npl, seed, 0, b, g, "cuda").cpu().numpy()
            assert set(planted.tolist()) <= set(gsel[b, g].tolist())


def test_scores_at_the_largest_block_count(ss, oracle_impl):
    """Scoring and selection at 65536 blocks per unit (the largest supported)
    with a ragged second sequence: each wave's staged tiles past a
    sequence's end read zeros through the buffer bounds and nothing is
    written past the end; scores and selection match the oracle."""
    rng = np.random.default_rng(21)
    B, Hq, Hkv, nmax, k = 2, 8, 2, 65536, 128
    nblk = np.array([65536, 40001], np.int32)
    a = torch.from_numpy(rng.standard_normal((B, Hkv, nmax, 128)).astype(np.float32))
    c = torch.from_numpy(rng.standard_normal((B, Hkv, nmax, 128)).astype(np.float32))
    meta = torch.stack([torch.minimum(a, c), torch.maximum(a, c)], 3).bfloat16().cuda().contiguous()
    del a, c
    q = torch.from_numpy(rng.standard_normal((B, Hq, 128)).astype(np.float32)).bfloat16().cuda()
    scores = torch.full((B, Hkv, nmax), 7.0, dtype=torch.float32, device="cuda")
    sel = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
    ss.ss_score_topk(q, meta, torch.from_numpy(nblk).cuda(), B, Hq, Hkv, nmax, 128, k, scores, sel)
    torch.cuda.synchronize()
    q_host = gu.u16(q)
    meta_host = gu.u16(meta)
    S = oracle_impl.score(q_host, meta_host, nblk, Hq, Hkv, nmax, 128)
    got = scores.cpu().numpy()
    assert np.all(got[1, :, 40001:] == 7.0), "scores written past the sequence's end"
    gu.check_scores(got, S, q_host, meta_host, nblk, Hq // Hkv)
    gu.check_selection(sel.cpu().numpy(), oracle_impl.select(S, nblk, k), S, nblk, k)


def test_topk_exact_ties(ss, oracle_impl):
    """Scores drawn from a handful of values (massive exact ties, +0 and -0,
    negatives): the GPU selection must equal the oracle's bit for bit."""
    rng = np.random.default_rng(5)
    for B, Hkv, nmax, k, nblk in [(2, 3, 1000, 37, [1000, 999]), (1, 2, 5000, 512, [5000]),
                                  (2, 2, 300, 300, [300, 17]), (1, 1, 16384, 512, [16384]),
                                  (3, 1, 64, 1, [64, 1, 2]), (1, 2, 4096, 128, [4096]), (1, 1, 30000, 700, [30000])]:
        vals = np.array([-3.5, -0.0, 0.0, 1.25, 1.25000012, 7.0, 246.0], np.float32)
        sc = vals[rng.integers(0, len(vals), size=(B, Hkv, nmax))]
        sel = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
        ss.ss_select_topk(torch.from_numpy(sc).cuda(), torch.tensor(nblk, dtype=torch.int32, device="cuda"), B, Hkv,
                          nmax, k, sel)
        ref = oracle_impl.select(sc.astype(np.float64), np.array(nblk, np.int32), k)
        np.testing.assert_array_equal(sel.cpu().numpy(), ref)


def test_topk_random_scores_match(ss, oracle_impl):
    """Continuous random scores (no ties) at the workloads' block counts and
    in every workgroup-width class of the kernel (up to 65536 blocks)."""
    rng = np.random.default_rng(6)
    for nmax, k in [(256, 16), (2048, 128), (4096, 128), (8192, 128), (16384, 512), (700, 699), (40000, 256),
                    (65536, 128)]:
        sc = (246 + 21 * rng.standard_normal((2, 2, nmax))).astype(np.float32)
        sel = torch.empty(2, 2, k, dtype=torch.int32, device="cuda")
        ss.ss_select_topk(torch.from_numpy(sc).cuda(), torch.full((2,), nmax, dtype=torch.int32, device="cuda"), 2, 2,
                          nmax, k, sel)
        ref = oracle_impl.select(sc.astype(np.float64), np.full(2, nmax, np.int32), k)
        np.testing.assert_array_equal(sel.cpu().numpy(), ref)


def test_topk_clustered_scores(ss, oracle_impl):
    """Score rows whose first radix digit takes one or a few values (a narrow
    band with far outliers, mixed signs, a single value with one larger),
    rows shorter than k and empty rows: the selections equal the oracle's."""
    rng = np.random.default_rng(11)
    B, Hkv, nmax, k = 4, 4, 8192, 128
    rows = []
    band = 30 + 1e-3 * rng.standard_normal(nmax)
    out = band.copy()
    out[::97] += 5e4  # 85 outliers, then the band
    rows.append(out)
    rows.append(0.5 * rng.standard_normal(nmax))  # mixed signs around zero
    one = np.full(nmax, 7.0)
    one[4000] = 8.0
    rows.append(one)  # massive ties below one larger value
    rows.append(np.concatenate([np.full(nmax // 2, -1.0), 1e-30 * np.arange(nmax // 2)]))  # subnormals and -1
    rows.append(np.where(rng.random(nmax) < 0.02, 1e6, 1.0) + 1e-3 * rng.standard_normal(nmax))  # ~164 above the rest
    rows.append(np.round(rng.standard_normal(nmax), 1))  # few distinct values
    while len(rows) < B * Hkv:
        rows.append(246 + 21 * rng.standard_normal(nmax))
    sc = np.stack(rows).reshape(B, Hkv, nmax).astype(np.float32)
    for nblk in ([nmax] * B, [nmax, 100, 0, 129]):
        sel = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
        ss.ss_select_topk(torch.from_numpy(sc).cuda(), torch.tensor(nblk, dtype=torch.int32, device="cuda"), B, Hkv,
                          nmax, k, sel)
        ref = oracle_impl.select(sc.astype(np.float64), np.array(nblk, np.int32), k)
        np.testing.assert_array_equal(sel.cpu().numpy(), ref)


def test_attention_skips_invalid_slots(ss, oracle_impl):
    """-1 entries anywhere and slots >= slot_limit are skipped."""
    w = workload("gqa1-blk32")  # B=2, Hq=Hkv=4, blk 32, 64 blocks, k=8
    slots = np.array([[[3, -1, 7, 70, 0, -1, 63, 5],
                       [-1, -1, -1, -1, -1, -1, -1, -1],
                       [64, 65, 1000, -1, 2, -1, -1, -1],
                       [10, 11, 12, 13, 14, 15, 16, 17]],
                      [[1, 2, 3, 4, 5, 6, 64, 65],
                       [10, -1, 11, -1, 12, -1, 13, -1],
                       [-1, -1, -1, -1, -1, -1, -1, 9],
                       [63, 62, 61, 60, 59, 58, 57, 56]]], np.int32)
    out = gu.run_attention(ss, w, torch.from_numpy(slots).cuda(), slot_limit=64).cpu().numpy()
    ora_slots = np.where(slots >= 64, -1, slots)
    ref = oracle_impl.attention(w.q_host, w.kv_host, w.unit_off_host, ora_slots, w.Hkv, w.blk)
    assert np.abs(out - ref).max() <= gu.ATTN_TOL
    assert np.all(out[0, 1] == 0)  # every entry skipped -> zero output


def test_attention_bounds_slots_by_unit_capacity(ss, oracle_impl):
    """With per-unit capacities, a slot at or above its unit's own capacity
    is skipped even when it lies below slot_limit.  The over-capacity slots
    sit in units that are not last, so each one addresses bytes inside the
    allocation (in the unit's 64-record region): reading it would not fault,
    and would change the output."""
    w = workload("gqa1-blk32")  # B=2, Hq=Hkv=4, blk 32, 64 records per unit, k=8
    cap = np.array([64, 10, 0, 30, 64, 5, 64, 20], np.int32)
    slots = np.array([[[3, 9, 7, 40, 0, 63, 62, 5],
                       [9, 10, 11, 40, 0, 1, 2, -1],
                       [0, 1, 2, 3, 4, 5, 6, 7],
                       [29, 30, 31, 50, 1, -1, 2, 3]],
                      [[1, 2, 3, 4, 5, 6, 64, 65],
                       [4, 5, 6, 7, 8, 0, 1, 63],
                       [10, -1, 11, -1, 12, -1, 13, 60],
                       [19, 20, 21, 0, 22, 1, 2, 3]]], np.int32)
    assert np.any((slots >= cap.reshape(2, 4, 1)) & (slots < 64))
    out = gu.run_attention(ss, w, torch.from_numpy(slots).cuda(), slot_limit=64,
                           capacity=torch.from_numpy(cap).cuda()).cpu().numpy()
    ora_slots = np.where((slots >= cap.reshape(2, 4, 1)) | (slots >= 64), -1, slots)
    ref = oracle_impl.attention(w.q_host, w.kv_host, w.unit_off_host, ora_slots, w.Hkv, w.blk)
    assert np.abs(out - ref).max() <= gu.ATTN_TOL
    assert np.all(out[0, 2] == 0)  # capacity 0: every entry skipped
    # without the capacities the same slots are read (the bound is what skips them)
    out_nocap = gu.run_attention(ss, w, torch.from_numpy(slots).cuda(), slot_limit=64).cpu().numpy()
    assert np.abs(out_nocap[0, 1] - ref[0, 1]).max() > 1e-3


def test_runs_are_bitwise_deterministic(ss):
    w = workload("gqa7-blk8-ragged")
    meta = gu.run_metadata(ss, w)
    res = []
    for _ in range(2):
        scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
        sel = torch.empty(w.B, w.Hkv, w.k, dtype=torch.int32, device="cuda")
        ss.ss_score_topk(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, w.k, scores, sel)
        out = gu.run_attention(ss, w, sel)
        res.append((sel.cpu().numpy(), out.cpu().numpy()))
    np.testing.assert_array_equal(res[0][0], res[1][0])
    np.testing.assert_array_equal(res[0][1].view(np.uint32), res[1][1].view(np.uint32))


def test_kernel_timing_hook(ss):
    """ss_time_next_kernel: the attached events bracket exactly one kernel
    (within the stream-recorded bracket around the same call), the call's
    result is unchanged, and the setting is consumed by that launch."""
    w = workload("gqa7-blk8-ragged")
    meta = gu.run_metadata(ss, w)
    scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
    ref = torch.empty_like(scores)
    ss.ss_score_blocks(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, ref)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev:
        e.record()
    torch.cuda.synchronize()
    ev[0].record()
    ss.ss_time_next_kernel(ev[1], ev[2])
    ss.ss_score_blocks(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, scores)
    ev[3].record()
    torch.cuda.synchronize()
    inner, outer = ev[1].elapsed_time(ev[2]), ev[0].elapsed_time(ev[3])
    print(f"[gpu] kernel {inner * 1e3:.1f} us inside a {outer * 1e3:.1f} us bracket", flush=True)
    assert 0 < inner <= outer
    assert ev[0].elapsed_time(ev[1]) >= 0 and ev[2].elapsed_time(ev[3]) >= 0
    valid_rows_equal(scores.cpu().numpy(), ref.cpu().numpy(), w.nblk_host)
    # consumed: the next launch does not touch the events again
    ss.ss_score_blocks(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, scores)
    torch.cuda.synchronize()
    assert ev[1].elapsed_time(ev[2]) == inner
    ss.ss_time_next_kernel(None, None)


def test_llama3_8b_shape_full_size(ss, oracle_impl):
    """The Llama-3-8B-shaped single layer at full size (B=32, 32/8 heads,
    32k context, blk 16, k=128, 64 planted blocks per head), every unit
    checked against the oracle."""
    cfg = synth.get(1)
    print(f"[gpu] {cfg.name}: generating", flush=True)
    w = gu.HbmWorkload(cfg.B, cfg.Hq, cfg.Hkv, cfg.blk, cfg.nblk_max, cfg.k, seed=0, n_plant=cfg.n_plant)
    meta = gu.run_metadata(ss, w)
    scores = torch.empty(w.B, w.Hkv, w.nblk_max, dtype=torch.float32, device="cuda")
    sel = torch.empty(w.B, w.Hkv, w.k, dtype=torch.int32, device="cuda")
    ss.ss_score_topk(w.q, meta, w.nblk, w.B, w.Hq, w.Hkv, w.nblk_max, w.d, w.k, scores, sel)
    out = gu.run_attention(ss, w, sel).cpu().numpy()
    gmeta = gu.u16(meta)
    print(f"[gpu] {cfg.name}: oracle", flush=True)
    om = oracle_meta(oracle_impl, w)
    np.testing.assert_array_equal(gmeta, om)
    S = oracle_impl.score(w.q_host, om, w.nblk_host, w.Hq, w.Hkv, w.nblk_max, w.d)
    osel = oracle_impl.select(S, w.nblk_host, w.k)
    gu.check_scores(scores.cpu().numpy(), S, w.q_host, om, w.nblk_host, w.Hq // w.Hkv)
    diff = gu.check_selection(sel.cpu().numpy(), osel, S, w.nblk_host, w.k)
    ref = oracle_impl.attention(w.q_host, w.kv_host, w.unit_off_host, osel, w.Hkv, w.blk)
    G = w.Hq // w.Hkv
    worst = 0.0
    for b in range(w.B):
        for g in range(w.Hkv):
            if (b, g) not in diff:
                worst = max(worst, float(np.abs(out[b, g * G:(g + 1) * G] - ref[b, g * G:(g + 1) * G]).max()))
    # attention on the oracle's own selection covers every unit
    out2 = gu.run_attention(ss, w, torch.from_numpy(osel).cuda()).cpu().numpy()
    worst2 = float(np.abs(out2 - ref).max())
    print(f"[gpu] {cfg.name}: tie-band units {len(diff)}, attention err {worst:.2e} / {worst2:.2e}")
    assert worst <= gu.ATTN_TOL and worst2 <= gu.ATTN_TOL

"""GPU parity over the HBM/DRAM hierarchy: whole decode steps
(ss_decode_layer: score, top-k, host resolve, gather from the pinned DRAM
pool, attention) against the oracle run on the same pool bytes, step after
step with drifting queries.

Lock-step rule: a (sequence, KV head) unit is compared exactly (slots,
miss rows, gathered cache bytes) and to 2e-3 (attention) as long as its
selections have equalled the oracle's at every step; a selection that
differs only inside the 1e-5 tie band is legitimate, and from then on the
two block caches of that unit hold different histories, so the unit leaves
the exact comparison (the count is reported and bounded).
"""
import dataclasses

import numpy as np
import pytest
import torch

import gpu_util as gu
import synth
from synth.configs import Config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ss():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2509_24626_amd import binding
    binding.lib()
    return binding


def lockstep(oracle_impl, cfg, seed, sample_b, steps, layer=0, flags=0, max_diverged_frac=0.25, parts=1):
    from paper_2509_24626_amd import harness as H
    lens = synth.gen.lengths(cfg, seed)
    nblk = (lens // cfg.blk).astype(np.int32)
    off, total = H.pool_layout(cfg, nblk)
    print(f"[gpu] {cfg.name}: pool {total / 2**30:.2f} GiB, sampled sequences {sample_b}, {parts} group(s)",
          flush=True)
    pool = H.HostPool(total, flags)
    try:
        L = H.build_hier_layer(cfg, seed, layer, pool, 0, nblk, progress=lambda m: print("[gpu]", m, flush=True),
                               parts=parts)
        qs = H.query_stream(cfg, seed, layer, steps)
        Hkv, k, G, rb = cfg.Hkv, cfg.k, cfg.G, cfg.record_bytes
        sb = list(sample_b)
        units = [b * Hkv + g for b in sb for g in range(Hkv)]
        nb_s = nblk[sb]
        cap_s = L.capacity[units]
        # oracle state for the sampled sequences
        meta_o = oracle_impl.build_metadata(pool.host, L.pool_off_host[units], nb_s, len(sb), Hkv, cfg.nblk_max,
                                            cfg.blk, 128)
        lru = oracle_impl.lru(len(sb), Hkv, nb_s, cap_s)
        img_off = np.concatenate([[0], np.cumsum(cap_s.astype(np.int64))[:-1]]) * rb
        image = np.zeros(int(cap_s.sum()) * rb + rb, np.uint8)
        pool_off_abs = L.pool_off_host[units]
        diverged = set()
        misses = []
        for t in range(steps + 1):
            q32, q = qs[t]
            L.step(t, q)
            torch.cuda.synchronize()
            misses.append(L.last_n_miss)
            qh = gu.u16(q)[sb]
            S = oracle_impl.score(qh, meta_o, nb_s, cfg.Hq, Hkv, cfg.nblk_max, 128)
            osel = oracle_impl.select(S, nb_s, k)
            gsel = L.sel.cpu().numpy()[sb]
            now = gu.check_selection(gsel, osel, S, nb_s, k)
            for (i, g) in now:
                diverged.add((i, g))
            oslots, omiss = lru.step(t, osel)
            oracle_impl.gather(omiss, pool.host, pool_off_abs, image, img_off, rb, Hkv)
            oout = oracle_impl.attention(qh, image, img_off, oslots, Hkv, cfg.blk)
            gslots = L.slots_h.numpy()[sb]
            gmiss = L.miss_h.numpy()[:L.last_n_miss]
            gout = L.out.cpu().numpy()[sb]
            for i, b in enumerate(sb):
                for g in range(Hkv):
                    if (i, g) in diverged:
                        continue
                    u = b * Hkv + g
                    np.testing.assert_array_equal(gslots[i, g], oslots[i, g], err_msg=f"slots t={t} b={b} g={g}")
                    gm = gmiss[(gmiss[:, 0] == b) & (gmiss[:, 1] == g)]
                    om = omiss[(omiss[:, 0] == i) & (omiss[:, 1] == g)]
                    np.testing.assert_array_equal(gm[:, 2:], om[:, 2:], err_msg=f"misses t={t} b={b} g={g}")
                    # every slot the selection uses holds the record the oracle gathered
                    base = int(L.cache_off_host[u])
                    region = L.cache[base:base + int(L.capacity[u]) * rb].cpu().numpy()
                    for s in oslots[i, g][oslots[i, g] >= 0]:
                        o = int(img_off[i * Hkv + g] + s * rb)
                        assert np.array_equal(region[s * rb:(s + 1) * rb], image[o:o + rb]), (t, b, g, s)
                    err = np.abs(gout[i, g * G:(g + 1) * G] - oout[i, g * G:(g + 1) * G]).max()
                    assert err <= gu.ATTN_TOL, (t, b, g, err)
        rate = [m / (L.units * k) for m in misses]
        print(f"[gpu] {cfg.name}: miss rate per step {[round(r, 3) for r in rate]}; "
              f"diverged units {len(diverged)}/{len(units)}", flush=True)
        assert len(diverged) <= max_diverged_frac * len(units)
        assert misses[0] == sum(min(k, int(n)) for n in nblk) * Hkv  # cold cache: everything misses
        L.close()
        return rate
    finally:
        pool.close()


SMALL = Config("hier-small-b3-ctx8k-blk16-k32-cache25", B=3, Hq=8, Hkv=2, d=128, blk=16, k=32, ctx=8192,
               placement="host", cache_frac=0.25, steps=6, drift=0.3)


def test_hier_small_lockstep(ss, oracle_impl):
    rate = lockstep(oracle_impl, SMALL, seed=3, sample_b=range(SMALL.B), steps=6)
    assert 0 < np.mean(rate[1:]) < 1


@pytest.mark.parametrize("parts", [2, 3])
def test_hier_small_pipelined_groups(ss, oracle_impl, parts):
    lockstep(oracle_impl, SMALL, seed=3, sample_b=range(SMALL.B), steps=6, parts=parts)


def test_hier_small_noncoherent_pool(ss, oracle_impl):
    lockstep(oracle_impl, SMALL, seed=4, sample_b=range(SMALL.B), steps=3, flags=1)


def test_hier_gqa7_blk8_small(ss, oracle_impl):
    cfg = dataclasses.replace(synth.get(4), name="qwen-gqa7-small", B=2, ctx=16384, k=64, steps=4)
    lockstep(oracle_impl, cfg, seed=5, sample_b=range(cfg.B), steps=4)


def test_hier_ragged_small(ss, oracle_impl):
    cfg = dataclasses.replace(synth.get(3), name="ragged-small", B=4, ctx_range=(2048, 6144), k=32, layers=1)
    lockstep(oracle_impl, cfg, seed=6, sample_b=range(cfg.B), steps=4)


def test_hier_128k_full_size_sampled(ss, oracle_impl):
    """The hierarchical 128k-context workload at full size (B=64, 32/8
    heads, 8192 blocks of 16 tokens, k=128, 25% cache, 16 drifting steps
    after the warm-up); the oracle follows 3 of the 64 sequences."""
    cfg = synth.get(2)
    rate = lockstep(oracle_impl, cfg, seed=0, sample_b=[0, 31, 63], steps=cfg.steps, parts=8)
    assert 0.05 < np.mean(rate[1:]) < 0.5


def test_hier_gqa7_full_size_sampled(ss, oracle_impl):
    """The Qwen-like GQA-7 fragmentation workload at full size (B=48, 28/4
    heads, 16384 blocks of 8 tokens, k=512, 15% cache, 8 steps)."""
    cfg = synth.get(4)
    lockstep(oracle_impl, cfg, seed=0, sample_b=[0, 47], steps=cfg.steps, parts=6)


def test_gather_bytes_and_range_checks(ss):
    """Standalone gather from a mapped host pool and from HBM: each valid
    row copies its record exactly; rows out of range are skipped."""
    from paper_2509_24626_amd import harness as H
    B, Hkv, nblk, cap = 3, 2, 50, 10
    for rb in (4096, 8192, 16384):
        pool = H.HostPool(B * Hkv * nblk * rb)
        try:
            rng = np.random.default_rng(rb)
            pool.u8[:] = rng.integers(0, 256, size=pool.nbytes, dtype=np.uint8)
            pool_off = np.arange(B * Hkv, dtype=np.int64) * nblk * rb
            cache_off = np.arange(B * Hkv, dtype=np.int64)[::-1].copy() * cap * rb
            rows = [(0, 0, 3, 1), (2, 1, 49, 9), (1, 0, 0, 0), (2, 0, 7, 4), (0, 1, 50, 2), (0, 1, 3, 10),
                    (3, 0, 1, 1), (1, 2, 1, 1), (-1, 0, 1, 1), (1, 1, 12, 5)]
            valid = rows[:4] + rows[-1:]
            miss = torch.tensor(rows, dtype=torch.int32, device="cuda")
            for src_name, src in (("host", pool.dev), ("hbm", torch.from_numpy(pool.u8.copy()).cuda())):
                cache = torch.zeros(B * Hkv * cap * rb, dtype=torch.uint8, device="cuda")
                ss.ss_gather_blocks(miss, len(rows), src, torch.from_numpy(pool_off).cuda(), cache,
                                    torch.from_numpy(cache_off).cuda(),
                                    torch.full((B,), nblk, dtype=torch.int32, device="cuda"),
                                    torch.full((B * Hkv,), cap, dtype=torch.int32, device="cuda"), B, Hkv, rb)
                c = cache.cpu().numpy()
                written = np.zeros(c.size, bool)
                for b, g, j, s in valid:
                    u = b * Hkv + g
                    dst = slice(cache_off[u] + s * rb, cache_off[u] + (s + 1) * rb)
                    src_b = slice(pool_off[u] + j * rb, pool_off[u] + (j + 1) * rb)
                    assert np.array_equal(c[dst], pool.u8[src_b]), (src_name, rb, b, g, j, s)
                    written[dst] = True
                assert np.all(c[~written] == 0), (src_name, rb)
        finally:
            pool.close()

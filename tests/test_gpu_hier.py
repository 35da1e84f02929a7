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


class Track:
    """The oracle following sampled sequences of one GPU layer step by step
    (its own metadata from the pool bytes, LRU cache, cache image)."""

    def __init__(self, oracle_impl, cfg, L, pool, sample_b, name=""):
        self.o, self.cfg, self.L, self.pool, self.name = oracle_impl, cfg, L, pool, name
        Hkv, rb = cfg.Hkv, cfg.record_bytes
        self.sb = list(sample_b)
        self.units = [b * Hkv + g for b in self.sb for g in range(Hkv)]
        self.nb_s = L.nblk_host[self.sb].astype(np.int32)
        cap_s = L.capacity[self.units]
        self.reserve = L.reserve
        if self.reserve:
            # with appends the oracle keeps a private copy of the sampled units'
            # records (the drawn inputs) plus room for the blocks it saves itself
            blocks = np.repeat(self.nb_s.astype(np.int64) + self.reserve, Hkv)
            self.src_off = np.concatenate([[0], np.cumsum(blocks)[:-1]]) * rb
            self.src = np.zeros(int(blocks.sum()) * rb, np.uint8)
            for i, u in enumerate(self.units):
                n = int(self.nb_s[i // Hkv]) * rb
                self.src[self.src_off[i]:self.src_off[i] + n] = pool.u8[L.pool_off_host[u]:L.pool_off_host[u] + n]
            self.src_blocks = self.nb_s + self.reserve
            self.open = np.zeros((len(self.sb), Hkv, rb // 2), np.uint16)
            self.len = self.nb_s * cfg.blk
            self.nb0 = self.nb_s.copy()
        else:
            self.src, self.src_off = pool.host, L.pool_off_host[self.units]
        self.kind, self.agg = L.meta_kind, L.agg
        build = oracle_impl.build_metadata if self.kind == 0 else oracle_impl.build_metadata_mean
        self.meta = build(self.src, self.src_off, self.nb_s, len(self.sb), Hkv, L.nblk_max, cfg.blk, 128)
        if self.kind != 0:  # the oracle's append writes cuboid rows; mean rows are made from its open records
            self.meta_cuboid = np.zeros((len(self.sb), Hkv, L.nblk_max, 2, 128), np.uint16)
        # block counts only bound which indices are valid: give the LRU the final ones
        self.lru = oracle_impl.lru(len(self.sb), Hkv, self.nb_s + self.reserve, cap_s)
        self.img_off = np.concatenate([[0], np.cumsum(cap_s.astype(np.int64))[:-1]]) * rb
        self.image = np.zeros(int(cap_s.sum()) * rb + rb, np.uint8)
        self.diverged = set()

    def append_and_save(self, new_kv):
        """The oracle's side of a step's saving: the sampled sequences' new
        tokens go to the private pool copy and to the open blocks."""
        kv = gu.u16(new_kv)[self.sb]
        self.o.save(kv[:, None], self.len, self.cfg.blk, self.src, self.src_off, self.src_blocks)
        if self.kind == 0:
            self.o.append(kv, self.len, self.nb_s, self.cfg.blk, self.L.nblk_max, self.open, self.meta)
            return
        before = self.nb_s.copy()
        self.o.append(kv, self.len, self.nb_s, self.cfg.blk, self.L.nblk_max, self.open, self.meta_cuboid)
        for i in np.nonzero(self.nb_s != before)[0]:
            j = int(self.nb_s[i]) - 1
            for g in range(self.cfg.Hkv):
                m = self.o.build_metadata_mean(self.open[i, g], np.zeros(1, np.int64), np.ones(1, np.int32), 1, 1, 1,
                                               self.cfg.blk, 128)
                self.meta[i, g, j] = m[0, 0, 0]

    def check_saved(self):
        """After the run: block counts, metadata rows and DRAM records of the
        blocks filled by appends, and the open blocks' filled rows."""
        cfg, L, Hkv, rb = self.cfg, self.L, self.cfg.Hkv, self.cfg.record_bytes
        import paper_2509_24626_amd.binding as ssb
        ssb.ss_kv_save_wait(L.saver)
        np.testing.assert_array_equal(L.nblk.cpu().numpy()[self.sb], self.nb_s)
        np.testing.assert_array_equal(L.len_dev.cpu().numpy()[self.sb], self.len)
        meta_g = L.meta.cpu().numpy().view(np.uint16)
        open_g = L.open.cpu().numpy().view(np.uint16)
        for i, b in enumerate(self.sb):
            n0, n1 = int(self.nb0[i]), int(self.nb_s[i])
            np.testing.assert_array_equal(meta_g[b, :, n0:n1], self.meta[i, :, n0:n1])
            p = int(self.len[i]) % cfg.blk
            for g in range(Hkv):
                u, iu = b * Hkv + g, i * Hkv + g
                got = self.pool.u8[L.pool_off_host[u] + n0 * rb:L.pool_off_host[u] + n1 * rb]
                np.testing.assert_array_equal(got, self.src[self.src_off[iu] + n0 * rb:self.src_off[iu] + n1 * rb])
                np.testing.assert_array_equal(open_g[b, g, :p * 128], self.open[i, g, :p * 128])

    def check(self, t, q):
        """Compares the GPU layer's step t (already run and synchronised)."""
        o, cfg, L, sb = self.o, self.cfg, self.L, self.sb
        Hkv, k, G, rb = cfg.Hkv, cfg.k, cfg.G, cfg.record_bytes
        qh = gu.u16(q)[sb]
        if self.kind == 0 and self.agg == 0:
            S = o.score(qh, self.meta, self.nb_s, cfg.Hq, Hkv, L.nblk_max, 128)
        else:
            S = o.score_variant(qh, self.meta, self.kind, self.agg, self.nb_s, cfg.Hq, Hkv, L.nblk_max, 128)
        osel = o.select(S, self.nb_s, k)
        gsel = L.sel.cpu().numpy()[sb]
        for (i, g) in gu.check_selection(gsel, osel, S, self.nb_s, k):
            self.diverged.add((i, g))
        oslots, omiss = self.lru.step(t, osel)
        o.gather(omiss, self.src, self.src_off, self.image, self.img_off, rb, Hkv)
        oout = o.attention(qh, self.image, self.img_off, oslots, Hkv, cfg.blk)
        if L.dev is None:
            gslots = L.slots_h.numpy()[sb]
            gmiss = L.miss_h.numpy()[:L.last_n_miss]
        else:  # device resolve: per-unit regions of miss rows
            gslots = L.slots.cpu().numpy()[sb]
            counts, rows, err = L.dev_miss_rows()
            assert err == 0, err
            gmiss = np.concatenate([rows[u, :counts[u]] for u in range(L.units)] + [np.zeros((0, 4), np.int32)])
        gout = L.out.cpu().numpy()[sb]
        for i, b in enumerate(sb):
            for g in range(Hkv):
                if (i, g) in self.diverged:
                    continue
                u = b * Hkv + g
                where = f"{self.name} t={t} b={b} g={g}"
                np.testing.assert_array_equal(gslots[i, g], oslots[i, g], err_msg="slots " + where)
                gm = gmiss[(gmiss[:, 0] == b) & (gmiss[:, 1] == g)]
                om = omiss[(omiss[:, 0] == i) & (omiss[:, 1] == g)]
                np.testing.assert_array_equal(gm[:, 2:], om[:, 2:], err_msg="misses " + where)
                # every slot the selection uses holds the record the oracle gathered
                base = int(L.cache_off_host[u])
                region = L.cache[base:base + int(L.capacity[u]) * rb].cpu().numpy()
                for s in oslots[i, g][oslots[i, g] >= 0]:
                    off = int(self.img_off[i * Hkv + g] + s * rb)
                    assert np.array_equal(region[s * rb:(s + 1) * rb], self.image[off:off + rb]), (where, s)
                err = np.abs(gout[i, g * G:(g + 1) * G] - oout[i, g * G:(g + 1) * G]).max()
                assert err <= gu.ATTN_TOL, (where, err)


_POOL = None


def _pool():
    """Host threads for the oracle's per-sequence work (its C calls release
    the GIL)."""
    global _POOL
    if _POOL is None:
        import os
        from concurrent.futures import ThreadPoolExecutor
        _POOL = ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0)))))
    return _POOL


class ParTrack:
    """The oracle following sequences of one GPU layer step by step, one
    independent oracle state per sequence (its metadata from the pool bytes,
    its LRU cache, its cache image), the sequences spread over host threads,
    so that every unit of a full-size batch can be followed.

    Per step and unit it checks
      * the selection against the oracle's scores under the tie-band rule
        (every step), and the GPU scores against the fp32 summation bound
        (the first `score_steps` steps);
      * slots and miss rows, bit-exact, for units whose selections have
        equalled the oracle's at every step so far (a legitimate tie-band
        difference gives the two caches different histories);
      * attention to 2e-3 whenever the unit's selection equals the oracle's
        at this step (its output depends on the selected blocks only);
      * gathered bytes: every record the GPU gathered this step, in the slot
        its miss row names, against the DRAM record of its block;
      * for the units of `image_b`, every slot the selection uses against
        the oracle's cache image (hits included)."""

    def __init__(self, oracle_impl, cfg, L, pool, sample_b, name="", score_steps=4, image_b=None):
        self.o, self.cfg, self.L, self.pool, self.name = oracle_impl, cfg, L, pool, name
        self.sb = list(sample_b)
        self.score_steps = score_steps
        self.image_b = set(self.sb if image_b is None else image_b)
        self.kind, self.agg = L.meta_kind, L.agg
        self.diverged = set()
        self.sel_differs = 0
        assert L.reserve == 0
        self.seq = dict(zip(self.sb, _pool().map(self._init_seq, self.sb)))

    @property
    def units(self):
        return [b * self.cfg.Hkv + g for b in self.sb for g in range(self.cfg.Hkv)]

    def _init_seq(self, b):
        o, cfg, L = self.o, self.cfg, self.L
        Hkv, rb = cfg.Hkv, cfg.record_bytes
        us = np.arange(b * Hkv, (b + 1) * Hkv)
        nb = L.nblk_host[b:b + 1].astype(np.int32)
        cap = L.capacity[us]
        build = o.build_metadata if self.kind == 0 else o.build_metadata_mean
        src_off = L.pool_off_host[us]
        meta = build(self.pool.host, src_off, nb, 1, Hkv, L.nblk_max, cfg.blk, 128)
        img_off = np.concatenate([[0], np.cumsum(cap.astype(np.int64))[:-1]]) * rb
        return {"nb": nb, "meta": meta, "src_off": src_off, "lru": o.lru(1, Hkv, nb, cap), "img_off": img_off,
                "image": np.zeros(int(cap.sum()) * rb + rb, np.uint8)}

    def _step_seq(self, b, t, qh, gsel, gscores, gslots, gmiss_u, gout):
        """The oracle's step t for sequence b and the per-unit comparisons;
        returns the units (g) whose selection left the exact comparison now."""
        o, cfg, L, st = self.o, self.cfg, self.L, self.seq[b]
        Hkv, k, G, rb = cfg.Hkv, cfg.k, cfg.G, cfg.record_bytes
        q1 = qh[b:b + 1]
        if self.kind == 0 and self.agg == 0:
            S = o.score(q1, st["meta"], st["nb"], cfg.Hq, Hkv, L.nblk_max, 128)
        else:
            S = o.score_variant(q1, st["meta"], self.kind, self.agg, st["nb"], cfg.Hq, Hkv, L.nblk_max, 128)
        if gscores is not None:
            if self.kind == 0 and self.agg == 0:
                gu.check_scores(gscores[b:b + 1], S, q1, st["meta"], st["nb"], G)
            else:
                gu.check_scores_variant(gscores[b:b + 1], S, q1, st["meta"], st["nb"], G, self.kind, self.agg)
        osel = o.select(S, st["nb"], k)
        new_div = [g for (_, g) in gu.check_selection(gsel[b:b + 1], osel, S, st["nb"], k)]
        oslots, omiss = st["lru"].step(t, osel)
        o.gather(omiss, self.pool.host, st["src_off"], st["image"], st["img_off"], rb, Hkv)
        oout = o.attention(q1, st["image"], st["img_off"], oslots, Hkv, cfg.blk)
        for g in range(Hkv):
            where = f"{self.name} t={t} b={b} g={g}"
            u = b * Hkv + g
            if np.array_equal(gsel[b, g], osel[0, g]):
                err = np.abs(gout[b, g * G:(g + 1) * G] - oout[0, g * G:(g + 1) * G]).max()
                assert err <= gu.ATTN_TOL, (where, err)
            if (b, g) in self.diverged or g in new_div:
                continue
            np.testing.assert_array_equal(gslots[b, g], oslots[0, g], err_msg="slots " + where)
            om = omiss[omiss[:, 1] == g]
            np.testing.assert_array_equal(gmiss_u[u][:, 2:], om[:, 2:], err_msg="misses " + where)
            if b in self.image_b:
                used = oslots[0, g][oslots[0, g] >= 0].astype(np.int64)
                rows = torch.from_numpy(int(L.cache_off_host[u]) // rb + used).cuda()
                got = L.cache.view(-1, rb).index_select(0, rows).cpu().numpy()
                want = st["image"].reshape(-1, rb)[int(st["img_off"][g]) // rb + used]
                assert np.array_equal(got, want), ("cache image " + where)
        return new_div

    def check(self, t, q):
        """Compares the GPU layer's step t (already run and synchronised)."""
        cfg, L = self.cfg, self.L
        Hkv, k, rb = cfg.Hkv, cfg.k, cfg.record_bytes
        qh = gu.u16(q)
        gsel = L.sel.cpu().numpy()
        gscores = L.scores.cpu().numpy() if t < self.score_steps else None
        gout = L.out.cpu().numpy()
        if L.dev is None:
            gslots = L.slots_h.numpy().copy()
            gmiss = L.miss_h.numpy()[:L.last_n_miss].copy()
            u_of = gmiss[:, 0].astype(np.int64) * Hkv + gmiss[:, 1]
            order = np.argsort(u_of, kind="stable")
            bounds = np.searchsorted(u_of[order], np.arange(L.units + 1))
            gmiss_u = [gmiss[order[bounds[u]:bounds[u + 1]]] for u in range(L.units)]
        else:  # device resolve: per-unit regions of miss rows
            gslots = L.slots.cpu().numpy()
            counts, rows, err = L.dev_miss_rows()
            assert err == 0, err
            gmiss_u = [rows[u, :counts[u]] for u in range(L.units)]
            gmiss = np.concatenate(gmiss_u + [np.zeros((0, 4), np.int32)])
        futs = [_pool().submit(self._step_seq, b, t, qh, gsel, gscores, gslots, gmiss_u, gout) for b in self.sb]
        for b, f in zip(self.sb, futs):
            for g in f.result():
                self.diverged.add((b, g))
        self._check_gathered(gmiss)

    def _check_gathered(self, gmiss, chunk=8192):
        """Every record gathered in this step holds its block's DRAM bytes."""
        L, rb, Hkv = self.L, self.cfg.record_bytes, self.cfg.Hkv
        if len(gmiss) == 0:
            return
        u = gmiss[:, 0].astype(np.int64) * Hkv + gmiss[:, 1]
        slot_row = L.cache_off_host[u] // rb + gmiss[:, 3]
        pool_row = L.pool_off_host[u] // rb + gmiss[:, 2]
        cache_rows = L.cache.view(-1, rb)
        pool_rows = self.pool.u8.reshape(-1, rb)
        for i in range(0, len(gmiss), chunk):
            got = cache_rows.index_select(0, torch.from_numpy(slot_row[i:i + chunk]).cuda()).cpu().numpy()
            want = pool_rows[pool_row[i:i + chunk]]
            if not np.array_equal(got, want):
                bad = i + int(np.nonzero((got != want).any(axis=1))[0][0])
                raise AssertionError(f"{self.name}: gathered record differs, miss row {gmiss[bad].tolist()}")


def group_samples(part_sizes):
    """One sequence from every sequence group (its first)."""
    ends = np.cumsum(part_sizes)
    return [int(e - n) for e, n in zip(ends, part_sizes)]


def lockstep(oracle_impl, cfg, seed, sample_b, steps, layer=0, flags=0, max_diverged_frac=0.25, parts=1, meta_kind=0,
             agg=0, dev_cache=False, nblk=None, image_b=None):
    from paper_2509_24626_amd import harness as H
    if nblk is None:
        nblk = (synth.gen.lengths(cfg, seed) // cfg.blk).astype(np.int32)
    nblk = np.asarray(nblk, np.int32)
    off, total = H.pool_layout(cfg, nblk)
    print(f"[gpu] {cfg.name}: pool {total / 2**30:.2f} GiB, sampled sequences {sample_b}, {parts} group(s)",
          flush=True)
    pool = H.HostPool(total, flags)
    try:
        L = H.build_hier_layer(cfg, seed, layer, pool, 0, nblk, progress=lambda m: print("[gpu]", m, flush=True),
                               parts=parts, meta_kind=meta_kind, agg=agg, dev_cache=dev_cache)
        qs = H.query_stream(cfg, seed, layer, steps)
        tr = ParTrack(oracle_impl, cfg, L, pool, sample_b, cfg.name, image_b=image_b)
        misses = []
        for t in range(steps + 1):
            L.step(t, qs[t][1])
            torch.cuda.synchronize()
            misses.append(L.last_n_miss if L.dev is None else int(L.dev_miss_rows()[0].sum()))
            tr.check(t, qs[t][1])
            print(f"[gpu] {cfg.name} step {t}: {misses[-1]} blocks gathered, checked "
                  f"{len(tr.units)} units, diverged so far {len(tr.diverged)}", flush=True)
        rate = [m / (L.units * cfg.k) for m in misses]
        print(f"[gpu] {cfg.name}: miss rate per step {[round(r, 3) for r in rate]}; "
              f"diverged units {len(tr.diverged)}/{len(tr.units)}", flush=True)
        assert len(tr.diverged) <= max_diverged_frac * len(tr.units)
        assert misses[0] == sum(min(cfg.k, int(n)) for n in nblk) * cfg.Hkv  # cold cache: everything misses
        L.close()
        return rate
    finally:
        pool.close()


def lockstep_with_save(oracle_impl, cfg, seed, sample_b, steps, parts=1, save_stream=False, meta_kind=0, agg=0,
                       dev_cache=False):
    """Decode steps that also append and save each step's new tokens
    (ss_append_kv, FlashD2H), so blocks fill during the run and become
    selectable; the oracle follows the sampled sequences on its own copy of
    their records."""
    from paper_2509_24626_amd import harness as H
    lens = synth.gen.lengths(cfg, seed)
    nblk = (lens // cfg.blk).astype(np.int32)
    reserve = steps // cfg.blk + 2
    off, total = H.pool_layout(cfg, nblk, reserve)
    print(f"[gpu] {cfg.name} with save: pool {total / 2**30:.2f} GiB, {steps} steps, reserve {reserve}, "
          f"sampled {sample_b}, {parts} group(s), save stream {save_stream}", flush=True)
    pool = H.HostPool(total)
    try:
        L = H.build_hier_layer(cfg, seed, 0, pool, 0, nblk, parts=parts, reserve=reserve, meta_kind=meta_kind, agg=agg,
                               dev_cache=dev_cache)
        L.enable_save(threads=2, save_stream=torch.cuda.Stream() if save_stream else None)
        sK, sV = synth.gen.channel_scales(cfg.Hkv, 128, seed, 0, "cuda")
        qs = H.query_stream(cfg, seed, 0, steps)
        tr = Track(oracle_impl, cfg, L, pool, sample_b, cfg.name + " +save")
        new_selected = 0
        for t in range(steps + 1):
            kv = synth.gen.new_tokens(cfg.B, cfg.Hkv, 128, sK, sV, seed, 0, t, "cuda")
            L.step_with_save(t, qs[t][1], kv)
            torch.cuda.synchronize()
            tr.check(t, qs[t][1])
            sel = L.sel.cpu().numpy()
            new_selected += int(sum((sel[b] >= nblk[b]).sum() for b in range(cfg.B)))
            tr.append_and_save(kv)
        tr.check_saved()
        filled = L.nblk.cpu().numpy() - nblk
        print(f"[gpu] blocks filled per sequence {sorted(set(filled.tolist()))}; selections of new blocks "
              f"{new_selected}; diverged {len(tr.diverged)}/{len(tr.units)}", flush=True)
        assert filled.min() >= 1 and int(L.overflow.item()) == 0
        assert len(tr.diverged) <= 0.25 * len(tr.units)
        L.close()
        return new_selected
    finally:
        pool.close()


# Units whose selection may legitimately leave the exact comparison in a
# full-size run.  A selection differs from the oracle's only when the GPU's
# fp32 scores (relative error below 3e-7) reorder two blocks whose fp64
# scores lie that close around the k-th; at the workloads' score spread
# (k-th gap ~2e-4 relative) that is ~0.1-0.2% of unit-steps at worst, so a
# few percent of the units over 8-16 steps.
FULL_DIVERGED_FRAC = 0.05

SMALL = Config("hier-small-b3-ctx8k-blk16-k32-cache25", B=3, Hq=8, Hkv=2, d=128, blk=16, k=32, ctx=8192,
               placement="host", cache_frac=0.25, steps=6, drift=0.3)


def test_hier_small_lockstep(ss, oracle_impl):
    rate = lockstep(oracle_impl, SMALL, seed=3, sample_b=range(SMALL.B), steps=6)
    assert 0 < np.mean(rate[1:]) < 1


def test_decode_layer_wait_deadline(ss, oracle_impl):
    """A host wait for a selection that passes the deadline set with
    ss_set_host_wait_timeout returns SS_ERR_TIMEOUT and leaves the block
    cache untouched.  The stream is held busy by ordinary work queued before
    the step (four fp32 8192^3 products, tens of milliseconds) against a
    2 ms deadline; after synchronising, the same step with the default
    deadline matches the oracle, which never saw the failed call."""
    from paper_2509_24626_amd import harness as H
    cfg = SMALL
    nblk = (synth.gen.lengths(cfg, 3) // cfg.blk).astype(np.int32)
    _, total = H.pool_layout(cfg, nblk)
    pool = H.HostPool(total)
    try:
        L = H.build_hier_layer(cfg, 3, 0, pool, 0, nblk, parts=2)
        qs = H.query_stream(cfg, 3, 0, 2)
        tr = Track(oracle_impl, cfg, L, pool, range(cfg.B), "deadline")
        L.step(0, qs[0][1])
        torch.cuda.synchronize()
        tr.check(0, qs[0][1])
        x = torch.randn(8192, 8192, device="cuda")
        torch.cuda.synchronize()
        ss.ss_set_host_wait_timeout(2)
        try:
            for _ in range(4):
                x = x @ x * 1e-4
            with pytest.raises(ss.SparseServeError) as e:
                L.step(1, qs[1][1])
            assert e.value.status == ss.SS_ERR_TIMEOUT, str(e.value)
            assert "step 1" in str(e.value)
        finally:
            ss.ss_set_host_wait_timeout(0)
        torch.cuda.synchronize()
        for t in (1, 2):
            L.step(t, qs[t][1])
            torch.cuda.synchronize()
            tr.check(t, qs[t][1])
        assert not tr.diverged
        L.close()
    finally:
        pool.close()


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


SAVE_SMALL = Config("hier-save-b3-ctx1k-blk16-k16-cache25", B=3, Hq=8, Hkv=2, d=128, blk=16, k=16, ctx=1024,
                    placement="host", cache_frac=0.25, steps=40, drift=0.3)


@pytest.mark.parametrize("save_stream", [False, True])
def test_hier_small_with_append_and_save(ss, oracle_impl, save_stream):
    """40 steps on 64-block sequences: every sequence fills 2 blocks, which
    are then selected and gathered back from the DRAM records FlashD2H
    wrote."""
    n = lockstep_with_save(oracle_impl, SAVE_SMALL, seed=12, sample_b=range(SAVE_SMALL.B), steps=40, parts=2,
                           save_stream=save_stream)
    assert n > 0


@pytest.mark.parametrize("kind,agg", [(1, 0), (0, 1), (1, 1)], ids=["mean-max", "cuboid-sum", "mean-sum"])
def test_hier_small_score_variants(ss, oracle_impl, kind, agg):
    """Whole decode steps with the mean-key metadata and the sum over the
    GQA group: selections, slots, misses, gathered bytes and attention."""
    lockstep(oracle_impl, SMALL, seed=14, sample_b=range(SMALL.B), steps=6, parts=2, meta_kind=kind, agg=agg)


@pytest.mark.parametrize("save_stream", [False, True])
def test_hier_small_with_append_and_save_device_resolve(ss, oracle_impl, save_stream):
    """The save side with the cache resolved on the GPU: blocks filled by
    appends enter the device block table (its room covers the reserve) and
    are selected and gathered back."""
    n = lockstep_with_save(oracle_impl, SAVE_SMALL, seed=16, sample_b=range(SAVE_SMALL.B), steps=40, parts=2,
                           save_stream=save_stream, dev_cache=True)
    assert n > 0


def test_hier_ragged_with_append_and_save_device_resolve(ss, oracle_impl):
    cfg = dataclasses.replace(synth.get(3), name="ragged-save-small-dev", B=4, ctx_range=(1024, 4096), k=16, layers=1)
    lockstep_with_save(oracle_impl, cfg, seed=17, sample_b=range(cfg.B), steps=36, dev_cache=True)


def test_hier_small_mean_metadata_with_save(ss, oracle_impl):
    """Appends build mean-key rows when blocks fill; those blocks are then
    selected through the mean-key scores."""
    n = lockstep_with_save(oracle_impl, SAVE_SMALL, seed=15, sample_b=range(SAVE_SMALL.B), steps=40, parts=2,
                           meta_kind=1, agg=1)
    assert n > 0


def test_hier_128k_full_size_mean_sum_every_unit(ss, oracle_impl):
    """The 128k workload at full size with mean-key metadata and the sum
    aggregation (8 steps); the oracle follows all 512 units."""
    cfg = synth.get(2)
    lockstep(oracle_impl, cfg, seed=0, sample_b=range(cfg.B), steps=8, parts=8, meta_kind=1, agg=1,
             max_diverged_frac=FULL_DIVERGED_FRAC, image_b=group_samples([8] * 8))


def test_hier_ragged_with_append_and_save(ss, oracle_impl):
    cfg = dataclasses.replace(synth.get(3), name="ragged-save-small", B=4, ctx_range=(1024, 4096), k=16, layers=1)
    lockstep_with_save(oracle_impl, cfg, seed=13, sample_b=range(cfg.B), steps=36)


def test_hier_128k_full_size_with_save_sampled(ss, oracle_impl):
    """The 128k workload at full size with appends and saves: 20 steps, so
    every sequence fills one block at step 16.  The oracle keeps a private
    copy of the DRAM records it follows, so it follows one sequence of each
    of the 8 groups (64 units) and the last one."""
    cfg = synth.get(2)
    lockstep_with_save(oracle_impl, cfg, seed=0, sample_b=group_samples([8] * 8) + [63], steps=20, parts=8,
                       save_stream=True)


@pytest.mark.parametrize("parts", [1, 3])
def test_hier_small_device_resolve(ss, oracle_impl, parts):
    """The decode step with the slot table resolved on the GPU
    (ss_decode_layer_dev): slots, misses, gathered bytes and attention in
    lock-step with the oracle."""
    lockstep(oracle_impl, SMALL, seed=3, sample_b=range(SMALL.B), steps=6, parts=parts, dev_cache=True)


def test_hier_many_units_one_group_device_resolve(ss, oracle_impl):
    """72 sequences x 16 KV heads in one group: 1152 units, so the gather of
    per-unit miss rows sums the units' counts in two LDS chunks (1024 + 128)."""
    cfg = dataclasses.replace(SMALL, name="hier-many-units-b72-h16", B=72, Hq=32, Hkv=16, ctx=1024, k=8, steps=4)
    lockstep(oracle_impl, cfg, seed=9, sample_b=[0, 35, 64, 71], steps=4, parts=1, dev_cache=True)


@pytest.mark.parametrize("dev_cache", [False, True])
def test_hier_empty_and_short_sequences(ss, oracle_impl, dev_cache):
    """A sequence with no blocks, ones with fewer blocks than k (padded
    selections, every block selected) and a longer one, in two groups."""
    cfg = dataclasses.replace(SMALL, name="hier-empty-short", B=5, k=8)
    lockstep(oracle_impl, cfg, seed=21, sample_b=range(cfg.B), steps=5, parts=2, dev_cache=dev_cache,
             nblk=[0, 3, 40, 1, 90])


def test_hier_gqa7_small_device_resolve(ss, oracle_impl):
    cfg = dataclasses.replace(synth.get(4), name="qwen-gqa7-small-dev", B=2, ctx=16384, k=64, steps=4)
    lockstep(oracle_impl, cfg, seed=5, sample_b=range(cfg.B), steps=4, dev_cache=True)


def test_hier_128k_full_size_device_resolve_every_unit(ss, oracle_impl):
    """The 128k workload at full size with the resolve on the GPU and the
    automatic groups (bench.py --resolve device); the oracle follows all
    512 units."""
    from paper_2509_24626_amd import harness as H
    cfg = synth.get(2)
    parts = H.default_parts(cfg.B)
    lockstep(oracle_impl, cfg, seed=0, sample_b=range(cfg.B), steps=cfg.steps, parts=parts, dev_cache=True,
             max_diverged_frac=FULL_DIVERGED_FRAC, image_b=group_samples(parts))


def test_hier_128k_full_size_every_unit(ss, oracle_impl):
    """The hierarchical 128k-context workload at full size (B=64, 32/8
    heads, 8192 blocks of 16 tokens, k=128, 25% cache, 16 drifting steps
    after the warm-up) in the launch configuration bench.py times (the
    host-side resolve, the automatic groups); the oracle follows all 64
    sequences (512 units)."""
    from paper_2509_24626_amd import harness as H
    cfg = synth.get(2)
    parts = H.default_parts(cfg.B)
    rate = lockstep(oracle_impl, cfg, seed=0, sample_b=range(cfg.B), steps=cfg.steps, parts=parts,
                    max_diverged_frac=FULL_DIVERGED_FRAC, image_b=group_samples(parts))
    assert 0.05 < np.mean(rate[1:]) < 0.5


def test_hier_gqa7_full_size_every_unit(ss, oracle_impl):
    """The Qwen-like GQA-7 fragmentation workload at full size (B=48, 28/4
    heads, 16384 blocks of 8 tokens, k=512, 15% cache, 8 steps) in the
    launch configuration bench.py times; the oracle follows all 192 units."""
    from paper_2509_24626_amd import harness as H
    cfg = synth.get(4)
    parts = H.default_parts(cfg.B)
    lockstep(oracle_impl, cfg, seed=0, sample_b=range(cfg.B), steps=cfg.steps, parts=parts,
             max_diverged_frac=FULL_DIVERGED_FRAC, image_b=group_samples(parts))


def test_hier_gqa7_full_size_device_resolve_every_unit(ss, oracle_impl):
    """The GQA-7 workload at full size with the resolve on the GPU and the
    automatic groups (bench.py --resolve device); every unit followed."""
    from paper_2509_24626_amd import harness as H
    cfg = synth.get(4)
    parts = H.default_parts(cfg.B)
    lockstep(oracle_impl, cfg, seed=0, sample_b=range(cfg.B), steps=cfg.steps, parts=parts, dev_cache=True,
             max_diverged_frac=FULL_DIVERGED_FRAC, image_b=group_samples(parts))


@pytest.mark.parametrize("mode", ["host", "device", "groups", "host-groups"])
def test_layers32_ragged_full_size_every_unit(ss, oracle_impl, mode):
    """The 32-layer ragged workload at full size (B=16, lengths U[8k, 64k],
    k=128, 30% cache per layer, 8 drifting steps): every step runs all 32
    layers; the oracle follows all 16 sequences (128 units) in each of 4
    layers, two of which read DRAM records shared with an earlier layer.
    The automatic groups of each schedule: each layer's step in turn with
    the resolve on host threads (host) or on the GPU (device), and the
    groups pipelined across layers in one call per step with the resolve on
    the GPU (groups, ss_decode_step_dev) or on host threads (host-groups,
    ss_decode_step)."""
    from paper_2509_24626_amd import harness as H
    cfg = synth.get(3)
    seed = 0
    nblk = (synth.gen.lengths(cfg, seed) // cfg.blk).astype(np.int32)
    log = lambda m: print("[gpu]", m, flush=True)
    dev_cache = mode in ("device", "groups")
    grouped = mode in ("groups", "host-groups")
    parts = H.default_parts(cfg.B, "groups" if grouped else "layers")
    pool, layers, n = H.build_hier_model(cfg, seed, nblk, progress=log, parts=parts, dev_cache=dev_cache)
    try:
        print(f"[gpu] {cfg.name}: {n} of {cfg.layers} layers with their own DRAM records", flush=True)
        assert n < cfg.layers  # the 32 layers do not fit the pinned budget
        followed = [0, n - 1, n, cfg.layers - 1]
        qs = [H.query_stream(cfg, seed, l, cfg.steps) for l in range(cfg.layers)]
        tracks = {l: ParTrack(oracle_impl, cfg, layers[l], pool, range(cfg.B), f"layer {l}",
                              image_b=group_samples(layers[0].part_sizes)) for l in followed}
        for t in range(cfg.steps + 1):
            if grouped:
                H.decode_step_groups(layers, t, [qs[l][t][1] for l in range(cfg.layers)])
            else:
                for l, L in enumerate(layers):
                    L.step(t, qs[l][t][1])
            torch.cuda.synchronize()
            for l, tr in tracks.items():
                tr.check(t, qs[l][t][1])
            misses = [L.last_n_miss if L.dev is None else int(L.dev_miss_rows()[0].sum()) for L in layers]
            rates = [m / (L.units * cfg.k) for m, L in zip(misses, layers)]
            print(f"[gpu] step {t}: miss rate over layers {min(rates):.3f}..{max(rates):.3f}", flush=True)
            if t == 0:
                assert all(m == sum(min(cfg.k, int(x)) for x in nblk) * cfg.Hkv for m in misses)
        units = sum(len(tr.units) for tr in tracks.values())
        div = sum(len(tr.diverged) for tr in tracks.values())
        print(f"[gpu] diverged units {div}/{units}", flush=True)
        assert div <= FULL_DIVERGED_FRAC * units
        # aliased layers read the same DRAM records but keep caches of their own
        assert layers[n].pool_off_host[0] == layers[0].pool_off_host[0]
        assert layers[n].cache.data_ptr() != layers[0].cache.data_ptr()
    finally:
        for L in layers:
            L.close()
        pool.close()


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


def random_shapes(n, seed):
    """Seeded small hierarchical configurations: batch, heads and group
    size, block size, k, ragged lengths, cache fraction, group count and
    the resolve path all vary."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        Hkv = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.choice([1, 2, 4, 7, 16]))
        blk = int(rng.choice([8, 16, 32]))
        k = int(rng.choice([4, 16, 33, 64, 128]))
        lo = int(rng.integers(1, 80)) * blk
        hi = lo + int(rng.integers(0, 300)) * blk
        B = int(rng.integers(1, 12))
        cfg = Config(f"random-shape-{seed}-{i}", B=B, Hq=Hkv * G, Hkv=Hkv, d=128, blk=blk, k=k,
                     ctx_range=(lo, hi), placement="host", cache_frac=float(rng.choice([0.1, 0.25, 0.6])),
                     steps=3, drift=float(rng.choice([0.3, 0.8])))
        parts = int(rng.integers(1, min(B, 4) + 1))
        out.append((cfg, parts, bool(rng.integers(0, 2))))
    return out


@pytest.mark.parametrize("cfg,parts,dev_cache", random_shapes(20, 31), ids=lambda x: getattr(x, "name", str(x)))
def test_hier_random_shapes(ss, oracle_impl, cfg, parts, dev_cache):
    lockstep(oracle_impl, cfg, seed=7, sample_b=range(cfg.B), steps=cfg.steps, parts=parts, dev_cache=dev_cache)

"""Composition of the C-ABI calls into decode-step layers, with torch used
only to hold device memory and streams.

HbmLayer   all KV blocks resident in HBM: score/top-k, then attention with
           the selection as the slot list.
HierLayer  KV blocks in a pinned, device-mapped DRAM pool and an LRU HBM
           block cache per (sequence, KV head): one ss_decode_layer call
           per step (score/top-k, resolve, gather, attention).

build_hbm_layer / build_hier_layer draw a seeded synthetic layer (synth)
on the GPU, build its metadata with ss_build_metadata, and for the
hierarchical case copy the records into the DRAM pool.  Nothing here
computes any part of the method itself.
"""
import ctypes
import math

import numpy as np
import torch

import synth
from synth import gen

from . import binding as ss

D = 128


def _dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).cuda()


class HostPool:
    """Pinned, device-mapped host memory from ss_host_alloc_mapped."""

    def __init__(self, nbytes, flags=0):
        self.nbytes = nbytes
        self.host, self.dev = ss.ss_host_alloc_mapped(nbytes, flags)
        # CPU views of the same bytes (no copy)
        buf = (ctypes.c_uint8 * nbytes).from_address(self.host)
        self.u8 = np.frombuffer(buf, dtype=np.uint8)
        self.t = torch.from_numpy(self.u8)

    def close(self):
        if self.host:
            self.t = None
            self.u8 = None
            ss.ss_host_free(self.host)
            self.host = 0


class HbmLayer:
    def __init__(self, cfg, kv, nblk_host, meta=None):
        self.cfg = cfg
        B, Hkv = cfg.B, cfg.Hkv
        self.units = B * Hkv
        self.kv = kv
        self.nblk_host = np.asarray(nblk_host, np.int32)
        self.nblk = _dev(self.nblk_host, np.int32)
        self.unit_off = _dev(np.arange(self.units, dtype=np.int64) * cfg.nblk_max * cfg.record_bytes, np.int64)
        self.meta = meta if meta is not None else torch.empty(B, Hkv, cfg.nblk_max, 2, D, dtype=torch.int16,
                                                              device="cuda")
        self.scores = torch.empty(B, Hkv, cfg.nblk_max, dtype=torch.float32, device="cuda")
        self.sel = torch.empty(B, Hkv, cfg.k, dtype=torch.int32, device="cuda")
        self.out = torch.empty(B, cfg.Hq, D, dtype=torch.float32, device="cuda")
        self.ws_bytes = ss.ss_sparse_attention_workspace(B, cfg.Hq, Hkv, D, cfg.blk, cfg.k)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device="cuda")

    def build_metadata(self):
        c = self.cfg
        ss.ss_build_metadata(self.kv, self.unit_off, self.nblk, c.B, c.Hkv, c.nblk_max, c.blk, D, self.meta)

    def select(self, q):
        c = self.cfg
        ss.ss_score_topk(q, self.meta, self.nblk, c.B, c.Hq, c.Hkv, c.nblk_max, D, c.k, self.scores, self.sel)

    def attend(self, q, slots=None):
        c = self.cfg
        ss.ss_sparse_attention(q, self.kv, self.unit_off, self.sel if slots is None else slots, None, c.nblk_max,
                               c.B, c.Hq, c.Hkv, D, c.blk, c.k, 1.0 / math.sqrt(D), self.out, self.ws, self.ws_bytes)

    def step(self, q):
        self.select(q)
        self.attend(q)
        return self.out


def build_hbm_layer(cfg, seed, layer=0):
    """Draws a synthetic HBM-resident layer; returns (HbmLayer, q fp32, q bf16)."""
    q32, q = gen.query(cfg.B, cfg.Hq, D, seed, "cuda", layer)
    sK, sV = gen.channel_scales(cfg.Hkv, D, seed, layer, "cuda")
    kv = torch.empty(cfg.B, cfg.Hkv, cfg.nblk_max, cfg.record_bytes // 2, dtype=torch.bfloat16, device="cuda")
    for b in range(cfg.B):
        kv[b], _ = gen.kv_records_seq(b, cfg.Hkv, cfg.nblk_max, cfg.blk, D, sK, sV, seed, layer, "cuda",
                                      q_bf16_b=q[b], n_plant=cfg.n_plant, shift=cfg.plant_shift)
    lens = gen.lengths(cfg, seed)
    L = HbmLayer(cfg, kv, (lens // cfg.blk).astype(np.int32))
    L.build_metadata()
    return L, q32, q


class HierLayer:
    """One layer of the hierarchical workload: its DRAM pool slice, HBM
    metadata, HBM block cache and step buffers."""

    def __init__(self, cfg, nblk_host, capacity, pool, pool_off_host, meta, parts=1, reserve=0, meta_kind=0, agg=0,
                 dev_cache=False):
        self.cfg = cfg
        self.dev = None  # the slot table on the GPU (ss_dev_cache) instead of the host handle
        self.meta_kind, self.agg = meta_kind, agg
        # blocks each unit may gain (appended tokens) beyond its initial count:
        # the metadata, the scores and the pool have room for them
        self.reserve = reserve
        self.nblk_max = cfg.nblk_max + reserve
        assert meta.shape[2] == self.nblk_max
        # parts: a group count (equal groups) or a list of group sizes
        if isinstance(parts, (list, tuple)):
            assert sum(parts) == cfg.B and all(p > 0 for p in parts)
            self.part_sizes = list(parts)
        else:
            n = max(1, min(parts, cfg.B))
            self.part_sizes = [cfg.B * (i + 1) // n - cfg.B * i // n for i in range(n)]
        self.parts = len(self.part_sizes)
        self.part_end = np.cumsum(self.part_sizes).astype(np.int32)
        B, Hkv, k = cfg.B, cfg.Hkv, cfg.k
        self.units = B * Hkv
        self.nblk_host = np.asarray(nblk_host, np.int32)
        self.capacity = np.ascontiguousarray(capacity, np.int32).reshape(-1)
        self.pool = pool
        self.pool_off_host = np.asarray(pool_off_host, np.int64)
        self.meta = meta
        self.handle = ss.ss_cache_create(B, Hkv, self.nblk_host, self.capacity, cfg.record_bytes)
        self.total_slots = ss.ss_cache_total_slots(self.handle)
        off = np.empty(self.units, np.int64)
        ss.ss_cache_region_offsets(self.handle, off)
        self.cache_off_host = off
        self.cache = torch.empty(max(self.total_slots, 1) * cfg.record_bytes, dtype=torch.uint8, device="cuda")
        self.cache_off = _dev(off, np.int64)
        self.cap_dev = _dev(self.capacity, np.int32)
        self.nblk = _dev(self.nblk_host, np.int32)
        self.pool_off = _dev(self.pool_off_host, np.int64)
        self.scores = torch.empty(B, Hkv, self.nblk_max, dtype=torch.float32, device="cuda")
        self.sel = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
        self.slots = torch.empty(B, Hkv, k, dtype=torch.int32, device="cuda")
        self.miss_cap = self.units * k
        self.miss = torch.empty(self.miss_cap, 4, dtype=torch.int32, device="cuda")
        # pinned, mapped, coherent host buffers the kernels read and write directly
        self._staging = HostPool(max(1, (2 * self.units * k + 4 * self.miss_cap) * 4))
        st = self._staging.t.view(torch.int32)
        self.sel_h = st[:self.units * k].view(B, Hkv, k)
        self.slots_h = st[self.units * k:2 * self.units * k].view(B, Hkv, k)
        self.miss_h = st[2 * self.units * k:2 * self.units * k + 4 * self.miss_cap].view(self.miss_cap, 4)
        self.out = torch.empty(B, cfg.Hq, D, dtype=torch.float32, device="cuda")
        # attention runs per sequence group; with the resolve on the GPU the groups'
        # attentions run on up to four streams at once (two in a one-layer call,
        # four when the groups are pipelined across layers), each with its own region
        one = max(ss.ss_sparse_attention_workspace(b, cfg.Hq, Hkv, D, cfg.blk, k) for b in set(self.part_sizes))
        self.ws_bytes = min(4, self.parts) * ((one + 255) // 256 * 256)
        self.ws = torch.empty(max(self.ws_bytes, 16), dtype=torch.uint8, device="cuda")
        p = ss._ptr
        self.buffers = ss.ss_layer_buffers(
            B=B, Hq=cfg.Hq, Hkv=Hkv, d=D, blk=cfg.blk, nblk_max=self.nblk_max, k=k, scale=1.0 / math.sqrt(D),
            meta=p(meta), nblk_dev=p(self.nblk), pool=pool.dev, pool_off_dev=p(self.pool_off), cache=self.handle,
            cache_base=p(self.cache), cache_off_dev=p(self.cache_off), capacity_dev=p(self.cap_dev),
            slot_limit=int(self.capacity.max()) if self.units else 0, scores=p(self.scores), sel_dev=p(self.sel),
            slots_dev=p(self.slots), miss_dev=p(self.miss), sel_host=p(self.sel_h), slots_host=p(self.slots_h),
            miss_host=p(self.miss_h), miss_cap=self.miss_cap, attn_ws=p(self.ws), attn_ws_bytes=self.ws_bytes,
            parts=self.parts, part_end=self.part_end.ctypes.data, meta_kind=meta_kind, agg=agg)
        self.last_n_miss = 0
        self.saver = None
        if dev_cache:
            self.dev = ss.ss_dev_cache_create(B, Hkv, self.nblk_host + reserve, self.capacity)
            assert ss.ss_dev_cache_total_slots(self.dev) == self.total_slots

    def step(self, t, q, events=None):
        if self.dev is not None:
            # nothing is waited for; misses are counted on the GPU (dev_miss_rows)
            ss.ss_decode_layer_dev(self.buffers, self.dev, t, q, self.out, None, events)
            self.last_n_miss = None
        else:
            self.last_n_miss = ss.ss_decode_layer(self.buffers, t, q, self.out, None, events)
        return self.out

    def reset_cache(self):
        """Empties the block cache: a fresh slot table over the same regions
        (host or GPU), so that the next step starts from a cold cache.  The
        HBM bytes stay as they are; every slot is empty, so none of them is
        read before a gather writes it."""
        torch.cuda.synchronize()
        cfg = self.cfg
        if self.dev is not None:
            ss.ss_dev_cache_destroy(self.dev)
            self.dev = None
            self.dev = ss.ss_dev_cache_create(cfg.B, cfg.Hkv, self.nblk_host + self.reserve, self.capacity)
        old = self.handle
        self.handle = ss.ss_cache_create(cfg.B, cfg.Hkv, self.nblk_host, self.capacity, cfg.record_bytes)
        ss.ss_cache_destroy(old)
        off = np.empty(self.units, np.int64)
        ss.ss_cache_region_offsets(self.handle, off)
        assert np.array_equal(off, self.cache_off_host)
        self.buffers.cache = self.handle

    def dev_miss_rows(self):
        """Device resolve: (per-unit miss counts, rows [units][k][4], error flags) of the last step."""
        counts, err = ss.ss_dev_cache_miss_counts(self.dev, self.units)
        rows = self.miss.view(self.units, self.cfg.k, 4).cpu().numpy()
        return counts, rows, err

    # ---------------------------------------------------------- save path
    def enable_save(self, threads=2, staging_slots=4, save_stream=None):
        """Appending and saving (FlashD2H) after each step: the open block of
        every unit in HBM, the token counts on the device, a saver into the
        pool's reserved blocks."""
        cfg = self.cfg
        assert self.reserve > 0, "build the layer with reserve > 0 blocks"
        B, Hkv = cfg.B, cfg.Hkv
        self.len_host = self.nblk_host.astype(np.int32) * cfg.blk  # sequences start block-aligned
        self.len_dev = _dev(self.len_host, np.int32)
        self.open = torch.empty(B, Hkv, cfg.record_bytes // 2, dtype=torch.int16, device="cuda")
        self.overflow = torch.zeros(1, dtype=torch.int32, device="cuda")
        self.pool_blocks = self.nblk_host + self.reserve
        self.saver = ss.ss_kv_saver_create(B, Hkv, cfg.blk, D, self.pool.host, self.pool_off_host,
                                           self.pool_blocks, 1, staging_slots, threads)
        self.save_stream = save_stream
        self.cache_blocks = self.nblk_host.copy()

    def step_with_save(self, t, q, new_kv, events=None):
        """One decode step of the layer with its save side.  The previous
        saves must be in the pool before this step's gather can read a block
        they completed, so they are waited for first; blocks filled so far
        become selectable; the step's new tokens (ready on the current
        stream) start their FlashD2H save, whose copy runs beside the decode
        when a save stream is set; decode; then the tokens are appended to
        the open blocks (metadata on a fill) for the next step."""
        cfg = self.cfg
        ss.ss_kv_save_wait(self.saver)
        nb = (self.len_host // cfg.blk).astype(np.int32)
        if np.any(nb != self.cache_blocks):
            ss.ss_cache_set_blocks(self.handle, nb)
            self.cache_blocks = nb
        if self.save_stream is not None:
            self.save_stream.wait_stream(torch.cuda.current_stream())
            new_kv.record_stream(self.save_stream)  # its memory is not reused before the copy ran
        ss.ss_kv_save(self.saver, new_kv, 1, self.len_host, self.save_stream)
        self.step(t, q, events)
        ss.ss_append_kv(new_kv, self.len_dev, self.nblk, cfg.B, cfg.Hkv, cfg.blk, D, self.nblk_max, self.open,
                        self.meta, self.overflow, meta_kind=self.meta_kind)
        self.len_host = self.len_host + 1
        return self.out

    def close(self):
        if self.dev is not None:
            ss.ss_dev_cache_destroy(self.dev)
            self.dev = None
        if self.saver:
            ss.ss_kv_saver_destroy(self.saver)
            self.saver = None
        if self.handle:
            ss.ss_cache_destroy(self.handle)
            self.handle = None
        if self._staging is not None:
            self.sel_h = self.slots_h = self.miss_h = None
            self._staging.close()
            self._staging = None


def cache_capacity(cfg, nblk):
    """Slots per unit: floor(cache_frac * blocks of the sequence), and never
    fewer than one step's selection, min(k, blocks), which attention needs in
    HBM at once (short sequences only; every benchmark sequence has more)."""
    n = np.asarray(nblk, np.int64)
    per_seq = np.maximum(np.floor(cfg.cache_frac * n.astype(np.float64)).astype(np.int64), np.minimum(cfg.k, n))
    return np.repeat(per_seq.astype(np.int32), cfg.Hkv)


def pool_layout(cfg, nblk, reserve=0):
    """Byte offsets of each unit's block array in a compact DRAM pool
    (nblk + reserve records per unit)."""
    per_unit = (np.repeat(np.asarray(nblk, np.int64), cfg.Hkv) + reserve) * cfg.record_bytes
    off = np.concatenate([[0], np.cumsum(per_unit)[:-1]]).astype(np.int64)
    return off, int(per_unit.sum())


def tent_parts(B, n):
    """Group sizes that grow then shrink (small first and last groups), so the
    link starts early and little work is left after the last gather."""
    n = max(1, min(n, B))
    w = np.array([min(i + 1, n - i) for i in range(n)], np.float64) ** 2
    sizes = np.maximum(1, np.floor(w / w.sum() * B)).astype(int)
    i = int(np.argmax(w))
    sizes[i] += B - int(sizes.sum())
    return [int(x) for x in sizes]


def ramp_parts(B, weights=(1, 2, 5, 10, 9, 4, 1)):
    """Group sizes that roughly double while the pipeline fills (each gather
    then lasts about as long as the next group's scoring, top-k and resolve, so
    the link does not idle between the first gathers), then shrink, so little
    work is left after the last gather.  For B = 64: 2, 4, 10, 20, 18, 8, 2."""
    w = np.asarray(weights, np.float64)
    n = min(len(w), B)
    if n < len(w):
        return tent_parts(B, n)
    sizes = np.maximum(1, np.round(w / w.sum() * B)).astype(int)
    i = int(np.argmax(w))
    sizes[i] += B - int(sizes.sum())
    if sizes[i] < 1:
        # small batches, where rounding up to one sequence per group overshoots:
        # one sequence each, the rest shared by largest remainder
        share = w / w.sum() * (B - n)
        sizes = 1 + np.floor(share).astype(int)
        order = np.argsort(-(share - np.floor(share)), kind="stable")
        sizes[order[:B - int(sizes.sum())]] += 1
    assert int(sizes.sum()) == B and sizes.min() >= 1
    return [int(x) for x in sizes]


def default_parts(B, schedule="layers"):
    """The decode step's automatic sequence groups.  One layer at a time
    ("layers"): seven ramp-shaped groups for batches of 40 or more, four
    (weights 2, 3, 5, 6) for 8 to 39, and otherwise one or two equal groups
    (per-group costs, a top-k launch and a resolve, favour few groups).
    Groups pipelined across layers ("groups"): the link fills and drains
    once per step, so the groups are equal, four of them (one per stream)."""
    if schedule == "groups":
        return max(1, min(4, B))
    if B >= 40:
        return ramp_parts(B)
    if B >= 8:
        return ramp_parts(B, weights=(2, 3, 5, 6))
    return max(1, min(2, round(B / 4)))


def build_hier_layer(cfg, seed, layer, pool, pool_base_off, nblk, progress=None, parts=1, reserve=0, meta_kind=0,
                     agg=0, dev_cache=False):
    """Draws one layer's KV per sequence on the GPU, builds its metadata in
    HBM and copies the records into `pool` at pool_base_off.  Returns the
    HierLayer (its pool offsets are relative to the pool base).  With
    reserve > 0 every unit has that many more pool records and metadata rows
    for blocks filled by appended tokens."""
    nblk = np.asarray(nblk, np.int32)
    sK, sV = gen.channel_scales(cfg.Hkv, D, seed, layer, "cuda")
    off, total = pool_layout(cfg, nblk, reserve)
    off = off + pool_base_off
    rows = (2,) if meta_kind == ss.SS_META_CUBOID else ()
    meta = torch.empty(cfg.B, cfg.Hkv, cfg.nblk_max + reserve, *rows, D, dtype=torch.int16, device="cuda")
    build = ss.ss_build_metadata if meta_kind == ss.SS_META_CUBOID else ss.ss_build_metadata_mean
    for b in range(cfg.B):
        n = int(nblk[b])
        if n == 0:
            continue
        rec, _ = gen.kv_records_seq(b, cfg.Hkv, n, cfg.blk, D, sK, sV, seed, layer, "cuda")
        rec = rec.contiguous()
        # metadata of this sequence, from the HBM copy of its records
        unit_off = _dev(np.arange(cfg.Hkv, dtype=np.int64) * n * cfg.record_bytes, np.int64)
        build(rec, unit_off, _dev([n], np.int32), 1, cfg.Hkv, cfg.nblk_max + reserve, cfg.blk, D, meta[b])
        for g in range(cfg.Hkv):
            start = int(off[b * cfg.Hkv + g])
            pool.t[start:start + n * cfg.record_bytes].copy_(rec[g].view(torch.uint8).reshape(-1))
        if progress and b % 16 == 15:
            progress(f"layer {layer}: {b + 1}/{cfg.B} sequences in the DRAM pool")
    torch.cuda.synchronize()
    L = HierLayer(cfg, nblk, cache_capacity(cfg, nblk), pool, off, meta, parts, reserve, meta_kind, agg, dev_cache)
    return L


def query_stream(cfg, seed, layer, steps, device="cuda"):
    """q for the warm-up step (index 0) and `steps` drifting steps after it."""
    q32, q = gen.query(cfg.B, cfg.Hq, D, seed, device, layer)
    qs = [(q32, q)]
    for s in range(1, steps + 1):
        q32, q = gen.drift(q32, cfg.drift, seed, layer, s)
        qs.append((q32, q))
    return qs


# Pinned host memory the pool may take.  A process can pin about 64 GiB on
# the MI355X hosts measured (the total over all allocation kinds); the rest
# of this allowance is left for step buffers.
POOL_BUDGET = 56 << 30


def decode_step_groups(layers, t, qs, events=None, between=None, stream=None):
    """Step t of every layer, the sequence groups pipelined across layers:
    group p's layer l+1 runs as soon as its layer l is attended.  With the
    device resolve (every layer built with dev_cache) ss_decode_step_dev,
    else ss_decode_step with the host resolve (each layer's last_n_miss is
    then set).  qs: per-layer query tensors.  Returns the per-layer outputs."""
    assert layers
    dev = [L.dev is not None for L in layers]
    assert all(dev) or not any(dev), "every layer resolves the same way"
    if all(dev):
        ss.ss_decode_step_dev([L.buffers for L in layers], [L.dev for L in layers], t, qs, [L.out for L in layers],
                              stream, between, events)
    else:
        n_miss = ss.ss_decode_step([L.buffers for L in layers], t, qs, [L.out for L in layers], stream, between,
                                   events)
        for L, m in zip(layers, n_miss):
            L.last_n_miss = int(m)
    return [L.out for L in layers]


def distinct_layers(cfg, nblk, budget=POOL_BUDGET):
    """How many layers get DRAM records of their own: all of them if the
    pool fits `budget`, else as many as fit.  Layer l then reads the records
    of layer l mod n (it still has its own queries, selections, HBM cache and
    misses, so the step's transfer volume is that of distinct layers)."""
    _, per_layer = pool_layout(cfg, nblk)
    if per_layer == 0:
        return cfg.layers
    return max(1, min(cfg.layers, budget // per_layer))


def build_hier_model(cfg, seed, nblk, flags=0, budget=POOL_BUDGET, progress=None, parts=1, dev_cache=False):
    """All cfg.layers layers over one DRAM pool (see distinct_layers).
    Returns (pool, layers, n_distinct)."""
    nblk = np.asarray(nblk, np.int32)
    n = distinct_layers(cfg, nblk, budget)
    _, per_layer = pool_layout(cfg, nblk)
    pool = HostPool(max(1, per_layer * n), flags)
    layers = []
    try:
        for l in range(cfg.layers):
            if l < n:
                L = build_hier_layer(cfg, seed, l, pool, l * per_layer, nblk, progress=progress, parts=parts,
                                     dev_cache=dev_cache)
            else:
                src = layers[l % n]
                L = HierLayer(cfg, nblk, src.capacity, pool, src.pool_off_host, src.meta, parts, dev_cache=dev_cache)
            layers.append(L)
    except BaseException:
        for L in layers:
            L.close()
        pool.close()
        raise
    return pool, layers, n


class PrefillExecutor:
    """Layer-segmented prefill of one prompt on the saving side (Section 3.4):
    the plan (ss_prefill_plan) runs the layers, or chunks of them, in
    batches.  A layer's new KV over the prompt, token-major [T][Hkv][2][d],
    lives in the one HBM buffer that every layer reuses (the model's
    projection would write it; it is drawn here).  Each plan item builds the
    metadata of the blocks its tokens complete, straight from that buffer,
    and saves its tokens to the DRAM pool with FlashD2H; when a layer ends,
    its tail tokens go to the layer's open block.  Every layer's metadata
    stays in HBM; only one layer's KV is there at a time."""

    def __init__(self, T, layers, Hkv, blk, max_inject, seed=0, meta_kind=0, threads=8, flags=0, same_kv=False):
        self.T, self.layers, self.Hkv, self.blk, self.max_inject = T, layers, Hkv, blk, max_inject
        self.seed, self.meta_kind = seed, meta_kind
        self.rb = 2 * blk * D * 2
        self.nfull = T // blk
        self.nmax = self.nfull + 1  # room for the block the tail will fill
        units = layers * Hkv
        self.pool = HostPool(units * self.nmax * self.rb, flags)
        self.pool_off = (np.arange(units, dtype=np.int64) * self.nmax * self.rb).reshape(layers, Hkv)
        self.items = ss.ss_prefill_plan(T, layers, max_inject)
        max_chunk = int((self.items[:, 3] - self.items[:, 2]).max())
        # one saver, pointed at each layer's records in turn
        self.saver = ss.ss_kv_saver_create(1, Hkv, blk, D, self.pool.host, self.pool_off[0],
                                           np.array([self.nmax], np.int32), max_chunk, 2, threads)
        self.same_kv = same_kv  # every layer's KV equal to layer 0's (timing the save side alone)
        rows = (2,) if meta_kind == ss.SS_META_CUBOID else ()
        self.meta = torch.zeros(layers, Hkv, self.nmax, *rows, D, dtype=torch.int16, device="cuda")
        self.buf = torch.empty(T, Hkv, 2, D, dtype=torch.bfloat16, device="cuda")  # one layer's KV
        self.open = torch.zeros(layers, Hkv, self.rb // 2, dtype=torch.int16, device="cuda")
        self.len_dev = torch.zeros(layers, dtype=torch.int32, device="cuda")
        self.nblk_dev = torch.zeros(layers, dtype=torch.int32, device="cuda")
        self.unit_off = _dev(np.arange(Hkv, dtype=np.int64) * 2 * D * 2, np.int64)
        self.scales = [gen.channel_scales(Hkv, D, seed, l, "cuda") for l in range(layers)]

    def layer_kv(self, l):
        sK, sV = self.scales[l]
        return gen.prefill_kv(self.T, self.Hkv, D, sK, sV, self.seed, l, "cuda")

    def run(self, progress=None):
        """Runs every batch of the plan; returns the number of batches."""
        T, blk, Hkv = self.T, self.blk, self.Hkv
        row = Hkv * 2 * D * 2  # bytes per token
        cur = -1
        for batch, l, t0, t1 in self.items.tolist():
            if l != cur:
                if cur < 0 or not self.same_kv:
                    self.buf.copy_(self.layer_kv(l))  # the layer's projection output
                if cur >= 0:
                    ss.ss_kv_saver_retarget(self.saver, self.pool_off[l], np.array([self.nmax], np.int32))
                cur = l
            j0, j1 = t0 // blk, t1 // blk  # blocks whose last token lies in [t0, t1)
            if j1 > j0:
                n = torch.tensor([j1 - j0], dtype=torch.int32, device="cuda")
                base = self.buf.data_ptr() + j0 * blk * row
                ss.ss_build_metadata_strided(base, self.unit_off, n, 1, Hkv, self.nmax, blk, D, blk * row, row,
                                             self.meta_kind, self.meta[l, :, j0:].data_ptr())
            ss.ss_kv_save(self.saver, self.buf.data_ptr() + t0 * row, t1 - t0, np.array([t0], np.int32))
            if t1 == T:
                # the tail of the prompt opens the layer's next block
                self.len_dev[l] = self.nfull * blk
                self.nblk_dev[l] = self.nfull
                for t in range(self.nfull * blk, T):
                    ss.ss_append_kv(self.buf[t], self.len_dev[l:l + 1], self.nblk_dev[l:l + 1], 1, Hkv, blk, D,
                                    self.nmax, self.open[l], self.meta[l], None, meta_kind=self.meta_kind)
                # the next layer's KV overwrites the buffer behind this layer's
                # copies (same stream); their host scatter continues meanwhile
            if progress:
                progress(batch, l, t0, t1)
        torch.cuda.synchronize()
        ss.ss_kv_save_wait(self.saver)
        return int(self.items[-1, 0]) + 1

    def close(self):
        if self.saver:
            ss.ss_kv_saver_destroy(self.saver)
            self.saver = None
        self.pool.close()

"""CPU oracle for SparseServe's decode-step hot path (arXiv 2509.24626).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline use this package; the product library never imports or loads it.

This module only marshals numpy arrays into the plain-C oracle in oracle.c
(fp64 arithmetic, plain loops) and returns numpy arrays.  bf16 tensors are
passed as uint16 bit patterns.  Memory given to the oracle must be host
memory (numpy arrays, or raw host addresses such as pinned host buffers).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

_c_i32p = ctypes.POINTER(ctypes.c_int32)
_c_i64p = ctypes.POINTER(ctypes.c_int64)


def lib():
    """Load liboracle.so, compiling it first if it is not there."""
    global _lib
    if _lib is None:
        other = os.environ.get("ORACLE_LIBRARY")  # another build of oracle.c (a sanitizer build)
        if other:
            _lib = load(other)
            return _lib
        if not os.path.exists(_build.LIB) or os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC):
            _build.build()
        _lib = load(_build.LIB)
    return _lib


def load(path):
    """Load an oracle shared object and declare its signatures."""
    L = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    L.oracle_build_metadata.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, sz, vp]
    L.oracle_score.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, vp]
    L.oracle_select.argtypes = [vp, vp, i32, i32, i32, i32, vp]
    L.oracle_lru_create.argtypes = [i32, i32, vp, vp]
    L.oracle_lru_create.restype = vp
    L.oracle_lru_destroy.argtypes = [vp]
    L.oracle_lru_step.argtypes = [vp, i64, vp, i32, vp, vp, i64, vp]
    L.oracle_lru_total_slots.argtypes = [vp]
    L.oracle_lru_total_slots.restype = i64
    L.oracle_lru_export.argtypes = [vp, vp, vp]
    L.oracle_gather.argtypes = [vp, i64, vp, vp, vp, vp, sz, i32]
    L.oracle_attention.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, ctypes.c_double, vp]
    L.oracle_append.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, vp, vp]
    L.oracle_save.argtypes = [vp, i32, vp, i32, i32, i32, i32, vp, vp, vp]
    L.oracle_build_metadata_mean.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, sz, vp]
    L.oracle_score_variant.argtypes = [vp, vp, i32, i32, vp, i32, i32, i32, i32, i32, vp]
    L.oracle_build_metadata_mean.restype = i32
    L.oracle_score_variant.restype = i32
    L.oracle_prefill_plan.argtypes = [i64, i32, i64, vp, i64]
    L.oracle_prefill_plan.restype = i64
    L.oracle_ws_decode.argtypes = [vp, i32, i32, i32, i32, i32, i32, sz]
    L.oracle_ws_decode.restype = i64
    L.oracle_ws_prefill.argtypes = [i64, i64, i64, i32, i32, i32, sz, i32]
    L.oracle_ws_prefill.restype = i64
    L.oracle_schedule.argtypes = [vp, i32, i64, vp, vp]
    for f in ("oracle_build_metadata", "oracle_score", "oracle_select", "oracle_lru_step",
              "oracle_gather", "oracle_attention", "oracle_append", "oracle_save", "oracle_schedule"):
        getattr(L, f).restype = i32
    return L


def _addr(x):
    """Host address of a numpy array or a raw integer address."""
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    if isinstance(x, int):
        return x
    raise TypeError(f"oracle needs host memory, got {type(x)}")


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with code {rc}")


def record_bytes(blk, d):
    """Bytes of one block record: K tile + channel-major V tile, bf16."""
    return 2 * blk * d * 2


class Oracle:
    """Bound oracle functions; `Oracle(lib_path)` loads a specific build."""

    def __init__(self, L=None):
        self.L = L if L is not None else lib()

    # O0
    def build_metadata(self, base, unit_off, nblk, B, Hkv, nblk_max, blk, d, meta=None):
        unit_off = _c(unit_off, np.int64)
        nblk = _c(nblk, np.int32)
        if meta is None:
            meta = np.zeros((B, Hkv, nblk_max, 2, d), dtype=np.uint16)
        _check(self.L.oracle_build_metadata(_addr(base), _addr(unit_off), _addr(nblk), B, Hkv, nblk_max,
                                            blk, d, record_bytes(blk, d), _addr(meta)), "build_metadata")
        return meta

    # O1
    def score(self, q, meta, nblk, Hq, Hkv, nblk_max, d):
        q = _c(q, np.uint16)
        meta = _c(meta, np.uint16)
        nblk = _c(nblk, np.int32)
        B = q.shape[0]
        S = np.empty((B, Hkv, nblk_max), dtype=np.float64)
        _check(self.L.oracle_score(_addr(q), _addr(meta), _addr(nblk), B, Hq, Hkv, nblk_max, d, _addr(S)), "score")
        return S

    # O2
    def select(self, S, nblk, k):
        S = _c(S, np.float64)
        nblk = _c(nblk, np.int32)
        B, Hkv, nblk_max = S.shape
        sel = np.empty((B, Hkv, k), dtype=np.int32)
        _check(self.L.oracle_select(_addr(S), _addr(nblk), B, Hkv, nblk_max, k, _addr(sel)), "select")
        return sel

    # O4
    def gather(self, miss, pool, pool_off, cache, cache_off, rec_bytes, Hkv):
        miss = _c(miss, np.int32).reshape(-1, 4)
        pool_off = _c(pool_off, np.int64)
        cache_off = _c(cache_off, np.int64)
        _check(self.L.oracle_gather(_addr(miss), miss.shape[0], _addr(pool), _addr(pool_off), _addr(cache),
                                    _addr(cache_off), rec_bytes, Hkv), "gather")

    # O5
    def attention(self, q, base, region_off, slots, Hkv, blk, scale=None):
        q = _c(q, np.uint16)
        region_off = _c(region_off, np.int64)
        slots = _c(slots, np.int32)
        B, Hq, d = q.shape
        k = slots.shape[-1]
        if scale is None:
            scale = 1.0 / np.sqrt(d)
        out = np.empty((B, Hq, d), dtype=np.float32)
        _check(self.L.oracle_attention(_addr(q), _addr(base), _addr(region_off), _addr(slots), B, Hq, Hkv, d,
                                       blk, k, float(scale), _addr(out)), "attention")
        return out

    # O6
    def append(self, new_kv, len_, nblk, blk, nblk_max, open_rec, meta):
        """new_kv uint16 [B][Hkv][2][d]; len_, nblk int32 [B] (updated in
        place); open_rec uint16 [B][Hkv][2*blk*d] and meta uint16
        [B][Hkv][nblk_max][2][d] (updated in place)."""
        new_kv = _c(new_kv, np.uint16)
        B, Hkv, _, d = new_kv.shape
        for a, dt in ((len_, np.int32), (nblk, np.int32), (open_rec, np.uint16), (meta, np.uint16)):
            assert isinstance(a, np.ndarray) and a.dtype == dt and a.flags.c_contiguous
        rc = self.L.oracle_append(_addr(new_kv), _addr(len_), _addr(nblk), B, Hkv, blk, d, nblk_max,
                                  _addr(open_rec), _addr(meta))
        if rc == 2:
            raise OverflowError("a filled block lies past nblk_max")
        _check(rc, "append")

    # O7
    def save(self, new_kv, len_, blk, pool, pool_off, pool_blocks):
        """new_kv uint16 [B][n_new][Hkv][2][d]; len_ int32 [B] (not changed);
        pool: host memory (array or address) updated in place."""
        new_kv = _c(new_kv, np.uint16)
        B, n_new, Hkv, _, d = new_kv.shape
        len_ = _c(len_, np.int32)
        pool_off = _c(pool_off, np.int64)
        pool_blocks = _c(pool_blocks, np.int32)
        rc = self.L.oracle_save(_addr(new_kv), n_new, _addr(len_), B, Hkv, blk, d, _addr(pool), _addr(pool_off),
                                _addr(pool_blocks))
        if rc == 2:
            raise OverflowError("a token lies past the unit's pool blocks")
        _check(rc, "save")

    # O11
    def build_metadata_mean(self, base, unit_off, nblk, B, Hkv, nblk_max, blk, d, meta=None):
        unit_off = _c(unit_off, np.int64)
        nblk = _c(nblk, np.int32)
        if meta is None:
            meta = np.zeros((B, Hkv, nblk_max, d), dtype=np.uint16)
        _check(self.L.oracle_build_metadata_mean(_addr(base), _addr(unit_off), _addr(nblk), B, Hkv, nblk_max, blk,
                                                 d, record_bytes(blk, d), _addr(meta)), "build_metadata_mean")
        return meta

    # O12
    def score_variant(self, q, meta, kind, agg, nblk, Hq, Hkv, nblk_max, d):
        """kind 0 cuboid / 1 mean-key metadata; agg 0 max / 1 sum over the group's heads."""
        q = _c(q, np.uint16)
        meta = _c(meta, np.uint16)
        nblk = _c(nblk, np.int32)
        B = q.shape[0]
        S = np.empty((B, Hkv, nblk_max), dtype=np.float64)
        _check(self.L.oracle_score_variant(_addr(q), _addr(meta), kind, agg, _addr(nblk), B, Hq, Hkv, nblk_max, d,
                                           _addr(S)), "score_variant")
        return S

    # O13
    def prefill_plan(self, T, layers, max_inject, cap=1 << 20):
        """Items int32 [n][4] = (batch, layer, tok_begin, tok_end)."""
        items = np.empty((cap, 4), np.int32)
        n = self.L.oracle_prefill_plan(T, layers, max_inject, _addr(items), cap)
        if n < 0:
            raise ValueError("oracle prefill_plan: invalid arguments")
        return items[:n].copy()

    # O8
    def ws_decode(self, sel_hist, w, record_bytes, fallback=0):
        """sel_hist int32 [m][layers][Hkv][k], oldest step first."""
        h = _c(sel_hist, np.int32)
        m, layers, Hkv, k = h.shape
        r = self.L.oracle_ws_decode(_addr(h), m, layers, Hkv, k, w, fallback, record_bytes)
        if r < 0:
            raise RuntimeError("oracle ws_decode failed")
        return int(r)

    # O9
    def ws_prefill(self, prompt, done, chunk, layers, Hkv, blk, record_bytes, layer_segmented):
        r = self.L.oracle_ws_prefill(prompt, done, chunk, layers, Hkv, blk, record_bytes, int(bool(layer_segmented)))
        if r < 0:
            raise RuntimeError("oracle ws_prefill failed")
        return int(r)

    # O10
    def schedule(self, ws, m_avl):
        ws = _c(ws, np.int64)
        admit = np.empty(ws.size, np.int32)
        used = ctypes.c_int64(0)
        _check(self.L.oracle_schedule(_addr(ws), ws.size, int(m_avl), _addr(admit), ctypes.addressof(used)),
               "schedule")
        return admit, used.value

    def lru(self, B, Hkv, nblk, cap):
        return LRU(self.L, B, Hkv, nblk, cap)


class LRU:
    """O3: the per-(sequence, KV head) LRU block cache of the oracle."""

    def __init__(self, L, B, Hkv, nblk, cap):
        self.L = L
        self.B, self.Hkv = B, Hkv
        nblk = _c(nblk, np.int32)
        cap = _c(cap, np.int32).reshape(-1)
        assert cap.size == B * Hkv
        self.cap = cap
        self.h = L.oracle_lru_create(B, Hkv, _addr(nblk), _addr(cap))
        if not self.h:
            raise MemoryError("oracle_lru_create")

    def __del__(self):
        if getattr(self, "h", None):
            self.L.oracle_lru_destroy(self.h)
            self.h = None

    def step(self, t, sel):
        sel = _c(sel, np.int32)
        k = sel.shape[-1]
        units = self.B * self.Hkv
        slots = np.empty((self.B, self.Hkv, k), dtype=np.int32)
        miss = np.empty((units * k, 4), dtype=np.int32)
        n = ctypes.c_int64(0)
        rc = self.L.oracle_lru_step(self.h, int(t), _addr(sel), k, _addr(slots), _addr(miss), units * k,
                                    ctypes.addressof(n))
        if rc == 3:
            raise OverflowError("selection larger than the unit's cache capacity")
        _check(rc, "lru_step")
        return slots, miss[: n.value].copy()

    def export(self):
        total = self.L.oracle_lru_total_slots(self.h)
        blocks = np.empty(total, dtype=np.int32)
        last = np.empty(total, dtype=np.int64)
        self.L.oracle_lru_export(self.h, _addr(blocks), _addr(last))
        return blocks, last

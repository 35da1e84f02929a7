"""ctypes binding of libsparseserve.so (include/sparseserve.h).

Argument marshalling only: every function here has the name of the C entry
point it calls and does no computation of its own.  Buffers may be torch
tensors (device or host), numpy arrays or raw integer addresses; streams
are torch streams, raw hipStream_t integers, or None for torch's current
stream.  A failing call raises SparseServeError with the library's message.
The library must be built (paper_2509_24626_amd/build.py); there is no
fallback path.
"""
import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# SS_LIBRARY names another build of the same library (the sanitizer builds
# of build_sanitized.py); there is still no fallback
LIB_PATH = os.environ.get("SS_LIBRARY") or os.path.join(_HERE, "_lib", "libsparseserve.so")

_lib = None

SS_OK = 0
SS_ERR_INVALID_ARG = 1
SS_ERR_UNSUPPORTED = 2
SS_ERR_CAPACITY = 3
SS_ERR_OOM = 4
SS_ERR_HIP = 5
SS_ERR_TIMEOUT = 6


class SparseServeError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"[{status}] {message}")
        self.status = status


_vp, _i32, _i64, _sz, _f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float


class ss_layer_buffers(ctypes.Structure):
    """Mirror of the C struct ss_layer_buffers (include/sparseserve.h)."""
    _fields_ = [("B", _i32), ("Hq", _i32), ("Hkv", _i32), ("d", _i32), ("blk", _i32), ("nblk_max", _i32),
                ("k", _i32), ("scale", _f32), ("meta", _vp), ("nblk_dev", _vp), ("pool", _vp),
                ("pool_off_dev", _vp), ("cache", _vp), ("cache_base", _vp), ("cache_off_dev", _vp),
                ("capacity_dev", _vp), ("slot_limit", _i32), ("scores", _vp), ("sel_dev", _vp),
                ("slots_dev", _vp), ("miss_dev", _vp), ("sel_host", _vp), ("slots_host", _vp),
                ("miss_host", _vp), ("miss_cap", _i64), ("attn_ws", _vp), ("attn_ws_bytes", _sz), ("parts", _i32),
                ("part_end", _vp), ("meta_kind", _i32), ("agg", _i32)]

_SIGNATURES = {
    "ss_abi_version": (_i32, []),
    "ss_status_string": (ctypes.c_char_p, [_i32]),
    "ss_last_error": (ctypes.c_char_p, []),
    "ss_host_alloc_mapped": (_i32, [_sz, ctypes.c_uint, _vp, _vp]),
    "ss_host_free": (_i32, [_vp]),
    "ss_time_next_kernel": (_i32, [_vp, _vp]),
    "ss_build_metadata": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "ss_score_blocks": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "ss_select_topk": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp]),
    "ss_score_topk": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp]),
    "ss_cache_create": (_i32, [_i32, _i32, _vp, _vp, _sz, _vp]),
    "ss_cache_destroy": (None, [_vp]),
    "ss_cache_total_slots": (_i64, [_vp]),
    "ss_cache_region_offsets": (_i32, [_vp, _vp]),
    "ss_cache_set_threads": (_i32, [_vp, _i32]),
    "ss_cache_resolve": (_i32, [_vp, _i64, _vp, _i32, _vp, _vp, _i64, _vp]),
    "ss_cache_resolve_range": (_i32, [_vp, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _i64, _vp]),
    "ss_cache_export": (_i32, [_vp, _vp, _vp]),
    "ss_gather_blocks": (_i32, [_vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _sz, _vp]),
    "ss_sparse_attention_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32]),
    "ss_score_topk_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32]),
    "ss_sparse_attention": (_i32, [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _f32, _vp,
                                   _vp, _sz, _vp]),
    "ss_decode_layer": (_i32, [ctypes.POINTER(ss_layer_buffers), _i64, _vp, _vp, _vp, _vp, _vp]),
    "ss_cache_set_blocks": (_i32, [_vp, _vp]),
    "ss_append_kv": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _i32, _vp, _vp]),
    "ss_build_metadata_mean": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "ss_score_blocks_variant": (_i32, [_vp, _vp, _i32, _i32, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp]),
    "ss_kv_saver_create": (_i32, [_i32, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _i32, _i32, _vp]),
    "ss_kv_saver_destroy": (None, [_vp]),
    "ss_kv_save": (_i32, [_vp, _vp, _i32, _vp, _vp]),
    "ss_kv_save_wait": (_i32, [_vp]),
    "ss_kv_saver_retarget": (_i32, [_vp, _vp, _vp]),
    "ss_ws_create": (_i32, [_i32, _i32, _i32, _sz, _vp]),
    "ss_ws_destroy": (None, [_vp]),
    "ss_ws_observe": (_i32, [_vp, _i32, _i64, _vp, _i32, _vp, _i32]),
    "ss_ws_decode_bytes": (_i32, [_vp, _vp, _i32, _vp, _vp]),
    "ss_ws_forget": (_i32, [_vp, _i64]),
    "ss_ws_prefill_bytes": (_i64, [_i64, _i64, _i64, _i32, _i32, _i32, _sz, _i32]),
    "ss_schedule_batch": (_i32, [_vp, _i32, _i64, _vp, _vp]),
    "ss_build_metadata_strided": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i64, _i64, _i32, _vp, _vp]),
    "ss_prefill_plan": (_i32, [_i64, _i32, _i64, _vp, _i64, _vp]),
    "ss_dev_cache_create": (_i32, [_i32, _i32, _vp, _vp, _vp, _vp]),
    "ss_dev_cache_destroy": (None, [_vp]),
    "ss_dev_cache_total_slots": (_i64, [_vp]),
    "ss_dev_cache_resolve": (_i32, [_vp, _i64, _i32, _i32, _vp, _i32, _vp, _vp, _vp, _vp]),
    "ss_dev_cache_miss_counts": (_i32, [_vp, _vp, _vp]),
    "ss_dev_cache_export": (_i32, [_vp, _vp, _vp]),
    "ss_dev_cache_total_misses": (_i32, [_vp, _vp]),
    "ss_decode_layer_dev": (_i32, [ctypes.POINTER(ss_layer_buffers), _vp, _i64, _vp, _vp, _vp, _vp]),
    "ss_set_host_wait_timeout": (_i32, [_i64]),
    "ss_decode_step_dev": (_i32, [_vp, _vp, _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp]),
    "ss_decode_step": (_i32, [_vp, _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "ss_sparse_attention_static": (_i32, [_vp, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _f32,
                                          _vp, _vp]),
}


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run paper_2509_24626_amd/build.py (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def exported_names():
    return list(_SIGNATURES)


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):  # torch.Tensor
        return x.data_ptr()
    if hasattr(x, "ctypes"):  # numpy.ndarray
        return x.ctypes.data
    raise TypeError(f"cannot pass {type(x)} as a buffer")


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(status):
    if status != SS_OK:
        raise SparseServeError(status, lib().ss_last_error().decode())


def ss_abi_version():
    return lib().ss_abi_version()


def ss_status_string(status):
    return lib().ss_status_string(status).decode()


def ss_last_error():
    return lib().ss_last_error().decode()


def ss_host_alloc_mapped(nbytes, flags=0):
    """Returns (host_address, device_address)."""
    h, d = ctypes.c_void_p(), ctypes.c_void_p()
    _check(lib().ss_host_alloc_mapped(nbytes, flags, ctypes.byref(h), ctypes.byref(d)))
    return h.value or 0, d.value or 0


def ss_host_free(host_address):
    _check(lib().ss_host_free(host_address))


def ss_time_next_kernel(start_event=None, stop_event=None):
    """Attach timing events to the next kernel this thread launches through
    the library (torch.cuda.Event objects or raw hipEvent_t values)."""
    ev = lambda e: None if e is None else (e if isinstance(e, int) else e.cuda_event)
    _check(lib().ss_time_next_kernel(ev(start_event), ev(stop_event)))


def ss_build_metadata(kv_base, unit_off, nblk, B, Hkv, nblk_max, blk, d, meta, stream=None):
    _check(lib().ss_build_metadata(_ptr(kv_base), _ptr(unit_off), _ptr(nblk), B, Hkv, nblk_max, blk, d, _ptr(meta),
                                   _stream(stream)))


def ss_score_blocks(q, meta, nblk, B, Hq, Hkv, nblk_max, d, scores, stream=None):
    _check(lib().ss_score_blocks(_ptr(q), _ptr(meta), _ptr(nblk), B, Hq, Hkv, nblk_max, d, _ptr(scores),
                                 _stream(stream)))


def ss_select_topk(scores, nblk, B, Hkv, nblk_max, k, sel, stream=None):
    _check(lib().ss_select_topk(_ptr(scores), _ptr(nblk), B, Hkv, nblk_max, k, _ptr(sel), _stream(stream)))


def ss_score_topk(q, meta, nblk, B, Hq, Hkv, nblk_max, d, k, scores, sel, stream=None):
    _check(lib().ss_score_topk(_ptr(q), _ptr(meta), _ptr(nblk), B, Hq, Hkv, nblk_max, d, k, _ptr(scores), _ptr(sel),
                               _stream(stream)))


def ss_cache_create(B, Hkv, nblk, capacity, record_bytes):
    """nblk: host int32 [B]; capacity: host int32 [B*Hkv]. Returns a handle."""
    h = ctypes.c_void_p()
    _check(lib().ss_cache_create(B, Hkv, _ptr(nblk), _ptr(capacity), record_bytes, ctypes.byref(h)))
    return h.value


def ss_cache_destroy(handle):
    lib().ss_cache_destroy(handle)


def ss_cache_total_slots(handle):
    return lib().ss_cache_total_slots(handle)


def ss_cache_region_offsets(handle, off):
    _check(lib().ss_cache_region_offsets(handle, _ptr(off)))


def ss_cache_set_threads(handle, n):
    _check(lib().ss_cache_set_threads(handle, n))


def ss_cache_resolve(handle, step, sel, k, slots, miss, miss_cap):
    """Host arrays; returns the number of miss rows written."""
    n = ctypes.c_int64(0)
    _check(lib().ss_cache_resolve(handle, step, _ptr(sel), k, _ptr(slots), _ptr(miss), miss_cap, ctypes.byref(n)))
    return n.value


def ss_cache_resolve_range(handle, step, b_begin, b_end, sel, k, slots, miss, miss_cap):
    """Host arrays holding the rows of sequences [b_begin, b_end); returns the miss rows written."""
    n = ctypes.c_int64(0)
    _check(lib().ss_cache_resolve_range(handle, step, b_begin, b_end, _ptr(sel), k, _ptr(slots), _ptr(miss),
                                        miss_cap, ctypes.byref(n)))
    return n.value


def ss_cache_export(handle, slot_block, slot_last):
    _check(lib().ss_cache_export(handle, _ptr(slot_block), _ptr(slot_last)))


def ss_gather_blocks(miss, n_miss, pool_base, pool_off, cache_base, cache_off, nblk, capacity, B, Hkv, record_bytes,
                     stream=None):
    _check(lib().ss_gather_blocks(_ptr(miss), n_miss, _ptr(pool_base), _ptr(pool_off), _ptr(cache_base),
                                  _ptr(cache_off), _ptr(nblk), _ptr(capacity), B, Hkv, record_bytes, _stream(stream)))


def ss_sparse_attention_workspace(B, Hq, Hkv, d, blk, k):
    return lib().ss_sparse_attention_workspace(B, Hq, Hkv, d, blk, k)


def ss_score_topk_workspace(B, Hq, Hkv, nblk_max, d, k):
    return int(lib().ss_score_topk_workspace(B, Hq, Hkv, nblk_max, d, k))


def ss_sparse_attention(q, kv_base, region_off, slots, capacity, slot_limit, B, Hq, Hkv, d, blk, k, scale, out,
                        workspace, ws_bytes, stream=None):
    _check(lib().ss_sparse_attention(_ptr(q), _ptr(kv_base), _ptr(region_off), _ptr(slots), _ptr(capacity),
                                     slot_limit, B, Hq, Hkv, d, blk, k, float(scale), _ptr(out), _ptr(workspace),
                                     ws_bytes, _stream(stream)))


def ss_sparse_attention_static(q, kv_base, region_off, slots, capacity, slot_limit, B, Hq, Hkv, d, blk, k, scale,
                               out, stream=None):
    _check(lib().ss_sparse_attention_static(_ptr(q), _ptr(kv_base), _ptr(region_off), _ptr(slots), _ptr(capacity),
                                            slot_limit, B, Hq, Hkv, d, blk, k, float(scale), _ptr(out),
                                            _stream(stream)))


def ss_decode_layer(buffers, step, q, out, stream=None, events=None):
    """buffers: an ss_layer_buffers; events: None or 7*parts raw hipEvent_t
    handles.  Returns the number of blocks gathered."""
    n = ctypes.c_int64(0)
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*events)
    _check(lib().ss_decode_layer(ctypes.byref(buffers), step, _ptr(q), _ptr(out), _stream(stream), ev,
                                 ctypes.byref(n)))
    return n.value


def ss_set_host_wait_timeout(ms):
    _check(lib().ss_set_host_wait_timeout(int(ms)))


def ss_cache_set_blocks(handle, nblk):
    import numpy as np
    nblk = np.ascontiguousarray(nblk, dtype=np.int32)
    _check(lib().ss_cache_set_blocks(handle, nblk.ctypes.data))


def ss_append_kv(new_kv, len_dev, nblk_dev, B, Hkv, blk, d, nblk_max, open_blocks, meta, overflow=None, stream=None,
                 meta_kind=0):
    _check(lib().ss_append_kv(_ptr(new_kv), _ptr(len_dev), _ptr(nblk_dev), B, Hkv, blk, d, nblk_max,
                              _ptr(open_blocks), _ptr(meta), meta_kind, _ptr(overflow), _stream(stream)))


SS_META_CUBOID, SS_META_MEAN = 0, 1
SS_AGG_MAX, SS_AGG_SUM = 0, 1


def ss_build_metadata_mean(kv_base, unit_off, nblk, B, Hkv, nblk_max, blk, d, meta, stream=None):
    _check(lib().ss_build_metadata_mean(_ptr(kv_base), _ptr(unit_off), _ptr(nblk), B, Hkv, nblk_max, blk, d,
                                        _ptr(meta), _stream(stream)))


def ss_score_blocks_variant(q, meta, meta_kind, agg, nblk, B, Hq, Hkv, nblk_max, d, scores, stream=None):
    _check(lib().ss_score_blocks_variant(_ptr(q), _ptr(meta), meta_kind, agg, _ptr(nblk), B, Hq, Hkv, nblk_max, d,
                                         _ptr(scores), _stream(stream)))


def ss_kv_saver_create(B, Hkv, blk, d, pool_host, pool_off, pool_blocks, max_new_tokens=1, staging_slots=4,
                       threads=2):
    """pool_host: host address; pool_off int64 [B*Hkv], pool_blocks int32 [B] (numpy)."""
    import numpy as np
    pool_off = np.ascontiguousarray(pool_off, dtype=np.int64)
    pool_blocks = np.ascontiguousarray(pool_blocks, dtype=np.int32)
    h = ctypes.c_void_p()
    _check(lib().ss_kv_saver_create(B, Hkv, blk, d, pool_host, pool_off.ctypes.data, pool_blocks.ctypes.data,
                                    max_new_tokens, staging_slots, threads, ctypes.byref(h)))
    return h.value


def ss_kv_saver_destroy(saver):
    lib().ss_kv_saver_destroy(saver)


def ss_kv_save(saver, new_kv, n_new, len_host, stream=None):
    import numpy as np
    len_host = np.ascontiguousarray(len_host, dtype=np.int32)
    _check(lib().ss_kv_save(saver, _ptr(new_kv), n_new, len_host.ctypes.data, _stream(stream)))


def ss_kv_save_wait(saver):
    _check(lib().ss_kv_save_wait(saver))


def ss_ws_create(layers, Hkv, window, record_bytes):
    h = ctypes.c_void_p()
    _check(lib().ss_ws_create(layers, Hkv, window, record_bytes, ctypes.byref(h)))
    return h.value


def ss_ws_destroy(ws):
    lib().ss_ws_destroy(ws)


def ss_ws_observe(ws, layer, step, req_ids, sel):
    """req_ids int64 [B]; sel int32 [B][Hkv][k] (host)."""
    import numpy as np
    req_ids = np.ascontiguousarray(req_ids, dtype=np.int64)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    _check(lib().ss_ws_observe(ws, layer, step, req_ids.ctypes.data, req_ids.size, sel.ctypes.data, sel.shape[-1]))


def ss_ws_decode_bytes(ws, req_ids, fallback_blocks=None):
    import numpy as np
    req_ids = np.ascontiguousarray(req_ids, dtype=np.int64)
    out = np.empty(req_ids.size, np.int64)
    fb = None if fallback_blocks is None else np.ascontiguousarray(fallback_blocks, dtype=np.int32)
    _check(lib().ss_ws_decode_bytes(ws, req_ids.ctypes.data, req_ids.size, None if fb is None else fb.ctypes.data,
                                    out.ctypes.data))
    return out


def ss_ws_forget(ws, req_id):
    _check(lib().ss_ws_forget(ws, req_id))


def ss_ws_prefill_bytes(prompt_tokens, done_tokens, chunk_tokens, layers, Hkv, blk, record_bytes, layer_segmented):
    r = lib().ss_ws_prefill_bytes(prompt_tokens, done_tokens, chunk_tokens, layers, Hkv, blk, record_bytes,
                                  int(bool(layer_segmented)))
    if r < 0:
        raise SparseServeError(SS_ERR_INVALID_ARG, "ss_ws_prefill_bytes: invalid arguments")
    return r


def ss_schedule_batch(ws_bytes, m_avl):
    """Returns (admit int32 [n], m_used)."""
    import numpy as np
    ws_bytes = np.ascontiguousarray(ws_bytes, dtype=np.int64)
    admit = np.empty(ws_bytes.size, np.int32)
    used = ctypes.c_int64(0)
    _check(lib().ss_schedule_batch(ws_bytes.ctypes.data, ws_bytes.size, m_avl, admit.ctypes.data,
                                   ctypes.byref(used)))
    return admit, used.value


def ss_build_metadata_strided(kv_base, unit_off, nblk, B, Hkv, nblk_max, blk, d, block_stride, row_stride, meta_kind,
                              meta, stream=None):
    _check(lib().ss_build_metadata_strided(_ptr(kv_base), _ptr(unit_off), _ptr(nblk), B, Hkv, nblk_max, blk, d,
                                           block_stride, row_stride, meta_kind, _ptr(meta), _stream(stream)))


def ss_prefill_plan(T, layers, max_inject):
    """Returns int32 [n][4] rows (batch, layer, tok_begin, tok_end)."""
    import numpy as np
    valid = T > 0 and layers > 0 and max_inject > 0  # otherwise the library reports the error
    per_layer = 1 if not valid or T <= max_inject else -(-T // max_inject)
    cap = max(1, per_layer * max(layers, 0))
    items = np.empty((cap, 4), np.int32)
    n = ctypes.c_int64(0)
    _check(lib().ss_prefill_plan(T, layers, max_inject, items.ctypes.data, cap, ctypes.byref(n)))
    return items[:n.value].copy()


def ss_kv_saver_retarget(saver, pool_off, pool_blocks):
    import numpy as np
    pool_off = np.ascontiguousarray(pool_off, dtype=np.int64)
    pool_blocks = np.ascontiguousarray(pool_blocks, dtype=np.int32)
    _check(lib().ss_kv_saver_retarget(saver, pool_off.ctypes.data, pool_blocks.ctypes.data))


def ss_dev_cache_create(B, Hkv, table_room, capacity, stream=None):
    import numpy as np
    table_room = np.ascontiguousarray(table_room, dtype=np.int32)
    capacity = np.ascontiguousarray(capacity, dtype=np.int32).reshape(-1)
    h = ctypes.c_void_p()
    _check(lib().ss_dev_cache_create(B, Hkv, table_room.ctypes.data, capacity.ctypes.data, _stream(stream),
                                     ctypes.byref(h)))
    return h.value


def ss_dev_cache_destroy(handle):
    lib().ss_dev_cache_destroy(handle)


def ss_dev_cache_total_slots(handle):
    return lib().ss_dev_cache_total_slots(handle)


def ss_dev_cache_resolve(handle, step, b_begin, b_end, sel, k, nblk, slots, miss, stream=None):
    _check(lib().ss_dev_cache_resolve(handle, step, b_begin, b_end, _ptr(sel), k, _ptr(nblk), _ptr(slots), _ptr(miss),
                                      _stream(stream)))


def ss_dev_cache_miss_counts(handle, units):
    """Returns (counts int32 [units], error flags)."""
    import numpy as np
    counts = np.empty(units, np.int32)
    err = ctypes.c_int32(0)
    _check(lib().ss_dev_cache_miss_counts(handle, counts.ctypes.data, ctypes.byref(err)))
    return counts, err.value


def ss_dev_cache_export(handle, slot_block, slot_last):
    _check(lib().ss_dev_cache_export(handle, _ptr(slot_block), _ptr(slot_last)))


def ss_decode_layer_dev(buffers, handle, step, q, out, stream=None, events=None):
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*events)
    _check(lib().ss_decode_layer_dev(ctypes.byref(buffers), handle, step, _ptr(q), _ptr(out), _stream(stream), ev))


# int (*)(void *ctx, int layer, int b_begin, int b_end, void *stream)
SS_BETWEEN_FN = ctypes.CFUNCTYPE(_i32, _vp, _i32, _i32, _i32, _vp)


def _addr_array(xs):
    if isinstance(xs, ctypes.Array):
        return xs
    return (ctypes.c_void_p * len(xs))(*[_ptr(x) if not isinstance(x, ss_layer_buffers) else ctypes.addressof(x)
                                         for x in xs])


def _between_cb(between, raised):
    if between is None:
        return None

    def _cb(_ctx, layer, b0, b1, stream_handle):
        try:
            between(layer, b0, b1, stream_handle)
            return SS_OK
        except BaseException as e:  # noqa: BLE001 -- re-raised after the call
            raised.append(e)
            return SS_ERR_INVALID_ARG
    return SS_BETWEEN_FN(_cb)


def ss_decode_step(buffers, step, qs, outs, stream=None, between=None, events=None):
    """The step over len(buffers) layers with the host resolve (each layer's
    buffers.cache), groups pipelined across layers.  Arguments as
    ss_decode_step_dev.  Returns each layer's missed blocks (numpy int64)."""
    import numpy as np
    n = len(buffers)
    arrs = [_addr_array(buffers), _addr_array(qs), _addr_array(outs)]
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*events)
    raised = []
    cb = _between_cb(between, raised)
    n_miss = np.zeros(max(n, 1), np.int64)
    st = lib().ss_decode_step(arrs[0], n, step, arrs[1], arrs[2], _stream(stream),
                              ctypes.cast(cb, ctypes.c_void_p) if cb is not None else None, None, ev,
                              n_miss.ctypes.data)
    if raised:
        raise raised[0]
    _check(st)
    return n_miss[:n]


def ss_decode_step_dev(buffers, handles, step, qs, outs, stream=None, between=None, events=None):
    """The step over len(buffers) layers, groups pipelined across layers.
    buffers: ss_layer_buffers per layer; handles: ss_dev_cache per layer;
    qs, outs: per-layer tensors or device addresses (or prebuilt ctypes
    arrays of addresses).  between: None, or a callable (layer, b_begin,
    b_end, stream_handle) that enqueues on that HIP stream the work producing
    the group's next-layer queries; an exception it raises stops the call and
    is raised again here.  events: None or 2*layers*groups raw hipEvent_t
    handles (None entries allowed)."""
    n = len(buffers)
    arrs = [_addr_array(buffers), _addr_array(handles), _addr_array(qs), _addr_array(outs)]
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*events)
    raised = []
    cb = _between_cb(between, raised)
    st = lib().ss_decode_step_dev(arrs[0], arrs[1], n, step, arrs[2], arrs[3], _stream(stream),
                                  ctypes.cast(cb, ctypes.c_void_p) if cb is not None else None, None, ev)
    if raised:
        raise raised[0]
    _check(st)


def ss_dev_cache_total_misses(handle):
    n = ctypes.c_int64(0)
    _check(lib().ss_dev_cache_total_misses(handle, ctypes.byref(n)))
    return n.value

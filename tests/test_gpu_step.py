"""The decode step with the sequence groups pipelined across layers (one
call per step: ss_decode_step_dev with the slot tables resolved on the GPU,
ss_decode_step with them resolved on host threads) against each layer's
step in turn (ss_decode_layer_dev, ss_decode_layer), whose parity with the
oracle the hierarchical tests establish unit by unit.  Both take the same kernels over the same groups,
so every layer's selection, slots and attention output must be identical
bit for bit, and so must the block caches after the run.

The between-layer callback stands for the rest of the model's layer: it
makes each group's next-layer queries from its attention output on the
group's stream.  Run per layer, the same arithmetic runs on the whole batch
after each layer's call.  Equal results show that the callback's work is
ordered after the group's attention and before its next scoring.  The
full-size run of the 32-layer workload against the oracle is in
test_gpu_hier.py (schedule "groups")."""
import dataclasses

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


def small_cfg(B=12, layers=4):
    """The 32-layer workload's shape, shortened: ragged lengths U[1k, 8k],
    k = 128 blocks (sequences shorter than that select all their blocks),
    30% cache per layer, 3 drifting steps."""
    return dataclasses.replace(synth.get(3), name=f"layers{layers}-b{B}-ragged1k8k-blk16-k128-cache30", B=B,
                               layers=layers, ctx_range=(1024, 8192), steps=3)


def build(cfg, seed, parts, dev=True):
    from paper_2509_24626_amd import harness as H
    nblk = (synth.gen.lengths(cfg, seed) // cfg.blk).astype(np.int32)
    pool, layers, n = H.build_hier_model(cfg, seed, nblk, parts=parts, dev_cache=dev)
    assert n == cfg.layers
    return pool, layers


def close(pool, layers):
    for L in layers:
        L.close()
    pool.close()


def next_query(base, out):
    """The stand-in for the rest of a layer: bf16(base + out / 2)."""
    return (base.float() + 0.5 * out).to(torch.bfloat16)


def _stream_of(handle):
    return torch.cuda.ExternalStream(handle) if handle else torch.cuda.default_stream()


@pytest.mark.parametrize("B,layers,parts,resolve", [
    (12, 4, 1, "device"), (12, 4, 4, "device"), (12, 4, 6, "device"), (12, 4, [2, 3, 5, 2], "device"),
    (13, 3, 4, "device"), (12, 1, 4, "device"),
    (12, 4, 1, "host"), (12, 4, 4, "host"), (12, 4, 6, "host"), (12, 4, [2, 3, 5, 2], "host"), (13, 3, 4, "host"),
    (12, 1, 4, "host")])
def test_groups_schedule_equals_layer_by_layer(ss, B, layers, parts, resolve):
    """Groups pipelined across layers, with the between-layer callback, give
    the per-layer path's results bit for bit at every step and layer, with
    the slot tables on the GPU or on the host; 6 groups share the four
    streams, the uneven groups put groups of different sizes on one stream's
    attention workspace, 13 sequences do not divide into the groups evenly,
    and a single layer makes no callback."""
    from paper_2509_24626_amd import harness as H
    cfg, seed = small_cfg(B=B, layers=layers), 3
    dev = resolve == "device"
    pa, A = build(cfg, seed, parts, dev)
    pb, Bm = build(cfg, seed, parts, dev)
    try:
        base = [H.query_stream(cfg, seed, l, cfg.steps) for l in range(cfg.layers)]
        qa = [torch.empty_like(base[l][0][1]) for l in range(cfg.layers)]
        qb = [torch.empty_like(base[l][0][1]) for l in range(cfg.layers)]
        calls = []
        for t in range(cfg.steps + 1):
            print(f"[gpu] parts {parts} step {t}", flush=True)
            for l, L in enumerate(A):
                qa[l].copy_(base[0][t][1] if l == 0 else next_query(base[l][t][1], A[l - 1].out))
                L.step(t, qa[l])

            def between(l, b0, b1, handle, t=t):
                calls.append((l, b0, b1))
                with torch.cuda.stream(_stream_of(handle)):
                    qb[l + 1][b0:b1].copy_(next_query(base[l + 1][t][1][b0:b1], Bm[l].out[b0:b1]))

            qb[0].copy_(base[0][t][1])
            H.decode_step_groups(Bm, t, qb, between=between)
            torch.cuda.synchronize()
            for l in range(cfg.layers):
                where = f"step {t} layer {l}"
                assert torch.equal(A[l].sel, Bm[l].sel), where
                assert torch.equal(A[l].slots, Bm[l].slots), where
                assert torch.equal(qa[l], qb[l]), where
                assert torch.equal(A[l].out, Bm[l].out), where
                if dev:
                    ca, _, ea = A[l].dev_miss_rows()
                    cb, _, eb = Bm[l].dev_miss_rows()
                    assert ea == eb == 0 and np.array_equal(ca, cb), where
                else:  # the layer's miss rows, compact in group order on both paths
                    n = A[l].last_n_miss
                    assert n == Bm[l].last_n_miss, where
                    assert np.array_equal(A[l].miss_h.numpy()[:n], Bm[l].miss_h.numpy()[:n]), where
        P = Bm[0].parts
        ends = np.cumsum(Bm[0].part_sizes)
        want = [(l, int(e - n), int(e)) for l in range(cfg.layers - 1) for e, n in zip(ends, Bm[0].part_sizes)]
        assert calls == want * (cfg.steps + 1)
        assert len(want) == (cfg.layers - 1) * P
        for l in range(cfg.layers):
            n = A[l].total_slots
            sa, la = np.empty(n, np.int32), np.empty(n, np.int64)
            sb, lb = np.empty(n, np.int32), np.empty(n, np.int64)
            if dev:
                ss.ss_dev_cache_export(A[l].dev, sa, la)
                ss.ss_dev_cache_export(Bm[l].dev, sb, lb)
                assert ss.ss_dev_cache_total_misses(A[l].dev) == ss.ss_dev_cache_total_misses(Bm[l].dev)
            else:
                ss.ss_cache_export(A[l].handle, sa, la)
                ss.ss_cache_export(Bm[l].handle, sb, lb)
            assert np.array_equal(sa, sb) and np.array_equal(la, lb), f"cache of layer {l}"
    finally:
        close(pa, A)
        close(pb, Bm)


@pytest.mark.parametrize("resolve", ["device", "host"])
def test_groups_schedule_without_callback_and_events(ss, resolve):
    """Without a callback the queries are taken as given: the results equal
    the per-layer path's; the gather timing events of every (layer, group)
    complete, each interval inside the step."""
    from paper_2509_24626_amd import harness as H
    cfg, seed = small_cfg(B=16, layers=3), 5
    pa, A = build(cfg, seed, 4, resolve == "device")
    pb, Bm = build(cfg, seed, 4, resolve == "device")
    try:
        qs = [H.query_stream(cfg, seed, l, cfg.steps) for l in range(cfg.layers)]
        P = Bm[0].parts
        for t in range(cfg.steps + 1):
            for l, L in enumerate(A):
                L.step(t, qs[l][t][1])
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * cfg.layers * P + 2)]
            for e in ev:  # creates the underlying events (the library records the gathers' on their dispatch)
                e.record()
            torch.cuda.synchronize()
            ev[-2].record()
            H.decode_step_groups(Bm, t, [qs[l][t][1] for l in range(cfg.layers)],
                                 events=[e.cuda_event for e in ev[:-2]])
            ev[-1].record()
            torch.cuda.synchronize()
            span = ev[-2].elapsed_time(ev[-1])
            for j in range(cfg.layers * P):
                a, b = ev[-2].elapsed_time(ev[2 * j]), ev[-2].elapsed_time(ev[2 * j + 1])
                assert 0 <= a <= b <= span, (t, j, a, b, span)
            for l in range(cfg.layers):
                assert torch.equal(A[l].slots, Bm[l].slots) and torch.equal(A[l].out, Bm[l].out), (t, l)
    finally:
        close(pa, A)
        close(pb, Bm)


@pytest.mark.parametrize("resolve", ["device", "host"])
def test_groups_schedule_callback_error_and_checks(ss, resolve):
    """An exception in the callback stops the call and is raised; what was
    enqueued finishes, the caller's stream is ordered after it, and the next
    step runs.  A step call made from inside the callback is refused.  Layers
    of different shapes and a workspace short of one region per stream are
    rejected before anything is enqueued."""
    from paper_2509_24626_amd import harness as H
    cfg, seed = small_cfg(layers=3), 7
    dev = resolve == "device"
    pool, Ls = build(cfg, seed, 4, dev)
    try:
        qs = [H.query_stream(cfg, seed, l, cfg.steps) for l in range(cfg.layers)]

        def boom(l, b0, b1, handle):
            if l == 1 and b0 > 0:
                raise RuntimeError("callback stopped the step")

        with pytest.raises(RuntimeError, match="callback stopped"):
            H.decode_step_groups(Ls, 0, [qs[l][0][1] for l in range(cfg.layers)], between=boom)
        torch.cuda.synchronize()

        def reenter(l, b0, b1, handle):  # a step call from inside the callback is refused, not deadlocked
            Ls[0].step(1, qs[0][1][1])

        with pytest.raises(ss.SparseServeError, match="between-layer callback"):
            H.decode_step_groups(Ls, 0, [qs[l][0][1] for l in range(cfg.layers)], between=reenter)
        torch.cuda.synchronize()
        H.decode_step_groups(Ls, 1, [qs[l][1][1] for l in range(cfg.layers)])
        torch.cuda.synchronize()
        if dev:
            for L in Ls:
                _, _, err = L.dev_miss_rows()
                assert err == 0

        def call(bufs):
            q2, o2 = [qs[0][2][1], qs[1][2][1]], [Ls[0].out, Ls[1].out]
            if dev:
                ss.ss_decode_step_dev(bufs, [Ls[0].dev, Ls[1].dev], 2, q2, o2)
            else:
                ss.ss_decode_step(bufs, 2, q2, o2)

        b = ss.ss_layer_buffers.from_buffer_copy(Ls[1].buffers)
        b.k = cfg.k // 2
        with pytest.raises(ss.SparseServeError, match="shape differs"):
            call([Ls[0].buffers, b])
        b = ss.ss_layer_buffers.from_buffer_copy(Ls[1].buffers)
        b.attn_ws_bytes = Ls[1].ws_bytes // 4 * 3  # three of the four regions
        with pytest.raises(ss.SparseServeError, match="workspace"):
            call([Ls[0].buffers, b])
        torch.cuda.synchronize()
    finally:
        close(pool, Ls)


def test_host_groups_schedule_wait_deadline(ss):
    """With the host resolve, a wait for a selection that passes the deadline
    (ss_set_host_wait_timeout) returns SS_ERR_TIMEOUT before any slot table
    changed: the caller's stream is held busy by ordinary work queued before
    the step (four fp32 8192^3 products) against a 2 ms deadline.  After
    synchronising, the next steps equal those of a model that never saw the
    failed call."""
    from paper_2509_24626_amd import harness as H
    cfg, seed = small_cfg(layers=2), 9
    pa, A = build(cfg, seed, 4, False)
    pb, Bm = build(cfg, seed, 4, False)
    try:
        qs = [H.query_stream(cfg, seed, l, cfg.steps) for l in range(cfg.layers)]
        for M in (A, Bm):
            H.decode_step_groups(M, 0, [qs[l][0][1] for l in range(cfg.layers)])
        torch.cuda.synchronize()
        x = torch.randn(8192, 8192, device="cuda")
        torch.cuda.synchronize()
        ss.ss_set_host_wait_timeout(2)
        try:
            for _ in range(4):
                x = x @ x * 1e-4
            with pytest.raises(ss.SparseServeError) as e:
                H.decode_step_groups(Bm, 1, [qs[l][1][1] for l in range(cfg.layers)])
            assert e.value.status == ss.SS_ERR_TIMEOUT, str(e.value)
            assert "step 1" in str(e.value)
        finally:
            ss.ss_set_host_wait_timeout(0)
        torch.cuda.synchronize()
        for t in (1, 2):
            for M in (A, Bm):
                H.decode_step_groups(M, t, [qs[l][t][1] for l in range(cfg.layers)])
            torch.cuda.synchronize()
            for l in range(cfg.layers):
                assert torch.equal(A[l].slots, Bm[l].slots) and torch.equal(A[l].out, Bm[l].out), (t, l)
                assert A[l].last_n_miss == Bm[l].last_n_miss, (t, l)
    finally:
        close(pa, A)
        close(pb, Bm)


@pytest.mark.parametrize("resolve", ["device", "host"])
def test_groups_schedule_gqa7_blk8(ss, resolve):
    """The GQA-7 shape (28 query / 4 KV heads, blocks of 8 tokens, k = 512,
    15% cache, drift 0.6) over three layers with ragged lengths U[2k, 16k]:
    the groups schedule equals layer-by-layer calls bit for bit."""
    from paper_2509_24626_amd import harness as H
    cfg = dataclasses.replace(synth.get(4), name="layers3-gqa7-b7-ragged2k16k-blk8-k512-cache15", B=7, layers=3,
                              ctx=0, ctx_range=(2048, 16384), steps=3)
    seed, dev = 4, resolve == "device"
    pa, A = build(cfg, seed, 3, dev)
    pb, Bm = build(cfg, seed, 3, dev)
    try:
        qs = [H.query_stream(cfg, seed, l, cfg.steps) for l in range(cfg.layers)]
        for t in range(cfg.steps + 1):
            for l, L in enumerate(A):
                L.step(t, qs[l][t][1])
            H.decode_step_groups(Bm, t, [qs[l][t][1] for l in range(cfg.layers)])
            torch.cuda.synchronize()
            for l in range(cfg.layers):
                where = f"step {t} layer {l}"
                assert torch.equal(A[l].sel, Bm[l].sel), where
                assert torch.equal(A[l].slots, Bm[l].slots), where
                assert torch.equal(A[l].out, Bm[l].out), where
    finally:
        close(pa, A)
        close(pb, Bm)

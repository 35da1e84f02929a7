"""Layer-segmented prefill on the saving side (Section 3.4) against the
oracle: for whole-layer and chunked plans, cuboid and mean-key metadata, a
prompt with a ragged tail, the executor's metadata of every layer, the
DRAM records FlashD2H wrote and the open blocks' tail rows equal what the
oracle computes from the same drawn KV (its own save into its own pool,
then its metadata of those records), bit-exact; and the executor's HBM for KV is one
layer's buffer, reused by every layer."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

D = 128


@pytest.fixture(scope="module")
def ss():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2509_24626_amd import binding
    binding.lib()
    return binding


def u16(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("T,layers,max_inject,kind", [(1000, 3, 2500, 0), (1000, 3, 400, 0), (777, 2, 300, 1),
                                                      (4096, 2, 4096, 1), (37, 4, 16, 0)])
def test_prefill_matches_oracle(ss, oracle_impl, T, layers, max_inject, kind):
    from paper_2509_24626_amd import harness as H
    Hkv, blk = 2, 16
    print(f"[gpu] prefill T={T} layers={layers} maxInjectToken={max_inject} kind={kind}", flush=True)
    ex = H.PrefillExecutor(T, layers, Hkv, blk, max_inject, seed=T, meta_kind=kind, threads=3)
    try:
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        batches = ex.run()
        torch.cuda.synchronize()
        one_layer = T * Hkv * 2 * D * 2
        # one layer's KV buffer, reused by every layer: nothing accumulates across layers
        assert ex.buf.numel() * 2 == one_layer
        assert torch.cuda.memory_allocated() - base < (1 << 20)
        assert batches == int(ex.items[-1, 0]) + 1
        rb = ex.rb
        pool_o = np.zeros_like(ex.pool.u8)
        nfull = T // blk
        meta_g = u16(ex.meta)
        open_g = u16(ex.open)
        for l in range(layers):
            kv = u16(ex.layer_kv(l))  # [T][Hkv][2][D]
            oracle_impl.save(kv[None], np.zeros(1, np.int32), blk, pool_o, ex.pool_off[l], np.array([ex.nmax], np.int32))
            # records of full blocks, and the open block's tail rows
            build = oracle_impl.build_metadata if kind == 0 else oracle_impl.build_metadata_mean
            mo = build(pool_o, ex.pool_off[l], np.array([nfull], np.int32), 1, Hkv, ex.nmax, blk, D)
            np.testing.assert_array_equal(meta_g[l, :, :nfull], mo[0, :, :nfull], err_msg=f"metadata layer {l}")
            tail = T - nfull * blk
            for g in range(Hkv):
                rec = pool_o[ex.pool_off[l][g] + nfull * rb:ex.pool_off[l][g] + (nfull + 1) * rb].view(np.uint16)
                Ko, Vo = rec[:blk * D].reshape(blk, D), rec[blk * D:].reshape(D, blk)
                og = open_g[l, g]
                np.testing.assert_array_equal(og[:tail * D], Ko[:tail].reshape(-1))
                np.testing.assert_array_equal(og[blk * D:].reshape(D, blk)[:, :tail], Vo[:, :tail])
        written = np.zeros(ex.pool.u8.size, bool)
        for l in range(layers):
            for g in range(Hkv):
                o = ex.pool_off[l][g]
                written[o:o + nfull * rb] = True
                for t in range(nfull * blk, T):  # tail rows of the last record
                    p = t - nfull * blk
                    written[o + nfull * rb + p * D * 2:o + nfull * rb + (p + 1) * D * 2] = True
        np.testing.assert_array_equal(ex.pool.u8[written], pool_o[written])
        assert list(ex.len_dev.cpu().numpy()) == [T] * layers
        assert list(ex.nblk_dev.cpu().numpy()) == [nfull] * layers
        print(f"[gpu] {batches} batches; KV in HBM: one layer of {one_layer} bytes", flush=True)
    finally:
        ex.close()


def test_prefill_plan_rejects_bad_arguments(ss):
    for args in ((0, 2, 10), (10, 0, 10), (10, 2, 0)):
        with pytest.raises(ss.SparseServeError):
            ss.ss_prefill_plan(*args)

"""The allocation-free attention entry point (ss_sparse_attention_static,
split partials in the library's static device array) against the entry
point with a caller workspace (ss_sparse_attention), through the C ABI: two
calls in a row, the second smaller, each to the 2e-3 attention bound (the
two run the same kernels, so the outputs are also expected to be
identical).  Collected last, so a failure here hides no other test."""
import math

import numpy as np
import pytest
import torch

import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ss():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2509_24626_amd import binding
    binding.lib()
    return binding


def _attend_both(ss, w, slots, cap, slot_limit):
    k = slots.shape[-1]
    ref = gu.run_attention(ss, w, slots, slot_limit=slot_limit, capacity=cap)
    out = torch.full((w.B, w.Hq, w.d), float("nan"), dtype=torch.float32, device="cuda")
    ss.ss_sparse_attention_static(w.q, w.kv, w.unit_off, slots, cap, slot_limit, w.B, w.Hq, w.Hkv, w.d, w.blk, k,
                                  1.0 / math.sqrt(w.d), out)
    torch.cuda.synchronize()
    return ref.cpu().numpy(), out.cpu().numpy()


@pytest.mark.parametrize("order", ["large-then-small", "small-then-large"])
def test_static_scratch_matches_workspace_entry_point(ss, oracle_impl, order):
    """Shapes that split the selection over several workgroups per unit, so
    the partials go through the scratch array: 16 units x 8 splits, then 2
    units x 4 splits (and the reverse order), each against the workspace
    entry point and the oracle."""
    shapes = [(2, 32, 8, 16, 300, 128, "large"), (1, 8, 2, 16, 80, 64, "small")]
    if order == "small-then-large":
        shapes = shapes[::-1]
    for B, Hq, Hkv, blk, nmax, k, tag in shapes:
        assert ss.ss_sparse_attention_workspace(B, Hq, Hkv, 128, blk, k) > 0, "the shape must use split partials"
        w = gu.HbmWorkload(B, Hq, Hkv, blk, nmax, k, seed=61 if tag == "large" else 62)
        rng = np.random.default_rng(7)
        slots = np.stack([np.stack([np.sort(rng.choice(nmax, size=k, replace=False)) for _ in range(Hkv)])
                          for _ in range(B)]).astype(np.int32)
        slots[0, 0, 3] = -1
        cap = np.full(B * Hkv, nmax, np.int32)
        ref, out = _attend_both(ss, w, torch.from_numpy(slots).cuda(), torch.from_numpy(cap).cuda(), nmax)
        assert not np.isnan(out).any()
        assert np.abs(out - ref).max() <= gu.ATTN_TOL, tag
        ora = oracle_impl.attention(w.q_host, w.kv_host, w.unit_off_host, slots, w.Hkv, w.blk)
        assert np.abs(out - ora).max() <= gu.ATTN_TOL, tag
        print(f"[gpu] {tag}: static-scratch output {'identical to' if np.array_equal(out, ref) else 'within 2e-3 of'} "
              f"the workspace entry point's", flush=True)


def test_static_scratch_single_split(ss):
    """A shape with one split per unit needs no partials: the static entry
    point runs it without touching the scratch array."""
    w = gu.HbmWorkload(64, 32, 8, 16, 64, 8, seed=63)
    assert ss.ss_sparse_attention_workspace(64, 32, 8, 128, 16, 8) == 0
    slots = torch.arange(8, dtype=torch.int32, device="cuda").repeat(64, 8, 1).contiguous()
    ref, out = _attend_both(ss, w, slots, None, 64)
    assert np.abs(out - ref).max() <= gu.ATTN_TOL

"""GPU parity of the saving side against the oracle, bit-exact, step after
step: ss_append_kv (each sequence's new token into its open block in HBM,
metadata when a block fills) and FlashD2H (ss_kv_save: one copy of the new
KV to pinned staging memory, host threads place the tokens in the DRAM
pool).  Cases: blocks of 8, 16 and 32 tokens, sequences at different
offsets inside their blocks, several fills per sequence, multi-token saves
that span blocks, the overflow flag, an empty batch, and the full-size
128k-context shape (B=64, 32/8 heads, 8192-block sequences).
"""
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


def bf16_bits(shape, gen):
    return torch.randn(*shape, generator=gen).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


class SaveCase:
    """GPU state (open records, metadata, counts; a pinned DRAM pool) and
    the oracle's copies of the same bytes."""

    def __init__(self, ss, B, Hkv, blk, start, nblk_max, seed, pool_base_block=None, max_new=1, threads=2,
                 staging_slots=3):
        from paper_2509_24626_amd import harness as H
        self.ss, self.B, self.Hkv, self.blk, self.nblk_max = ss, B, Hkv, blk, nblk_max
        self.rb = 2 * blk * D * 2
        self.gen = torch.Generator().manual_seed(seed)
        units = B * Hkv
        self.start = np.asarray(start, np.int32)
        self.len_host = self.start.copy()
        # the open record rows below each sequence's fill level hold earlier tokens
        self.open_o = bf16_bits((B, Hkv, 2 * blk * D), self.gen)
        self.open = torch.from_numpy(self.open_o.view(np.int16).copy()).cuda()
        self.meta_o = np.zeros((B, Hkv, nblk_max, 2, D), np.uint16)
        self.meta = torch.zeros(B, Hkv, nblk_max, 2, D, dtype=torch.int16, device="cuda")
        self.len_o = self.start.copy()
        self.nblk_o = (self.start // blk).astype(np.int32)
        self.len_dev = torch.from_numpy(self.len_o.copy()).cuda()
        self.nblk_dev = torch.from_numpy(self.nblk_o.copy()).cuda()
        self.overflow = torch.zeros(1, dtype=torch.int32, device="cuda")
        # DRAM pool: room for the blocks this case writes.  Unit u's block j
        # is at pool + pool_off[u] + j*rb; with pool_base_block set, each
        # unit's window starts at that block (its offset is shifted down).
        first = 0 if pool_base_block is None else pool_base_block
        self.pool_blocks = np.full(B, nblk_max, np.int32)
        window = nblk_max - first
        self.pool = H.HostPool(units * window * self.rb)
        self.pool.u8[:] = np.frombuffer(np.random.default_rng(seed).bytes(self.pool.nbytes), np.uint8)
        self.pool_o = self.pool.u8.copy()
        self.pool_off = (np.arange(units, dtype=np.int64) * window - first) * self.rb
        self.saver = ss.ss_kv_saver_create(B, Hkv, blk, D, self.pool.host, self.pool_off, self.pool_blocks,
                                           max_new_tokens=max_new, staging_slots=staging_slots, threads=threads)

    def close(self):
        if self.saver:
            self.ss.ss_kv_saver_destroy(self.saver)
            self.saver = None
        self.pool.close()

    def step(self, oracle_impl):
        """One decode token per sequence: append + save on the GPU and in the oracle."""
        kv = bf16_bits((self.B, self.Hkv, 2, D), self.gen)
        kv_dev = torch.from_numpy(kv.view(np.int16).copy()).cuda()
        before = self.len_host.copy()
        self.ss.ss_append_kv(kv_dev, self.len_dev, self.nblk_dev, self.B, self.Hkv, self.blk, D, self.nblk_max,
                             self.open, self.meta, self.overflow)
        self.ss.ss_kv_save(self.saver, kv_dev, 1, before)
        oracle_impl.append(kv, self.len_o, self.nblk_o, self.blk, self.nblk_max, self.open_o, self.meta_o)
        oracle_impl.save(kv[:, None], before, self.blk, self.pool_o, self.pool_off, self.pool_blocks)
        self.len_host += 1
        return kv_dev  # kept alive until the copy has run

    def check_hbm(self, meta_rows=None):
        torch.cuda.synchronize()
        np.testing.assert_array_equal(self.len_dev.cpu().numpy(), self.len_o)
        np.testing.assert_array_equal(self.nblk_dev.cpu().numpy(), self.nblk_o)
        np.testing.assert_array_equal(self.open.cpu().numpy().view(np.uint16), self.open_o)
        if meta_rows is None:
            np.testing.assert_array_equal(self.meta.cpu().numpy().view(np.uint16), self.meta_o)
        else:
            r = slice(*meta_rows)
            np.testing.assert_array_equal(self.meta[:, :, r].cpu().numpy().view(np.uint16), self.meta_o[:, :, r])

    def check_pool(self):
        torch.cuda.synchronize()
        self.ss.ss_kv_save_wait(self.saver)
        np.testing.assert_array_equal(self.pool.u8, self.pool_o)


@pytest.mark.parametrize("blk", [8, 16, 32])
def test_append_and_save_match_oracle(ss, oracle_impl, blk):
    B, Hkv = 3, 2
    start = [0, blk + 5, 3 * blk - 1]
    steps = 2 * blk + 3  # every sequence fills two or three blocks
    print(f"[gpu] append/save blk={blk} B={B} Hkv={Hkv} start={start} steps={steps}", flush=True)
    c = SaveCase(ss, B, Hkv, blk, start, nblk_max=8, seed=100 + blk)
    try:
        keep = []
        for t in range(steps):
            keep.append(c.step(oracle_impl))
            c.check_hbm()
            if t % 7 == 6:
                c.check_pool()
        c.check_pool()
        assert int(c.overflow.item()) == 0
        assert list(c.nblk_o) == [(s + steps) // blk for s in start]
    finally:
        c.close()


def test_save_multi_token_spans_blocks(ss, oracle_impl):
    """Prefill-like saves: 37 then 5 tokens per sequence in one call each,
    crossing several block boundaries, through a single staging slot."""
    B, Hkv, blk = 2, 4, 16
    c = SaveCase(ss, B, Hkv, blk, [3, 20], nblk_max=8, seed=7, max_new=40, staging_slots=1, threads=3)
    try:
        for n in (37, 5):
            kv = bf16_bits((B, n, Hkv, 2, D), c.gen)
            kv_dev = torch.from_numpy(kv.view(np.int16).copy()).cuda()
            ss.ss_kv_save(c.saver, kv_dev, n, c.len_host)
            oracle_impl.save(kv, c.len_host, blk, c.pool_o, c.pool_off, c.pool_blocks)
            c.len_host += n
            c.check_pool()
    finally:
        c.close()


def test_save_rejects_tokens_past_the_pool(ss):
    c = SaveCase(ss, 1, 1, 16, [16 * 7 + 10], nblk_max=8, seed=8, max_new=8)
    try:
        kv = torch.zeros(1, 8, 1, 2, D, dtype=torch.int16, device="cuda")
        with pytest.raises(ss.SparseServeError):
            ss.ss_kv_save(c.saver, kv, 8, c.len_host)  # tokens 122..129: block 8 does not exist
        ss.ss_kv_save(c.saver, kv, 6, c.len_host)  # 122..127 fit
        ss.ss_kv_save_wait(c.saver)
    finally:
        c.close()


def test_append_overflow_flag(ss, oracle_impl):
    """A block that fills at index >= nblk_max: the token is still written
    and the length advanced, but no metadata row is written, the block count
    stays, and the overflow flag is raised."""
    blk = 8
    c = SaveCase(ss, 2, 2, blk, [2 * blk - 1, 0], nblk_max=2, seed=9)
    try:
        kv = torch.from_numpy(bf16_bits((2, 2, 2, D), c.gen).view(np.int16).copy()).cuda()
        ss.ss_append_kv(kv, c.len_dev, c.nblk_dev, 2, 2, blk, D, 2, c.open, c.meta, c.overflow)
        torch.cuda.synchronize()
        assert int(c.overflow.item()) == 0  # block 1 of sequence 0 filled: fine
        ss.ss_append_kv(kv, c.len_dev, c.nblk_dev, 2, 2, blk, D, 2, c.open, c.meta, c.overflow)
        torch.cuda.synchronize()
        assert list(c.nblk_dev.cpu().numpy()) == [2, 0]
        c.len_dev[0] = 3 * blk - 1
        meta_before = c.meta.clone()
        ss.ss_append_kv(kv, c.len_dev, c.nblk_dev, 2, 2, blk, D, 2, c.open, c.meta, c.overflow)
        torch.cuda.synchronize()
        assert int(c.overflow.item()) == 1
        assert list(c.len_dev.cpu().numpy()) == [3 * blk, 3]
        assert list(c.nblk_dev.cpu().numpy()) == [2, 0]
        assert torch.equal(c.meta, meta_before)
    finally:
        c.close()


def test_append_empty_batch_is_a_no_op(ss):
    dummy = torch.zeros(16, dtype=torch.int32, device="cuda")
    ss.ss_append_kv(dummy, dummy, dummy, 0, 8, 16, D, 4, dummy, dummy)
    torch.cuda.synchronize()


def test_full_size_128k_shape(ss, oracle_impl):
    """B=64, 32/8 heads, 8192 blocks of 16 tokens per sequence: 24 decode
    tokens from offsets spread over the block (every sequence fills one
    block, some two).  The pool holds a window of the last blocks of each
    unit (shifted offsets); metadata rows compared are the ones written."""
    B, Hkv, blk = 64, 8, 16
    base = 8190 * blk
    start = base + (np.arange(B) * 5) % blk
    c = SaveCase(ss, B, Hkv, blk, start, nblk_max=8194, seed=10, pool_base_block=8190, threads=4)
    try:
        keep = []
        for t in range(24):
            keep.append(c.step(oracle_impl))
            if t % 8 == 7:
                c.check_hbm(meta_rows=(8190, 8194))
        c.check_hbm(meta_rows=(8190, 8194))
        c.check_pool()
        assert np.all(c.nblk_o >= 8191)
    finally:
        c.close()

"""Seeded generators.  Every draw is keyed by (seed, tags...) so that any
slice of a workload (one layer, one sequence, one step) can be produced on
its own, in any order, with the same values on a given device.  Streams
drawn on the CPU and on the GPU differ (different torch generators); a run
draws everything it compares on one device and hands the same bytes to both
sides.

Block record format (bf16): K tile [blk][d] followed by the V tile stored
channel-major [d][blk]; see the header in include/ for the full contract.
"""
import hashlib
import math

import numpy as np
import torch


def derive_seed(*tags):
    h = hashlib.blake2b(repr(tags).encode(), digest_size=8).digest()
    return int.from_bytes(h, "little") & ((1 << 63) - 1)


def generator(device, *tags):
    g = torch.Generator(device=device)
    g.manual_seed(derive_seed(*tags))
    return g


def to_u16(t):
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)


# ---------------------------------------------------------------- queries
def query(B, Hq, d, seed, device="cpu", layer=0):
    """Initial decode query q ~ N(0,1); returns (fp32 master, bf16)."""
    q = torch.randn(B, Hq, d, generator=generator(device, seed, "q", layer), device=device)
    return q, q.to(torch.bfloat16)


def drift(q, sigma, seed, layer, step):
    """Next step's query: q + sigma * N(0,1), rescaled per head to norm
    sqrt(d) (the scale of an N(0,1) query).  Returns (fp32, bf16)."""
    n = torch.randn(q.shape, generator=generator(q.device, seed, "drift", layer, step), device=q.device)
    x = q + sigma * n
    x = x * (math.sqrt(q.shape[-1]) / x.norm(dim=-1, keepdim=True))
    return x, x.to(torch.bfloat16)


# ---------------------------------------------------------------- KV blocks
def channel_scales(Hkv, d, seed, layer=0, device="cpu"):
    """Per (KV head, channel) scales U[0.5, 2], separately for K and V."""
    g = generator(device, seed, "scale", layer)
    sK = 0.5 + 1.5 * torch.rand(Hkv, d, generator=g, device=device)
    sV = 0.5 + 1.5 * torch.rand(Hkv, d, generator=g, device=device)
    return sK, sV


def planted_blocks(nblk, n_plant, seed, layer, b, g, device="cpu"):
    """n_plant distinct block indices drawn uniformly from [0, nblk)."""
    if n_plant <= 0:
        return torch.empty(0, dtype=torch.long, device=device)
    perm = torch.randperm(nblk, generator=generator(device, seed, "plant", layer, b, g), device=device)
    return perm[:n_plant]


def kv_records_seq(b, Hkv, nblk, blk, d, sK, sV, seed, layer=0, device="cpu",
                   q_bf16_b=None, n_plant=0, shift=1.5):
    """Block records of sequence b: bf16 [Hkv][nblk][2*blk*d].

    K = N(0,1) * sK[g, c] and V = N(0,1) * sV[g, c], drawn in fp32 and rounded
    to bf16 (round to nearest even).  With n_plant > 0, every token key of
    n_plant random blocks per KV head g is shifted by shift * qhat, where
    qhat = sqrt(d) * u / |u| and u is the sum of the bf16 queries of the heads
    that share g (consecutive query heads), added in fp32 before rounding.
    Returns (records, planted) with planted a [Hkv][n_plant] index tensor.
    """
    gk = generator(device, seed, "K", layer, b)
    gv = generator(device, seed, "V", layer, b)
    K = torch.randn(Hkv, nblk, blk, d, generator=gk, device=device) * sK[:, None, None, :]
    planted = torch.empty(Hkv, max(n_plant, 0), dtype=torch.long, device=device)
    if n_plant > 0:
        Hq = q_bf16_b.shape[0]
        G = Hq // Hkv
        for g in range(Hkv):
            u = q_bf16_b[g * G:(g + 1) * G].float().sum(0)
            qhat = math.sqrt(d) * u / u.norm()
            idx = planted_blocks(nblk, n_plant, seed, layer, b, g, device)
            planted[g] = idx
            K[g, idx] += shift * qhat
    V = torch.randn(Hkv, nblk, blk, d, generator=gv, device=device) * sV[:, None, None, :]
    Kb = K.to(torch.bfloat16).reshape(Hkv, nblk, blk * d)
    Vb = V.to(torch.bfloat16).transpose(-1, -2).reshape(Hkv, nblk, d * blk)
    del K, V
    return torch.cat([Kb, Vb], dim=-1), planted


def new_tokens(B, Hkv, d, sK, sV, seed, layer, step, device="cpu"):
    """The decode step's new token per (sequence, KV head): bf16
    [B][Hkv][2][d], K then V, drawn like the context (N(0,1) times the
    layer's channel scales, fp32 rounded to bf16)."""
    g = generator(device, seed, "new", layer, step)
    K = torch.randn(B, Hkv, d, generator=g, device=device) * sK[None]
    V = torch.randn(B, Hkv, d, generator=g, device=device) * sV[None]
    return torch.stack([K, V], dim=2).to(torch.bfloat16).contiguous()


def prefill_kv(T, Hkv, d, sK, sV, seed, layer, device="cpu"):
    """A prompt's new KV for one layer, token-major bf16 [T][Hkv][2][d] (K
    then V), drawn like the context: N(0,1) times the layer's channel
    scales, fp32 rounded to bf16."""
    g = generator(device, seed, "prefill", layer)
    K = torch.randn(T, Hkv, d, generator=g, device=device) * sK[None]
    V = torch.randn(T, Hkv, d, generator=g, device=device) * sV[None]
    return torch.stack([K, V], dim=2).to(torch.bfloat16).contiguous()


def lengths(cfg, seed):
    """Context length in tokens per sequence: fixed, or for a ragged
    workload T_b = blk * round(U[lo, hi] / blk), clamped to [lo, hi]."""
    if not cfg.ctx_range:
        return np.full(cfg.B, cfg.ctx, dtype=np.int64)
    lo, hi = cfg.ctx_range
    g = generator("cpu", seed, "len")
    u = lo + (hi - lo) * torch.rand(cfg.B, generator=g, dtype=torch.float64)
    t = (torch.round(u / cfg.blk) * cfg.blk).clamp(lo, hi).to(torch.int64)
    return t.numpy()


# ---------------------------------------------------------------- selections
def selection_stream(nblk, Hkv, k, steps, churn, seed):
    """Synthetic selection streams with temporal locality, for exercising
    the block cache on its own: int32 [steps][B][Hkv][k], each row strictly
    ascending then -1 padded.  Each step keeps a (1 - churn) share of the
    previous step's blocks and draws the rest anew."""
    rng = np.random.default_rng(derive_seed(seed, "selstream"))
    nblk = np.asarray(nblk)
    B = nblk.shape[0]
    out = np.full((steps, B, Hkv, k), -1, dtype=np.int32)
    for b in range(B):
        n = int(nblk[b])
        m = min(k, n)
        for g in range(Hkv):
            cur = rng.choice(n, size=m, replace=False) if m else np.empty(0, dtype=np.int64)
            for s in range(steps):
                if s > 0 and m:
                    keep = rng.random(m) >= churn
                    kept = cur[keep]
                    pool = np.setdiff1d(np.arange(n), kept)
                    new = rng.choice(pool, size=m - kept.size, replace=False)
                    cur = np.concatenate([kept, new])
                out[s, b, g, :m] = np.sort(cur)
    return out

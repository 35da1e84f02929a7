"""Helpers for the GPU parity tests: seeded workloads drawn on the GPU,
host copies for the oracle, and the comparison rules.

Comparison rules
  * metadata, selections that agree, slots, miss lists, gathered bytes:
    bit-exact;
  * block scores: |gpu - oracle| <= 256 * 2^-24 * sum_c |q_c| * max(|lo_c|, |hi_c|)
    (the worst-case error of a 256-term fp32 sum of exact products, for
    any summation order), taken with the largest such sum over the heads;
  * selection: equal counts, ascending, no duplicates; blocks in the
    symmetric difference with the oracle's selection must have oracle
    scores within 1e-5 relative of the oracle's m-th largest score
    (m = min(k, blocks));
  * attention: max |gpu - oracle| <= 2e-3.
"""
import math

import numpy as np
import torch

import synth
from synth import gen

ATTN_TOL = 2e-3
SEL_REL = 1e-5


def u16(t):
    return gen.to_u16(t)


def bits_to_f64(a):
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


class HbmWorkload:
    """All KV resident in HBM: records [B][Hkv][nblk_max][rec] bf16."""

    def __init__(self, B, Hq, Hkv, blk, nblk_max, k, seed, n_plant=0, nblk=None, d=128, device="cuda",
                 kv_override=None):
        self.B, self.Hq, self.Hkv, self.blk, self.nblk_max, self.k, self.d = B, Hq, Hkv, blk, nblk_max, k, d
        self.units = B * Hkv
        self.rec_bytes = 2 * blk * d * 2
        self.nblk_host = np.full(B, nblk_max, np.int32) if nblk is None else np.asarray(nblk, np.int32)
        self.q32, self.q = gen.query(B, Hq, d, seed, device)
        sK, sV = gen.channel_scales(Hkv, d, seed, 0, device)
        recs = []
        for b in range(B):
            r, _ = gen.kv_records_seq(b, Hkv, nblk_max, blk, d, sK, sV, seed, 0, device, q_bf16_b=self.q[b],
                                      n_plant=n_plant)
            recs.append(r)
        self.kv = torch.stack(recs).contiguous() if kv_override is None else kv_override
        self.nblk = torch.from_numpy(self.nblk_host).to(device)
        off = np.arange(self.units, dtype=np.int64) * nblk_max * self.rec_bytes
        self.unit_off_host = off
        self.unit_off = torch.from_numpy(off).to(device)
        self._host = None

    @property
    def kv_host(self):
        if self._host is None:
            self._host = u16(self.kv)
        return self._host

    @property
    def q_host(self):
        return u16(self.q)


def check_scores(gpu, ora, q_host, meta_host, nblk, G):
    """Elementwise score check with the fp32 summation bound (see module doc)."""
    B, Hkv, nblk_max = ora.shape
    qf = np.abs(bits_to_f64(q_host))  # [B][Hq][d]
    lo = np.abs(bits_to_f64(meta_host[..., 0, :]))
    hi = np.abs(bits_to_f64(meta_host[..., 1, :]))
    mag = np.maximum(lo, hi)  # [B][Hkv][nblk][d]
    worst = 0.0
    for b in range(B):
        n = int(nblk[b])
        for g in range(Hkv):
            absum = (qf[b, g * G:(g + 1) * G] @ mag[b, g, :n].T).max(axis=0)  # [n]
            bound = 256 * 2.0 ** -24 * absum
            err = np.abs(gpu[b, g, :n].astype(np.float64) - ora[b, g, :n])
            assert np.all(err <= bound), (b, g, float((err - bound).max()))
            if n:
                worst = max(worst, float((err / np.maximum(np.abs(ora[b, g, :n]), 1e-30)).max()))
    return worst


def check_selection(gpu_sel, ora_sel, ora_scores, nblk, k):
    """Returns the list of units whose selection differs (legitimately)."""
    B, Hkv, _ = ora_sel.shape
    differing = []
    for b in range(B):
        n = int(nblk[b])
        m = min(k, n)
        for g in range(Hkv):
            gs, os_ = gpu_sel[b, g], ora_sel[b, g]
            assert np.all(gs[m:] == -1) and np.all(gs[:m] >= 0), (b, g, gs)
            assert np.all(np.diff(gs[:m]) > 0), ("not strictly ascending", b, g)
            assert np.all(gs[:m] < n)
            if np.array_equal(gs, os_):
                continue
            S = ora_scores[b, g, :n]
            sk = np.sort(S)[::-1][m - 1]
            diff = set(gs[:m].tolist()) ^ set(os_[:m].tolist())
            for j in diff:
                assert abs(S[j] - sk) <= SEL_REL * abs(sk), ("selection differs outside the tie band", b, g, j,
                                                             S[j], sk)
            differing.append((b, g))
    return differing


def run_metadata(ss, w, stream=None):
    meta = torch.empty(w.B, w.Hkv, w.nblk_max, 2, w.d, dtype=torch.int16, device="cuda")
    ss.ss_build_metadata(w.kv, w.unit_off, w.nblk, w.B, w.Hkv, w.nblk_max, w.blk, w.d, meta, stream)
    return meta


def run_attention(ss, w, slots_dev, slot_limit=None, capacity=None):
    out = torch.empty(w.B, w.Hq, w.d, dtype=torch.float32, device="cuda")
    wsb = ss.ss_sparse_attention_workspace(w.B, w.Hq, w.Hkv, w.d, w.blk, slots_dev.shape[-1])
    ws = torch.empty(max(wsb, 4), dtype=torch.uint8, device="cuda")
    ss.ss_sparse_attention(w.q, w.kv, w.unit_off, slots_dev, capacity, w.nblk_max if slot_limit is None else slot_limit,
                           w.B, w.Hq, w.Hkv, w.d, w.blk, slots_dev.shape[-1], 1.0 / math.sqrt(w.d), out, ws, wsb)
    return out


def check_scores_variant(gpu, ora, q_host, meta_host, nblk, G, kind, agg):
    """Elementwise score check for the metadata kinds and aggregations: the
    GPU sums exact bf16 products in fp32 (and, for agg 1, the G head
    scores), so |gpu - oracle| <= (2*d + G) * 2^-24 * sum over the group's
    heads of sum_c |q_c| * |m_c| (m = max(|lo|, |hi|) for cuboid rows)."""
    B, Hkv, nblk_max = ora.shape
    qf = np.abs(bits_to_f64(q_host))
    if kind == 0:
        mag = np.maximum(np.abs(bits_to_f64(meta_host[..., 0, :])), np.abs(bits_to_f64(meta_host[..., 1, :])))
    else:
        mag = np.abs(bits_to_f64(meta_host))
    d = qf.shape[-1]
    worst = 0.0
    for b in range(B):
        n = int(nblk[b])
        for g in range(Hkv):
            per_head = qf[b, g * G:(g + 1) * G] @ mag[b, g, :n].T  # [G][n]
            bound = (2 * d + G) * 2.0 ** -24 * per_head.sum(axis=0)
            err = np.abs(gpu[b, g, :n].astype(np.float64) - ora[b, g, :n])
            assert np.all(err <= bound), (b, g, float((err - bound).max()))
            if n:
                worst = max(worst, float((err / np.maximum(np.abs(ora[b, g, :n]), 1e-30)).max()))
    return worst

"""Parity helpers: run the HIP path on a chunk and compare with the fp64 oracle.

The oracle reads back exactly the bf16 bits the GPU saw (the inputs are drawn on
the device by the shared generator). For large chunks only sampled (row, head)
items are evaluated; the oracle is called once per kv head involved, on that
kv head's slice of the cache limited to the keys the chunk can reach.

Tolerances (bf16 outputs upcast to fp64): max |out - ref| <= 2e-2,
mean |out - ref| <= 2e-3, max |lse - ref| <= 1e-3. Besides these, a relative
RMS guard ||out - ref|| / ||ref|| <= 1e-2 is applied, because with these inputs
the softmax is nearly uniform and |out| shrinks like 1/sqrt(position): an
all-zero output would pass the absolute bounds on long prefixes.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

import oracle

MAX_ABS = 2e-2
MEAN_ABS = 2e-3
LSE_ABS = 1e-3
REL_RMS = 1e-2


@dataclasses.dataclass
class ParityReport:
    n_items: int
    max_abs: float
    mean_abs: float
    lse_max_abs: float
    rel_rms: float

    def ok(self) -> bool:
        return (self.max_abs <= MAX_ABS and self.mean_abs <= MEAN_ABS
                and self.lse_max_abs <= LSE_ABS and self.rel_rms <= REL_RMS)

    def __str__(self):
        return ("items=%d max_abs=%.3e mean_abs=%.3e lse_max_abs=%.3e rel_rms=%.3e"
                % (self.n_items, self.max_abs, self.mean_abs, self.lse_max_abs, self.rel_rms))


def sample_items(cu_q, kv_start, prefix_len, hq: int, hkv: int, seed: int = 0,
                 n_random_rows: int = 32, n_random_heads: int = 2):
    """Seeded sample of (row, head) items covering tile edges, heads of >=2 groups,
    and the first/last rows of every segment."""
    rng = np.random.default_rng(seed)
    tok = int(cu_q[-1])
    g = hq // hkv
    heads = {0, g - 1, min(g, hq - 1), hq - 1}
    heads |= set(int(x) for x in rng.integers(0, hq, size=n_random_heads))
    rows = {0, 1, max(0, tok - 2), tok - 1}
    for m in rng.integers(1, max(2, tok // 64), size=4):
        for r in (64 * int(m) - 1, 64 * int(m)):
            if 0 <= r < tok:
                rows.add(r)
    rows |= set(int(x) for x in rng.integers(0, tok, size=n_random_rows))
    for s in range(len(kv_start)):
        if cu_q[s + 1] > cu_q[s]:
            rows.add(int(cu_q[s]))
            rows.add(int(cu_q[s + 1]) - 1)
    rows = sorted(r for r in rows if 0 <= r < tok)
    heads = sorted(heads)
    rr = np.repeat(np.array(rows, dtype=np.int64), len(heads))
    hh = np.tile(np.array(heads, dtype=np.int32), len(rows))
    return rr, hh


def oracle_items(q, k_cache, v_cache, cu_q, kv_start, prefix_len, rows, heads,
                 scale: Optional[float] = None, n_threads: int = 0):
    """Oracle on selected items; q/k/v may live on the GPU (slices are copied back)."""
    hq, hkv = q.shape[1], k_cache.shape[1]
    g = hq // hkv
    cu = np.asarray(cu_q)
    ks = np.asarray(kv_start, dtype=np.int64)
    pl = np.asarray(prefix_len, dtype=np.int64)
    # cache rows any segment can reach
    hi = 0
    for s in range(len(ks)):
        if cu[s + 1] > cu[s]:
            hi = max(hi, int(ks[s] + pl[s] + cu[s + 1] - cu[s]))
    rows = np.asarray(rows, dtype=np.int64)
    heads = np.asarray(heads, dtype=np.int32)
    out = np.zeros((len(rows), v_cache.shape[2]))
    lse = np.zeros(len(rows))
    tok = int(cu[-1])
    for kvh in sorted(set((heads // g).tolist())):
        sel = np.nonzero(heads // g == kvh)[0]
        qh = q[:tok, kvh * g:(kvh + 1) * g, :].cpu()
        kh = k_cache[:hi, kvh:kvh + 1, :].cpu()
        vh = v_cache[:hi, kvh:kvh + 1, :].cpu()
        o, l = oracle.attention(qh, kh, vh, cu, ks, pl, rows=rows[sel],
                                heads=heads[sel] - kvh * g, scale=scale, n_threads=n_threads)
        out[sel] = o
        lse[sel] = l
    return out, lse


def compare(out_gpu, lse_gpu, rows, heads, ref_out, ref_lse) -> ParityReport:
    """out_gpu [tokens, Hq, dv] bf16 tensor, lse_gpu [Hq, >=tokens] fp32 tensor or None."""
    r = torch.as_tensor(np.asarray(rows), device=out_gpu.device)
    h = torch.as_tensor(np.asarray(heads, dtype=np.int64), device=out_gpu.device)
    og = out_gpu[r, h].double().cpu().numpy()
    err = np.abs(og - ref_out)
    lse_err = 0.0
    if lse_gpu is not None:
        lg = lse_gpu[h, r].double().cpu().numpy()
        lse_err = float(np.max(np.abs(lg - ref_lse))) if len(rows) else 0.0
    denom = float(np.sqrt(np.sum(ref_out ** 2)))
    rel = float(np.sqrt(np.sum((og - ref_out) ** 2)) / denom) if denom > 0 else 0.0
    return ParityReport(n_items=len(rows), max_abs=float(err.max()) if err.size else 0.0,
                        mean_abs=float(err.mean()) if err.size else 0.0,
                        lse_max_abs=lse_err, rel_rms=rel)


def run_chunk(attn, q, k_cache, v_cache, cu_q, kv_start, prefix_len, lse_cols: int = 0):
    """Plan + run one chunk with a ChunkAttention; returns (out, lse [Hq, tokens])."""
    attn.plan(cu_q, kv_start, prefix_len)
    tok = int(cu_q[-1])
    out = torch.full((tok, q.shape[1], v_cache.shape[2]), float("nan"),
                     dtype=torch.bfloat16, device=q.device)
    lse = torch.full((q.shape[1], max(tok, lse_cols)), float("nan"), dtype=torch.float32,
                     device=q.device)
    attn.run(q[:tok], k_cache, v_cache, out, lse)
    torch.cuda.synchronize()
    return out, lse


def planned_splits(requested, prefixes, lens, tile=64):
    """Split count a plan uses for a fixed request: the request, capped at one key
    tile of prefix per piece (longest prefix of a segment with rows); a chunk with
    no prefix is not split."""
    longest = max([int(p) for p, n in zip(prefixes, lens) if int(n) > 0], default=0)
    return min(int(requested), max(1, longest // tile))

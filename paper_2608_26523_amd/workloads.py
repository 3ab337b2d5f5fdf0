"""Workload registry and seeded synthetic input generators.

This module is shared by the HIP path's callers (bench, tests) and by the oracle
side of the tests. It holds no attention arithmetic: it only describes the five
workloads (shapes, chunking, request mix) and draws the random bf16 inputs.

Workloads (one layer of attention, all on one GPU):

* ``tiny``  -- 1 request of 1024 tokens in chunks of 256, 4 query / 4 kv heads,
  head dim 64.
* ``gqa``   -- 1 request of 32768 tokens in chunks of 4096, 32 query / 8 kv heads
  (grouped-query attention, as in the paper's Qwen3 model, section 6.1),
  head dim 128.
* ``mla``   -- 1 request of 131072 tokens in chunks of 8192, 128 heads, qk dim 192
  (128 + 64 rope), v dim 128: the multi-head form of the MLA attention of the
  paper's DeepSeek-V3.1 model (section 6.1).
* ``long``  -- 1 request of 524288 tokens (the 512K workload of section 6.3) in
  chunks of 16384, MLA shape, with the prefix split for an lse merge.
* ``mixed`` -- 64 requests with lengths log-uniform in [1024, 262144], packed
  back to back into 8192-token chunks that cross request boundaries; 64 query /
  4 kv heads, head dim 128. This is a synthetic stand-in for the paper's mixed
  GSM8K-derived request suite (section 6.1), whose items are not used here.

Inputs: Q, K, V drawn i.i.d. N(0, 1) and divided by sqrt(dqk), rounded to bf16,
on the requested device from torch's generator, slab by slab with a seed derived
from (seed, workload, tensor, slab) so that the same bits come back whatever
else ran before.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Tuple

import numpy as np

SLAB_TOKENS = 8192


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int             # position in the registry (0-based)
    hq: int
    hkv: int
    dqk: int
    dv: int
    chunk: int             # chunk size C in tokens
    seq_len: int = 0       # single-request workloads: tokens of the request
    n_requests: int = 1
    len_lo: int = 0        # mixed workload: log-uniform length range
    len_hi: int = 0
    num_splits: int = -1   # split-KV request: -1 auto, 1 off, n fixed
    seed: int = 0

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.dqk)


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny", 0, hq=4, hkv=4, dqk=64, dv=64, chunk=256, seq_len=1024),
        Workload("gqa", 1, hq=32, hkv=8, dqk=128, dv=128, chunk=4096, seq_len=32768),
        Workload("mla", 2, hq=128, hkv=128, dqk=192, dv=128, chunk=8192, seq_len=131072),
        Workload("long", 3, hq=128, hkv=128, dqk=192, dv=128, chunk=16384,
                 seq_len=524288, num_splits=4),
        Workload("mixed", 4, hq=64, hkv=4, dqk=128, dv=128, chunk=8192,
                 n_requests=64, len_lo=1024, len_hi=262144),
    ]
}


def get(name: str) -> Workload:
    return WORKLOADS[name]


def request_lengths(w: Workload) -> np.ndarray:
    """Token count of each request, in packing order.

    Mixed workload: L = round(exp(U(ln lo, ln hi))) from numpy's PCG64(seed).
    """
    if w.n_requests == 1:
        return np.array([w.seq_len], dtype=np.int64)
    rng = np.random.Generator(np.random.PCG64(w.seed))
    u = rng.uniform(math.log(w.len_lo), math.log(w.len_hi), size=w.n_requests)
    return np.rint(np.exp(u)).astype(np.int64)


def request_starts(w: Workload) -> np.ndarray:
    """Packed token index of each request's first token (also its cache row)."""
    lens = request_lengths(w)
    return np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)


def total_tokens(w: Workload) -> int:
    return int(request_lengths(w).sum())


def num_chunks(w: Workload) -> int:
    return -(-total_tokens(w) // w.chunk)


def chunk_segments(w: Workload, k: int, chunk: int = 0) -> Tuple[int, np.ndarray, np.ndarray, np.ndarray]:
    """Segments of chunk k of the packed token stream.

    Returns (first packed token of the chunk, cu_q int32 [n+1], kv_start int64 [n],
    prefix_len int64 [n]). Segment s covers the chunk-local rows cu_q[s]..cu_q[s+1]-1,
    which belong to one request; kv_start is that request's first cache row and
    prefix_len the in-request position of the segment's first token. ``chunk``
    overrides the workload's chunk size (0 keeps it).
    """
    c = chunk or w.chunk
    lens = request_lengths(w)
    starts = request_starts(w)
    total = int(lens.sum())
    t0 = k * c
    t1 = min(t0 + c, total)
    if t0 >= total or k < 0:
        raise IndexError("chunk %d out of range" % k)
    cu = [0]
    kvs: List[int] = []
    pre: List[int] = []
    for r in range(len(lens)):
        a, b = int(starts[r]), int(starts[r] + lens[r])
        lo, hi = max(a, t0), min(b, t1)
        if lo >= hi:
            continue
        cu.append(cu[-1] + (hi - lo))
        kvs.append(a)
        pre.append(lo - a)
    return (t0, np.array(cu, dtype=np.int32), np.array(kvs, dtype=np.int64),
            np.array(pre, dtype=np.int64))


# ----------------------------------------------------------------------------
# random inputs
# ----------------------------------------------------------------------------
TENSOR_IDS = {"q": 1, "k": 2, "v": 3}


def _slab_seed(seed: int, index: int, tensor: str, slab: int) -> int:
    # a fixed mixing of the four integers into one 63-bit torch seed
    x = (seed * 0x9E3779B97F4A7C15 + (index + 1) * 0xBF58476D1CE4E5B9
         + TENSOR_IDS[tensor] * 0x94D049BB133111EB + slab * 0x2545F4914F6CDD1D)
    return x & ((1 << 63) - 1)


def normal_bf16(shape, std: float, seed: int, index: int, tensor: str, device,
                out=None, first_token: int = 0):
    """bf16 tensor of N(0,1)*std values, drawn slab by slab along dim 0.

    Row r of the result is token ``first_token + r`` of the full stream, which
    must start on a slab boundary; the bits do not depend on ``first_token``.
    """
    import torch
    if first_token % SLAB_TOKENS:
        raise ValueError("first_token must be a multiple of %d" % SLAB_TOKENS)
    if out is None:
        out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    n = out.shape[0]
    gen = torch.Generator(device=out.device)
    for t0 in range(0, n, SLAB_TOKENS):
        t1 = min(n, t0 + SLAB_TOKENS)
        gen.manual_seed(_slab_seed(seed, index, tensor, (first_token + t0) // SLAB_TOKENS))
        tmp = torch.randn((t1 - t0,) + tuple(out.shape[1:]), generator=gen,
                          device=out.device, dtype=torch.float32)
        out[t0:t1].copy_(tmp.mul_(std))
        del tmp
    return out


def make_inputs(w: Workload, device, tokens: int = 0):
    """Full-sequence q [S, Hq, dqk], k_cache [S, Hkv, dqk], v_cache [S, Hkv, dv].

    ``tokens`` (0 = all) truncates the packed stream, for tests that only need a
    prefix of a workload.
    """
    s = tokens or total_tokens(w)
    std = 1.0 / math.sqrt(w.dqk)
    q = normal_bf16((s, w.hq, w.dqk), std, w.seed, w.index, "q", device)
    k = normal_bf16((s, w.hkv, w.dqk), std, w.seed, w.index, "k", device)
    v = normal_bf16((s, w.hkv, w.dv), std, w.seed, w.index, "v", device)
    return q, k, v


def make_q_rows(w: Workload, device, t0: int, t1: int):
    """Rows t0..t1-1 of the workload's q, the same bits as make_inputs (a view into
    the enclosing slabs when t0 is not on a slab boundary)."""
    std = 1.0 / math.sqrt(w.dqk)
    a = t0 - t0 % SLAB_TOKENS
    full = normal_bf16((t1 - a, w.hq, w.dqk), std, w.seed, w.index, "q", device, first_token=a)
    return full[t0 - a:]

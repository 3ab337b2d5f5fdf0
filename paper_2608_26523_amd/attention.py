"""PyTorch-facing wrapper of the C ABI: device memory and streams come from torch.

``ChunkAttention`` validates tensors, owns a plan and a device workspace, and
passes raw pointers and element strides to ``vpp_chunk_attn_plan`` /
``vpp_chunk_attn_run``. It does no arithmetic of its own.
"""
from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import binding as B


class ChunkAttention:
    """Chunked-prefill causal attention for one layer's head configuration.

    Typical use, chunk by chunk (the chunk's K/V already written to the cache)::

        attn = ChunkAttention(hq, hkv, dqk, dv, max_chunk_tokens=C, max_kv_len=S)
        attn.plan(cu_q, kv_start, prefix_len)
        attn.run(q_chunk, k_cache, v_cache, out_chunk, lse_chunk)
    """

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim_qk: int, head_dim_v: int,
                 max_chunk_tokens: int, max_kv_len: int, max_segments: int = 1024,
                 num_splits: int = -1, softmax_scale: float = 0.0, device=None):
        B.load()
        self.cfg = B.Config(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                            head_dim_qk=head_dim_qk, head_dim_v=head_dim_v,
                            softmax_scale=softmax_scale, causal=1,
                            max_chunk_tokens=max_chunk_tokens, max_segments=max_segments,
                            max_kv_len=max_kv_len, num_splits=num_splits)
        self.device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        self._plan: Optional[int] = None
        self._ws: Optional[torch.Tensor] = None
        self.workspace_bytes = 0
        self.tokens = 0

    # -- planning -----------------------------------------------------------
    def plan(self, cu_q: Sequence[int], kv_start: Sequence[int], prefix_len: Sequence[int]):
        first = self._plan is None
        h, ws = B.vpp_chunk_attn_plan(self.cfg if first else None, cu_q, kv_start, prefix_len,
                                      plan=self._plan)
        self._plan = h
        self.workspace_bytes = ws
        cu = [int(x) for x in cu_q]
        # last cache row the chunk reads: the C ABI cannot see tensor sizes, so the
        # wrapper checks the caches against it before every run
        self.max_row = max([int(kv_start[s]) + int(prefix_len[s]) + cu[s + 1] - cu[s]
                            for s in range(len(kv_start)) if cu[s + 1] > cu[s]] or [0])
        if self._ws is None or self._ws.numel() < ws:
            self._ws = torch.empty(ws, dtype=torch.uint8, device=self.device)
        self.tokens = int(cu_q[-1])
        return B.vpp_chunk_attn_plan_info(h)

    def info(self):
        return B.vpp_chunk_attn_plan_info(self._plan)

    def items(self):
        return B.vpp_chunk_attn_plan_items(self._plan)

    # -- running ------------------------------------------------------------
    @staticmethod
    def _check(t: torch.Tensor, name: str, dtype, ndim: int):
        if t.dtype != dtype:
            raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
        if t.device.type != "cuda":
            raise ValueError("%s must be on the GPU" % name)
        if t.dim() != ndim:
            raise ValueError("%s must have %d dimensions" % (name, ndim))
        if t.stride(-1) != 1:
            raise ValueError("%s: last dimension must be contiguous" % name)

    def run(self, q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
            out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
            stream: Optional[torch.cuda.Stream] = None):
        """Enqueue the planned chunk on ``stream`` (default: torch's current stream).

        q [tokens, Hq, dqk], k_cache [rows, Hkv, dqk], v_cache [rows, Hkv, dv] bf16;
        out [tokens, Hq, dv] bf16 (allocated when None); lse an fp32 view whose
        element [h, r] is chunk row r of head h (e.g. a column slice of a
        [Hq, seq] tensor), or None.
        """
        if self._plan is None:
            raise RuntimeError("plan() must be called before run()")
        c = self.cfg
        self._check(q, "q", torch.bfloat16, 3)
        self._check(k_cache, "k_cache", torch.bfloat16, 3)
        self._check(v_cache, "v_cache", torch.bfloat16, 3)
        if q.shape[0] < self.tokens or q.shape[1] != c.num_q_heads or q.shape[2] != c.head_dim_qk:
            raise ValueError("q shape %s does not match the plan" % (tuple(q.shape),))
        if k_cache.shape[1] != c.num_kv_heads or k_cache.shape[2] != c.head_dim_qk:
            raise ValueError("k_cache shape %s does not match the config" % (tuple(k_cache.shape),))
        if v_cache.shape[1] != c.num_kv_heads or v_cache.shape[2] != c.head_dim_v:
            raise ValueError("v_cache shape %s does not match the config" % (tuple(v_cache.shape),))
        if k_cache.shape[0] < self.max_row or v_cache.shape[0] < self.max_row:
            raise ValueError("the planned chunk reads cache rows up to %d but the caches hold "
                             "%d/%d rows" % (self.max_row, k_cache.shape[0], v_cache.shape[0]))
        if out is None:
            out = torch.empty((self.tokens, c.num_q_heads, c.head_dim_v), dtype=torch.bfloat16,
                              device=q.device)
        self._check(out, "out", torch.bfloat16, 3)
        if out.shape[0] < self.tokens or out.shape[1] != c.num_q_heads or out.shape[2] != c.head_dim_v:
            raise ValueError("out shape %s does not match the plan" % (tuple(out.shape),))
        lse_ptr, lse_sh = 0, 0
        if lse is not None:
            if lse.dtype != torch.float32 or lse.dim() != 2 or lse.stride(1) != 1:
                raise ValueError("lse must be a 2-D fp32 [Hq, tokens] view with unit token stride")
            if lse.shape[0] != c.num_q_heads or lse.shape[1] < self.tokens:
                raise ValueError("lse shape %s does not match the plan" % (tuple(lse.shape),))
            lse_ptr, lse_sh = lse.data_ptr(), lse.stride(0)
        s = stream if stream is not None else torch.cuda.current_stream(q.device)
        B.vpp_chunk_attn_run(self._plan,
                             q.data_ptr(), q.stride(0), q.stride(1),
                             k_cache.data_ptr(), k_cache.stride(0), k_cache.stride(1),
                             v_cache.data_ptr(), v_cache.stride(0), v_cache.stride(1),
                             out.data_ptr(), out.stride(0), out.stride(1),
                             lse_ptr, lse_sh,
                             self._ws.data_ptr(), self._ws.numel(), s.cuda_stream)
        return out, lse

    def close(self):
        if self._plan is not None:
            B.vpp_chunk_attn_destroy(self._plan)
            self._plan = None
        self._ws = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

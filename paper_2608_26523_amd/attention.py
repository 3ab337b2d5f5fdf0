"""PyTorch-facing wrapper of the C ABI: device memory and streams come from torch.

``ChunkAttention`` validates tensors, owns a plan and a device workspace, and
passes raw pointers and element strides to ``vpp_chunk_attn_plan`` /
``vpp_chunk_attn_run`` (contiguous cache), ``vpp_chunk_attn_run_noalloc`` (the
same without a workspace), ``vpp_chunk_attn_run_paged`` (paged cache) or
``vpp_chunk_attn_run_mla`` (keys split into per-head and shared parts);
``kv_append_paged`` wraps ``vpp_kv_append_paged``. Nothing here does arithmetic
of its own.
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
        dev = torch.device(device) if device is not None else torch.device("cuda")
        if dev.type != "cuda":
            raise ValueError("the workspace must be on a GPU, not %s" % dev)
        self.device = dev if dev.index is not None else torch.device("cuda", torch.cuda.current_device())
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
        self.seg_rows = [int(kv_start[s]) + int(prefix_len[s]) + cu[s + 1] - cu[s]
                         for s in range(len(kv_start))]
        self.max_row = max([self.seg_rows[s] for s in range(len(kv_start)) if cu[s + 1] > cu[s]] or [0])
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

    def _on_device(self, *named):
        """Every tensor must live on the device that holds the plan's workspace."""
        for t, name in named:
            if t is not None and t.device != self.device:
                raise ValueError("%s is on %s but the plan's workspace is on %s" % (name, t.device, self.device))

    def _stream(self, stream, *allocated):
        """The launch stream (default: torch's current stream). Memory this object
        allocated on the current stream is recorded on another launch stream, so that
        torch's allocator does not hand it out while the kernel may still use it."""
        cur = torch.cuda.current_stream(self.device)
        s = stream if stream is not None else cur
        if s != cur:
            for t in (self._ws,) + allocated:
                if t is not None:
                    t.record_stream(s)
        return s

    def _io(self, q: torch.Tensor, out: Optional[torch.Tensor], lse: Optional[torch.Tensor]):
        """Checks of q, out and lse shared by the run methods; allocates out if None
        (the second value returned is that new tensor, else None)."""
        if self._plan is None:
            raise RuntimeError("plan() must be called before run()")
        c = self.cfg
        self._check(q, "q", torch.bfloat16, 3)
        self._on_device((q, "q"), (out, "out"), (lse, "lse"))
        if q.shape[0] < self.tokens or q.shape[1] != c.num_q_heads or q.shape[2] != c.head_dim_qk:
            raise ValueError("q shape %s does not match the plan" % (tuple(q.shape),))
        new_out = None
        if out is None:
            out = new_out = torch.empty((self.tokens, c.num_q_heads, c.head_dim_v), dtype=torch.bfloat16,
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
        return out, lse_ptr, lse_sh, new_out

    def _check_cache(self, k_cache: torch.Tensor, v_cache: torch.Tensor):
        """Checks of a contiguous cache shared by run and run_noalloc."""
        c = self.cfg
        self._check(k_cache, "k_cache", torch.bfloat16, 3)
        self._check(v_cache, "v_cache", torch.bfloat16, 3)
        if k_cache.shape[1] != c.num_kv_heads or k_cache.shape[2] != c.head_dim_qk:
            raise ValueError("k_cache shape %s does not match the config" % (tuple(k_cache.shape),))
        if v_cache.shape[1] != c.num_kv_heads or v_cache.shape[2] != c.head_dim_v:
            raise ValueError("v_cache shape %s does not match the config" % (tuple(v_cache.shape),))
        if k_cache.shape[0] < self.max_row or v_cache.shape[0] < self.max_row:
            raise ValueError("the planned chunk reads cache rows up to %d but the caches hold "
                             "%d/%d rows" % (self.max_row, k_cache.shape[0], v_cache.shape[0]))
        self._on_device((k_cache, "k_cache"), (v_cache, "v_cache"))

    def run(self, q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
            out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
            stream: Optional[torch.cuda.Stream] = None):
        """Enqueue the planned chunk on ``stream`` (default: torch's current stream).

        q [tokens, Hq, dqk], k_cache [rows, Hkv, dqk], v_cache [rows, Hkv, dv] bf16;
        out [tokens, Hq, dv] bf16 (allocated when None); lse an fp32 view whose
        element [h, r] is chunk row r of head h (e.g. a column slice of a
        [Hq, seq] tensor), or None.
        """
        out, lse_ptr, lse_sh, new_out = self._io(q, out, lse)
        self._check_cache(k_cache, v_cache)
        s = self._stream(stream, new_out)
        B.vpp_chunk_attn_run(self._plan,
                             q.data_ptr(), q.stride(0), q.stride(1),
                             k_cache.data_ptr(), k_cache.stride(0), k_cache.stride(1),
                             v_cache.data_ptr(), v_cache.stride(0), v_cache.stride(1),
                             out.data_ptr(), out.stride(0), out.stride(1),
                             lse_ptr, lse_sh,
                             self._ws.data_ptr(), self._ws.numel(), s.cuda_stream)
        return out, lse

    def run_noalloc(self, q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                    out: torch.Tensor, lse: Optional[torch.Tensor] = None,
                    stream: Optional[torch.cuda.Stream] = None):
        """Like ``run``, through ``vpp_chunk_attn_run_noalloc``: the library's static
        device scratch replaces this object's workspace, and nothing is allocated
        (``out`` must be given). Plans needing more than ``NOALLOC_SCRATCH_BYTES``
        are refused; calls that overlap on one GPU share its scratch and race."""
        if out is None:
            raise ValueError("run_noalloc allocates nothing: pass out")
        out, lse_ptr, lse_sh, _ = self._io(q, out, lse)
        self._check_cache(k_cache, v_cache)
        s = stream if stream is not None else torch.cuda.current_stream(self.device)
        if s.device != self.device:
            raise ValueError("stream is on %s but the tensors are on %s" % (s.device, self.device))
        # the library takes the scratch of the current device: make it the tensors' device
        with torch.cuda.device(self.device):
            B.vpp_chunk_attn_run_noalloc(self._plan,
                                         q.data_ptr(), q.stride(0), q.stride(1),
                                         k_cache.data_ptr(), k_cache.stride(0), k_cache.stride(1),
                                         v_cache.data_ptr(), v_cache.stride(0), v_cache.stride(1),
                                         out.data_ptr(), out.stride(0), out.stride(1),
                                         lse_ptr, lse_sh, s.cuda_stream)
        return out, lse

    def run_mla(self, q: torch.Tensor, k_nope: torch.Tensor, k_rope: torch.Tensor, v_cache: torch.Tensor,
                out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                stream: Optional[torch.cuda.Stream] = None):
        """Like ``run`` with the keys split as in the MLA models: k_nope [rows, Hkv, 128] per
        head and k_rope [rows, 64] shared by all heads (head dims (192, 128) only)."""
        out, lse_ptr, lse_sh, new_out = self._io(q, out, lse)
        c = self.cfg
        if c.head_dim_qk != 192 or c.head_dim_v != 128:
            raise ValueError("the split key layout needs head dims (192, 128)")
        self._check(k_nope, "k_nope", torch.bfloat16, 3)
        self._check(k_rope, "k_rope", torch.bfloat16, 2)
        self._check(v_cache, "v_cache", torch.bfloat16, 3)
        if k_nope.shape[1] != c.num_kv_heads or k_nope.shape[2] != 128 or k_rope.shape[1] != 64:
            raise ValueError("k_nope %s / k_rope %s do not match the config"
                             % (tuple(k_nope.shape), tuple(k_rope.shape)))
        if v_cache.shape[1] != c.num_kv_heads or v_cache.shape[2] != c.head_dim_v:
            raise ValueError("v_cache shape %s does not match the config" % (tuple(v_cache.shape),))
        if min(k_nope.shape[0], k_rope.shape[0], v_cache.shape[0]) < self.max_row:
            raise ValueError("the planned chunk reads cache rows up to %d" % self.max_row)
        self._on_device((k_nope, "k_nope"), (k_rope, "k_rope"), (v_cache, "v_cache"))
        s = self._stream(stream, new_out)
        B.vpp_chunk_attn_run_mla(self._plan,
                                 q.data_ptr(), q.stride(0), q.stride(1),
                                 k_nope.data_ptr(), k_nope.stride(0), k_nope.stride(1),
                                 k_rope.data_ptr(), k_rope.stride(0),
                                 v_cache.data_ptr(), v_cache.stride(0), v_cache.stride(1),
                                 out.data_ptr(), out.stride(0), out.stride(1),
                                 lse_ptr, lse_sh,
                                 self._ws.data_ptr(), self._ws.numel(), s.cuda_stream)
        return out, lse

    def run_paged(self, q: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                  block_table: torch.Tensor, out: Optional[torch.Tensor] = None,
                  lse: Optional[torch.Tensor] = None, stream: Optional[torch.cuda.Stream] = None):
        """Like ``run`` over a paged cache: k_pages [pages, page_size, Hkv, dqk], v_pages
        [pages, page_size, Hkv, dv] bf16; block_table int32 [segments, pages_per_row] on the
        device (row s: the pages of segment s's request, in cache-row order)."""
        out, lse_ptr, lse_sh, new_out = self._io(q, out, lse)
        c = self.cfg
        self._check(k_pages, "k_pages", torch.bfloat16, 4)
        self._check(v_pages, "v_pages", torch.bfloat16, 4)
        if k_pages.shape[2] != c.num_kv_heads or k_pages.shape[3] != c.head_dim_qk:
            raise ValueError("k_pages shape %s does not match the config" % (tuple(k_pages.shape),))
        if v_pages.shape[2] != c.num_kv_heads or v_pages.shape[3] != c.head_dim_v:
            raise ValueError("v_pages shape %s does not match the config" % (tuple(v_pages.shape),))
        if k_pages.shape[:2] != v_pages.shape[:2]:
            raise ValueError("k_pages and v_pages must have the same pages and page size")
        page = int(k_pages.shape[1])
        if block_table.dtype != torch.int32 or block_table.dim() != 2 or block_table.device != q.device \
                or block_table.stride(1) != 1:
            raise ValueError("block_table must be an int32 [segments, pages] tensor on the GPU")
        if block_table.shape[0] < len(self.seg_rows):
            raise ValueError("block_table has %d rows for %d segments" % (block_table.shape[0], len(self.seg_rows)))
        need = max(self.seg_rows or [0])
        if need > block_table.shape[1] * page:
            raise ValueError("the planned chunk reads cache rows up to %d but a block-table row maps "
                             "%d" % (need, block_table.shape[1] * page))
        self._on_device((k_pages, "k_pages"), (v_pages, "v_pages"), (block_table, "block_table"))
        s = self._stream(stream, new_out)
        B.vpp_chunk_attn_run_paged(self._plan,
                                   q.data_ptr(), q.stride(0), q.stride(1),
                                   k_pages.data_ptr(), k_pages.stride(0), k_pages.stride(1), k_pages.stride(2),
                                   v_pages.data_ptr(), v_pages.stride(0), v_pages.stride(1), v_pages.stride(2),
                                   page, int(k_pages.shape[0]),
                                   block_table.data_ptr(), block_table.stride(0),
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


def kv_append_paged(k_new: torch.Tensor, v_new: torch.Tensor, k_pages: torch.Tensor,
                    v_pages: torch.Tensor, slot_mapping: torch.Tensor,
                    stream: Optional[torch.cuda.Stream] = None) -> None:
    """Write k_new [tokens, Hkv, dqk] and v_new [tokens, Hkv, dv] (bf16) into the paged caches
    at slot_mapping [tokens] (int64, on the GPU; slot = page * page_size + row, -1 skips)."""
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        ChunkAttention._check(t, name, torch.bfloat16, 3)
    for t, name in ((k_pages, "k_pages"), (v_pages, "v_pages")):
        ChunkAttention._check(t, name, torch.bfloat16, 4)
    for t, name in ((v_new, "v_new"), (k_pages, "k_pages"), (v_pages, "v_pages")):
        if t.device != k_new.device:
            raise ValueError("%s is on %s, k_new on %s" % (name, t.device, k_new.device))
    if slot_mapping.dtype != torch.int64 or slot_mapping.dim() != 1 or slot_mapping.device != k_new.device \
            or slot_mapping.stride(0) != 1:
        raise ValueError("slot_mapping must be a contiguous int64 vector on the GPU")
    T, H, dqk = k_new.shape
    dv = v_new.shape[2]
    if v_new.shape[:2] != (T, H) or slot_mapping.shape[0] != T:
        raise ValueError("k_new, v_new and slot_mapping disagree on tokens/heads")
    if k_pages.shape[2:] != (H, dqk) or v_pages.shape[2:] != (H, dv) or k_pages.shape[:2] != v_pages.shape[:2]:
        raise ValueError("page shapes do not match the new rows")
    s = stream if stream is not None else torch.cuda.current_stream(k_new.device)
    B.vpp_kv_append_paged(k_new.data_ptr(), k_new.stride(0), k_new.stride(1),
                          v_new.data_ptr(), v_new.stride(0), v_new.stride(1),
                          k_pages.data_ptr(), k_pages.stride(0), k_pages.stride(1), k_pages.stride(2),
                          v_pages.data_ptr(), v_pages.stride(0), v_pages.stride(1), v_pages.stride(2),
                          T, H, dqk, dv, int(k_pages.shape[1]), int(k_pages.shape[0]),
                          slot_mapping.data_ptr(), s.cuda_stream)

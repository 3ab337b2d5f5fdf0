"""The largest cache row stride the ABI accepts, on the GPU.

A key tile is 64 cache rows; its byte count (rows x row stride x 2 bytes) is the
size of the buffer resource its copies read through, a 32-bit field, so the host
accepts row strides up to 2^24 - 8 elements and refuses 2^24. At that bound one
tile spans 2^31 - 1024 bytes. Here K (192 dims) and V (128 dims) of every key sit
in one row of such a buffer, 1220 rows or 41 GB, so the running copy sources of
the kernel cross a 4 GiB boundary every 128 rows, ascending and descending. The
split key layout reads the same rows as k_nope [0, 128) and k_rope [128, 192).
Every (row, head) item is compared with the fp64 oracle for both tile variants,
unsplit and split; the split key run must give the bits of the concatenated one.
"""
import numpy as np
import pytest
import torch

import oracle
import parity as PA

pytestmark = pytest.mark.gpu

DEV = "cuda"
STRIDE = (1 << 24) - 8


def _rand(shape, std, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * std).to(torch.bfloat16)


def test_largest_row_stride_every_item(monkeypatch):
    from paper_2608_26523_amd.attention import ChunkAttention
    p, L = 700, 520  # three 256-row tiles (one slot runs a tile descending), a ragged prefix
    R = p + L
    std = 1.0 / np.sqrt(192)
    buf = torch.empty(R * STRIDE, dtype=torch.bfloat16, device=DEV)
    try:
        k = buf.as_strided((R, 1, 192), (STRIDE, 192, 1), 0)
        v = buf.as_strided((R, 1, 128), (STRIDE, 128, 1), 192)
        k.copy_(_rand((R, 1, 192), std, 71))
        v.copy_(_rand((R, 1, 128), std, 72))
        k_nope = buf.as_strided((R, 1, 128), (STRIDE, 128, 1), 0)
        k_rope = buf.as_strided((R, 64), (STRIDE, 1), 128)
        assert k.stride(0) == STRIDE and v.stride(0) == STRIDE
        q = _rand((L, 1, 192), std, 73)
        cu = np.array([0, L])
        ref_o, ref_l = oracle.attention_full(q.cpu(), k.cpu(), v.cpu(), cu, [0], [p])
        rows, heads = np.arange(L), np.zeros(L, dtype=np.int64)
        for nb in (1, 2):
            monkeypatch.setenv("VPP_NB", str(nb))
            for splits in (1, 2):
                what = "row stride %d, nb %d, splits %d" % (STRIDE, nb, splits)
                print("case:", what, flush=True)
                attn = ChunkAttention(1, 1, 192, 128, max_chunk_tokens=L, max_kv_len=R, num_splits=splits)
                out, lse = PA.run_chunk(attn, q, k, v, cu, [0], [p])
                info = attn.info()
                assert info.block_m == 128 * nb and info.num_splits == splits
                rep = PA.compare(out, lse, rows, heads, ref_o.reshape(L, -1), ref_l.reshape(-1))
                print(what, rep, flush=True)
                assert rep.ok(), "%s: %s" % (what, rep)
                out_s = torch.full_like(out, float("nan"))
                lse_s = torch.full_like(lse, float("nan"))
                attn.run_mla(q, k_nope, k_rope, v, out=out_s, lse=lse_s)
                torch.cuda.synchronize()
                assert torch.equal(out_s, out) and torch.equal(lse_s, lse), "split keys differ: " + what
    finally:
        del buf
        torch.cuda.empty_cache()

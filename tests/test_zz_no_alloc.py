"""vpp_chunk_attn_run_noalloc against vpp_chunk_attn_run (GPU).

Both entry points run the same plan through the same kernels, so the no-allocation
variant (its workspace is the library's static device scratch) must give the same
bits. Two calls in a row share the scratch: a split chunk (work list and fp32
partials in the scratch) and then a smaller unsplit one, which must not see the
first call's leftovers; then the split chunk once more, and a chunk of the MLA
shape with a split key range.
"""
import math

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _rand(shape, std, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * std).to(torch.bfloat16)


def _both(attn, q, k, v, cu, kvs, pre):
    from paper_2608_26523_amd import binding as B
    attn.plan(cu, kvs, pre)
    assert attn.workspace_bytes <= B.NOALLOC_SCRATCH_BYTES
    tok = int(cu[-1])
    hq, dv = attn.cfg.num_q_heads, attn.cfg.head_dim_v
    ref = torch.full((tok, hq, dv), 7.0, dtype=torch.bfloat16, device=DEV)
    ref_lse = torch.full((hq, tok), 7.0, dtype=torch.float32, device=DEV)
    attn.run(q[:tok], k, v, ref, ref_lse)
    out = torch.full((tok, hq, dv), -3.0, dtype=torch.bfloat16, device=DEV)
    lse = torch.full((hq, tok), -3.0, dtype=torch.float32, device=DEV)
    attn.run_noalloc(q[:tok], k, v, out, lse)
    torch.cuda.synchronize()
    return ref, ref_lse, out, lse


@pytest.mark.parametrize("dims", [(128, 128), (192, 128)])
def test_noalloc_equals_run_twice_with_smaller_second_call(dims):
    from paper_2608_26523_amd.attention import ChunkAttention
    dqk, dv = dims
    hq, hkv = (8, 2) if dqk == 128 else (4, 4)
    T = 4200
    std = 1.0 / math.sqrt(dqk)
    k = _rand((T, hkv, dqk), std, 11 + dqk)
    v = _rand((T, hkv, dv), std, 12 + dqk)
    q = _rand((1024, hq, dqk), std, 13 + dqk)
    attn = ChunkAttention(hq, hkv, dqk, dv, max_chunk_tokens=1024, max_kv_len=T, num_splits=3)
    cases = [
        ("split, two segments", np.array([0, 700, 1000]), [0, 3300], [3000, 400]),
        ("smaller, one segment", np.array([0, 200]), [0], [100]),
        ("split again", np.array([0, 700, 1000]), [0, 3300], [3000, 400]),
    ]
    for what, cu, kvs, pre in cases:
        print("case:", dims, what, flush=True)
        ref, ref_lse, out, lse = _both(attn, q, k, v, cu, kvs, pre)
        assert attn.info().num_splits == (3 if pre[0] >= 192 else 1)
        assert torch.equal(out, ref), what
        assert torch.equal(lse, ref_lse), what
        assert bool(torch.isfinite(out.float()).all())

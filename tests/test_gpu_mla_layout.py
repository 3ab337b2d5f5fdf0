"""Split key layout of the MLA models (vpp_chunk_attn_run_mla) on the GPU.

K[j][h] = (k_nope[j][h][0..127], k_rope[j][0..63]): the run over the split
layout must give the same bits as the contiguous run over the concatenated keys
(the kernels do the same arithmetic; only the LDS copy of K differs), for both
tile variants, split and unsplit key ranges and multi-segment chunks, and at the
mla workload's full size. One case is also checked against the fp64 oracle.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import parity as PA

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _rand(shape, std, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * std).to(torch.bfloat16)


def _attn(hq, max_tok, max_kv, splits=1):
    from paper_2608_26523_amd.attention import ChunkAttention
    return ChunkAttention(hq, hq, 192, 128, max_chunk_tokens=max_tok, max_kv_len=max_kv, num_splits=splits)


def _split_keys(rows, heads, seed):
    std = 1.0 / math.sqrt(192)
    k_nope = _rand((rows, heads, 128), std, seed)
    k_rope = _rand((rows, 64), std, seed + 1)
    k_full = torch.cat([k_nope, k_rope.unsqueeze(1).expand(rows, heads, 64)], dim=2).contiguous()
    return k_nope, k_rope, k_full


# (heads, segments (kv_start, prefix, len), cache rows, splits)
CASES = [
    (4, [(0, 0, 300)], 300, 1),
    (2, [(0, 130, 257)], 387, 1),
    (4, [(0, 90, 300), (390, 0, 45), (435, 700, 170)], 1305, 1),
    (2, [(0, 1000, 131)], 1131, 3),
    (8, [(0, 4096, 256)], 4352, 4),
]


SPLIT_OFF = ("split key ranges are switched off for the split key layout: a run with 4 splits "
             "over a 524288-row cache faulted the GPU and its cause is not yet shown")


@pytest.mark.parametrize("nb", [1, 2])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_split_keys_equal_concatenated(case, nb, monkeypatch):
    monkeypatch.setenv("VPP_NB", str(nb))
    hq, segs, T, splits = CASES[case]
    if splits > 1:
        pytest.skip(SPLIT_OFF)
    print("case:", case, CASES[case], "nb", nb, flush=True)
    k_nope, k_rope, k_full = _split_keys(T, hq, 10 + case)
    v = _rand((T, hq, 128), 1.0 / math.sqrt(192), 20 + case)
    tok = sum(s[2] for s in segs)
    q = _rand((tok, hq, 192), 1.0 / math.sqrt(192), 30 + case)
    cu = np.cumsum([0] + [s[2] for s in segs])
    kvs, pre = [s[0] for s in segs], [s[1] for s in segs]
    attn = _attn(hq, tok, T, splits)
    attn.plan(cu, kvs, pre)
    lse_a = torch.empty((hq, tok), dtype=torch.float32, device=DEV)
    lse_b = torch.full_like(lse_a, 7.0)
    out_a, _ = attn.run(q, k_full, v, lse=lse_a)
    out_b, _ = attn.run_mla(q, k_nope, k_rope, v, lse=lse_b)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b), "split-key output differs from the concatenated keys"
    assert torch.equal(lse_a, lse_b)


def test_split_keys_vs_oracle():
    hq, T = 4, 900
    segs = [(0, 300, 200), (500, 0, 150)]
    k_nope, k_rope, k_full = _split_keys(T, hq, 40)
    v = _rand((T, hq, 128), 1.0 / math.sqrt(192), 41)
    tok = sum(s[2] for s in segs)
    q = _rand((tok, hq, 192), 1.0 / math.sqrt(192), 42)
    cu = np.cumsum([0] + [s[2] for s in segs])
    kvs, pre = [s[0] for s in segs], [s[1] for s in segs]
    attn = _attn(hq, tok, T)
    attn.plan(cu, kvs, pre)
    out, lse = attn.run_mla(q, k_nope, k_rope, v, lse=torch.empty((hq, tok), dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
    # the oracle gets the keys assembled on the host by the definition above
    kc = torch.cat([k_nope.cpu(), k_rope.cpu().unsqueeze(1).expand(T, hq, 64)], dim=2).contiguous()
    ro, rl = oracle.attention_full(q.cpu(), kc, v.cpu(), cu, kvs, pre)
    rows = np.repeat(np.arange(tok), hq)
    heads = np.tile(np.arange(hq), tok)
    rep = PA.compare(out, lse, rows, heads, ro.reshape(tok * hq, -1), rl.T.reshape(-1))
    print(rep, flush=True)
    assert rep.ok(), str(rep)


def test_split_keys_refuse_split_plans():
    """The split key layout refuses plans with a split key range (switched off, see SPLIT_OFF)."""
    from paper_2608_26523_amd import binding as B
    hq, T = 2, 1131
    k_nope, k_rope, _ = _split_keys(T, hq, 60)
    v = _rand((T, hq, 128), 0.1, 61)
    q = _rand((131, hq, 192), 0.1, 62)
    attn = _attn(hq, 131, T, splits=3)
    attn.plan([0, 131], [0], [1000])
    with pytest.raises(B.VppError) as e:
        attn.run_mla(q, k_nope, k_rope, v)
    assert e.value.status == B.VPP_ERR_UNSUPPORTED


def test_split_keys_full_size_mla_chunk():
    """mla workload, chunk 8 (prefix 65536, 8192 queries, 128 heads)."""
    from paper_2608_26523_amd import workloads as W
    w = W.get("mla")
    c = 8
    t0, cu, kvs, pre = W.chunk_segments(w, c)
    rows = int(pre[0]) + int(cu[-1])
    print("case: mla chunk", c, "rows", rows, flush=True)
    k_nope, k_rope, k_full = _split_keys(rows, w.hq, 50)
    v = W.normal_bf16((rows, w.hkv, w.dv), 1.0 / math.sqrt(w.dqk), w.seed, w.index, "v", DEV)
    q = W.make_q_rows(w, DEV, t0, t0 + int(cu[-1]))
    attn = _attn(w.hq, w.chunk, rows)
    attn.plan(cu, kvs, pre)
    out_a, _ = attn.run(q, k_full, v)
    del k_full
    out_b, _ = attn.run_mla(q, k_nope, k_rope, v)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b)

"""Split key layout of the MLA models (vpp_chunk_attn_run_mla) on the GPU.

K[j][h] = (k_nope[j][h][0..127], k_rope[j][0..63]): the run over the split
layout must give the same bits as the contiguous run over the concatenated keys
(the kernels do the same arithmetic; only the LDS copy of K differs), for both
tile variants, split and unsplit key ranges and multi-segment chunks, and at the
full sizes of the mla workload and of the long workload (the latter with the
split keys also given as views into the concatenated keys, whose row strides
make every running copy address cross 4 GiB boundaries). One case is also
checked against the fp64 oracle.
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


@pytest.mark.parametrize("nb", [1, 2])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_split_keys_equal_concatenated(case, nb, monkeypatch):
    monkeypatch.setenv("VPP_NB", str(nb))
    hq, segs, T, splits = CASES[case]
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


def test_split_keys_full_size_long_chunk():
    """long workload, last chunk (prefix 507904, 16384 queries, 128 heads, 4 splits):
    the split keys as contiguous tensors and as strided views into the concatenated
    keys (a 24 GiB span, so 64-bit address arithmetic carries in every copy stream)."""
    from paper_2608_26523_amd import workloads as W
    w = W.get("long")
    c = W.num_chunks(w) - 1
    t0, cu, kvs, pre = W.chunk_segments(w, c)
    rows = int(pre[0]) + int(cu[-1])
    print("case: long chunk", c, "rows", rows, "splits", w.num_splits, flush=True)
    std = 1.0 / math.sqrt(w.dqk)
    k_full = W.normal_bf16((rows, w.hkv, w.dqk), std, w.seed, w.index, "k", DEV)
    k_full[:, 1:, 128:] = k_full[:, :1, 128:]          # one shared rope part per row
    v = W.normal_bf16((rows, w.hkv, w.dv), std, w.seed, w.index, "v", DEV)
    q = W.make_q_rows(w, DEV, t0, t0 + int(cu[-1]))
    nope_view, rope_view = k_full[:, :, :128], k_full[:, 0, 128:]
    assert nope_view.stride(0) == w.hkv * 192 and rope_view.stride(0) == w.hkv * 192
    k_nope, k_rope = nope_view.contiguous(), rope_view.contiguous()
    from paper_2608_26523_amd.attention import ChunkAttention
    attn = ChunkAttention(w.hq, w.hkv, w.dqk, w.dv, max_chunk_tokens=w.chunk, max_kv_len=rows,
                          num_splits=w.num_splits)
    attn.plan(cu, kvs, pre)
    assert attn.info().num_splits == w.num_splits
    tok = int(cu[-1])
    lse = [torch.full((w.hq, tok), float(i), dtype=torch.float32, device=DEV) for i in range(3)]
    out_a, _ = attn.run(q, k_full, v, lse=lse[0])
    out_b, _ = attn.run_mla(q, nope_view, rope_view, v, lse=lse[1])
    out_c, _ = attn.run_mla(q, k_nope, k_rope, v, lse=lse[2])
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out_a).all())
    assert torch.equal(out_a, out_b), "strided split keys differ from the concatenated keys"
    assert torch.equal(out_a, out_c), "contiguous split keys differ from the concatenated keys"
    assert torch.equal(lse[0], lse[1]) and torch.equal(lse[0], lse[2])
    del k_full, k_nope, k_rope, v, q
    torch.cuda.empty_cache()

"""HIP path vs the fp64 oracle at the workloads' full sizes (GPU).

Each workload runs with the head configuration, chunk size, cache length and
split request that the benchmark uses, on every chunk of gqa, mla and long and
on selected mixed chunks. The oracle evaluates a seeded sample of (row, head)
items per chunk (tile edges, segment ends, heads of several kv groups, random
rows), and every item of gqa's first two chunks; the other outputs of the
sampled chunks are checked against properties that hold at any size (on a
subset of chunks for the long prompts, where they cost the most):

* each output element is a convex combination of the visible values of its
  column, so it lies within [min, max] of that column over the cache rows the
  chunk can reach (plus one bf16 rounding);
* lse_i - ln(i + 1) lies within [min_j s_ij, max_j s_ij], and
  |s_ij| <= scale * |q_i| * max_j |k_j| (Cauchy-Schwarz).
"""
import math

import numpy as np
import pytest
import torch

import parity as PA

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _attn(w, max_kv):
    from paper_2608_26523_amd.attention import ChunkAttention
    return ChunkAttention(w.hq, w.hkv, w.dqk, w.dv, max_chunk_tokens=w.chunk,
                          max_kv_len=max_kv, num_splits=w.num_splits)


def _kv(w, rows):
    from paper_2608_26523_amd import workloads as W
    std = 1.0 / math.sqrt(w.dqk)
    k = W.normal_bf16((rows, w.hkv, w.dqk), std, w.seed, w.index, "k", DEV)
    v = W.normal_bf16((rows, w.hkv, w.dv), std, w.seed, w.index, "v", DEV)
    return k, v


def _properties(w, q, k, v, cu, kvs, pre, out, lse):
    """Bounds every output must satisfy (see the module docstring)."""
    tok = int(cu[-1])
    g = w.group
    assert bool(torch.isfinite(out[:tok]).all()), "non-finite output"
    assert bool(torch.isfinite(lse[:, :tok]).all()), "non-finite lse"
    for s in range(len(kvs)):
        r0, r1 = int(cu[s]), int(cu[s + 1])
        if r0 == r1:
            continue
        a, p = int(kvs[s]), int(pre[s])
        vis = slice(a, a + p + (r1 - r0))
        vmin = v[vis].float().amin(0).repeat_interleave(g, 0)          # [Hq, dv]
        vmax = v[vis].float().amax(0).repeat_interleave(g, 0)
        o = out[r0:r1].float()
        slack = (vmax.abs().amax() + vmin.abs().amax()) * 2.0 ** -8
        assert bool((o >= vmin - slack).all()) and bool((o <= vmax + slack).all()), \
            "segment %d: output outside the convex hull of its values" % s
        kn = k[vis].float().norm(dim=2).amax(0).repeat_interleave(g, 0)  # [Hq]
        qn = q[r0:r1].float().norm(dim=2)                               # [rows, Hq]
        bound = (w.scale * qn * kn).t()                                 # [Hq, rows]
        pos = torch.arange(p, p + r1 - r0, device=DEV, dtype=torch.float64)
        dev = lse[:, r0:r1].double() - torch.log(pos + 1).unsqueeze(0)
        assert bool((dev.abs() <= bound.double() * (1 + 1e-3) + 1e-3).all()), \
            "segment %d: lse outside its Cauchy-Schwarz bound" % s


def _check_chunk(w, attn, q, k, v, cu, kvs, pre, what, seed, properties=True):
    print("case:", what, flush=True)
    out, lse = PA.run_chunk(attn, q, k, v, cu, kvs, pre)
    rows, heads = PA.sample_items(cu, kvs, pre, w.hq, w.hkv, seed=seed)
    ro, rl = PA.oracle_items(q, k, v, cu, kvs, pre, rows, heads, scale=w.scale)
    rep = PA.compare(out, lse, rows, heads, ro, rl)
    print(what, "splits=%d" % attn.info().num_splits, rep, flush=True)
    assert rep.ok(), "%s: %s" % (what, rep)
    if properties:
        _properties(w, q, k, v, cu, kvs, pre, out, lse)
    else:
        assert bool(torch.isfinite(out.float()).all()) and bool(torch.isfinite(lse[:, :int(cu[-1])]).all())
    return attn.info()


def _single_request(name, chunks, properties=None):
    """Sampled oracle parity on the given chunks; the any-size property checks on the
    chunks in `properties` (default: all of them)."""
    from paper_2608_26523_amd import workloads as W
    w = W.get(name)
    hi = (max(chunks) + 1) * w.chunk
    k, v = _kv(w, hi)
    attn = _attn(w, w.seq_len)
    infos = []
    for c in chunks:
        t0, cu, kvs, pre = W.chunk_segments(w, c)
        q = W.make_q_rows(w, DEV, t0, t0 + int(cu[-1]))
        infos.append(_check_chunk(w, attn, q, k, v, cu, kvs, pre,
                                  "%s chunk %d prefix %d" % (name, c, int(pre[0])), seed=c,
                                  properties=properties is None or c in properties))
        del q
    del k, v
    torch.cuda.empty_cache()
    return infos


def test_gqa_every_chunk():
    from paper_2608_26523_amd import workloads as W
    _single_request("gqa", list(range(W.num_chunks(W.get("gqa")))))


def test_gqa_first_chunks_every_item():
    """gqa chunks 0 and 1 compared with the oracle on every (row, head): 4096 rows x 32
    heads each, about 5e11 fp64 flop on the host."""
    from paper_2608_26523_amd import workloads as W
    w = W.get("gqa")
    k, v = _kv(w, 2 * w.chunk)
    attn = _attn(w, w.seq_len)
    for c in (0, 1):
        t0, cu, kvs, pre = W.chunk_segments(w, c)
        tok = int(cu[-1])
        q = W.make_q_rows(w, DEV, t0, t0 + tok)
        print("case: gqa chunk %d, every item" % c, flush=True)
        out, lse = PA.run_chunk(attn, q, k, v, cu, kvs, pre)
        rows = np.repeat(np.arange(tok, dtype=np.int64), w.hq)
        heads = np.tile(np.arange(w.hq, dtype=np.int32), tok)
        ro, rl = PA.oracle_items(q, k, v, cu, kvs, pre, rows, heads, scale=w.scale)
        rep = PA.compare(out, lse, rows, heads, ro, rl)
        print("gqa chunk %d every item:" % c, rep, flush=True)
        assert rep.n_items == tok * w.hq and rep.ok(), rep


def test_mla_every_chunk():
    from paper_2608_26523_amd import workloads as W
    n = W.num_chunks(W.get("mla"))
    _single_request("mla", list(range(n)), properties={0, 1, 8, n - 1})


def test_long_every_chunk_split():
    from paper_2608_26523_amd import workloads as W
    n = W.num_chunks(W.get("long"))
    infos = _single_request("long", list(range(n)), properties={0, 4, 16, n - 1})
    # a prefix of at least 4 key tiles gets the requested 4-way split
    assert infos[0].num_splits == 1 and all(i.num_splits == 4 for i in infos[1:])


def test_mixed_chunks():
    """Sampled oracle parity on the mixed workload's packed chunks: the first and last, the
    one packing most requests, the deepest single-request chunk, every chunk of three or
    more requests, every chunk the automatic split count cuts, and every 32nd chunk."""
    from paper_2608_26523_amd import binding as B
    from paper_2608_26523_amd import workloads as W
    w = W.get("mixed")
    n = W.num_chunks(w)
    segs = [W.chunk_segments(w, c) for c in range(n)]
    most = max(range(n), key=lambda c: len(segs[c][2]))
    single = [c for c in range(n) if len(segs[c][2]) == 1]
    deepest = max(single, key=lambda c: int(segs[c][3][0]))
    assert int(segs[deepest][3][0]) >= 65536
    assert int(segs[n - 1][1][-1]) < w.chunk or W.total_tokens(w) % w.chunk == 0
    # the split counts the planner picks (host only)
    cfg = B.Config(num_q_heads=w.hq, num_kv_heads=w.hkv, head_dim_qk=w.dqk, head_dim_v=w.dv,
                   softmax_scale=0.0, causal=1, max_chunk_tokens=w.chunk, max_segments=256,
                   max_kv_len=W.total_tokens(w), num_splits=w.num_splits)
    planned = {}
    for c in range(n):
        h, _ = B.vpp_chunk_attn_plan(cfg, segs[c][1], segs[c][2], segs[c][3])
        planned[c] = B.vpp_chunk_attn_plan_info(h).num_splits
        B.vpp_chunk_attn_destroy(h)
    split = [c for c in range(n) if planned[c] > 1]
    packed = [c for c in range(n) if len(segs[c][2]) >= 3]
    # chunk 98: 43 rows behind a 118844-key prefix next to two short requests; the
    # simulated launch cuts it four ways
    assert 98 in split and len(split) >= 8 and len(packed) >= 8
    picks = sorted({0, most, deepest, n - 1} | set(split) | set(packed) | set(range(0, n, 32)))
    k, v = _kv(w, W.total_tokens(w))
    attn = _attn(w, W.total_tokens(w))
    for c in picks:
        t0, cu, kvs, pre = segs[c]
        q = W.make_q_rows(w, DEV, t0, t0 + int(cu[-1]))
        info = _check_chunk(w, attn, q, k, v, cu, kvs, pre,
                            "mixed chunk %d (%d segments, first prefix %d)" % (c, len(kvs), int(pre[0])),
                            seed=c, properties=c in {0, most, deepest, 98, n - 1})
        assert info.num_splits == planned[c]
        del q
    del k, v
    torch.cuda.empty_cache()

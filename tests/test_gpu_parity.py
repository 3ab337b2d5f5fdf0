"""HIP path vs the fp64 oracle, element by element, on small and ragged chunks (GPU).

Sizes are chosen so the oracle evaluates every (row, head) item in seconds while
the chunks still span several 128-row query tiles, several 64-key tiles and a
ragged tail; every supported head-dim pair, GQA and MHA, multi-segment packed
chunks, zero-length segments and forced split counts are covered.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import parity as PA

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _attn(hq, hkv, dqk, dv, max_tok, max_kv, splits=-1, scale=0.0):
    from paper_2608_26523_amd.attention import ChunkAttention
    return ChunkAttention(hq, hkv, dqk, dv, max_chunk_tokens=max_tok, max_kv_len=max_kv,
                          num_splits=splits, softmax_scale=scale)


def _rand(shape, std, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * std).to(torch.bfloat16)


def _full_check(attn, q, k, v, cu, kvs, pre, scale=None, what=""):
    print("case:", what, flush=True)
    out, lse = PA.run_chunk(attn, q, k, v, cu, kvs, pre)
    ro, rl = oracle.attention_full(q[:int(cu[-1])].cpu(), k.cpu(), v.cpu(), cu, kvs, pre,
                                   scale=scale)
    hq = q.shape[1]
    tok = int(cu[-1])
    rows = np.repeat(np.arange(tok), hq)
    heads = np.tile(np.arange(hq), tok)
    rep = PA.compare(out, lse, rows, heads, ro.reshape(tok * hq, -1), rl.T.reshape(-1))
    print(what, rep, flush=True)
    assert rep.ok(), "%s: %s" % (what, rep)
    return out, lse


def test_library_loaded_is_in_tree():
    from paper_2608_26523_amd import binding
    lib = binding.load()
    assert lib._name == binding.LIB_PATH


def test_tiny_workload_all_chunks():
    from paper_2608_26523_amd import workloads as W
    w = W.get("tiny")
    q, k, v = W.make_inputs(w, DEV)
    attn = _attn(w.hq, w.hkv, w.dqk, w.dv, w.chunk, w.seq_len)
    for c in range(W.num_chunks(w)):
        t0, cu, kvs, pre = W.chunk_segments(w, c)
        _full_check(attn, q[t0:], k, v, cu, kvs, pre, what="tiny chunk %d" % c)


CASES = [
    # (hq, hkv, dqk, dv, segments (kv_start, prefix, len), cache rows, splits)
    (4, 4, 64, 64, [(0, 0, 300)], 300, 1),
    (4, 1, 128, 128, [(0, 77, 200)], 277, 1),
    (2, 2, 192, 128, [(0, 130, 257)], 387, 1),
    (8, 2, 128, 128, [(0, 0, 100), (100, 0, 37), (137, 500, 90)], 727, -1),
    (2, 2, 192, 128, [(0, 63, 1), (64, 0, 0), (64, 5, 129)], 198, 1),
    (4, 2, 128, 128, [(0, 700, 150)], 850, 2),
    (2, 1, 192, 128, [(0, 1000, 131), (1131, 0, 64)], 1195, 3),
    (4, 4, 64, 64, [(0, 20, 40), (60, 300, 200)], 560, 5),
    (2, 2, 128, 128, [(0, 0, 10)], 10, 4),        # more splits than key tiles
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_ragged_cases(case):
    hq, hkv, dqk, dv, segs, T, splits = CASES[case]
    tok = sum(s[2] for s in segs)
    std = 1.0 / math.sqrt(dqk)
    q = _rand((tok, hq, dqk), std, 100 + case)
    k = _rand((T, hkv, dqk), std, 200 + case)
    v = _rand((T, hkv, dv), std, 300 + case)
    cu = np.cumsum([0] + [s[2] for s in segs])
    kvs = [s[0] for s in segs]
    pre = [s[1] for s in segs]
    attn = _attn(hq, hkv, dqk, dv, max(tok, 1), T, splits=splits)
    _full_check(attn, q, k, v, cu, kvs, pre, what="case %d %s" % (case, CASES[case]))
    info = attn.info()
    if splits >= 1:
        assert info.num_splits == PA.planned_splits(splits, pre, [s[2] for s in segs])


def test_zero_keys_count_visible_keys():
    """K == 0: lse = ln(i+1) exactly up to fp32 rounding; out = running mean of V."""
    hq, dqk, dv, p, L = 2, 128, 128, 1000, 300
    T = p + L
    q = _rand((L, hq, dqk), 1 / math.sqrt(dqk), 7)
    k = torch.zeros((T, 1, dqk), dtype=torch.bfloat16, device=DEV)
    v = _rand((T, 1, dv), 1.0, 8)
    attn = _attn(hq, 1, dqk, dv, L, T)
    out, lse = PA.run_chunk(attn, q, k, v, [0, L], [0], [p])
    pos = torch.arange(p, p + L, device=DEV, dtype=torch.float64)
    want = torch.log(pos + 1)
    err = (lse.double() - want.unsqueeze(0)).abs()
    ulp = torch.finfo(torch.float32).eps * want.abs().max()
    assert float(err.max()) <= 4 * float(ulp) + 1e-6, float(err.max())
    mean = torch.cumsum(v[:, 0].double(), 0) / torch.arange(1, T + 1, device=DEV).unsqueeze(1)
    ref = mean[p:p + L].unsqueeze(1).expand(L, hq, dv)
    assert float((out.double() - ref).abs().max()) <= 2e-2


def test_unit_values_give_ones():
    hq, dqk, dv, p, L = 4, 192, 128, 333, 260
    T = p + L
    q = _rand((L, hq, dqk), 1.0, 9)       # large scores: far from uniform
    k = _rand((T, hq, dqk), 1.0, 10)
    v = torch.ones((T, hq, dv), dtype=torch.bfloat16, device=DEV)
    attn = _attn(hq, hq, dqk, dv, L, T)
    out, _ = PA.run_chunk(attn, q, k, v, [0, L], [0], [p])
    assert float((out.double() - 1).abs().max()) <= 4e-3


def test_planted_keys_no_leak():
    """q_i parallel to a chosen key: out_i == v_{j*}; j* on the diagonal, the first key,
    a key of the previous request in the same chunk must not be reachable."""
    d, dv = 128, 128
    T = 1024
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 2, size=(T, d)) * 2 - 1
    kk = torch.tensor(codes / 8.0, dtype=torch.float32)             # |k|^2 = 2
    k = kk.to(torch.bfloat16).unsqueeze(1).to(DEV)
    v = _rand((T, 1, dv), 1.0, 11)
    # two requests packed in one chunk: request A = rows 0..399, request B = 400..1023
    segs = [(0, 300, 100), (400, 0, 624)]
    cu = [0, 100, 724]
    targets = []
    for (base, p, L) in segs:
        for r in range(L):
            i = p + r
            j = i if r % 3 == 0 else (0 if r % 3 == 1 else int(rng.integers(0, i + 1)))
            targets.append(base + j)
    targets = np.array(targets)
    q = (kk[targets] * 40.0).to(torch.bfloat16).unsqueeze(1).to(DEV)  # score 80 vs <= ~50
    attn = _attn(1, 1, d, dv, 724, T, scale=1.0)
    out, _ = PA.run_chunk(attn, q, k, v, cu, [s[0] for s in segs], [s[1] for s in segs])
    want = v[torch.as_tensor(targets, device=DEV), 0]
    err = (out[:, 0].double() - want.double()).abs().max()
    assert float(err) <= 1e-2, float(err)


@pytest.mark.parametrize("nb", [1, 2])
@pytest.mark.parametrize("splits", [2, 3, 4])
def test_planted_keys_across_split_pieces(splits, nb, monkeypatch):
    """Forced splits: q_i parallel to a key j* that lies in a split piece other than the
    last, at piece boundaries and key-tile edges (64m - 1, 64m), at key 0, at random
    earlier keys and on the diagonal. out_i must be v_{j*}; the result must also match
    the oracle on every item. Several query tiles, so some slots run a tile's keys in
    descending order."""
    monkeypatch.setenv("VPP_NB", str(nb))
    d, dv = 128, 128
    p, L = 3000, 700
    T = p + L
    rng = np.random.default_rng(40 + splits)
    codes = rng.integers(0, 2, size=(T, d)) * 2 - 1
    kk = torch.tensor(codes / 8.0, dtype=torch.float32)             # |k|^2 = 2
    k = kk.to(torch.bfloat16).unsqueeze(1).to(DEV)
    v = _rand((T, 1, dv), 1.0, 41 + splits)
    # piece boundaries of an n-way split of the 3000-key prefix (tile-aligned)
    bounds = [((p // 64) * b // splits) * 64 for b in range(1, splits)]
    special = [0, 63, 64, 127, 128] + [x for b in bounds for x in (b - 1, b, b + 63, b + 64)]
    targets = []
    for r in range(L):
        i = p + r
        if r % 4 == 0:
            j = i                                         # the diagonal
        elif r % 4 == 1:
            j = special[(r // 4) % len(special)]          # edges of pieces and tiles
        elif r % 4 == 2:
            j = int(rng.integers(0, bounds[-1]))          # somewhere before the last piece
        else:
            j = int(rng.integers(0, i + 1))
        targets.append(j)
    targets = np.array(targets)
    assert all(b in targets or b - 1 in targets for b in bounds)
    q = (kk[targets] * 40.0).to(torch.bfloat16).unsqueeze(1).to(DEV)  # score 80 vs <= ~50
    attn = _attn(1, 1, d, dv, L, T, splits=splits, scale=1.0)
    out, lse = PA.run_chunk(attn, q, k, v, [0, L], [0], [p])
    info = attn.info()
    assert info.num_splits == splits and info.block_m == 128 * nb
    want = v[torch.as_tensor(targets, device=DEV), 0]
    err = (out[:, 0].double() - want.double()).abs().max()
    assert float(err) <= 1e-2, float(err)
    _full_check(attn, q, k, v, np.array([0, L]), [0], [p], scale=1.0,
                what="planted keys, %d splits, nb %d" % (splits, nb))


def test_split_matches_unsplit_and_determinism():
    hq, hkv, dqk, dv, p, L = 8, 2, 128, 128, 4000, 384
    T = p + L
    std = 1 / math.sqrt(dqk)
    q = _rand((L, hq, dqk), std, 12)
    k = _rand((T, hkv, dqk), std, 13)
    v = _rand((T, hkv, dv), std, 14)
    a1 = _attn(hq, hkv, dqk, dv, L, T, splits=1)
    o1, l1 = PA.run_chunk(a1, q, k, v, [0, L], [0], [p])
    o1b, l1b = PA.run_chunk(a1, q, k, v, [0, L], [0], [p])
    assert torch.equal(o1, o1b) and torch.equal(l1, l1b), "two runs differ"
    for n in (2, 7):
        an = _attn(hq, hkv, dqk, dv, L, T, splits=n)
        on, ln = PA.run_chunk(an, q, k, v, [0, L], [0], [p])
        assert float((on.double() - o1.double()).abs().max()) <= 8e-3
        assert float((ln - l1).abs().max()) <= 1e-4


def test_chunked_equals_unchunked():
    hq, hkv, dqk, dv, S, C = 4, 2, 128, 128, 1024, 256
    std = 1 / math.sqrt(dqk)
    q = _rand((S, hq, dqk), std, 15)
    k = _rand((S, hkv, dqk), std, 16)
    v = _rand((S, hkv, dv), std, 17)
    full = _attn(hq, hkv, dqk, dv, S, S, splits=1)
    of, lf = PA.run_chunk(full, q, k, v, [0, S], [0], [0])
    ch = _attn(hq, hkv, dqk, dv, C, S, splits=1)
    for c0 in range(0, S, C):
        oc, lc = PA.run_chunk(ch, q[c0:], k, v, [0, C], [0], [c0])
        # tile-aligned chunk boundaries, no split: the same products, summed in an order
        # that differs only where a tile runs its keys in the other direction (a slot's
        # second tile streams them descending, and the partner depends on the chunk), so
        # the results agree to rounding: a bf16 ulp of out (|out| < 0.5 here) and fp32
        # rounding of lse
        assert float((oc.double() - of[c0:c0 + C].double()).abs().max()) <= 2.0 ** -9, "chunk at %d" % c0
        assert float((lc - lf[:, c0:c0 + C]).abs().max()) <= 1e-5


def test_gqa_equals_replicated_mha():
    hq, hkv, dqk, dv, p, L = 8, 2, 128, 128, 200, 200
    T = p + L
    std = 1 / math.sqrt(dqk)
    q = _rand((L, hq, dqk), std, 18)
    k = _rand((T, hkv, dqk), std, 19)
    v = _rand((T, hkv, dv), std, 20)
    g = _attn(hq, hkv, dqk, dv, L, T, splits=1)
    og, lg = PA.run_chunk(g, q, k, v, [0, L], [0], [p])
    m = _attn(hq, hq, dqk, dv, L, T, splits=1)
    om, lm = PA.run_chunk(m, q, k.repeat_interleave(hq // hkv, 1).contiguous(),
                          v.repeat_interleave(hq // hkv, 1).contiguous(), [0, L], [0], [p])
    assert torch.equal(og, om) and torch.equal(lg, lm)


def test_packed_equals_per_request():
    hq, hkv, dqk, dv = 4, 1, 128, 128
    lens = [300, 77, 500]
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    T = int(sum(lens))
    std = 1 / math.sqrt(dqk)
    q = _rand((T, hq, dqk), std, 21)
    k = _rand((T, hkv, dqk), std, 22)
    v = _rand((T, hkv, dv), std, 23)
    t0, t1 = 200, 700
    cu, kvs, pre = [0], [], []
    for a, L in zip(starts, lens):
        lo, hi = max(a, t0), min(a + L, t1)
        if lo < hi:
            cu.append(cu[-1] + hi - lo)
            kvs.append(int(a))
            pre.append(int(lo - a))
    pk = _attn(hq, hkv, dqk, dv, t1 - t0, T, splits=1)
    op, lp = PA.run_chunk(pk, q[t0:], k, v, cu, kvs, pre)
    for s in range(len(kvs)):
        a = kvs[s]
        n = cu[s + 1] - cu[s]
        one = _attn(hq, hkv, dqk, dv, n, T, splits=1)
        o1, l1 = PA.run_chunk(one, q[a + pre[s]:], k, v, [0, n], [a], [pre[s]])
        assert float((op[cu[s]:cu[s + 1]].double() - o1.double()).abs().max()) == 0.0
        assert float((lp[:, cu[s]:cu[s + 1]] - l1).abs().max()) == 0.0


@pytest.mark.parametrize("nb", [1, 2])
@pytest.mark.parametrize("dims", [(64, 64), (128, 128), (192, 128)])
def test_both_tile_variants(nb, dims, monkeypatch):
    """Both kernel variants (32-row and 64-row waves), forced, on a ragged packed chunk."""
    monkeypatch.setenv("VPP_NB", str(nb))
    dqk, dv = dims
    hq, hkv = 4, 2
    segs = [(0, 90, 300), (390, 0, 45), (435, 700, 170)]
    T = 435 + 700 + 170
    tok = sum(s[2] for s in segs)
    std = 1.0 / math.sqrt(dqk)
    q = _rand((tok, hq, dqk), std, 400 + dqk + nb)
    k = _rand((T, hkv, dqk), std, 500 + dqk + nb)
    v = _rand((T, hkv, dv), std, 600 + dqk + nb)
    cu = np.cumsum([0] + [s[2] for s in segs])
    attn = _attn(hq, hkv, dqk, dv, tok, T, splits=1)
    _full_check(attn, q, k, v, cu, [s[0] for s in segs], [s[1] for s in segs],
                what="nb=%d dims=%s" % (nb, dims))
    assert attn.info().block_m == 32 * nb * 4


@pytest.mark.parametrize("nb", [1, 2])
@pytest.mark.parametrize("dims", [(64, 64), (192, 128)])
def test_tile_variants_split(nb, dims, monkeypatch):
    """Both kernel variants with the key range of one ragged request split three ways."""
    monkeypatch.setenv("VPP_NB", str(nb))
    dqk, dv = dims
    hq, hkv = 2, 1
    prefix, rows = 1000, 300
    T = prefix + rows
    std = 1.0 / math.sqrt(dqk)
    q = _rand((rows, hq, dqk), std, 700 + dqk + nb)
    k = _rand((T, hkv, dqk), std, 800 + dqk + nb)
    v = _rand((T, hkv, dv), std, 900 + dqk + nb)
    cu = np.array([0, rows])
    attn = _attn(hq, hkv, dqk, dv, rows, T, splits=3)
    _full_check(attn, q, k, v, cu, [0], [prefix], what="split nb=%d dims=%s" % (nb, dims))
    assert attn.info().num_splits == 3


def _random_mix(seed):
    """A seeded random chunk: 1-4 segments (empty ones allowed), ragged lengths,
    prefixes up to 1500 rows, one of the head and dim pairs, a split count."""
    rng = np.random.default_rng(seed)
    heads = [(4, 4), (8, 2), (6, 3), (2, 1)][rng.integers(4)]
    dims = [(64, 64), (128, 128), (192, 128)][rng.integers(3)]
    n = int(rng.integers(1, 5))
    segs, row = [], 0
    for _ in range(n):
        ln = int(rng.integers(0, 300)) if rng.random() > 0.15 else 0
        p = int(rng.integers(0, 1500)) if rng.random() > 0.25 else 0
        segs.append((row, p, ln))
        row += p + ln + int(rng.integers(0, 40))
    if sum(s[2] for s in segs) == 0:
        segs[0] = (segs[0][0], segs[0][1], 1 + int(rng.integers(0, 200)))
        row = max(row, segs[0][0] + segs[0][1] + segs[0][2])
    splits = [-1, 1, 2, 3][rng.integers(4)]
    nb = [1, 2][rng.integers(2)]
    return heads, dims, segs, row, splits, nb


@pytest.mark.parametrize("seed", range(12))
def test_random_mixes(seed, monkeypatch):
    (hq, hkv), (dqk, dv), segs, T, splits, nb = _random_mix(seed)
    monkeypatch.setenv("VPP_NB", str(nb))
    tok = sum(s[2] for s in segs)
    std = 1.0 / math.sqrt(dqk)
    q = _rand((tok, hq, dqk), std, 400 + seed)
    k = _rand((T, hkv, dqk), std, 500 + seed)
    v = _rand((T, hkv, dv), std, 600 + seed)
    cu = np.cumsum([0] + [s[2] for s in segs])
    attn = _attn(hq, hkv, dqk, dv, tok, T, splits=splits)
    _full_check(attn, q, k, v, cu, [s[0] for s in segs], [s[1] for s in segs],
                what="random mix %d: heads %d/%d dims %d/%d nb %d splits %d segs %s" %
                (seed, hq, hkv, dqk, dv, nb, splits, segs))


def test_side_stream_and_growing_workspace():
    """Runs on a side stream (default priority), with a re-plan that grows the workspace in
    between, give the same bits as runs on torch's current stream; device="cuda" without an
    index resolves to the current device."""
    from paper_2608_26523_amd.attention import ChunkAttention
    hq, hkv, d = 4, 2, 128
    std = 1.0 / math.sqrt(d)
    T = 3000
    k = _rand((T, hkv, d), std, 700)
    v = _rand((T, hkv, d), std, 701)
    q = _rand((1024, hq, d), std, 702)
    # the second case splits its 2600-key prefix (few workgroups): more workspace
    cases = [([0, 200], [0], [100]), ([0, 300], [0], [2600])]
    ref = []
    a_ref = ChunkAttention(hq, hkv, d, d, max_chunk_tokens=1024, max_kv_len=T, device="cuda")
    assert a_ref.device == torch.device("cuda", torch.cuda.current_device())
    for cu, ks, pl in cases:
        a_ref.plan(cu, ks, pl)
        ref.append(a_ref.run(q[:cu[-1]], k, v)[0].clone())
    side = torch.cuda.Stream()
    a = ChunkAttention(hq, hkv, d, d, max_chunk_tokens=1024, max_kv_len=T)
    outs = []
    for cu, ks, pl in cases:
        ws_before = a.workspace_bytes
        a.plan(cu, ks, pl)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            o, _ = a.run(q[:cu[-1]], k, v, stream=side)
        outs.append(o)
    assert a.workspace_bytes > ws_before
    torch.cuda.synchronize()
    for o, r in zip(outs, ref):
        assert torch.equal(o, r)

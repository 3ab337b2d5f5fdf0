"""Paged KV cache on the GPU: vpp_chunk_attn_run_paged and vpp_kv_append_paged.

* The paged run must give the same bits as the contiguous run over the same
  rows (the kernels do the same arithmetic in the same order; only the copy
  addresses differ), for every head-dim pair, both tile variants, split and
  unsplit, several page sizes and multi-segment chunks with one block-table row
  per segment, pages in random order.
* One case per head-dim pair is also checked against the fp64 oracle on the
  rows gathered by the reference page mapping (oracle/paged.py).
* The append kernel must write exactly the reference scatter (bit-exact),
  leave every other slot untouched and skip slot -1; chunk-by-chunk append +
  paged attention must equal the contiguous path.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import parity as PA
from oracle import paged as OP

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _rand(shape, std, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=DEV) * std).to(torch.bfloat16)


def _attn(hq, hkv, dqk, dv, max_tok, max_kv, splits=-1):
    from paper_2608_26523_amd.attention import ChunkAttention
    return ChunkAttention(hq, hkv, dqk, dv, max_chunk_tokens=max_tok, max_kv_len=max_kv,
                          num_splits=splits)


def _paginate(k, v, seg_rows, kv_start, page, seed, extra_pages=3):
    """Scatter each segment's cache rows [kv_start, kv_start + rows) into pages in a
    random order. Returns k_pages, v_pages, block_table (device int32) and the host
    table."""
    rng = np.random.default_rng(seed)
    per_seg = [int(math.ceil(r / page)) for r in seg_rows]
    width = max(per_seg)
    total = sum(per_seg) + extra_pages
    perm = rng.permutation(total)
    bt = np.zeros((len(seg_rows), width), dtype=np.int32)
    pos = 0
    for s, n in enumerate(per_seg):
        bt[s, :n] = perm[pos:pos + n]
        bt[s, n:] = perm[pos]               # padding entries: a valid page
        pos += n
    hkv, dqk, dv = k.shape[1], k.shape[2], v.shape[2]
    # garbage in every page first, so any read of a wrong page shows
    k_pages = _rand((total, page, hkv, dqk), 3.0, seed + 1)
    v_pages = _rand((total, page, hkv, dv), 3.0, seed + 2)
    for s, rows in enumerate(seg_rows):
        for i in range(per_seg[s]):
            r0, r1 = i * page, min(rows, (i + 1) * page)
            src0 = kv_start[s] + r0
            k_pages[int(bt[s, i]), :r1 - r0] = k[src0:src0 + r1 - r0]
            v_pages[int(bt[s, i]), :r1 - r0] = v[src0:src0 + r1 - r0]
    return k_pages, v_pages, torch.as_tensor(bt, device=DEV), bt


def _run_both(attn, q, k, v, k_pages, v_pages, bt_dev, cu, kvs_contig, kvs_paged, pre):
    tok = int(cu[-1])
    hq = q.shape[1]
    out_c = torch.empty((tok, hq, v.shape[2]), dtype=torch.bfloat16, device=DEV)
    lse_c = torch.empty((hq, tok), dtype=torch.float32, device=DEV)
    attn.plan(cu, kvs_contig, pre)
    attn.run(q, k, v, out_c, lse_c)
    out_p = torch.full_like(out_c, 7.0)
    lse_p = torch.full_like(lse_c, 7.0)
    attn.plan(cu, kvs_paged, pre)
    attn.run_paged(q, k_pages, v_pages, bt_dev, out_p, lse_p)
    torch.cuda.synchronize()
    return out_c, lse_c, out_p, lse_p


# (hq, hkv, dqk, dv, segments (prefix, len), page, splits)
CASES = [
    (4, 2, 64, 64, [(90, 300), (0, 45), (700, 170)], 64, 1),
    (4, 2, 128, 128, [(90, 300), (0, 45), (700, 170)], 128, 1),
    (2, 2, 192, 128, [(130, 257), (5, 1)], 256, 1),
    (4, 1, 128, 128, [(1000, 131)], 64, 3),
    (2, 1, 192, 128, [(2000, 64), (63, 100)], 512, 2),
    (8, 2, 64, 64, [(4096, 256)], 1024, 4),
]


@pytest.mark.parametrize("nb", [1, 2])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_paged_equals_contiguous(case, nb, monkeypatch):
    monkeypatch.setenv("VPP_NB", str(nb))
    hq, hkv, dqk, dv, segs, page, splits = CASES[case]
    print("case:", case, CASES[case], "nb", nb, flush=True)
    std = 1.0 / math.sqrt(dqk)
    seg_rows = [p + n for (p, n) in segs]
    kv_contig = list(np.cumsum([0] + seg_rows[:-1]))
    T = sum(seg_rows)
    k = _rand((T, hkv, dqk), std, 10 + case)
    v = _rand((T, hkv, dv), std, 20 + case)
    tok = sum(n for (_, n) in segs)
    q = _rand((tok, hq, dqk), std, 30 + case)
    cu = np.cumsum([0] + [n for (_, n) in segs])
    pre = [p for (p, _) in segs]
    k_pages, v_pages, bt_dev, _ = _paginate(k, v, seg_rows, kv_contig, page, 40 + case)
    attn = _attn(hq, hkv, dqk, dv, tok, T, splits=splits)
    out_c, lse_c, out_p, lse_p = _run_both(attn, q, k, v, k_pages, v_pages, bt_dev, cu, kv_contig,
                                           [0] * len(segs), pre)
    assert torch.equal(out_c, out_p), "paged output differs from contiguous"
    assert torch.equal(lse_c, lse_p), "paged lse differs from contiguous"
    if splits > 1:
        assert attn.info().num_splits == splits


@pytest.mark.parametrize("dims", [(64, 64), (128, 128), (192, 128)])
def test_paged_vs_oracle(dims):
    dqk, dv = dims
    hq, hkv, page = 4, 2, 128
    segs = [(200, 150), (0, 70), (333, 90)]
    print("case: paged oracle", dims, flush=True)
    std = 1.0 / math.sqrt(dqk)
    seg_rows = [p + n for (p, n) in segs]
    kv_contig = list(np.cumsum([0] + seg_rows[:-1]))
    T = sum(seg_rows)
    k = _rand((T, hkv, dqk), std, 50 + dqk)
    v = _rand((T, hkv, dv), std, 60 + dqk)
    tok = sum(n for (_, n) in segs)
    q = _rand((tok, hq, dqk), std, 70 + dqk)
    cu = np.cumsum([0] + [n for (_, n) in segs])
    pre = [p for (p, _) in segs]
    k_pages, v_pages, bt_dev, bt = _paginate(k, v, seg_rows, kv_contig, page, 80 + dqk)
    attn = _attn(hq, hkv, dqk, dv, tok, T)
    attn.plan(cu, [0] * len(segs), pre)
    out, lse = attn.run_paged(q, k_pages, v_pages, bt_dev,
                              lse=torch.empty((hq, tok), dtype=torch.float32, device=DEV))
    torch.cuda.synchronize()
    # the oracle sees only the pages: gather each request's rows by the reference mapping
    kp = k_pages.cpu().view(torch.int16).numpy()
    vp = v_pages.cpu().view(torch.int16).numpy()
    kc = np.concatenate([OP.contiguous_rows(kp, bt[s], seg_rows[s]) for s in range(len(segs))])
    vc = np.concatenate([OP.contiguous_rows(vp, bt[s], seg_rows[s]) for s in range(len(segs))])
    kc = torch.from_numpy(kc).view(torch.bfloat16)
    vc = torch.from_numpy(vc).view(torch.bfloat16)
    ro, rl = oracle.attention_full(q.cpu(), kc, vc, cu, kv_contig, pre)
    rows = np.repeat(np.arange(tok), hq)
    heads = np.tile(np.arange(hq), tok)
    rep = PA.compare(out, lse, rows, heads, ro.reshape(tok * hq, -1), rl.T.reshape(-1))
    print(dims, rep, flush=True)
    assert rep.ok(), str(rep)


def test_kv_append_bit_exact():
    from paper_2608_26523_amd import binding as B
    from paper_2608_26523_amd.attention import kv_append_paged
    hkv, dqk, dv, page, npages = 3, 192, 128, 64, 11
    segs_cu = [0, 100, 100, 230]          # three segments, one empty
    kv_start, pre = [0, 64, 0], [37, 0, 300]
    tok = segs_cu[-1]
    rng = np.random.default_rng(3)
    perm = rng.permutation(npages).astype(np.int32)
    # segment 0 covers cache rows 37..136 (table entries 0..2), segment 2 rows
    # 300..429 (entries 4..6): distinct pages, so no two tokens share a slot
    bt = np.full((3, 7), perm[6], dtype=np.int32)
    bt[0, :3] = perm[:3]
    bt[2, 4:7] = perm[3:6]
    slots = B.vpp_paged_slot_mapping(segs_cu, kv_start, pre, bt, page)
    assert len(set(slots.tolist())) == tok
    assert np.array_equal(slots, OP.slot_mapping(segs_cu, kv_start, pre, bt, page))
    slots[[5, 77]] = -1                    # padding tokens
    k_new = _rand((tok, hkv, dqk), 1.0, 90)
    v_new = _rand((tok, hkv, dv), 1.0, 91)
    k_pages = _rand((npages, page, hkv, dqk), 1.0, 92)
    v_pages = _rand((npages, page, hkv, dv), 1.0, 93)
    want_k = OP.append(k_pages.cpu().view(torch.int16).numpy(), k_new.cpu().view(torch.int16).numpy(), slots)
    want_v = OP.append(v_pages.cpu().view(torch.int16).numpy(), v_new.cpu().view(torch.int16).numpy(), slots)
    kv_append_paged(k_new, v_new, k_pages, v_pages, torch.as_tensor(slots, device=DEV))
    torch.cuda.synchronize()
    assert np.array_equal(k_pages.cpu().view(torch.int16).numpy(), want_k)
    assert np.array_equal(v_pages.cpu().view(torch.int16).numpy(), want_v)


@pytest.mark.parametrize("dims", [(128, 128), (192, 128)])
def test_chunked_prefill_through_paged_cache(dims):
    """Prompt in chunks: append each chunk's K/V into pages, then paged attention;
    bit-identical to the contiguous path on the same rows."""
    from paper_2608_26523_amd import binding as B
    from paper_2608_26523_amd.attention import kv_append_paged
    dqk, dv = dims
    hq, hkv, page, S, C = 4, 2, 128, 1100, 256
    std = 1.0 / math.sqrt(dqk)
    q = _rand((S, hq, dqk), std, 100)
    k = _rand((S, hkv, dqk), std, 101)
    v = _rand((S, hkv, dv), std, 102)
    npages = (S + page - 1) // page + 2
    rng = np.random.default_rng(7)
    bt = rng.permutation(npages)[:(S + page - 1) // page].astype(np.int32)[None, :]
    bt_dev = torch.as_tensor(bt, device=DEV)
    k_pages = torch.zeros((npages, page, hkv, dqk), dtype=torch.bfloat16, device=DEV)
    v_pages = torch.zeros((npages, page, hkv, dv), dtype=torch.bfloat16, device=DEV)
    attn_c = _attn(hq, hkv, dqk, dv, C, S)
    attn_p = _attn(hq, hkv, dqk, dv, C, S)
    for c0 in range(0, S, C):
        n = min(C, S - c0)
        print("case: chunk at", c0, dims, flush=True)
        cu, pre = [0, n], [c0]
        slots = B.vpp_paged_slot_mapping(cu, [0], pre, bt, page)
        kv_append_paged(k[c0:c0 + n], v[c0:c0 + n], k_pages, v_pages, torch.as_tensor(slots, device=DEV))
        attn_c.plan(cu, [0], pre)
        oc, _ = attn_c.run(q[c0:c0 + n], k, v)
        attn_p.plan(cu, [0], pre)
        op, _ = attn_p.run_paged(q[c0:c0 + n], k_pages, v_pages, bt_dev)
        torch.cuda.synchronize()
        assert torch.equal(oc, op), "chunk at %d differs" % c0


def test_paged_full_size_mla_last_chunk_pool_over_4gib():
    """mla's last chunk (prefix 122880, 8192 rows, 128 heads, dims 192/128) over a paged
    cache of 128-row pages in random order: a 10.7 GB page pool, so page addresses run
    far past 4 GiB. Sampled (row, head) items against the oracle, evaluated on rows
    gathered from the pool by the reference page mapping (oracle/paged.contiguous_rows)."""
    from paper_2608_26523_amd import workloads as W
    from paper_2608_26523_amd.attention import ChunkAttention
    w = W.get("mla")
    c = W.num_chunks(w) - 1
    t0, cu, kvs, pre = W.chunk_segments(w, c)
    tok = int(cu[-1])
    rows = int(pre[0]) + tok
    page, extra = 128, 4
    npg = (rows + page - 1) // page
    print("case: paged mla chunk %d, %d rows in %d pages of %d" % (c, rows, npg, page), flush=True)
    rng = np.random.default_rng(15)
    perm = rng.permutation(npg + extra).astype(np.int32)
    bt = perm[:npg][None, :].copy()
    std = 1.0 / math.sqrt(w.dqk)
    idx = torch.as_tensor(bt[0].astype(np.int64), device=DEV)
    k_pages = torch.full((npg + extra, page, w.hkv, w.dqk), 3.0, dtype=torch.bfloat16, device=DEV)
    k = W.normal_bf16((rows, w.hkv, w.dqk), std, w.seed, w.index, "k", DEV)
    k_pages.index_copy_(0, idx, k.view(npg, page, w.hkv, w.dqk))
    del k
    v_pages = torch.full((npg + extra, page, w.hkv, w.dv), 3.0, dtype=torch.bfloat16, device=DEV)
    v = W.normal_bf16((rows, w.hkv, w.dv), std, w.seed, w.index, "v", DEV)
    v_pages.index_copy_(0, idx, v.view(npg, page, w.hkv, w.dv))
    del v
    assert k_pages.numel() * 2 > (4 << 30) and v_pages.numel() * 2 > (4 << 30)
    q = W.make_q_rows(w, DEV, t0, t0 + tok)
    attn = ChunkAttention(w.hq, w.hkv, w.dqk, w.dv, max_chunk_tokens=w.chunk, max_kv_len=rows,
                          num_splits=w.num_splits)
    attn.plan(cu, [0], pre)
    out = torch.full((tok, w.hq, w.dv), float("nan"), dtype=torch.bfloat16, device=DEV)
    lse = torch.full((w.hq, tok), float("nan"), dtype=torch.float32, device=DEV)
    attn.run_paged(q, k_pages, v_pages, torch.as_tensor(bt, device=DEV), out, lse)
    torch.cuda.synchronize()
    r_items, h_items = PA.sample_items(cu, [0], pre, w.hq, w.hkv, seed=c)
    g = w.hq // w.hkv
    ro = np.zeros((len(r_items), w.dv))
    rl = np.zeros(len(r_items))
    for kvh in sorted(set((h_items // g).tolist())):
        sel = np.nonzero(h_items // g == kvh)[0]
        kp = k_pages[:, :, kvh].cpu().view(torch.int16).numpy().view(np.uint16)
        vp = v_pages[:, :, kvh].cpu().view(torch.int16).numpy().view(np.uint16)
        kg = OP.contiguous_rows(kp, bt[0], rows)[:, None, :]
        vg = OP.contiguous_rows(vp, bt[0], rows)[:, None, :]
        qh = q[:, kvh * g:(kvh + 1) * g].cpu()
        o, l = oracle.attention(qh, kg, vg, cu, [0], pre, rows=r_items[sel],
                                heads=h_items[sel] - kvh * g, scale=w.scale)
        ro[sel], rl[sel] = o, l
    rep = PA.compare(out, lse, r_items, h_items, ro, rl)
    print("paged mla chunk %d:" % c, rep, flush=True)
    assert rep.ok(), rep
    assert bool(torch.isfinite(out.float()).all())

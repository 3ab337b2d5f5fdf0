"""The C ABI on the host (no GPU): exports, planner invariants, argument checks."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_26523_amd import binding as B
from paper_2608_26523_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vpp_chunk_attn.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(vpp_\w+)\s*\(", text)))


def test_header_symbols_exported():
    lib = B.load()
    names = header_functions()
    assert "vpp_chunk_attn_plan" in names and "vpp_chunk_attn_run" in names
    for n in names:
        assert hasattr(lib, n), "symbol %s declared in the header is not exported" % n
    assert sorted(B.EXPORTED) == names


def cfg(hq=8, hkv=2, dqk=128, dv=128, max_tok=4096, max_seg=16, max_kv=1 << 20, splits=-1,
        causal=1, scale=0.0):
    return B.Config(num_q_heads=hq, num_kv_heads=hkv, head_dim_qk=dqk, head_dim_v=dv,
                    softmax_scale=scale, causal=causal, max_chunk_tokens=max_tok,
                    max_segments=max_seg, max_kv_len=max_kv, num_splits=splits)


def plan_status(c, cu, ks, pl):
    lib = B.load()
    cu = np.ascontiguousarray(cu, dtype=np.int32)
    ks = np.ascontiguousarray(ks, dtype=np.int64)
    pl = np.ascontiguousarray(pl, dtype=np.int64)
    h = ctypes.c_void_p(None)
    ws = ctypes.c_size_t(0)
    st = lib.vpp_chunk_attn_plan(ctypes.byref(c) if c is not None else None, len(ks),
                                 cu.ctypes.data, ks.ctypes.data, pl.ctypes.data,
                                 ctypes.byref(h), ctypes.byref(ws))
    if h.value:
        B.vpp_chunk_attn_destroy(h.value)
    return st


@pytest.mark.parametrize("bad,status", [
    (dict(hq=6, hkv=4), B.VPP_ERR_INVALID_ARG),
    (dict(dqk=96, dv=96), B.VPP_ERR_UNSUPPORTED),
    (dict(dqk=128, dv=64), B.VPP_ERR_UNSUPPORTED),
    (dict(causal=0), B.VPP_ERR_UNSUPPORTED),
    (dict(splits=0), B.VPP_ERR_INVALID_ARG),
    (dict(splits=17), B.VPP_ERR_INVALID_ARG),
    (dict(scale=-1.0), B.VPP_ERR_INVALID_ARG),
    (dict(max_tok=0), B.VPP_ERR_INVALID_ARG),
])
def test_config_errors(bad, status):
    assert plan_status(cfg(**bad), [0, 10], [0], [0]) == status


@pytest.mark.parametrize("cu,ks,pl", [
    ([1, 10], [0], [0]),                 # cu_q[0] != 0
    ([0, 10, 5], [0, 20], [0, 0]),       # decreasing
    ([0, 10], [-1], [0]),                # negative kv_start
    ([0, 10], [0], [-5]),                # negative prefix
    ([0, 5000], [0], [0]),               # more rows than max_chunk_tokens
    ([0, 10], [(1 << 20) - 5], [0]),     # runs past max_kv_len
])
def test_metadata_errors(cu, ks, pl):
    assert plan_status(cfg(), cu, ks, pl) == B.VPP_ERR_INVALID_ARG


def test_too_many_segments_and_null_args():
    assert plan_status(cfg(max_seg=2), [0, 1, 2, 3], [0, 1, 2], [0, 0, 0]) == B.VPP_ERR_INVALID_ARG
    lib = B.load()
    ws = ctypes.c_size_t(0)
    h = ctypes.c_void_p(None)
    assert lib.vpp_chunk_attn_plan(None, 1, None, None, None, ctypes.byref(h),
                                   ctypes.byref(ws)) == B.VPP_ERR_INVALID_ARG
    assert lib.vpp_chunk_attn_plan_info(None, None) == B.VPP_ERR_INVALID_ARG
    assert B.vpp_status_str(B.VPP_ERR_WORKSPACE) == "workspace too small"
    lib.vpp_chunk_attn_destroy(None)


def test_refill_must_keep_config():
    h, _ = B.vpp_chunk_attn_plan(cfg(), [0, 100], [0], [0])
    try:
        B.vpp_chunk_attn_plan(None, [0, 300], [0], [500], plan=h)      # refill, same config
        assert B.vpp_chunk_attn_plan_info(h).num_tokens == 300
        with pytest.raises(B.VppError):
            B.vpp_chunk_attn_plan(cfg(hq=16), [0, 10], [0], [0], plan=h)
    finally:
        B.vpp_chunk_attn_destroy(h)


def check_plan(c, cu, ks, pl):
    h, ws = B.vpp_chunk_attn_plan(c, cu, ks, pl)
    try:
        info = B.vpp_chunk_attn_plan_info(h)
        items = B.vpp_chunk_attn_plan_items(h)
    finally:
        B.vpp_chunk_attn_destroy(h)
    bm, bn, n = info.block_m, info.block_n, info.num_splits
    # two entries per work slot (one workgroup per slot and head); a second entry
    # without rows is empty
    assert info.num_work_items == len(items) and len(items) % 2 == 0
    # the launch runs one workgroup per slot and head
    assert info.num_slots * 2 == len(items)
    assert ws == info.workspace_bytes and ws >= len(items) * 32
    slots = items.reshape(-1, 2)
    assert np.all(slots[:, 0]["nrows"] >= 1)
    seg_of = lambda row0: int(np.searchsorted(cu, row0, side="right") - 1)  # noqa: E731
    # tiles: rows partition the chunk, positions and bases follow the segments
    tiles = {}
    for it in items[items["nrows"] > 0]:
        tiles.setdefault(int(it["row0"]), []).append(it)
    assert info.num_tiles == len(tiles)
    covered = np.zeros(int(cu[-1]), dtype=np.int32)
    pairs = 0
    bounds = {}
    for row0, its in tiles.items():
        assert len(its) == n
        t = its[0]
        assert 1 <= t["nrows"] <= bm
        covered[row0:row0 + t["nrows"]] += 1
        s = seg_of(row0)
        assert row0 + t["nrows"] <= cu[s + 1], "a tile crosses a segment boundary"
        assert t["pos0"] == pl[s] + row0 - cu[s]
        assert t["kv_base"] == ks[s]
        # pieces cover [0, last position + 1) exactly, in order, tile-aligned inside;
        # every piece below the last ends inside the prefix, at a boundary common to
        # all tiles of the segment
        rng = sorted((int(x["split"]), int(x["key_begin"]), int(x["key_end"])) for x in its)
        assert [r[0] for r in rng] == list(range(n))
        assert rng[0][1] == 0 and rng[-1][2] == t["pos0"] + t["nrows"]
        for a, b in zip(rng, rng[1:]):
            assert a[2] == b[1] and a[2] % bn == 0 and a[2] <= pl[s]
        assert bounds.setdefault(s, [r[1] for r in rng]) == [r[1] for r in rng]
        pairs += int(t["nrows"]) * int(t["pos0"]) + int(t["nrows"]) * (int(t["nrows"]) + 1) // 2
    assert np.all(covered == 1)
    assert info.pairs == pairs
    # a slot pairs a tile with its partner from the other end of the same segment,
    # in the same piece; the pair's key counts add up alike within a (segment,
    # piece) group, and groups run longest first
    groups = {}
    order = []
    for a, b in slots:
        s = seg_of(int(a["row0"]))
        ln = int(a["key_end"] - a["key_begin"])
        if b["nrows"]:
            assert seg_of(int(b["row0"])) == s and b["split"] == a["split"] and b["row0"] > a["row0"]
            ln += int(b["key_end"] - b["key_begin"])
        key = (s, int(a["split"]))
        if key not in groups:
            order.append(key)
        groups.setdefault(key, []).append((ln, bool(b["nrows"])))
    for key, lens in groups.items():
        full = [x for x, two in lens if two]
        if full:
            assert max(full) - min(full) <= bm, (key, lens)
        # the groups' slots are contiguous
    seen = [(seg_of(int(a["row0"])), int(a["split"])) for a, _ in slots]
    assert [k for i, k in enumerate(seen) if i == 0 or seen[i - 1] != k] == order, "a group is not contiguous"
    glen = [max(x for x, _ in groups[k]) for k in order]
    assert all(x >= y for x, y in zip(glen, glen[1:]))
    return info


@pytest.mark.parametrize("name", ["tiny", "gqa", "mla", "long"])
def test_plan_workload_chunks(name):
    w = W.get(name)
    c = cfg(hq=w.hq, hkv=w.hkv, dqk=w.dqk, dv=w.dv, max_tok=w.chunk, max_kv=w.seq_len,
            splits=w.num_splits)
    for k in sorted({0, 1, W.num_chunks(w) - 1}):
        _, cu, ks, pl = W.chunk_segments(w, k)
        info = check_plan(c, cu, ks, pl)
        if w.num_splits > 0:
            # a fixed count applies once the prefix has a key tile per piece
            assert info.num_splits == min(w.num_splits, max(1, int(pl[0]) // 64))


def test_plan_mixed_chunks():
    w = W.get("mixed")
    c = cfg(hq=w.hq, hkv=w.hkv, dqk=w.dqk, dv=w.dv, max_tok=w.chunk,
            max_kv=W.total_tokens(w), max_seg=256)
    n = W.num_chunks(w)
    multi = 0
    for k in list(range(0, n, 23)) + [n - 1]:
        _, cu, ks, pl = W.chunk_segments(w, k)
        multi += len(ks) > 1
        check_plan(c, cu, ks, pl)
    assert multi > 0, "no sampled chunk spans a request boundary"


@pytest.mark.parametrize("splits", [2, 3, 5, 16])
def test_plan_forced_splits_ragged(splits):
    c = cfg(splits=splits)
    check_plan(c, [0, 1, 1, 130, 400], [0, 7, 7, 500], [63, 0, 1000, 37])


def test_auto_split_only_when_few_workgroups():
    # one tile x 8 heads with a long prefix: too few workgroups -> split
    info = check_plan(cfg(), [0, 100], [0], [200000])
    assert info.num_splits > 1
    # a full 4096-row chunk over 32 heads: plenty of workgroups -> no split
    info = check_plan(cfg(hq=32, hkv=8), [0, 4096], [0], [200000])
    assert info.num_splits == 1


def test_auto_split_follows_the_simulated_launch():
    """Automatic splits come from a model of the launch: a chunk whose work sits in a few
    long slots of one segment (mixed chunk 98: 43 rows behind a 118844-key prefix, next to
    two short requests) is split; chunks whose slots fill the chip evenly are not."""
    w = W.get("mixed")
    c = cfg(hq=w.hq, hkv=w.hkv, dqk=w.dqk, dv=w.dv, max_tok=w.chunk, max_kv=W.total_tokens(w), max_seg=256)
    _, cu, ks, pl = W.chunk_segments(w, 98)
    assert len(ks) == 3 and int(max(pl)) > 100000
    assert check_plan(c, cu, ks, pl).num_splits > 1
    _, cu, ks, pl = W.chunk_segments(w, 200)        # one request deep in its prefix, one fresh
    assert check_plan(c, cu, ks, pl).num_splits > 1
    for name in ("gqa", "mla"):
        w = W.get(name)
        c = cfg(hq=w.hq, hkv=w.hkv, dqk=w.dqk, dv=w.dv, max_tok=w.chunk, max_kv=w.seq_len)
        for k in range(W.num_chunks(w)):
            _, cu, ks, pl = W.chunk_segments(w, k)
            assert check_plan(c, cu, ks, pl).num_splits == 1, (name, k)


def test_run_argument_checks_before_any_device_work():
    """Errors the host can detect are returned before any HIP call (works without a GPU)."""
    lib = B.load()
    h, ws = B.vpp_chunk_attn_plan(cfg(), [0, 64], [0], [0])
    try:
        good = 1 << 20            # aligned fake addresses: never dereferenced on these paths
        base = dict(q=good, qs=(8 * 128, 128), k=good, ks=(2 * 128, 128), v=good,
                    vs=(2 * 128, 128), o=good, os=(8 * 128, 128), lse=0, lsh=0,
                    ws=good, wsb=ws)

        def call(**over):
            a = dict(base)
            a.update(over)
            return lib.vpp_chunk_attn_run(h, a["q"], a["qs"][0], a["qs"][1], a["k"], a["ks"][0],
                                          a["ks"][1], a["v"], a["vs"][0], a["vs"][1], a["o"],
                                          a["os"][0], a["os"][1], a["lse"], a["lsh"], a["ws"],
                                          a["wsb"], None)
        assert call(q=0) == B.VPP_ERR_INVALID_ARG
        assert call(k=good + 2) == B.VPP_ERR_INVALID_ARG
        assert call(qs=(8 * 128 + 4, 128)) == B.VPP_ERR_INVALID_ARG
        assert call(os=(0, 128)) == B.VPP_ERR_INVALID_ARG
        assert call(lse=good, lsh=10) == B.VPP_ERR_INVALID_ARG        # stride < tokens
        assert call(ws=0) == B.VPP_ERR_WORKSPACE
        assert call(ws=good + 64) == B.VPP_ERR_WORKSPACE
        assert call(wsb=ws - 1) == B.VPP_ERR_WORKSPACE
        assert lib.vpp_chunk_attn_run(None, good, 1024, 128, good, 256, 128, good, 256, 128,
                                      good, 1024, 128, 0, 0, good, ws, None) == B.VPP_ERR_INVALID_ARG
    finally:
        B.vpp_chunk_attn_destroy(h)


def test_cache_row_stride_boundary():
    """A key tile (64 rows of the cache row stride, 2 bytes an element) must span less
    than 2^31 bytes: row strides up to 2^24 - 8 elements pass the argument checks,
    2^24 is refused. The workspace is one byte short, so a stride that passes stops
    at the workspace check and no device work is ever enqueued."""
    lib = B.load()
    h, ws = B.vpp_chunk_attn_plan(cfg(), [0, 64], [0], [0])
    try:
        good = 1 << 20
        ok, bad = (1 << 24) - 8, 1 << 24

        def call(k_st=256, v_st=256, q_st=1024):
            return lib.vpp_chunk_attn_run(h, good, q_st, 128, good, k_st, 128, good, v_st, 128,
                                          good, 1024, 128, 0, 0, good, ws - 1, None)
        assert call(k_st=ok) == B.VPP_ERR_WORKSPACE
        assert call(v_st=ok) == B.VPP_ERR_WORKSPACE
        assert call(k_st=bad) == B.VPP_ERR_INVALID_ARG
        assert call(v_st=bad) == B.VPP_ERR_INVALID_ARG
        # query strides are not tile-bounded: only the 32-bit element-stride limit applies
        assert call(q_st=bad) == B.VPP_ERR_WORKSPACE
        assert call(q_st=1 << 25) == B.VPP_ERR_INVALID_ARG
    finally:
        B.vpp_chunk_attn_destroy(h)


def test_split_key_row_stride_boundary():
    lib = B.load()
    h, ws = B.vpp_chunk_attn_plan(cfg(hq=2, hkv=2, dqk=192, dv=128), [0, 64], [0], [0])
    try:
        good = 1 << 20

        def call(kr_st):
            return lib.vpp_chunk_attn_run_mla(h, good, 384, 192, good, 256, 128, good, kr_st, good, 256, 128,
                                              good, 256, 128, None, 0, good, ws - 1, None)
        assert call((1 << 24) - 8) == B.VPP_ERR_WORKSPACE
        assert call(1 << 24) == B.VPP_ERR_INVALID_ARG
    finally:
        B.vpp_chunk_attn_destroy(h)


def test_noalloc_limit_and_refusals_before_any_device_work():
    """run_noalloc refuses a plan whose workspace exceeds its static scratch, and a NULL
    plan, before any HIP call; the header's size is the binding's."""
    import re
    hdr = open(os.path.join(ROOT, "include", "vpp_chunk_attn.h")).read()
    m = re.search(r"#define VPP_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", hdr)
    assert m and int(m.group(1)) << int(m.group(2)) == B.NOALLOC_SCRATCH_BYTES
    lib = B.load()
    good = 1 << 20
    # one 256-row tile, 128 heads, 16 splits over a long prefix: 16 x 256 x 128 x 128 x 4 B of partials
    c = cfg(hq=128, hkv=128, dqk=192, dv=128, splits=16)
    h, ws = B.vpp_chunk_attn_plan(c, [0, 256], [0], [500000])
    try:
        assert ws > B.NOALLOC_SCRATCH_BYTES
        st = lib.vpp_chunk_attn_run_noalloc(h, good, 128 * 192, 192, good, 128 * 192, 192, good, 128 * 128,
                                            128, good, 128 * 128, 128, 0, 0, None)
        assert st == B.VPP_ERR_WORKSPACE
    finally:
        B.vpp_chunk_attn_destroy(h)
    assert lib.vpp_chunk_attn_run_noalloc(None, good, 1024, 128, good, 256, 128, good, 256, 128,
                                          good, 1024, 128, 0, 0, None) == B.VPP_ERR_INVALID_ARG


def test_empty_chunk_plans_to_nothing():
    info = check_plan(cfg(), [0, 0, 0], [0, 5], [3, 0])
    assert info.num_work_items == 0 and info.num_tokens == 0


def test_tile_rows_follow_chunk_size(monkeypatch):
    monkeypatch.delenv("VPP_NB", raising=False)
    # 4096 rows x 32 heads = 512 workgroups of 256 rows (at most two per CU) with
    # short key ranges -> 128-row tiles
    info = check_plan(cfg(hq=32, hkv=8), [0, 4096], [0], [0])
    assert info.block_m == 128
    # the same chunk behind a long prefix -> 256-row tiles
    info = check_plan(cfg(hq=32, hkv=8), [0, 4096], [0], [20480])
    assert info.block_m == 256
    # 16384 rows x 32 heads: enough 256-row workgroups
    info = check_plan(cfg(hq=32, hkv=8, max_tok=16384), [0, 16384], [0], [0])
    assert info.block_m == 256
    # dqk = 192 keeps the 64-row waves whatever the size
    info = check_plan(cfg(hq=8, hkv=8, dqk=192, dv=128), [0, 256], [0], [0])
    assert info.block_m == 256
    # every item's rows fit the tile
    for n in (1, 127, 128, 129, 300):
        check_plan(cfg(hq=4, hkv=2), [0, n], [0], [17])


# Random segment mixes through the same invariant checks: empty and ragged
# segments, long prefixes, forced and automatic splits, every head-dim pair.
from hypothesis import HealthCheck, given, settings, strategies as st  # noqa: E402

_HEADS = [(4, 4), (8, 2), (32, 8), (128, 128)]
_DIMS = [(64, 64), (128, 128), (192, 128)]


@st.composite
def _segment_mix(draw):
    n = draw(st.integers(1, 8))
    lens = draw(st.lists(st.integers(0, 700), min_size=n, max_size=n))
    if sum(lens) == 0:
        lens[0] = draw(st.integers(1, 700))
    prefixes = draw(st.lists(st.integers(0, 300000), min_size=n, max_size=n))
    starts, row = [], 0
    for ln, p in zip(lens, prefixes):       # each segment's own cache region
        starts.append(row)
        row += p + ln + draw(st.integers(0, 50))
    hq, hkv = draw(st.sampled_from(_HEADS))
    dqk, dv = draw(st.sampled_from(_DIMS))
    splits = draw(st.sampled_from([-1, 1, 2, 3, 7, 16]))
    return lens, prefixes, starts, row, (hq, hkv, dqk, dv), splits


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(_segment_mix())
def test_plan_random_segment_mixes(mix):
    lens, prefixes, starts, rows, (hq, hkv, dqk, dv), splits = mix
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    c = cfg(hq=hq, hkv=hkv, dqk=dqk, dv=dv, max_tok=int(cu[-1]), max_kv=max(rows, 1), splits=splits)
    info = check_plan(c, cu, starts, prefixes)
    if splits > 0:
        # a fixed count, capped at one key tile of prefix per piece (longest prefix
        # of a segment with rows)
        longest = max([p for p, n in zip(prefixes, lens) if n > 0], default=0)
        assert info.num_splits == min(splits, max(1, longest // 64))

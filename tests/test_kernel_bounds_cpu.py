"""Host model of the attention kernel's indexing, checked on the CPU for many plans.

The launch runs num_slots x num_heads workgroups; a workgroup reads work-list
entries 2*slot and 2*slot + 1, runs the first entry's key tiles ascending and the
second's descending. Per tile loop it issues the copies of the key tiles of visits
0 and 1 up front, then in step t the K copy of visit t+2 and the V copy of visit
t+1, through the same running values the kernel keeps (first key of the K copy,
visits left). This model replays exactly those updates and checks that

* every work-list read is inside the list;
* every copy with rows reads only keys inside its entry's range [key_begin, key_end)
  (so cache rows stay inside the cache the plan was checked against);
* every key of the range is copied exactly once for K and once for V, and each visit
  of the loop consumes the tile that was copied for it.
"""
import numpy as np
import pytest

from paper_2608_26523_amd import binding as B
from paper_2608_26523_amd import workloads as W

BN = 64


def _cfg(hq, hkv, dqk, dv, max_tok, max_kv, splits, max_seg=256):
    return B.Config(num_q_heads=hq, num_kv_heads=hkv, head_dim_qk=dqk, head_dim_v=dv, softmax_scale=0.0,
                    causal=1, max_chunk_tokens=max_tok, max_segments=max_seg, max_kv_len=max_kv,
                    num_splits=splits)


def _tile_rows(kt, ke, valid):
    return min(BN, ke - kt) if valid else 0


def _replay_entry(it, rev):
    """Copies (visit, first key, rows) of K and V for one entry, as the kernel issues them."""
    kb, ke = int(it["key_begin"]), int(it["key_end"])
    ntiles = (ke - kb + BN - 1) // BN
    dkt = -BN if rev else BN
    kt_first = kb + (ntiles - 1) * BN if rev else kb
    k_copies, v_copies = [], []
    if ntiles > 0:
        k_copies.append((0, kt_first, _tile_rows(kt_first, ke, True)))
        v_copies.append((0, kt_first, _tile_rows(kt_first, ke, True)))
        if ntiles > 1:
            k_copies.append((1, kt_first + dkt, _tile_rows(kt_first + dkt, ke, True)))
    kt_k, k_left = kt_first + 2 * dkt, ntiles - 2
    # steps: pairs of full steps while two tiles remain, then one last step (no copies)
    t = 0
    steps = []
    while t + 1 < ntiles:
        steps += [(t, True), (t + 1, True)]
        t += 2
    if t < ntiles:
        steps.append((t, False))
    visits = []
    for t, has_next in steps:
        visits.append(kt_first + t * dkt)
        k_n = min(BN, ke - kt_k) if k_left > 0 else 0
        v_n = min(BN, ke - (kt_k - dkt)) if k_left >= 0 else 0
        if has_next:
            k_copies.append((t + 2, kt_k, k_n))
            v_copies.append((t + 1, kt_k - dkt, v_n))
        kt_k += dkt
        k_left -= 1
    return kb, ke, ntiles, visits, k_copies, v_copies


def _check_plan(cfg, cu, kvs, pre):
    h, ws = B.vpp_chunk_attn_plan(cfg, cu, kvs, pre)
    try:
        info = B.vpp_chunk_attn_plan_info(h)
        items = B.vpp_chunk_attn_plan_items(h)
    finally:
        B.vpp_chunk_attn_destroy(h)
    n = len(items)
    assert info.num_slots * 2 == n
    # the grid: every workgroup's entries are inside the list
    for slot in range(info.num_slots):
        for sub in (0, 1):
            e = 2 * slot + sub
            assert 0 <= e < n
            it = items[e]
            if it["nrows"] == 0:
                assert sub == 1
                break
            kb, ke, ntiles, visits, kc, vc = _replay_entry(it, rev=sub == 1)
            assert 0 <= kb <= ke
            assert visits == sorted(visits, reverse=sub == 1)
            for copies in (kc, vc):
                got = {}
                for vis, kt, rows in copies:
                    if rows > 0:
                        assert vis < ntiles
                        assert kb <= kt and kt + rows <= ke, (it, vis, kt, rows)
                        assert kt == visits[vis], "copied tile is not the tile of its visit"
                        got[vis] = (kt, rows)
                    else:
                        assert vis >= ntiles, "a needed tile was not copied"
                assert sorted(got) == list(range(ntiles))
                assert sum(r for _, r in got.values()) == ke - kb
                assert {kt for kt, _ in got.values()} == set(visits)
    return info


@pytest.mark.parametrize("name", ["tiny", "gqa", "mla", "long"])
def test_workload_chunks_in_bounds(name):
    w = W.get(name)
    c = _cfg(w.hq, w.hkv, w.dqk, w.dv, w.chunk, w.seq_len, w.num_splits)
    for k in sorted({0, 1, 2, W.num_chunks(w) // 2, W.num_chunks(w) - 1}):
        _, cu, kvs, pre = W.chunk_segments(w, k)
        _check_plan(c, cu, kvs, pre)


def test_mixed_chunks_in_bounds():
    w = W.get("mixed")
    c = _cfg(w.hq, w.hkv, w.dqk, w.dv, w.chunk, W.total_tokens(w), w.num_splits)
    n = W.num_chunks(w)
    for k in list(range(0, n, 17)) + [n - 1]:
        _, cu, kvs, pre = W.chunk_segments(w, k)
        _check_plan(c, cu, kvs, pre)


@pytest.mark.parametrize("seed", range(60))
def test_random_plans_in_bounds(seed):
    rng = np.random.default_rng(seed)
    nseg = int(rng.integers(1, 6))
    lens = [int(rng.integers(0, 900)) if rng.random() > 0.15 else 0 for _ in range(nseg)]
    if sum(lens) == 0:
        lens[0] = 1 + int(rng.integers(0, 500))
    pre = [int(rng.integers(0, 5000)) if rng.random() > 0.2 else 0 for _ in range(nseg)]
    kvs, row = [], 0
    for ln, p in zip(lens, pre):
        kvs.append(row)
        row += p + ln + int(rng.integers(0, 70))
    hq, hkv = [(4, 4), (8, 2), (2, 1), (16, 16)][int(rng.integers(4))]
    dqk, dv = [(64, 64), (128, 128), (192, 128)][int(rng.integers(3))]
    splits = [-1, 1, 2, 3, 5, 16][int(rng.integers(6))]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    _check_plan(_cfg(hq, hkv, dqk, dv, int(cu[-1]), row, splits), cu, kvs, pre)

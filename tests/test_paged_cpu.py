"""Paged-cache entry points on the host: slot mapping against its reference, and the
argument checks that reject bad paged calls before any device work."""
import numpy as np
import pytest

from oracle import paged as OP
from paper_2608_26523_amd import binding as B


def _cfg(hq=4, hkv=2, dqk=128, dv=128):
    return B.Config(num_q_heads=hq, num_kv_heads=hkv, head_dim_qk=dqk, head_dim_v=dv, softmax_scale=0.0,
                    causal=1, max_chunk_tokens=4096, max_segments=16, max_kv_len=1 << 20, num_splits=-1)


@pytest.mark.parametrize("page", [64, 128, 1024])
def test_slot_mapping_matches_reference(page):
    rng = np.random.default_rng(page)
    n = 4
    lens = rng.integers(0, 300, size=n)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    pre = rng.integers(0, 5000, size=n).astype(np.int64)
    kvs = (rng.integers(0, 4, size=n) * 64).astype(np.int64)
    width = int(max((kvs + pre + lens) // page + 1))
    bt = rng.integers(0, 10_000, size=(n, width)).astype(np.int32)
    got = B.vpp_paged_slot_mapping(cu, kvs, pre, bt, page)
    assert np.array_equal(got, OP.slot_mapping(cu, kvs, pre, bt, page))


def test_slot_mapping_rejects_short_table():
    bt = np.zeros((1, 2), np.int32)
    with pytest.raises(B.VppError):
        B.vpp_paged_slot_mapping([0, 10], [0], [120], bt, 64)   # row 129 needs entry 2
    with pytest.raises(B.VppError):
        B.vpp_paged_slot_mapping([0, 10], [0], [0], -np.ones((1, 2), np.int32), 64)


def _plan(kv_start=0):
    h, ws = B.vpp_chunk_attn_plan(_cfg(), [0, 100], [kv_start], [50])
    return h, ws


FAKE = 1 << 20  # aligned, never dereferenced: every case fails its checks first


@pytest.mark.parametrize("page,kv_start,bt,ok_expected", [
    (32, 0, FAKE, False),     # below the key tile
    (96, 0, FAKE, False),     # not a power of two
    (128, 0, 0, False),       # no block table
    (128, 0, FAKE + 2, False),  # misaligned block table
    (128, 32, FAKE, False),   # kv_start not a multiple of 64: a tile would straddle pages
])
def test_run_paged_rejects(page, kv_start, bt, ok_expected):
    h, ws = _plan(kv_start)
    try:
        st = B.load().vpp_chunk_attn_run_paged(h, FAKE, 512, 128, FAKE, 4096, 256, 128, FAKE, 4096, 256, 128,
                                               page, 8, bt, 4, FAKE, 512, 128, None, 0, FAKE, ws, None)
        assert st == B.VPP_ERR_INVALID_ARG
    finally:
        B.vpp_chunk_attn_destroy(h)


@pytest.mark.parametrize("kw", [
    dict(dqk=100), dict(dv=0), dict(page=48), dict(page=192), dict(heads=0), dict(pages=0),
    dict(tokens=-1), dict(slots=FAKE + 4),
])
def test_kv_append_rejects(kw):
    a = dict(dqk=128, dv=128, page=64, heads=2, pages=4, tokens=10, slots=FAKE)
    a.update(kw)
    st = B.load().vpp_kv_append_paged(FAKE, 256, 128, FAKE, 256, 128, FAKE, 16384, 256, 128,
                                      FAKE, 16384, 256, 128, a["tokens"], a["heads"], a["dqk"], a["dv"],
                                      a["page"], a["pages"], a["slots"], None)
    assert st == B.VPP_ERR_INVALID_ARG


def test_kv_append_no_tokens_is_a_no_op():
    st = B.load().vpp_kv_append_paged(0, 256, 128, 0, 256, 128, 0, 16384, 256, 128,
                                      0, 16384, 256, 128, 0, 2, 128, 128, 64, 4, 0, None)
    assert st == B.VPP_OK


def test_run_mla_rejects():
    lib = B.load()
    h, ws = B.vpp_chunk_attn_plan(_cfg(), [0, 100], [0], [50])        # (128, 128): no split keys
    try:
        st = lib.vpp_chunk_attn_run_mla(h, FAKE, 512, 128, FAKE, 512, 128, FAKE, 64, FAKE, 512, 128,
                                        FAKE, 512, 128, None, 0, FAKE, ws, None)
        assert st == B.VPP_ERR_UNSUPPORTED
    finally:
        B.vpp_chunk_attn_destroy(h)
    h, ws = B.vpp_chunk_attn_plan(_cfg(hq=2, hkv=2, dqk=192, dv=128), [0, 100], [0], [50])
    try:
        for kr, kr_st in ((0, 64), (FAKE + 8, 64), (FAKE, 60), (FAKE, 0)):
            st = lib.vpp_chunk_attn_run_mla(h, FAKE, 384, 192, FAKE, 256, 128, kr, kr_st, FAKE, 256, 128,
                                            FAKE, 256, 128, None, 0, FAKE, ws, None)
            assert st == B.VPP_ERR_INVALID_ARG, (kr, kr_st)
    finally:
        B.vpp_chunk_attn_destroy(h)

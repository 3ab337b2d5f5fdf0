"""Workload registry and input generator (CPU)."""
import numpy as np
import pytest
import torch

from paper_2608_26523_amd import workloads as W


def test_partial_q_rows_match_full_stream():
    w = W.get("tiny")
    q, _, _ = W.make_inputs(w, "cpu", tokens=3 * W.SLAB_TOKENS // 4)
    w2 = W.Workload("t2", 7, hq=2, hkv=1, dqk=64, dv=64, chunk=W.SLAB_TOKENS, seq_len=3 * W.SLAB_TOKENS)
    full, _, _ = W.make_inputs(w2, "cpu")
    part = W.make_q_rows(w2, "cpu", W.SLAB_TOKENS, 3 * W.SLAB_TOKENS - 5)
    assert torch.equal(part, full[W.SLAB_TOKENS:3 * W.SLAB_TOKENS - 5])
    assert q.shape == (3 * W.SLAB_TOKENS // 4, w.hq, w.dqk)
    mid = W.make_q_rows(w2, "cpu", 4096 + 5, 2 * W.SLAB_TOKENS + 3)
    assert torch.equal(mid, full[4096 + 5:2 * W.SLAB_TOKENS + 3])
    with pytest.raises(ValueError):
        W.normal_bf16((4, 2, 64), 1.0, 0, 7, "q", "cpu", first_token=5)


def test_mixed_workload_shape():
    w = W.get("mixed")
    lens = W.request_lengths(w)
    assert len(lens) == 64 and lens.min() >= 1024 and lens.max() <= 262144
    n = W.num_chunks(w)
    covered = 0
    deepest = 0
    for c in range(n):
        t0, cu, kvs, pre = W.chunk_segments(w, c)
        assert t0 == covered and int(cu[-1]) <= w.chunk
        assert np.all(np.diff(cu) > 0)
        covered += int(cu[-1])
        if len(kvs) == 1:
            deepest = max(deepest, int(pre[0]))
    assert covered == W.total_tokens(w)
    assert deepest >= 65536      # the p >= 64K single-segment chunks exist


@pytest.mark.parametrize("name", ["tiny", "gqa", "mla", "long"])
def test_single_request_chunks(name):
    w = W.get(name)
    assert W.num_chunks(w) * w.chunk == w.seq_len
    for c in range(W.num_chunks(w)):
        t0, cu, kvs, pre = W.chunk_segments(w, c)
        assert t0 == c * w.chunk and list(cu) == [0, w.chunk]
        assert list(kvs) == [0] and list(pre) == [c * w.chunk]

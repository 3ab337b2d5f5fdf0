"""Pins for the fp64 oracle: checks against facts other than the oracle itself.

Each pin takes ``attn`` -- a callable with the signature of ``oracle.attention_full``
(q, k, v, cu_q, kv_start, prefix_len, scale=None) -> (out [tok, Hq, dv], lse [Hq, tok])
-- and raises AssertionError when the fact does not hold. The same battery runs
against the real oracle (tests/test_oracle_pins.py) and against copies of it with
planted mistakes (tests/test_oracle_mutants.py), which must each fail a pin.

The facts come from the mathematics of Eq. (1) with the causal rule (section 2.1)
and the chunk semantics (section 2.4), and from independent library routines:

* torch's float64 scaled_dot_product_attention and logsumexp, given an explicit
  mask in which query position i sees key positions 0..i (the causal rule at
  absolute positions: torch's own is_causal flag aligns differently when a chunk
  has fewer queries than keys, so it is not used);
* closed forms: the first token sees only itself; all-zero keys give the running
  mean of values and lse = ln(i+1); all-one values give ones;
* planted keys: a query parallel to one key picks out that key's value;
* exact invariances: adding a constant vector to every key shifts lse by
  scale*<q, c> and leaves out unchanged; adding a constant to every value adds it
  to out; doubling q and halving the scale changes nothing;
* causality: changing key/value rows after a query's position leaves its row
  unchanged, changing the row at its position does not;
* chunked == unchunked, packed == per-request, GQA == replicated MHA.
"""
from __future__ import annotations

import math

import numpy as np
import torch

TOL = 1e-11


def bf16(x) -> torch.Tensor:
    """float array -> bf16 CPU tensor (round to nearest even)."""
    return torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)


def rand_qkv(rng: np.random.Generator, tok, hq, hkv, dqk, dv, T=None):
    T = T or tok
    q = bf16(rng.standard_normal((tok, hq, dqk)) / math.sqrt(dqk))
    k = bf16(rng.standard_normal((T, hkv, dqk)) / math.sqrt(dqk))
    v = bf16(rng.standard_normal((T, hkv, dv)) / math.sqrt(dqk))
    return q, k, v


def sdpa_reference(q, k, v, cu_q, kv_start, prefix_len, scale=None):
    """torch float64 SDPA per segment with an explicit absolute-position mask."""
    tok, hq, dqk = q.shape
    hkv, dv = v.shape[1], v.shape[2]
    g = hq // hkv
    scale = scale if scale is not None else 1.0 / math.sqrt(dqk)
    out = np.zeros((tok, hq, dv))
    lse = np.zeros((hq, tok))
    for s in range(len(kv_start)):
        r0, r1 = int(cu_q[s]), int(cu_q[s + 1])
        if r1 == r0:
            continue
        p, base = int(prefix_len[s]), int(kv_start[s])
        nk = p + (r1 - r0)
        qs = q[r0:r1].double().permute(1, 0, 2)                      # [Hq, L, d]
        ks = k[base:base + nk].double().permute(1, 0, 2).repeat_interleave(g, 0)
        vs = v[base:base + nk].double().permute(1, 0, 2).repeat_interleave(g, 0)
        pos_q = torch.arange(p, p + (r1 - r0)).unsqueeze(1)
        pos_k = torch.arange(nk).unsqueeze(0)
        mask = pos_k <= pos_q                                         # [L, nk]
        o = torch.nn.functional.scaled_dot_product_attention(
            qs, ks, vs, attn_mask=mask, scale=scale)
        sc = torch.matmul(qs, ks.transpose(1, 2)) * scale
        sc = sc.masked_fill(~mask, float("-inf"))
        out[r0:r1] = o.permute(1, 0, 2).numpy()
        lse[:, r0:r1] = torch.logsumexp(sc, dim=-1).numpy()
    return out, lse


def _close(a, b, tol=TOL, what=""):
    err = float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) if np.size(a) else 0.0
    assert err <= tol, "%s: max abs err %.3e > %.1e" % (what, err, tol)


# ----------------------------------------------------------------------------
# pins
# ----------------------------------------------------------------------------
SDPA_CASES = [
    # (hq, hkv, dqk, dv, segments as (kv_start, prefix, len), T)
    (1, 1, 8, 8, [(0, 0, 24)], 24),
    (2, 1, 8, 8, [(0, 16, 12)], 28),
    (4, 2, 16, 12, [(0, 5, 9), (14, 0, 7), (21, 30, 5)], 56),
    (4, 4, 12, 16, [(3, 40, 17)], 60),
    (6, 2, 8, 4, [(0, 0, 1), (1, 63, 2), (66, 0, 40)], 106),
]


def pin_sdpa(attn, seed=0):
    rng = np.random.default_rng(seed)
    for hq, hkv, dqk, dv, segs, T in SDPA_CASES:
        tok = sum(s[2] for s in segs)
        q, k, v = rand_qkv(rng, tok, hq, hkv, dqk, dv, T=T)
        cu = np.cumsum([0] + [s[2] for s in segs])
        kvs = [s[0] for s in segs]
        pre = [s[1] for s in segs]
        out, lse = attn(q, k, v, cu, kvs, pre)
        ro, rl = sdpa_reference(q, k, v, cu, kvs, pre)
        _close(out, ro, 1e-12, "out vs torch SDPA %s" % ((hq, hkv, dqk, dv, segs),))
        _close(lse, rl, 1e-12, "lse vs torch logsumexp %s" % ((hq, hkv, dqk, dv, segs),))


def pin_sdpa_custom_scale(attn, seed=1):
    rng = np.random.default_rng(seed)
    q, k, v = rand_qkv(rng, 20, 2, 2, 8, 8, T=30)
    for sc in (0.5, 1.0, 0.0625):
        out, lse = attn(q, k, v, [0, 20], [0], [10], scale=sc)
        ro, rl = sdpa_reference(q, k, v, [0, 20], [0], [10], scale=sc)
        _close(out, ro, 1e-12, "out scale=%g" % sc)
        _close(lse, rl, 1e-12, "lse scale=%g" % sc)


def pin_first_token(attn, seed=2):
    """Position 0 sees only key 0: out = v_0, lse = scale*<q_0, k_0>."""
    rng = np.random.default_rng(seed)
    q, k, v = rand_qkv(rng, 10, 4, 2, 16, 8)
    # three requests each starting in this chunk at position 0
    cu, kvs, pre = [0, 3, 7, 10], [0, 3, 7], [0, 0, 0]
    out, lse = attn(q, k, v, cu, kvs, pre)
    for r in (0, 3, 7):
        for h in range(4):
            g = h // 2
            _close(out[r, h], v[r, g].double().numpy(), 0.0, "first-token out")
            want = (q[r, h].double() @ k[r, g].double()).item() / 4.0
            _close(lse[h, r], want, 1e-15, "first-token lse")


def pin_zero_keys(attn, seed=3):
    """K == 0: every visible key has weight 1/(i+1); lse = ln(i+1)."""
    rng = np.random.default_rng(seed)
    q, _, v = rand_qkv(rng, 48, 2, 1, 8, 8, T=80)
    k = torch.zeros((80, 1, 8), dtype=torch.bfloat16)
    out, lse = attn(q, k, v, [0, 48], [0], [32])
    vv = v[:, 0].double().numpy()
    for r in range(48):
        i = 32 + r
        want = vv[:i + 1].mean(axis=0)
        for h in range(2):
            _close(out[r, h], want, 1e-13, "zero-key mean row %d" % r)
            _close(lse[h, r], math.log(i + 1), 1e-13, "zero-key lse row %d" % r)


def pin_unit_values(attn, seed=4):
    """V == 1: the softmax weights sum to one, so out == 1."""
    rng = np.random.default_rng(seed)
    q, k, _ = rand_qkv(rng, 30, 3, 1, 8, 8, T=50)
    v = torch.ones((50, 1, 5), dtype=torch.bfloat16)
    out, _ = attn(q, k, v, [0, 12, 30], [0, 20], [8, 2])
    _close(out, np.ones_like(out), 1e-14, "unit values")


def pin_planted_keys(attn, seed=5):
    """q_i parallel to one chosen key j* <= i: out_i ~= v_{j*} to ~1e-9."""
    rng = np.random.default_rng(seed)
    d, T = 16, 200
    # distinct sign patterns, so every other key differs from the chosen one in
    # at least one coordinate: its score is lower by >= 2*160/16 = 20
    codes = rng.choice(1 << d, size=T, replace=False)
    bits = (codes[:, None] >> np.arange(d)[None, :]) & 1
    kk = ((2.0 * bits - 1.0) / 4.0)[:, None, :]
    k = bf16(kk)
    v = bf16(rng.standard_normal((T, 1, 8)))
    p, L = 120, 64
    targets = np.array([rng.integers(0, p + r + 1) for r in range(L)])
    targets[0], targets[1], targets[5] = p, 0, p + 5      # diagonal, first key
    q = bf16(np.stack([kk[t, 0] * 160.0 for t in targets])[:, None, :])
    out, _ = attn(q, k, v, [0, L], [0], [p], scale=1.0)
    for r in range(L):
        _close(out[r, 0], v[targets[r], 0].double().numpy(), 1e-6,
               "planted key row %d -> key %d" % (r, targets[r]))


def pin_key_translation(attn, seed=6):
    """k_j + c for every j: lse shifts by scale*<q,c>, out is unchanged (exact inputs)."""
    rng = np.random.default_rng(seed)
    d = 8
    q = bf16(rng.integers(-2, 3, size=(16, 2, d)) / 4.0)
    kk = rng.integers(-3, 4, size=(40, 1, d)).astype(np.float64)
    c = rng.integers(-2, 3, size=(d,)).astype(np.float64)
    v = bf16(rng.standard_normal((40, 1, 4)))
    cu, kvs, pre = [0, 16], [0], [24]
    o1, l1 = attn(q, bf16(kk), v, cu, kvs, pre)
    o2, l2 = attn(q, bf16(kk + c), v, cu, kvs, pre)
    shift = (q.double().numpy() @ c) / math.sqrt(d)          # [tok, Hq]
    _close(o2, o1, 1e-12, "key translation out")
    _close(l2, l1 + shift.T, 1e-12, "key translation lse")


def pin_value_translation(attn, seed=7):
    """v_j + c for every j: out shifts by c."""
    rng = np.random.default_rng(seed)
    q, k, _ = rand_qkv(rng, 16, 2, 2, 8, 4, T=40)
    vv = rng.integers(-4, 5, size=(40, 2, 4)).astype(np.float64)
    c = np.array([1.0, -2.0, 0.5, 3.0])
    o1, _ = attn(q, k, bf16(vv), [0, 16], [0], [24])
    o2, _ = attn(q, k, bf16(vv + c), [0, 16], [0], [24])
    _close(o2, o1 + c, 1e-12, "value translation")


def pin_scale_covariance(attn, seed=8):
    """(2q, scale/2) gives exactly the same scores as (q, scale)."""
    rng = np.random.default_rng(seed)
    q, k, v = rand_qkv(rng, 16, 2, 1, 8, 8, T=40)
    o1, l1 = attn(q, k, v, [0, 16], [0], [24], scale=0.3)
    o2, l2 = attn((q.float() * 2).bfloat16(), k, v, [0, 16], [0], [24], scale=0.15)
    _close(o2, o1, 1e-14, "scale covariance out")
    _close(l2, l1, 1e-14, "scale covariance lse")


def pin_causality(attn, seed=9):
    """A row depends on key/value rows 0..i of its request and on nothing after."""
    rng = np.random.default_rng(seed)
    q, k, v = rand_qkv(rng, 20, 2, 1, 8, 8, T=40)
    cu, kvs, pre = [0, 20], [0], [20]
    o1, l1 = attn(q, k, v, cu, kvs, pre)
    r = 7
    i = 20 + r
    k2, v2 = k.clone(), v.clone()
    k2[i + 1:] = bf16(rng.standard_normal((40 - i - 1, 1, 8)))
    v2[i + 1:] = bf16(rng.standard_normal((40 - i - 1, 1, 8)))
    o2, l2 = attn(q, k2, v2, cu, kvs, pre)
    _close(o2[:r + 1], o1[:r + 1], 0.0, "future keys leaked into rows <= %d" % r)
    _close(l2[:, :r + 1], l1[:, :r + 1], 0.0, "future keys leaked into lse")
    k3, v3 = k.clone(), v.clone()
    v3[i] = v3[i] + 1.0
    o3, _ = attn(q, k3, v3, cu, kvs, pre)
    assert np.all(np.abs(o3[r] - o1[r]) > 1e-6), "row %d ignores its own key" % r
    assert np.all(np.abs(o3[:r] - o1[:r]) == 0.0), "earlier rows see a later key"


def pin_chunked_equals_unchunked(attn, seed=10):
    rng = np.random.default_rng(seed)
    S, C = 96, 32
    q, k, v = rand_qkv(rng, S, 4, 2, 8, 8)
    o_full, l_full = attn(q, k, v, [0, S], [0], [0])
    for c0 in range(0, S, C):
        o, l = attn(q[c0:c0 + C], k, v, [0, C], [0], [c0])
        _close(o, o_full[c0:c0 + C], 0.0, "chunk at %d vs whole sequence" % c0)
        _close(l, l_full[:, c0:c0 + C], 0.0, "chunk lse at %d" % c0)


def pin_packed_equals_per_request(attn, seed=11):
    rng = np.random.default_rng(seed)
    lens = [13, 40, 7, 25]
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    T = int(sum(lens))
    q, k, v = rand_qkv(rng, T, 2, 1, 8, 8)
    # one packed chunk covering rows 10..69 of the stream
    t0, t1 = 10, 70
    cu, kvs, pre = [0], [], []
    for a, L in zip(starts, lens):
        lo, hi = max(a, t0), min(a + L, t1)
        if lo < hi:
            cu.append(cu[-1] + hi - lo)
            kvs.append(int(a))
            pre.append(int(lo - a))
    o, l = attn(q[t0:t1], k, v, cu, kvs, pre)
    for s in range(len(kvs)):
        a = kvs[s]
        L = lens[list(starts).index(a)]
        o_r, l_r = attn(q[a:a + L], k[a:a + L], v[a:a + L], [0, L], [0], [0])
        r0, r1 = cu[s], cu[s + 1]
        _close(o[r0:r1], o_r[pre[s]:pre[s] + (r1 - r0)], 0.0, "packed segment %d" % s)
        _close(l[:, r0:r1], l_r[:, pre[s]:pre[s] + (r1 - r0)], 0.0, "packed lse %d" % s)


def pin_gqa_equals_mha(attn, seed=12):
    rng = np.random.default_rng(seed)
    q, k, v = rand_qkv(rng, 24, 6, 2, 8, 8, T=40)
    o1, l1 = attn(q, k, v, [0, 24], [0], [16])
    o2, l2 = attn(q, k.repeat_interleave(3, dim=1), v.repeat_interleave(3, dim=1),
                  [0, 24], [0], [16])
    _close(o1, o2, 0.0, "GQA vs replicated heads")
    _close(l1, l2, 0.0, "GQA lse vs replicated heads")


ALL_PINS = [
    pin_sdpa, pin_sdpa_custom_scale, pin_first_token, pin_zero_keys, pin_unit_values,
    pin_planted_keys, pin_key_translation, pin_value_translation,
    pin_scale_covariance, pin_causality, pin_chunked_equals_unchunked,
    pin_packed_equals_per_request, pin_gqa_equals_mha,
]

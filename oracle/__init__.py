"""fp64 CPU oracle for chunked-prefill causal attention.

TEST INFRASTRUCTURE ONLY: this package is the checker, not the product. Only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it. It shares no code with the HIP library under
``paper_2608_26523_amd/``, and the product never imports it.

It evaluates Eq. (1) of the paper (section 2.1), softmax(Q K^T * scale) V, with
the causal rule of section 2.1 applied at each query's in-request position and
the chunk semantics of section 2.4 (a chunk's queries see the cached prefix of
their own request plus the earlier tokens of the chunk). The arithmetic lives in
``vpp_oracle.c`` (plain C, fp64); this module only builds it, marshals
arguments and checks shapes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vpp_oracle.c")
LIB_PATH = os.path.join(_HERE, "libvpp_oracle.so")

_libs = {}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc -O2 (no fast-math) into oracle/libvpp_oracle.so."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
               "-o", tmp, _SRC, "-lm", "-lpthread"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load(path: Optional[str] = None):
    """Load (once per path) the compiled oracle; ``path`` defaults to the in-tree build."""
    path = path or LIB_PATH
    lib = _libs.get(path)
    if lib is None:
        if path == LIB_PATH and not os.path.exists(LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(path)
        p = ctypes.c_void_p
        i64 = ctypes.c_int64
        i32 = ctypes.c_int32
        lib.vpp_oracle_attn.restype = ctypes.c_int
        lib.vpp_oracle_attn.argtypes = [
            p, i64, i64, p, i64, i64, p, i64, i64,
            i32, i32, i32, i32, ctypes.c_double,
            i32, p, p, p,
            i64, p, p, p, p, i32]
        lib.vpp_oracle_default_threads.restype = i32
        lib.vpp_oracle_default_threads.argtypes = []
        _libs[path] = lib
    return lib


def default_threads() -> int:
    return int(_load().vpp_oracle_default_threads())


def _bits(x) -> np.ndarray:
    """bf16 tensor/array -> uint16 bit-pattern ndarray (no copy when possible)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            if x.dtype != torch.bfloat16:
                raise TypeError("oracle inputs must be bfloat16")
            return x.detach().cpu().view(torch.int16).numpy().view(np.uint16)
    except ImportError:  # pragma: no cover
        pass
    a = np.asarray(x)
    if a.dtype != np.uint16:
        raise TypeError("numpy oracle inputs must be uint16 bf16 bit patterns")
    return a


def attention(q, k, v, cu_q: Sequence[int], kv_start: Sequence[int],
              prefix_len: Sequence[int], rows: Optional[Sequence[int]] = None,
              heads: Optional[Sequence[int]] = None, scale: Optional[float] = None,
              n_threads: int = 0, lib_path: Optional[str] = None
              ) -> Tuple[np.ndarray, np.ndarray]:
    """Oracle attention for selected (row, head) items.

    q: [tokens, Hq, dqk] bf16; k: [T, Hkv, dqk] bf16; v: [T, Hkv, dv] bf16 (any
    strides with a contiguous last dim). cu_q/kv_start/prefix_len describe the
    chunk's segments (see vpp_oracle.h). rows/heads select items; when both are
    None every (row, head) pair is evaluated, row-major. scale defaults to
    1/sqrt(dqk). Returns (out [n_items, dv] float64, lse [n_items] float64).
    """
    qb, kb, vb = _bits(q), _bits(k), _bits(v)
    if qb.ndim != 3 or kb.ndim != 3 or vb.ndim != 3:
        raise ValueError("q, k, v must be 3-D [tokens, heads, dim]")
    for a in (qb, kb, vb):
        if a.strides[2] != 2:
            raise ValueError("last dimension must be contiguous")
    hq, dqk = qb.shape[1], qb.shape[2]
    hkv, dv = vb.shape[1], vb.shape[2]
    if kb.shape[1] != hkv or kb.shape[2] != dqk:
        raise ValueError("k shape mismatch")
    cu = np.ascontiguousarray(cu_q, dtype=np.int32)
    ks = np.ascontiguousarray(kv_start, dtype=np.int64)
    pl = np.ascontiguousarray(prefix_len, dtype=np.int64)
    n_seg = len(ks)
    if len(cu) != n_seg + 1 or len(pl) != n_seg:
        raise ValueError("segment metadata lengths disagree")
    if int(cu[-1]) > qb.shape[0]:
        raise ValueError("cu_q[-1] exceeds the number of query rows")
    # every key the items can touch must exist in the cache arrays
    for s in range(n_seg):
        if cu[s + 1] > cu[s] and ks[s] + pl[s] + (cu[s + 1] - cu[s]) > kb.shape[0]:
            raise ValueError("segment %d reaches past the end of the cache" % s)
    if rows is None and heads is None:
        tok = int(cu[-1])
        r = np.repeat(np.arange(tok, dtype=np.int64), hq)
        h = np.tile(np.arange(hq, dtype=np.int32), tok)
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        h = np.ascontiguousarray(heads, dtype=np.int32)
        if r.shape != h.shape:
            raise ValueError("rows and heads must have the same length")
    n = int(r.shape[0])
    out = np.zeros((n, dv), dtype=np.float64)
    lse = np.zeros((n,), dtype=np.float64)
    if scale is None:
        scale = 1.0 / float(np.sqrt(dqk))
    lib = _load(lib_path)
    ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    rc = lib.vpp_oracle_attn(
        ptr(qb), qb.strides[0] // 2, qb.strides[1] // 2,
        ptr(kb), kb.strides[0] // 2, kb.strides[1] // 2,
        ptr(vb), vb.strides[0] // 2, vb.strides[1] // 2,
        hq, hkv, dqk, dv, float(scale),
        n_seg, ptr(cu), ptr(ks), ptr(pl),
        n, ptr(r), ptr(h), ptr(out), ptr(lse), int(n_threads))
    if rc != 0:
        raise RuntimeError("vpp_oracle_attn failed with code %d" % rc)
    return out, lse


def attention_full(q, k, v, cu_q, kv_start, prefix_len, scale=None, n_threads=0,
                   lib_path=None):
    """Every (row, head) of the chunk, reshaped to out [tokens, Hq, dv], lse [Hq, tokens]."""
    qb = _bits(q)
    tok, hq = int(np.asarray(cu_q)[-1]), qb.shape[1]
    out, lse = attention(q, k, v, cu_q, kv_start, prefix_len, scale=scale,
                         n_threads=n_threads, lib_path=lib_path)
    return out.reshape(tok, hq, -1), lse.reshape(tok, hq).T.copy()

"""Chunked-prefill causal attention for AMD MI355X (gfx950).

The hot path of VPP (virtual pipeline parallelism for chunked prefill): a chunk
of C query tokens at prefix offset p attends causally to the p cached prefix
tokens plus itself. The arithmetic runs in hand-written HIP kernels behind the C
ABI of include/vpp_chunk_attn.h; this package holds the ctypes binding, a thin
torch wrapper (device memory and streams only) and the workload registry.
"""
from . import binding  # noqa: F401
from . import workloads  # noqa: F401

__all__ = ["binding", "workloads", "ChunkAttention"]


def __getattr__(name):
    if name == "ChunkAttention":
        from .attention import ChunkAttention
        return ChunkAttention
    raise AttributeError(name)

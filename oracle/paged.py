"""Reference definitions of the paged KV cache (plain numpy, host).

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): the checker of
``vpp_chunk_attn_run_paged``, ``vpp_kv_append_paged`` and
``vpp_paged_slot_mapping``; it shares no code with the library.

A paged cache holds the rows of each request in fixed-size pages: cache row j
of a request whose block-table row is ``bt`` lives in page ``bt[j // P]`` at
row ``j % P``. Attention over a paged cache is attention over the contiguous
rows this mapping yields (section 2.4's chunk semantics are unchanged), so the
attention oracle runs on ``contiguous_rows``.
"""
from __future__ import annotations

import numpy as np


def contiguous_rows(pages: np.ndarray, bt_row: np.ndarray, nrows: int) -> np.ndarray:
    """Rows 0 .. nrows-1 of one request, gathered from pages [num_pages, P, ...]."""
    P = pages.shape[1]
    out = np.empty((nrows,) + pages.shape[2:], dtype=pages.dtype)
    for j in range(nrows):
        out[j] = pages[int(bt_row[j // P]), j % P]
    return out


def slot_mapping(cu_q, kv_start, prefix_len, block_table, page_size) -> np.ndarray:
    """Slot (page * P + row) of every chunk row: segment s's row r sits at cache row
    kv_start[s] + prefix_len[s] + (r - cu_q[s]) of its request."""
    slots = np.zeros(int(cu_q[-1]), dtype=np.int64)
    for s in range(len(kv_start)):
        for r in range(int(cu_q[s]), int(cu_q[s + 1])):
            j = int(kv_start[s]) + int(prefix_len[s]) + (r - int(cu_q[s]))
            slots[r] = int(block_table[s][j // page_size]) * page_size + j % page_size
    return slots


def append(pages: np.ndarray, rows: np.ndarray, slots: np.ndarray) -> np.ndarray:
    """The pages after writing rows[t] at slots[t] (slots outside the cache are skipped)."""
    out = pages.copy()
    P = pages.shape[1]
    cap = pages.shape[0] * P
    for t, sl in enumerate(slots):
        sl = int(sl)
        if 0 <= sl < cap:
            out[sl // P, sl % P] = rows[t]
    return out

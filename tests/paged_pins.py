"""Pins of the paged-cache reference (``oracle/paged.py``), CPU only.

Each pin takes the module under test, so the same checks run on the real
reference and on copies of it with planted mistakes. Expected values are
literals worked out by hand from the page mapping (cache row j of a request
with block-table row bt lives in page bt[j // P] at row j % P), or come from a
plain numpy reshape of the page pool; none is computed by the reference itself.
"""
from __future__ import annotations

import numpy as np


def pin_slot_mapping_by_hand(m):
    """Two segments, 64-row pages, a table written out by hand.

    Segment 0: rows 0..2 at cache rows 126, 127, 128 of its request (kv_start 0,
    prefix 126). Rows 126 and 127 are in table entry 1 (page 3), rows 62 and 63 of
    it; row 128 is in entry 2 (page 9), row 0. Segment 1: rows 3..4 at cache rows
    64, 65 (kv_start 64, prefix 0): entry 1 of its own table row (page 2), rows 0, 1.
    """
    bt = np.array([[7, 3, 9], [5, 2, 8]], dtype=np.int32)
    got = m.slot_mapping([0, 3, 5], [0, 64], [126, 0], bt, 64)
    want = [3 * 64 + 62, 3 * 64 + 63, 9 * 64 + 0, 2 * 64 + 0, 2 * 64 + 1]
    assert list(np.asarray(got)) == want, (list(got), want)


def pin_slot_mapping_page_boundary(m):
    """A segment whose rows cross two page boundaries (page size 4, table [6, 1, 4]):
    cache rows 2..9 -> entries 0, 0, 1, 1, 1, 1, 2, 2 at in-page rows 2, 3, 0, 1, 2, 3, 0, 1."""
    bt = np.array([[6, 1, 4]], dtype=np.int32)
    got = m.slot_mapping([0, 8], [0], [2], bt, 4)
    want = [26, 27, 4, 5, 6, 7, 16, 17]
    assert list(np.asarray(got)) == want, (list(got), want)


def _pool(num_pages, page, width=1):
    """pages[pg, r, c] = 100 * pg + 10 * r + c (small integers, exact in any dtype)."""
    pg = np.arange(num_pages)[:, None, None]
    r = np.arange(page)[None, :, None]
    c = np.arange(width)[None, None, :]
    return (100 * pg + 10 * r + c).astype(np.int64)


def pin_contiguous_identity(m):
    """With the identity table the gathered rows are the pool read in order."""
    pages = _pool(4, 3, 2)
    got = m.contiguous_rows(pages, np.arange(4, dtype=np.int32), 10)
    want = pages.reshape(12, 2)[:10]
    assert np.array_equal(got, want)


def pin_contiguous_by_hand(m):
    """Page size 2, table [2, 0, 1], 5 rows: pages 2, 2, 0, 0, 1 at in-page rows 0, 1, 0, 1, 0."""
    pages = _pool(3, 2, 1)
    got = m.contiguous_rows(pages, np.array([2, 0, 1], dtype=np.int32), 5)
    assert list(got[:, 0]) == [200, 210, 0, 10, 100], list(got[:, 0])


def pin_contiguous_reversed(m):
    """A reversed table reads the pool's pages back to front, rows in order within each."""
    pages = _pool(3, 2, 1)
    got = m.contiguous_rows(pages, np.array([2, 1, 0], dtype=np.int32), 6)
    assert list(got[:, 0]) == [200, 210, 100, 110, 0, 10], list(got[:, 0])


def pin_append_by_hand(m):
    """Three pages of two rows; rows 1..5 go to slots 5, -1, 0, 6, 3: slot 5 is page 2
    row 1, slot 0 is page 0 row 0, slot 3 is page 1 row 1; -1 and 6 (one past the
    pool) are skipped; every other row keeps its old value."""
    pages = -np.ones((3, 2, 1), dtype=np.int64)
    rows = np.array([[1], [2], [3], [4], [5]], dtype=np.int64)
    got = m.append(pages, rows, np.array([5, -1, 0, 6, 3], dtype=np.int64))
    want = np.array([[[3], [-1]], [[-1], [5]], [[-1], [1]]], dtype=np.int64)
    assert np.array_equal(got, want), got[:, :, 0]
    assert np.array_equal(pages, -np.ones((3, 2, 1), dtype=np.int64)), "input pages modified"


def pin_append_then_gather(m):
    """Rows appended at the slots of a slot mapping are read back, in order, by the
    gather of the same table (slot mapping, append and gather agree on the mapping)."""
    bt = np.array([[4, 0, 2]], dtype=np.int32)
    slots = m.slot_mapping([0, 5], [0], [1], bt, 2)   # cache rows 1..5 of the request
    pages = np.zeros((5, 2, 1), dtype=np.int64)
    rows = np.array([[11], [12], [13], [14], [15]], dtype=np.int64)
    filled = m.append(pages, rows, slots)
    got = m.contiguous_rows(filled, bt[0], 6)
    assert list(got[:, 0]) == [0, 11, 12, 13, 14, 15], list(got[:, 0])


PINS = [pin_slot_mapping_by_hand, pin_slot_mapping_page_boundary, pin_contiguous_identity,
        pin_contiguous_by_hand, pin_contiguous_reversed, pin_append_by_hand, pin_append_then_gather]

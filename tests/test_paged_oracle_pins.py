"""The paged-cache reference against hand-worked pins, and planted mistakes in copies
of it that a pin must catch (CPU only).

The mutants are textual edits of ``oracle/paged.py`` loaded as separate modules;
the real reference is not touched. They are the plausible mistakes of a page
mapping: page index and in-page row swapped, an off-by-one table entry, the wrong
table row for a segment, the prefix or the request base ignored, a skipped bound
that lets an out-of-range slot through, and row/page swapped in the scatter.
"""
import os
import types

import pytest

import paged_pins as PP
from oracle import paged as OP

SRC = OP.__file__

MUTANTS = {
    "gather_div_mod_swapped": [("pages[int(bt_row[j // P]), j % P]", "pages[int(bt_row[j % P]), j // P]")],
    "gather_table_off_by_one": [("pages[int(bt_row[j // P]), j % P]",
                                 "pages[int(bt_row[min(j // P + 1, len(bt_row) - 1)]), j % P]")],
    "slots_div_mod_swapped": [("int(block_table[s][j // page_size]) * page_size + j % page_size",
                               "int(block_table[s][j % page_size]) * page_size + j // page_size")],
    "slots_wrong_table_row": [("int(block_table[s][j // page_size])", "int(block_table[0][j // page_size])")],
    "slots_prefix_ignored": [("j = int(kv_start[s]) + int(prefix_len[s]) + (r - int(cu_q[s]))",
                              "j = int(kv_start[s]) + (r - int(cu_q[s]))")],
    "slots_base_ignored": [("j = int(kv_start[s]) + int(prefix_len[s]) + (r - int(cu_q[s]))",
                            "j = int(prefix_len[s]) + (r - int(cu_q[s]))")],
    "append_bound_inclusive": [("if 0 <= sl < cap:", "if 0 <= sl <= cap and sl < cap + P:")],
    "append_negative_wraps": [("if 0 <= sl < cap:", "if sl < cap:")],
    "append_row_page_swapped": [("out[sl // P, sl % P] = rows[t]",
                                 "out[sl % pages.shape[0], (sl // pages.shape[0]) % P] = rows[t]")],
}


def _load_mutant(name, edits):
    text = open(SRC).read()
    for old, new in edits:
        assert old in text, "paged reference changed; update mutant %s" % name
        text = text.replace(old, new)
    mod = types.ModuleType("paged_mutant_" + name)
    exec(compile(text, "<%s>" % name, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("pin", PP.PINS, ids=lambda f: f.__name__)
def test_reference_passes_pin(pin):
    pin(OP)


def _caught(mod):
    for pin in PP.PINS:
        try:
            pin(mod)
        except Exception:   # a wrong value or an out-of-range access both expose the mistake
            return pin.__name__
    return None


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _load_mutant(name, MUTANTS[name])
    assert _caught(mod) is not None, "no pin catches mutant %s" % name


def test_mutant_sources_apply():
    # every edit still matches the current reference text (guards against silent no-op mutants)
    text = open(SRC).read()
    for name, edits in MUTANTS.items():
        for old, _ in edits:
            assert old in text, name
    assert os.path.exists(SRC)

"""Planted mistakes in copies of the oracle must each fail at least one pin (CPU only).

Every mutant is a textual edit of oracle/vpp_oracle.c compiled into a temporary
directory; the real oracle is not touched. The edits are the plausible mistakes
an implementation of causal chunked attention can make: the mask off by one,
the prefix or the request base ignored, the wrong kv head for a query head, a
dropped scale, lse in the wrong logarithm base, a value row shifted against its
key, an extra term in the denominator, a flipped exponent sign.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins as P

SRC = os.path.join(os.path.dirname(oracle.__file__), "vpp_oracle.c")

MUTANTS = {
    "mask_excludes_diagonal": [("j <= i; ++j) {\n        const uint16_t* krow",
                                "j < i; ++j) {\n        const uint16_t* krow"),
                               ("for (int64_t j = 0; j <= i; ++j) {\n        const double e",
                                "for (int64_t j = 0; j < i; ++j) {\n        const double e"),
                               ("for (int64_t j = 0; j <= i; ++j) wsum",
                                "for (int64_t j = 0; j < i; ++j) wsum")],
    "prefix_ignored": [("const int64_t i = J->prefix_len[seg] + (r - J->cu_q[seg]);",
                        "const int64_t i = (r - J->cu_q[seg]);")],
    "request_base_ignored": [("const int64_t base = J->kv_start[seg];",
                              "const int64_t base = 0;")],
    "gqa_modulo_mapping": [("const int32_t g = h / group;",
                            "const int32_t g = h % J->hkv; (void)group;")],
    "scale_dropped": [("s[j] = J->scale * dot;", "s[j] = dot;")],
    "lse_log2": [("J->lse[n] = m + log(l);", "J->lse[n] = m + log2(l);")],
    "value_row_shifted": [("J->v + (base + j) * J->v_st",
                           "J->v + (base + j - (j > 0)) * J->v_st")],
    "extra_denominator_term": [("double l = 0.0;", "double l = 1.0;")],
    "exponent_sign_flipped": [("const double e = exp(s[j] - m);",
                               "const double e = exp(m - s[j]);")],
}


# The oracle's own self-check (weights sum to one) is switched off in every
# mutant so that each planted mistake has to be caught by a pin's value check.
NO_SELFCHECK = ("if (!(fabs(wsum - 1.0) <= 1e-12)) return VPP_ORACLE_ESELFCHECK;",
                "(void)wsum;")


def _build_mutant(tmp_path, name, edits):
    text = open(SRC).read()
    for old, new in list(edits) + [NO_SELFCHECK]:
        assert old in text, "oracle source changed; update mutant %s" % name
        text = text.replace(old, new)
    src = tmp_path / ("%s.c" % name)
    src.write_text(text)
    lib = tmp_path / ("lib%s.so" % name)
    hdr_dir = os.path.dirname(SRC)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-I", hdr_dir,
                    "-o", str(lib), str(src), "-lm", "-lpthread"], check=True)
    return str(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    lib = _build_mutant(tmp_path, name, MUTANTS[name])

    def attn(*a, **kw):
        return oracle.attention_full(*a, lib_path=lib, **kw)

    caught = []
    for pin in P.ALL_PINS:
        try:
            pin(attn)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, "mutant %s passed every pin" % name


def test_unmutated_copy_passes(tmp_path):
    lib = _build_mutant(tmp_path, "identity", [])

    def attn(*a, **kw):
        return oracle.attention_full(*a, lib_path=lib, **kw)

    for pin in P.ALL_PINS:
        pin(attn)

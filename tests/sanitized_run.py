"""Run CPU tests against a sanitizer-instrumented build of one native library.

Invoked in a subprocess by tests/test_sanitizers_cpu.py (with the matching
sanitizer runtime preloaded): ``python sanitized_run.py {oracle|sched|attn} LIB [TEST ...]``.
For the oracle it runs the oracle pins through LIB; for the schedule model and the
attention library it points the binding at LIB and runs the given pytest files.
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path[:0] = [ROOT, HERE]


def main():
    which, lib, tests = sys.argv[1], sys.argv[2], sys.argv[3:]
    if which == "oracle":
        import oracle
        import oracle_pins as P

        def attn(*a, **kw):
            return oracle.attention_full(*a, lib_path=lib, **kw)
        for pin in P.ALL_PINS:
            pin(attn)
        print("oracle pins passed under the sanitizers", flush=True)
        return 0
    if which == "attn":
        from paper_2608_26523_amd import binding
        binding.LIB_PATH = lib
        assert binding.load()._name == lib
    elif which == "sched":
        from paper_2608_26523_amd import schedule
        schedule.LIB_PATH = lib
    else:
        raise SystemExit("unknown library %s" % which)
    import pytest
    return pytest.main(["-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu"] + tests)


if __name__ == "__main__":
    sys.exit(main())

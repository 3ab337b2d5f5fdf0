"""The native host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Each library is rebuilt with the sanitizers into a temporary directory and
exercised in a subprocess that preloads the matching runtime (Python itself is
not instrumented):

* the fp64 oracle (gcc): every oracle pin;
* the schedule model (g++): the schedule tests;
* the attention library's host code (hipcc, sanitizers on the host side only:
  the planner, argument checks and introspection): the ABI, planner, kernel
  index-model and paged host tests, none of which needs a GPU.

A copy of the oracle with a planted out-of-bounds read must abort under the same
setup, which shows the instrumentation is live.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
RUNNER = os.path.join(HERE, "sanitized_run.py")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
       "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _gcc_asan():
    return subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()


def _clang_asan():
    import glob
    hits = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    return hits[0] if hits else None


def _run(preload, which, lib, tests=()):
    env = dict(os.environ)
    env.update(ENV)
    env["LD_PRELOAD"] = preload
    return subprocess.run([sys.executable, RUNNER, which, lib] + list(tests), env=env,
                          capture_output=True, text=True, timeout=900)


def _build_oracle(tmp_path, src_text=None, name="liboracle_san.so"):
    src = os.path.join(ROOT, "oracle", "vpp_oracle.c")
    if src_text is not None:
        p = tmp_path / "oracle_copy.c"
        p.write_text(src_text)
        src = str(p)
    lib = str(tmp_path / name)
    subprocess.run(["gcc", "-std=c11", "-fPIC", "-shared"] + SAN +
                   ["-I", os.path.join(ROOT, "oracle"), "-o", lib, src, "-lm", "-lpthread"], check=True)
    return lib


def test_oracle_under_sanitizers(tmp_path):
    lib = _build_oracle(tmp_path)
    r = _run(_gcc_asan(), "oracle", lib)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "oracle pins passed" in r.stdout


def test_planted_overflow_is_caught(tmp_path):
    text = open(os.path.join(ROOT, "oracle", "vpp_oracle.c")).read()
    old = "for (int64_t j = 0; j <= i; ++j) wsum"
    assert old in text
    lib = _build_oracle(tmp_path, text.replace(old, "for (int64_t j = 0; j <= i + 4096; ++j) wsum"), "libbad.so")
    r = _run(_gcc_asan(), "oracle", lib)
    assert r.returncode != 0 and "AddressSanitizer" in r.stderr


def test_schedule_model_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libsched_san.so")
    subprocess.run(["g++", "-std=c++17", "-fPIC", "-shared"] + SAN +
                   ["-I", os.path.join(ROOT, "include"), "-o", lib,
                    os.path.join(ROOT, "paper_2608_26523_amd", "csrc", "vpp_sched.cpp")], check=True)
    r = _run(_gcc_asan(), "sched", lib, [os.path.join(HERE, "test_schedule_cpu.py")])
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]


def test_attention_host_code_under_sanitizers(tmp_path):
    rt = _clang_asan()
    if rt is None:
        pytest.skip("no clang AddressSanitizer runtime in this ROCm install")
    from paper_2608_26523_amd import build as Bld
    lib = str(tmp_path / "libvpp_san.so")
    # sanitizers on the host side only: -Xarch_host before each -fsanitize
    host_san = ["-g", "-fno-omit-frame-pointer",
                "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all"]
    Bld.build(extra_flags=host_san, out=lib)
    tests = [os.path.join(HERE, t) for t in ("test_abi_cpu.py", "test_kernel_bounds_cpu.py", "test_paged_cpu.py")]
    r = _run(rt, "attn", lib, tests)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]

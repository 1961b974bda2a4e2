"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

- The C oracle, built with gcc -fsanitize=address,undefined, runs a set of its
  pins and a ragged selection in a child process with the gcc sanitizer runtime
  preloaded.
- The C ABI layer (ress_api.cpp), built with host sanitizers only (each
  -fsanitize= behind -Xarch_host: the device code is untouched) and linked with
  launchers that enqueue nothing, runs the host-side argument checks in a child
  process with clang's sanitizer runtime preloaded.
A sanitizer report or a failed check fails the test."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run_child(code_or_args, preload, timeout=600):
    env = dict(os.environ, LD_PRELOAD=preload, OMP_NUM_THREADS="4", **SAN_ENV)
    env["PYTHONPATH"] = os.pathsep.join([ROOT, HERE] + [env.get("PYTHONPATH", "")])
    r = subprocess.run([sys.executable] + code_or_args, capture_output=True, text=True, env=env, timeout=timeout)
    report = [l for l in (r.stdout + r.stderr).splitlines() if "Sanitizer" in l or "runtime error:" in l]
    assert r.returncode == 0 and not report, (r.returncode, report[:10], r.stderr[-3000:])
    return r.stdout


def test_harness_reports_a_planted_overflow(tmp_path):
    """The set-up itself: a heap overflow planted in a tiny C library is reported."""
    src = tmp_path / "bad.c"
    src.write_text("#include <stdlib.h>\nint bad(int n) { int *a = malloc(4 * n); int s = a[n]; free(a); return s; }\n")
    lib = tmp_path / "libbad.so"
    subprocess.run(["gcc", "-O0", "-g", "-fsanitize=address,undefined", "-fPIC", "-shared", str(src), "-o", str(lib)],
                   check=True)
    preload = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    with pytest.raises(AssertionError, match="heap-buffer-overflow"):
        _run_child(["-c", f"import ctypes; ctypes.CDLL({str(lib)!r}).bad(8)"], preload)


def test_oracle_under_sanitizers(tmp_path):
    lib = tmp_path / "libress_oracle_san.so"
    subprocess.run(["gcc", "-std=c99", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                    os.path.join(ROOT, "oracle", "ress_oracle.c"), "-o", str(lib), "-lm"], check=True)
    preload = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    code = f"""
import numpy as np
import oracle, pins, synth
with oracle.use_library({str(lib)!r}):
    for check in (pins.check_pool, pins.check_select_driver, pins.check_trajectory, pins.check_track_best,
                  pins.check_margin, pins.check_cdf_threshold, pins.check_drift_max, pins.check_edges,
                  pins.check_attention, pins.check_zero_sparsity):
        check()
    L = synth.make_layer(3, 150, 5, H=2, bq=128, bk=64, sparsity=0.6, seed=5, name="ragged")
    for crit, tau in ((0, 0.0), (1, 0.7), (3, 0.0)):
        oracle.select(L.q, L.k, L.v, L.gram, L.budgets, N=L.N, bq=L.bq, bk=L.bk, n_special=L.n_special_tail,
                      rounds=5, criterion=crit, cdf_tau=tau)
print("oracle checks ok")
"""
    out = _run_child(["-c", code], preload)
    assert "oracle checks ok" in out


def test_abi_layer_under_sanitizers(tmp_path):
    rt = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        pytest.skip("clang sanitizer runtime not found")
    inc = ["-I" + os.path.join(ROOT, "include"), "-I" + os.path.join(ROOT, "paper_2609_35593_amd", "csrc")]
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
    base = [HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Xclang", "-target-feature",
            "-Xclang", "-packed-fp32-ops", *inc, "-x", "hip", "-c"]
    api_o, stub_o, lib = tmp_path / "api.o", tmp_path / "stub.o", tmp_path / "libress_san.so"
    subprocess.run([*base, *san, os.path.join(ROOT, "paper_2609_35593_amd", "csrc", "ress_api.cpp"), "-o", str(api_o)],
                   check=True, capture_output=True)
    subprocess.run([*base, os.path.join(HERE, "sanitize", "launch_stubs.cpp"), "-o", str(stub_o)], check=True,
                   capture_output=True)
    subprocess.run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", str(api_o), str(stub_o), "-o", str(lib)],
                   check=True, capture_output=True)
    out = _run_child([os.path.join(HERE, "sanitize", "abi_checks.py"), str(lib)], rt[-1])
    assert "abi checks ok" in out

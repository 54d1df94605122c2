"""Native code under AddressSanitizer and UndefinedBehaviorSanitizer, on the
CPU (no GPU: device code is not instrumented).

* The host side of libnetsim (netsim.cpp, fabric.cpp: validation, routing,
  decomposition, the stream front end, device layout up to the first device
  call) is rebuilt with the host compilation instrumented, and the host-side
  tests run against that build in a subprocess with the sanitizer runtime
  preloaded.
* The oracle (netsim_oracle.c) is rebuilt with gcc's sanitizers and its pin
  tests run against that build the same way.
* A bounds-checked host model of the default solver's one-workgroup rate
  solve (the gather, both phases of a freezing round, the write-back) runs
  at every number of path records in flight per thread from 1 to 8 over
  re-solve sizes of the 4096-GPU workload.

Every check must report no error; sanitizer reports make the subprocess fail.
"""

import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = "/opt/rocm/bin/hipcc"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:verify_asan_link_order=0",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}

pytestmark = pytest.mark.slow


def _run(cmd, env=None, timeout=900):
    r = subprocess.run(cmd, cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=timeout)
    assert r.returncode == 0, r.stdout[-4000:]
    return r.stdout


def _env(preload, **kw):
    env = dict(os.environ)
    env.update(SAN_ENV)
    env["LD_PRELOAD"] = preload
    env.update(kw)
    return env


def test_solve_mask_index_model(tmp_path):
    exe = str(tmp_path / "solve_mask_index")
    _run(["g++", "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=undefined", "-o", exe,
          os.path.join(ROOT, "tests", "native", "solve_mask_index.cpp")])
    out = _run([exe], env=_env(""))
    for d in range(1, 9):
        assert f"depth {d}: 132 cases, in bounds" in out, out


def test_oracle_under_sanitizers(tmp_path):
    lib = str(tmp_path / "oracle_san.so")
    _run(["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-o", lib,
          os.path.join(ROOT, "oracle", "netsim_oracle.c"), "-lm"])
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], stdout=subprocess.PIPE,
                          text=True).stdout.strip()
    ubsan = subprocess.run(["gcc", "-print-file-name=libubsan.so"], stdout=subprocess.PIPE,
                           text=True).stdout.strip()
    out = _run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                "tests/test_oracle_pins.py", "tests/test_oracle_next4.py",
                "tests/test_oracle_timeline.py", "-k", "not c3"],
               env=_env(f"{asan}:{ubsan}", NETSIM_ORACLE_LIB=lib))
    assert " passed" in out and "failed" not in out


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="no hipcc")
def test_host_library_under_sanitizers(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2505_01616_amd import build as b
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rt:
        pytest.skip("no clang AddressSanitizer runtime")
    lib = str(tmp_path / "libnetsim_san.so")
    flags = [f for f in b.FLAGS if f != "-O3"]
    srcs = [os.path.join(b.CSRC, s) for s in b.SOURCES]
    # the host compilation only is instrumented
    _run([HIPCC, *flags, "-O1", "-g", "-Xarch_host", "-fsanitize=address",
          "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=undefined",
          "-I", os.path.join(ROOT, "include"), "-I", b.CSRC, "-o", lib, *srcs])
    out = _run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                "tests/test_lib_host.py", "tests/test_trace_host.py", "tests/test_next4_host.py"],
               env=_env(rt[0], NETSIM_LIB=lib))
    assert " passed" in out and "failed" not in out
    shutil.rmtree(tmp_path, ignore_errors=True)

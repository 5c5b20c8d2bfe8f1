"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU): libdg is rebuilt with both sanitizers on its host code (its
device code is not instrumented), and the host ABI tests (every entry point's
argument checks, the workspace and bound queries with their buffer carving, the
error text) run against that build with the sanitizer runtime preloaded.  They
must pass, and the sanitizers must report nothing."""
import os
import subprocess
import sys

import pytest

from conftest import ROOT

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang"
SAN_EXIT = 87


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                    reason="the ROCm compilers are not available")
def test_host_abi_checks_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    if os.environ.get("LD_PRELOAD") or os.path.exists("/etc/ld.so.preload"):
        pytest.skip("a preloaded library is already in place; it is not replaced")
    sys.path.insert(0, ROOT)
    from paper_2405_05231_amd import build

    lib = str(tmp_path / "libdg_san.so")
    flags = [f for f in build.FLAGS if f != "-O3"]
    san = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer"]
    cmd = [HIPCC, *flags, "-O1", "-g", *[x for f in san for x in ("-Xarch_host", f)],
           "-I", build.INCLUDE, "-I", build.CSRC, *build.sources(), "-o", lib]
    b = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert b.returncode == 0, b.stderr[-3000:]
    # the build is instrumented
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms

    runtime = subprocess.run([CLANG, "--print-file-name=libclang_rt.asan-x86_64.so"],
                             capture_output=True, text=True, check=True).stdout.strip()
    env = dict(os.environ, DG_LIB_PATH=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS=f"detect_leaks=0:exitcode={SAN_EXIT}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:exitcode={SAN_EXIT}")
    # the binding loads that build
    probe = ("from paper_2405_05231_amd import _lib; import sys; "
             "sys.exit(0 if _lib.load()._name == sys.argv[1] else 3)")
    p = subprocess.run([sys.executable, "-c", probe, lib], capture_output=True, text=True,
                       env=env, cwd=ROOT, timeout=300)
    assert p.returncode == 0, p.stderr[-3000:]
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"),
                        "-q", "-p", "no:cacheprovider"], capture_output=True, text=True, env=env,
                       cwd=ROOT, timeout=600)
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, \
        r.stderr[-3000:]
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]

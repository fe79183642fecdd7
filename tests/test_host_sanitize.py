"""Host code of the library under AddressSanitizer + UndefinedBehaviorSanitizer
(CPU only): tests/sanitize/host_checks.cpp drives configuration validation,
workspace sizing for the largest supported shapes, every entry point's
argument checks and the router / renderer.  The runtime's host half is built
with the sanitizers (its device code is unchanged), the router and the driver
with ROCm's clang++, and the kernels' objects come from the regular build or
are compiled here."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2606_12154_amd import build as B  # noqa: E402

CLANGXX = "/opt/rocm/llvm/bin/clang++"
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
CXX_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
INC = ["-I" + os.path.join(ROOT, "include"), "-I" + B.CSRC]


def _run(cmd, **kw):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, **kw)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout[-4000:]
    return r.stdout


@pytest.mark.skipif(not (os.path.exists(B.HIPCC) and os.path.exists(CLANGXX)), reason="ROCm toolchain not present")
def test_host_code_under_asan_ubsan(tmp_path):
    objs = []
    jobs = []
    # Kernel translation units (their launchers are host code too, but the
    # driver reaches none of them): reuse the regular build when current.
    for src in B.SOURCES:
        if src in ("runtime.hip", "router.cpp"):
            continue
        o = os.path.join(B.BUILD, os.path.splitext(src)[0] + ".o")
        if not (os.path.exists(o) and os.path.getmtime(o) >= os.path.getmtime(os.path.join(B.CSRC, src))):
            o = str(tmp_path / (os.path.splitext(src)[0] + ".o"))
            jobs.append([B.HIPCC] + B.FLAGS + ["-c", os.path.join(B.CSRC, src), "-o", o])
        objs.append(o)
    rt = str(tmp_path / "runtime_san.o")
    jobs.append([B.HIPCC] + B.FLAGS + ["-O1", "-g"] + HOST_SAN + ["-c", os.path.join(B.CSRC, "runtime.hip"), "-o", rt])
    ro = str(tmp_path / "router_san.o")
    jobs.append([CLANGXX, "-std=c++17", "-O1", "-g", "-fPIC"] + CXX_SAN + INC +
                ["-c", os.path.join(B.CSRC, "router.cpp"), "-o", ro])
    dr = str(tmp_path / "host_checks.o")
    jobs.append([CLANGXX, "-std=c++17", "-O1", "-g"] + CXX_SAN + INC +
                ["-c", os.path.join(ROOT, "tests", "sanitize", "host_checks.cpp"), "-o", dr])
    procs = [subprocess.Popen(j, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True) for j in jobs]
    for j, p in zip(jobs, procs):
        out = p.communicate()[0]
        assert p.returncode == 0, " ".join(j) + "\n" + out[-4000:]
    exe = str(tmp_path / "host_checks")
    _run([CLANGXX] + CXX_SAN + [dr, rt, ro] + objs + ["-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
                                                     "-o", exe])
    env = dict(os.environ)
    # Leaks are checked; the HIP runtime's own process-lifetime allocations
    # are not the library's.
    supp = tmp_path / "lsan.supp"
    supp.write_text("leak:libamdhip64\nleak:libhsa-runtime64\nleak:libamd_comgr\n")
    env["ASAN_OPTIONS"] = "detect_leaks=1:halt_on_error=1"
    env["LSAN_OPTIONS"] = f"suppressions={supp}"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "host checks passed" in r.stdout, r.stdout[-6000:]
    assert "runtime error" not in r.stdout and "ERROR: AddressSanitizer" not in r.stdout, r.stdout[-6000:]

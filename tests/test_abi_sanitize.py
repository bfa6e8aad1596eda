"""Host AddressSanitizer + UndefinedBehaviorSanitizer over the C ABI's
validation paths (CPU only, no GPU calls).

The runtime's host code (ifvs_host.hip) is compiled with both sanitizers on
its host side only (each -fsanitize= after -Xarch_host; the device code is
built as usual), linked with the other objects into a separate library, and
exercised by tests/abi_sanitize.cpp, itself built with the sanitizers: every
entry point on a NULL handle, every malformed index-descriptor field, and a
well-formed load (IFVS_E_HIP without a GPU).  A memory error, a leak of the
library's own allocations or undefined behaviour fails the run."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
CLANGXX = "/opt/rocm/llvm/bin/clang++"
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    from paper_2607_22922_amd import build as BLD
    if not (shutil.which(BLD.HIPCC) or os.path.exists(BLD.HIPCC)) or not os.path.exists(CLANGXX):
        pytest.skip("hipcc / clang++ not available")
    out = tmp_path_factory.mktemp("abi_san")
    os.makedirs(BLD.BUILD, exist_ok=True)
    objs = []
    deps = [os.path.join(BLD.CSRC, f) for f in os.listdir(BLD.CSRC) if f.endswith(".h")]
    deps.append(os.path.join(ROOT, "include", "ifvs.h"))
    newest_dep = max(os.path.getmtime(p) for p in deps)
    for src in BLD.SOURCES:
        if src == "ifvs_host.hip":
            continue
        obj = os.path.join(BLD.BUILD, src.replace(".hip", ".o"))
        path = os.path.join(BLD.CSRC, src)
        if not os.path.exists(obj) or os.path.getmtime(obj) < max(os.path.getmtime(path), newest_dep):
            obj = BLD._compile(src)
        objs.append(obj)
    host_obj = str(out / "ifvs_host_san.o")
    r = subprocess.run([BLD.HIPCC, *BLD.FLAGS, *SAN_HOST, "-g", "-c", os.path.join(BLD.CSRC, "ifvs_host.hip"),
                        "-o", host_obj], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    lib = str(out / "libifvs_san.so")
    r = subprocess.run([BLD.HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", lib, host_obj, *objs],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    exe = str(out / "abi_sanitize")
    r = subprocess.run([CLANGXX, "-std=c++17", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                        "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
                        os.path.join(ROOT, "tests", "abi_sanitize.cpp"), "-L", str(out), "-lifvs_san",
                        "-Wl,-rpath," + str(out), "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return lib, exe


def test_sanitized_library_is_instrumented(sanitized):
    lib, _ = sanitized
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms


def test_validation_paths_under_asan_and_ubsan(sanitized):
    _, exe = sanitized
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["LSAN_OPTIONS"] = "suppressions=" + os.path.join(ROOT, "tests", "abi_sanitize.supp")
    env["HIP_VISIBLE_DEVICES"] = ""          # no device: the well-formed load must fail cleanly
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    report = r.stdout + r.stderr
    assert "AddressSanitizer" not in report and "runtime error" not in report, report[-6000:]
    assert r.returncode == 0, report[-6000:]
    assert "all statuses as documented" in r.stdout

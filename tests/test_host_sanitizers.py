"""The host side of the C ABI (argument validation, split plans, workspace
sizes, status strings) under AddressSanitizer and UndefinedBehaviorSanitizer.

The library is rebuilt with the sanitizers on its host code only (the device
code is compiled as usual and never runs), then the ABI tests run against it
in a child process that preloads the sanitizer runtime.  No GPU is needed."""
import glob
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# host-only instrumentation: every -fsanitize= applies to the host pass alone
SANITIZE = ("-O1 -g -Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
            "-Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer "
            "-shared-libsan").split()


def asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def build_sanitized(out):
    from paper_2609_20734_amd import build as B
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    flags = [f for f in B.HIPCC_FLAGS if f != "-O3"] + SANITIZE
    cmd = [hipcc, *flags, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(B.PKG, "csrc"),
           *B.sources(), "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert res.returncode == 0, (res.stdout + res.stderr)[-4000:]
    return out


def sanitized_tree(tmp_path, lib):
    """A copy of the package (the sanitized build as its liboda.so), the
    header and the ABI tests, so the tests load the instrumented library."""
    tree = tmp_path / "tree"
    shutil.copytree(os.path.join(ROOT, "paper_2609_20734_amd"), tree / "paper_2609_20734_amd",
                    ignore=shutil.ignore_patterns("__pycache__", "*.so", "*.so.tmp"))
    shutil.copy(lib, tree / "paper_2609_20734_amd" / "liboda.so")
    shutil.copytree(os.path.join(ROOT, "include"), tree / "include")
    (tree / "tests").mkdir()
    for f in ("conftest.py", "test_abi.py"):
        shutil.copy(os.path.join(ROOT, "tests", f), tree / "tests" / f)
    return tree


def test_abi_checks_pass_under_host_sanitizers(tmp_path):
    rt = asan_runtime()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime in this toolchain")
    lib = build_sanitized(str(tmp_path / "liboda_sanitized.so"))
    # the instrumented library needs the sanitizer runtime, i.e. the build took effect
    dyn = subprocess.run(["readelf", "-d", lib], capture_output=True, text=True).stdout
    assert "libclang_rt.asan" in dyn, dyn
    tree = sanitized_tree(tmp_path, lib)
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, LD_LIBRARY_PATH=os.path.dirname(rt) + os.pathsep + env.get("LD_LIBRARY_PATH", ""),
               ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    # the child reports which library it loaded: the instrumented copy, not the in-tree build
    probe = subprocess.run([sys.executable, "-c", "import paper_2609_20734_amd._lib as L; print(L.LIB_PATH)"],
                           env=env, capture_output=True, text=True, timeout=300, cwd=str(tree))
    assert probe.returncode == 0, probe.stderr[-3000:]
    assert probe.stdout.strip() == str(tree / "paper_2609_20734_amd" / "liboda.so"), probe.stdout
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          str(tree / "tests" / "test_abi.py")],
                         env=env, capture_output=True, text=True, timeout=600, cwd=str(tree))
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out

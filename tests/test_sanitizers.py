"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

1. The C oracle (oracle/csrc/oracle.c), built with gcc and both sanitizers, runs
   tests/test_oracle_native.py (all but the planted-mistake builds, which compile their
   own copies): plan, ring, copies, binary16 conversions, OpenMP threads.
2. libhvdx's host code (every .hip source built with hipcc, the sanitizers applied to
   the host side only) runs tests/test_abi_host.py: the fusion plan, the ring
   partition, the broadcast layout and every argument check, through the C-ABI, with no
   GPU.
Each run is a child process with the sanitizer runtime preloaded; any report ends it
with an error.  A planted out-of-bounds write and a planted signed overflow, built the
same two ways, must be caught, so a silent harness cannot pass.
"""
import glob
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
CLANG = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang")
ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}
GCC_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
# host side only: each option after -Xarch_host, so no device code is instrumented
HIP_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
           "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g", "-O1"]


def runtime(compiler, name):
    try:
        out = subprocess.run([compiler, f"-print-file-name={name}"], capture_output=True, text=True, check=True)
    except (OSError, subprocess.CalledProcessError):
        return None
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def child(script, preload, timeout=900):
    env = dict(os.environ, LD_PRELOAD=preload, **ENV)
    return subprocess.run([sys.executable, "-c", script], cwd=ROOT, env=env, capture_output=True, text=True,
                          timeout=timeout)


def drive(pkg_dir, test_file, extra=()):
    """Child script: import from pkg_dir first, check that, run one test file."""
    return textwrap.dedent(f"""
        import sys
        sys.path[:0] = [{pkg_dir!r}, {ROOT!r}, {os.path.join(ROOT, 'tests')!r}]
        import pytest
        sys.exit(pytest.main(["-q", "-p", "no:cacheprovider", {test_file!r}, *{list(extra)!r}]))
    """)


@pytest.fixture(scope="module")
def gcc_asan():
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    lib = runtime("gcc", "libasan.so")
    if lib is None:
        pytest.skip("gcc's AddressSanitizer runtime not found")
    return lib


@pytest.fixture(scope="module")
def clang_asan():
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    lib = runtime(CLANG, "libclang_rt.asan-x86_64.so")
    if lib is None:
        pytest.skip("clang's AddressSanitizer runtime not found")
    return lib


PLANTED_C = """
#include <stdlib.h>
int planted_oob(int n) { int* a = (int*)malloc(sizeof(int) * n); a[n] = 1; int v = a[0]; free(a); return v; }
int planted_overflow(int x) { return x + 2147483647; }
"""


def planted_caught(lib_path, preload):
    for call in ("planted_oob(4)", "planted_overflow(5)"):
        script = f"import ctypes; L = ctypes.CDLL({lib_path!r}); print(L.{call})"
        r = child(script, preload, timeout=120)
        text = r.stdout + r.stderr
        if r.returncode == 0 or not ("AddressSanitizer" in text or "runtime error" in text):
            return f"{call} not caught (rc {r.returncode})"
    return None


def test_oracle_under_sanitizers(tmp_path, gcc_asan):
    pkg = tmp_path / "pkg"
    (pkg / "oracle").mkdir(parents=True)
    for f in glob.glob(os.path.join(ROOT, "oracle", "*.py")):
        shutil.copy(f, pkg / "oracle")
    lib = pkg / "oracle" / "liboracle.so"
    subprocess.run(["gcc", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", "-Wall",
                    "-Wextra", "-Werror", *GCC_SAN, "-o", str(lib), os.path.join(ROOT, "oracle", "csrc", "oracle.c")],
                   check=True)
    planted = tmp_path / "planted.c"
    planted.write_text(PLANTED_C)
    subprocess.run(["gcc", "-fPIC", "-shared", *GCC_SAN, "-o", str(tmp_path / "libplanted.so"), str(planted)],
                   check=True)
    assert planted_caught(str(tmp_path / "libplanted.so"), gcc_asan) is None

    check = f"import oracle.native as n; assert n.lib_path[0] == {str(lib)!r}, n.lib_path"
    script = drive(str(pkg), os.path.join(ROOT, "tests", "test_oracle_native.py"), ["-k", "not planted"])
    script = script.replace("import pytest", check + "\nimport pytest", 1)
    r = child(script, gcc_asan)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout


def test_library_host_code_under_sanitizers(tmp_path, clang_asan):
    pkg = tmp_path / "pkg" / "paper_1802_05799_amd"
    pkg.mkdir(parents=True)
    for f in glob.glob(os.path.join(ROOT, "paper_1802_05799_amd", "*.py")):
        shutil.copy(f, pkg)
    sys.path.insert(0, os.path.join(ROOT, "paper_1802_05799_amd"))
    try:
        import build as B  # the library's own flags
    finally:
        sys.path.pop(0)
    csrc = os.path.join(ROOT, "paper_1802_05799_amd", "csrc")
    flags = [f for f in B.HIP_FLAGS if f != "-O3"]
    subprocess.run([HIPCC, *flags, *HIP_SAN, "-I", os.path.join(ROOT, "include"), "-I", csrc, "-o",
                    str(pkg / "libhvdx.so"), *sorted(glob.glob(os.path.join(csrc, "*.hip")))], check=True,
                   capture_output=True)
    planted = tmp_path / "planted.hip"
    planted.write_text('extern "C" {\n' + PLANTED_C.replace("#include <stdlib.h>", "") + "}\n")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-fPIC", "-shared", "-include", "stdlib.h", *HIP_SAN, "-o",
                    str(tmp_path / "libplanted.so"), str(planted)], check=True, capture_output=True)
    assert planted_caught(str(tmp_path / "libplanted.so"), clang_asan) is None

    check = f"import paper_1802_05799_amd as hv; assert hv.LIB_PATH == {str(pkg / 'libhvdx.so')!r}, hv.LIB_PATH"
    script = drive(str(pkg.parent), os.path.join(ROOT, "tests", "test_abi_host.py"))
    script = script.replace("import pytest", check + "\nimport pytest", 1)
    r = child(script, clang_asan)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout

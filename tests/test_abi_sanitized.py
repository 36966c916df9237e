"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Every library source is compiled as usual for gfx950, with the sanitizers on
the host side only (each -fsanitize flag is applied to the host pass), and
linked into the C program tests/sanitize/abi_validation.c, which drives the
entry points through include/tls.h from C: pure host functions (version,
status strings, workspace sizing over a sweep of shapes and budgets, the
largest layouts the library takes) and calls that host validation must
reject before anything is enqueued.  No GPU is needed; leak detection is on.
A planted heap overflow, built and linked the same way, must be caught, so a
green run means the sanitizers were really active.
"""
import concurrent.futures
import glob
import importlib.util
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_07815_amd", "csrc")
DRIVER = os.path.join(ROOT, "tests", "sanitize", "abi_validation.c")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang"
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
C_SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")

pytestmark = pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                                reason="needs hipcc and ROCm's clang")


def _build_flags():
    spec = importlib.util.spec_from_file_location("tls_build", os.path.join(ROOT, "paper_2604_07815_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    flags = [f for f in mod.CFLAGS if f != "-O3"]
    return flags + ["-O1", "-g"] + HOST_SAN


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ... failed:\n{r.stderr[-4000:]}"
    return r


def _c_object(src, out):
    _run([CLANG, "-std=c11", "-O1", "-g", *C_SAN, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
          "-I", "/opt/rocm/include", "-c", src, "-o", out])


def _link(objs, exe):
    _run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
          "-fsanitize=undefined", "-o", exe, *objs])


@pytest.fixture(scope="module")
def library_objects(tmp_path_factory):
    d = tmp_path_factory.mktemp("asan_lib")
    flags = _build_flags()
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))

    def one(src):
        obj = str(d / (os.path.basename(src) + ".o"))
        _run([HIPCC, *flags, "-c", src, "-o", obj])
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        return list(ex.map(one, srcs))


def test_sanitizers_catch_a_planted_overflow(tmp_path):
    """The toolchain set-up itself: a one-past-the-end heap read must abort."""
    src = tmp_path / "planted.c"
    src.write_text("#include <stdlib.h>\n"
                   "int main(int argc, char** argv) {\n"
                   "  (void)argv; int* p = malloc(4 * sizeof(int));\n"
                   "  int v = p[argc + 3];\n"
                   "  free(p); return v == 12345;\n}\n")
    obj, exe = str(tmp_path / "planted.o"), str(tmp_path / "planted")
    _c_object(str(src), obj)
    _link([obj], exe)
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=60)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr


def test_abi_host_code_is_clean_under_asan_ubsan(library_objects, tmp_path):
    drv, exe = str(tmp_path / "abi_validation.o"), str(tmp_path / "abi_validation")
    _c_object(DRIVER, drv)
    _link([drv, *library_objects], exe)
    r = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=120)
    report = r.stdout + r.stderr
    assert "AddressSanitizer" not in report and "runtime error:" not in report and "LeakSanitizer" not in report, \
        report[-4000:]
    assert r.returncode == 0, report[-4000:]
    assert "all host-side checks passed" in r.stdout

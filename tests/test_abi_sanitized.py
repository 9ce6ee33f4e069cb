"""The C ABI shim under host AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU).

The library is rebuilt with the sanitizers on its host pass (build.py's
sanitize option; the GPU code is unchanged) and tests/test_abi.py runs
against it in a child process with the ASan runtime preloaded.  A second
child passes a partition table shorter than the P it declares, so the shim
reads past it: ASan must report that read, which shows the instrumentation
is live."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"

pytestmark = pytest.mark.slow


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    if not os.path.exists(CLANG):
        pytest.skip("ROCm clang not installed")
    rt = subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True).stdout.strip()
    if not os.path.exists(rt):
        pytest.skip("no ASan runtime")
    sys.path.insert(0, os.path.join(ROOT, "paper_2609_28053_amd"))
    import build as b
    lib = b.build(out=str(tmp_path_factory.mktemp("asan") / "libeqb_asan.so"), sanitize=True)
    env = dict(os.environ, EQB_LIB=lib, LD_PRELOAD=rt, PYTHONMALLOC="malloc",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return lib, env


def test_abi_checks_run_clean_under_asan_and_ubsan(sanitized):
    lib, env = sanitized
    res = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"), "-q",
                          "-p", "no:cacheprovider"], env=env, capture_output=True, text=True, cwd=ROOT,
                         timeout=300)
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    assert "Sanitizer" not in res.stdout + res.stderr


def test_sanitizer_reports_a_planted_overread(sanitized):
    lib, env = sanitized
    probe = textwrap.dedent("""
        import ctypes, os
        lib = ctypes.CDLL(os.environ["EQB_LIB"])
        V, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.eqb_route_topk.argtypes = [V, V, i64, i32, i32, V, V, V, V, i32, V, V, V]
        arr = (ctypes.c_int64 * 2)(0, 10)              # P + 1 = 2 entries ...
        fake = ctypes.c_void_p(0x10000)
        lib.eqb_route_topk(fake, fake, 10, 8, 2, fake, fake, fake, ctypes.cast(arr, V), 5, None, None, None)
    """)                                               # ... declared as P = 5
    res = subprocess.run([sys.executable, "-c", probe], env=env, capture_output=True, text=True, timeout=120)
    assert res.returncode != 0
    assert "AddressSanitizer: heap-buffer-overflow" in res.stderr
    assert "make_table" in res.stderr

"""The C ABI's host-side argument validation under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

The validation sources are built a second time with both sanitizers on their host pass
(`build.build_sanitized`), and every case of tests/test_abi.py then runs in a child
process against that library, with the sanitizer runtime preloaded and every report
fatal. A positive control first shows that the same set-up does stop a process on a
heap overflow in host code, so a clean run means something."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from paper_2608_06690_amd import build as B  # noqa: E402

# In the child: swap the binding's library for the sanitized one, keeping every
# declared argument and result type (test code only; the package loads its own
# library and nothing else).
PLUGIN = textwrap.dedent('''
    import ctypes, os

    def pytest_configure(config):
        from paper_2608_06690_amd import _native as N
        san = ctypes.CDLL(os.environ["PMPE_SAN_LIB"])
        n = 0
        for name, fp in list(N._lib.__dict__.items()):
            if isinstance(fp, ctypes._CFuncPtr):
                f = getattr(san, name)
                f.argtypes, f.restype = fp.argtypes, fp.restype
                n += 1
        assert n >= 20, n
        # the sanitizer runtime is in the process and the library calls into it
        ctypes.CDLL(None).__asan_report_load8
        N._lib = san
''')


def child_env(tmp_path):
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": B.sanitizer_runtime(),
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "PMPE_SAN_LIB": B.build_sanitized(),
        "PYTHONPATH": os.pathsep.join([str(tmp_path), ROOT, env.get("PYTHONPATH", "")]),
        "PYTHONDONTWRITEBYTECODE": "1",
    })
    return env


@pytest.fixture(scope="module")
def san_env(tmp_path_factory):
    tmp = tmp_path_factory.mktemp("san")
    (tmp / "pmpe_san_swap.py").write_text(PLUGIN)
    return tmp, child_env(tmp)


def test_sanitized_library_is_instrumented(san_env):
    lib = B.build_sanitized()
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms and "__ubsan_handle" in syms


def test_positive_control_heap_overflow_is_fatal(san_env):
    tmp, env = san_env
    src = tmp / "overflow.cpp"
    src.write_text(textwrap.dedent('''
        #include <cstdlib>
        extern "C" int read_past_end(int n) {
          int* a = (int*)std::malloc(n * sizeof(int));
          for (int i = 0; i < n; ++i) a[i] = i;
          volatile int v = a[n];  // one element past the allocation
          std::free(a);
          return v;
        }
    '''))
    so = tmp / "liboverflow.so"
    r = subprocess.run([B.hipcc(), "-shared", "-fPIC", "-g", "-Xarch_host", "-fsanitize=address",
                        "-shared-libasan", str(src), "-o", str(so)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    code = f"import ctypes; ctypes.CDLL({str(so)!r}).read_past_end(4); print('not caught')"
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "heap-buffer-overflow" in r.stderr, (r.returncode, r.stderr[-2000:])


def test_abi_error_cases_clean_under_sanitizers(san_env):
    tmp, env = san_env
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"), "-q", "-x",
           "-p", "pmpe_san_swap", "-p", "no:cacheprovider", "-m", "not gpu"]
    r = subprocess.run(cmd, env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in out and "failed" not in out
    # the child ran the ABI module's cases, not an empty selection
    n = int(out.split(" passed")[0].split()[-1])
    assert n >= 20, out[-2000:]

"""Host sanitizer runs, CPU only.

- The oracle, built by gcc with AddressSanitizer and UndefinedBehaviorSanitizer,
  runs its pin tests.
- The C-ABI library, its host code built with clang's ASan and UBSan (the device
  code is the ordinary gfx950 build), runs the host-side validation tests.

Each run is a child interpreter with the sanitizer runtime preloaded (the
interpreter itself is not instrumented), and any finding ends it with a
non-zero status.  A planted error in a scratch source, built with the same
flags, first checks that each toolchain reports at all."""
import os
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2204_05436_amd import build as B  # noqa: E402

SAN_ENV = {
    "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:exitcode=23",
    "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
}

# the child: point the oracle or the binding at the sanitized build, then run pytest
RUNNER = textwrap.dedent("""
    import sys
    sys.path.insert(0, %r)
    kind, lib, *tests = sys.argv[1:]
    if kind == "oracle":
        import oracle
        oracle.build = lambda *a, **k: lib
    else:
        from paper_2204_05436_amd import hotline
        hotline.LIB_PATH = lib
    import pytest
    # -s: a sanitizer report goes to the real stderr, not into pytest's capture
    sys.exit(pytest.main(["-q", "-s", "-p", "no:cacheprovider", "-m", "not gpu", *tests]))
""" % ROOT)

PLANTED_C = textwrap.dedent("""
    #include <limits.h>
    #include <stdlib.h>
    int heap_overflow(int n) { int* a = malloc(n * sizeof(int)); a[n] = 1; int r = a[0]; free(a); return r; }
    int add_one(int x) { return x + 1; }
""")
PLANTED_HIP = "extern \"C\" {\n" + PLANTED_C.replace("malloc(n", "(int*)malloc(n") + "}\n"


def _env(runtime):
    env = dict(os.environ, **SAN_ENV)
    env["LD_PRELOAD"] = " ".join(p for p in (runtime, os.environ.get("LD_PRELOAD", "")) if p)
    return env


def _child(code, args, runtime, timeout=600):
    r = subprocess.run([sys.executable, "-c", code, *args], cwd=ROOT, env=_env(runtime),
                       capture_output=True, text=True, timeout=timeout)
    return r.returncode, r.stdout + r.stderr


def _clean(rc, out):
    assert rc == 0, out[-6000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]


def _planted(lib, runtime):
    call = "import ctypes, sys; getattr(ctypes.CDLL(sys.argv[1]), sys.argv[2])(int(sys.argv[3]))"
    rc, out = _child(call, [lib, "heap_overflow", "4"], runtime, 120)
    assert rc != 0 and "heap-buffer-overflow" in out, out[-3000:]
    rc, out = _child(call, [lib, "add_one", str(2**31 - 1)], runtime, 120)
    assert rc != 0 and "signed integer overflow" in out, out[-3000:]


@pytest.fixture(scope="module")
def gcc_asan():
    r = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path):
        pytest.fail("gcc's libasan not found")
    return path


def test_gcc_sanitizers_report_a_planted_error(tmp_path, gcc_asan):
    src = tmp_path / "planted.c"
    src.write_text(PLANTED_C)
    lib = str(tmp_path / "libplanted.so")
    subprocess.check_call(["gcc", "-O1", *oracle.SAN_FLAGS, "-shared", "-fPIC", str(src), "-o", lib])
    _planted(lib, gcc_asan)


def test_oracle_pins_under_asan_ubsan(tmp_path, gcc_asan):
    lib = oracle.build(out=str(tmp_path / "liboracle_san.so"), sanitize=True)
    _clean(*_child(RUNNER, ["oracle", lib, "tests/test_oracle_pins.py"], gcc_asan))


def test_hipcc_host_sanitizers_report_a_planted_error(tmp_path):
    src = tmp_path / "planted.hip"
    src.write_text(PLANTED_HIP)
    obj, lib = str(tmp_path / "planted.o"), str(tmp_path / "libplanted.so")
    subprocess.check_call([B.HIPCC, *B.FLAGS, "-O1", *B.SAN_FLAGS, "-c", str(src), "-o", obj],
                          stderr=subprocess.DEVNULL)
    subprocess.check_call([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", obj, "-o", lib,
                           *B.SAN_LINK], stderr=subprocess.DEVNULL)
    _planted(lib, B.host_san_runtime())


@pytest.mark.slow
def test_library_host_validation_under_asan_ubsan(tmp_path):
    lib = B.build(verbose=False, out=str(tmp_path / "libhotline_san.so"), host_sanitize=True,
                  build_dir=str(tmp_path))
    _clean(*_child(RUNNER, ["hotline", lib, "tests/test_abi.py"], B.host_san_runtime()))

r"""Build libhotline.so (HIP, gfx950) in-tree: one hipcc compile per source, in
parallel, then a shared-library link.  Usage: python -m paper_2204_05436_amd.build

``python -m paper_2204_05436_amd.build --host-sanitize OUT.so`` builds a copy
whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer checks
(the device code is the ordinary gfx950 build).  It links against the shared
clang sanitizer runtime, which a process that loads it must preload
(``LD_PRELOAD`` set to the path ``host_san_runtime()`` returns), with
``ASAN_OPTIONS=detect_leaks=0`` since the interpreter around it is not
instrumented.  ROCm's ASan runtime also intercepts the HSA device-memory
allocator for device-side checking, which needs XNACK; where that is off its
first device allocation fails, so such a copy serves host-only runs.
``--sanitizers undefined`` builds a UBSan-only copy (its runtime intercepts
no allocator), which runs on a GPU as well; the GPU tests against it:

    python -m paper_2204_05436_amd.build --host-sanitize /tmp/libhl_ubsan.so --sanitizers undefined
    HOTLINE_LIB=/tmp/libhl_ubsan.so UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 \
    LD_PRELOAD=$(hipcc -print-file-name=libclang_rt.ubsan_standalone-x86_64.so) \
    python -m pytest tests -m gpu -x -s

UBSan's ``function`` check is always left out: it puts type data at the entry
of every host function whose address is taken, the kernels' host-side launch
handles included, and with it on the launches went through without an error
while no kernel wrote anything.  ``vptr`` is left out with it (the host code
has no polymorphic classes)."""
from __future__ import annotations

import argparse
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libhotline.so")
BUILD = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument",
]


def san_flags(sanitizers: str = "address,undefined"):
    """(compile flags, link flags) of a host-sanitized build: every -fsanitize=
    applies to the host pass alone."""
    cc = ["-Xarch_host", "-g", "-Xarch_host", "-fno-omit-frame-pointer"]
    ld = []
    for s in sanitizers.split(","):
        cc += ["-Xarch_host", "-fsanitize=" + s]
        ld += ["-Xarch_host", "-fsanitize=" + s]
    cc += ["-Xarch_host", "-fno-sanitize=function,vptr", "-Xarch_host", "-fno-sanitize-recover=undefined"]
    return cc, ld + ["-shared-libsan"]


SAN_FLAGS, SAN_LINK = san_flags()


def host_san_runtime(sanitizers: str = "address,undefined") -> str:
    """The shared clang sanitizer runtime that a process loading a host-sanitized
    build preloads: ASan's (which carries the UBSan handlers too) when ASan is on,
    else the standalone UBSan one."""
    name = "asan" if "address" in sanitizers.split(",") else "ubsan_standalone"
    r = subprocess.run([HIPCC, f"-print-file-name=libclang_rt.{name}-x86_64.so"],
                       capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError(f"clang {name} runtime not found: " + r.stdout + r.stderr)
    return path


def _compile(src: str, build_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if "warning" in err:
        sys.stderr.write(err + "\n")
    return obj


def build(verbose: bool = True, out: str = OUT, host_sanitize: bool = False,
          build_dir: str | None = None, sanitizers: str = "address,undefined") -> str:
    if build_dir is None:
        build_dir = BUILD if not host_sanitize else os.path.join(BUILD, "san")
    os.makedirs(build_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    cc, ld = san_flags(sanitizers) if host_sanitize else ((), ())
    extra = cc
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, build_dir, extra), srcs))
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp,
           *ld]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--host-sanitize", metavar="OUT", default=None,
                    help="build a host-sanitized copy of the library at OUT instead")
    ap.add_argument("--sanitizers", default="address,undefined",
                    help="the -fsanitize= list of --host-sanitize (default address,undefined)")
    a = ap.parse_args()
    if a.host_sanitize:
        build(out=os.path.abspath(a.host_sanitize), host_sanitize=True, sanitizers=a.sanitizers)
    else:
        build()

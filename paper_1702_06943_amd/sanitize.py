"""Host AddressSanitizer + UndefinedBehaviorSanitizer build of libtoc.so and a run
of the host-side tests against it (CPU only; the device code is built without
sanitizers).

Usage: python -m paper_1702_06943_amd.sanitize [pytest args...]
Builds _build/asan/libtoc.so with every host translation unit under
-fsanitize=address,undefined (hipcc: after -Xarch_host; the C++ host sources with
the same clang, so one sanitizer runtime serves all), then runs the encoder, image
layout and physical-encoding tests with that library (TOC_LIB_PATH) and the
clang ASan runtime preloaded.  Exits with pytest's status.
"""

import glob
import os
import subprocess
import sys

from . import build as B

ASAN_DIR = os.path.join(B.BUILD, "asan")
ASAN_LIB = os.path.join(ASAN_DIR, "libtoc.so")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined"]
TESTS = ["tests/test_encode_abi.py", "tests/test_layout.py", "tests/test_phys.py",
         "tests/test_ingest_host.py"]


def runtime():
    libs = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not libs:
        raise RuntimeError("clang ASan runtime not found under /opt/rocm/llvm")
    return libs[-1]


def build_asan(verbose=False):
    os.makedirs(ASAN_DIR, exist_ok=True)
    clang = "/opt/rocm/llvm/bin/clang++"
    objs = []
    for src in B.HOST_SOURCES:
        o = os.path.join(ASAN_DIR, src.replace(".cpp", ".o"))
        B._run([clang, "-O1", "-g", "-fno-omit-frame-pointer", "-std=c++17", "-fPIC", *SAN,
                "-I", B.INCLUDE, "-c", os.path.join(B.CSRC, src), "-o", o], verbose)
        objs.append(o)
    host_san = [x for f in SAN for x in ("-Xarch_host", f)]
    for src in B.HIP_SOURCES:
        o = os.path.join(ASAN_DIR, src.replace(".hip", ".o"))
        B._run([B.HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", f"--offload-arch={B.ARCH}",
                *B.NO_PACKED_FP32, *host_san, "-I", B.INCLUDE, "-c", os.path.join(B.CSRC, src),
                "-o", o], verbose)
        objs.append(o)
    B._run([B.HIPCC, "-shared", "-fPIC", f"--offload-arch={B.ARCH}", "-Xarch_host",
            "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-shared-libsan", *objs,
            "-o", ASAN_LIB, "-lpthread"], verbose)
    return ASAN_LIB


def main(argv):
    build_asan()
    env = dict(os.environ)
    env["TOC_LIB_PATH"] = ASAN_LIB
    env["LD_PRELOAD"] = runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:detect_odr_violation=0:verify_asan_link_order=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        *TESTS, *argv], cwd=B.ROOT, env=env)
    return r.returncode


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))

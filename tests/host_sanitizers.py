"""Run the C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only; no GPU call is made).

Builds a copy of the library whose host code is instrumented (the device code
is built as usual; the sanitizer flags apply to the host side only), then runs
tests/test_abi.py against it with the ASan runtime preloaded.  Exits with the
test run's status.  Usage: python -m tests.host_sanitizers [out_dir]
"""
from __future__ import annotations

import concurrent.futures
import os
import shlex
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2609_25537_amd import build  # noqa: E402

SAN = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined"


def main() -> int:
    out = sys.argv[1] if len(sys.argv) > 1 else tempfile.mkdtemp(prefix="cmc_san_")
    os.makedirs(out, exist_ok=True)
    flags = build.FLAGS + ["-g", "-fno-omit-frame-pointer"] + shlex.split(SAN)

    def compile_one(src):
        obj = os.path.join(out, src.replace(".hip", ".o"))
        subprocess.run([build.HIPCC, *flags, "-c", os.path.join(build.CSRC, src), "-o", obj], check=True)
        return obj

    with concurrent.futures.ThreadPoolExecutor(6) as ex:
        objs = list(ex.map(compile_one, build.SOURCES))
    lib = os.path.join(out, "libcmc_san.so")
    subprocess.run([build.HIPCC, f"--offload-arch={build.ARCH}", "-shared", "-fPIC", *shlex.split(SAN), "-o", lib,
                    *objs], check=True)
    clang = os.path.join(os.path.dirname(build.HIPCC), "..", "llvm", "bin", "clang")
    rt = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True, check=True).stdout.strip()
    env = dict(os.environ, LD_PRELOAD=rt, CMC_LIBRARY=lib, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"), "-q", "-x",
                        "-p", "no:cacheprovider"], env=env, cwd=ROOT)
    return r.returncode


if __name__ == "__main__":
    sys.exit(main())

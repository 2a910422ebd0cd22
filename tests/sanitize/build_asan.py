"""Builds libmkor with AddressSanitizer and UndefinedBehaviorSanitizer on
its host code (the device code is built as usual), for the host-side ABI
tests: tests/test_sanitized_host.py runs tests/test_abi_host.py against it
with clang's ASan runtime preloaded.  CPU only.

    python tests/sanitize/build_asan.py     -> tests/sanitize/_build/libmkor_asan.so
"""
import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
from paper_2306_01685_amd import build as B  # noqa: E402

OUT = os.path.join(HERE, "_build")
LIB = os.path.join(OUT, "libmkor_asan.so")
# each sanitizer flag applies to the host compilation only
SAN = ("-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined "
       "-Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer -Xarch_host -g").split()


def asan_runtime() -> str:
    """clang's shared ASan runtime (it carries the UBSan handlers too)."""
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang ASan runtime not found under /opt/rocm/llvm")
    return hits[-1]


def _compile(src):
    obj = os.path.join(OUT, os.path.basename(src) + ".o")
    cmd = [B.HIPCC, *B.COMMON_FLAGS, *B.DEVICE_FLAGS, *SAN, "-c", src, "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd)}\n{r.stderr[-4000:]}")
    return obj


def build() -> str:
    os.makedirs(OUT, exist_ok=True)
    with ThreadPoolExecutor(max_workers=8) as ex:
        objs = list(ex.map(_compile, B.sources()))
    # the runtime is preloaded into the process, so the library leaves the
    # sanitizer symbols for the dynamic linker to resolve
    cmd = [B.HIPCC, "-shared", "-fPIC", f"--offload-arch={B.ARCH}", *objs, *B.LINK_FLAGS, "-o", LIB + ".tmp"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd)}\n{r.stderr[-4000:]}")
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build())

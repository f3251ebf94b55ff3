"""Build the HIP encoder-stage library (gfx950) in-tree.

Compiles every ``csrc/*.hip`` with hipcc for gfx950 (and the host-only
``csrc/*.cpp``) and links them into
``paper_2202_11836_amd/libskystage.so``.  Always recompiles (the caller asks
for a fresh build); sources compile in parallel.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD_DIR = os.path.join(PKG, "_build")
LIB_NAME = "libskystage.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# -packed-fp32-ops: keep the compiler from emitting packed fp32 VALU ops.
COMMON_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def _sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                  if f.endswith(".hip") or f.endswith(".cpp"))


def _compile(src: str) -> str:
    base, ext = os.path.splitext(os.path.basename(src))
    obj = os.path.join(BUILD_DIR, base + ext.replace(".", "_") + ".o")
    if ext == ".cpp":  # host-only code
        cmd = [HIPCC, "-O3", "-std=c++17", "-fPIC", "-c", src, "-o", obj]
    else:
        cmd = [HIPCC] + COMMON_FLAGS + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    if shutil.which(HIPCC) is None and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found ({HIPCC})")
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = _sources()
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH} from {len(srcs)} sources", file=sys.stderr)
    return LIB_PATH


# Host code with AddressSanitizer and UndefinedBehaviorSanitizer (device
# code unchanged): each sanitizer flag applies to the host compilation only.
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_DIR = os.path.join(BUILD_DIR, "sanitized")
SAN_LIB = os.path.join(SAN_DIR, "libskystage_sanitized.so")


def _hash_sources() -> str:
    import hashlib
    hsh = hashlib.sha256()
    for src in _sources() + [os.path.join(os.path.dirname(PKG), "include", f)
                             for f in sorted(os.listdir(os.path.join(os.path.dirname(PKG), "include")))]:
        hsh.update(src.encode())
        hsh.update(open(src, "rb").read())
    for f in sorted(os.listdir(CSRC)):
        if f.endswith(".h"):
            hsh.update(open(os.path.join(CSRC, f), "rb").read())
    return hsh.hexdigest()


def sanitizer_runtime() -> str:
    """The AddressSanitizer runtime of the compiler hipcc drives (the
    process that loads the sanitized library must preload it)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "lib", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/lib/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        rd = subprocess.run([clang, "--print-runtime-dir"], capture_output=True, text=True).stdout.strip()
        path = os.path.join(rd, "libclang_rt.asan-x86_64.so")
    if not os.path.exists(path):
        raise RuntimeError("AddressSanitizer runtime not found")
    return path


def build_sanitized() -> str:
    """Build libskystage_sanitized.so (host code under ASan + UBSan) into
    _build/sanitized; reused while the sources are unchanged."""
    os.makedirs(SAN_DIR, exist_ok=True)
    stamp = os.path.join(SAN_DIR, "sources.sha256")
    digest = _hash_sources()
    if os.path.exists(SAN_LIB) and os.path.exists(stamp) and open(stamp).read() == digest:
        return SAN_LIB

    def comp(src):
        base, ext = os.path.splitext(os.path.basename(src))
        obj = os.path.join(SAN_DIR, base + ext.replace(".", "_") + ".o")
        if ext == ".cpp":
            cmd = [HIPCC, "-O1", "-g", "-std=c++17", "-fPIC"] + SAN_HOST + ["-c", src, "-o", obj]
        else:
            cmd = [HIPCC] + COMMON_FLAGS[:1] + ["-O1", "-g"] + COMMON_FLAGS[2:] + SAN_HOST + [
                "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"sanitized build failed for {src}:\n{r.stderr}")
        return obj

    srcs = _sources()
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(comp, srcs))
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC"] + SAN_HOST + ["-o", SAN_LIB] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stderr}")
    with open(stamp, "w") as fh:
        fh.write(digest)
    return SAN_LIB


if __name__ == "__main__":
    build(verbose=True)

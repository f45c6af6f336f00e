"""Build libdsattn.so in-tree with hipcc for gfx950.

    python -m paper_2606_16317_amd.build            # build (always recompiles)
    python -m paper_2606_16317_amd.build --asm DIR  # also keep the gfx950 assembly in DIR
    python -m paper_2606_16317_amd.build --sanitize # host-sanitizer build, libdsattn_san.so

The sanitizer build instruments the host code (argument checks, threshold mapping, token
order, launch wrappers) with AddressSanitizer and UndefinedBehaviorSanitizer; the GPU code
is compiled exactly as in the normal build.  It links the shared clang sanitizer runtime,
so a process that loads it must have that runtime loaded first (a program built with
``-fsanitize=address -shared-libsan``, or ``LD_PRELOAD`` of ``asan_runtime()``).
"""

from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_NAME = "libdsattn.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
SAN_LIB_PATH = os.path.join(PKG_DIR, "libdsattn_san.so")
ARCH = "gfx950"

SOURCES = ["fa_fwd_kernel.hip", "reorder_kernel.hip", "quant_kernel.hip", "dsattn_api.cpp"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def compile_flags() -> list:
    return [
        f"--offload-arch={ARCH}",
        "-O3",
        "-std=c++17",
        "-fPIC",
        # packed fp32 VALU forms stay off: plain scalar fp32 code only
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall",
        f"-I{INCLUDE}",
        f"-I{CSRC}",
    ]


def sanitize_flags() -> list:
    """Host-only AddressSanitizer + UndefinedBehaviorSanitizer (every -fsanitize= is
    preceded by -Xarch_host, so no GPU code is instrumented)."""
    flags = []
    for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=undefined",
              "-fno-omit-frame-pointer", "-shared-libsan", "-g"):
        flags += ["-Xarch_host", f]
    return flags


def asan_runtime() -> str:
    """Path of the shared clang AddressSanitizer runtime the sanitizer build links."""
    out = subprocess.run([os.path.join(os.path.dirname(hipcc()), "..", "llvm", "bin", "clang"),
                          "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True, check=True).stdout.strip()
    return os.path.realpath(out)


def build(verbose: bool = False, asm_dir: str | None = None, sanitize: bool = False) -> str:
    """Compile every source into LIB_PATH, or SAN_LIB_PATH with sanitize=True (always
    recompiles); return the path."""
    cc = hipcc()
    out_path = SAN_LIB_PATH if sanitize else LIB_PATH
    tmp = out_path + ".tmp"
    cmd = [cc, *compile_flags(), *(sanitize_flags() if sanitize else []), "-shared", "-o", tmp]
    for src in SOURCES:
        path = os.path.join(CSRC, src)
        if src.endswith(".cpp"):
            cmd += ["-x", "hip", path]
        else:
            cmd.append(path)
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out_path)
    if asm_dir:
        os.makedirs(asm_dir, exist_ok=True)
        src = os.path.join(CSRC, "fa_fwd_kernel.hip")
        out = os.path.join(asm_dir, "fa_fwd_kernel.s")
        subprocess.run([cc, *compile_flags(), "--cuda-device-only", "-S", src, "-o", out],
                       check=True)
    return out_path


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--asm", default=None, help="also write gfx950 assembly into this dir")
    ap.add_argument("--sanitize", action="store_true",
                    help="host-sanitizer build (libdsattn_san.so) instead of the normal one")
    ap.add_argument("-v", "--verbose", action="store_true")
    args = ap.parse_args(argv)
    path = build(verbose=args.verbose, asm_dir=args.asm, sanitize=args.sanitize)
    print(path)


if __name__ == "__main__":
    sys.exit(main())

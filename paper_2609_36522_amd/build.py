"""Build libparaanya.so (gfx950) in-tree with hipcc.

    python -m paper_2609_36522_amd.build [--sanitized]

Compiles the HIP kernels and the host library into one shared object next to this
file. Packed-fp32 VALU instructions are disabled for every device compilation. With
--sanitized it also builds the host-sanitized copy and the ABI driver the tests run.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libparaanya.so")

SOURCES = ["paraanya.cpp", "paraanya_parareal.cpp", "host_common.cpp", "k_solver.hip", "k_epsnet.hip", "k_parareal.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def command(out: str = LIB) -> list:
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-x", "hip", "-Wall", "-Wshadow", "-Werror=shadow", "-fvisibility=hidden", "-Wno-unused-command-line-argument",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC, *srcs, "-o", out]


# Host-sanitized copy of the library (AddressSanitizer + UndefinedBehaviorSanitizer on the host
# code only; every sanitizer flag is scoped to the host compilation, the device code is built as
# for the library) and the C driver that exercises its ABI (tests/sanitize/abi_driver.cpp).
SAN_DIR = os.path.join(ROOT, "tests", "sanitize", "_build")
SAN_LIB = os.path.join(SAN_DIR, "libparaanya_san.so")
SAN_DRIVER = os.path.join(SAN_DIR, "abi_driver")
SAN_DRIVER_SRC = os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp")
_HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def sanitized_commands() -> tuple:
    """(library command, driver command) of the host-sanitized build."""
    lib = command(SAN_LIB + ".tmp")
    lib = lib[:-2] + ["-g", *_HOST_SAN] + lib[-2:]
    drv = [hipcc(), "-O1", "-g", "-std=c++17", *_HOST_SAN, "-I", INCLUDE, SAN_DRIVER_SRC,
           "-L", SAN_DIR, "-lparaanya_san", f"-Wl,-rpath,{SAN_DIR}", "-o", SAN_DRIVER + ".tmp"]
    return lib, drv


def _finish(r, what: str, verbose: bool) -> None:
    out, err = r.communicate() if hasattr(r, "communicate") else (r.stdout, r.stderr)
    msgs = "\n".join(line for line in ((out or "") + (err or "")).splitlines()
                     if "packed-fp32-ops" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"{what}: hipcc failed ({r.returncode}):\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, flush=True)


def build(verbose: bool = False, sanitized: bool = False) -> str:
    """Compile every source and atomically replace the library. Returns its path.

    sanitized: also build the host-sanitized library and its ABI driver (the two library
    builds run side by side)."""
    tmp = LIB + ".tmp"
    cmd = command(tmp)
    procs = [(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True), "library", cmd)]
    if sanitized:
        os.makedirs(SAN_DIR, exist_ok=True)
        lib_cmd, _ = sanitized_commands()
        procs.append((subprocess.Popen(lib_cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True),
                      "sanitized library", lib_cmd))
    for p, what, c in procs:
        if verbose:
            print(" ".join(c), flush=True)
        _finish(p, what, verbose)
    os.replace(tmp, LIB)
    if sanitized:
        os.replace(SAN_LIB + ".tmp", SAN_LIB)
        _, drv_cmd = sanitized_commands()
        if verbose:
            print(" ".join(drv_cmd), flush=True)
        _finish(subprocess.run(drv_cmd, capture_output=True, text=True), "sanitizer driver", verbose)
        os.replace(SAN_DRIVER + ".tmp", SAN_DRIVER)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv, sanitized="--sanitized" in sys.argv))

"""Host-sanitized build of the C ABI's host code, for the CPU tests.

The host side of ee_abi.cpp (argument validation, workspace layout, launch
sequencing) is compiled with AddressSanitizer and UndefinedBehaviorSanitizer
(device code is not instrumented) and linked with the kernel objects of the
normal build into a library that tests/test_hostcheck.py loads in a process
that preloads the ASan runtime.  Nothing here runs on a GPU.
"""

import glob
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2402_00518_amd")
BUILD = os.path.join(PKG, "_build")
ROCM = "/opt/rocm"


def asan_runtime():
    """The clang ASan runtime that matches the ROCm compiler, or None."""
    hits = sorted(glob.glob(os.path.join(ROCM, "llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")))
    return hits[-1] if hits else None


def kernel_objects():
    objs = [os.path.join(BUILD, f) for f in ("kernels.hip.o", "optim.hip.o", "decode.hip.o")]
    return objs if all(os.path.exists(o) for o in objs) else None


def build(out_dir: str) -> str:
    """Compile and link the sanitized library into out_dir; returns its path."""
    from paper_2402_00518_amd.build import ARCH, hipcc

    obj = os.path.join(out_dir, "ee_abi_checked.o")
    lib = os.path.join(out_dir, "libeetune_checked.so")
    compile_cmd = [
        hipcc(), "-x", "hip", f"--offload-arch={ARCH}", "-O1", "-g", "-std=c++17", "-fPIC",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", os.path.join(ROOT, "include"),
        "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
        "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
        "-c", os.path.join(PKG, "csrc", "ee_abi.cpp"), "-o", obj,
    ]
    link_cmd = [
        os.path.join(ROCM, "llvm/bin/clang++"), "-shared", "-fPIC", "-fsanitize=address,undefined",
        "-shared-libasan", "-o", lib, obj, *kernel_objects(),
        "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}",
    ]
    for cmd in (compile_cmd, link_cmd):
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"host-checked build failed: {' '.join(cmd)}\n{r.stderr}")
    return lib

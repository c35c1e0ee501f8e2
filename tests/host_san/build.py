"""Host-sanitized build of the library for the CPU-side boundary checks.

The units with the boundary's host logic (agn_api.hip: argument checks,
context set-up and tear-down, the host bookkeeping of the commit order;
init.cpp: the initial parameters) are compiled with AddressSanitizer and
UndefinedBehaviorSanitizer on their host code (device code is built as
usual), and linked with the kernel units of the regular in-tree build into
libagn_san.so.  abi_host_checks.cpp is compiled the same way and linked
against it.  Used by tests/test_host_sanitizers.py; nothing here runs on a
GPU.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_1710_02368_amd", "csrc")
OBJS = os.path.join(ROOT, "paper_1710_02368_amd", "_build")
ROCM = "/opt/rocm"
CLANG = os.path.join(ROCM, "llvm", "bin", "clang++")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer"]
HOST_UNITS = ("agn_api.hip", "init.cpp")


def asan_runtime_dir():
    base = os.path.join(ROCM, "llvm", "lib", "clang")
    for v in sorted(os.listdir(base), reverse=True):
        d = os.path.join(base, v, "lib", "linux")
        if os.path.exists(os.path.join(d, "libclang_rt.asan-x86_64.so")):
            return d
    raise RuntimeError("no AddressSanitizer runtime under " + base)


def run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(" ".join(cmd) + "\n" + r.stdout + r.stderr)


def build(out_dir):
    """Build libagn_san.so and the checks program in out_dir; returns the
    program's path."""
    kernel_objs = [os.path.join(OBJS, f) for f in sorted(os.listdir(OBJS))
                   if f.endswith(".o") and f[:-2] not in HOST_UNITS]
    objs = []
    for unit in HOST_UNITS:
        obj = os.path.join(out_dir, unit + ".o")
        lang = ["-x", "hip"] if unit.endswith(".cpp") else []
        run([HIPCC, "-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Xclang", "-target-feature",
             "-Xclang", "-packed-fp32-ops", *SAN_HOST, "-I", os.path.join(ROOT, "include"), "-I", CSRC, *lang,
             "-c", os.path.join(CSRC, unit), "-o", obj])
        objs.append(obj)
    rt = asan_runtime_dir()
    lib = os.path.join(out_dir, "libagn_san.so")
    san = ["-fsanitize=address,undefined", "-shared-libasan"]
    run([CLANG, "-shared", "-fPIC", *san, *objs, *kernel_objs, "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
         "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", lib])
    exe = os.path.join(out_dir, "abi_host_checks")
    run([CLANG, "-g", "-O1", "-std=c++17", "-fno-omit-frame-pointer", *san, "-I", os.path.join(ROOT, "include"),
         os.path.join(HERE, "abi_host_checks.cpp"), "-L", out_dir, "-lagn_san", "-Wl,-rpath," + out_dir,
         "-Wl,-rpath," + rt, "-o", exe])
    return exe

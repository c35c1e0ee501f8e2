"""Build the plain C99 test program agn_c_round.c against include/agn.h and
the in-tree libagn.so (gcc; the HIP runtime's C API for device buffers).
Warnings are errors for the program and the library header; the ROCm headers
are system headers."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PKG = os.path.join(ROOT, "paper_1710_02368_amd")
ROCM = "/opt/rocm"


def build(out_dir):
    exe = os.path.join(out_dir, "agn_c_round")
    cmd = ["gcc", "-std=c99", "-O1", "-Wall", "-Wextra", "-pedantic", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-isystem", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           os.path.join(HERE, "agn_c_round.c"), "-L", PKG, "-lagn", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath," + PKG, "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(" ".join(cmd) + "\n" + r.stdout + r.stderr)
    return exe

"""Code size (.text bytes) of each kernel instantiation of one source file.

Compiles the file for gfx950 to device assembly, assembles it, and lists the
size of every kernel symbol, e.g. the K-loop unroll variants of the GEMM
(template argument 3 of ``gemm_kernel``).  Runs on the build machine (no
GPU).  Usage::

    python -m paper_2608_13757_amd.code_size kern_gemm.hip
"""
import os
import re
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = "/opt/rocm"


def sizes(src):
    path = os.path.join(HERE, "csrc", src)
    with tempfile.TemporaryDirectory() as d:
        asm, obj = os.path.join(d, "k.s"), os.path.join(d, "k.o")
        subprocess.check_call([f"{ROCM}/bin/hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang",
                               "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(HERE, "csrc"),
                               "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S", "-x", "hip", path,
                               "-o", asm], stderr=subprocess.DEVNULL)
        subprocess.check_call([f"{ROCM}/llvm/bin/llvm-mc", "-triple", "amdgcn-amd-amdhsa", "-mcpu=gfx950",
                               "-filetype=obj", asm, "-o", obj])
        out = subprocess.check_output([f"{ROCM}/llvm/bin/llvm-readelf", "-s", "--wide", obj], text=True)
    res = {}
    for line in out.splitlines():
        f = line.split()
        if len(f) >= 8 and f[3] == "FUNC":
            name = f[7]
            m = re.search(r"(\w+?_kernel)I(.*)EEvN", name)
            if m:
                args = ", ".join(v if t == "i" else ("true" if v == "1" else "false")
                                 for t, v in re.findall(r"L([ib])(\d+)E", m.group(2) + "E"))
                res[(m.group(1).split("N_1")[-1].lstrip("0123456789"), args)] = int(f[2])
    return res


def main():
    src = sys.argv[1] if len(sys.argv) > 1 else "kern_gemm.hip"
    for (k, args), n in sorted(sizes(src).items()):
        print(f"{k}<{args}> {n}")


if __name__ == "__main__":
    main()

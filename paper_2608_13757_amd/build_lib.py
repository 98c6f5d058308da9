"""Build libbfs.so (hipcc, gfx950) in-tree."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libbfs.so")
SOURCES = ["plan.cpp", "runtime.hip", "kern_interp.hip", "kern_stream3.hip", "kern_gemm.hip", "kern_attn.hip", "kern_moe.hip",
           "kern_rms.hip", "kern_adamw.hip", "kern_chain.hip"]
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-parameter", "-Wno-unused-result"]


def build(verbose: bool = False) -> str:
    objs = []
    bdir = os.path.join(HERE, "_build")
    os.makedirs(bdir, exist_ok=True)
    procs = []
    for src in SOURCES:
        obj = os.path.join(bdir, src + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else ["-x", "hip"]
        cmd = ["/opt/rocm/bin/hipcc", *FLAGS[:-3], "-c", *lang, os.path.join(CSRC, src), "-o", obj,
               "-Wall", "-Wno-unused-parameter"]
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        objs.append(obj)
    failed = False
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode()
        lines = [l for l in text.splitlines() if "packed-fp32-ops" not in l]
        if p.returncode != 0 or verbose:
            sys.stderr.write("\n".join(lines) + "\n")
        failed |= p.returncode != 0
    if failed:
        raise RuntimeError("libbfs build failed")
    tmp = OUT + ".tmp"
    subprocess.check_call(["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

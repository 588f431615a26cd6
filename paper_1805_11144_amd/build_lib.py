"""Build libmergesim.so in-tree: host C++ with g++, the HIP runtime and kernels
with hipcc for gfx950, linked by hipcc.  Always rebuilds (a few seconds)."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "libmergesim.so")
BUILD = os.path.join(HERE, "_build")

HOST_SOURCES = ["build.cpp", "ir.cpp", "planner.cpp", "launch_plan.cpp", "plan_json.cpp", "abi_host.cpp"]
HIP_SOURCES = ["runtime.hip"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")

HOST_FLAGS = ["-std=c++17", "-O3", "-fPIC", "-mavx2", "-mfma", "-Wall", "-Wextra",
              "-I" + INCLUDE]
HIP_FLAGS = ["-std=c++17", "-O3", "-fPIC", "--offload-arch=gfx950", "-I" + INCLUDE,
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout)
        raise RuntimeError(f"build step failed: {cmd[0]} {cmd[-1]}")
    return r.stdout


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    procs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        procs.append((["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj], obj))
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        procs.append(([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj], obj))
    running = [(subprocess.Popen(c, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True), c, o)
               for c, o in procs]
    failed = []
    for p, c, o in running:
        out, _ = p.communicate()
        if p.returncode != 0:
            failed.append(" ".join(c) + "\n" + out)
        elif verbose and out.strip():
            print(out)
        objs.append(o)
    if failed:
        sys.stderr.write("\n".join(failed))
        raise RuntimeError("libmergesim build failed")
    tmp = OUT + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp, "-lpthread"])
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))

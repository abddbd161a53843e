"""Builds the host-only executor test library: the library's C ABI, planner,
cost model and executor sources compiled with g++ against the queue
simulator in this directory instead of the HIP runtime (test infrastructure)."""
import fcntl
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2609_06172_amd", "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("capi.cpp", "planner.cpp", "cost.cpp", "executor.cpp")] + \
          [os.path.join(HERE, "hip_sim.cpp")]
OUT = os.path.join(HERE, "_build", "libautouvm_sim.so")


def build():
    """Compile if any source or header is newer than the library; returns its path."""
    deps = SOURCES + glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(ROOT, "include", "*.h")) + \
        glob.glob(os.path.join(HERE, "hip", "*.h"))
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    # one build at a time (parallel test workers share the output)
    with open(OUT + ".lock", "w") as lock:
        fcntl.flock(lock, fcntl.LOCK_EX)
        if os.path.exists(OUT) and os.path.getmtime(OUT) >= max(os.path.getmtime(d) for d in deps):
            return OUT
        tmp = f"{OUT}.{os.getpid()}.tmp"
        cmd = ["g++", "-O1", "-g", "-fPIC", "-shared", "-std=c++17", "-Wall", "-Wno-unused-function",
               "-I" + HERE, "-I" + os.path.join(ROOT, "include"), "-I" + CSRC] + SOURCES + ["-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build())

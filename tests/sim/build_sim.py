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
# the same sources with AddressSanitizer and UndefinedBehaviorSanitizer (host
# code only: nothing here is GPU code); load it into a process that preloads
# the ASan runtime (see sanitizer_env)
OUT_SAN = os.path.join(HERE, "_build", "libautouvm_sim_asan.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def sanitizer_env():
    """Environment for a child process that loads the sanitized library."""
    rt = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    cxx = subprocess.run(["g++", "-print-file-name=libstdc++.so"], capture_output=True, text=True).stdout.strip()
    env = dict(os.environ)
    # the C++ runtime too: the ASan interceptor of exception throws needs it
    # resolved at start-up, and the Python interpreter does not link it
    env["LD_PRELOAD"] = f"{rt}:{os.path.realpath(cxx)}"
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["AUVM_SIM_SANITIZE"] = "1"
    return env


def build(sanitize=None):
    """Compile if any source or header is newer than the library; returns its
    path.  sanitize (default: the AUVM_SIM_SANITIZE environment variable)
    builds the sanitized variant."""
    if sanitize is None:
        sanitize = os.environ.get("AUVM_SIM_SANITIZE") == "1"
    out = OUT_SAN if sanitize else OUT
    flags = SAN_FLAGS if sanitize else []
    deps = SOURCES + glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(ROOT, "include", "*.h")) + \
        glob.glob(os.path.join(HERE, "hip", "*.h"))
    os.makedirs(os.path.dirname(OUT), exist_ok=True)
    # one build at a time (parallel test workers share the output)
    with open(out + ".lock", "w") as lock:
        fcntl.flock(lock, fcntl.LOCK_EX)
        if os.path.exists(out) and os.path.getmtime(out) >= max(os.path.getmtime(d) for d in deps):
            return out
        tmp = f"{out}.{os.getpid()}.tmp"
        cmd = ["g++", "-O1", "-g", "-fPIC", "-shared", "-std=c++17", "-pthread", "-Wall", "-Wno-unused-function"] + flags + [
               "-I" + HERE, "-I" + os.path.join(ROOT, "include"), "-I" + CSRC] + SOURCES + ["-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


if __name__ == "__main__":
    import sys
    print(build(sanitize="--sanitize" in sys.argv))

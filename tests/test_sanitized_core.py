"""The C++ core (C ABI, planner, cost model, executor) under AddressSanitizer
and UndefinedBehaviorSanitizer: the host-only build of the same sources
(tests/sim, against the queue simulator) runs the executor's simulator suite
and the library-versus-oracle planner suites in a child process that
preloads the ASan runtime; any sanitizer report aborts it."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def test_core_suites_under_address_and_undefined_behavior_sanitizers():
    sys.path.insert(0, os.path.join(HERE, "sim"))
    import build_sim
    build_sim.build(sanitize=True)
    sel = ("golden or random_traces_bit_exact or object_granularity_bit_exact or kv_tensors or "
           "policy_defaults or touch_traces or read_only or caller_bound or timing_tracks or stall or "
           "new_budget or noalloc or object_plans")
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-s", "-p", "no:cacheprovider", "-p", "no:xdist",
           os.path.join(HERE, "test_executor_sim.py"), os.path.join(HERE, "test_capi_cpu.py"), "-k", sel]
    r = subprocess.run(cmd, cwd=ROOT, env=build_sim.sanitizer_env(), capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error" not in tail, tail
    assert " passed" in r.stdout, tail

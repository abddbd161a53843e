"""auvm_run_noalloc (the entry point for callers that cannot allocate) against
auvm_run on the GPU: a whole training step of the small LLaMA-style model
(attention and RMSNorm backward kernels, whose workspaces move to the static
scratch) gives bit-identical losses, gradients, moments and weights, on two
calls in a row, the second with a smaller input; a workspace above the
scratch's size is refused before anything runs."""
import dataclasses

import numpy as np
import pytest

from workloads import configs, init, trace

pytestmark = pytest.mark.gpu


def _step(cfg, noalloc):
    from paper_2609_06172_amd.session import Session
    w = trace.build(cfg, keep_grads=True)
    print(f"{cfg.name} {cfg.batch} x {cfg.prompt_len}, run_noalloc={noalloc}", flush=True)
    s = Session(w, device=0)                  # T+A+P at the config's factor, timing off
    if noalloc:
        s.ctx.run_noalloc(0, len(w.kernels))
    else:
        s.run_all()
    assert s.ctx.get_executed() == s.ctx.get_schedule()
    out = {"losses": s.read("losses")}
    for n in init.param_names(w):
        for suffix in (".grad", ".master", ".m", ".v", ""):
            out[n + suffix] = s.read(n + suffix)
    s.close()
    return out


def test_noalloc_step_equals_run_twice_with_a_smaller_second_input():
    big = configs.TRAIN_SMALL
    small = dataclasses.replace(big, batch=1, prompt_len=64)
    for cfg in (big, small):
        got = _step(cfg, True)
        ref = _step(cfg, False)
        assert got.keys() == ref.keys()
        for k in ref:
            assert got[k].tobytes() == ref[k].tobytes(), k


def test_noalloc_refuses_a_workspace_above_the_scratch():
    from paper_2609_06172_amd.capi import E_RANGE, AuvmError
    from paper_2609_06172_amd.session import Session
    from workloads.format import DT_BF16, DT_F32, MODE_R, MODE_W, OP_RMSNORM_BWD
    from gpu_util import single_kernel
    T, H = (8 << 20) // 4 + 64, 4               # rstd: 4T bytes, 256 above 8 MiB
    ops = [("x", (T, H), DT_F32, MODE_R, None), ("g", (H,), DT_BF16, MODE_R, None),
           ("dy", (T, H), DT_F32, MODE_R, None), ("dx", (T, H), DT_F32, MODE_W, None),
           ("dxb", (T, H), DT_BF16, MODE_W, None), ("dg", (H,), DT_F32, MODE_W, None),
           ("rstd", (T,), DT_F32, MODE_W, None)]
    w, _ = single_kernel(OP_RMSNORM_BWD, (T, H, 0), ops)
    for t in w.tensors:                       # inputs valid on the host (zeros), never launched
        t.host_init = True
    s = Session(w, device=0, M=w.footprint, fill=False)
    with pytest.raises(AuvmError) as e:
        s.ctx.run_noalloc(0, 1)
    assert e.value.code == E_RANGE and "workspace" in str(e.value)
    assert s.ctx.get_executed() == [] and s.ctx.get_counters()["kernels_run"] == 0
    s.close()

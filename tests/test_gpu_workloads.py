"""GPU parity at the full benchmark sizes, in both launch configurations:
cnn_fwd with the automatic plan, and the plan cnn_plan_find measures to be
fastest (the one the benchmark times, through cnn_fwd_plan_ws when it needs
a workspace).

Every output of every workload is compared with the fp64 oracle's (its
library-convolution route, computed once per workload on the host's cores
and pinned to the loop nest by the CPU tests), against the normwise and the
componentwise-conditioned bars.  A checksum identity, which holds at any
size, is checked as well:
    sum_{b,k,w,h} Out = sum_{c,r,s} (sum_k Ker[k,c,r,s]) * (sum_{b,w,h} In[b,c,sw*w+r,sh*h+s]).
"""
import functools

import numpy as np
import pytest

import oracle
from paper_2105_13480_amd import cnn, inputs

from gpu_helpers import TOL, errors, out_tensor, run, say, to_gpu

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=1)
def _oracle_full(name):
    """(In, Ker, Out, sum|In*Ker|) of a workload; the fp64 oracle over every
    output (one workload held at a time)."""
    w = inputs.BY_NAME[name]
    In, Ker = inputs.make_inputs(w)
    say(f"[workload] oracle {name}: {w.flops / 1e9:.2f} GFLOP")
    want, absv = oracle.conv_lib(In, Ker, w.sw, w.sh, with_abs=True)
    return In, Ker, want, absv


def _checksum(In64, Ker64, w):
    ks = Ker64.sum(axis=0)
    ka = np.abs(Ker64).sum(axis=0)
    tot = tot_abs = 0.0
    for r in range(w.Nr):
        for s in range(w.Ns):
            win = In64[:, :, r::w.sw, s::w.sh][:, :, :w.Nw, :w.Nh]
            tot += float((win.sum(axis=(0, 2, 3)) * ks[:, r, s]).sum())
            tot_abs += float((np.abs(win).sum(axis=(0, 2, 3)) * ka[:, r, s]).sum())
    return tot, tot_abs


@pytest.mark.parametrize("mode_out", ["fp32_out", "bf16_out"])
@pytest.mark.parametrize("plan_src", ["auto", "find"])
@pytest.mark.parametrize("name", [w.name for w in inputs.WORKLOADS])
def test_workload(name, plan_src, mode_out):
    w = inputs.BY_NAME[name]
    if w.dtype == "f32" and mode_out == "bf16_out":
        pytest.skip("fp32 workload has fp32 output only")
    mode = "f32" if w.dtype == "f32" else ("bf16" if mode_out == "fp32_out" else "bf16_obf16")
    In, Ker, want, absv = _oracle_full(name)
    if plan_src == "auto":  # what cnn_fwd runs: the model's best workspace-free plan
        plan = cnn.plan_tiles(cnn.problem(*w.dims()), cnn.DTYPES[mode], cnn.K_AUTO_NO_WORKSPACE)
    else:
        dIn, dKer = to_gpu(In), to_gpu(Ker)
        dOut = out_tensor(w.Nb, w.Nk, w.Nw, w.Nh, mode, 0.0)
        plan, _ = cnn.plan_find(dIn, dKer, dOut, w.sw, w.sh)
        del dIn, dKer, dOut
    say(f"[workload] {name} mode={mode} {plan_src} plan={plan.as_dict()['kernel']} "
        f"v{plan.variant} tk={plan.tk} tp={plan.tp} tc={plan.tc} kc={plan.kc} grid={plan.grid}")
    got = run(In, Ker, w.sw, w.sh, mode, plan=None if plan_src == "auto" else plan)
    assert got.shape == (w.Nb, w.Nk, w.Nw, w.Nh)
    assert np.isfinite(got).all()
    tol = TOL[mode]
    nw, cond, pt = errors(got, want, absv)
    say(f"[workload] {name} {mode} {plan_src}: every output: normwise {nw:.3e} "
        f"conditioned {cond:.3e} (pointwise {pt:.3e}, not gated)")
    assert nw <= tol and cond <= tol
    tot, tot_abs = _checksum(oracle.widen(In), oracle.widen(Ker), w)
    assert abs(got.sum() - tot) <= tol * tot_abs


def test_fwd_allocates_no_device_memory():
    """cnn_fwd's first call on each workload computes and caches a plan and
    launches it; it allocates no device memory (the plan never needs a
    workspace).  The kernels' code is loaded first, by running the same plan
    through cnn_fwd_plan, so that loading it is not counted."""
    import torch
    bufs = []
    for w in inputs.WORKLOADS:
        mode = "f32" if w.dtype == "f32" else "bf16"
        In, Ker = inputs.make_inputs(w)
        dIn, dKer = to_gpu(In), to_gpu(Ker)
        dOut = out_tensor(w.Nb, w.Nk, w.Nw, w.Nh, mode, 0.0)
        plan = cnn.plan_tiles(cnn.problem(*w.dims()), cnn.DTYPES[mode], cnn.K_AUTO_NO_WORKSPACE)
        assert plan.ws_bytes == 0
        say(f"[workload] load the code of {w.name} plan {plan.as_dict()['kernel']} v{plan.variant}")
        cnn.fwd_plan(dIn, dKer, dOut, plan, w.sw, w.sh)
        bufs.append((w, dIn, dKer, dOut))
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for w, dIn, dKer, dOut in bufs:
        say(f"[workload] first cnn_fwd call on {w.name}")
        cnn.fwd(dIn, dKer, dOut, w.sw, w.sh)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0, (free0, free1)

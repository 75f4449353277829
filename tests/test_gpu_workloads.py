"""GPU parity at the full benchmark sizes, in both launch configurations:
cnn_fwd with the automatic plan, and the plan cnn_plan_find measures to be
fastest (the one the benchmark times).

The tiny workload is compared element by element.  For the large ones the
oracle computes a sample of outputs one by one -- random points plus the
first and last output of every tile boundary it can reach cheaply -- and a
checksum identity, which holds at any size, covers every output:
    sum_{b,k,w,h} Out = sum_{c,r,s} (sum_k Ker[k,c,r,s]) * (sum_{b,w,h} In[b,c,sw*w+r,sh*h+s]).
"""
import numpy as np
import pytest

import oracle
from paper_2105_13480_amd import cnn, inputs

from gpu_helpers import TOL, errors, out_tensor, run, say, to_gpu

pytestmark = pytest.mark.gpu


def _sample_points(w, plan, n=3000, seed=0):
    rng = np.random.default_rng(seed)
    pts = [np.stack([rng.integers(0, m, size=n) for m in (w.Nb, w.Nk, w.Nw, w.Nh)], axis=1)]
    # outputs on both sides of composite-tile boundaries and feature-tile edges
    hw, npix = w.Nw * w.Nh, w.Nb * w.Nw * w.Nh
    edges = []
    tp, tk = max(int(plan.tp), 1), max(int(plan.tk), 1)
    for f in list(range(0, npix, tp))[:: max(1, npix // tp // 64)] + [npix - 1]:
        for q in (f - 1, f, min(f + tp - 1, npix - 1)):
            if 0 <= q < npix:
                for k in {0, min(tk - 1, w.Nk - 1), min(tk, w.Nk - 1), w.Nk - 1}:
                    edges.append((q // hw, k, (q % hw) // w.Nh, q % w.Nh))
    pts.append(np.array(edges, dtype=np.int64).reshape(-1, 4))
    return np.unique(np.concatenate(pts), axis=0)


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


@pytest.mark.parametrize("plan_src", ["auto", "find"])
@pytest.mark.parametrize("mode_out", ["fp32_out", "bf16_out"])
@pytest.mark.parametrize("name", [w.name for w in inputs.WORKLOADS])
def test_workload(name, mode_out, plan_src):
    w = inputs.BY_NAME[name]
    if w.dtype == "f32" and mode_out == "bf16_out":
        pytest.skip("fp32 workload has fp32 output only")
    mode = "f32" if w.dtype == "f32" else ("bf16" if mode_out == "fp32_out" else "bf16_obf16")
    In, Ker = inputs.make_inputs(w)
    if plan_src == "auto":
        plan = cnn.plan(cnn.problem(*w.dims()), cnn.DTYPES[mode])
    else:
        dIn, dKer = to_gpu(In), to_gpu(Ker)
        dOut = out_tensor(w.Nb, w.Nk, w.Nw, w.Nh, mode, 0.0)
        plan, _ = cnn.plan_find(dIn, dKer, dOut, w.sw, w.sh)
        del dIn, dKer, dOut
    say(f"[workload] {name} mode={mode} {plan_src} plan={plan.as_dict()['kernel']} "
        f"v{plan.variant} tk={plan.tk} tp={plan.tp} tc={plan.tc} grid={plan.grid}")
    got = run(In, Ker, w.sw, w.sh, mode, plan=None if plan_src == "auto" else plan)
    assert got.shape == (w.Nb, w.Nk, w.Nw, w.Nh)
    assert np.isfinite(got).all()
    tol = TOL[mode]
    if w.Nb * w.Nk * w.Nw * w.Nh <= 1 << 16:
        want, absv = oracle.conv(In, Ker, w.sw, w.sh, with_abs=True)
        nw, cond, _ = errors(got, want, absv)
    else:
        idx = _sample_points(w, plan)
        want, absv = oracle.conv_points(In, Ker, idx, w.sw, w.sh, with_abs=True)
        g = got[idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3]]
        nw, cond, _ = errors(g, want, absv)
    say(f"[workload] {name} {mode}: normwise {nw:.3e} conditioned {cond:.3e}")
    assert nw <= tol and cond <= tol
    tot, tot_abs = _checksum(oracle.widen(In), oracle.widen(Ker), w)
    assert abs(got.sum() - tot) <= tol * tot_abs

"""Shared helpers of the GPU tests: host<->device marshalling of the seeded
inputs and the error metrics.  No convolution arithmetic lives here."""
from __future__ import annotations

import sys

import numpy as np

from paper_2105_13480_amd import cnn, inputs

TOL = {"f32": 1e-5, "bf16": 2e-2, "bf16_obf16": 2e-2}


def say(msg: str):
    """Name the case before each GPU step (flushed, so it survives a crash)."""
    print(msg, flush=True)
    sys.stdout.flush()


def to_gpu(arr: np.ndarray):
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def out_tensor(Nb, Nk, Nw, Nh, mode: str, fill=float("nan")):
    import torch
    dt = torch.bfloat16 if mode == "bf16_obf16" else torch.float32
    return torch.full((Nb, Nk, Nw, Nh), fill, dtype=dt, device="cuda")


def to_host64(t) -> np.ndarray:
    """Exact float64 values of a float32 or bfloat16 GPU tensor."""
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return inputs.bf16_bits_to_f32(bits).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


def run(In: np.ndarray, Ker: np.ndarray, sw: int, sh: int, mode: str, plan=None,
        stream=None, fill=float("nan")):
    """Upload, run cnn_fwd (or cnn_fwd_plan, or cnn_fwd_plan_ws with a workspace of
    the plan's size), synchronise, return float64 Out."""
    import torch
    Nb, Nc, Nx, Ny = In.shape
    Nk, _, Nr, Ns = Ker.shape
    Nw, Nh = (Nx - Nr) // sw + 1, (Ny - Ns) // sh + 1
    dIn, dKer = to_gpu(In), to_gpu(Ker)
    dOut = out_tensor(Nb, Nk, Nw, Nh, mode, fill)
    if plan is None:
        cnn.fwd(dIn, dKer, dOut, sw, sh, stream=stream)
    elif plan.ws_bytes > 0:  # the caller's workspace (cnn_fwd_plan_ws)
        ws = torch.empty(plan.ws_bytes, dtype=torch.uint8, device="cuda")
        cnn.fwd_plan_ws(dIn, dKer, dOut, plan, ws, sw, sh, stream=stream)
        torch.cuda.synchronize()
        del ws
    else:
        cnn.fwd_plan(dIn, dKer, dOut, plan, sw, sh, stream=stream)
    torch.cuda.synchronize()
    return to_host64(dOut)


def errors(got: np.ndarray, want: np.ndarray, absv: np.ndarray):
    """(normwise, componentwise-conditioned, pointwise) max relative errors.

    normwise      max|g - o| / max|o|
    conditioned   max|g - o| / A, A = sum |In * Ker| (rounding-error scale of
                  any fp32 summation order); where A == 0 the error must be 0
    pointwise     max|g - o| / |o| over |o| > 0 (reported, not gated: the
                  zero-mean kernel makes outputs cross zero)
    """
    d = np.abs(got - want)
    scale = np.abs(want).max() if want.size else 0.0
    normwise = float(d.max() / scale) if scale > 0 else float(d.max() if d.size else 0.0)
    pos = absv > 0
    cond = float((d[pos] / absv[pos]).max()) if pos.any() else 0.0
    if (~pos).any() and d[~pos].max() > 0:
        cond = float("inf")
    nz = np.abs(want) > 0
    point = float((d[nz] / np.abs(want[nz])).max()) if nz.any() else 0.0
    return normwise, cond, point


def variant_dims(kernel, vid, dt, tk, tp, tc, stencils):
    """Problem sizes on which instantiation `vid` is what cnn_plan_tiles
    picks for (kernel, tk, tp, tc): ragged channel, feature and output
    tails, several tiles.  `stencils` lists the (Nr, Ns) to try.  None if
    no candidate fits."""
    for stencil in stencils:
        dims = _variant_dims_one(kernel, vid, dt, tk, tp, tc, stencil)
        if dims is not None:
            return dims
    return None


def variant_plan(dims, dt, kernel, tk, tp, tc, vid, bud=None):
    """The plan of instantiation `vid` for (kernel, tk, tp, tc) on problem
    dims: cnn_plan_tiles' choice if it is `vid`, else the candidate of that
    instantiation (several instantiations may implement one tiling); None
    if it does not fit."""
    prob = cnn.problem(*dims)
    try:
        pl = cnn.plan_tiles(prob, dt, kernel, tk, tp, tc, bud)
        if pl.variant == vid:
            return pl
    except cnn.CnnError:
        pl = None
    match = [c for c in cnn.plan_candidates(prob, dt, bud)
             if c.variant == vid and c.kernel == kernel and c.tk == tk and
             (tp == 0 or c.tp == tp or kernel != cnn.K_SROWS)]
    same = [c for c in match if pl is not None and c.tp == pl.tp]
    return (same or match or [None])[0]


def _fits(dims, dt, kernel, tk, tp, tc, vid):
    return variant_plan(dims, dt, kernel, tk, tp, tc, vid, cnn.budget()) is not None


def _variant_dims_one(kernel, vid, dt, tk, tp, tc, stencil):
    Nr, Ns = stencil
    if kernel == cnn.K_ROWS:
        return rows_dims(vid, dt, stencil)
    if kernel == cnn.K_SROWS:  # stride 2, Nc % 16 == 0, L | Nw (raw-Ker form: Nc >= 16 L)
        for dims in [(2, 32, 300, 7, 28, Nr, Ns, 2, 2), (3, 16, 64, 8, 12, Nr, Ns, 2, 2),
                     (2, 128, 300, 28, 14, Nr, Ns, 2, 2)]:
            if _fits(dims, dt, kernel, tk, 0, tc, vid):
                return dims
        return None
    if kernel == cnn.K_GEMM1:  # 1x1, Nc % 8 == 0; stride 1 (Nw*Nh % 4 == 0) or 2 (Nh % 4 == 0)
        cands = [(3, tc + 8, tk + 7, 6, 10, 1, 1, 1, 1), (2, 2 * tc + 16, tk - 5, 8, 14, 1, 1, 1, 1),
                 (1, 24, tk + 7, 4, 5, 1, 1, 1, 1), (3, tc + 8, tk + 7, 6, 8, 1, 1, 2, 2),
                 (2, 2 * tc + 16, tk - 5, 7, 12, 1, 1, 2, 2)]
        for dims in cands:
            if _fits(dims, dt, kernel, tk, tp, tc, vid):
                return dims
        return None
    if kernel == cnn.K_SPLITC and Nr == Ns and Nr in (1, 3) and tk == 32:
        # channel-slice kernel: Nc % 16 == 0 (the last stage 16 channels), ragged Nk
        for dims in [(1, 48, 39, 7, 7, Nr, Ns, 1, 1), (2, 96, 45, 5, 9, Nr, Ns, 2, 1)]:
            if _fits(dims, dt, kernel, tk, tp, tc, vid):
                return dims
        return None
    if kernel == cnn.K_SMALLC:  # few channels: Nc*Nr rows must fit the K-steps
        nc = 3 if Nr == 7 else 9
        cands = [(3, nc, tk + 7, 9, 13, Nr, Ns, 2, 2), (2, nc, tk + 7, 7, 13, Nr, Ns, 1, 1),
                 (2, nc, 5, 11, 6, Nr, Ns, 2, 1)]
    else:
        cands = []
    cands += [(3, tc + 5, tk + 7, 9, 13, Nr, Ns, 1, 2), (2, tc + 5, tk + 7, 7, 13, Nr, Ns, 1, 1),
             (3, tc + 8, tk + 7, 9, 13, Nr, Ns, 1, 2), (2, tc + 8, tk + 7, 7, 13, Nr, Ns, 1, 1),
             (3, tc + 8, max(1, tk - 5), 9, 13, Nr, Ns, 1, 2),
             (2, tc + 8, tk + 7, 4, 5, Nr, Ns, 2, 1), (2, tc + 8, tk + 7, 6, 8, Nr, Ns, 2, 2),
             (2, tc + 3, max(1, tk - 5), 5, 9, Nr, Ns, 1, 1), (1, tc + 5, tk + 3, 6, 7, Nr, Ns, 1, 1),
             (2, tc + 5, tk + 7, 4, 5, Nr, Ns, 2, 1), (1, tc + 5, tk + 7, 3, 4, Nr, Ns, 1, 1)]
    for dims in cands:
        if _fits(dims, dt, kernel, tk, tp, tc, vid):
            return dims
    return None


def variant_info(vid):
    return next(v for v in cnn.variants() if v.variant == vid)


def rows_dims(vid, dt, stencil):
    """A stride-1 problem the row-streaming instantiation `vid` is chosen
    for: two k tiles (ragged), a ragged channel tail, a band of several
    row groups."""
    v = variant_info(vid)
    nr, ns, mb, ncp = v.nr, v.ns, v.mode, int(v.tc)
    nc = ncp - 8                           # Nc % 8 == 0, last group half empty
    nh = (29 if mb == 1 else 45) - (ns - 1) if ns > 1 else (30 if mb == 1 else 50)
    for dims in [(2, nc, 71, 10, nh, nr, ns, 1, 1), (3, nc, 64, 6, nh + 1, nr, ns, 1, 1)]:
        for L in (dims[3], 5, 2, 1):
            if dims[3] % L:
                continue
            if _fits(dims, dt, cnn.K_ROWS, 64, L * dims[4], 0, vid):
                return dims
    return None


def variant_cases():
    """(kernel, vid, dtype, tk, tp, tc, stencils to try) of every
    instantiation the library holds (cnn_variants)."""
    out = []
    for v in cnn.variants():
        if v.nr:
            stencils = [(v.nr, v.ns)]
        elif v.kernel == cnn.K_SMALLC:
            stencils = [(7, 7), (5, 5)]
        else:
            stencils = [(5, 2), (1, 1), (3, 3)]
        tc = 0 if v.kernel == cnn.K_ROWS else int(v.tc)
        out.append((v.kernel, v.variant, v.dtype, int(v.tk), int(v.tp), tc, stencils))
    return out

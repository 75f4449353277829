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
    """Upload, run cnn_fwd (or cnn_fwd_plan), synchronise, return float64 Out."""
    import torch
    Nb, Nc, Nx, Ny = In.shape
    Nk, _, Nr, Ns = Ker.shape
    Nw, Nh = (Nx - Nr) // sw + 1, (Ny - Ns) // sh + 1
    dIn, dKer = to_gpu(In), to_gpu(Ker)
    dOut = out_tensor(Nb, Nk, Nw, Nh, mode, fill)
    if plan is None:
        cnn.fwd(dIn, dKer, dOut, sw, sh, stream=stream)
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


def variant_dims(kernel, vid, dt, tk, tp, tc, stencil):
    """Problem sizes on which instantiation `vid` is what cnn_plan_tiles
    picks for (kernel, tk, tp, tc): ragged channel, feature and output
    tails, several tiles.  None if no candidate fits."""
    Nr, Ns = stencil
    if kernel == cnn.K_ROWS:
        return rows_dims(vid, dt, stencil)
    if kernel == cnn.K_SROWS:  # stride 2, Nc % 16 == 0, Nh % 4 == 0, L | Nw
        from oracle import select as osel
        L = next(r[4] for r in osel.SROWS if r[0] == vid)
        dims = {7: (2, 32, 300, 7, 28, Nr, Ns, 2, 2), 4: (3, 16, 64, 8, 12, Nr, Ns, 2, 2)}[L]
        try:
            pl = cnn.plan_tiles(cnn.problem(*dims), dt, kernel, tk, 0, tc, cnn.budget())
        except cnn.CnnError:
            return None
        return dims if pl.variant == vid else None
    if kernel == cnn.K_GEMM1:  # 1x1, Nc % 8 == 0; stride 1 (Nw*Nh % 4 == 0) or 2 (Nh % 4 == 0)
        cands = [(3, tc + 8, tk + 7, 6, 10, 1, 1, 1, 1), (2, 2 * tc + 16, tk - 5, 8, 14, 1, 1, 1, 1),
                 (1, 24, tk + 7, 4, 5, 1, 1, 1, 1), (3, tc + 8, tk + 7, 6, 8, 1, 1, 2, 2),
                 (2, 2 * tc + 16, tk - 5, 7, 12, 1, 1, 2, 2)]
        for dims in cands:
            try:
                pl = cnn.plan_tiles(cnn.problem(*dims), dt, kernel, tk, tp, tc, cnn.budget())
            except cnn.CnnError:
                continue
            if pl.variant == vid:
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
        try:
            pl = cnn.plan_tiles(cnn.problem(*dims), dt, kernel, tk, tp, tc, cnn.budget())
        except cnn.CnnError:
            continue
        if pl.variant == vid:
            return dims
    return None


def rows_dims(vid, dt, stencil):
    """A stride-1 problem the row-streaming instantiation `vid` is chosen
    for: two k tiles (ragged), a ragged channel tail, a band of several
    row groups; the (tp = L*Nh) is returned as dims[-1] of the tuple."""
    from oracle import select as osel
    row = next(r for r in osel.ROWS if r[0] == vid)
    _, _, nr, ns, mb, ncg, _, _ = row
    nc = 16 * ncg - 8                      # Nc % 8 == 0, last group half empty
    nh = (29 if mb == 1 else 45) - (ns - 1) if ns > 1 else (30 if mb == 1 else 50)
    for dims in [(2, nc, 71, 10, nh, nr, ns, 1, 1), (3, nc, 64, 6, nh + 1, nr, ns, 1, 1)]:
        for L in (dims[3], 5, 2, 1):
            if dims[3] % L:
                continue
            try:
                pl = cnn.plan_tiles(cnn.problem(*dims), dt, cnn.K_ROWS, 64, L * dims[4], 0,
                                    cnn.budget())
            except cnn.CnnError:
                continue
            if pl.variant == vid:
                return dims
    return None


def variant_cases():
    """(kernel, vid, dtype, tk, tp, tc, stencil) of every implicit-GEMM
    instantiation, from the oracle's independent tables."""
    from oracle import select as osel
    out = []
    for vid, dt, wm, wn, mb, nb, tc in osel.IGEMM:
        out.append((cnn.K_IGEMM, vid, dt, 32 * wm * mb, 32 * wn * nb, tc, (3, 3)))
    for vid, dt, wm, wn, mb, nb, tc, nr, ns, _ in osel.IGEMM4:
        out.append((cnn.K_IGEMM_WIDE, vid, dt, 32 * wm * mb, 32 * wn * nb, tc,
                    (nr, ns) if nr else (5, 2)))
    for vid, dt, wm, wn, mb, nb, tc, nr, ns, *_ in osel.IGEMM3:
        tk = 32 * wm * mb
        out.append((cnn.K_IGEMM_DMA, vid, dt, tk, 32 * wn * nb, tc,
                    (nr, ns) if nr else ((1, 1) if vid % 100 in (10, 11, 12) else (5, 2))))
    for vid, dt, wm, wn, mb, nb, tc, nr, ns, kres, _, _ in osel.STREAM:
        out.append((cnn.K_STREAM, vid, dt, 32 * wm * mb, 32 * wn * nb, tc, (nr, ns)))
    for vid, dt, wp, wk, mbp, nbk, tc, _ in osel.GEMM1:
        out.append((cnn.K_GEMM1, vid, dt, 32 * wk * nbk, 32 * wp * mbp, tc, (1, 1)))
    for vid, dt, nr, ns, L in osel.SROWS:
        out.append((cnn.K_SROWS, vid, dt, 256, 0, 16, (nr, ns)))
    for vid, dt, nr, ns, mb, ncg, _, _ in osel.ROWS:
        out.append((cnn.K_ROWS, vid, dt, 64, 0, 0, (nr, ns)))
    for vid, dt, nb, ks in osel.SMALLC:
        out.append((cnn.K_SMALLC, vid, dt, 64, 128 * nb, 0, (7, 7) if ks <= 12 else (5, 5)))
    for vid, dt, wm, wn, mb, nb, tc, nr, ns, _, rawk, pw in osel.IGEMM2:
        tk = 32 * wm * mb
        kern = cnn.K_POINTWISE if pw else (cnn.K_IGEMM_RAWK if rawk else cnn.K_IGEMM_PIPE)
        out.append((kern, vid, dt, tk, 32 * wn * nb, tc,
                    (nr, ns) if nr else ((1, 1) if tk >= 256 else (5, 2))))
    return out

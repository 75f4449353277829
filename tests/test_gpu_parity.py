"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bars: fp32 max relative error 1e-5, bf16 inputs with fp32 accumulation 2e-2,
both normwise and componentwise-conditioned (see gpu_helpers.errors).
Integer inputs make every fp32 partial sum exact, so those cases must match
the oracle bit for bit; a delta kernel must reproduce a strided copy of In
bit for bit.
"""
import numpy as np
import pytest

import oracle
from paper_2105_13480_amd import cnn, inputs

from gpu_helpers import (TOL, errors, out_tensor, run, say, to_gpu, to_host64, variant_cases,
                         variant_dims, variant_plan)

pytestmark = pytest.mark.gpu

MODES = {"f32": cnn.CNN_F32, "bf16": cnn.CNN_BF16, "bf16_obf16": cnn.CNN_BF16_OBF16}


def _arrays(dims, mode, seed, dist=("uniform", -1.0, 1.0), kdist=("he",)):
    return inputs.make_arrays(*dims, "f32" if mode == "f32" else "bf16",
                              seed_in=seed, seed_ker=seed + 1, in_dist=dist, ker_dist=kdist)


# ---- mid-size problems: whole output compared element by element ---------
MID = [
    (3, 40, 70, 13, 11, 3, 3, 1, 1),     # ragged everywhere
    (2, 37, 33, 9, 14, 3, 2, 2, 1),      # Nr != Ns, sw != sh
    (1, 64, 96, 20, 20, 3, 3, 2, 2),
    (4, 17, 5, 7, 7, 5, 5, 1, 1),
    (3, 70, 130, 10, 10, 1, 1, 1, 1),    # 1x1
    (2, 48, 40, 9, 8, 1, 1, 2, 2),       # 1x1 stride 2
    (2, 3, 64, 30, 30, 7, 7, 2, 2),      # stem-like, few channels
    (1, 1, 1, 1, 1, 1, 1, 1, 1),         # degenerate
    (1, 1, 1, 5, 3, 4, 2, 3, 1),
    (5, 2, 3, 1, 9, 1, 3, 1, 2),
]


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("dims", MID)
def test_mid_size_auto_plan(dims, mode):
    say(f"[parity] auto plan dims={dims} mode={mode}")
    In, Ker = _arrays(dims, mode, seed=sum(dims))
    sw, sh = dims[7], dims[8]
    got = run(In, Ker, sw, sh, mode)
    want, absv = oracle.conv(In, Ker, sw, sh, with_abs=True)
    nw, cond, _ = errors(got, want, absv)
    assert nw <= TOL[mode] and cond <= TOL[mode], (nw, cond)


@pytest.mark.parametrize("case", variant_cases(), ids=lambda c: f"v{c[1]}")
def test_every_igemm_variant_exact_integers(case):
    kernel, vid, dt, tk, tp, tc, stencils = case
    mode = {0: "f32", 1: "bf16", 2: "bf16_obf16"}[dt]
    dims = variant_dims(kernel, vid, dt, tk, tp, tc, stencils)
    assert dims is not None, f"no test shape fits instantiation {vid}"
    In, Ker = _arrays(dims, mode, seed=vid, dist=("int", -2, 2), kdist=("int", -2, 2))
    pl = variant_plan(dims, dt, kernel, tk, tp, tc, vid)
    assert pl is not None and pl.variant == vid
    say(f"[parity] variant {vid} tk={tk} tp={tp} tc={tc} dims={dims} grid={pl.grid}")
    got = run(In, Ker, dims[7], dims[8], mode, plan=pl)
    want = oracle.conv(In, Ker, dims[7], dims[8])
    if mode == "bf16_obf16":
        want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(want.astype(np.float32))).astype(np.float64)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
def test_smallc_runs_of_tiles_exact(mode):
    """The few-channel kernel walks a run of tiles per workgroup (two
    workgroups per CU): 896 tiles of two 64-feature k tiles, so each
    workgroup takes several tiles and repacks its Ker image when the k tile
    changes; every output compared exactly on integer inputs."""
    dims = (32, 3, 128, 56, 56, 7, 7, 2, 2)
    dt = cnn.DTYPES[mode]
    In, Ker = _arrays(dims, mode, seed=77, dist=("int", -2, 2), kdist=("int", -2, 2))
    pl = min((c for c in cnn.plan_candidates(cnn.problem(*dims), dt)
              if c.kernel == cnn.K_SMALLC and c.tk == 64), key=lambda c: c.model_us)
    assert pl.grid > 2 * cnn.device_budget(0).cus, "more tiles than resident workgroups"
    say(f"[parity] smallc runs v{pl.variant} tp={pl.tp} grid={pl.grid} mode={mode}")
    got = run(In, Ker, dims[7], dims[8], mode, plan=pl)
    want = oracle.conv_lib(In, Ker, dims[7], dims[8], False)
    if mode == "bf16_obf16":
        want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(want.astype(np.float32))).astype(np.float64)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("mode", list(MODES))
def test_direct_kernel_exact_integers(mode):
    dims = (2, 7, 9, 11, 6, 3, 2, 2, 1)
    In, Ker = _arrays(dims, mode, seed=3, dist=("int", -2, 2), kdist=("int", -2, 2))
    pl = cnn.plan_tiles(cnn.problem(*dims), MODES[mode], cnn.K_DIRECT)
    say(f"[parity] direct kernel dims={dims} mode={mode}")
    got = run(In, Ker, dims[7], dims[8], mode, plan=pl)
    want = oracle.conv(In, Ker, dims[7], dims[8])
    if mode == "bf16_obf16":
        want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(want.astype(np.float32))).astype(np.float64)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("kernel", ["auto", "direct"])
@pytest.mark.parametrize("mode", ["f32", "bf16"])
@pytest.mark.parametrize("geom", [(3, 3, 1, 1), (3, 2, 2, 1), (1, 1, 2, 2), (7, 7, 2, 2)])
def test_delta_kernel_is_strided_copy(geom, mode, kernel):
    """Ker[k,c,r,s] = [c == k mod Nc][r == r0][s == s0] copies In exactly."""
    Nr, Ns, sw, sh = geom
    Nb, Nc, Nk, Nw, Nh = 2, 5, 11, 9, 7
    dims = (Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)
    In, _ = _arrays(dims, mode, seed=31)
    for r0, s0 in [(0, 0), (Nr - 1, Ns - 1), (Nr // 2, 0)]:
        Ker32 = np.zeros((Nk, Nc, Nr, Ns), dtype=np.float32)
        for k in range(Nk):
            Ker32[k, k % Nc, r0, s0] = 1.0
        Ker = Ker32 if mode == "f32" else inputs.f32_to_bf16_bits(Ker32)
        pl = None
        if kernel == "direct":
            pl = cnn.plan_tiles(cnn.problem(*dims), MODES[mode], cnn.K_DIRECT)
        say(f"[parity] delta kernel geom={geom} r0={r0} s0={s0} mode={mode} kernel={kernel}")
        got = run(In, Ker, sw, sh, mode, plan=pl)
        In64 = oracle.widen(In)
        for k in range(Nk):
            want = In64[:, k % Nc, r0::sw, s0::sh][:, :Nw, :Nh]
            assert np.array_equal(got[:, k], want)


def test_out_is_overwritten_not_read():
    dims = (2, 9, 33, 6, 7, 3, 3, 1, 1)
    In, Ker = _arrays(dims, "bf16", seed=41)
    say("[parity] Out prefilled with NaN and with 1e30")
    a = run(In, Ker, 1, 1, "bf16", fill=float("nan"))
    b = run(In, Ker, 1, 1, "bf16", fill=1e30)
    assert np.isfinite(a).all() and np.array_equal(a, b)


def test_repeatable_bitwise():
    w = inputs.BY_NAME["conv3x3_b32"]
    dims = (4,) + w.dims()[1:]
    In, Ker = _arrays(dims, "bf16", seed=43)
    say(f"[parity] run twice dims={dims}")
    a = run(In, Ker, 1, 1, "bf16")
    b = run(In, Ker, 1, 1, "bf16")
    assert np.array_equal(a, b)


def test_nondefault_stream():
    import torch
    dims = (2, 16, 40, 12, 12, 3, 3, 1, 1)
    In, Ker = _arrays(dims, "bf16", seed=47)
    s = torch.cuda.Stream()
    say("[parity] launch on a side stream")
    with torch.cuda.stream(s):
        got = run(In, Ker, 1, 1, "bf16", stream=s)
    want, absv = oracle.conv(In, Ker, 1, 1, with_abs=True)
    nw, cond, _ = errors(got, want, absv)
    assert nw <= TOL["bf16"] and cond <= TOL["bf16"]


def test_bad_arguments_raise_before_launch():
    import torch
    dims = (1, 2, 3, 4, 4, 3, 3, 1, 1)
    In, Ker = _arrays(dims, "f32", seed=1)
    dIn, dKer = to_gpu(In), to_gpu(Ker)
    out = out_tensor(1, 3, 4, 4, "f32")
    with pytest.raises(cnn.CnnError) as e:
        cnn.fwd_ptr(dIn.data_ptr(), dKer.data_ptr(), dIn.data_ptr(), dims, cnn.CNN_F32)
    assert e.value.status == -5
    with pytest.raises(cnn.CnnError):
        cnn.fwd_ptr(dIn.data_ptr(), dKer.data_ptr(), out.data_ptr(), dims, 9)
    torch.cuda.synchronize()


@pytest.mark.parametrize("mode", ["bf16", "f32"])
def test_plan_find_exact_and_cached(mode):
    """cnn_plan_find times every candidate tiling, leaves the returned plan's
    result in Out, and cnn_fwd then uses the fastest candidate that needs no
    workspace (the returned one when it needs none)."""
    import torch
    dims = (3, 40, 70, 13, 11, 3, 3, 1, 1)
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = dims
    rng = np.random.default_rng(77)
    Nx, Ny = sw * (Nw - 1) + Nr, sh * (Nh - 1) + Ns
    In = rng.integers(-2, 3, size=(Nb, Nc, Nx, Ny)).astype(np.float32)
    Ker = rng.integers(-2, 3, size=(Nk, Nc, Nr, Ns)).astype(np.float32)
    if mode == "bf16":
        In, Ker = inputs.f32_to_bf16_bits(In), inputs.f32_to_bf16_bits(Ker)
    want = oracle.conv(In, Ker, sw, sh)
    dIn, dKer = to_gpu(In), to_gpu(Ker)
    dOut = out_tensor(Nb, Nk, Nw, Nh, mode)
    say(f"[parity] plan_find dims={dims} mode={mode}")
    pl, ms = cnn.plan_find(dIn, dKer, dOut, sw, sh)
    torch.cuda.synchronize()
    assert ms > 0
    assert np.array_equal(to_host64(dOut), want)
    cached = cnn.plan_lookup(cnn.problem(*dims), MODES[mode])
    assert cached.ws_bytes == 0
    if pl.ws_bytes == 0:
        assert (cached.kernel, cached.variant, cached.tk, cached.tp, cached.tc) == \
            (pl.kernel, pl.variant, pl.tk, pl.tp, pl.tc)
    dOut.fill_(float("nan"))
    say(f"[parity] cnn_fwd after plan_find dims={dims} mode={mode}")
    cnn.fwd(dIn, dKer, dOut, sw, sh)
    torch.cuda.synchronize()
    assert np.array_equal(to_host64(dOut), want)


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
@pytest.mark.parametrize("shape", [
    (3, 72, 70, 10, 14, 1, 1, 1, 1),   # stride 1, Nh even: aligned pairs
    (2, 80, 40, 9, 13, 1, 1, 1, 1),    # Nh odd: element path
    (3, 72, 70, 10, 14, 1, 1, 2, 2),   # stride 2, Nh even: 8-byte gather
    (2, 64, 33, 7, 9, 1, 1, 2, 2),     # stride 2, Nh odd
    (2, 64, 33, 6, 8, 1, 1, 2, 1),     # stride only along w
    (2, 64, 33, 6, 8, 1, 1, 1, 3),     # stride 3 along h
])
@pytest.mark.parametrize("tk", [64, 128, 256])
def test_pointwise_gather_exact(shape, tk, mode):
    """The 1x1 gather kernels (every tiling, every load path) on small
    integers: bit-exact with the oracle in the fp32-Out mode, and within
    bf16 rounding of it in the bf16-Out mode."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = shape
    tp = {64: 256, 128: 256, 256: 128}[tk]
    try:
        pl = cnn.plan_tiles(cnn.problem(*shape), MODES[mode], cnn.K_POINTWISE, tk, tp, 64)
    except cnn.CnnError:
        pytest.skip("tiling does not fit this shape")
    rng = np.random.default_rng(sum(shape) + tk)
    Nx, Ny = sw * (Nw - 1) + Nr, sh * (Nh - 1) + Ns
    In = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nb, Nc, Nx, Ny)).astype(np.float32))
    Ker = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nk, Nc, Nr, Ns)).astype(np.float32))
    want = oracle.conv(In, Ker, sw, sh)
    say(f"[parity] pointwise gather shape={shape} tk={tk} mode={mode} v{pl.variant} tp={pl.tp}")
    got = run(In, Ker, sw, sh, mode, plan=pl)
    if mode == "bf16":
        assert np.array_equal(got, want)
    else:
        assert np.array_equal(got, oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32))))


# ---- row-streaming kernel: bands, row groups, store paths -----------------
ROWS_SHAPES = [
    (2, 56, 71, 10, 56, 3, 3, 1, 1),   # Ny = 58 (two 32-position blocks), 16-byte stores
    (3, 64, 64, 9, 30, 3, 3, 1, 1),    # Ny = 32 exactly, Nh % 4 != 0: element stores
    (3, 64, 64, 9, 28, 3, 3, 1, 1),    # one 32-position block, 16-byte stores
    (2, 24, 40, 8, 62, 3, 3, 1, 1),    # Ny = 64 exactly, two channel groups, one k tile
    (2, 24, 40, 12, 44, 3, 3, 1, 1),   # two channel groups, 16-byte stores
    (1, 32, 130, 12, 13, 3, 3, 1, 1),  # three k tiles, ragged
    (1, 32, 130, 12, 12, 3, 3, 1, 1),  # three k tiles, 16-byte stores
    (2, 56, 70, 6, 50, 1, 1, 1, 1),    # 1x1
    (2, 56, 70, 6, 48, 1, 1, 1, 1),    # 1x1, 16-byte stores
]


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
@pytest.mark.parametrize("shape", ROWS_SHAPES)
def test_rows_bands_exact(shape, mode):
    """Every band length L (dividing Nw): single partial group, several full
    groups, a partial last group; bit-exact with the oracle on integers."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = shape
    rng = np.random.default_rng(sum(shape))
    Nx, Ny = Nw + Nr - 1, Nh + Ns - 1
    In = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nb, Nc, Nx, Ny)).astype(np.float32))
    Ker = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nk, Nc, Nr, Ns)).astype(np.float32))
    want = oracle.conv(In, Ker, sw, sh)
    if mode == "bf16_obf16":
        want = oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32)))
    bands = [L for L in range(1, Nw + 1) if Nw % L == 0]
    for L in bands:
        pl = cnn.plan_tiles(cnn.problem(*shape), MODES[mode], cnn.K_ROWS, 64, L * Nh, 0)
        say(f"[parity] rows shape={shape} L={L} v{pl.variant} grid={pl.grid} mode={mode}")
        got = run(In, Ker, sw, sh, mode, plan=pl)
        assert np.array_equal(got, want), f"band length {L}"


def test_rows_float_headline_shape():
    """The 56x56 3x3 layer on uniform inputs through the row kernel at every
    band length the plan search tries: every output within the bf16
    tolerance of the fp64 oracle."""
    w = inputs.BY_NAME["conv3x3_b32"]
    In, Ker = inputs.make_inputs(w)
    want, absv = oracle.conv(In, Ker, 1, 1, with_abs=True)
    for L in (4, 7, 8):
        pl = cnn.plan_tiles(cnn.problem(*w.dims()), cnn.CNN_BF16, cnn.K_ROWS, 64, L * w.Nh, 0)
        say(f"[parity] rows headline v{pl.variant} tp={pl.tp} grid={pl.grid}")
        got = run(In, Ker, 1, 1, "bf16", plan=pl)
        nw, cond, _ = errors(got, want, absv)
        assert nw <= TOL["bf16"] and cond <= TOL["bf16"], (L, nw, cond)


# ---- 1x1 stride-1 GEMM kernel: stages, k tiles, tiles across images --------
GEMM1_SHAPES = [
    (3, 72, 71, 6, 10, 1, 1, 1, 1),     # Nc = 72: a second stage of 8 channels
    (2, 64, 300, 4, 5, 1, 1, 1, 1),     # two k tiles of 256, 20-pixel images
    (5, 40, 130, 7, 12, 1, 1, 1, 1),    # 84-pixel images, tiles span images
    (1, 128, 64, 14, 14, 1, 1, 1, 1),   # one 196-pixel image
    (2, 24, 40, 6, 6, 1, 1, 1, 1),      # Nc < one stage: Ker blocks past Nc
    (3, 8, 33, 4, 4, 1, 1, 1, 1),       # a single 8-channel block
]


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
@pytest.mark.parametrize("shape", GEMM1_SHAPES)
def test_gemm1_exact(shape, mode):
    """Every 1x1 GEMM instantiation of the mode, its balanced tile and a
    small tile (several tiles per image or images per tile): bit-exact with
    the oracle on integer inputs."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = shape
    rng = np.random.default_rng(sum(shape) + 11)
    In = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nb, Nc, Nw, Nh)).astype(np.float32))
    Ker = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nk, Nc, 1, 1)).astype(np.float32))
    want = oracle.conv(In, Ker, 1, 1)
    if mode == "bf16_obf16":
        want = oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32)))
    dt = MODES[mode]
    for v in cnn.variants():
        if v.kernel != cnn.K_GEMM1 or v.dtype != dt or v.mode != 0:
            continue
        vid, tk, tpmax, tc = v.variant, v.tk, v.tp, v.tc
        for cus in (256, 3):  # balanced tile; few slots -> the largest tile
            pl = cnn.plan_tiles(cnn.problem(*shape), dt, cnn.K_GEMM1, tk, tpmax, tc,
                                cnn.budget(cus, 160 * 1024, 128, 2))
            assert pl.variant == vid and pl.tp % 4 == 0
            say(f"[parity] gemm1 shape={shape} v{vid} tp={pl.tp} grid={pl.grid} mode={mode}")
            got = run(In, Ker, 1, 1, mode, plan=pl)
            assert np.array_equal(got, want), (vid, pl.tp)


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
@pytest.mark.parametrize("shape", GEMM1_SHAPES + [(1, 1000, 33, 12, 20, 1, 1, 1, 1),
                                                  (4, 8, 256, 2, 2, 1, 1, 1, 1),
                                                  (3, 16, 257, 6, 10, 1, 1, 1, 1)])
def test_gemm1_ring_exact(shape, mode):
    """The 1x1 GEMM kernel with whole-image tiles and both operands copied
    by DMA into a four-stage ring: bit-exact with the oracle on integer
    inputs (ragged last stage, a 240-pixel image, k tiles past Nk, 4-pixel
    images).  With bf16 Out a tile's run leaves as whole 16-byte units only
    when it starts and ends on 16-byte boundaries: Nk = 71 with 60-pixel
    images never does, Nk = 257 does for images 0 and 2 and not for image 1
    of the first k tile, so both store paths run side by side."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = shape
    rng = np.random.default_rng(sum(shape) + 13)
    In = inputs.f32_to_bf16_bits(rng.integers(-3, 4, size=(Nb, Nc, Nw, Nh)).astype(np.float32))
    Ker = inputs.f32_to_bf16_bits(rng.integers(-3, 4, size=(Nk, Nc, 1, 1)).astype(np.float32))
    want = oracle.conv(In, Ker, 1, 1)
    if mode == "bf16_obf16":
        want = oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32)))
    dt = MODES[mode]
    ran = 0
    for v in cnn.variants():
        if v.kernel != cnn.K_GEMM1 or v.dtype != dt or v.mode != 2:
            continue
        vid, tk, tpmax, tc = v.variant, v.tk, v.tp, v.tc
        pl = cnn.plan_tiles(cnn.problem(*shape), dt, cnn.K_GEMM1, tk, tpmax, tc)
        assert pl.variant == vid and pl.tp == Nw * Nh and pl.grid == Nb * -(-Nk // tk)
        say(f"[parity] gemm1 ring shape={shape} v{vid} grid={pl.grid} mode={mode}")
        got = run(In, Ker, 1, 1, mode, plan=pl)
        assert np.array_equal(got, want), vid
        ran += 1
    assert ran == 1


# ---- stride-2 row-band kernel: chunks, k tiles, bands, the last element -----
SROWS_SHAPES = [
    (2, 32, 300, 7, 28, 3, 3, 2, 2),    # Ny = 57: two k tiles (the second ragged), one band
    (3, 16, 64, 8, 12, 3, 3, 2, 2),     # one chunk, features past Nk, two bands of 4
    (1, 48, 256, 14, 28, 3, 3, 2, 2),   # three chunks, two bands of 7
    (2, 16, 40, 28, 4, 3, 3, 2, 2),     # Nh = 4: short rows, 4 or 7 bands
    (2, 16, 40, 7, 27, 3, 3, 2, 2),     # Nh = 27 (Ny = 55): a ragged row end
    (1, 32, 70, 8, 13, 3, 3, 2, 2),     # Nh = 13, two bands of 4, features past Nk
    (2, 16, 200, 7, 28, 3, 3, 2, 2),    # one chunk: first-tile rows left for the end
    (1, 128, 160, 4, 28, 3, 3, 2, 2),   # eight chunks, a second tile of 32 features
    (2, 128, 300, 7, 27, 3, 3, 2, 2),   # eight chunks, Nh = 27; k range 2 has one tile of 44
    (1, 160, 256, 14, 28, 3, 3, 2, 2),  # ten chunks per tile: seven store rows, three do not
    (2, 64, 129, 8, 12, 3, 3, 2, 2),    # four chunks (= L for bands of 4), a second tile of 1
]


def _srows_raw_ker_ids():
    """Row-band instantiations that need no workspace (the raw-Ker form)."""
    w = inputs.BY_NAME["conv3x3_s2_b64"]
    out = set()
    for mode in ("bf16", "bf16_obf16"):
        for c in cnn.plan_candidates(cnn.problem(*w.dims()), MODES[mode], cnn.budget()):
            if c.kernel == cnn.K_SROWS and c.ws_bytes == 0:
                out.add(c.variant)
    return out


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
@pytest.mark.parametrize("shape", SROWS_SHAPES)
def test_srows_exact(shape, mode):
    """Every stride-2 row-band instantiation of the mode whose band divides
    Nw: bit-exact with the oracle on integer inputs.  In's element count is
    even and its last row's final load starts 2 bytes into a dword, so the
    last-element patch runs."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = shape
    rng = np.random.default_rng(sum(shape) + 29)
    Nx, Ny = 2 * (Nw - 1) + Nr, 2 * (Nh - 1) + Ns
    In = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nb, Nc, Nx, Ny)).astype(np.float32))
    Ker = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nk, Nc, Nr, Ns)).astype(np.float32))
    want = oracle.conv(In, Ker, 2, 2)
    if mode == "bf16_obf16":
        want = oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32)))
    dt = MODES[mode]
    ran = 0
    for v in cnn.variants():
        vid, L = v.variant, v.mode
        if v.kernel != cnn.K_SROWS or v.dtype != dt or (v.nr, v.ns) != (Nr, Ns) or Nw % L:
            continue
        pl = variant_plan(shape, dt, cnn.K_SROWS, 256, L * Nh, 16, vid)
        if pl is None and Nc < 16 * L and vid in _srows_raw_ker_ids():
            continue  # the raw-Ker form needs at least L chunks of 16 channels
        assert pl is not None and pl.variant == vid and pl.grid == Nb * (Nw // L) * -(-Nk // 256)
        say(f"[parity] srows shape={shape} v{vid} L={L} grid={pl.grid} mode={mode}")
        got = run(In, Ker, 2, 2, mode, plan=pl)
        assert np.array_equal(got, want), (vid, L)
        ran += 1
    assert ran > 0


def test_srows_float_strided_shape():
    """The strided 3x3 layer (64 images, 128 -> 256 channels, 28x28 outputs)
    on uniform inputs through every row-band instantiation that fits it:
    every output within the bf16 tolerance of the fp64 oracle."""
    w = inputs.BY_NAME["conv3x3_s2_b64"]
    In, Ker = inputs.make_inputs(w)
    want, absv = oracle.conv(In, Ker, 2, 2, with_abs=True)
    ran = 0
    for v in cnn.variants():
        if v.kernel != cnn.K_SROWS or v.dtype != cnn.CNN_BF16 or w.Nw % v.mode:
            continue
        pl = variant_plan(w.dims(), cnn.CNN_BF16, cnn.K_SROWS, 256, v.mode * w.Nh, 16, v.variant)
        say(f"[parity] srows strided v{pl.variant} tp={pl.tp} grid={pl.grid}")
        got = run(In, Ker, 2, 2, "bf16", plan=pl)
        nw, cond, _ = errors(got, want, absv)
        assert nw <= TOL["bf16"] and cond <= TOL["bf16"], (v.variant, nw, cond)
        ran += 1
    assert ran > 0


# ---- 1x1 GEMM kernel, strides 2 and 2: the even input rows and columns -----
GEMM1_S2_SHAPES = [
    (3, 72, 71, 6, 8, 1, 1, 2, 2),      # In 11x15 (odd rows: unaligned loads), two stages
    (2, 64, 300, 4, 4, 1, 1, 2, 2),     # two k tiles of 256, 16-pixel images
    (5, 40, 130, 7, 12, 1, 1, 2, 2),    # 84-pixel images, tiles span images
    (1, 256, 64, 28, 28, 1, 1, 2, 2),   # one 784-pixel image, In 55x55
    (2, 24, 40, 6, 4, 1, 1, 2, 2),      # Nc < one stage
]


@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
@pytest.mark.parametrize("shape", GEMM1_S2_SHAPES)
def test_gemm1_stride2_exact(shape, mode):
    """Every stride-2 1x1 GEMM instantiation of the mode, at its balanced
    tile and at the largest: bit-exact with the oracle on integer inputs
    (In's element count is even and its last element sits in the second
    half of a straddling dword in the last-row cases, so the patch runs)."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = shape
    rng = np.random.default_rng(sum(shape) + 13)
    Nx, Ny = 2 * Nw - 1, 2 * Nh - 1
    In = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nb, Nc, Nx, Ny)).astype(np.float32))
    Ker = inputs.f32_to_bf16_bits(rng.integers(-2, 3, size=(Nk, Nc, 1, 1)).astype(np.float32))
    want = oracle.conv(In, Ker, 2, 2)
    if mode == "bf16_obf16":
        want = oracle.widen(inputs.f32_to_bf16_bits(want.astype(np.float32)))
    dt = MODES[mode]
    ran = 0
    for v in cnn.variants():
        if v.kernel != cnn.K_GEMM1 or v.dtype != dt or v.mode != 1:
            continue
        vid, tk, tpmax, tc = v.variant, v.tk, v.tp, v.tc
        for cus in (256, 3):
            pl = cnn.plan_tiles(cnn.problem(*shape), dt, cnn.K_GEMM1, tk, tpmax, tc,
                                cnn.budget(cus, 160 * 1024, 128, 2))
            assert pl.variant == vid and pl.tp % 4 == 0
            say(f"[parity] gemm1 s2 shape={shape} v{vid} tp={pl.tp} grid={pl.grid} mode={mode}")
            got = run(In, Ker, 2, 2, mode, plan=pl)
            assert np.array_equal(got, want), (vid, pl.tp)
            ran += 1
    assert ran > 0


# ---- channel slices (CNN_K_SPLITC, Case 2 of Sec. 2.1) --------------------
SPLITC_CASES = [
    ((1, 16, 16, 16, 16, 3, 3, 1, 1), "f32", 64, 64, 8),         # the tiny workload: 2 stages
    ((1, 70, 40, 7, 7, 3, 3, 1, 1), "bf16", 64, 64, 32),         # 3 stages, the last ragged
    ((2, 200, 48, 6, 5, 3, 2, 2, 1), "bf16_obf16", 64, 64, 32),  # 7 stages, strides (2, 1)
    ((1, 37, 20, 9, 4, 1, 1, 1, 1), "f32", 64, 64, 8),           # 1x1, ragged channel tail
    ((3, 45, 150, 5, 6, 3, 3, 1, 1), "bf16", 128, 256, 16),      # two k tiles, the second ragged
    ((1, 300, 20, 4, 4, 3, 3, 1, 1), "f32", 64, 64, 8),          # 38 stages: kc 37 and 38
]


def _splitc_kcs(Nc, tc, kc_plan):
    stages = -(-Nc // tc)
    return sorted({1, 2, stages - 1, stages, kc_plan} & set(range(1, stages + 1)))


@pytest.mark.parametrize("case", SPLITC_CASES)
def test_splitc_exact(case):
    """Channel slices: bit-exact with the oracle on integer inputs for kc =
    1, 2, stages - 1 (some slices empty), stages and the plan's own kc.
    Integer partial sums are exact in fp32, so the slice order cannot show."""
    dims, mode, tk, tp, tc = case
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = dims
    In, Ker = _arrays(dims, mode, seed=sum(dims) + 31, dist=("int", -3, 3), kdist=("int", -3, 3))
    want = oracle.conv(In, Ker, sw, sh)
    if mode == "bf16_obf16":
        want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(want.astype(np.float32))).astype(np.float64)
    pl = cnn.plan_tiles(cnn.problem(*dims), MODES[mode], cnn.K_SPLITC, tk, tp, tc)
    assert pl.kernel == cnn.K_SPLITC
    for kc in _splitc_kcs(Nc, tc, pl.kc):
        pl.kc, pl.ws_bytes = kc, 4 * kc * Nb * Nk * Nw * Nh
        say(f"[parity] splitc dims={dims} mode={mode} v{pl.variant} grid={pl.grid} kc={kc}")
        got = run(In, Ker, sw, sh, mode, plan=pl)
        assert np.array_equal(got, want), kc


# channel-slice kernel (tk 32, tp 64, tc 32): Nc % 16 == 0; the cases span a
# ragged 16-channel last stage, ragged Nk, tiles across images, strides,
# 1x1, several stages per slice and empty slices
CSLICE_CASES = [
    (1, 512, 512, 7, 7, 3, 3, 1, 1),   # the batch-1 deep layer
    (1, 48, 39, 7, 7, 3, 3, 1, 1),     # stages of 32 and 16 channels, 39 features
    (2, 96, 45, 5, 9, 3, 3, 2, 1),     # strides (2, 1), tiles across two images
    (3, 80, 70, 6, 7, 3, 3, 1, 2),     # strides (1, 2), three k tiles
    (4, 256, 100, 5, 5, 3, 3, 2, 2),   # stride 2, two p tiles over four images
    (2, 64, 33, 9, 13, 1, 1, 1, 1),    # 1x1
]


@pytest.mark.parametrize("dims,tc", [(d, tc) for tc in (32, 16, 64) for d in CSLICE_CASES
                                     if tc == 32 or d[5] == 3])
@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
def test_cslice_exact(dims, tc, mode):
    """Channel-slice kernel (stages of 32, 16 or 64 channels): bit-exact with the
    oracle on integer inputs for kc = 1, 2, stages - 1, stages and the plan's
    own kc (integer partial sums are exact in fp32)."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = dims
    In, Ker = _arrays(dims, mode, seed=sum(dims) + 57, dist=("int", -3, 3), kdist=("int", -3, 3))
    want = oracle.conv(In, Ker, sw, sh)
    if mode == "bf16_obf16":
        want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(want.astype(np.float32))).astype(np.float64)
    pl = cnn.plan_tiles(cnn.problem(*dims), MODES[mode], cnn.K_SPLITC, 32, 64, tc)
    assert pl.kernel == cnn.K_SPLITC and 2500 <= pl.variant <= 2507
    for kc in _splitc_kcs(Nc, tc, pl.kc):
        pl.kc, pl.ws_bytes = kc, 4 * kc * Nb * Nk * Nw * Nh
        say(f"[parity] cslice dims={dims} mode={mode} v{pl.variant} grid={pl.grid} kc={kc}")
        got = run(In, Ker, sw, sh, mode, plan=pl)
        assert np.array_equal(got, want), kc


@pytest.mark.parametrize("dims", [d for d in CSLICE_CASES if d[5] == 3])
@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
def test_cslice_direct_exact(dims, mode):
    """Direct channel-slice form (one slice of 128-channel stages, 1024
    threads, Out written by the slice itself, no workspace): bit-exact with
    the oracle on integer inputs, ragged last stages (Nc = 48, 80, 96)
    included; a slice count other than 1 is refused before HIP."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = dims
    In, Ker = _arrays(dims, mode, seed=sum(dims) + 13, dist=("int", -3, 3), kdist=("int", -3, 3))
    want = oracle.conv(In, Ker, sw, sh)
    if mode == "bf16_obf16":
        want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(want.astype(np.float32))).astype(np.float64)
    pl = cnn.plan_tiles(cnn.problem(*dims), MODES[mode], cnn.K_SPLITC, 32, 64, 128)
    assert pl.variant in (2510, 2511) and pl.kc == 1 and pl.ws_bytes == 0
    say(f"[parity] cslice direct dims={dims} mode={mode} v{pl.variant} grid={pl.grid}")
    got = run(In, Ker, sw, sh, mode, plan=pl)
    assert np.array_equal(got, want)
    if -(-Nc // 128) > 1:
        q = cnn.Plan.from_buffer_copy(pl)
        q.kc = 2
        with pytest.raises(cnn.CnnError):
            run(In, Ker, sw, sh, mode, plan=q)


def test_cslice_direct_is_the_workspace_free_bf16_out_late_layer_plan():
    """cnn_fwd's plan for the batch-1 deep layer with bf16 Out (no fp32
    atomic target) is the direct channel-slice form, within the bf16-Out
    tolerance of the fp64 oracle."""
    w = inputs.BY_NAME["late3x3_b1"]
    In, Ker = inputs.make_inputs(w)
    pl = cnn.plan_tiles(cnn.problem(*w.dims()), cnn.CNN_BF16_OBF16, cnn.K_AUTO_NO_WORKSPACE)
    assert pl.kernel == cnn.K_SPLITC and pl.variant == 2511 and pl.ws_bytes == 0
    say("[parity] cnn_fwd late3x3_b1 bf16 Out (direct channel slices)")
    got = run(In, Ker, 1, 1, "bf16_obf16", plan=pl)
    want, absv = oracle.conv(In, Ker, 1, 1, with_abs=True)
    nw, cond, _ = errors(got, want, absv)
    assert nw < TOL["bf16_obf16"] and cond < TOL["bf16_obf16"], (nw, cond)


@pytest.mark.parametrize("dims", CSLICE_CASES)
def test_cslice_atomic_exact(dims):
    """Workspace-free channel slices (atomic adds into a zeroed fp32 Out):
    bit-exact with the oracle on integer inputs, whose sums are exact in any
    order, for kc = 1, 2, stages - 1, stages and the plan's own kc; every
    call overwrites Out (a NaN fill first)."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = dims
    In, Ker = _arrays(dims, "bf16", seed=sum(dims) + 91, dist=("int", -3, 3), kdist=("int", -3, 3))
    want = oracle.conv(In, Ker, sw, sh)
    vid = 2508 if Nr == 3 else 2509
    pl = variant_plan(dims, cnn.CNN_BF16, cnn.K_SPLITC, 32, 64, 32, vid)
    assert pl is not None and pl.variant == vid and pl.ws_bytes == 0
    for kc in _splitc_kcs(Nc, 32, pl.kc):
        pl.kc = kc
        say(f"[parity] cslice atomic dims={dims} v{vid} grid={pl.grid} kc={kc}")
        got = run(In, Ker, sw, sh, "bf16", plan=pl)
        assert np.array_equal(got, want), kc


def test_cslice_atomic_in_graph():
    """The atomic-sum channel split (zero fill, then atomic adds into Out)
    captured into a HIP graph and replayed several times, with eager work
    and a NaN fill of Out between replays: every replay equals the oracle
    exactly on integer inputs (exact in any summation order)."""
    import torch
    dims = (1, 96, 70, 7, 7, 3, 3, 1, 1)
    In, Ker = _arrays(dims, "bf16", seed=123, dist=("int", -3, 3), kdist=("int", -3, 3))
    want = oracle.conv(In, Ker, 1, 1)
    pl = variant_plan(dims, cnn.CNN_BF16, cnn.K_SPLITC, 32, 64, 32, 2508)
    assert pl is not None and pl.ws_bytes == 0 and pl.kc > 1
    dIn, dKer = to_gpu(In), to_gpu(Ker)
    out = out_tensor(1, 70, 7, 7, "bf16")
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    say(f"[parity] cslice atomic graph capture kc={pl.kc}")
    with torch.cuda.graph(g, stream=s):
        cnn.fwd_plan(dIn, dKer, out, pl)
    for i in range(4):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        say(f"[parity] cslice atomic graph replay {i}")
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(to_host64(out), want), i


# batch-1 deep layers beyond the benchmark workloads (1x1 2048 -> 512 and
# 512 -> 2048, 1x1 at 14x14, 3x3 at 14x14, 3x3 at batch 2): the model's plan
# (channel slices with a workspace) and cnn_fwd's workspace-free plan
DEEP_B1 = [(1, 2048, 512, 7, 7, 1, 1, 1, 1), (1, 512, 2048, 7, 7, 1, 1, 1, 1),
           (1, 1024, 256, 14, 14, 1, 1, 1, 1), (1, 256, 256, 14, 14, 3, 3, 1, 1),
           (2, 512, 512, 7, 7, 3, 3, 1, 1)]


@pytest.mark.parametrize("dims", DEEP_B1)
@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
def test_batch1_deep_layers(dims, mode):
    """Every output of the model's plan and of cnn_fwd within the tolerance
    of the fp64 oracle on uniform inputs and He-normal Ker."""
    In, Ker = _arrays(dims, mode, seed=sum(dims) + 3)
    want, absv = oracle.conv(In, Ker, dims[7], dims[8], with_abs=True)
    pl = cnn.plan(cnn.problem(*dims), MODES[mode])
    for tag, plan in (("model", pl), ("cnn_fwd", None)):
        say(f"[parity] deep batch-1 dims={dims} mode={mode} {tag} "
            f"{'v%d kc=%d' % (pl.variant, pl.kc) if plan else ''}")
        got = run(In, Ker, dims[7], dims[8], mode, plan=plan)
        nw, cond, _ = errors(got, want, absv)
        assert nw < TOL[mode] and cond < TOL[mode], (tag, nw, cond)


def test_cslice_atomic_is_the_workspace_free_late_layer_plan():
    """cnn_fwd's plan for the batch-1 deep layer (no workspace) is the atomic
    channel-slice one, within the bf16 tolerance of the fp64 oracle."""
    w = inputs.BY_NAME["late3x3_b1"]
    In, Ker = inputs.make_inputs(w)
    pl = cnn.plan_tiles(cnn.problem(*w.dims()), cnn.CNN_BF16, cnn.K_AUTO_NO_WORKSPACE)
    assert pl.kernel == cnn.K_SPLITC and pl.variant == 2508 and pl.ws_bytes == 0
    say("[parity] cnn_fwd late3x3_b1 (atomic channel slices)")
    got = run(In, Ker, 1, 1, "bf16")
    want, absv = oracle.conv(In, Ker, 1, 1, with_abs=True)
    nw, cond, _ = errors(got, want, absv)
    assert nw < TOL["bf16"] and cond < TOL["bf16"], (nw, cond)


@pytest.mark.parametrize("tiles", [(64, 64, 32), (32, 64, 32), (32, 64, 16), (32, 64, 64)])
@pytest.mark.parametrize("mode", ["bf16", "bf16_obf16"])
def test_splitc_float_late_layer(mode, tiles):
    """The batch-1 deep layer (512 -> 512 channels, 7x7 outputs) on uniform
    inputs with its split plans (16 slices; the CNN_K_IGEMM tiles and the
    channel-slice kernel): every output within the bf16 tolerance of the
    fp64 oracle."""
    w = inputs.BY_NAME["late3x3_b1"]
    In, Ker = inputs.make_inputs(w)
    pl = cnn.plan_tiles(cnn.problem(*w.dims()), MODES[mode], cnn.K_SPLITC, *tiles)
    assert pl.kc > 1
    say(f"[parity] splitc late3x3_b1 mode={mode} v{pl.variant} grid={pl.grid} kc={pl.kc}")
    got = run(In, Ker, 1, 1, mode, plan=pl)
    want, absv = oracle.conv(In, Ker, 1, 1, with_abs=True)
    nw, cond, _ = errors(got, want, absv)
    assert nw < TOL[mode] and cond < TOL[mode], (nw, cond)


def test_splitc_caller_workspace_in_graph():
    """cnn_fwd_plan_ws with a caller workspace, captured into a HIP graph and
    replayed several times with eager work in between: every replay equals
    the eager result bit for bit (the reduction order is fixed)."""
    import torch
    dims = (1, 70, 40, 7, 7, 3, 3, 1, 1)
    In, Ker = _arrays(dims, "bf16", seed=77)
    pl = cnn.plan_tiles(cnn.problem(*dims), cnn.CNN_BF16, cnn.K_SPLITC, 64, 64, 32)
    dIn, dKer = to_gpu(In), to_gpu(Ker)
    ws = torch.empty(pl.ws_bytes // 4, dtype=torch.float32, device="cuda")
    ref = out_tensor(1, 40, 7, 7, "bf16")
    say(f"[parity] splitc eager kc={pl.kc}")
    cnn.fwd_plan_ws(dIn, dKer, ref, pl, ws)
    torch.cuda.synchronize()
    out = out_tensor(1, 40, 7, 7, "bf16")
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    say("[parity] splitc graph capture")
    with torch.cuda.graph(g, stream=s):
        cnn.fwd_plan_ws(dIn, dKer, out, pl, ws)
    for i in range(4):
        out.fill_(float("nan"))
        ws.fill_(float("nan"))
        torch.cuda.synchronize()
        say(f"[parity] splitc graph replay {i}")
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), i
    want = oracle.conv(In, Ker, 1, 1)
    assert np.abs(to_host64(ref) - want).max() <= TOL["bf16"] * np.abs(want).max()

"""Pins of the fp64 convolution oracle against facts fixed outside it.

Each check uses a route to the answer that does not go through the oracle's
loop nest: a library convolution, a library matrix product, array slicing,
closed forms, or exact integer arithmetic.  Shapes are chosen so that a
swapped r/s, a stride applied to the wrong axis, a transposed Ker index, a
dropped channel or a sign error fails at least one test.
"""
import itertools

import numpy as np
import pytest
import torch
import scipy.signal

import oracle
from paper_2105_13480_amd import inputs


def _rand(shape, rng, kind="float"):
    if kind == "int":
        return rng.integers(-3, 4, size=shape).astype(np.float64)
    return rng.uniform(-1.0, 1.0, size=shape)


def _shape_cases():
    # (Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh): asymmetric on purpose
    return [
        (1, 1, 1, 1, 1, 1, 1, 1, 1),
        (2, 3, 4, 5, 6, 3, 2, 1, 1),
        (1, 2, 3, 4, 3, 2, 3, 2, 1),
        (3, 2, 1, 3, 4, 3, 3, 1, 2),
        (2, 4, 3, 3, 2, 5, 3, 3, 2),
        (1, 3, 2, 2, 5, 1, 1, 2, 3),
        (2, 5, 6, 4, 4, 3, 3, 2, 2),
        (1, 1, 2, 7, 1, 2, 1, 1, 1),
        (1, 2, 2, 1, 7, 1, 4, 1, 3),
    ]


def _dims_of(case):
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = case
    return Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, sw * (Nw - 1) + Nr, sh * (Nh - 1) + Ns


@pytest.mark.parametrize("case", _shape_cases())
@pytest.mark.parametrize("kind", ["float", "int"])
def test_matches_torch_conv2d(case, kind):
    """Library pin: torch CPU conv2d in float64 computes the same
    cross-correlation (no kernel flip, no padding, strides per axis)."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny = _dims_of(case)
    rng = np.random.default_rng(hash(case) % 2**32)
    In = _rand((Nb, Nc, Nx, Ny), rng, kind)
    Ker = _rand((Nk, Nc, Nr, Ns), rng, kind)
    got = oracle.conv(In, Ker, sw, sh)
    ref = torch.nn.functional.conv2d(torch.from_numpy(In), torch.from_numpy(Ker),
                                     stride=(sw, sh)).numpy()
    assert got.shape == (Nb, Nk, Nw, Nh)
    if kind == "int":
        assert np.array_equal(got, ref)
    else:
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", _shape_cases()[1:6])
def test_matches_scipy_correlate(case):
    """Library pin: per-channel scipy 2-D correlation ('valid'), summed over
    c, then subsampled by the strides."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny = _dims_of(case)
    rng = np.random.default_rng(7)
    In = _rand((Nb, Nc, Nx, Ny), rng, "int")
    Ker = _rand((Nk, Nc, Nr, Ns), rng, "int")
    got = oracle.conv(In, Ker, sw, sh)
    for b in range(Nb):
        for k in range(Nk):
            full = sum(scipy.signal.correlate2d(In[b, c], Ker[k, c], mode="valid")
                       for c in range(Nc))
            assert np.array_equal(got[b, k], full[::sw, ::sh])


def test_brute_force_int_python():
    """Brute force on tiny integer inputs in Python int arithmetic via an
    explicit im2col matrix (rows = output pixels, columns = (c, r, s))."""
    rng = np.random.default_rng(11)
    grid = list(itertools.product([1, 2, 3], [1, 2, 3, 5], [1, 2, 3, 5], [1, 2], [1, 3],
                                  [1, 2, 4], [1, 2, 4], [1, 2, 3]))
    picks = rng.choice(len(grid), size=60, replace=False)
    for gi in picks:
        sw_, Nr, Ns, Nb, Nc, Nw, Nh, sh_ = grid[gi]
        Nk = 1 + (gi % 3)
        Nx, Ny = sw_ * (Nw - 1) + Nr, sh_ * (Nh - 1) + Ns
        In = rng.integers(-3, 4, size=(Nb, Nc, Nx, Ny))
        Ker = rng.integers(-3, 4, size=(Nk, Nc, Nr, Ns))
        cols = [(c, r, s) for c in range(Nc) for r in range(Nr) for s in range(Ns)]
        kmat = [[int(Ker[k, c, r, s]) for (c, r, s) in cols] for k in range(Nk)]
        got = oracle.conv(In.astype(np.float64), Ker.astype(np.float64), sw_, sh_)
        for b in range(Nb):
            for w in range(Nw):
                for h in range(Nh):
                    row = [int(In[b, c, sw_ * w + r, sh_ * h + s]) for (c, r, s) in cols]
                    for k in range(Nk):
                        want = sum(a * x for a, x in zip(row, kmat[k]))
                        assert got[b, k, w, h] == want


@pytest.mark.parametrize("sw,sh", [(1, 1), (2, 2), (1, 3), (3, 1)])
def test_pointwise_is_matmul(sw, sh):
    """Identity: a 1x1 kernel is a matrix product on the subsampled input."""
    Nb, Nc, Nk, Nw, Nh = 3, 7, 5, 4, 6
    rng = np.random.default_rng(3)
    In = rng.standard_normal((Nb, Nc, sw * (Nw - 1) + 1, sh * (Nh - 1) + 1))
    Ker = rng.standard_normal((Nk, Nc, 1, 1))
    got = oracle.conv(In, Ker, sw, sh)
    sub = In[:, :, ::sw, ::sh].reshape(Nb, Nc, Nw * Nh)
    ref = np.matmul(Ker[:, :, 0, 0], sub).reshape(Nb, Nk, Nw, Nh)
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)
    Ii = rng.integers(-5, 6, size=In.shape).astype(np.float64)
    Ki = rng.integers(-5, 6, size=Ker.shape).astype(np.float64)
    subi = Ii[:, :, ::sw, ::sh].reshape(Nb, Nc, Nw * Nh)
    refi = np.matmul(Ki[:, :, 0, 0], subi).reshape(Nb, Nk, Nw, Nh)
    assert np.array_equal(oracle.conv(Ii, Ki, sw, sh), refi)


@pytest.mark.parametrize("Nr,Ns,sw,sh", [(3, 3, 1, 1), (3, 2, 2, 1), (5, 3, 2, 3), (1, 4, 1, 2)])
def test_delta_kernel_is_strided_copy(Nr, Ns, sw, sh):
    """Identity: Ker = [c == k mod Nc][r == r0][s == s0] copies
    In[b, k mod Nc, sw*w + r0, sh*h + s0] exactly, for arbitrary floats."""
    Nb, Nc, Nk, Nw, Nh = 2, 3, 5, 4, 5
    Nx, Ny = sw * (Nw - 1) + Nr, sh * (Nh - 1) + Ns
    rng = np.random.default_rng(5)
    In = rng.standard_normal((Nb, Nc, Nx, Ny)).astype(np.float32)
    for r0 in range(Nr):
        for s0 in range(Ns):
            Ker = np.zeros((Nk, Nc, Nr, Ns), dtype=np.float32)
            for k in range(Nk):
                Ker[k, k % Nc, r0, s0] = 1.0
            got = oracle.conv(In, Ker, sw, sh)
            for k in range(Nk):
                want = In[:, k % Nc, r0::sw, s0::sh][:, :Nw, :Nh].astype(np.float64)
                assert np.array_equal(got[:, k], want)


def test_all_ones_closed_form():
    """Closed form: all-ones In and Ker give Nc*Nr*Ns everywhere."""
    for (Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh) in [(2, 3, 4, 5, 6, 3, 2, 1, 2), (1, 16, 16, 16, 16, 3, 3, 1, 1)]:
        In = np.ones((Nb, Nc, sw * (Nw - 1) + Nr, sh * (Nh - 1) + Ns))
        Ker = np.ones((Nk, Nc, Nr, Ns))
        assert np.all(oracle.conv(In, Ker, sw, sh) == Nc * Nr * Ns)


def test_checksum_identity():
    """sum_{b,k,w,h} Out = sum_{c,r,s} (sum_k Ker[k,c,r,s]) *
    (sum_{b,w,h} In[b,c,sw*w+r,sh*h+s]), the right side by slicing."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh = 3, 4, 5, 6, 7, 3, 2, 2, 1
    rng = np.random.default_rng(9)
    In = rng.integers(-4, 5, size=(Nb, Nc, sw * (Nw - 1) + Nr, sh * (Nh - 1) + Ns)).astype(np.float64)
    Ker = rng.integers(-4, 5, size=(Nk, Nc, Nr, Ns)).astype(np.float64)
    lhs = oracle.conv(In, Ker, sw, sh).sum()
    ksum = Ker.sum(axis=0)
    rhs = 0.0
    for c in range(Nc):
        for r in range(Nr):
            for s in range(Ns):
                rhs += ksum[c, r, s] * In[:, c, r::sw, s::sh][:, :Nw, :Nh].sum()
    assert lhs == rhs


def test_linearity_exact():
    """Out is linear in In and in Ker (exact on integers)."""
    case = (2, 3, 4, 5, 4, 3, 3, 2, 1)
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny = _dims_of(case)
    rng = np.random.default_rng(13)
    I1, I2 = (rng.integers(-3, 4, size=(Nb, Nc, Nx, Ny)).astype(np.float64) for _ in range(2))
    K1, K2 = (rng.integers(-3, 4, size=(Nk, Nc, Nr, Ns)).astype(np.float64) for _ in range(2))
    assert np.array_equal(oracle.conv(I1 + 2 * I2, K1, sw, sh),
                          oracle.conv(I1, K1, sw, sh) + 2 * oracle.conv(I2, K1, sw, sh))
    assert np.array_equal(oracle.conv(I1, K1 - 3 * K2, sw, sh),
                          oracle.conv(I1, K1, sw, sh) - 3 * oracle.conv(I1, K2, sw, sh))


def test_abs_sum():
    """Abs = sum |In*Ker|: equals Out when every product is >= 0, equals
    -Out when every product is <= 0, and bounds |Out| always."""
    case = (2, 3, 4, 5, 4, 3, 2, 1, 2)
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny = _dims_of(case)
    rng = np.random.default_rng(17)
    In = rng.uniform(0, 1, size=(Nb, Nc, Nx, Ny))
    Ker = rng.uniform(0, 1, size=(Nk, Nc, Nr, Ns))
    out, ab = oracle.conv(In, Ker, sw, sh, with_abs=True)
    np.testing.assert_allclose(ab, out, rtol=1e-15)
    out, ab = oracle.conv(In, -Ker, sw, sh, with_abs=True)
    np.testing.assert_allclose(ab, -out, rtol=1e-15)
    In2 = rng.uniform(-1, 1, size=In.shape)
    out, ab = oracle.conv(In2, Ker - 0.5, sw, sh, with_abs=True)
    assert np.all(ab >= np.abs(out))
    ref_abs = torch.nn.functional.conv2d(torch.from_numpy(np.abs(In2)),
                                         torch.from_numpy(np.abs(Ker - 0.5)),
                                         stride=(sw, sh)).numpy()
    np.testing.assert_allclose(ab, ref_abs, rtol=1e-12)


def test_points_match_full():
    case = (2, 3, 4, 6, 5, 3, 3, 2, 1)
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny = _dims_of(case)
    rng = np.random.default_rng(19)
    In = rng.standard_normal((Nb, Nc, Nx, Ny))
    Ker = rng.standard_normal((Nk, Nc, Nr, Ns))
    full, fabs_ = oracle.conv(In, Ker, sw, sh, with_abs=True)
    idx = np.stack([rng.integers(0, n, size=50) for n in (Nb, Nk, Nw, Nh)], axis=1)
    pts, pabs = oracle.conv_points(In, Ker, idx, sw, sh, with_abs=True)
    for i, (b, k, w, h) in enumerate(idx):
        assert pts[i] == full[b, k, w, h]
        assert pabs[i] == fabs_[b, k, w, h]


def test_bf16_inputs_widen_exactly():
    """bf16 bit patterns are read as the top half of a float32."""
    vals = np.array([1.0, -2.5, 0.0078125, 3.0e38, -1.0e-30], dtype=np.float32)
    bits = inputs.f32_to_bf16_bits(vals)
    back = oracle.widen(bits)
    assert np.array_equal(back, inputs.bf16_bits_to_f32(bits).astype(np.float64))
    assert back[0] == 1.0 and back[1] == -2.5 and back[2] == 0.0078125


def test_bad_extent_rejected():
    with pytest.raises(ValueError):
        oracle.conv(np.zeros((1, 1, 4, 4)), np.zeros((1, 1, 3, 3)), 2, 2)
    with pytest.raises(ValueError):
        oracle.conv(np.zeros((1, 2, 4, 4)), np.zeros((1, 1, 3, 3)), 1, 1)
    with pytest.raises(ValueError):
        oracle.conv_points(np.zeros((1, 1, 4, 4)), np.zeros((1, 1, 3, 3)),
                           np.array([[0, 0, 2, 0]]), 1, 1)


@pytest.mark.parametrize("case", _shape_cases())
def test_library_route_matches_loop_nest(case):
    """conv_lib (a library convolution, used for every output of the
    full-size workloads) equals the loop nest output by output, Abs too."""
    Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny = _dims_of(case)
    rng = np.random.default_rng(7 + hash(case) % 2**31)
    In = _rand((Nb, Nc, Nx, Ny), rng, "int")
    Ker = _rand((Nk, Nc, Nr, Ns), rng, "int")
    got, got_abs = oracle.conv_lib(In, Ker, sw, sh, with_abs=True)
    want, want_abs = oracle.conv(In, Ker, sw, sh, with_abs=True)
    assert np.array_equal(got, want) and np.array_equal(got_abs, want_abs)


@pytest.mark.parametrize("name", [w.name for w in inputs.WORKLOADS])
def test_library_route_at_full_size(name):
    """At every benchmark workload's full size, conv_lib agrees with the loop
    nest's single-point route on a sample of outputs (corners included) to
    fp64 rounding of sum |In * Ker|."""
    w = inputs.BY_NAME[name]
    In, Ker = inputs.make_inputs(w)
    got, got_abs = oracle.conv_lib(In, Ker, w.sw, w.sh, with_abs=True)
    rng = np.random.default_rng(11)
    idx = np.stack([rng.integers(0, m, size=300) for m in (w.Nb, w.Nk, w.Nw, w.Nh)], axis=1)
    corners = np.array(list(itertools.product((0, w.Nb - 1), (0, w.Nk - 1),
                                              (0, w.Nw - 1), (0, w.Nh - 1))))
    idx = np.concatenate([idx, corners])
    want, want_abs = oracle.conv_points(In, Ker, idx, w.sw, w.sh, with_abs=True)
    sel = (idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3])
    assert np.all(np.abs(got[sel] - want) <= 1e-13 * want_abs)
    assert np.allclose(got_abs[sel], want_abs, rtol=1e-13, atol=0)

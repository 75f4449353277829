"""C ABI checks that need no GPU: the library loads, exports every symbol
include/cnn.h declares, rejects bad arguments before any HIP call, its
host-side model (Eq. (1), composite-tile costs, the closed form) equals the
oracle's, and the plans the selector makes are pinned by facts of the paper:
their Eq. (1) terms count the loads of Listing 3's point loops, and no plan
moves less than the Table 1 lower bound."""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

from oracle import eq1 as oeq1
from paper_2105_13480_amd import cnn, inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "cnn.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(cnn_\w+)\(", text, re.M)))


def test_header_and_binding_agree():
    assert _declared_functions() == sorted(cnn.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = cnn.lib()
    for name in _declared_functions():
        assert hasattr(L, name), name
    assert L.cnn_abi_version() == 2


def test_strerror_covers_all_codes():
    L = cnn.lib()
    for code in cnn.STATUS:
        assert L.cnn_strerror(code)
    assert L.cnn_strerror(12345) == b"unknown status"


DIMS = (2, 3, 4, 5, 6, 3, 3, 1, 1)


def _fwd(ptrs=(0x1000, 0x100000, 0x200000), dims=DIMS, dtype=cnn.CNN_F32):
    return cnn.lib().cnn_fwd(*ptrs, *dims, dtype, None)


def test_null_pointers_rejected():
    assert _fwd(ptrs=(0, 0x100000, 0x200000)) == -1
    assert _fwd(ptrs=(0x1000, 0, 0x200000)) == -1
    assert _fwd(ptrs=(0x1000, 0x100000, 0)) == -1
    assert b"non-NULL" in cnn.lib().cnn_last_error()


@pytest.mark.parametrize("i", range(9))
def test_sizes_below_one_rejected(i):
    dims = list(DIMS)
    dims[i] = 0
    assert _fwd(dims=tuple(dims)) == -2
    dims[i] = -3
    assert _fwd(dims=tuple(dims)) == -2


def test_bad_dtype_rejected():
    assert _fwd(dtype=7) == -3
    assert _fwd(dtype=-1) == -3


def test_overflow_rejected():
    assert _fwd(dims=(1 << 20, 1, 1, 1 << 10, 1 << 10, 1, 1, 1, 1)) == -4
    assert _fwd(dims=(1, 1, 1, 1, 1, 1 << 31, 1, 1, 1)) == -4
    assert _fwd(dims=(1, 1, 1, 1 << 20, 1, 1, 1, 1 << 12, 1)) == -4


def test_alias_rejected():
    # Out = [0x200000, +2*4*5*6*4 bytes); In covers 2*3*7*8*4 bytes from its base
    assert _fwd(ptrs=(0x200000 - 8, 0x100000, 0x200000)) == -5
    assert _fwd(ptrs=(0x1000, 0x200000 + 16, 0x200000)) == -5
    assert b"overlaps" in cnn.lib().cnn_last_error()


def test_fwd_plan_rejects_foreign_plan():
    p = cnn.problem(*DIMS)
    pl = cnn.plan(p, cnn.CNN_F32, cnn.budget())
    q = cnn.problem(2, 3, 4, 5, 6, 3, 3, 1, 2)
    st = cnn.lib().cnn_fwd_plan(0x1000, 0x100000, 0x200000, ctypes.byref(q), cnn.CNN_F32,
                                ctypes.byref(pl), None)
    assert st == -8
    st = cnn.lib().cnn_fwd_plan(0x1000, 0x100000, 0x200000, ctypes.byref(p), cnn.CNN_BF16,
                                ctypes.byref(pl), None)
    assert st == -8


def test_plan_tiles_unknown_tiling_unsupported():
    p = cnn.problem(*DIMS)
    with pytest.raises(cnn.CnnError) as e:
        cnn.plan_tiles(p, cnn.CNN_F32, cnn.K_IGEMM, 64, 96, 8, cnn.budget())
    assert e.value.status == -6


def _problems():
    rng = np.random.default_rng(21)
    out = [oeq1.Problem(*w.dims()) for w in inputs.WORKLOADS]
    for _ in range(25):
        Nr, Ns = rng.integers(1, 6, size=2)
        out.append(oeq1.Problem(int(rng.integers(1, 5)), int(rng.integers(1, 40)),
                                int(rng.integers(1, 300)), int(rng.integers(1, 30)),
                                int(rng.integers(1, 30)), int(Nr), int(Ns),
                                int(rng.integers(1, 4)), int(rng.integers(1, 4))))
    return out


@pytest.mark.parametrize("halo", [0, 1])
def test_eq1_matches_oracle(halo):
    rng = np.random.default_rng(5)
    for p in _problems():
        for _ in range(4):
            t = oeq1.Tiles(*(int(rng.integers(1, n + 1)) for n in (p.Nb, p.Nk, p.Nc, p.Nw, p.Nh)))
            terms, fp = cnn.eq1_cost(cnn.problem(*p.__dict__.values()), cnn.Tiles(*t.__dict__.values()), halo)
            want = oeq1.eq1_terms(p, t, "exact" if halo else "paper")
            wfp = oeq1.eq1_footprint(p, t, "exact" if halo else "paper")
            if halo:
                assert terms == tuple(float(x) for x in want) and fp == wfp
            else:
                np.testing.assert_allclose(terms, want, rtol=1e-13)
                np.testing.assert_allclose(fp, wfp, rtol=1e-13)


def test_slab_cost_matches_oracle():
    for p in _problems():
        for tk, tp in [(32, 32), (64, 256), (256, 128), (7, 50)]:
            got = cnn.slab_cost(cnn.problem(*p.__dict__.values()), tk, tp)
            assert got == tuple(float(x) for x in oeq1.slab_terms(p, tk, tp))


BUDGETS = [(256, 160 * 1024, 128, 2), (64, 64 * 1024, 64, 1), (8, 160 * 1024, 128, 2)]


def _key(pl):
    return (pl.kernel, pl.variant, pl.tk, pl.tp, pl.tc, pl.kc)


def _better(a, b):
    """The selector's documented order: less model time; within 2 % of each
    other, fewer predicted HBM bytes, then fewer Eq. (1) bytes, then the
    lower instantiation id, then the larger tile."""
    lo = min(a.model_us, b.model_us)
    if abs(a.model_us - b.model_us) > 0.02 * lo:
        return a.model_us < b.model_us
    for x, y in ((a.hbm_bytes, b.hbm_bytes), (a.eq1_bytes, b.eq1_bytes), (a.variant, b.variant)):
        if x != y:
            return x < y
    return a.tp > b.tp


@pytest.mark.parametrize("dtype", [0, 1, 2])
def test_plan_is_the_model_minimum(dtype):
    """cnn_plan's choice is a candidate of cnn_plan_candidates and no
    candidate comes before it in the model's order; the choice among the
    candidates that need no workspace (what cnn_fwd runs) likewise among
    those."""
    for p in _problems():
        prob = cnn.problem(*p.__dict__.values())
        for bud in BUDGETS:
            cands = cnn.plan_candidates(prob, dtype, cnn.budget(*bud))
            free = [c for c in cands if c.ws_bytes == 0]
            pl = cnn.plan(prob, dtype, cnn.budget(*bud))
            assert _key(pl) in {_key(c) for c in cands}, (p, bud)
            assert pl.model_us <= 1.02 * min(c.model_us for c in cands)
            assert not any(_better(c, pl) for c in cands if _key(c) != _key(pl)), (p, bud)
            pf = cnn.plan_tiles(prob, dtype, cnn.K_AUTO_NO_WORKSPACE, bud=cnn.budget(*bud))
            assert pf.ws_bytes == 0
            if not free:
                assert pf.kernel == cnn.K_DIRECT
                continue
            assert _key(pf) in {_key(c) for c in free}, (p, bud)
            assert not any(_better(c, pf) for c in free if _key(c) != _key(pf)), (p, bud)


def test_model_time_is_at_least_the_hbm_floor():
    """Every candidate's predicted time is at least its HBM bytes (Eq. (3)
    at the XCD level) at the bandwidth of their read/write mix -- a device
    copy's 5.0 TB/s for half writes or fewer, rising linearly with the write
    share to a fill's 6.9 TB/s -- plus the 2 us launch; the stem's traffic
    is write-dominated (its Out is nine tenths), so it takes the floor's
    upper end."""
    def floor_us(pl):
        out, ker, inp = cnn.hbm_bytes(pl)
        total = out + ker + inp
        w = out / total
        gbs = 5000.0 if w <= 0.5 else 5000.0 + (6900.0 - 5000.0) * (w - 0.5) / 0.5
        return total / (gbs * 1e3) + 2.0
    for w in inputs.WORKLOADS:
        prob = cnn.problem(*w.dims())
        for c in cnn.plan_candidates(prob, cnn.DTYPES["f32" if w.dtype == "f32" else "bf16"],
                                     cnn.budget()):
            if c.kernel in (cnn.K_DIRECT, cnn.K_SPLITC):
                continue  # direct plans price compulsory bytes; split plans add a reduce
            assert c.model_us >= floor_us(c) * (1 - 1e-9), (w.name, c.variant, c.model_us)
    stem = inputs.BY_NAME["stem7x7_s2_b64"]
    out, ker, inp = cnn.hbm_bytes(cnn.plan(cnn.problem(*stem.dims()), cnn.DTYPES["bf16"], cnn.budget()))
    assert out / (out + ker + inp) > 0.85


def test_candidates_are_complete_plans():
    for w in inputs.WORKLOADS:
        prob = cnn.problem(*w.dims())
        for dt in ((0,) if w.dtype == "f32" else (1, 2)):
            cands = cnn.plan_candidates(prob, dt, cnn.budget())
            assert cands
            for c in cands:
                assert c.kernel != cnn.K_AUTO and c.grid >= 1 and c.model_us > 0
                assert c.flops == w.flops and c.mfma_flops >= c.flops
                assert c.hbm_bytes >= 0.99 * c.compulsory_bytes
                if c.kernel != cnn.K_DIRECT:
                    assert c.hbm_bytes == pytest.approx(sum(cnn.hbm_bytes(c, 8, 4 << 20)))


def _composite_loads(p, tk, tp):
    """Loads of Listing 3 run over a composite tiling, counted literally:
    for every tile of tk features by tp consecutive outputs of the flattened
    (b, w, h) index, with all Nc channels (W_c = N_c), the set of In
    elements its point loops read, its Ker tile and its Out tile.  Returns
    (Out stores, Ker loads, In loads) in elements."""
    hw, npix = p.Nw * p.Nh, p.Nb * p.Nw * p.Nh
    out = ker = inn = 0
    for k0 in range(0, p.Nk, tk):
        kk = min(tk, p.Nk - k0)
        for f in range(0, npix, tp):
            outs = range(f, min(f + tp, npix))
            pos = set()
            for q in outs:
                b, w, h = q // hw, (q % hw) // p.Nh, q % p.Nh
                for r in range(p.Nr):
                    for s_ in range(p.Ns):
                        pos.add((b, p.sw * w + r, p.sh * h + s_))
            inn += len(pos) * p.Nc
            ker += kk * p.Nc * p.Nr * p.Ns
            out += kk * len(outs)
    return out, ker, inn


SMALL = [(2, 24, 70, 6, 8, 3, 3, 1, 1), (1, 16, 40, 8, 12, 3, 3, 2, 2),
         (3, 16, 33, 4, 6, 1, 1, 1, 1), (2, 8, 20, 5, 7, 5, 3, 2, 1),
         (2, 3, 64, 6, 6, 7, 7, 2, 2), (1, 48, 300, 4, 4, 1, 1, 2, 2)]


@pytest.mark.parametrize("dims", SMALL)
@pytest.mark.parametrize("dtype", [0, 1])
def test_candidate_eq1_terms_count_listing3_loads(dims, dtype):
    """Sec. 2, Eq. (1) on the plans themselves: for every candidate tiling,
    Out and Ker terms equal the literal counts of Listing 3's stores and
    loads at the plan's (tk, tp); the In term (whole staged input rows)
    covers every input element the tile's point loops read, and equals that
    count when the tiles are whole rows of one image (or whole images) and
    the stride does not skip input rows or columns."""
    P = oeq1.Problem(*dims)
    prob = cnn.problem(*dims)
    hw = P.Nw * P.Nh
    n = 0
    for c in cnn.plan_candidates(prob, dtype, cnn.budget()):
        if c.kernel == cnn.K_DIRECT:
            continue
        o, k, i = _composite_loads(P, c.tk, c.tp)
        assert (c.eq1_elems[0], c.eq1_elems[1]) == (o, k), (c.as_dict(), o, k)
        assert c.eq1_elems[2] >= i
        whole = (c.tp % P.Nh == 0 and hw % c.tp == 0) or c.tp % hw == 0
        if whole and P.sw <= P.Nr and P.sh <= P.Ns:
            assert c.eq1_elems[2] == i, c.as_dict()
        n += 1
    assert n > 0


def _table1_bound_cases():
    out = [(w.dims(), 0 if w.dtype == "f32" else 1) for w in inputs.WORKLOADS
           if w.sw <= w.Nr and w.sh <= w.Ns]
    rng = np.random.default_rng(12)
    while len(out) < len(inputs.WORKLOADS) + 20:
        Nr, Ns = (int(x) for x in rng.integers(1, 6, size=2))
        sw, sh = int(rng.integers(1, Nr + 1)), int(rng.integers(1, Ns + 1))
        dims = (int(rng.integers(1, 9)), int(rng.integers(1, 200)), int(rng.integers(1, 400)),
                int(rng.integers(1, 40)), int(rng.integers(1, 40)), Nr, Ns, sw, sh)
        out.append((dims, int(rng.integers(0, 3))))
    return out


@pytest.mark.parametrize("dims,dtype", _table1_bound_cases())
def test_candidate_eq1_at_least_the_table1_bound(dims, dtype):
    """Sec. 2.1: with M_L = M the Table 1 costs are lower bounds.  Every
    candidate plan, seen as P = min(grid, CUs) processors whose fast memory
    M (elements) is its LDS footprint plus its Out tile, moves at least P
    times the Table 1 cost in Eq. (1) elements.  (Checked where the stride
    does not exceed the stencil: the relaxation's In tile of sw*sh*T_bhw
    elements assumes every input row and column between reads is read.)"""
    P_ = oeq1.Problem(*dims)
    prob = cnn.problem(*dims)
    bud = cnn.budget()
    e_in = 4 if dtype == 0 else 2
    for c in cnn.plan_candidates(prob, dtype, bud):
        if c.kernel == cnn.K_DIRECT:
            continue
        P = min(c.grid, bud.cus)
        M = c.lds_bytes / e_in + c.tk * c.tp
        bound = P * oeq1.table1_cost(P_, P, M)
        assert sum(c.eq1_elems) >= bound * (1 - 1e-12), (c.as_dict(), bound)


def test_plan_reports_eq1_and_compulsory_bytes():
    w = inputs.BY_NAME["conv3x3_b32"]
    p = oeq1.Problem(*w.dims())
    pl = cnn.plan(cnn.problem(*w.dims()), cnn.CNN_BF16, cnn.budget())
    o, k, i = oeq1.slab_terms(p, pl.tk, pl.tp)
    assert tuple(pl.eq1_elems) == (o, k, i)
    assert pl.eq1_bytes == 4 * o + 2 * (k + i)
    comp = 2 * (w.Nb * w.Nc * w.Nx * w.Ny + w.Nk * w.Nc * 9) + 4 * w.Nb * w.Nk * w.Nw * w.Nh
    assert pl.compulsory_bytes == comp
    assert pl.flops == w.flops


def test_every_instantiation_has_a_fitting_test_shape():
    """The GPU variant test needs, for each instantiation, a problem it fits;
    check on the CPU that one exists."""
    import sys
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from gpu_helpers import variant_cases, variant_dims
    cases = variant_cases()
    assert len({c[1] for c in cases}) == len(cases)
    for case in cases:
        kernel, vid, dt, tk, tp, tc, stencils = case
        assert variant_dims(kernel, vid, dt, tk, tp, tc, stencils) is not None, vid


def test_plan_find_and_lookup_validate_before_hip():
    L = cnn.lib()
    p = cnn.problem(*DIMS)
    pl = cnn.Plan()
    assert L.cnn_plan_find(0x1000, 0x100000, 0x200000, None, cnn.CNN_F32, None,
                           ctypes.byref(pl), None) == -1
    assert L.cnn_plan_find(0, 0x100000, 0x200000, ctypes.byref(p), cnn.CNN_F32, None,
                           ctypes.byref(pl), None) == -1
    assert L.cnn_plan_find(0x1000, 0x100000, 0x200000, ctypes.byref(p), 9, None,
                           ctypes.byref(pl), None) == -3
    q = cnn.problem(2, 3, 4, 0, 6, 3, 3, 1, 1)
    assert L.cnn_plan_find(0x1000, 0x100000, 0x200000, ctypes.byref(q), cnn.CNN_F32, None,
                           ctypes.byref(pl), None) == -2
    assert L.cnn_plan_find(0x200000 - 8, 0x100000, 0x200000, ctypes.byref(p), cnn.CNN_F32,
                           None, ctypes.byref(pl), None) == -5
    assert L.cnn_plan_lookup(None, cnn.CNN_F32, ctypes.byref(pl)) == -1
    assert L.cnn_plan_lookup(ctypes.byref(p), 5, ctypes.byref(pl)) == -3
    assert L.cnn_plan_lookup(ctypes.byref(q), cnn.CNN_F32, ctypes.byref(pl)) == -2


SPLITC_PLANS = [((1, 16, 16, 16, 16, 3, 3, 1, 1), cnn.CNN_F32, 64, 64, 8),
                ((1, 224, 64, 64, 110, 1, 1, 1, 1), cnn.CNN_BF16, 64, 64, 32),  # 7 stages, grid 110
                ((1, 512, 512, 7, 7, 3, 3, 1, 1), cnn.CNN_BF16, 64, 64, 32),
                ((1, 512, 512, 7, 7, 3, 3, 1, 1), cnn.CNN_BF16_OBF16, 128, 128, 32),
                ((2, 200, 48, 6, 5, 3, 2, 2, 1), cnn.CNN_BF16, 64, 64, 32),
                ((64, 24, 16, 28, 28, 3, 3, 1, 1), cnn.CNN_F32, 64, 64, 8)]


@pytest.mark.parametrize("case", SPLITC_PLANS)
def test_splitc_plan_is_the_staging_tiling_split_over_channels(case):
    """CNN_K_SPLITC (Case 2 of Sec. 2.1, W_c < N_c): the CNN_K_IGEMM tiling
    with kc channel slices of ceil(stages/kc) stages, none empty; enough
    slices for two workgroups per CU unless every stage is its own slice,
    and no more; a workspace of kc fp32 partial Outs."""
    dims, dt, tk, tp, tc = case
    bud = cnn.budget()
    p = cnn.problem(*dims)
    base = cnn.plan_tiles(p, dt, cnn.K_IGEMM, tk, tp, tc, bud)
    sp = cnn.plan_tiles(p, dt, cnn.K_SPLITC, tk, tp, tc, bud)
    same = ("variant", "tk", "tp", "tc", "grid", "lds_bytes", "slab_rows")
    assert [getattr(sp, f) for f in same] == [getattr(base, f) for f in same]
    assert sp.kernel == cnn.K_SPLITC and base.kc == 0 and base.ws_bytes == 0
    Nb, Nc, Nk, Nw, Nh = dims[:5]
    stages = -(-Nc // tc)

    def nonempty(k):  # k slices of ceil(stages/k) stages: none empty
        return (k - 1) * -(-stages // k) < stages

    kc = sp.kc
    assert 1 <= kc <= stages and nonempty(kc)
    assert base.grid * kc >= 2 * bud.cus or kc == stages
    for k in range(1, kc):  # no smaller valid count is enough
        assert not (nonempty(k) and base.grid * k >= 2 * bud.cus), k
    assert sp.ws_bytes == 4 * kc * Nb * Nk * Nw * Nh


def test_splitc_bad_slice_count_rejected_before_hip():
    dims = (1, 16, 16, 16, 16, 3, 3, 1, 1)
    p = cnn.problem(*dims)
    pl = cnn.plan_tiles(p, cnn.CNN_F32, cnn.K_SPLITC, 64, 64, 8, cnn.budget())
    L = cnn.lib()
    nout = 16 * 16 * 16
    for kc, ws in [(0, 0), (3, 4 * 3 * nout), (2, 4 * 2 * nout - 4), (-1, 4 * nout)]:
        q = cnn.Plan.from_buffer_copy(pl)
        q.kc, q.ws_bytes = kc, ws
        st = L.cnn_fwd_plan_ws(0x1000, 0x100000, 0x200000, ctypes.byref(p), cnn.CNN_F32,
                               ctypes.byref(q), 0x4000000, 1 << 30, None)
        assert st == -8, (kc, ws)


def test_channel_slice_plans():
    """The channel-slice instantiations (CNN_K_SPLITC, tk 32, tp 64): on the
    batch-1 deep layer the workspace form keeps 16 fp32 partial Outs and is
    the model's plan; the atomic-sum form needs no workspace and is the
    workspace-free plan (the one cnn_fwd runs); a workspace size on the
    atomic form, or none on the ordered form, is refused before HIP."""
    bud = cnn.budget()
    p = cnn.problem(1, 512, 512, 7, 7, 3, 3, 1, 1)
    ws = cnn.plan(p, cnn.CNN_BF16, bud)
    assert (ws.kernel, ws.variant, ws.kc, ws.grid) == (cnn.K_SPLITC, 2500, 16, 16)
    assert ws.ws_bytes == 4 * 16 * 512 * 49
    free = cnn.plan_tiles(p, cnn.CNN_BF16, cnn.K_AUTO_NO_WORKSPACE, 0, 0, 0, bud)
    assert (free.kernel, free.variant, free.kc, free.ws_bytes) == (cnn.K_SPLITC, 2508, 16, 0)
    assert free.model_us > ws.model_us
    # bf16 Out has no atomic form: its workspace-free plan is the direct one
    # (one slice of 128-channel stages)
    free_b = cnn.plan_tiles(p, cnn.CNN_BF16_OBF16, cnn.K_AUTO_NO_WORKSPACE, 0, 0, 0, bud)
    assert (free_b.kernel, free_b.variant, free_b.kc, free_b.ws_bytes) == (cnn.K_SPLITC, 2511, 1, 0)
    L = cnn.lib()
    for pl, bad_ws in [(free, 4 * 16 * 512 * 49), (ws, 0)]:
        q = cnn.Plan.from_buffer_copy(pl)
        q.ws_bytes = bad_ws
        st = L.cnn_fwd_plan_ws(0x1000, 0x10000000, 0x20000000, ctypes.byref(p), cnn.CNN_BF16,
                               ctypes.byref(q), 0x40000000, 1 << 30, None)
        assert st == -8, pl.variant


def test_workspace_plans_need_the_workspace_form():
    """cnn_fwd_plan never allocates: a plan that needs a workspace is
    refused before any HIP call; cnn_fwd_plan_ws checks the workspace."""
    dims = (1, 16, 16, 16, 16, 3, 3, 1, 1)
    p = cnn.problem(*dims)
    pl = cnn.plan_tiles(p, cnn.CNN_F32, cnn.K_SPLITC, 64, 64, 8, cnn.budget())
    assert pl.ws_bytes > 0
    L = cnn.lib()
    args = (0x1000, 0x100000, 0x200000, ctypes.byref(p), cnn.CNN_F32, ctypes.byref(pl))
    assert L.cnn_fwd_plan(*args, None) == -6
    assert b"cnn_fwd_plan_ws" in L.cnn_last_error()
    assert L.cnn_fwd_plan_ws(*args, None, 0, None) == -1
    assert L.cnn_fwd_plan_ws(*args, 0x4000000, pl.ws_bytes - 16, None) == -2
    assert L.cnn_fwd_plan_ws(*args, 0x4000008, pl.ws_bytes, None) == -2


def test_edited_plan_beyond_32bit_ranges_rejected():
    """A plan edited onto a problem whose In exceeds the 2 GiB its kernel
    addresses with 32-bit offsets is refused (CNN_E_PLAN) before any
    launch, not run with clamped loads and dropped stores."""
    small = (32, 64, 64, 56, 56, 3, 3, 1, 1)
    big = (8192, 64, 64, 56, 56, 3, 3, 1, 1)  # In: 8192*64*58*58*2 bytes > 2 GiB
    pl = cnn.plan_tiles(cnn.problem(*small), cnn.CNN_BF16, cnn.K_ROWS, 64, 7 * 56, 0, cnn.budget())
    q = cnn.Plan.from_buffer_copy(pl)
    q.prob = cnn.problem(*big)
    q.grid = pl.grid // 32 * 8192
    st = cnn.lib().cnn_fwd_plan(1 << 40, 1 << 42, 1 << 44, ctypes.byref(q.prob), cnn.CNN_BF16,
                                ctypes.byref(q), None)
    assert st == -8
    with pytest.raises(cnn.CnnError):
        cnn.plan_tiles(cnn.problem(*big), cnn.CNN_BF16, cnn.K_ROWS, 64, 7 * 56, 0, cnn.budget())


def test_closed_form_matches_oracle():
    """cnn_closed_form (Table 1 of Sec. 2.1) against the oracle's Table 1
    row, tiles, cost and relaxed capacity, on random problems, processor
    counts and capacities spanning all three rows, in both capacity modes."""
    rng = np.random.default_rng(7)
    rows = set()
    for _ in range(300):
        Nr, Ns = (int(x) for x in rng.integers(1, 8, size=2))
        dims = (int(rng.integers(1, 65)), int(rng.integers(1, 1025)), int(rng.integers(1, 1025)),
                int(rng.integers(1, 113)), int(rng.integers(1, 113)), Nr, Ns,
                int(rng.integers(1, 3)), int(rng.integers(1, 3)))
        P = float(2 ** int(rng.integers(0, 11)))
        M = float(10 ** rng.uniform(2, 8))
        p = oeq1.Problem(*dims)
        for mode in (0, 1):
            cf = cnn.closed_form(cnn.problem(*dims), P, M, mode)
            ML = M if mode == 0 else oeq1.relaxed_capacity(M, Nr, Ns, dims[7], dims[8])
            row, tk, tb = oeq1.table1_tiles(p, P, ML)
            cost = oeq1.table1_cost(p, P, ML)
            assert abs(cf.M_L - ML) <= 1e-12 * M
            assert cf.row == row and cf.split_c == (row != 1)
            for got, want in ((cf.Tk, tk), (cf.Tbhw, tb), (cf.cost, cost)):
                assert abs(got - want) <= 1e-9 * abs(want), (dims, P, M, mode, got, want)
            rows.add(row)
    assert rows == {1, 2, 3}


def test_closed_form_rejects_bad_arguments():
    L = cnn.lib()
    p = cnn.problem(1, 2, 3, 4, 5, 3, 3, 1, 1)
    out = cnn.ClosedForm()
    assert L.cnn_closed_form(None, 4.0, 100.0, 0, ctypes.byref(out)) == -1
    assert L.cnn_closed_form(ctypes.byref(p), 4.0, 100.0, 0, None) == -1
    for P, M, mode in [(0.5, 100.0, 0), (4.0, 0.0, 0), (4.0, -1.0, 1), (4.0, 100.0, 2)]:
        assert L.cnn_closed_form(ctypes.byref(p), P, M, mode, ctypes.byref(out)) == -2
    q = cnn.problem(1, 0, 3, 4, 5, 3, 3, 1, 1)
    assert L.cnn_closed_form(ctypes.byref(q), 4.0, 100.0, 0, ctypes.byref(out)) == -2


def _hbm_brute(pl, xcds, l2):
    """cnn_hbm_bytes by enumeration: XCD x runs the x-th contiguous run of
    the tile index; its In traffic is every (b, x) input row that any output
    of its tiles reads with any stencil row, each once (all channels and
    columns), plus the rows of every gap between two such rows (in the
    flattened b*Nx + x order) that is shorter than a 128-byte line; its Ker
    traffic is each k tile it meets once (l2 large) or once per tile (l2 =
    1).  The stride-2 row-band kernels write Out at the measured rate of
    1.18 bytes per byte."""
    p = pl.prob
    hw, npix = p.Nw * p.Nh, p.Nb * p.Nw * p.Nh
    Ny = p.sh * (p.Nh - 1) + p.Ns
    e_in = 4 if pl.dtype == cnn.CNN_F32 else 2
    e_out = 2 if pl.dtype == cnn.CNN_BF16_OBF16 else 4
    n_k = -(-p.Nk // pl.tk)
    tiles = -(-npix // pl.tp) * n_k
    q, rem = divmod(tiles, xcds)
    ker = lambda kt: e_in * min(pl.tk, p.Nk - kt * pl.tk) * p.Nc * p.Nr * p.Ns
    in_b = ker_b = 0
    for x in range(xcds):
        cnt = q + (1 if x < rem else 0)
        t0 = x * q + min(x, rem)
        rows, kts, per_tile = set(), set(), 0
        for t in range(t0, t0 + cnt):
            pt, kt = divmod(t, n_k)
            kts.add(kt)
            per_tile += ker(kt)
            for f in range(pt * pl.tp, min((pt + 1) * pl.tp, npix)):
                b, w = f // hw, (f % hw) // p.Nh
                rows.update((b, p.sw * w + r) for r in range(p.Nr))
        Nx = p.sw * (p.Nw - 1) + p.Nr
        flat = sorted(b * Nx + x for b, x in rows)
        gaps = sum(n - m - 1 for m, n in zip(flat, flat[1:])
                   if 0 < (n - m - 1) * Ny * e_in < 128)
        in_b += (len(rows) + gaps) * p.Nc * Ny * e_in
        ker_b += sum(ker(k) for k in kts) if l2 > 1 else per_tile
    out = npix * p.Nk
    extra = 8 * pl.kc * out if pl.kernel == cnn.K_SPLITC else 0
    rate = 1.18 if pl.kernel == cnn.K_SROWS else 1.0
    return e_out * out * rate + extra, ker_b, in_b


@pytest.mark.parametrize("dims,dt,kernel,tk,tp,tc", [
    ((3, 40, 70, 13, 11, 3, 3, 1, 1), cnn.CNN_BF16, cnn.K_IGEMM, 64, 64, 32),
    ((2, 37, 130, 9, 14, 3, 2, 1, 1), cnn.CNN_BF16_OBF16, cnn.K_IGEMM, 128, 128, 32),
    ((2, 16, 33, 7, 9, 3, 3, 1, 1), cnn.CNN_F32, cnn.K_IGEMM, 64, 64, 8),
    ((2, 64, 64, 8, 20, 3, 3, 1, 1), cnn.CNN_BF16, cnn.K_ROWS, 64, 160, 0),
    ((3, 72, 300, 6, 10, 1, 1, 1, 1), cnn.CNN_BF16, cnn.K_GEMM1, 256, 256, 64),
    ((1, 70, 40, 7, 7, 3, 3, 1, 1), cnn.CNN_BF16, cnn.K_SPLITC, 64, 64, 32),
    ((3, 48, 300, 7, 12, 1, 1, 2, 2), cnn.CNN_BF16, cnn.K_GEMM1, 256, 256, 32),   # rows skipped
    ((2, 32, 300, 7, 28, 3, 3, 2, 2), cnn.CNN_BF16, cnn.K_SROWS, 256, 196, 16),
    ((2, 5, 9, 6, 7, 2, 3, 3, 1), cnn.CNN_F32, cnn.K_IGEMM, 64, 64, 8),           # sw > Nr
])
def test_hbm_bytes_matches_enumeration(dims, dt, kernel, tk, tp, tc):
    pl = cnn.plan_tiles(cnn.problem(*dims), dt, kernel, tk, tp, tc, cnn.budget())
    for xcds in (1, 3, 8):
        for l2 in (1 << 40, 1):
            got = cnn.hbm_bytes(pl, xcds, l2)
            want = _hbm_brute(pl, xcds, l2)
            assert all(abs(g - w) <= 1e-9 * max(1.0, w) for g, w in zip(got, want)), \
                (xcds, l2, got, want)


def test_hbm_bytes_rejects_bad_arguments():
    L = cnn.lib()
    pl = cnn.plan_tiles(cnn.problem(1, 16, 16, 16, 16, 3, 3, 1, 1), cnn.CNN_F32, cnn.K_IGEMM,
                        64, 64, 8, cnn.budget())
    terms = (ctypes.c_double * 3)()
    assert L.cnn_hbm_bytes(None, 8, 1 << 22, terms) == -1
    assert L.cnn_hbm_bytes(ctypes.byref(pl), 0, 1 << 22, terms) == -2
    assert L.cnn_hbm_bytes(ctypes.byref(pl), 8, 0, terms) == -2
    d = cnn.plan_tiles(cnn.problem(1, 16, 16, 16, 16, 3, 3, 1, 1), cnn.CNN_F32, cnn.K_DIRECT,
                       bud=cnn.budget())
    assert L.cnn_hbm_bytes(ctypes.byref(d), 8, 1 << 22, terms) == -8


def test_static_scratch_entry_validates_before_hip():
    """cnn_fwd_plan_static refuses, before any HIP call, a plan needing more
    than CNN_STATIC_SCRATCH_BYTES of workspace, and bad arguments."""
    L = cnn.lib()
    dims = (1, 512, 512, 56, 56, 3, 3, 1, 1)
    p = cnn.problem(*dims)
    big = cnn.plan_tiles(p, cnn.CNN_BF16, cnn.K_SPLITC, 64, 64, 32, cnn.budget())
    assert big.ws_bytes > cnn.STATIC_SCRATCH_BYTES
    ptrs = (1 << 40, 1 << 42, 1 << 44)
    assert L.cnn_fwd_plan_static(*ptrs, ctypes.byref(p), cnn.CNN_BF16, ctypes.byref(big), None) == -6
    assert b"CNN_STATIC_SCRATCH_BYTES" in L.cnn_last_error()
    small = cnn.problem(1, 16, 16, 16, 16, 3, 3, 1, 1)
    pl = cnn.plan_tiles(small, cnn.CNN_F32, cnn.K_SPLITC, 64, 64, 8, cnn.budget())
    assert L.cnn_fwd_plan_static(0, 0x100000, 0x200000, ctypes.byref(small), cnn.CNN_F32,
                                 ctypes.byref(pl), None) == -1
    assert L.cnn_fwd_plan_static(*ptrs, ctypes.byref(p), cnn.CNN_F32, ctypes.byref(pl),
                                 None) == -8
    q = cnn.Plan.from_buffer_copy(pl)
    q.kc = 3
    assert L.cnn_fwd_plan_static(0x1000, 0x100000, 0x200000, ctypes.byref(small), cnn.CNN_F32,
                                 ctypes.byref(q), None) == -8


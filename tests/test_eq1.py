"""Pins of the oracle's Eq. (1)/(4) model (Sec. 2, 2.1) against brute force.

* Listing 3 is simulated literally on tiny problems: every tile collects the
  set of In, Ker and Out elements its point loops touch, and the set sizes
  are summed.  That count must equal the exact-halo Eq. (1); for stride 1
  and dividing tiles it must also equal the formula as printed.
* The Case 1a closed form is checked against brute-force minimisation of the
  relaxed cost Eq. (4) over integer tile sizes.
* Table 1 is checked to lower-bound a brute-force search of Eq. (4) and to be
  continuous across its regime boundaries.
* The composite-tile slab count is checked against the set of input rows the
  tile's outputs actually read.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import eq1
from oracle.eq1 import Problem, Tiles


def _listing3_counts(p: Problem, t: Tiles):
    """Literal simulation of Listing 3's loads/stores, returned as
    (Out stores, Ker loads, In loads) in elements."""
    out_n = ker_n = in_n = 0
    rng = lambda n, T: [range(i, min(i + T, n)) for i in range(0, n, T)]
    for kt in rng(p.Nk, t.Tk):
        for bt in rng(p.Nb, t.Tb):
            for wt in rng(p.Nw, t.Tw):
                for ht in rng(p.Nh, t.Th):
                    for ct in rng(p.Nc, t.Tc):
                        in_set, ker_set = set(), set()
                        for b, c, w, h in itertools.product(bt, ct, wt, ht):
                            for r in range(p.Nr):
                                for s in range(p.Ns):
                                    in_set.add((b, c, p.sw * w + r, p.sh * h + s))
                        for k, c in itertools.product(kt, ct):
                            for r in range(p.Nr):
                                for s in range(p.Ns):
                                    ker_set.add((k, c, r, s))
                        in_n += len(in_set)
                        ker_n += len(ker_set)
                    out_n += len(kt) * len(bt) * len(wt) * len(ht)
    return out_n, ker_n, in_n


_CASES = [
    (Problem(2, 4, 3, 4, 6, 3, 3, 1, 1), Tiles(1, 2, 1, 2, 3)),
    (Problem(2, 4, 3, 4, 6, 3, 3, 2, 2), Tiles(1, 2, 1, 2, 3)),
    (Problem(3, 3, 5, 5, 4, 3, 2, 2, 1), Tiles(2, 2, 2, 2, 3)),
    (Problem(1, 2, 4, 7, 5, 5, 3, 1, 3), Tiles(1, 3, 2, 3, 2)),
    (Problem(2, 3, 2, 3, 3, 2, 2, 2, 2), Tiles(2, 2, 3, 3, 3)),
    (Problem(1, 5, 3, 6, 6, 1, 1, 1, 1), Tiles(1, 2, 2, 4, 4)),
]


@pytest.mark.parametrize("p,t", _CASES)
def test_exact_halo_equals_listing3(p, t):
    assert p.sw <= p.Nr and p.sh <= p.Ns
    sim = _listing3_counts(p, t)
    assert eq1.eq1_terms(p, t, "exact") == sim


def test_paper_formula_equals_listing3_when_tiles_divide_stride1():
    p, t = Problem(2, 4, 3, 4, 6, 3, 3, 1, 1), Tiles(1, 1, 2, 2, 3)
    sim = _listing3_counts(p, t)
    assert eq1.eq1_terms(p, t, "paper") == tuple(float(v) for v in sim)
    assert eq1.eq1_cost(p, t, "paper") == float(sum(sim))


def test_paper_halo_overcounts_for_stride2():
    """The printed halo sigma*T + R - 1 counts sigma-1 rows/cols a tile never
    reads; the exact halo sigma*(T-1) + R matches the simulation."""
    p, t = Problem(2, 4, 3, 4, 6, 3, 3, 2, 2), Tiles(1, 3, 4, 2, 3)
    o, k, i = _listing3_counts(p, t)
    po, pk, pi = eq1.eq1_terms(p, t, "paper")
    assert (po, pk) == (o, k) and pi > i
    assert eq1.eq1_terms(p, t, "exact") == (o, k, i)


@pytest.mark.parametrize("p,t", _CASES)
def test_footprint_is_max_tile_working_set(p, t):
    """Eq. (1) constraint, exact halo: the largest (full) tile's In+Ker+Out set."""
    full = Tiles(t.Tb, t.Tk, t.Tc, t.Tw, t.Th)
    in_el = t.Tb * t.Tc * len({(p.sw * w + r) for w in range(t.Tw) for r in range(p.Nr)}) * \
        len({(p.sh * h + s) for h in range(t.Th) for s in range(p.Ns)})
    want = in_el + t.Tw * t.Th * t.Tb * t.Tk + p.Nr * p.Ns * t.Tk * t.Tc
    assert eq1.eq1_footprint(p, full, "exact") == want


@pytest.mark.parametrize("RS,ss", [(9, 1), (9, 4), (1, 1), (49, 4), (25, 1)])
def test_case1a_closed_form_vs_brute_force(RS, ss):
    """Minimise Nr Ns / Tbhw + sw sh / Tk over integers with Tk*Tbhw <= ML."""
    ML = 4096
    best = None
    for tk in range(1, ML + 1):
        tb = ML // tk
        f = RS / tb + ss / tk
        if best is None or f < best[0]:
            best = (f, tk, tb)
    sw = sh = int(math.isqrt(ss))
    Nr = Ns = int(math.isqrt(RS))
    tk_c, tb_c = eq1.case1a_tiles(ML, Nr, Ns, sw, sh)
    assert abs(tk_c * tb_c - ML) < 1e-9 * ML
    assert abs(tb_c / tk_c - RS / ss) < 1e-9 * RS / ss
    f_c = RS / tb_c + ss / tk_c
    assert abs(f_c - 2 * math.sqrt(RS * ss / ML)) < 1e-12
    assert best[0] >= f_c - 1e-12            # continuous optimum is a lower bound
    assert best[0] <= f_c * 1.01             # and is (nearly) attained
    assert abs(best[1] - tk_c) <= 0.1 * tk_c + 1


def test_relaxed_capacity_identity():
    """M_L solves M_L + 3K sqrt(M_L) = M with K = sqrt(sw sh Nr Ns)."""
    for M, (Nr, Ns, sw, sh) in itertools.product([1e3, 65536.0, 1e7], [(3, 3, 1, 1), (3, 3, 2, 2), (7, 7, 2, 2), (1, 1, 1, 1)]):
        ML = eq1.relaxed_capacity(M, Nr, Ns, sw, sh)
        K = math.sqrt(sw * sh * Nr * Ns)
        assert 0 < ML < M
        assert abs(ML + 3 * K * math.sqrt(ML) - M) < 1e-9 * M


def test_relaxed_capacity_gives_valid_tile_square_spatial():
    """With Tb = 1 and square spatial tiles, the Case 1a tile at M_L fits M
    once the halo is put back (the paper's claim, checked where its
    treatment of b, h, w as one index holds)."""
    for M in [16384.0, 65536.0, 262144.0]:
        for Nr, sw in [(3, 1), (3, 2), (5, 1)]:
            ML = eq1.relaxed_capacity(M, Nr, Nr, sw, sw)
            tk, tbhw = eq1.case1a_tiles(ML, Nr, Nr, sw, sw)
            T = math.sqrt(tbhw)
            g = (sw * T + Nr - 1) ** 2 * 1 * 1 + tbhw * tk + Nr * Nr * tk * 1
            assert g <= M * (1 + 1e-12)


def _eq4_brute_min(p: Problem, P: int, ML: int):
    Nbhw = p.Nb * p.Nw * p.Nh
    total = p.Nk * p.Nc * Nbhw
    best = math.inf
    divs = lambda n: [d for d in range(1, n + 1) if n % d == 0]
    for Wk in divs(p.Nk):
        for Wc in divs(p.Nc):
            rest = total // P
            if total % P or rest % (Wk * Wc):
                continue
            Wbhw = rest // (Wk * Wc)
            if Wbhw > Nbhw:
                continue
            for Tk in range(1, Wk + 1):
                Tb = min(Wbhw, ML // Tk)
                if Tb < 1:
                    continue
                best = min(best, eq1.eq4_cost(p, P, Wk, Wbhw, Tk, Tb))
    return best


@pytest.mark.parametrize("ML", [16, 64, 256, 700, 1024, 4096, 1 << 16])
def test_table1_lower_bounds_eq4(ML):
    """Table 1 (its rows 1, 2 and 3: ML = 700 lies between A = 512 and the
    Case 2a threshold, about 845, for this problem) lower-bounds a
    brute-force minimisation of Eq. (4) and is nearly attained."""
    p = Problem(1, 16, 32, 8, 8, 3, 3, 1, 1)
    P = 4
    bound = eq1.table1_cost(p, P, ML)
    brute = _eq4_brute_min(p, P, ML)
    assert bound <= brute * (1 + 1e-12)
    assert brute <= 1.6 * bound


def test_table1_continuous_at_regime_boundaries():
    p = Problem(2, 64, 128, 14, 14, 3, 3, 2, 2)
    P = 16
    Nbhw = p.Nb * p.Nw * p.Nh
    A = p.Nk * Nbhw / P
    V = p.Nk * p.Nc * Nbhw / P
    Q = p.Nr * p.Ns * p.sw * p.sh
    thr = V ** (2 / 3) * Q ** (1 / 3)
    for x in (A, thr):
        lo, hi = eq1.table1_cost(p, P, x * (1 - 1e-9)), eq1.table1_cost(p, P, x * (1 + 1e-9))
        assert abs(lo - hi) < 1e-6 * lo
    assert abs(eq1.case1a_cost(p, P, A / 2) - eq1.table1_cost(p, P, A / 2)) < 1e-9 * A


@pytest.mark.parametrize("p,P", [(Problem(2, 64, 128, 14, 14, 3, 3, 2, 2), 16),
                                 (Problem(1, 512, 512, 7, 7, 3, 3, 1, 1), 256),
                                 (Problem(8, 3, 64, 56, 56, 7, 5, 2, 1), 64)])
def test_table1_tiles_attain_the_row_cost_in_eq4(p, P):
    """Each Table 1 row's tiles, put into the Eq. (4) objective with the
    row's W (W_c = N_c in row 1; W = T, W_c < N_c in rows 2 and 3), give the
    row's cost; rows 1 and 3 fill M_L; row 2's tiles are a stationary point
    (no nearby tile pair costs less) and fit M_L."""
    Nbhw = p.Nb * p.Nw * p.Nh
    A = p.Nk * Nbhw / P
    V = p.Nk * p.Nc * Nbhw / P
    thr = V ** (2 / 3) * (p.Nr * p.Ns * p.sw * p.sh) ** (1 / 3)
    rows = set()
    for ML in [A / 3, 2 * max(A, thr)] + ([(A + thr) / 2] if A < thr else []):
        row, tk, tb = eq1.table1_tiles(p, P, ML)
        rows.add(row)
        want = eq1.table1_cost(p, P, ML)
        if row == 1:
            assert ML <= A
            got = eq1.eq4_cost(p, P, p.Nk, Nbhw / P, tk, tb)  # Wk Wbhw = Nk Nbhw / P
            assert abs(tk * tb - ML) < 1e-9 * ML
        else:
            got = eq1.eq4_cost(p, P, tk, tb, tk, tb)
            if row == 3:
                assert abs(tk * tb - ML) < 1e-9 * ML and ML < thr
            else:
                assert tk * tb <= ML * (1 + 1e-12) and ML >= thr
                for fk in (0.97, 1.0, 1.03):
                    for fb in (0.97, 1.0, 1.03):
                        assert eq1.eq4_cost(p, P, tk * fk, tb * fb, tk * fk, tb * fb) >= got * (1 - 1e-12)
        assert abs(got - want) < 1e-9 * want, (row, got, want)
    assert rows >= {1, 2}


@pytest.mark.parametrize("p", [Problem(3, 2, 2, 5, 7, 3, 3, 1, 1), Problem(2, 2, 2, 4, 6, 3, 2, 2, 1),
                               Problem(4, 1, 1, 3, 3, 1, 1, 1, 1), Problem(2, 1, 1, 6, 5, 5, 3, 2, 2)])
@pytest.mark.parametrize("T", [1, 4, 7, 12, 32])
def test_slab_rows_match_rows_touched(p, T):
    """For sw <= Nr the contiguous slab of a composite tile is exactly the set
    of (b, x) input rows its outputs read."""
    n = p.Nb * p.Nw * p.Nh
    for f in range(0, n, T):
        last = min(f + T, n) - 1
        rows = set()
        for q in range(f, last + 1):
            b, w = q // (p.Nw * p.Nh), (q % (p.Nw * p.Nh)) // p.Nh
            for r in range(p.Nr):
                rows.add((b, p.sw * w + r))
        assert eq1.slab_rows(p, f, last) == len(rows)


def test_slab_terms_equal_box_terms_for_row_tiles():
    """A composite tile of Tw whole rows inside one image is the box tile
    (Tb=1, Tw, Th=Nh); both forms of the In term then agree."""
    p = Problem(3, 4, 8, 6, 5, 3, 3, 1, 1)
    for Tw in (1, 2, 3, 6):
        o, k, i = eq1.slab_terms(p, 4, Tw * p.Nh)
        assert (o, k, i) == eq1.eq1_terms(p, Tiles(1, 4, 1, Tw, p.Nh), "exact")

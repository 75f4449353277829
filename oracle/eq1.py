"""Data-movement model of the paper, written out -- TEST INFRASTRUCTURE ONLY.

Part of the oracle: the GPU library has its own, independent implementation
of the same formulas, and tests compare the two.

Notation follows the paper.  A problem is (Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)
with sw, sh the strides sigma_w, sigma_h; a box tiling is
(Tb, Tk, Tc, Tw, Th).  All volumes are counted in tensor ELEMENTS.

* :func:`eq1_cost` / :func:`eq1_footprint` -- Eq. (1), Sec. 2: the volume
  moved by the single-level tiled loop nest (Listing 2/3) and the fast-memory
  footprint of one tile.  ``halo="paper"`` is the formula as printed (real
  division, halo sigma*T + R - 1).  ``halo="exact"`` counts what Listing 3
  moves when tile counts are rounded up and edge tiles are clipped, with the
  exact halo extent sigma*(T-1) + R of a tile of T outputs.
* :func:`slab_cost` -- the same three Eq. (1) terms for "composite" tiles:
  T_bhw consecutive outputs of the flattened (b, w, h) index (Sec. 2 treats
  b, h, w as one composite index), each loading whole input rows.
* :func:`eq4_cost`, :func:`case1a_tiles`, :func:`case1a_cost`,
  :func:`relaxed_capacity`, :func:`table1_cost`, :func:`table1_tiles` --
  Sec. 2.1: the relaxed problem Eq. (4), its Case 1a optimum Eq. (6), the
  capacity M_L that makes the relaxed optimum a valid tiling, the Table 1
  optima and the tiles of each Table 1 row (Cases 1a, 2a, 2b).
"""
from __future__ import annotations

import math
from dataclasses import dataclass


@dataclass(frozen=True)
class Problem:
    Nb: int
    Nc: int
    Nk: int
    Nw: int
    Nh: int
    Nr: int
    Ns: int
    sw: int = 1
    sh: int = 1

    @property
    def Nx(self) -> int:
        """Input rows: sigma_w*(Nw-1) + Nr (valid convolution)."""
        return self.sw * (self.Nw - 1) + self.Nr

    @property
    def Ny(self) -> int:
        """Input columns: sigma_h*(Nh-1) + Ns."""
        return self.sh * (self.Nh - 1) + self.Ns


@dataclass(frozen=True)
class Tiles:
    Tb: int
    Tk: int
    Tc: int
    Tw: int
    Th: int


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def _tile_sizes(n: int, t: int):
    """Extents of the ceil(n/t) tiles of size t covering 0..n-1 (last clipped)."""
    return [min(t, n - i) for i in range(0, n, t)]


def eq1_terms(p: Problem, t: Tiles, halo: str = "paper"):
    """The three Eq. (1) terms (Out, Ker, In) in elements.

    paper: Out = Nb Nk Nw Nh;
           Ker = Nk Nc Nr Ns Nw Nh Nb / (Tw Th Tb);
           In  = Nb Nc (sw Tw + Nr - 1)(sh Th + Ns - 1) Nw Nh Nk / (Tw Th Tk).
    exact: Out as above; Ker loaded once per (b, w, h) tile;
           In loaded once per (b, w, h) tile per k tile, each load the clipped
           box Tb' x Nc x (sw(Tw'-1)+Nr) x (sh(Th'-1)+Ns).
    """
    out = p.Nb * p.Nk * p.Nw * p.Nh
    if halo == "paper":
        ker = p.Nk * p.Nc * p.Nr * p.Ns * p.Nw * p.Nh * p.Nb / (t.Tw * t.Th * t.Tb)
        inp = (p.Nb * p.Nc * (p.sw * t.Tw + p.Nr - 1) * (p.sh * t.Th + p.Ns - 1)
               * p.Nw * p.Nh * p.Nk / (t.Tw * t.Th * t.Tk))
        return float(out), float(ker), float(inp)
    if halo == "exact":
        n_bhw = _ceil_div(p.Nb, t.Tb) * _ceil_div(p.Nw, t.Tw) * _ceil_div(p.Nh, t.Th)
        ker = n_bhw * p.Nk * p.Nc * p.Nr * p.Ns
        xs = sum(p.sw * (tw - 1) + p.Nr for tw in _tile_sizes(p.Nw, t.Tw))
        ys = sum(p.sh * (th - 1) + p.Ns for th in _tile_sizes(p.Nh, t.Th))
        inp = _ceil_div(p.Nk, t.Tk) * p.Nc * p.Nb * xs * ys
        return out, ker, inp
    raise ValueError("halo must be 'paper' or 'exact'")


def eq1_cost(p: Problem, t: Tiles, halo: str = "paper"):
    """Eq. (1) total data movement in elements."""
    o, k, i = eq1_terms(p, t, halo)
    return o + k + i


def eq1_footprint(p: Problem, t: Tiles, halo: str = "paper") -> int:
    """Left side of the Eq. (1) capacity constraint (one tile, elements).

    In tile (with halo) x Tb x Tc + Out tile Tw Th Tb Tk + Ker tile Nr Ns Tk Tc.
    """
    if halo == "paper":
        x, y = p.sw * t.Tw + p.Nr - 1, p.sh * t.Th + p.Ns - 1
    elif halo == "exact":
        x, y = p.sw * (t.Tw - 1) + p.Nr, p.sh * (t.Th - 1) + p.Ns
    else:
        raise ValueError("halo must be 'paper' or 'exact'")
    return x * y * t.Tb * t.Tc + t.Tw * t.Th * t.Tb * t.Tk + p.Nr * p.Ns * t.Tk * t.Tc


def slab_rows(p: Problem, first: int, last: int) -> int:
    """Input rows a composite tile stages: outputs first..last (inclusive) of
    the flattened (b, w, h) index need, per image, input rows
    sw*w .. sw*w + Nr - 1 of every output row w they touch.  The tile stages
    the contiguous range of flattened (b, x) input rows from the first such
    row to the last one."""
    hw = p.Nw * p.Nh
    b0, w0 = first // hw, (first % hw) // p.Nh
    b1, w1 = last // hw, (last % hw) // p.Nh
    return (b1 * p.Nx + p.sw * w1 + p.Nr) - (b0 * p.Nx + p.sw * w0)


def slab_terms(p: Problem, Tk: int, Tbhw: int):
    """Eq. (1) terms (Out, Ker, In) for composite tiles of Tbhw outputs of the
    flattened (b, w, h) index and Tk output channels, each tile loading whole
    input rows (all Ny columns) for every channel."""
    n_pix = p.Nb * p.Nw * p.Nh
    out = n_pix * p.Nk
    n_p = _ceil_div(n_pix, Tbhw)
    ker = n_p * p.Nk * p.Nc * p.Nr * p.Ns
    rows = sum(slab_rows(p, f, min(f + Tbhw, n_pix) - 1) for f in range(0, n_pix, Tbhw))
    inp = _ceil_div(p.Nk, Tk) * p.Nc * p.Ny * rows
    return out, ker, inp


def slab_cost(p: Problem, Tk: int, Tbhw: int) -> int:
    o, k, i = slab_terms(p, Tk, Tbhw)
    return o + k + i


# ---- Sec. 2.1: relaxed problem and closed forms -------------------------

def eq4_cost(p: Problem, P: int, Wk: float, Wbhw: float, Tk: float, Tbhw: float) -> float:
    """Eq. (4): cost_L = Wk Wbhw + (Nk Nc Nbhw / P)(Nr Ns / Tbhw + sw sh / Tk)."""
    Nbhw = p.Nb * p.Nw * p.Nh
    return Wk * Wbhw + (p.Nk * p.Nc * Nbhw / P) * (p.Nr * p.Ns / Tbhw + p.sw * p.sh / Tk)


def case1a_tiles(ML: float, Nr: int, Ns: int, sw: int, sh: int):
    """Case 1a optimum of Eq. (4): Tk = sqrt(ML sw sh / (Nr Ns)),
    Tbhw = sqrt(ML Nr Ns / (sw sh)).  Their product is ML and their ratio
    Tbhw / Tk is Nr Ns / (sw sh)."""
    tk = math.sqrt(ML * sw * sh / (Nr * Ns))
    tbhw = math.sqrt(ML * Nr * Ns / (sw * sh))
    return tk, tbhw


def case1a_cost(p: Problem, P: int, ML: float) -> float:
    """Eq. (6): Nk Nbhw / P + 2 (Nk Nc Nbhw / P) sqrt(Nr Ns sw sh / ML)."""
    Nbhw = p.Nb * p.Nw * p.Nh
    return (p.Nk * Nbhw / P
            + 2.0 * (p.Nk * p.Nc * Nbhw / P) * math.sqrt(p.Nr * p.Ns * p.sw * p.sh / ML))


def relaxed_capacity(M: float, Nr: int, Ns: int, sw: int, sh: int) -> float:
    """M_L = M - (1/2) * 3K (sqrt(9K^2 + 4M) - 3K), K = sqrt(sw sh Nr Ns)."""
    K = math.sqrt(sw * sh * Nr * Ns)
    return M - 0.5 * (3.0 * K * (math.sqrt(9.0 * K * K + 4.0 * M) - 3.0 * K))


def table1_cost(p: Problem, P: int, ML: float) -> float:
    """Table 1: optimal Eq. (4) cost for loop orders with c innermost.

    Three regimes, selected by ML against Nk Nbhw / P and
    (Nk Nc Nbhw / P)^(2/3) (Nr Ns sw sh)^(1/3).
    """
    Nbhw = p.Nb * p.Nw * p.Nh
    V = p.Nk * p.Nc * Nbhw / P
    Q = p.Nr * p.Ns * p.sw * p.sh
    if p.Nk * Nbhw / P >= ML:
        return p.Nk * Nbhw / P + 2.0 * V * math.sqrt(Q / ML)
    thr = V ** (2.0 / 3.0) * Q ** (1.0 / 3.0)
    if ML >= thr:
        return 3.0 * thr
    return ML + 2.0 * V / math.sqrt(ML) * math.sqrt(Q)


def table1_tiles(p: Problem, P: int, ML: float):
    """(row, Tk, Tbhw) of the Table 1 optimum.

    Row 1 (Nk Nbhw / P >= ML): Case 1a, W_c = N_c, Tk and Tbhw of
    :func:`case1a_tiles`.  Row 2 (ML >= V^(2/3) Q^(1/3), V = Nk Nc Nbhw / P,
    Q = Nr Ns sw sh): Case 2a, W_c < N_c with T = W,
    Tk = (V / (Nr Ns))^(1/3) (sw sh)^(2/3),
    Tbhw = (V / (sw sh))^(1/3) (Nr Ns)^(2/3).  Row 3: Case 2b, the Case 1a
    expressions (the capacity binds).
    """
    Nbhw = p.Nb * p.Nw * p.Nh
    V = p.Nk * p.Nc * Nbhw / P
    RS, ss = p.Nr * p.Ns, p.sw * p.sh
    if p.Nk * Nbhw / P >= ML:
        return (1,) + case1a_tiles(ML, p.Nr, p.Ns, p.sw, p.sh)
    if ML >= V ** (2.0 / 3.0) * (RS * ss) ** (1.0 / 3.0):
        return 2, (V / RS) ** (1.0 / 3.0) * ss ** (2.0 / 3.0), (V / ss) ** (1.0 / 3.0) * RS ** (2.0 / 3.0)
    return (3,) + case1a_tiles(ML, p.Nr, p.Ns, p.sw, p.sh)

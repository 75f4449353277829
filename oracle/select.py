"""Brute-force reference of the tile-size selector -- TEST INFRASTRUCTURE ONLY.

The library's selector evaluates the paper's Eq. (1) (Sec. 2) for every
tiling its kernels implement and picks one; this module restates the same
rule, over a candidate list typed in here independently, so tests can check
the library's choice (an integer decision) exactly.

Rule
----
A candidate is (tk, tp, tc): tk output features by tp consecutive outputs
of the flattened (b, w, h) index per workgroup, tc input features per LDS
stage, with `acc` fp32 accumulators per lane.  It is feasible when its LDS
footprint -- the halo'd In slab (whole input rows) and the Ker tile -- fits
the LDS budget and `acc` fits the accumulator budget.  Its cost is
Eq. (1) in bytes for composite tiles (``eq1.slab_terms``), converted to
time on P = `cus` processors:

    rounds * (slots / cus) * max(tile_flops / mfma_rate, (bytes / tiles) / 64)

with slots = cus * min(wg_per_cu, floor(lds / footprint)), tile_flops the
MFMA work of one tile padded to whole blocks, mfma_rate 4096 (bf16) or
256 (fp32) flops per CU per clock, 64 bytes per CU per clock from L2.
Lowest time wins; ties go to larger tk, then tp, then tc, then lower id.
If nothing fits, the direct kernel is used.
"""
from __future__ import annotations

import math

from . import eq1

F32, BF16, BF16_OBF16 = 0, 1, 2

# (id, dtype, wm, wn, mb, nb, tc) of the implicit-GEMM kernels; tk = 32*wm*mb,
# tp = 32*wn*nb, acc = 16*mb*nb.
IGEMM = [
    (100, F32, 1, 4, 2, 2, 8), (101, F32, 2, 2, 2, 2, 8), (102, F32, 1, 4, 1, 2, 8),
    (103, F32, 2, 2, 1, 1, 8), (104, F32, 1, 4, 2, 1, 8),
    (200, BF16, 1, 4, 2, 2, 32), (201, BF16, 2, 2, 2, 2, 32), (202, BF16, 2, 2, 2, 4, 16),
    (203, BF16, 4, 1, 2, 4, 16), (204, BF16, 1, 4, 1, 2, 32), (205, BF16, 2, 2, 1, 1, 32),
    (206, BF16, 1, 4, 2, 1, 32),
    (300, BF16_OBF16, 1, 4, 2, 2, 32), (301, BF16_OBF16, 2, 2, 2, 2, 32),
    (302, BF16_OBF16, 2, 2, 2, 4, 16), (303, BF16_OBF16, 4, 1, 2, 4, 16),
    (304, BF16_OBF16, 1, 4, 1, 2, 32), (305, BF16_OBF16, 2, 2, 1, 1, 32),
    (306, BF16_OBF16, 1, 4, 2, 1, 32),
]


def _max_slab(p: eq1.Problem, tp: int) -> int:
    n = p.Nb * p.Nw * p.Nh
    return max(eq1.slab_rows(p, f, min(f + tp, n) - 1) for f in range(0, n, tp))


def candidates(p: eq1.Problem, dtype: int, cus: int, lds_bytes: int, acc_regs: int,
               wg_per_cu: int):
    """Yield (time, tk, tp, tc, id, info) for every feasible candidate."""
    e_in = 4 if dtype == F32 else 2
    e_out = 2 if dtype == BF16_OBF16 else 4
    kv = 1 if dtype == F32 else 8
    vec = 4 if dtype == F32 else 16
    rate = 256.0 if dtype == F32 else 4096.0
    RS = p.Nr * p.Ns
    npix = p.Nb * p.Nw * p.Nh
    for vid, dt, wm, wn, mb, nb, tc in IGEMM:
        if dt != dtype:
            continue
        tk, tp, acc = 32 * wm * mb, 32 * wn * nb, 16 * mb * nb
        S = _max_slab(p, tp)
        groups = tc // kv
        lds = (groups * S * p.Ny + RS * groups * tk) * vec
        if lds > lds_bytes or acc > acc_regs:
            continue
        tiles = math.ceil(npix / tp) * math.ceil(p.Nk / tk)
        occ = max(1, min(lds_bytes // lds, wg_per_cu))
        slots = cus * occ
        rounds = math.ceil(tiles / slots)
        o, k, i = eq1.slab_terms(p, tk, tp)
        nbytes = e_out * o + e_in * (k + i)
        tile_flops = 2.0 * tk * tp * (math.ceil(p.Nc / tc) * tc) * RS
        tile_clk = max(tile_flops / rate, (nbytes / tiles) / 64.0)
        t = rounds * slots / cus * tile_clk
        yield t, tk, tp, tc, vid, {"grid": tiles, "lds": lds, "slab": S, "bytes": nbytes,
                                   "terms": (o, k, i)}


def choose(p: eq1.Problem, dtype: int, cus=256, lds_bytes=160 * 1024, acc_regs=128,
           wg_per_cu=2):
    """(kernel, variant id, tk, tp, tc) the rule above selects."""
    best = None
    for t, tk, tp, tc, vid, info in candidates(p, dtype, cus, lds_bytes, acc_regs, wg_per_cu):
        key = (t, -tk, -tp, -tc, vid)
        if best is None or key < best[0]:
            best = (key, (2, vid, tk, tp, tc))
    if best is None:
        return (1, 1, 1, 1, p.Nc)
    return best[1]

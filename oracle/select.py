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

Two implicit-GEMM families are ranked in tiers.  Tier 1 (the pipelined
bf16 kernel) double-buffers both LDS tiles: footprint
2 * 16 * (tc/8 * even(S*Ny) + blk), blk = RS * tc/8 * tk vectors rounded up
to a multiple of 256; it also needs its stencil to match a compile-time
one (or be generic), ceil(S*Ny/2) <= 256 * maxp slab position pairs, and
(tp // (Nw*Nh) + 2) images to span < 2^31 bytes of In and of Out.
Tier 0 holds the wide-staging bf16 kernel -- footprint
2 * 16 * (tc/8 * ceil8(S*Ny) + blk), tc/8 * ceil(S*Ny/8) <= 256*maxi items,
the same 2^31-byte span rule as below -- and the DMA-staged bf16 kernel:
footprint
16 * (tc/8 * S*Ny + nbuf * 256 * (ndi + ndk)); it needs tc*S*nbr <= 256*ndi
natural-copy blocks (nbr = (Ny + 14) // 8 per row), RS*tc/8*tk <= 256*ndk Ker
vectors, S*Ny <= 256*mpos positions, and (imgs*Nc + tc) input planes and imgs
output images to span < 2^31 bytes.  Each later tier is ranked only if no
candidate of the earlier tiers fits; tier 2 (the plain staging kernel) last.
If nothing fits, the direct kernel is used.

Before all tiers the automatic choice takes a specialized family when one
fits (`_special`): the 1x1 GEMM kernel for 1x1 layers (the first row of
GEMM1 whose stride mode, size limits, LDS image and balanced tile fit),
else the row-streaming kernel for stride 1 (the first row of ROWS that fits,
with the band that needs the fewest rounds of row groups per workgroup, the
largest such), else the stride-2 row-band kernel (the largest band that
divides Nw, then the lowest id).  These are not ranked by the cost above.
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


# (id, dtype, wm, wn, mb, nb, tc, nr, ns, maxp, rawk, pw) of the pipelined
# kernel; rawk = 1: Ker staged from its raw rows (Nc must be a multiple of 8),
# LDS rows of (taps*tc/8 rounded up to odd) 16-byte chunks per feature;
# pw = 1: 1x1 gather, stages the tile's outputs (pairs: ceil(tp/2)).
IGEMM2 = [
    (400, BF16, 1, 4, 2, 2, 16, 3, 3, 3, 0, 0), (401, BF16, 2, 2, 2, 2, 16, 3, 3, 3, 0, 0),
    (402, BF16, 2, 2, 2, 4, 16, 3, 3, 3, 0, 0), (404, BF16, 1, 4, 2, 2, 32, 3, 3, 2, 0, 0),
    (410, BF16, 1, 4, 2, 2, 16, 0, 0, 4, 0, 0), (411, BF16, 2, 2, 2, 4, 16, 0, 0, 4, 0, 0),
    (412, BF16, 4, 1, 2, 4, 16, 0, 0, 4, 0, 0),
    (420, BF16, 1, 4, 2, 2, 16, 3, 3, 3, 1, 0), (421, BF16, 2, 2, 2, 2, 16, 3, 3, 3, 1, 0),
    (422, BF16, 2, 2, 2, 4, 16, 3, 3, 3, 1, 0), (424, BF16, 1, 4, 2, 2, 32, 3, 3, 2, 1, 0),
    (430, BF16, 1, 4, 2, 2, 16, 1, 1, 4, 1, 0), (431, BF16, 2, 2, 2, 4, 16, 1, 1, 4, 1, 0),
    (432, BF16, 4, 1, 2, 4, 16, 1, 1, 4, 1, 0),
    (440, BF16, 4, 1, 2, 4, 64, 1, 1, 1, 1, 1), (441, BF16, 2, 2, 2, 4, 64, 1, 1, 1, 1, 1),
    (442, BF16, 1, 4, 2, 2, 64, 1, 1, 1, 1, 1),
    (500, BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 3, 0, 0), (501, BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 3, 0, 0),
    (502, BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 3, 0, 0), (504, BF16_OBF16, 1, 4, 2, 2, 32, 3, 3, 2, 0, 0),
    (510, BF16_OBF16, 1, 4, 2, 2, 16, 0, 0, 4, 0, 0), (511, BF16_OBF16, 2, 2, 2, 4, 16, 0, 0, 4, 0, 0),
    (512, BF16_OBF16, 4, 1, 2, 4, 16, 0, 0, 4, 0, 0),
    (520, BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 3, 1, 0), (521, BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 3, 1, 0),
    (522, BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 3, 1, 0), (524, BF16_OBF16, 1, 4, 2, 2, 32, 3, 3, 2, 1, 0),
    (530, BF16_OBF16, 1, 4, 2, 2, 16, 1, 1, 4, 1, 0), (531, BF16_OBF16, 2, 2, 2, 4, 16, 1, 1, 4, 1, 0),
    (532, BF16_OBF16, 4, 1, 2, 4, 16, 1, 1, 4, 1, 0),
    (540, BF16_OBF16, 4, 1, 2, 4, 64, 1, 1, 1, 1, 1), (541, BF16_OBF16, 2, 2, 2, 4, 64, 1, 1, 1, 1, 1),
    (542, BF16_OBF16, 1, 4, 2, 2, 64, 1, 1, 1, 1, 1),
]


# (id, dtype, wm, wn, mb, nb, tc, nr, ns, nbuf, ndi, ndk, mpos) of the
# DMA-staged kernel.
IGEMM3 = [
    (600, BF16, 1, 4, 2, 2, 16, 3, 3, 3, 6, 5, 3),
    (602, BF16, 2, 2, 2, 2, 16, 3, 3, 2, 7, 9, 3), (603, BF16, 2, 2, 2, 4, 16, 3, 3, 2, 6, 9, 3),
    (610, BF16, 1, 4, 2, 2, 16, 0, 0, 3, 4, 1, 2), (611, BF16, 2, 2, 2, 4, 16, 0, 0, 3, 4, 2, 2),
    (612, BF16, 4, 1, 2, 4, 16, 0, 0, 3, 4, 2, 2), (613, BF16, 1, 4, 2, 1, 16, 0, 0, 2, 6, 13, 4),
    (700, BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 3, 6, 5, 3),
    (702, BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 2, 7, 9, 3),
    (703, BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 2, 6, 9, 3),
    (710, BF16_OBF16, 1, 4, 2, 2, 16, 0, 0, 3, 4, 1, 2),
    (711, BF16_OBF16, 2, 2, 2, 4, 16, 0, 0, 3, 4, 2, 2),
    (712, BF16_OBF16, 4, 1, 2, 4, 16, 0, 0, 3, 4, 2, 2),
    (713, BF16_OBF16, 1, 4, 2, 1, 16, 0, 0, 2, 6, 13, 4),
]


# (id, dtype, wm, wn, mb, nb, tc, nr, ns, maxi) of the wide-staging kernel.
IGEMM4 = [
    (800, BF16, 1, 4, 2, 2, 16, 3, 3, 1), (801, BF16, 1, 4, 2, 2, 32, 3, 3, 2),
    (802, BF16, 2, 2, 2, 4, 16, 3, 3, 2), (803, BF16, 2, 2, 2, 2, 16, 3, 3, 1),
    (810, BF16, 4, 1, 2, 4, 32, 1, 1, 1), (811, BF16, 2, 2, 2, 4, 32, 1, 1, 1),
    (812, BF16, 4, 1, 2, 4, 64, 1, 1, 1), (820, BF16, 1, 4, 2, 2, 16, 0, 0, 2),
    (900, BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 1), (901, BF16_OBF16, 1, 4, 2, 2, 32, 3, 3, 2),
    (902, BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 2), (903, BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 1),
    (910, BF16_OBF16, 4, 1, 2, 4, 32, 1, 1, 1), (911, BF16_OBF16, 2, 2, 2, 4, 32, 1, 1, 1),
    (912, BF16_OBF16, 4, 1, 2, 4, 64, 1, 1, 1), (920, BF16_OBF16, 1, 4, 2, 2, 16, 0, 0, 2),
]


# (id, dtype, nb, ks) of the few-channel kernel: tk = 64, tp = 128*nb,
# K = flattened (c, r, s padded to 8), ceil(Nc*Nr/2) <= ks K-steps, Ns <= 8.
SMALLC = [
    (1000, BF16, 2, 12), (1001, BF16, 1, 12), (1002, BF16, 2, 24),
    (1100, BF16_OBF16, 2, 12), (1101, BF16_OBF16, 1, 12), (1102, BF16_OBF16, 2, 24),
]


# (id, dtype, wm, wn, mb, nb, tc, nr, ns, kres, mpos, ndma) of the persistent
# streaming kernel: tk = 32*wm*mb, tp = 32*wn*nb, 64*wm*wn threads; kres
# keeps all of Ker in LDS (Nk <= tk), packed as MFMA operands (tc/8 vectors
# per tap and feature per stage), else two raw-row stages; the slab must fit mpos transposed
# positions and ndma 16-byte natural-copy blocks per thread (rows copied as
# ceil((Ny+14)/8) blocks); grid = workgroup slots.
STREAM = [
    (1300, BF16, 2, 4, 1, 2, 16, 3, 3, 1, 1, 2),
    (1310, BF16, 2, 4, 2, 1, 16, 3, 3, 0, 2, 3),
    (1400, BF16_OBF16, 2, 4, 1, 2, 16, 3, 3, 1, 1, 2),
    (1410, BF16_OBF16, 2, 4, 2, 1, 16, 3, 3, 0, 2, 3),
]


# (id, dtype, nr, ns, mb, ncg, waves, rpw) of the row-streaming kernel: tk =
# 64, stride 1, input rows of at most 32*mb positions, Nc rounded up to 16
# equal to 16*ncg, `waves` waves of which each pair takes rpw rows of a
# group (wr = rpw*waves/2 rows per group); a tile is L whole output rows of
# one image (tp = L*Nh, L | Nw).  Where several fit, the lowest id.
ROWS = [
    (1500, BF16, 3, 3, 1, 4, 8, 1), (1501, BF16, 3, 3, 1, 2, 8, 1),
    (1502, BF16, 3, 3, 2, 4, 8, 1), (1503, BF16, 3, 3, 2, 2, 8, 1),
    (1504, BF16, 1, 1, 2, 4, 8, 1),
    (1600, BF16_OBF16, 3, 3, 1, 4, 8, 1), (1601, BF16_OBF16, 3, 3, 1, 2, 8, 1),
    (1602, BF16_OBF16, 3, 3, 2, 4, 8, 1), (1603, BF16_OBF16, 3, 3, 2, 2, 8, 1),
    (1604, BF16_OBF16, 1, 1, 2, 4, 8, 1),
]


# (id, dtype, wp, wk, mbp, nbk, tc, s2) of the 1x1 GEMM kernel: tk =
# 32*wk*nbk, tp <= 32*wp*mbp (a multiple of 4), Nc % 8 == 0; s2 = 0: strides
# 1 and Nw*Nh % 4 == 0; s2 = 1: strides 2 and 2, Nh % 4 == 0; s2 = 2: strides
# 1, a tile is one image (tp = Nw*Nh <= 32*wp*mbp - 8, Nw*Nh % 4 == 0), LDS
# a ring of 4 stages.
GEMM1 = [
    (1700, BF16, 2, 4, 4, 2, 64, 0), (1701, BF16, 4, 2, 2, 2, 64, 0),
    (1702, BF16, 2, 4, 4, 2, 32, 1), (1709, BF16, 2, 4, 4, 2, 32, 2),
    (1800, BF16_OBF16, 2, 4, 4, 2, 64, 0), (1801, BF16_OBF16, 4, 2, 2, 2, 64, 0),
    (1802, BF16_OBF16, 2, 4, 4, 2, 32, 1), (1809, BF16_OBF16, 2, 4, 4, 2, 32, 2),
]


# (id, dtype, nr, ns, L) of the stride-2 row-band kernel: tk = 256, tc = 16,
# strides 2 and 2, Nc % 16 == 0, Nh <= 32, Ny <= 64; a tile is
# L whole output rows of one image (tp = L*Nh, L | Nw); eight waves.
SROWS = [
    (1900, BF16, 3, 3, 7), (1901, BF16, 3, 3, 4),
    (2000, BF16_OBF16, 3, 3, 7), (2001, BF16_OBF16, 3, 3, 4),
]


def stream_grid(p: eq1.Problem, tk: int, tp: int, threads: int, lds: int, cus: int,
                lds_bytes: int, wg_per_cu: int) -> int:
    """Workgroups a streaming plan launches: its slots, at most its tiles."""
    slots = cus * max(1, min(wg_per_cu * 256 // threads, lds_bytes // lds))
    return min(slots, -(-(p.Nb * p.Nw * p.Nh) // tp) * -(-p.Nk // tk))


def balanced_tp(p: eq1.Problem, tp_max: int, tk: int, slots: int, min_rounds: int = 1) -> int:
    """Outputs per tile: as many rounds of `slots` workgroups as tiles of
    tp_max outputs need, and within them the most (hence smallest, equal)
    tiles -- each processor's share N/P of Eq. (2).  Even, never below 32;
    min_rounds > 1 asks for that many tiles per slot (persistent kernels)."""
    npix = p.Nb * p.Nw * p.Nh
    nk = -(-p.Nk // tk)
    rounds = max(min_rounds, -(-(-(-npix // tp_max) * nk) // slots))
    ptiles = max(1, (rounds * slots) // nk)
    tp = -(-npix // ptiles)
    if tp % 2:
        tp += 1
    return min(tp_max, max(tp, min(tp_max, 32)))


def _max_slab(p: eq1.Problem, tp: int) -> int:
    n = p.Nb * p.Nw * p.Nh
    return max(eq1.slab_rows(p, f, min(f + tp, n) - 1) for f in range(0, n, tp))


def _cost(p, dtype, tk, tp, tc, lds, cus, lds_bytes, wg_per_cu):
    e_in = 4 if dtype == F32 else 2
    e_out = 2 if dtype == BF16_OBF16 else 4
    rate = 256.0 if dtype == F32 else 4096.0
    RS = p.Nr * p.Ns
    npix = p.Nb * p.Nw * p.Nh
    tiles = math.ceil(npix / tp) * math.ceil(p.Nk / tk)
    occ = max(1, min(lds_bytes // lds, wg_per_cu))
    slots = cus * occ
    rounds = math.ceil(tiles / slots)
    o, k, i = eq1.slab_terms(p, tk, tp)
    nbytes = e_out * o + e_in * (k + i)
    tile_flops = 2.0 * tk * tp * (math.ceil(p.Nc / tc) * tc) * RS
    tile_clk = max(tile_flops / rate, (nbytes / tiles) / 64.0)
    return rounds * slots / cus * tile_clk, {"grid": tiles, "lds": lds, "bytes": nbytes,
                                             "terms": (o, k, i)}


def candidates(p: eq1.Problem, dtype: int, cus: int, lds_bytes: int, acc_regs: int,
               wg_per_cu: int, tier: int = 2):
    """Yield (time, tk, tp, tc, id, info) for every feasible candidate of a tier."""
    RS = p.Nr * p.Ns
    e_out = 2 if dtype == BF16_OBF16 else 4
    if tier == 0:
        for vid, dt, wm, wn, mb, nb, tc, nr, ns, maxi in IGEMM4:
            if dt != dtype or (nr > 0 and (nr, ns) != (p.Nr, p.Ns)):
                continue
            tk, tp, acc = 32 * wm * mb, 32 * wn * nb, 16 * mb * nb
            S = _max_slab(p, tp)
            if (tc // 8) * math.ceil(S * p.Ny / 8) > 256 * maxi:
                continue
            imgs = tp // (p.Nw * p.Nh) + 2
            if ((imgs * p.Nc + tc) * p.Nx * p.Ny * 2 >= 2 ** 31
                    or imgs * p.Nk * p.Nw * p.Nh * e_out >= 2 ** 31):
                continue
            blk = math.ceil(RS * (tc // 8) * tk / 256) * 256
            sn8 = math.ceil(S * p.Ny / 8) * 8
            lds = 2 * ((tc // 8) * sn8 + blk) * 16
            if lds > lds_bytes or acc > acc_regs:
                continue
            t, info = _cost(p, dtype, tk, tp, tc, lds, cus, lds_bytes, wg_per_cu)
            yield t, tk, tp, tc, vid, info
        nbr = (p.Ny + 14) // 8
        for vid, dt, wm, wn, mb, nb, tc, nr, ns, nbuf, ndi, ndk, mpos in IGEMM3:
            if dt != dtype or (nr > 0 and (nr, ns) != (p.Nr, p.Ns)):
                continue
            tk, tp, acc = 32 * wm * mb, 32 * wn * nb, 16 * mb * nb
            S = _max_slab(p, tp)
            if (tc * S * nbr > 256 * ndi or RS * (tc // 8) * tk > 256 * ndk
                    or S * p.Ny > 256 * mpos):
                continue
            imgs = tp // (p.Nw * p.Nh) + 2
            if ((imgs * p.Nc + tc) * p.Nx * p.Ny * 2 >= 2 ** 31
                    or imgs * p.Nk * p.Nw * p.Nh * e_out >= 2 ** 31):
                continue
            lds = ((tc // 8) * S * p.Ny + nbuf * 256 * (ndi + ndk)) * 16
            if lds > lds_bytes or acc > acc_regs:
                continue
            t, info = _cost(p, dtype, tk, tp, tc, lds, cus, lds_bytes, wg_per_cu)
            yield t, tk, tp, tc, vid, info
        return
    if tier == 1:
        for vid, dt, wm, wn, mb, nb, tc, nr, ns, maxp, rawk, pw in IGEMM2:
            if dt != dtype or (nr > 0 and (nr, ns) != (p.Nr, p.Ns)):
                continue
            if rawk and (p.Nc % 8 or (p.Nk + 512) * p.Nc * RS * 2 >= 2 ** 31):
                continue
            tk, tp_max, acc = 32 * wm * mb, 32 * wn * nb, 16 * mb * nb
            if rawk:
                row = RS * tc // 8
                row += 1 - row % 2
                blk = math.ceil(tk * row / 64) * 64
            else:
                blk = math.ceil(RS * (tc // 8) * tk / 256) * 256

            def lds_of(S, t):
                per_group = (t + 1) // 2 * 2 if pw else (S * p.Ny + 1) // 2 * 2
                return 2 * ((tc // 8) * per_group + blk) * 16

            wgs = max(1, min(wg_per_cu, lds_bytes // lds_of(_max_slab(p, tp_max), tp_max)))
            tp = balanced_tp(p, tp_max, tk, cus * wgs)
            S = _max_slab(p, tp)
            if math.ceil((tp if pw else S * p.Ny) / 2) > 256 * maxp:
                continue
            imgs = tp_max // (p.Nw * p.Nh) + 2
            if (imgs * p.Nc * p.Nx * p.Ny * 2 >= 2 ** 31
                    or imgs * p.Nk * p.Nw * p.Nh * e_out >= 2 ** 31):
                continue
            lds = lds_of(S, tp)
            if lds > lds_bytes or acc > acc_regs:
                continue
            t, info = _cost(p, dtype, tk, tp, tc, lds, cus, lds_bytes, wg_per_cu)
            yield t, tk, tp, tc, vid, info
        for vid, dt, wm, wn, mb, nb, tc, nr, ns, kres, mpos, ndma in STREAM:
            if dt != dtype or (nr, ns) != (p.Nr, p.Ns) or p.Nc % 8:
                continue
            tk, tp_max, acc, threads = 32 * wm * mb, 32 * wn * nb, 16 * mb * nb, 64 * wm * wn
            if kres and p.Nk > tk:
                continue
            if ((p.Nk + 512) * p.Nc * RS * 2 >= 2 ** 31 or p.Nb * p.Nc * p.Nx * p.Ny * 2 >= 2 ** 31
                    or p.Nb * p.Nk * p.Nw * p.Nh * e_out >= 2 ** 31):
                continue
            rc = (RS * tc // 8) | 1
            kvecs = -(-(tk * rc) // 64) * 64
            n_cc = -(-p.Nc // tc)

            nbr = (p.Ny + 14) // 8

            ker_vecs = n_cc * RS * (tc // 8) * tk if kres else 2 * kvecs

            def lds_t(S):
                return (2 * threads * ndma + (tc // 8) * S * p.Ny + ker_vecs) * 16

            lds_full = lds_t(_max_slab(p, tp_max))
            slots = cus * max(1, min(wg_per_cu * 256 // threads, lds_bytes // lds_full))
            tp = balanced_tp(p, tp_max, tk, slots, 2)
            S = _max_slab(p, tp)
            if S * p.Ny > threads * mpos or tc * S * nbr > threads * ndma:
                continue
            lds = lds_t(S)
            if lds > lds_bytes or acc > acc_regs:
                continue
            t, info = _cost(p, dtype, tk, tp, tc, lds, cus, lds_bytes, wg_per_cu)
            yield t, tk, tp, tc, vid, info
        for vid, dt, nb, ks in SMALLC:
            if dt != dtype or p.Ns > 8 or -(-(p.Nc * p.Nr) // 2) > ks:
                continue
            if (p.Nb * p.Nc * p.Nx * p.Ny * 2 >= 2 ** 31 or p.Nk * p.Nc * RS * 2 >= 2 ** 31):
                continue
            tk, tp_max, acc = 64, 128 * nb, 32 * nb
            if (tp_max // (p.Nw * p.Nh) + 2) * p.Nk * p.Nw * p.Nh * e_out >= 2 ** 31:
                continue

            def lds_s(S):
                return ks * 2 * 64 * 16 + p.Nc * S * (p.Ny + 8) * 2

            wgs = max(1, min(wg_per_cu, lds_bytes // lds_s(_max_slab(p, tp_max))))
            tp = balanced_tp(p, tp_max, tk, cus * wgs)
            lds = lds_s(_max_slab(p, tp))
            if lds > lds_bytes or acc > acc_regs:
                continue
            t, info = _cost(p, dtype, tk, tp, p.Nc, lds, cus, lds_bytes, wg_per_cu)
            yield t, tk, tp, p.Nc, vid, info
        return
    kv = 1 if dtype == F32 else 8
    vec = 4 if dtype == F32 else 16
    for vid, dt, wm, wn, mb, nb, tc in IGEMM:
        if dt != dtype:
            continue
        tk, tp, acc = 32 * wm * mb, 32 * wn * nb, 16 * mb * nb
        S = _max_slab(p, tp)
        groups = tc // kv
        lds = (groups * S * p.Ny + RS * groups * tk) * vec
        if lds > lds_bytes or acc > acc_regs:
            continue
        t, info = _cost(p, dtype, tk, tp, tc, lds, cus, lds_bytes, wg_per_cu)
        yield t, tk, tp, tc, vid, info


def _special(p: eq1.Problem, dtype: int, cus: int, lds_bytes: int, acc_regs: int,
             wg_per_cu: int):
    """(kernel, id, tk, tp, tc) of the specialized tier, or None."""
    e_out = 2 if dtype == BF16_OBF16 else 4
    lds_cap = min(lds_bytes, 160 * 1024)
    out_big = p.Nb * p.Nk * p.Nw * p.Nh * e_out >= 2 ** 31
    # 1x1 GEMM: In planes of Nx x Ny for 1x1 taps
    for vid, dt, wp, wk, mbp, nbk, tc, s2 in GEMM1:
        if dt != dtype or p.Nr != 1 or p.Ns != 1 or p.Nc % 8:
            continue
        if s2 == 1 and not (p.sw == 2 and p.sh == 2 and p.Nh % 4 == 0):
            continue
        if s2 != 1 and not (p.sw == 1 and p.sh == 1 and (p.Nw * p.Nh) % 4 == 0):
            continue
        tk, tpmax, acc = 32 * wk * nbk, 32 * wp * mbp, 16 * mbp * nbk
        if s2 == 2 and p.Nw * p.Nh > tpmax - 8:
            continue
        if s2 == 2:  # four stages of whole 512-unit copy rounds (16-byte units)
            units = tk * 4 + tc * (((tpmax - 8) // 8) | 1)
            nt = 64 * wp * wk
            lds = 4 * -(-units // nt) * nt * 16
        else:
            lds = 2 * (tc * (tpmax + 16) + tk * (tc + 8)) * 2
        nx, ny = p.sw * (p.Nw - 1) + 1, p.sh * (p.Nh - 1) + 1
        if (lds > lds_cap or p.Nb * p.Nc * nx * ny * 2 >= 2 ** 30
                or p.Nk * p.Nc * 2 >= 2 ** 30 or out_big):
            continue
        occ = max(1, min(wg_per_cu, lds_bytes // lds))
        tp = min(tpmax, -(-balanced_tp(p, tpmax, tk, cus * occ, 1) // 4) * 4)
        if s2 == 2:
            tp = p.Nw * p.Nh
        if tp % 4 or tp < 4 or acc > acc_regs:
            continue
        return (11, vid, tk, tp, tc)
    # stride-1 row streaming
    for vid, dt, nr, ns, mb, ncg, waves, rpw in ROWS:
        if (dt != dtype or (nr, ns) != (p.Nr, p.Ns) or p.sw != 1 or p.sh != 1 or p.Nc % 8
                or -(-p.Nc // 16) * 16 != 16 * ncg or p.Nh + p.Ns - 1 > 32 * mb):
            continue
        if (p.Nb * p.Nc * p.Nx * p.Ny * 2 >= 2 ** 31 or p.Nk * p.Nc * nr * ns * 2 >= 2 ** 31
                or out_big):
            continue
        wr, nt, ncp = rpw * waves // 2, 64 * waves, 16 * ncg
        ring = (2 * wr + nr - 1) * ncp * 32 * mb * 2
        copies = -(-(64 * ncp * nr * ns // 8) // nt)
        plane = 66 if ring >= copies * nt * 16 else 64   # padded B-operand planes
        lds = ncg * nr * ns * 2 * plane * 16 + ring
        acc = 16 * mb * ns * rpw
        if lds > lds_cap or acc > acc_regs * 8 // waves:
            continue
        nk = -(-p.Nk // 64)
        band, best = 0, None
        for l in range(1, p.Nw + 1):
            if p.Nw % l:
                continue
            rounds = -(-(p.Nb * (p.Nw // l) * nk) // cus) * -(-l // wr)
            if best is None or rounds <= best:
                band, best = l, rounds
        return (10, vid, 64, band * p.Nh, p.Nc)
    # stride-2 row bands
    pick = None
    for vid, dt, nr, ns, L in SROWS:
        if (dt != dtype or (nr, ns) != (p.Nr, p.Ns) or p.sw != 2 or p.sh != 2 or p.Nc % 16
                or p.Nh > 32 or p.Ny > 64 or p.Nw % L):
            continue
        rows = 2 * (L - 1) + nr if nr >= 2 else L
        blk = -(-(nr * ns * 2 * 256) // 256) * 256
        ws = -(-p.Nk // 256) * (p.Nc // 16) * blk * 16
        lds = (4 * ns * 2 * 256 + 2 * 2 * rows * 64) * 16
        acc = 32 * ((L + 1) // 2) - 16 * (L % 2)
        if (p.Nb * p.Nc * p.Nx * p.Ny * 2 >= 2 ** 31 or ws >= 2 ** 31 or out_big
                or lds > lds_cap or acc > acc_regs):
            continue
        if pick is None or L > pick[0]:
            pick = (L, vid)
    if pick is not None:
        return (12, pick[1], 256, pick[0] * p.Nh, 16)
    return None


def choose(p: eq1.Problem, dtype: int, cus=256, lds_bytes=160 * 1024, acc_regs=128,
           wg_per_cu=2):
    """(kernel, variant id, tk, tp, tc) the rule above selects; kernels 11,
    10 and 12 are the specialized 1x1 GEMM, row-streaming and stride-2 row-band
    families, 7 the wide-staging family, 6 the DMA-staged one, 5 the register-staged
    pipelined one (8 when it stages raw Ker rows, 3 for its 1x1 gather),
    4 the few-channel one, 9 the persistent streaming one, 2 the plain
    staging one, 1 the direct kernel."""
    special = _special(p, dtype, cus, lds_bytes, acc_regs, wg_per_cu)
    if special is not None:
        return special
    rawk_ids = {row[0] for row in IGEMM2 if row[10]}
    pw_ids = {row[0] for row in IGEMM2 if row[11]}
    best = None
    for tier in (0, 1, 2):
        for t, tk, tp, tc, vid, info in candidates(p, dtype, cus, lds_bytes, acc_regs,
                                                   wg_per_cu, tier):
            key = (t, -tk, -tp, -tc, vid)
            if best is None or key < best[0]:
                if tier == 0:
                    kern = 7 if vid >= 800 else 6
                elif tier == 1:
                    if vid >= 1300:
                        kern = 9
                    elif vid >= 1000:
                        kern = 4
                    else:
                        kern = 3 if vid in pw_ids else (8 if vid in rawk_ids else 5)
                else:
                    kern = 2
                best = (key, (kern, vid, tk, tp, tc))
        if best is not None:
            break
    if best is None:
        return (1, 1, 1, 1, p.Nc)
    return best[1]

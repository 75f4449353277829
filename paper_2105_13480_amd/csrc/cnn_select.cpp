// Tile-size selection from the paper's data-movement model (Sec. 2, Eq. (1)).
//
// For every kernel instantiation of the requested dtype the selector
//   1. computes the tile footprint -- the halo'd In slab and the Ker tile in
//      LDS, the Out tile in accumulator registers (the two halves of the
//      paper's fast memory M) -- and drops tilings that exceed the budget;
//   2. evaluates Eq. (1) for that tiling: Out written once, Ker re-read once
//      per (b,w,h) tile, the halo'd In slab re-read once per k tile (exact
//      halo, edge tiles clipped), in bytes;
//   3. turns it into a time: a CU processes ceil(tiles / slots) rounds of
//      `slots / cus` tiles, each tile bound by its MFMA work (padded to
//      whole MFMA blocks) or its share of the Eq. (1) traffic, whichever is
//      larger.  This accounts for the P processors of Eq. (2) that the
//      sequential Eq. (1) leaves out: a tiling with fewer tiles than
//      workgroup slots leaves CUs idle however little data it moves.
// The smallest time wins; ties go to the larger tk, then the larger tp,
// then the larger tc, then the lower instantiation id.  The pipelined bf16
// kernel (conv_igemm2) is tier 1; the plain staging kernel (conv_igemm) is
// considered only when no tier-1 instantiation fits; the direct kernel
// takes problems no implicit-GEMM tiling fits.
#include <math.h>
#include <cmath>
#include <string.h>

#include <algorithm>
#include <vector>

#include "internal.h"

namespace cnnlib {

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Walk the composite tiles of tp outputs; return the largest slab and
// (optionally) the total number of slab rows over all tiles.
static int64_t walk_slabs(const cnn_problem& p, int64_t tp, int64_t* total_rows) {
  const int64_t hw = p.Nw * p.Nh;
  const int64_t npix = p.Nb * hw;
  const int64_t Nx = p.sw * (p.Nw - 1) + p.Nr;
  int64_t mx = 0, tot = 0;
  for (int64_t f = 0; f < npix; f += tp) {
    const int64_t last = std::min(f + tp, npix) - 1;
    const int64_t b0 = f / hw, w0 = (f % hw) / p.Nh;
    const int64_t b1 = last / hw, w1 = (last % hw) / p.Nh;
    const int64_t S = (b1 * Nx + p.sw * w1 + p.Nr) - (b0 * Nx + p.sw * w0);
    mx = std::max(mx, S);
    tot += S;
  }
  if (total_rows) *total_rows = tot;
  return mx;
}

int64_t slab_rows_max(const cnn_problem& p, int64_t tp) { return walk_slabs(p, tp, nullptr); }

void slab_terms(const cnn_problem& p, int64_t tk, int64_t tp, double terms[3]) {
  const int64_t npix = p.Nb * p.Nw * p.Nh;
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  int64_t rows = 0;
  walk_slabs(p, tp, &rows);
  terms[0] = (double)(npix * p.Nk);
  terms[1] = (double)(ceil_div(npix, tp) * p.Nk * p.Nc * p.Nr * p.Ns);
  terms[2] = (double)ceil_div(p.Nk, tk) * (double)(p.Nc * Ny) * (double)rows;
}

void eq1_terms(const cnn_problem& p, const cnn_tiles& t, int exact, double terms[3],
               double* footprint) {
  const double Nb = (double)p.Nb, Nc = (double)p.Nc, Nk = (double)p.Nk, Nw = (double)p.Nw,
               Nh = (double)p.Nh, Nr = (double)p.Nr, Ns = (double)p.Ns, sw = (double)p.sw,
               sh = (double)p.sh;
  terms[0] = Nb * Nk * Nw * Nh;
  if (!exact) {
    terms[1] = Nk * Nc * Nr * Ns * Nw * Nh * Nb / ((double)t.Tw * t.Th * t.Tb);
    terms[2] = Nb * Nc * (sw * t.Tw + Nr - 1) * (sh * t.Th + Ns - 1) * Nw * Nh * Nk /
               ((double)t.Tw * t.Th * t.Tk);
    if (footprint)
      *footprint = (sw * t.Tw + Nr - 1) * (sh * t.Th + Ns - 1) * t.Tb * t.Tc +
                   (double)t.Tw * t.Th * t.Tb * t.Tk + Nr * Ns * t.Tk * t.Tc;
    return;
  }
  // Exact: ceil tile counts, clipped edge tiles, halo sigma*(T-1) + R.
  const int64_t nb = ceil_div(p.Nb, t.Tb), nw = ceil_div(p.Nw, t.Tw), nh = ceil_div(p.Nh, t.Th);
  terms[1] = (double)(nb * nw * nh) * (double)(p.Nk * p.Nc * p.Nr * p.Ns);
  int64_t xs = 0, ys = 0;
  for (int64_t i = 0; i < p.Nw; i += t.Tw) xs += p.sw * (std::min(t.Tw, p.Nw - i) - 1) + p.Nr;
  for (int64_t i = 0; i < p.Nh; i += t.Th) ys += p.sh * (std::min(t.Th, p.Nh - i) - 1) + p.Ns;
  terms[2] = (double)ceil_div(p.Nk, t.Tk) * (double)(p.Nc * p.Nb) * (double)xs * (double)ys;
  if (footprint)
    *footprint = (double)(p.sw * (t.Tw - 1) + p.Nr) * (double)(p.sh * (t.Th - 1) + p.Ns) *
                     (double)(t.Tb * t.Tc) +
                 (double)(t.Tw * t.Th * t.Tb * t.Tk) + (double)(p.Nr * p.Ns * t.Tk * t.Tc);
}

// Byte ranges each family addresses with 32-bit buffer offsets (the kernels
// clamp their buffer descriptors just below 2 GiB): a plan outside them is
// never made, and a plan handed in is rejected (plan_ranges_ok).
static const int64_t k2G = 1LL << 31;

static int64_t in_elems(const cnn_problem& p) {
  return p.Nb * p.Nc * (p.sw * (p.Nw - 1) + p.Nr) * (p.sh * (p.Nh - 1) + p.Ns);
}

// images a tile of up to tp outputs touches, plus one of slack each side
static int64_t tile_images(const cnn_problem& p, int64_t tp) { return tp / (p.Nw * p.Nh) + 2; }

bool ranges_ok_tile(const cnn_problem& p, int dtype, int64_t tp, int64_t tc_extra) {
  const int64_t Nx = p.sw * (p.Nw - 1) + p.Nr, Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t imgs = tile_images(p, tp);
  return (imgs * p.Nc + tc_extra) * Nx * Ny * 2 < k2G &&
         imgs * p.Nk * p.Nw * p.Nh * out_bytes(dtype) < k2G;
}

bool ranges_ok_rawk(const cnn_problem& p) {
  // Ker rows up to Nk + tk + 64 are addressed
  return (p.Nk + 512) * p.Nc * p.Nr * p.Ns * 2 < k2G;
}

bool ranges_ok_whole(const cnn_problem& p, int dtype, int64_t in_limit) {
  return in_elems(p) * 2 < in_limit && p.Nk * p.Nc * p.Nr * p.Ns * 2 < in_limit &&
         p.Nb * p.Nk * p.Nw * p.Nh * out_bytes(dtype) < k2G;
}

bool ranges_ok_smallc(const VariantS& v, const cnn_problem& p, int dtype) {
  return in_elems(p) * 2 < k2G && p.Nk * p.Nc * p.Nr * p.Ns * 2 < k2G &&
         tile_images(p, v.tp) * p.Nk * p.Nw * p.Nh * out_bytes(dtype) < k2G;
}

bool ranges_ok_srows(const VariantQ& v, const cnn_problem& p, int dtype) {
  // (the raw-Ker form addresses Ker up to the end of the last 256-feature
  // range, and puts Out offsets up to 288 features past the end in the
  // scalar offset beside an out-of-range lane offset)
  const int64_t ker_end = (p.Nk + 255) / 256 * 256 * p.Nc * p.Nr * p.Ns * 2;
  return in_elems(p) * 2 < k2G && srows_ws_bytes(v, p) < k2G && ker_end < k2G &&
         (p.Nb * p.Nk + 288) * p.Nw * p.Nh * out_bytes(dtype) < k2G;
}

static double model_us(const cnn_plan_t& pl, const cnn_budget& bud, double w_out);

// Plan fields shared by the implicit-GEMM families (the model's time is set
// once the plan is complete).
static bool eval_tiling(const cnn_problem& p, int dtype, int id, int64_t tk, int64_t tp,
                        int64_t tc, int64_t acc, int64_t S, int64_t lds, int64_t ws,
                        const cnn_budget& bud, cnn_plan_t* plan) {
  const int64_t RS = p.Nr * p.Ns;
  const int64_t npix = p.Nb * p.Nw * p.Nh;
  if (lds > bud.lds_bytes || acc > bud.acc_regs) return false;
  const int64_t n_p = ceil_div(npix, tp), n_k = ceil_div(p.Nk, tk);
  const int64_t grid = n_p * n_k;
  if (grid > 0x7fffffffLL) return false;

  double terms[3];
  slab_terms(p, tk, tp, terms);
  const double e_in = in_bytes(dtype), e_out = out_bytes(dtype);
  const double bytes = e_out * terms[0] + e_in * (terms[1] + terms[2]);
  const double tile_flops =
      2.0 * tk * tp * (double)(ceil_div(p.Nc, tc) * tc) * (double)RS;

  memset(plan, 0, sizeof(*plan));
  plan->prob = p;
  plan->dtype = dtype;
  plan->kernel = CNN_K_IGEMM;
  plan->variant = id;
  plan->tk = tk;
  plan->tp = tp;
  plan->tc = tc;
  plan->grid = grid;
  plan->lds_bytes = lds;
  plan->slab_rows = S;
  plan->ws_bytes = ws;
  for (int i = 0; i < 3; ++i) plan->eq1_elems[i] = terms[i];
  plan->eq1_bytes = bytes;
  plan->mfma_flops = tile_flops * (double)grid;
  return true;
}

// Plain staging kernel (conv_igemm).
static bool eval_variant(const cnn_problem& p, int dtype, const Variant& v,
                         const cnn_budget& bud, cnn_plan_t* plan) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t S = slab_rows_max(p, v.tp);
  const int64_t lds = igemm_lds_bytes(v, S, Ny, p.Nr * p.Ns);
  return eval_tiling(p, dtype, v.id, v.tk, v.tp, v.tc, v.acc, S, lds, 0, bud, plan);
}

// Wide-staging pipelined kernel (conv_igemm4).
static bool eval_variant4(const cnn_problem& p, int dtype, const Variant4& v,
                          const cnn_budget& bud, cnn_plan_t* plan) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t S = slab_rows_max(p, v.tp);
  if (!igemm4_fits(v, p, S) || !ranges_ok_tile(p, dtype, v.tp, v.tc)) return false;
  const int64_t lds = igemm4_lds_bytes(v, S, Ny, p.Nr * p.Ns);
  return eval_tiling(p, dtype, v.id, v.tk, v.tp, v.tc, v.acc, S, lds, igemm4_ws_bytes(v, p),
                     bud, plan);
}

// DMA-staged kernel (conv_igemm3).
static bool eval_variant3(const cnn_problem& p, int dtype, const Variant3& v,
                          const cnn_budget& bud, cnn_plan_t* plan) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t S = slab_rows_max(p, v.tp);
  if (!igemm3_fits(v, p, S) || !ranges_ok_tile(p, dtype, v.tp, v.tc)) return false;
  const int64_t lds = igemm3_lds_bytes(v, S, Ny);
  return eval_tiling(p, dtype, v.id, v.tk, v.tp, v.tc, v.acc, S, lds, igemm3_ws_bytes(v, p),
                     bud, plan);
}

// Outputs per tile for a kernel whose tiles hold up to TP outputs: the
// fewest rounds of `slots` concurrent workgroups that TP-output tiles need,
// then the smallest tile that still fits in those rounds, so every
// workgroup of every round gets the same share (the P processors of
// Eq. (2) each take N/P).  Rounded up to an even count (the kernels stage
// outputs in pairs), at least 32 outputs (one MFMA block).  min_rounds > 1
// asks for at least that many tiles per slot (persistent kernels).
int64_t balanced_tp(const cnn_problem& p, int64_t TP, int64_t tk, int64_t slots,
                    int64_t min_rounds) {
  const int64_t npix = p.Nb * p.Nw * p.Nh;
  const int64_t n_k = ceil_div(p.Nk, tk);
  const int64_t rounds = std::max(min_rounds, ceil_div(ceil_div(npix, TP) * n_k, slots));
  const int64_t ptiles = std::max<int64_t>(1, rounds * slots / n_k);
  int64_t tp = ceil_div(npix, ptiles);
  tp += tp & 1;
  return std::min(TP, std::max<int64_t>(tp, std::min<int64_t>(TP, 32)));
}

// Kernel family of a pipelined-kernel instantiation.
int v2_family(const Variant2& v) {
  return v.pw ? CNN_K_POINTWISE : v.rawk ? CNN_K_IGEMM_RAWK : CNN_K_IGEMM_PIPE;
}

// Pipelined kernel (conv_igemm2): its stencil must match a compile-time one
// (or be generic) and its slab must fit the per-thread staging registers;
// raw-Ker instantiations need Nc % 8 == 0 and Ker well below 2 GiB.
static bool eval_variant2(const cnn_problem& p, int dtype, const Variant2& v,
                          const cnn_budget& bud, cnn_plan_t* plan) {
  if (v.nr > 0 && (v.nr != p.Nr || v.ns != p.Ns)) return false;
  // (rows up to Nk + tk + 64 are addressed with 32-bit byte offsets)
  if (v.rawk && (p.Nc % 8 != 0 || !ranges_ok_rawk(p))) return false;
  if (!ranges_ok_tile(p, dtype, v.tp, 0)) return false;
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t lds_full = igemm2_lds_bytes(v, slab_rows_max(p, v.tp), Ny, p.Nr * p.Ns, v.tp);
  const int64_t occ = std::max<int64_t>(1, std::min<int64_t>(bud.wg_per_cu, bud.lds_bytes / lds_full));
  const int64_t tp = balanced_tp(p, v.tp, v.tk, bud.cus * occ, 1);
  const int64_t S = slab_rows_max(p, tp);
  const int64_t pairs = v.pw ? (tp + 1) / 2 : (S * Ny + 1) / 2;
  if (pairs > 256 * (int64_t)v.maxp) return false;
  const int64_t lds = igemm2_lds_bytes(v, S, Ny, p.Nr * p.Ns, tp);
  return eval_tiling(p, dtype, v.id, v.tk, tp, v.tc, v.acc, S, lds, igemm2_ws_bytes(v, p),
                     bud, plan);
}

// Few-channel kernel (conv_smallc): the flattened (c, r) rows must fit the
// registers' K-steps, the stencil at most 8 wide, the slab in LDS, and the
// tensors the 32-bit offsets.
static bool eval_smallc(const cnn_problem& p, int dtype, const VariantS& v, const cnn_budget& bud, cnn_plan_t* plan) {
  if (p.Ns > 8 || (p.Nc * p.Nr + 1) / 2 > v.ks || !smallc_stencil_ok(v, p) ||
      !ranges_ok_smallc(v, p, dtype))
    return false;
  const int64_t lds_full = smallc_lds_bytes(v, p, slab_rows_max(p, v.tp));
  const int64_t occ = std::max<int64_t>(1, std::min<int64_t>(bud.wg_per_cu, bud.lds_bytes / lds_full));
  const int64_t tp = balanced_tp(p, v.tp, v.tk, bud.cus * occ, 1);
  const int64_t S = slab_rows_max(p, tp);
  const int64_t lds = smallc_lds_bytes(v, p, S);
  // one stage holds every channel (tc = Nc)
  return eval_tiling(p, dtype, v.id, v.tk, tp, p.Nc, v.acc, S, lds, 0, bud, plan);
}

// Row-streaming kernel (conv_rows): stride 1, fixed stencil, Nc % 8 == 0,
// input rows of at most 32*mb positions; a tile is L whole output rows of
// one image (L divides Nw, tp = L*Nh) by 64 features, all Nc channels.
static bool eval_rows(const cnn_problem& p, int dtype, const VariantR& v, const cnn_budget& bud,
                      int64_t L, cnn_plan_t* plan) {
  if (!rows_fits(v, p) || !ranges_ok_whole(p, dtype, k2G)) return false;
  const int64_t lds = rows_lds_bytes(v, p);
  if (lds > std::min<int64_t>(bud.lds_bytes, 160 * 1024)) return false;
  if (L < 1 || p.Nw % L) return false;
  const int64_t tp = L * p.Nh;
  // the accumulator budget is per lane at two waves per SIMD (8 per
  // workgroup); a 4-wave workgroup (one wave per SIMD) has twice the registers
  cnn_budget b2 = bud;
  b2.acc_regs = bud.acc_regs * 8 / v.waves;
  if (!eval_tiling(p, dtype, v.id, v.tk, tp, p.Nc, v.acc, L + p.Nr - 1, lds, 0, b2, plan))
    return false;
  // the products run over whole 32-position blocks of the input row and
  // 16-channel groups, every tap at unshifted positions
  plan->mfma_flops = 2.0 * (double)(ceil_div(p.Nk, v.tk) * v.tk) * (double)(p.Nb * p.Nw) *
                     (double)(32 * v.mb) * (double)(16 * v.ncg) * (double)(p.Nr * p.Ns);
  return true;
}

// 1x1 stride-1 GEMM kernel (conv_gemm1): tiles of tp consecutive pixels
// (a multiple of 4, balanced over the CUs) by tk features.
static bool eval_gemm1(const cnn_problem& p, int dtype, const VariantG& v, const cnn_budget& bud, cnn_plan_t* plan) {
  const int64_t lds = gemm1_lds_bytes(v);
  if (lds > std::min<int64_t>(bud.lds_bytes, 160 * 1024)) return false;
  if (!ranges_ok_whole(p, dtype, 1LL << 30)) return false;
  const int64_t occ = std::max<int64_t>(1, std::min<int64_t>(bud.wg_per_cu, bud.lds_bytes / lds));
  int64_t tp = balanced_tp(p, v.tp, v.tk, bud.cus * occ, 1);
  tp = std::min<int64_t>(v.tp, (tp + 3) / 4 * 4);
  if (v.s2 == 2) tp = p.Nw * p.Nh;  // a tile is one image
  if (!gemm1_fits(v, p, tp)) return false;
  return eval_tiling(p, dtype, v.id, v.tk, tp, v.tc, v.acc, 1, lds, 0, bud, plan);
}

// Stride-2 row-band kernel (conv_srows): fixed stencil, tiles of the
// instantiation's L whole output rows of one image by 256 features, 16
// channels per chunk, Ker repacked into the workspace.
static bool eval_srows(const cnn_problem& p, int dtype, const VariantQ& v, const cnn_budget& bud, cnn_plan_t* plan) {
  if (!srows_fits(v, p) || !ranges_ok_srows(v, p, dtype)) return false;
  const int64_t ws = srows_ws_bytes(v, p);
  const int64_t lds = srows_lds_bytes(v);
  if (lds > std::min<int64_t>(bud.lds_bytes, 160 * 1024)) return false;
  // the accumulator budget is per lane at two waves per SIMD; a 4-wave
  // workgroup (one wave per SIMD) has twice the registers
  cnn_budget b2 = bud;
  b2.acc_regs = bud.acc_regs * 8 / v.waves;
  if (!eval_tiling(p, dtype, v.id, v.tk, v.L * p.Nh, 16, v.acc, srows_slab_rows(v), lds, ws,
                   b2, plan))
    return false;
  // a 32-position MFMA block per output row
  plan->mfma_flops = 2.0 * (double)(ceil_div(p.Nk, v.tk) * v.tk) * (double)(p.Nb * p.Nw * 32) *
                     (double)(p.Nc * p.Nr * p.Ns);
  if (v.form == 2) {
    // the raw-Ker form walks its 256 features as two 128-feature tiles in
    // turn, each streaming the band's In again: Eq. (1)'s In term is that
    // of 128-feature tiles
    double t[3];
    slab_terms(p, 128, v.L * p.Nh, t);
    plan->eq1_elems[2] = t[2];
    plan->eq1_bytes = out_bytes(dtype) * plan->eq1_elems[0] +
                      in_bytes(dtype) * (plan->eq1_elems[1] + plan->eq1_elems[2]);
  }
  return true;
}

// The XCD / L2 level the two-level model (Eq. (3) one level up) sees: 8 XCDs
// of one 4 MiB L2 each on MI355X.
static const int64_t kXcds = 8;
static const int64_t kL2Bytes = 4LL << 20;

// Rates of one MI355X the time model converts work and bytes with, all
// measured on the device (not datasheet figures): the engine clock; the
// bf16 MFMA rate sustained on operands of these workloads' value ranges
// (64 % of the 4096 flop/clk/CU datasheet rate: the clock drops with the
// data-dependent power; fp32 MFMA is taken at its datasheet rate); the HBM
// bandwidth of a large device copy (read plus write) and of a large fill
// (writes only); a kernel launch.
static const double kClkGHz = 2.4;
static const double kMfmaRealBf16 = 0.64;
static const double kHbmGBs = 5000.0;
static const double kFillGBs = 6900.0;
static const double kLaunchUs = 2.0;
// HBM writes per byte of Out of the stride-2 row-band kernels (row-piece
// stores, partial lines), measured with WRITE_SIZE.
static const double kSrowsWriteRate = 1.18;

// MFMA throughput per CU per clock for the dtype's operand type.
static double mfma_rate(int dtype) { return dtype == CNN_F32 ? 256.0 : 4096.0; }

// What each kernel family's implementation adds to the work and the bytes,
// fitted (least squares on log time) to every candidate of the seven
// benchmark workloads timed on one MI355X: the fraction of the sustained
// MFMA rate its inner loop reaches; a fixed cost per workgroup (set-up,
// the resident Ker tile); and the time of one channel stage when it is not
// MFMA-bound: a latency plus the stage's share of the Eq. (1) traffic at a
// per-CU bandwidth.
struct FamilyCost {
  double mfma_eff;      // of the sustained MFMA rate
  double wg_us;         // per workgroup
  double stage_us;      // per stage, latency
  double stage_gbs;     // per stage, Eq. (1) bytes per CU per second (GB/s)
};

static FamilyCost family_cost(int kernel, int variant) {
  switch (kernel) {
    case CNN_K_ROWS: return {0.73, 6.37, 0.01, 58.0};
    case CNN_K_SROWS: {
      int n = 0;
      const VariantQ* vq = variants_srows(&n);
      for (int i = 0; i < n; ++i) {
        if (vq[i].id != variant) continue;
        if (vq[i].form == 2) return {0.50, 4.30, 0.11, 48.3};   // Ker repacked on chip
        if (vq[i].form == 3) return {0.625, 1.43, 0.11, 48.3};  // B operands in registers
      }
      return {0.53, 1.39, 0.11, 48.3};
    }
    case CNN_K_GEMM1: {
      int n = 0;
      const VariantG* vg = variants_gemm1(&n);
      for (int i = 0; i < n; ++i)
        if (vg[i].id == variant && vg[i].s2 == 2) return {0.99, 1.22, 0.40, 50.0};  // DMA ring
      return {0.36, 1.28, 0.56, 50.1};
    }
    case CNN_K_SMALLC: {
      int n = 0;
      const VariantS* vs = variants_smallc(&n);
      for (int i = 0; i < n; ++i)
        if (vs[i].id == variant && vs[i].nc) return {0.17, 1.52, 0.17, 49.7};  // stencil compiled in
      return {0.17, 1.66, 0.17, 49.7};
    }
    case CNN_K_IGEMM_RAWK: return {0.49, 1.67, 2.41, 29.5};
    case CNN_K_POINTWISE: return {0.98, 37.19, 0.41, 100.0};
    case CNN_K_IGEMM_PIPE: return {0.74, 3.80, 2.51, 30.2};
    case CNN_K_IGEMM_DMA: return {0.55, 6.62, 0.93, 34.8};
    case CNN_K_IGEMM_WIDE: return {1.00, 0.00, 7.53, 100.0};
    case CNN_K_SPLITC: {
      int n = 0;
      const VariantC* vc = variants_cslice(&n);
      // a stage's loads at once; atomic sums cost 1.3 us more; the direct
      // form's 128-channel stages (one 1024-thread workgroup per CU) run
      // about 5 us each, bound by one CU's outstanding requests
      for (int i = 0; i < n; ++i)
        if (vc[i].id == variant)
          return {0.50, vc[i].mode == 1 ? 2.30 : 1.00, vc[i].mode == 2 ? 2.90 : 1.50, 50.0};
      return {0.51, 3.07, 1.65, 4.1};
    }
    case CNN_K_IGEMM: return {0.40, 0.00, 2.14, 3.4};
    default: return {0.25, 0.0, 0.0, 1.0};  // direct: fp32 vector FMAs
  }
}

// The bandwidth HBM sustains for a mix of reads and writes with write share
// w: a device copy's (half of each, or more reads) up to a fill's (writes
// only), linear in w.
static double hbm_gbs(double w) {
  return w <= 0.5 ? kHbmGBs : kHbmGBs + (kFillGBs - kHbmGBs) * (w - 0.5) / 0.5;
}

// The selector's time model for a finished plan, in microseconds.  The
// busiest CU runs ceil(workgroups / CUs) workgroups, up to `occ` of them at
// once (as LDS allows); each walks its channel stages, a stage taking the
// longer of its MFMA work and its latency plus its Eq. (1) bytes at the
// family's stage bandwidth.  The whole is at least the plan's HBM bytes
// (Eq. (3) at the XCD level), of which the share w_out is written, at the
// bandwidth of that mix.  Channel-split plans add their reduce pass; every
// plan adds its launch.
static double model_us(const cnn_plan_t& pl, const cnn_budget& bud, double w_out) {
  const cnn_problem& p = pl.prob;
  const FamilyCost fc = family_cost(pl.kernel, pl.variant);
  const double clk_per_us = kClkGHz * 1e3;
  const double cus = (double)bud.cus;
  const double n_out = (double)(p.Nb * p.Nk * p.Nw * p.Nh);
  if (pl.kernel == CNN_K_DIRECT) {
    // 64 lanes x 4 SIMDs x one fp32 FMA (2 flops) per clock per CU
    const double t = pl.flops / (cus * 512.0 * clk_per_us * fc.mfma_eff);
    return std::max(t, pl.hbm_bytes / (hbm_gbs(w_out) * 1e3)) + kLaunchUs;
  }
  const double kc = pl.kernel == CNN_K_SPLITC ? (double)pl.kc : 1.0;
  const double wgs = (double)pl.grid * kc;
  const double per_cu = std::ceil(wgs / cus);
  const double tc = pl.tc > 0 ? (double)pl.tc : (double)p.Nc;
  const double n_st = std::ceil(std::ceil((double)p.Nc / tc) / kc);  // stages per workgroup
  // (a stride-2 row-band workgroup fills the register file: one wave per
  // SIMD with accumulators in AGPRs, or two of about 256 registers each)
  const int64_t occ =
      pl.kernel == CNN_K_SROWS
          ? 1
          : std::max<int64_t>(1, std::min<int64_t>(bud.wg_per_cu,
                                                   bud.lds_bytes / std::max<int64_t>(1, pl.lds_bytes)));
  const double rate = mfma_rate(pl.dtype) * (pl.dtype == CNN_F32 ? 1.0 : kMfmaRealBf16) *
                      clk_per_us * fc.mfma_eff;                    // flops per us per CU
  const double stage_flops = pl.mfma_flops / wgs / n_st;
  const double stage_bytes = pl.eq1_bytes / wgs / n_st;
  const double t_stage =
      std::max(stage_flops / rate, fc.stage_us + stage_bytes / (fc.stage_gbs * 1e3));
  double t = std::ceil(per_cu / (double)occ) * (fc.wg_us + n_st * t_stage);
  t = std::max(t, pl.hbm_bytes / (hbm_gbs(w_out) * 1e3));
  if (pl.kernel == CNN_K_SPLITC && pl.ws_bytes == 0 && pl.kc > 1)  // atomic sums: zero fill
    t += kLaunchUs + 4.0 * n_out / (kFillGBs * 1e3);
  else if (pl.kernel == CNN_K_SPLITC && pl.ws_bytes > 0)  // the reduce: kc partials read, Out written
    t += kLaunchUs + 4.0 * (kc + 1.0) * n_out / (kHbmGBs * 1e3);
  return t + kLaunchUs;
}

static void fill_common(const cnn_problem& p, int dtype, const cnn_budget& bud,
                        cnn_plan_t* plan) {
  const int64_t Nx = p.sw * (p.Nw - 1) + p.Nr, Ny = p.sh * (p.Nh - 1) + p.Ns;
  const double e_in = in_bytes(dtype), e_out = out_bytes(dtype);
  // Compulsory traffic: In elements that some output reads, Ker, Out once.
  const double rows_read = (p.sw >= p.Nr) ? (double)(p.Nw * p.Nr) : (double)Nx;
  const double cols_read = (p.sh >= p.Ns) ? (double)(p.Nh * p.Ns) : (double)Ny;
  plan->compulsory_bytes = e_in * ((double)(p.Nb * p.Nc) * rows_read * cols_read +
                                   (double)(p.Nk * p.Nc * p.Nr * p.Ns)) +
                           e_out * (double)(p.Nb * p.Nk * p.Nw * p.Nh);
  plan->flops = 2.0 * (double)p.Nb * p.Nk * p.Nc * p.Nr * p.Ns * p.Nw * p.Nh;
  double w_out;  // share of the HBM bytes that are writes
  if (plan->kernel == CNN_K_DIRECT) {
    plan->mfma_flops = 0.0;
    plan->hbm_bytes = plan->compulsory_bytes;
    w_out = e_out * (double)(p.Nb * p.Nk * p.Nw * p.Nh) / plan->compulsory_bytes;
  } else {
    double t[3];
    hbm_terms(*plan, kXcds, kL2Bytes, t);
    plan->hbm_bytes = t[0] + t[1] + t[2];
    w_out = plan->hbm_bytes > 0.0 ? t[0] / plan->hbm_bytes : 0.0;
  }
  plan->model_us = model_us(*plan, bud, w_out);
}

void direct_plan(const cnn_problem& p, int dtype, const cnn_budget& bud, cnn_plan_t* plan) {
  memset(plan, 0, sizeof(*plan));
  plan->prob = p;
  plan->dtype = dtype;
  plan->kernel = CNN_K_DIRECT;
  plan->variant = 1;
  plan->tk = 1;
  plan->tp = 1;
  plan->tc = p.Nc;
  const int64_t out = p.Nb * p.Nk * p.Nw * p.Nh;
  plan->grid = std::min<int64_t>((out + 255) / 256, 65536);
  // Each thread reads its own In window and Ker row: Eq. (1) with unit tiles.
  cnn_tiles t = {1, 1, p.Nc, 1, 1};
  double terms[3];
  eq1_terms(p, t, 1, terms, nullptr);
  for (int i = 0; i < 3; ++i) plan->eq1_elems[i] = terms[i];
  plan->eq1_bytes = out_bytes(dtype) * terms[0] + in_bytes(dtype) * (terms[1] + terms[2]);
  fill_common(p, dtype, bud, plan);
}

// Eq. (3) one level up: the plan's tiles split over `xcds` processors (the
// XCDs, each with an L2 of l2 bytes) as the kernels assign them -- XCD x
// runs the x-th of `xcds` contiguous runs of the tile index (tile = pixel
// tile * n_ktiles + k tile) -- each XCD reading from HBM the union of the
// input rows its tiles read,
// and each Ker tile its run meets once if those Ker tiles fit its L2 beside
// the largest slab, else once per tile.  terms: Out written (with the fp32
// partial Outs of channel-split plans, written and read once), Ker read,
// In read; bytes.
void hbm_terms(const cnn_plan_t& pl, int64_t xcds, int64_t l2, double terms[3]) {
  const cnn_problem& p = pl.prob;
  const int64_t hw = p.Nw * p.Nh, npix = p.Nb * hw;
  const int64_t Nx = p.sw * (p.Nw - 1) + p.Nr, Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t tp = pl.tp, tk = pl.tk;
  const int64_t n_p = ceil_div(npix, tp), n_k = ceil_div(p.Nk, tk), tiles = n_p * n_k;
  const double e_in = in_bytes(pl.dtype), e_out = out_bytes(pl.dtype);
  const double row_bytes = e_in * (double)p.Nc * (double)Ny;  // one (b, x) row, all channels
  auto ker_bytes = [&](int64_t kt) {
    return e_in * (double)(std::min(tk, p.Nk - kt * tk) * p.Nc * p.Nr * p.Ns);
  };
  double in_b = 0.0, ker_b = 0.0;
  const int64_t q = tiles / xcds, rem = tiles % xcds;
  for (int64_t x = 0; x < xcds; ++x) {
    const int64_t cnt = q + (x < rem ? 1 : 0);
    if (cnt == 0) continue;
    const int64_t t0 = x * q + std::min(x, rem), t1 = t0 + cnt;
    // input rows read: output row (b, w) reads rows b*Nx + sw*w .. + Nr - 1;
    // the output rows are visited in increasing order, so a running end
    // counts each row once.  Rows between strided reads are not read, but
    // a gap shorter than a 128-byte line shares its lines with the rows
    // around it, which HBM delivers whole: such gaps count as read.
    const int64_t gap_max = (int64_t)((128.0 - 1.0) / (e_in * (double)Ny));  // rows
    int64_t rows = 0, end = -1, max_slab = 0;
    for (int64_t pt = t0 / n_k; pt <= (t1 - 1) / n_k; ++pt) {
      const int64_t f = pt * tp, last = std::min(f + tp, npix) - 1;
      const int64_t r0 = f / p.Nh, r1 = last / p.Nh;  // flattened (b, w) output rows
      max_slab = std::max(max_slab, (r1 / p.Nw) * Nx + p.sw * (r1 % p.Nw) + p.Nr -
                                        ((r0 / p.Nw) * Nx + p.sw * (r0 % p.Nw)));
      for (int64_t r = r0; r <= r1; ++r) {
        const int64_t g0 = (r / p.Nw) * Nx + p.sw * (r % p.Nw), g1 = g0 + p.Nr;
        const int64_t from = (end >= 0 && g0 > end && g0 - end <= gap_max) ? end : std::max(g0, end);
        if (g1 > from) rows += g1 - from;
        end = std::max(end, g1);
      }
    }
    in_b += (double)rows * row_bytes;
    double set = 0.0, per_tile = 0.0;
    for (int64_t kt = 0; kt < n_k; ++kt) {  // k tiles the run meets
      bool met = cnt >= n_k;
      for (int64_t t = t0; !met && t < t1; ++t) met = t % n_k == kt;
      if (met) set += ker_bytes(kt);
    }
    for (int64_t t = t0; t < t1; ++t) per_tile += ker_bytes(t % n_k);
    ker_b += set + (double)max_slab * row_bytes <= (double)l2 ? set : per_tile;
  }
  const double out = (double)npix * (double)p.Nk;
  terms[0] = e_out * out + (pl.kernel == CNN_K_SPLITC ? 8.0 * pl.kc * out : 0.0);
  // The stride-2 row-band kernels store Out as row pieces (Nh values per
  // feature row) that rarely fill a 128-byte line; the L2 merges most
  // neighbouring pieces but writes some lines twice: measured WRITE_SIZE is
  // 17-20 % above Out on the 3x3 stride-2 layer (fp32 Out).
  if (pl.kernel == CNN_K_SROWS) terms[0] *= kSrowsWriteRate;
  terms[1] = ker_b;
  terms[2] = in_b;
  if (pl.kernel == CNN_K_SROWS) {
    // the raw-Ker form streams a band's In once per 128-feature tile, the
    // tiles one after the other: its XCD's bands (tens of 100-KiB-scale
    // slabs) do not stay in the L2 from one tile to the next
    int n = 0;
    const VariantQ* vq = variants_srows(&n);
    for (int i = 0; i < n; ++i)
      if (vq[i].id == pl.variant && vq[i].form == 2)
        terms[2] *= (double)ceil_div(p.Nk, 128) / (double)ceil_div(p.Nk, 256);
  }
}

// Table 1 of Sec. 2.1: the closed-form optimum of Eq. (4).  The relaxed
// capacity solves M_L + 3K sqrt(M_L) = M.
void closed_form(const cnn_problem& p, double P, double M, int capacity_mode,
                 cnn_closed_form_t* out) {
  const double RS = (double)(p.Nr * p.Ns), ss = (double)(p.sw * p.sh), Q = RS * ss;
  const double Nbhw = (double)p.Nb * (double)p.Nw * (double)p.Nh;
  const double A = (double)p.Nk * Nbhw / P;   // Out per processor
  const double V = A * (double)p.Nc;          // products per processor
  double ML = M;
  if (capacity_mode == 1) {
    const double K = std::sqrt(Q);
    ML = M - 0.5 * 3.0 * K * (std::sqrt(9.0 * K * K + 4.0 * M) - 3.0 * K);
  }
  const double ridge = std::cbrt(V * V) * std::cbrt(Q);  // V^(2/3) Q^(1/3)
  out->M_L = ML;
  if (A >= ML || ML < ridge) {  // the capacity binds: Cases 1a and 2b
    out->row = A >= ML ? 1 : 3;
    out->Tk = std::sqrt(ML * ss / RS);
    out->Tbhw = std::sqrt(ML * RS / ss);
    out->cost = (A >= ML ? A : ML) + 2.0 * V * std::sqrt(Q / ML);
  } else {                      // Case 2a: the unconstrained optimum fits
    out->row = 2;
    out->Tk = std::cbrt(V / RS) * std::cbrt(ss * ss);
    out->Tbhw = std::cbrt(V / ss) * std::cbrt(RS * RS);
    out->cost = 3.0 * ridge;
  }
  out->split_c = out->row != 1;
}

// Case 2 of Sec. 2.1 (W_c < N_c) on one GPU: the plain staging plan with its
// channel loop split over kc workgroup slices of ceil(stages/kc) stages.  kc
// is the smallest count with no empty slice that gives at least two
// workgroups per CU, else one slice per stage.  The workspace holds kc fp32
// partial Outs.
static void splitc_finish(const cnn_problem& p, const cnn_budget& bud, cnn_plan_t* plan) {
  const int64_t stages = ceil_div(p.Nc, plan->tc);
  int64_t kc = std::min<int64_t>(stages, std::max<int64_t>(1, ceil_div(2 * bud.cus, plan->grid)));
  while (ceil_div(stages, ceil_div(stages, kc)) != kc) ++kc;  // ends at kc = stages
  plan->kernel = CNN_K_SPLITC;
  plan->kc = (int32_t)kc;
  plan->ws_bytes = 4 * kc * p.Nb * p.Nk * p.Nw * p.Nh;
}

// Channel-slice kernel (conv_cslice): a split form only.
static bool eval_cslice(const cnn_problem& p, int dtype, const VariantC& v,
                        const cnn_budget& bud, cnn_plan_t* plan) {
  if (!cslice_fits(v, p)) return false;
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t S = slab_rows_max(p, v.tp);
  const int64_t lds = cslice_lds_bytes(v, S, Ny);
  if (!eval_tiling(p, dtype, v.id, v.tk, v.tp, v.tc, 16, S, lds, 0, bud, plan)) return false;
  splitc_finish(p, bud, plan);
  if (v.mode == 1) plan->ws_bytes = 0;  // the slices add into Out
  if (v.mode == 2) {                     // one slice writing Out
    plan->kc = 1;
    plan->ws_bytes = 0;
  }
  return true;
}

// Candidate order: the smaller model time; within 2 % of it, fewer
// predicted HBM bytes (Eq. (3) at the XCD level), then fewer Eq. (1) bytes,
// then the lower instantiation id.
static bool better(const cnn_plan_t& a, const cnn_plan_t& b) {
  const double lo = std::min(a.model_us, b.model_us);
  if (std::fabs(a.model_us - b.model_us) > 0.02 * lo) return a.model_us < b.model_us;
  if (a.hbm_bytes != b.hbm_bytes) return a.hbm_bytes < b.hbm_bytes;
  if (a.eq1_bytes != b.eq1_bytes) return a.eq1_bytes < b.eq1_bytes;
  if (a.variant != b.variant) return a.variant < b.variant;
  return a.tp > b.tp;
}

// Every tiling the kernels implement that fits the budget, as complete plans
// (model fields set); at most cap are written, the count is returned.
int enumerate_plans(const cnn_problem& p, int dtype, const cnn_budget& bud, cnn_plan_t* out,
                    int cap) {
  int n = 0;
  auto add = [&](cnn_plan_t& cand, int kernel) {
    cand.kernel = kernel;
    fill_common(p, dtype, bud, &cand);
    if (n < cap) out[n] = cand;
    ++n;
  };
  cnn_plan_t cand;
  int n4 = 0, n3 = 0, n2 = 0, n1 = 0;
  const Variant4* vs4 = variants4(&n4);
  for (int i = 0; i < n4; ++i)
    if (vs4[i].dtype == dtype && eval_variant4(p, dtype, vs4[i], bud, &cand))
      add(cand, CNN_K_IGEMM_WIDE);
  const Variant3* vs3 = variants3(&n3);
  for (int i = 0; i < n3; ++i)
    if (vs3[i].dtype == dtype && eval_variant3(p, dtype, vs3[i], bud, &cand))
      add(cand, CNN_K_IGEMM_DMA);
  const Variant2* vs2 = variants2(&n2);
  for (int i = 0; i < n2; ++i)
    if (vs2[i].dtype == dtype && eval_variant2(p, dtype, vs2[i], bud, &cand))
      add(cand, v2_family(vs2[i]));
  int nsc = 0;
  const VariantS* vss = variants_smallc(&nsc);
  for (int i = 0; i < nsc; ++i)
    if (vss[i].dtype == dtype && eval_smallc(p, dtype, vss[i], bud, &cand))
      add(cand, CNN_K_SMALLC);
  int ngm = 0;
  const VariantG* vgm = variants_gemm1(&ngm);
  for (int i = 0; i < ngm; ++i)
    if (vgm[i].dtype == dtype && eval_gemm1(p, dtype, vgm[i], bud, &cand))
      add(cand, CNN_K_GEMM1);
  int nsq = 0;
  const VariantQ* vsq = variants_srows(&nsq);
  for (int i = 0; i < nsq; ++i)
    if (vsq[i].dtype == dtype && eval_srows(p, dtype, vsq[i], bud, &cand))
      add(cand, CNN_K_SROWS);
  // row streaming: every band length L dividing Nw, up to 4 groups' rows
  int nrw = 0;
  const VariantR* vrw = variants_rows(&nrw);
  for (int i = 0; i < nrw; ++i) {
    if (vrw[i].dtype != dtype) continue;
    for (int64_t L = 1; L <= std::min<int64_t>(p.Nw, 4 * vrw[i].wr); ++L)
      if (p.Nw % L == 0 && eval_rows(p, dtype, vrw[i], bud, L, &cand))
        add(cand, CNN_K_ROWS);
  }
  const Variant* vs = variants(&n1);
  for (int i = 0; i < n1; ++i)
    if (vs[i].dtype == dtype && vs[i].kernel == CNN_K_IGEMM &&
        eval_variant(p, dtype, vs[i], bud, &cand)) {
      cnn_plan_t plain = cand;
      add(plain, CNN_K_IGEMM);
      // too few tiles for the chip and more than one stage: the split form
      if (cand.grid < bud.cus && ceil_div(p.Nc, cand.tc) > 1) {
        splitc_finish(p, bud, &cand);
        add(cand, CNN_K_SPLITC);
      }
    }
  int ncs = 0;
  const VariantC* vcs = variants_cslice(&ncs);
  for (int i = 0; i < ncs; ++i)
    if (vcs[i].dtype == dtype && eval_cslice(p, dtype, vcs[i], bud, &cand) &&
        cand.grid < bud.cus && ceil_div(p.Nc, cand.tc) > 1)
      add(cand, CNN_K_SPLITC);
  if (n == 0) {
    direct_plan(p, dtype, bud, &cand);
    if (cap > 0) out[0] = cand;
    n = 1;
  }
  return n;
}

int select_plan(const cnn_problem& p, int dtype, const cnn_budget& bud, int kernel,
                int64_t tk, int64_t tp, int64_t tc, cnn_plan_t* out) {
  if (kernel == CNN_K_DIRECT) {
    direct_plan(p, dtype, bud, out);
    return CNN_OK;
  }
  if (kernel == CNN_K_AUTO || kernel == CNN_K_AUTO_NO_WORKSPACE) {
    // The model's choice among all candidates, or among those that need no
    // workspace.
    const bool ws_free = kernel == CNN_K_AUTO_NO_WORKSPACE;
    std::vector<cnn_plan_t> c(256);
    int n = enumerate_plans(p, dtype, bud, c.data(), (int)c.size());
    if (n > (int)c.size()) {
      c.resize(n);
      n = enumerate_plans(p, dtype, bud, c.data(), n);
    }
    const cnn_plan_t* best = nullptr;
    for (int i = 0; i < n; ++i)
      if ((!ws_free || c[i].ws_bytes == 0) && (!best || better(c[i], *best))) best = &c[i];
    if (!best) {
      direct_plan(p, dtype, bud, out);
      return CNN_OK;
    }
    *out = *best;
    return CNN_OK;
  }
  if (kernel == CNN_K_SPLITC) {
    int n = 0;
    const Variant* vs = variants(&n);
    for (int i = 0; i < n; ++i) {
      const Variant& v = vs[i];
      if (v.dtype != dtype || v.kernel != CNN_K_IGEMM || v.tk != tk || v.tp != tp || v.tc != tc)
        continue;
      if (!eval_variant(p, dtype, v, bud, out)) continue;
      splitc_finish(p, bud, out);
      out->kernel = CNN_K_SPLITC;
      fill_common(p, dtype, bud, out);
      return CNN_OK;
    }
    const VariantC* vc = variants_cslice(&n);
    for (int i = 0; i < n; ++i) {
      const VariantC& v = vc[i];
      if (v.dtype != dtype || v.tk != tk || v.tp != tp || v.tc != tc) continue;
      if (!eval_cslice(p, dtype, v, bud, out)) continue;
      out->kernel = CNN_K_SPLITC;
      fill_common(p, dtype, bud, out);
      return CNN_OK;
    }
    return CNN_E_UNSUPPORTED;
  }
  // A requested family and tiling: the instantiations that implement it,
  // the model's best of them.
  bool found = false;
  cnn_plan_t best;
  auto consider = [&](cnn_plan_t& cand, int family) {
    cand.kernel = family;
    fill_common(p, dtype, bud, &cand);
    if (!found || better(cand, best)) {
      best = cand;
      found = true;
    }
  };
  cnn_plan_t cand;
  if (kernel == CNN_K_ROWS) {  // tp = L*Nh whole rows (0: the model's band), tc always Nc
    int nr = 0;
    const VariantR* vr = variants_rows(&nr);
    for (int i = 0; i < nr; ++i) {
      const VariantR& v = vr[i];
      if (v.dtype != dtype || v.tk != tk || tp % p.Nh) continue;
      if (tp > 0) {
        if (eval_rows(p, dtype, v, bud, tp / p.Nh, &cand)) consider(cand, CNN_K_ROWS);
      } else {
        for (int64_t L = 1; L <= p.Nw; ++L)
          if (p.Nw % L == 0 && eval_rows(p, dtype, v, bud, L, &cand)) consider(cand, CNN_K_ROWS);
      }
    }
  } else if (kernel == CNN_K_GEMM1) {  // tp: the instantiation's largest tile
    int ng = 0;
    const VariantG* vg = variants_gemm1(&ng);
    for (int i = 0; i < ng; ++i) {
      const VariantG& v = vg[i];
      if (v.dtype != dtype || v.tk != tk || v.tp != tp || v.tc != tc) continue;
      if (eval_gemm1(p, dtype, v, bud, &cand)) consider(cand, CNN_K_GEMM1);
    }
  } else if (kernel == CNN_K_SROWS) {  // tp = L*Nh names the band; 0: any
    int nq = 0;
    const VariantQ* vq = variants_srows(&nq);
    for (int i = 0; i < nq; ++i) {
      const VariantQ& v = vq[i];
      if (v.dtype != dtype || v.tk != tk || (tp != 0 && tp != v.L * p.Nh) || (tc != 0 && tc != 16))
        continue;
      if (eval_srows(p, dtype, v, bud, &cand)) consider(cand, CNN_K_SROWS);
    }
  } else if (kernel == CNN_K_IGEMM_WIDE) {
    int n4 = 0;
    const Variant4* vs4 = variants4(&n4);
    for (int i = 0; i < n4; ++i) {
      const Variant4& v = vs4[i];
      if (v.dtype == dtype && v.tk == tk && v.tp == tp && v.tc == tc &&
          eval_variant4(p, dtype, v, bud, &cand))
        consider(cand, CNN_K_IGEMM_WIDE);
    }
  } else if (kernel == CNN_K_IGEMM_DMA) {
    int n3 = 0;
    const Variant3* vs3 = variants3(&n3);
    for (int i = 0; i < n3; ++i) {
      const Variant3& v = vs3[i];
      if (v.dtype == dtype && v.tk == tk && v.tp == tp && v.tc == tc &&
          eval_variant3(p, dtype, v, bud, &cand))
        consider(cand, CNN_K_IGEMM_DMA);
    }
  } else if (kernel == CNN_K_SMALLC) {  // tc: always Nc
    int ns = 0;
    const VariantS* vss = variants_smallc(&ns);
    for (int i = 0; i < ns; ++i) {
      const VariantS& v = vss[i];
      if (v.dtype == dtype && v.tk == tk && v.tp == tp && eval_smallc(p, dtype, v, bud, &cand))
        consider(cand, CNN_K_SMALLC);
    }
  } else if (kernel == CNN_K_IGEMM_PIPE || kernel == CNN_K_IGEMM_RAWK ||
             kernel == CNN_K_POINTWISE) {  // tp: the instantiation's largest tile
    int n2 = 0;
    const Variant2* vs2 = variants2(&n2);
    for (int i = 0; i < n2; ++i) {
      const Variant2& v = vs2[i];
      if (v.dtype == dtype && v2_family(v) == kernel && v.tk == tk && v.tp == tp &&
          v.tc == tc && eval_variant2(p, dtype, v, bud, &cand))
        consider(cand, kernel);
    }
  } else if (kernel == CNN_K_IGEMM) {
    int n = 0;
    const Variant* vs = variants(&n);
    for (int i = 0; i < n; ++i) {
      const Variant& v = vs[i];
      if (v.dtype == dtype && v.kernel == CNN_K_IGEMM && v.tk == tk && v.tp == tp &&
          v.tc == tc && eval_variant(p, dtype, v, bud, &cand))
        consider(cand, CNN_K_IGEMM);
    }
  } else {
    return CNN_E_UNSUPPORTED;
  }
  if (!found) return CNN_E_UNSUPPORTED;
  *out = best;
  return CNN_OK;
}

// The instantiation table of every family (cnn_variants).
int list_variants(cnn_variant_t* out, int cap) {
  int n = 0;
  auto add = [&](int kernel, int id, int dtype, int nr, int ns, int mode, int64_t tk, int64_t tp,
                 int64_t tc) {
    if (n < cap) {
      cnn_variant_t& o = out[n];
      o.kernel = kernel;
      o.variant = id;
      o.dtype = dtype;
      o.nr = nr;
      o.ns = ns;
      o.mode = mode;
      o.tk = tk;
      o.tp = tp;
      o.tc = tc;
    }
    ++n;
  };
  int c = 0;
  const Variant* v1 = variants(&c);
  for (int i = 0; i < c; ++i)
    if (v1[i].kernel == CNN_K_IGEMM)
      add(CNN_K_IGEMM, v1[i].id, v1[i].dtype, 0, 0, 0, v1[i].tk, v1[i].tp, v1[i].tc);
  const Variant2* v2 = variants2(&c);
  for (int i = 0; i < c; ++i)
    add(v2_family(v2[i]), v2[i].id, v2[i].dtype, v2[i].nr, v2[i].ns, 0, v2[i].tk, v2[i].tp,
        v2[i].tc);
  const Variant3* v3 = variants3(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_IGEMM_DMA, v3[i].id, v3[i].dtype, v3[i].nr, v3[i].ns, 0, v3[i].tk, v3[i].tp,
        v3[i].tc);
  const Variant4* v4 = variants4(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_IGEMM_WIDE, v4[i].id, v4[i].dtype, v4[i].nr, v4[i].ns, 0, v4[i].tk, v4[i].tp,
        v4[i].tc);
  const VariantS* vsc = variants_smallc(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_SMALLC, vsc[i].id, vsc[i].dtype, vsc[i].nr, vsc[i].ns, 0, vsc[i].tk, vsc[i].tp, 0);
  const VariantR* vr = variants_rows(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_ROWS, vr[i].id, vr[i].dtype, vr[i].nr, vr[i].ns, vr[i].mb, vr[i].tk, 0,
        16 * vr[i].ncg);
  const VariantG* vg = variants_gemm1(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_GEMM1, vg[i].id, vg[i].dtype, 1, 1, vg[i].s2, vg[i].tk, vg[i].tp, vg[i].tc);
  const VariantQ* vq = variants_srows(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_SROWS, vq[i].id, vq[i].dtype, vq[i].nr, vq[i].ns, vq[i].L, vq[i].tk, 0, 16);
  const VariantC* vc = variants_cslice(&c);
  for (int i = 0; i < c; ++i)
    add(CNN_K_SPLITC, vc[i].id, vc[i].dtype, vc[i].nr, vc[i].ns, vc[i].mode, vc[i].tk, vc[i].tp,
        vc[i].tc);
  return n;
}

}  // namespace cnnlib

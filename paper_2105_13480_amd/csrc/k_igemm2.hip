// Implicit-GEMM convolution on bf16 MFMA, pipelined (gfx950).
//
// Same tile schedule as conv_igemm (paper Sec. 2.1 / Listing 3 with
// W_c = N_c: a workgroup keeps a tk x tp Out tile in accumulators and walks
// the input features tc at a time), with the data movement rebuilt for the
// CDNA4 memory system:
//
// * Ker, fixed stencils (RAWK) with Nc a multiple of 8: the stage's raw Ker
//   rows -- for each feature, its TC channels times all taps, one
//   contiguous run of memory -- are copied with 16-byte buffer->LDS DMA,
//   one padding chunk per row so the A-operand reads of 8 consecutive
//   features hit distinct LDS banks.  A lane reads its feature's 8
//   channels x RS taps (16*RS contiguous bytes) and builds each tap's
//   MFMA operand with four v_perm: no repack kernel, no workspace.
// * Ker, other problems: repacked once per call by pack_ker into the exact
//   LDS image of every (k tile, c stage) block, [tap][c/8][k][8], which a
//   workgroup streams with 16-byte global->LDS DMA loads.
// * The halo'd In slab (whole input rows, see conv_igemm) is loaded as
//   dwords -- two consecutive positions of one channel per lane, so each
//   wave-wide load is a 256-byte contiguous run -- eight channels per work
//   item, transposed in registers with v_perm into two 16-byte
//   [8 channels] vectors and written to LDS as [c/8][position][8].
//   Positions whose address is odd are assembled from two aligned dwords
//   with a funnel shift; pairs that straddle an image use two 16-bit loads.
// * Two LDS buffers per operand: the loads of stage i+1 are in flight while
//   stage i runs on the MFMA units; one barrier per stage.
// * The tile size a.tp is a run-time value up to TP (the lanes' capacity):
//   the selector shrinks it so the tiles fill the machine's workgroup slots
//   evenly (the P processors of Eq. (2) each get the same share).
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

// ---- Ker repack ------------------------------------------------------------
// Packed layout: block (kt, cc) of RS*G*TK vectors (G = TC/8), each block
// padded to `blk_vecs` vectors (a multiple of 256); vector (tap, g, kk)
// holds Ker[kt*TK+kk][cc*TC + 8g + 0..7][tap], zero where k >= Nk or
// c >= Nc.
__global__ __launch_bounds__(256) void pack_ker_bf16(const bf16_t* __restrict__ Ker,
                                                      u32x4_t* __restrict__ P, ConvArgs a,
                                                      int TK, int TC, int blk_vecs,
                                                      int64_t total_vecs) {
  const int RS = a.Nr * a.Ns;
  const int G = TC / 8;
  const int n_cc = (a.Nc + TC - 1) / TC;
  for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < total_vecs;
       v += (int64_t)gridDim.x * 256) {
    const int64_t blk = v / blk_vecs;
    const int in_blk = (int)(v - blk * blk_vecs);
    u32x4_t out = {0u, 0u, 0u, 0u};
    if (in_blk < RS * G * TK) {
      const int kt = (int)(blk / n_cc);
      const int cc = (int)(blk - (int64_t)kt * n_cc);
      const int kk = in_blk % TK;
      const int rest = in_blk / TK;
      const int g = rest % G;
      const int tap = rest / G;
      const int k = kt * TK + kk;
      if (k < a.Nk) {
        const bf16_t* src = Ker + ((int64_t)k * a.Nc) * RS + tap;
        const int cb = cc * TC + 8 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = cb + 2 * i;
          const uint32_t lo = c < a.Nc ? src[(int64_t)c * RS] : 0u;
          const uint32_t hi = c + 1 < a.Nc ? src[(int64_t)(c + 1) * RS] : 0u;
          out[i] = lo | (hi << 16);
        }
      }
    }
    P[v] = out;
  }
}

// ---- In staging ---------------------------------------------------------------
// Work items are pairs of consecutive slab positions (pos, pos+1) of one
// 8-channel group; a wave's lanes always share the group, so the channel
// offset of each load is a wave-uniform (scalar) buffer offset and the
// per-lane offsets are computed once per tile.  How a pair is read is
// decided once per tile:
//   kAligned   Ny even: every pair starts on a 4-byte boundary in every
//              channel plane and never straddles an image -> one dword.
//   kFunnel    otherwise, if no pair straddles an image: two aligned dwords
//              and a 16-bit funnel shift (v_alignbit); which of the two
//              alignments a channel needs follows from c*Nx*Ny's parity.
//   kElement   a pair straddles an image: two 16-bit loads per pair.
// Loads go through buffer descriptors based at the tile's first image, so
// offsets are 32-bit and reads past the tensor return 0 instead of faulting.
//   kStride2   (1x1 gather, stride 2 along h) one 8-byte load covers the
//              pair's two elements, 4 bytes apart; v_perm packs them.
enum { kAligned = 0, kFunnel = 1, kElement = 2, kStride2 = 3 };

// Extent rounded up to whole dwords: a dword holding a tensor's last
// 16-bit element must not count as out of range (the extra bytes share the
// element's 4-byte word, so they are mapped, and are never used).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// 16-byte buffer -> LDS copy (lane i's 16 bytes land at lds + 16 i, lds
// wave-uniform); out-of-range reads give zeros.  Device-only builtin.
__device__ __forceinline__ void dma16b(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR(void, lds), 16, voff, 0, 0, 0);
#endif
}

// Raw-Ker LDS row: RS*TC/8 16-byte chunks of one feature, padded to an odd
// count (row strides of 8 consecutive features then start in distinct
// 4-bank groups).
__host__ __device__ constexpr int rawk_row_chunks(int RS, int TC) {
  return (RS * TC / 8) | 1;
}

// ODDY: the input rows have odd length, so pairs need the funnel or the
// element path (and two words per pair in flight); with Ny even every pair
// is one aligned dword.  The launcher picks the instantiation from Ny.
template <typename TO, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int MAXP,
          bool RAWK, bool PW, bool ODDY>
__global__ __launch_bounds__(256) void conv_igemm2(const bf16_t* __restrict__ In,
                                                   const u32x4_t* __restrict__ Kp,
                                                   TO* __restrict__ Out, ConvArgs a,
                                                   int blk_vecs) {
  constexpr int TK = 32 * WM * MB;
  constexpr int G = TC / 8;
  constexpr int KSTEPS = G / 2;
  static_assert(WM * WN == 4, "four waves");
  static_assert(TC % 16 == 0, "whole MFMA K-steps per stage");
  const int Nr = NR > 0 ? NR : a.Nr;
  const int Ns = NS > 0 ? NS : a.Ns;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  // positions per channel group (even: pairs never cross groups); the 1x1
  // gather (PW) stages the tile's outputs, the others its input rows
  const int SN = PW ? ((a.tp + 1) & ~1) : ((a.slab_max * a.Ny + 1) & ~1);
  u32x4_t* inbuf = reinterpret_cast<u32x4_t*>(smem);  // [2][G][SN]
  u32x4_t* kerbuf = inbuf + 2 * G * SN;                 // [2][blk_vecs]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, half = lane >> 5;

  static_assert(!RAWK || (NR > 0 && NS > 0), "raw Ker needs a compile-time stencil");
  static_assert(!PW || (NR == 1 && NS == 1 && RAWK), "the gather is for raw-Ker 1x1 stencils");
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int pt = tile / a.n_ktiles;
  const int kt = tile - pt * a.n_ktiles;
  const int p0 = pt * a.tp;
  const int k0 = kt * TK;
  const int plast = min(p0 + a.tp, a.npix) - 1;
  const int b0 = p0 / a.hw, w0 = (p0 - b0 * a.hw) / a.Nh;
  const int b1 = plast / a.hw, w1 = (plast - b1 * a.hw) / a.Nh;
  const int G0 = b0 * a.Nx + a.sw * w0;
  const int S = b1 * a.Nx + a.sw * w1 + Nr - G0;
  const int SNt = PW ? plast - p0 + 1 : S * a.Ny;
  const int npairs = (SNt + 1) >> 1;

  // Output side: LDS position of each lane's (r, s) = (0, 0) tap and its
  // Out byte offset (k = 0) from the tile's first image.  Lanes past the
  // tile's last output take that output's place: they compute and store
  // the identical value, so no store needs a pixel mask.
  int pix[NB];
  uint32_t obyte[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int p = p0 + (wn * NB + nb) * 32 + l32;
    const int pc = p <= plast ? p : plast;
    const int b = pc / a.hw;
    const int q = pc - b * a.hw;
    const int w = q / a.Nh;
    const int h = q - w * a.Nh;
    pix[nb] = PW ? pc - p0 : (b * a.Nx + a.sw * w - G0) * a.Ny + a.sh * h;
    obyte[nb] = (uint32_t)(((int64_t)(b - b0) * a.Nk * a.hw + q) * (int64_t)sizeof(TO));
  }

  // Input side.
  // Descriptor base: the tile's first image rounded down to an even element,
  // so dword offsets relative to it are dword-aligned in memory.
  const int64_t base_el = ((int64_t)b0 * a.in_img) & ~(int64_t)1;
  const __amdgpu_buffer_rsrc_t in_rsrc = make_rsrc(In + base_el, (a.in_total - base_el) * 2);
  int path;
  if constexpr (PW) {
    // Pairs are outputs (2i, 2i+1) of the tile (p0 and Nh even keep them in
    // one output row).  Stride 1 along h: the two elements are adjacent
    // and, with Ny even, dword-aligned.  Stride 2: 4 bytes apart, one
    // 8-byte load, unless the tile holds the tensor's last input row, where
    // the load could reach past the end.
    const bool even = (a.Nh & 1) == 0 && (p0 & 1) == 0;
    if (even && a.sh == 1 && (a.Ny & 1) == 0)
      path = kAligned;
    else if (even && a.sh == 2 && !(b1 == a.Nb - 1 && w1 == a.Nw - 1))
      path = kStride2;
    else
      path = kElement;
  } else if constexpr (!ODDY) {
    path = kAligned;  // Ny even: pairs are aligned and never straddle an image
  } else {
    path = kFunnel;
    for (int b = b0 + 1; b <= b1; ++b)
      if ((((int64_t)b * a.Nx - G0) * a.Ny) & 1) path = kElement;
  }
  const int gpos0 = G0 * a.Ny;
  uint32_t voff[MAXP], voff2[MAXP];  // byte offsets (channel 0) of pos / of pos+1
  bool pvalid[MAXP];
  int pdst[MAXP];
#pragma unroll
  for (int j = 0; j < MAXP; ++j) {
    const int pr = tid + 256 * j;
    pvalid[j] = pr < npairs;
    const int pos = 2 * (pvalid[j] ? pr : 0);
    pdst[j] = pos;
    if constexpr (PW) {
      // element of output p: In[b][c][sw*w][sh*h] (channel 0 here)
      auto gather = [&](int p) -> uint32_t {
        const int b = p / a.hw;
        const int q = p - b * a.hw;
        const int w = q / a.Nh;
        const int h = q - w * a.Nh;
        return (uint32_t)(((int64_t)b * a.in_img - base_el + (int64_t)a.sw * w * a.Ny +
                           (int64_t)a.sh * h) * 2);
      };
      voff[j] = gather(p0 + pos);
      voff2[j] = gather(min(p0 + pos + 1, plast));
    } else {
      const int gp = gpos0 + pos;
      const int b = gp / a.nxny;
      const int r0 = gp - b * a.nxny;
      voff[j] = (uint32_t)(((int64_t)b * a.in_img - base_el + r0) * 2);
      // second position: next element, or the next image's first element
      const int b2 = (r0 + 1 == a.nxny) ? b + 1 : b;
      const int r2 = (r0 + 1 == a.nxny) ? 0 : r0 + 1;
      voff2[j] = (uint32_t)(((int64_t)b2 * a.in_img - base_el + r2) * 2);
    }
  }

  uint32_t pre[G][MAXP][8];
  uint32_t pre2[G][MAXP][8];  // second word of a pair (row paths; unused by the gather)
  // Gather staging (1x1 kernels), the stage starting at c0: channel
  // q = 8g + i into every pair slot (slots past the tile reload position
  // 0).  One uniform switch on the load path per stage, then straight-line
  // loads; a channel past Nc loads channel Nc-1 and write_in zeroes it.
  auto load_path = [&](auto tag, int c0) __attribute__((always_inline)) {
    constexpr int P = decltype(tag)::value;
#pragma unroll
    for (int q = 0; q < 8 * G; ++q) {
      const int g = q >> 3, i = q & 7;
      const int c = c0 + q;
      const uint32_t so = (uint32_t)((int64_t)min(c, a.Nc - 1) * a.nxny * 2);
#pragma unroll
      for (int j = 0; j < MAXP; ++j) {
        if constexpr (P == kAligned) {
          pre[g][j][i] = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, voff[j], so, 0);
        } else if constexpr (P == kStride2) {
          const u32x2_t d = __builtin_bit_cast(
              u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(in_rsrc, voff[j], so, 0));
          pre[g][j][i] = __builtin_amdgcn_perm(d[1], d[0], 0x05040100u);
        } else {
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, voff[j], so, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, voff2[j], so, 0);
          pre[g][j][i] = lo | (hi << 16);
        }
      }
    }
  };
  // Slab staging (row-staged kernels): one uniform switch on the load path
  // per stage, then straight-line loads of every channel (a channel past Nc
  // loads channel Nc-1; write_in zeroes it).  The words of a pair are
  // combined only in write_in, so no load waits for another.
  auto load_rows_p = [&](auto tag, int c0) __attribute__((always_inline)) {
    constexpr int P = decltype(tag)::value;
#pragma unroll
    for (int q = 0; q < 8 * G; ++q) {
      const int g = q >> 3, i = q & 7;
      const uint32_t so = (uint32_t)((int64_t)min(c0 + q, a.Nc - 1) * a.nxny * 2);
#pragma unroll
      for (int j = 0; j < MAXP; ++j) {
        if constexpr (P == kAligned) {
          pre[g][j][i] = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, voff[j], so, 0);
        } else if constexpr (P == kFunnel) {
          // the two aligned dwords around the pair
          const uint32_t lo_off = (voff[j] + (so & 2u)) & ~3u;
          pre[g][j][i] = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, lo_off, so & ~3u, 0);
          pre2[g][j][i] = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, lo_off + 4, so & ~3u, 0);
        } else {
          // the pair's two elements
          pre[g][j][i] = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, voff[j], so, 0);
          pre2[g][j][i] = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, voff2[j], so, 0);
        }
      }
    }
  };
  auto load_rows = [&](int c0) __attribute__((always_inline)) {
    if constexpr (!ODDY)
      load_rows_p(std::integral_constant<int, kAligned>(), c0);
    else if (path == kFunnel)
      load_rows_p(std::integral_constant<int, kFunnel>(), c0);
    else
      load_rows_p(std::integral_constant<int, kElement>(), c0);
  };
  auto load_in = [&](int c0) __attribute__((always_inline)) {
    if constexpr (PW) {
      if (path == kAligned)
        load_path(std::integral_constant<int, kAligned>(), c0);
      else if (path == kStride2)
        load_path(std::integral_constant<int, kStride2>(), c0);
      else
        load_path(std::integral_constant<int, kElement>(), c0);
    } else {
      load_rows(c0);
    }
  };
  // Each pair as one dword (funnel shift or packing per load path), then
  // 8 channels transposed into the two 16-byte vectors of the pair.
  auto write_path = [&](auto tag, u32x4_t* buf, int c0) __attribute__((always_inline)) {
    constexpr int P = decltype(tag)::value;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      // channels past Nc were loaded as channel Nc-1: zero them
      uint32_t keep[8], par[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        keep[i] = c0 + 8 * g + i < a.Nc ? ~0u : 0u;
        par[i] = (uint32_t)(((int64_t)(c0 + 8 * g + i) * a.nxny) & 1);
      }
#pragma unroll
      for (int j = 0; j < MAXP; ++j) {
        if (pvalid[j]) {
          uint32_t wd[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            if constexpr (P == kFunnel && !PW) {
              const uint32_t sh = (((voff[j] >> 1) + par[i]) & 1u) * 16u;
              wd[i] = __builtin_amdgcn_alignbit(pre2[g][j][i], pre[g][j][i], sh);
            } else if constexpr (P == kElement && !PW) {
              wd[i] = pre[g][j][i] | (pre2[g][j][i] << 16);
            } else {
              wd[i] = pre[g][j][i];
            }
          }
          u32x4_t lo, hi;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t e0 = wd[2 * i] & keep[2 * i];
            const uint32_t e1 = wd[2 * i + 1] & keep[2 * i + 1];
            lo[i] = __builtin_amdgcn_perm(e1, e0, 0x05040100u);
            hi[i] = __builtin_amdgcn_perm(e1, e0, 0x07060302u);
          }
          buf[g * SN + pdst[j]] = lo;
          buf[g * SN + pdst[j] + 1] = hi;
        }
      }
    }
  };
  auto write_in = [&](u32x4_t* buf, int c0) __attribute__((always_inline)) {
    if (PW || !ODDY)
      write_path(std::integral_constant<int, kAligned>(), buf, c0);
    else if (path == kFunnel)
      write_path(std::integral_constant<int, kFunnel>(), buf, c0);
    else
      write_path(std::integral_constant<int, kElement>(), buf, c0);
  };
  const int n_cc = (a.Nc + TC - 1) / TC;
  // Raw Ker: LDS chunk slot v of a stage is feature k0 + v / RC chunk
  // v % RC of that feature's run (chunks past RS*TC/8 are padding).
  constexpr int RS_C = (NR > 0 ? NR : 1) * (NS > 0 ? NS : 1);
  constexpr int RC = rawk_row_chunks(RS_C, TC);
  constexpr int RAW_VECS = (TK * RC + 63) / 64 * 64;
  constexpr int RAW_DMA = (RAW_VECS + 255) / 256;
  const __amdgpu_buffer_rsrc_t ker_rsrc =
      make_rsrc(reinterpret_cast<const bf16_t*>(Kp), (int64_t)a.Nk * a.Nc * RS_C * 2);
  uint32_t raw_off[RAWK ? RAW_DMA : 1];
  if constexpr (RAWK) {
#pragma unroll
    for (int j = 0; j < RAW_DMA; ++j) {
      const int v = tid + 256 * j;
      const int kk = v / RC;
      const int part = v - kk * RC;
      // padding chunks and rows past Nk read whatever is in range (or zeros)
      raw_off[j] = (uint32_t)((((int64_t)(k0 + kk) * a.Nc) * RS_C) * 2 + 16 * part);
    }
  }
  auto dma_ker = [&](int cc, u32x4_t* dst) {
    if constexpr (RAWK) {
      const uint32_t so = (uint32_t)(cc * TC * RS_C * 2);
#pragma unroll
      for (int j = 0; j < RAW_DMA; ++j)
        if (256 * j + wave * 64 < RAW_VECS)
          dma16b(ker_rsrc, dst + 256 * j + wave * 64, raw_off[j] + so);
    } else {
      const u32x4_t* src = Kp + ((int64_t)kt * n_cc + cc) * blk_vecs;
      for (int v0 = wave * 64; v0 < blk_vecs; v0 += 256)
        __builtin_amdgcn_global_load_lds(src + v0 + lane, LDS_PTR(void, dst + v0), 16, 0, 0);
    }
  };

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;

  dma_ker(0, kerbuf);
  load_in(0);
  for (int cc = 0; cc < n_cc; ++cc) {
    const int buf = cc & 1;
    u32x4_t* ib = inbuf + buf * G * SN;
    const u32x4_t* kb = kerbuf + buf * blk_vecs;
    write_in(ib, cc * TC);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    const bool more = cc + 1 < n_cc;
    if (more) {
      dma_ker(cc + 1, kerbuf + (buf ^ 1) * blk_vecs);
      load_in((cc + 1) * TC);
    }
    auto tap_step = [&](int rr, int ss) {
      const int tap = rr * Ns + ss;
      const int toff = rr * a.Ny + ss;
      const u32x4_t* kt_base = kb + tap * G * TK + (wm * MB) * 32 + l32;
#pragma unroll
      for (int j = 0; j < KSTEPS; ++j) {
        const int grp = 2 * j + half;
        u32x4_t av[MB], bv[NB];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) av[mb] = kt_base[grp * TK + mb * 32];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) bv[nb] = ib[grp * SN + pix[nb] + toff];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, av[mb]), __builtin_bit_cast(bf16x8_t, bv[nb]),
                acc[mb][nb], 0, 0, 0);
      }
    };
    if constexpr (RAWK) {
      // Per K-step group: the lane's 8 channels x RS taps of each of its
      // features (RS 16-byte LDS reads), then one operand per tap.
      constexpr int RSD = RS_C * 4;  // dwords of a lane's run
#pragma unroll
      for (int j = 0; j < KSTEPS; ++j) {
        const int grp = 2 * j + half;
        // whole group in range (Nc % 8 == 0); masked, not branched on
        const uint32_t gmask = cc * TC + 8 * grp < a.Nc ? ~0u : 0u;
        uint32_t raw[MB][RSD];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const u32x4_t* src = kb + ((wm * MB + mb) * 32 + l32) * RC + grp * RS_C;
#pragma unroll
          for (int q = 0; q < RS_C; ++q) {
            const u32x4_t v = src[q];
#pragma unroll
            for (int d = 0; d < 4; ++d) raw[mb][4 * q + d] = v[d] & gmask;
          }
        }
#pragma unroll
        for (int r = 0; r < NR; ++r) {
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            const int tap = r * NS + s;
            const int toff = r * a.Ny + s;
            u32x4_t av[MB], bv[NB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                // elements (channel 2i, tap) and (channel 2i+1, tap) of the run
                const int e0 = (2 * i) * RS_C + tap, e1 = e0 + RS_C;
                const uint32_t sel = ((e0 & 1) ? 0x0302u : 0x0100u) |
                                     ((e1 & 1) ? 0x07060000u : 0x05040000u);
                av[mb][i] = __builtin_amdgcn_perm(raw[mb][e1 >> 1], raw[mb][e0 >> 1], sel);
              }
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bv[nb] = ib[grp * SN + pix[nb] + toff];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
#pragma unroll
              for (int nb = 0; nb < NB; ++nb)
                acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8_t, av[mb]), __builtin_bit_cast(bf16x8_t, bv[nb]),
                    acc[mb][nb], 0, 0, 0);
          }
        }
      }
    } else if constexpr (NR > 0 && NS > 0) {
#pragma unroll
      for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int s = 0; s < NS; ++s) tap_step(r, s);
    } else {
      for (int r = 0; r < Nr; ++r)
        for (int s = 0; s < Ns; ++s) tap_step(r, s);
    }
  }

  // Epilogue: register j of a 32x32 accumulator holds feature
  // m = 8*(j/4) + 4*half + j%4 of output l32.  The feature offset minus the
  // lane-dependent 4*half is wave-uniform and goes in the scalar offset.
  const __amdgpu_buffer_rsrc_t out_rsrc =
      make_rsrc(Out + (int64_t)b0 * a.Nk * a.hw,
                (a.out_total - (int64_t)b0 * a.Nk * a.hw) * (int64_t)sizeof(TO));
  const uint32_t half_off = (uint32_t)(4 * half * a.hw * (int)sizeof(TO));
  const bool k_full = k0 + TK <= a.Nk;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int kw = k0 + (wm * MB + mb) * 32 + 8 * (j >> 2) + (j & 3);  // wave-uniform
      const uint32_t so = (uint32_t)kw * (uint32_t)a.hw * (uint32_t)sizeof(TO);
      if (k_full || kw + 4 * half < a.Nk) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if constexpr (sizeof(TO) == 4) {
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[mb][nb][j]), out_rsrc,
                                                  obyte[nb] + half_off, so, 0);
          } else {
            __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc[mb][nb][j]), out_rsrc,
                                                  obyte[nb] + half_off, so, 0);
          }
        }
      }
    }
  }
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, WM, WN, MB, NB, TC, NR, NS, MAXP, RAWK, PW): tk = 32*WM*MB,
// tp = 32*WN*NB (the largest tile; plans may use fewer outputs per tile);
// NR = NS = 0 reads the stencil size at run time; MAXP position pairs per
// thread bound the slab (ceil(S*Ny/2) <= 256*MAXP; with PW, ceil(tp/2));
// RAWK stages raw Ker; PW gathers the 1x1 inputs of the tile's outputs.
#define CNN_IGEMM2_VARIANTS(X)                          \
  X(400, CNN_BF16, 1, 4, 2, 2, 16, 3, 3, 3, 0, 0)          \
  X(401, CNN_BF16, 2, 2, 2, 2, 16, 3, 3, 3, 0, 0)          \
  X(402, CNN_BF16, 2, 2, 2, 4, 16, 3, 3, 3, 0, 0)          \
  X(404, CNN_BF16, 1, 4, 2, 2, 32, 3, 3, 2, 0, 0)          \
  X(410, CNN_BF16, 1, 4, 2, 2, 16, 0, 0, 4, 0, 0)          \
  X(411, CNN_BF16, 2, 2, 2, 4, 16, 0, 0, 4, 0, 0)          \
  X(412, CNN_BF16, 4, 1, 2, 4, 16, 0, 0, 4, 0, 0)          \
  X(420, CNN_BF16, 1, 4, 2, 2, 16, 3, 3, 3, 1, 0)          \
  X(421, CNN_BF16, 2, 2, 2, 2, 16, 3, 3, 3, 1, 0)          \
  X(422, CNN_BF16, 2, 2, 2, 4, 16, 3, 3, 3, 1, 0)          \
  X(424, CNN_BF16, 1, 4, 2, 2, 32, 3, 3, 2, 1, 0)          \
  X(430, CNN_BF16, 1, 4, 2, 2, 16, 1, 1, 4, 1, 0)          \
  X(431, CNN_BF16, 2, 2, 2, 4, 16, 1, 1, 4, 1, 0)          \
  X(432, CNN_BF16, 4, 1, 2, 4, 16, 1, 1, 4, 1, 0)          \
  X(440, CNN_BF16, 4, 1, 2, 4, 64, 1, 1, 1, 1, 1)          \
  X(441, CNN_BF16, 2, 2, 2, 4, 64, 1, 1, 1, 1, 1)          \
  X(442, CNN_BF16, 1, 4, 2, 2, 64, 1, 1, 1, 1, 1)          \
  X(500, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 3, 0, 0)    \
  X(501, CNN_BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 3, 0, 0)    \
  X(502, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 3, 0, 0)    \
  X(504, CNN_BF16_OBF16, 1, 4, 2, 2, 32, 3, 3, 2, 0, 0)    \
  X(510, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 0, 0, 4, 0, 0)    \
  X(511, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 0, 0, 4, 0, 0)    \
  X(512, CNN_BF16_OBF16, 4, 1, 2, 4, 16, 0, 0, 4, 0, 0)    \
  X(520, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 3, 1, 0)    \
  X(521, CNN_BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 3, 1, 0)    \
  X(522, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 3, 1, 0)    \
  X(524, CNN_BF16_OBF16, 1, 4, 2, 2, 32, 3, 3, 2, 1, 0)    \
  X(530, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 1, 1, 4, 1, 0)    \
  X(531, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 1, 1, 4, 1, 0)    \
  X(532, CNN_BF16_OBF16, 4, 1, 2, 4, 16, 1, 1, 4, 1, 0)    \
  X(540, CNN_BF16_OBF16, 4, 1, 2, 4, 64, 1, 1, 1, 1, 1)    \
  X(541, CNN_BF16_OBF16, 2, 2, 2, 4, 64, 1, 1, 1, 1, 1)    \
  X(542, CNN_BF16_OBF16, 1, 4, 2, 2, 64, 1, 1, 1, 1, 1)

static const Variant2 kVariants2[] = {
#define CNN_ROW2(id, dt, wm, wn, mb, nb, tc, nr, ns, maxp, rawk, pw) \
  {id, dt, 32 * (wm) * (mb), 32 * (wn) * (nb), tc, 16 * (mb) * (nb), nr, ns, maxp, rawk, pw},
    CNN_IGEMM2_VARIANTS(CNN_ROW2)
#undef CNN_ROW2
};

const Variant2* variants2(int* count) {
  *count = (int)(sizeof(kVariants2) / sizeof(kVariants2[0]));
  return kVariants2;
}

int64_t igemm2_blk_vecs(const Variant2& v, int64_t RS) {
  if (v.rawk) {
    const int64_t n = v.tk * (int64_t)rawk_row_chunks((int)RS, v.tc);
    return (n + 63) / 64 * 64;
  }
  const int64_t n = RS * (v.tc / 8) * v.tk;
  return (n + 255) / 256 * 256;
}

int64_t igemm2_lds_bytes(const Variant2& v, int64_t slab_rows, int64_t Ny, int64_t RS,
                         int64_t tp) {
  const int64_t sn = v.pw ? (tp + 1) / 2 * 2 : (slab_rows * Ny + 1) / 2 * 2;
  return 2 * ((v.tc / 8) * sn + igemm2_blk_vecs(v, RS)) * 16;
}

int64_t igemm2_ws_bytes(const Variant2& v, const cnn_problem& p) {
  if (v.rawk) return 0;
  const int64_t n_kt = (p.Nk + v.tk - 1) / v.tk, n_cc = (p.Nc + v.tc - 1) / v.tc;
  return n_kt * n_cc * igemm2_blk_vecs(v, p.Nr * p.Ns) * 16;
}

template <int DT, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int MAXP, int RAWK,
          int PW>
static hipError_t launch_one2(const void* In, const void* Ker, void* Out, void* ws,
                              const ConvArgs& a, int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  constexpr int TK = 32 * WM * MB;
  const int64_t RS = (int64_t)a.Nr * a.Ns;
  int64_t blk;
  const void* kp = Ker;
  if (RAWK) {
    blk = (TK * (int64_t)rawk_row_chunks((int)RS, TC) + 63) / 64 * 64;
  } else {
    blk = (RS * (TC / 8) * TK + 255) / 256 * 256;
    const int64_t n_kt = (a.Nk + TK - 1) / TK, n_cc = (a.Nc + TC - 1) / TC;
    const int64_t total = n_kt * n_cc * blk;
    int64_t pgrid = (total + 255) / 256;
    if (pgrid > 4096) pgrid = 4096;
    hipLaunchKernelGGL(pack_ker_bf16, dim3((unsigned)pgrid), dim3(256), 0, stream,
                       (const bf16_t*)Ker, (u32x4_t*)ws, a, TK, TC, (int)blk, total);
    kp = ws;
  }
  auto kern = (!PW && (a.Ny & 1))
                  ? conv_igemm2<TO, WM, WN, MB, NB, TC, NR, NS, MAXP, (RAWK != 0), (PW != 0), true>
                  : conv_igemm2<TO, WM, WN, MB, NB, TC, NR, NS, MAXP, (RAWK != 0), (PW != 0), false>;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(256), (unsigned)lds, stream,
                     (const bf16_t*)In, (const u32x4_t*)kp, (TO*)Out, a, (int)blk);
  return hipGetLastError();
}

hipError_t launch_igemm2(const Variant2& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASE2(id, dt, wm, wn, mb, nb, tc, nr, ns, maxp, rawk, pw)                    \
  case id:                                                                              \
    return launch_one2<dt, wm, wn, mb, nb, tc, nr, ns, maxp, rawk, pw>(In, Ker, Out, ws, a, \
                                                                       lds_bytes, stream);
    CNN_IGEMM2_VARIANTS(CNN_CASE2)
#undef CNN_CASE2
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

// Implicit-GEMM convolution for few input channels and wide stencils
// (bf16 MFMA, gfx950), e.g. a 3-channel 7x7 input layer.
//
// Same tile schedule as the other implicit-GEMM kernels (paper Sec. 2.1,
// Listing 3 with W_c = N_c; tiles of tp consecutive outputs of the
// flattened (b, w, h) index by 64 features), but with Nc*Nr*Ns small the
// whole contraction fits one stage, so the K dimension of the MFMA is the
// flattened (c, r, s) index instead of channels:
//
// * K order: q = c*Nr + r, then s padded to 8, so each 8-element K-group of
//   a lane is one (c, r) row of the stencil -- 8 consecutive input columns.
//   ceil(Nc*Nr/2) MFMA K-steps of 16; padded taps carry zero weights.
// * Ker (A operand): packed once per workgroup into an LDS image
//   [K-step][lane half][feature][8] -- one 16-byte read per operand.
// * In (B operand): the tile's halo'd slab -- every input row the tile's
//   outputs touch, all Nc channels -- staged once in its natural layout
//   (row stride Ny + 8 rounded up to 8, columns past Ny zero) by unaligned
//   16-byte loads of 8 columns, and each operand gathered at the lane's
//   output position plus the (c, r) offset: eight 16-bit LDS reads, or four
//   32-bit reads when the h stride is 2 (the position is then even).
// * Ker runs (Ns <= 8 taps of one (k, c, r)) are one unaligned 16-byte load
//   each, the taps past Ns masked to zero.
// * A 16-byte load whose last dword straddles the end of its tensor loses
//   that dword to the range check; the only element that matters there is
//   the tensor's last, loaded once and patched in.
// * One tile per workgroup and several workgroups per CU: a workgroup's
//   Out stores (the dominant HBM traffic of such layers) overlap other
//   workgroups' staging and MFMA work.
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_s(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// Dividers for the launch's runtime divisors (made on the host).
struct SmallcDiv {
  FastDiv cpr, nx, hw, nh, nr, kt;
  FastDiv s0;  // slab rows of the first tile (most tiles have as many)
  int S0;
};

// KS: largest number of K-steps (ceil(Nc*Nr/2)) the registers hold.  SH2:
// sh == 2 (operands gathered with 32-bit LDS reads).  FC, FR, FS, FST: a
// fixed stencil (Nc, Nr, Ns and both strides) compiled in, 0 for any: the
// address arithmetic and the K-step count then fold at compile time (the
// 3-channel 7x7 stride-2 input layer).  Two workgroups per CU (two waves per
// SIMD) run at once, so a wave keeps to 256 registers.
template <typename TO, int NB, int KS, bool SH2, int FC = 0, int FR = 0, int FS = 0, int FST = 0>
__global__ __launch_bounds__(256, 2) void conv_smallc(const bf16_t* __restrict__ In,
                                                   const bf16_t* __restrict__ Ker,
                                                   TO* __restrict__ Out, ConvArgs a,
                                                   SmallcDiv dv) {
  const int Nc = FC ? FC : a.Nc, Nr = FR ? FR : a.Nr, Ns = FS ? FS : a.Ns;
  const int sw = FST ? FST : a.sw, sh = FST ? FST : a.sh;
  auto div_nr = [&](int q) -> int {
    if constexpr (FR != 0) return q / FR;
    else return fdiv(q, dv.nr);
  };
  constexpr int MB = 2;         // 64 features per tile, shared by the 4 waves
  constexpr int TK = 32 * MB;
  constexpr int KVEC = KS * 2 * TK;  // Ker image vectors
  static_assert(KVEC % 256 == 0, "whole Ker image vectors per thread");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* kimg = reinterpret_cast<u32x4_t*>(smem);           // [KS][2][TK]
  bf16_t* slab = reinterpret_cast<bf16_t*>(kimg + KVEC);      // [Nc][S][RSTR]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

  // ---- several tiles per workgroup, strided by the grid: at any time the
  // workgroups of an XCD work on neighbouring tiles, whose slabs share halo
  // rows in its L2.  The Ker image is packed again only when the k tile
  // changes, and each next tile's slab loads are issued before the current
  // tile's products.
  const int n_tiles = a.n_ptiles * a.n_ktiles;
  const int G = (int)gridDim.x;
  const int t_first = xcd_remap(blockIdx.x, gridDim.x);
  const int RSTR = (a.Ny + 15) & ~7;                       // LDS row stride (elements)
  const int nq = Nc * Nr;                              // (c, r) rows of the stencil
  const int nks = (nq + 1) >> 1;                           // K-steps
  const int cpr = RSTR / 8;                                // 16-byte chunks per slab row
  const __amdgpu_buffer_rsrc_t ir = rsrc_s(In, a.in_total * 2);
  const uint32_t in_last =
      t_first < n_tiles ? __builtin_amdgcn_raw_buffer_load_b16(ir, (uint32_t)((a.in_total - 1) * 2), 0, 0)
                        : 0u;

  // Tile geometry: the first slab row G0 (flattened b, x) and the slab
  // rows S of tile t (its outputs p0 .. plast).
  struct Geo {
    int p0, plast, k0, kt, b0, G0, S;
    FastDiv fs;  // divider for S
  };
  auto geo = [&](int t) {
    Geo g;
    const int pt = fdiv(t, dv.kt);
    g.kt = t - pt * a.n_ktiles;
    g.p0 = pt * a.tp;
    g.k0 = g.kt * TK;
    g.plast = min(g.p0 + a.tp, a.npix) - 1;
    g.b0 = fdiv(g.p0, dv.hw);
    const int w0 = fdiv(g.p0 - g.b0 * a.hw, dv.nh);
    const int b1 = fdiv(g.plast, dv.hw), w1 = fdiv(g.plast - b1 * a.hw, dv.nh);
    g.G0 = g.b0 * a.Nx + sw * w0;
    g.S = b1 * a.Nx + sw * w1 + Nr - g.G0;
    g.fs = g.S == dv.S0 ? dv.s0 : make_fastdiv((uint32_t)g.S);
    return g;
  };

  // Slab loads: element (c, row, col) of the LDS image is In[b][c][x][col]
  // for flattened input row G0 + row = b*Nx + x, zero for col >= Ny.  Chunk
  // (c, row, k8) = columns 8 k8 .. +7, one unaligned 16-byte load; a thread
  // holds chunks tid + 256 u (u < U) of the tile in flight, more in batches.
  constexpr int U = 4;
  u32x4_t sv[U];
  int soff[U];
  auto slab_load = [&](const Geo& g, int e0) __attribute__((always_inline)) {
    const int n = Nc * g.S * cpr;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = min(e0 + tid + 256 * u, n - 1);
      const int crow = fdiv(e, dv.cpr);
      const int k8 = e - crow * cpr;
      const int c = fdiv(crow, g.fs);
      const int row = crow - c * g.S;
      const int gr = g.G0 + row;
      const int b = fdiv(gr, dv.nx);
      const int x = gr - b * a.Nx;
      soff[u] = (int)((int64_t)b * a.in_img + (int64_t)c * a.nxny + (int64_t)x * a.Ny) + 8 * k8;
      sv[u] = __builtin_bit_cast(
          u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ir, (uint32_t)(soff[u] * 2), 0, 0));
    }
  };
  auto slab_write = [&](const Geo& g, int e0) __attribute__((always_inline)) {
    const int n = Nc * g.S * cpr;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = e0 + tid + 256 * u;
      if (e >= n) continue;
      const int crow = fdiv(e, dv.cpr);
      const int k8 = e - crow * cpr;
      const int d = (int)(a.in_total - 1) - soff[u];
      u32x4_t vv = sv[u];
#pragma unroll
      for (int t = 0; t < 8; t += 2) {
        uint32_t w = vv[t >> 1];
        if (d == t) w = (w & 0xffff0000u) | in_last;
        if (d == t + 1) w = (w & 0xffffu) | (in_last << 16);
        const int col = 8 * k8 + t;
        const uint32_t keep = (col < a.Ny ? 0xffffu : 0u) | (col + 1 < a.Ny ? 0xffff0000u : 0u);
        vv[t >> 1] = w & keep;
      }
      *reinterpret_cast<u32x4_t*>(slab + crow * RSTR + 8 * k8) = vv;
    }
  };

  // Ker image: vector (j, h, kk) holds Ker[k0+kk][c][r][0..7] for the
  // (c, r) row q = 2j + h, zero past Ns, nq or Nk.  All of a thread's
  // loads are issued before any is used.
  auto load_kimg = [&](int k0) __attribute__((always_inline)) {
    const int64_t ker_total = (int64_t)a.Nk * Nc * Nr * Ns;
    const __amdgpu_buffer_rsrc_t kr = rsrc_s(Ker, ker_total * 2);
    const uint32_t ker_last =
        __builtin_amdgcn_raw_buffer_load_b16(kr, (uint32_t)((ker_total - 1) * 2), 0, 0);
    constexpr int PER = KVEC / 256;
    u32x4_t e[PER];
    int ebase[PER];
    bool eok[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int v = tid + 256 * u;
      const int kk = v % TK;
      const int jh = v / TK;  // 2j + h == q
      const int k = k0 + kk;
      eok[u] = k < a.Nk && jh < nq;
      const int q = eok[u] ? jh : 0;
      const int c = div_nr(q), r = q - c * Nr;
      ebase[u] = (((eok[u] ? k : 0) * Nc + c) * Nr + r) * Ns;
      e[u] = __builtin_bit_cast(
          u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(kr, (uint32_t)(ebase[u] * 2), 0, 0));
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      u32x4_t vv = e[u];
      const int d = (int)(ker_total - 1) - ebase[u];
#pragma unroll
      for (int t = 0; t < 8; t += 2) {
        // taps t, t+1 of the run: zero past Ns (and for invalid vectors);
        // the tensor's last element patched in
        uint32_t w = vv[t >> 1];
        if (d == t) w = (w & 0xffff0000u) | ker_last;
        if (d == t + 1) w = (w & 0xffffu) | (ker_last << 16);
        const uint32_t keep = (eok[u] ? (t < Ns ? 0xffffu : 0u) | (t + 1 < Ns ? 0xffff0000u : 0u)
                                      : 0u);
        vv[t >> 1] = w & keep;
      }
      kimg[tid + 256 * u] = vv;
    }
  };

  const uint32_t half_off = (uint32_t)(4 * half * a.hw * (int)sizeof(TO));
  int kt_img = -1;  // k tile of the Ker image in LDS
  if (t_first < n_tiles) slab_load(geo(t_first), 0);
  for (int t = t_first; t < n_tiles; t += G) {
    const Geo g = geo(t);
    const int n_chunks = Nc * g.S * cpr;
    __syncthreads();  // the previous tile's operand reads are done
    if (g.kt != kt_img) {
      load_kimg(g.k0);
      kt_img = g.kt;
    }
    // this tile's slab: the first batch is in flight (issued a tile ago)
    for (int e0 = 0; e0 < n_chunks; e0 += 256 * U) {
      if (e0 > 0) slab_load(g, e0);
      slab_write(g, e0);
    }
    __syncthreads();
    if (t + G < n_tiles) slab_load(geo(t + G), 0);  // lands during this tile's products

    // Output side: each lane's slab position and Out offset; lanes past the
    // tile's last output recompute and rewrite it (no store masks).
    int pbase[NB];
    uint32_t obyte[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int p = g.p0 + (wave * NB + nb) * 32 + l32;
      const int pc = p <= g.plast ? p : g.plast;
      const int b = fdiv(pc, dv.hw);
      const int q = pc - b * a.hw;
      const int w = fdiv(q, dv.nh);
      const int h = q - w * a.Nh;
      pbase[nb] = (b * a.Nx + sw * w - g.G0) * RSTR + sh * h;
      obyte[nb] = (uint32_t)(((int64_t)(b - g.b0) * a.Nk * a.hw + q) * (int64_t)sizeof(TO));
    }

    f32x16_t acc[MB][NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;

#pragma unroll
    for (int j = 0; j < KS; ++j) {
      if (j < nks) {
        const int q = min(2 * j + half, nq - 1);  // past nq: weights are zero
        const int c = div_nr(q), r = q - c * Nr;
        const int qoff = (c * g.S + r) * RSTR;
        u32x4_t bv[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const bf16_t* src = slab + qoff + pbase[nb];
          if constexpr (SH2) {
            // the position's first column is even: 4-byte-aligned words
#pragma unroll
            for (int d = 0; d < 4; ++d) bv[nb][d] = reinterpret_cast<const uint32_t*>(src)[d];
          } else {
#pragma unroll
            for (int d = 0; d < 4; ++d)
              bv[nb][d] = (uint32_t)src[2 * d] | ((uint32_t)src[2 * d + 1] << 16);
          }
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const u32x4_t av = kimg[(2 * j + half) * TK + mb * 32 + l32];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, av), __builtin_bit_cast(bf16x8_t, bv[nb]),
                acc[mb][nb], 0, 0, 0);
        }
      }
    }

    // Epilogue: register j of a 32x32 accumulator holds feature
    // 8*(j/4) + 4*half + j%4 of output l32.
    const __amdgpu_buffer_rsrc_t out_rsrc =
        rsrc_s(Out + (int64_t)g.b0 * a.Nk * a.hw,
               (a.out_total - (int64_t)g.b0 * a.Nk * a.hw) * (int64_t)sizeof(TO));
    const bool k_full = g.k0 + TK <= a.Nk;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int kw = g.k0 + mb * 32 + 8 * (j >> 2) + (j & 3);
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
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, NB, KS, FC, FR, FS, FST): tk = 64, tp = 128*NB (largest tile);
// KS = most K-steps, ceil(Nc*Nr/2) <= KS; any Ns <= 8, any stride, unless
// FC..FST fix the stencil (1003, 1103: 3 channels, 7x7, stride 2).
#define CNN_SMALLC_VARIANTS(X)                   \
  X(1000, CNN_BF16, 2, 12, 0, 0, 0, 0)           \
  X(1001, CNN_BF16, 1, 12, 0, 0, 0, 0)           \
  X(1002, CNN_BF16, 2, 24, 0, 0, 0, 0)           \
  X(1003, CNN_BF16, 2, 12, 3, 7, 7, 2)           \
  X(1100, CNN_BF16_OBF16, 2, 12, 0, 0, 0, 0)     \
  X(1101, CNN_BF16_OBF16, 1, 12, 0, 0, 0, 0)     \
  X(1102, CNN_BF16_OBF16, 2, 24, 0, 0, 0, 0)     \
  X(1103, CNN_BF16_OBF16, 2, 12, 3, 7, 7, 2)

static const VariantS kVariantsS[] = {
#define CNN_ROWS(id, dt, nb, ks, fc, fr, fs, fst) \
  {id, dt, 64, 128 * (nb), ks, 16 * 2 * (nb), fc, fr, fs, fst},
    CNN_SMALLC_VARIANTS(CNN_ROWS)
#undef CNN_ROWS
};

bool smallc_stencil_ok(const VariantS& v, const cnn_problem& p) {
  return v.nc == 0 || (p.Nc == v.nc && p.Nr == v.nr && p.Ns == v.ns && p.sw == v.st && p.sh == v.st);
}

const VariantS* variants_smallc(int* count) {
  *count = (int)(sizeof(kVariantsS) / sizeof(kVariantsS[0]));
  return kVariantsS;
}

int64_t smallc_lds_bytes(const VariantS& v, const cnn_problem& p, int64_t slab_rows) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  return (int64_t)v.ks * 2 * v.tk * 16 + p.Nc * slab_rows * ((Ny + 15) & ~(int64_t)7) * 2;
}

template <int DT, int NB, int KS, int FC, int FR, int FS, int FST>
static hipError_t launch_s(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                           int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  auto kern = FST ? conv_smallc<TO, NB, KS, FST == 2, FC, FR, FS, FST>
                  : a.sh == 2 ? conv_smallc<TO, NB, KS, true> : conv_smallc<TO, NB, KS, false>;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  // two workgroups per CU fill the registers; each takes every grid-th tile
  const int64_t wgs = std::min<int64_t>(a.grid, 2 * (int64_t)device_cus());
  SmallcDiv dv;
  dv.cpr = make_fastdiv((uint32_t)(((a.Ny + 15) & ~7) / 8));
  dv.nx = make_fastdiv((uint32_t)a.Nx);
  dv.hw = make_fastdiv((uint32_t)a.hw);
  dv.nh = make_fastdiv((uint32_t)a.Nh);
  dv.nr = make_fastdiv((uint32_t)a.Nr);
  dv.kt = make_fastdiv((uint32_t)a.n_ktiles);
  {
    // the first tile's slab rows, as the kernel's geometry computes them
    const int plast = (int)std::min<int64_t>(a.tp, a.npix) - 1;
    const int b1 = plast / a.hw, w1 = (plast - b1 * a.hw) / a.Nh;
    dv.S0 = b1 * a.Nx + a.sw * w1 + a.Nr;
    dv.s0 = make_fastdiv((uint32_t)dv.S0);
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)wgs), dim3(256), (unsigned)lds, stream,
                     (const bf16_t*)In, (const bf16_t*)Ker, (TO*)Out, a, dv);
  return hipGetLastError();
}

hipError_t launch_smallc(const VariantS& v, const void* In, const void* Ker, void* Out,
                         const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASES(id, dt, nb, ks, fc, fr, fs, fst) \
  case id:                                        \
    return launch_s<dt, nb, ks, fc, fr, fs, fst>(In, Ker, Out, a, lds_bytes, stream);
    CNN_SMALLC_VARIANTS(CNN_CASES)
#undef CNN_CASES
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

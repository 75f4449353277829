// Implicit-GEMM convolution on MFMA (gfx950).
//
// The paper's tile schedule (Sec. 2.1, Listing 3, with W_c = N_c, i.e. its
// Case 1): each workgroup owns an output tile -- tk output features by tp
// consecutive outputs of the flattened (b, w, h) index (the paper's
// composite T_bhw) -- keeps it resident in accumulator registers, and walks
// the input features tc at a time.  For every c step it copies the halo'd
// In tile and the Ker tile from HBM into LDS, then runs the point loops
// (taps r, s; features k; outputs b, w, h; channels c) as MFMA products.
//
// GEMM view: D[k][p] += A[k][(c,r,s)] * B[(c,r,s)][p] with A = Ker and
// B = the im2col view of In.  Per tap (r, s) the contraction runs over c:
//   * bf16: v_mfma_f32_32x32x16_bf16 -- each lane feeds 8 consecutive c;
//   * fp32: v_mfma_f32_32x32x2f32    -- each lane feeds 1 c.
// Output features are the MFMA rows (M) and outputs the columns (N), so a
// half-wave's 32 results of one accumulator register are 32 consecutive
// outputs in Out's [b][k][w][h] order: every store is a contiguous run.
//
// In tile ("slab"): a tile of consecutive outputs touches whole output rows
// (b, w), so it reads the contiguous range of flattened (b, x) input rows
// from the first row's sw*w to the last row's sw*w + Nr - 1, all Ny
// columns.  It is staged channel-group-major, [c/KV][row][y][KV], KV = 8
// channels per 16-byte vector for bf16: lane reads of one tap are then
// 16-byte vectors at consecutive positions.
// Ker tile: staged [tap][c/KV][k][KV], so A reads are consecutive vectors.
//
// Split channels (the paper's Case 2, P_c > 1): launched with gridDim.y = kc,
// workgroup (tile, z) walks only the channels [z*cs, z*cs + cs) (cs a
// multiple of TC, so no stage straddles two slices) and writes its fp32
// partial tile to slice z of a workspace laid out as Out; splitc_reduce then
// adds the kc slices in slice order (a fixed order: the result does not
// depend on which workgroup finishes first) and writes Out.  Unsplit
// launches have gridDim.y = 1 and cs >= Nc.
#include "internal.h"
#include "common.h"

namespace cnnlib {

template <typename TI> struct Pack;
template <> struct Pack<float> {
  static constexpr int KV = 1;
  typedef float V;
};
template <> struct Pack<bf16_t> {
  static constexpr int KV = 8;
  typedef u32x4_t V;
};

__device__ __forceinline__ void mfma32(f32x16_t& acc, float a, float b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma32(f32x16_t& acc, const u32x4_t& a, const u32x4_t& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}

// Gather KV channels (c, c+1, ...) of one position into an LDS vector;
// channels at or beyond Nc read as zero.
__device__ __forceinline__ float gather(const float* __restrict__ p, int64_t cstride, int c, int Nc) {
  return c < Nc ? p[(int64_t)c * cstride] : 0.f;
}
__device__ __forceinline__ u32x4_t gather(const bf16_t* __restrict__ p, int64_t cstride, int c, int Nc) {
  u32x4_t v;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = (c + 2 * i < Nc) ? p[(int64_t)(c + 2 * i) * cstride] : 0u;
    const uint32_t hi = (c + 2 * i + 1 < Nc) ? p[(int64_t)(c + 2 * i + 1) * cstride] : 0u;
    v[i] = lo | (hi << 16);
  }
  return v;
}

template <typename TI, typename TO, int WM, int WN, int MB, int NB, int TC>
__global__ __launch_bounds__(256) void conv_igemm(const TI* __restrict__ In,
                                                  const TI* __restrict__ Ker,
                                                  TO* __restrict__ Out, ConvArgs a, int cs) {
  constexpr int KV = Pack<TI>::KV;
  typedef typename Pack<TI>::V V;
  constexpr int TK = 32 * WM * MB;
  constexpr int TP = 32 * WN * NB;
  constexpr int G = TC / KV;      // channel groups per stage
  constexpr int KSTEPS = G / 2;   // MFMA K-steps per tap (two groups each)
  static_assert(WM * WN == 4, "four waves per workgroup");
  static_assert(TC % (2 * KV) == 0, "stage must hold whole MFMA K-steps");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int SN = a.slab_max * a.Ny;  // LDS positions per channel group
  V* lds_in = reinterpret_cast<V*>(smem);
  V* lds_ker = lds_in + G * SN;
  const int RS = a.Nr * a.Ns;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, half = lane >> 5;

  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int pt = tile / a.n_ktiles;
  const int kt = tile - pt * a.n_ktiles;
  const int p0 = pt * TP;
  const int k0 = kt * TK;
  const int plast = min(p0 + TP, a.npix) - 1;

  // Input rows of the tile: flattened (b, x) rows G0 .. G0 + S - 1.
  const int b0 = p0 / a.hw, w0 = (p0 - b0 * a.hw) / a.Nh;
  const int b1 = plast / a.hw, w1 = (plast - b1 * a.hw) / a.Nh;
  const int G0 = b0 * a.Nx + a.sw * w0;
  const int S = b1 * a.Nx + a.sw * w1 + a.Nr - G0;
  const int SNt = S * a.Ny;

  // Per lane and N-block: LDS position of the output's (r, s) = (0, 0) tap
  // and the Out offset of its k = 0 plane.  Outputs past the end reuse the
  // last valid one for reading and are not stored.
  int pix[NB];
  int64_t obase[NB];
  bool pval[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int p = p0 + (wn * NB + nb) * 32 + l32;
    pval[nb] = p <= plast;
    const int pc = p <= plast ? p : plast;
    const int b = pc / a.hw;
    const int q = pc - b * a.hw;
    const int w = q / a.Nh;
    const int h = q - w * a.Nh;
    pix[nb] = (b * a.Nx + a.sw * w - G0) * a.Ny + a.sh * h;
    obase[nb] = (int64_t)b * a.Nk * a.hw + q;
  }

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;

  const int gpos0 = G0 * a.Ny;  // flattened (b, x, y) index of the slab start
  const int c_begin = (int)blockIdx.y * cs;
  const int c_end = min(a.Nc, c_begin + cs);
  Out += (int64_t)blockIdx.y * a.out_total;  // this slice's partial Out
  for (int c0 = c_begin; c0 < c_end; c0 += TC) {
    __syncthreads();  // previous stage fully consumed
    // In slab: positions are consecutive in y, then x, then b.
    // (unrolled so that several positions' loads are in flight together)
#pragma unroll 2
    for (int pos = tid; pos < SNt; pos += 256) {
      const int gp = gpos0 + pos;
      const int b = gp / a.nxny;
      const TI* src = In + (int64_t)b * a.in_img + (gp - b * a.nxny);
#pragma unroll
      for (int g = 0; g < G; ++g) lds_in[g * SN + pos] = gather(src, a.nxny, c0 + g * KV, a.Nc);
    }
    // Ker tile, [tap][group][k].
#pragma unroll 4
    for (int idx = tid; idx < RS * G * TK; idx += 256) {
      const int kk = idx % TK;
      const int rest = idx / TK;
      const int g = rest % G;
      const int tap = rest / G;
      const int k = k0 + kk;
      V v;
      if (k < a.Nk) {
        v = gather(Ker + (int64_t)k * a.Nc * RS + tap, RS, c0 + g * KV, a.Nc);
      } else {
        v = V{};
      }
      lds_ker[idx] = v;
    }
    __syncthreads();

    for (int r = 0; r < a.Nr; ++r) {
      for (int s = 0; s < a.Ns; ++s) {
        const int tap = r * a.Ns + s;
        const int toff = r * a.Ny + s;
        const V* kt_base = lds_ker + tap * G * TK + (wm * MB) * 32 + l32;
#pragma unroll
        for (int j = 0; j < KSTEPS; ++j) {
          const int grp = 2 * j + half;
          V av[MB], bv[NB];
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) av[mb] = kt_base[grp * TK + mb * 32];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) bv[nb] = lds_in[grp * SN + pix[nb] + toff];
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) mfma32(acc[mb][nb], av[mb], bv[nb]);
        }
      }
    }
  }

  // Epilogue: register j of a 32x32 accumulator holds row
  // m = 8*(j/4) + 4*half + j%4 (output feature) of column l32 (output).
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int k = k0 + (wm * MB + mb) * 32 + 8 * (j >> 2) + 4 * half + (j & 3);
      if (k < a.Nk) {
        const int64_t koff = (int64_t)k * a.hw;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          if (pval[nb]) Out[obase[nb] + koff] = from_f32<TO>(acc[mb][nb][j]);
      }
    }
  }
}

// ---- instantiation table ------------------------------------------------
// (id, dtype, WM, WN, MB, NB, TC): tk = 32*WM*MB, tp = 32*WN*NB.
#define CNN_IGEMM_VARIANTS(X)              \
  X(100, CNN_F32, 1, 4, 2, 2, 8)           \
  X(101, CNN_F32, 2, 2, 2, 2, 8)           \
  X(102, CNN_F32, 1, 4, 1, 2, 8)           \
  X(103, CNN_F32, 2, 2, 1, 1, 8)           \
  X(104, CNN_F32, 1, 4, 2, 1, 8)           \
  X(200, CNN_BF16, 1, 4, 2, 2, 32)         \
  X(201, CNN_BF16, 2, 2, 2, 2, 32)         \
  X(202, CNN_BF16, 2, 2, 2, 4, 16)         \
  X(203, CNN_BF16, 4, 1, 2, 4, 16)         \
  X(204, CNN_BF16, 1, 4, 1, 2, 32)         \
  X(205, CNN_BF16, 2, 2, 1, 1, 32)         \
  X(206, CNN_BF16, 1, 4, 2, 1, 32)         \
  X(300, CNN_BF16_OBF16, 1, 4, 2, 2, 32)   \
  X(301, CNN_BF16_OBF16, 2, 2, 2, 2, 32)   \
  X(302, CNN_BF16_OBF16, 2, 2, 2, 4, 16)   \
  X(303, CNN_BF16_OBF16, 4, 1, 2, 4, 16)   \
  X(304, CNN_BF16_OBF16, 1, 4, 1, 2, 32)   \
  X(305, CNN_BF16_OBF16, 2, 2, 1, 1, 32)   \
  X(306, CNN_BF16_OBF16, 1, 4, 2, 1, 32)

template <int DT> struct DtypeTypes;
template <> struct DtypeTypes<CNN_F32> { typedef float TI; typedef float TO; };
template <> struct DtypeTypes<CNN_BF16> { typedef bf16_t TI; typedef float TO; };
template <> struct DtypeTypes<CNN_BF16_OBF16> { typedef bf16_t TI; typedef bf16_t TO; };

static const Variant kVariants[] = {
#define CNN_ROW(id, dt, wm, wn, mb, nb, tc) \
  {id, CNN_K_IGEMM, dt, 32 * (wm) * (mb), 32 * (wn) * (nb), tc, 256, 16 * (mb) * (nb)},
    CNN_IGEMM_VARIANTS(CNN_ROW)
#undef CNN_ROW
};

const Variant* variants(int* count) {
  *count = (int)(sizeof(kVariants) / sizeof(kVariants[0]));
  return kVariants;
}

int64_t igemm_lds_bytes(const Variant& v, int64_t slab_rows, int64_t Ny, int64_t RS) {
  const int64_t kv = v.dtype == CNN_F32 ? 1 : 8;
  const int64_t vec = v.dtype == CNN_F32 ? 4 : 16;
  const int64_t groups = v.tc / kv;
  return (groups * slab_rows * Ny + RS * groups * v.tk) * vec;
}

template <int DT, int WM, int WN, int MB, int NB, int TC>
static hipError_t launch_one(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                             int64_t lds, hipStream_t stream, int kc, int cs, bool split) {
  typedef typename DtypeTypes<DT>::TI TI;
  typedef typename DtypeTypes<DT>::TO TO;
  // split launches write fp32 partial sums whatever the Out type: the bf16
  // instantiation with fp32 Out
  if constexpr (DT == CNN_BF16_OBF16)
    if (split)
      return launch_one<CNN_BF16, WM, WN, MB, NB, TC>(In, Ker, Out, a, lds, stream, kc, cs, true);
  auto kern = conv_igemm<TI, TO, WM, WN, MB, NB, TC>;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid, (unsigned)kc), dim3(256), (unsigned)lds, stream,
                     (const TI*)In, (const TI*)Ker, (TO*)Out, a, cs);
  return hipGetLastError();
}

// Out[o] = sum over z = 0 .. kc-1, in that order, of Part[z][o].  Slices
// are loaded 16 (then 4) at a time, independent loads in flight together;
// the additions stay in slice order.
template <typename TO>
__global__ __launch_bounds__(256) void splitc_reduce(const float* __restrict__ Part,
                                                     TO* __restrict__ Out, int kc, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n; o += stride) {
    const float* p = Part + o;
    float s;
    int z;
    if (kc >= 16) {
      float v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = p[(int64_t)i * n];
      s = v[0];
#pragma unroll
      for (int i = 1; i < 16; ++i) s += v[i];
      z = 16;
    } else {
      s = p[0];
      z = 1;
    }
    for (; z + 16 <= kc; z += 16) {
      float v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = p[(int64_t)(z + i) * n];
#pragma unroll
      for (int i = 0; i < 16; ++i) s += v[i];
    }
    for (; z + 4 <= kc; z += 4) {
      float v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] = p[(int64_t)(z + i) * n];
#pragma unroll
      for (int i = 0; i < 4; ++i) s += v[i];
    }
    for (; z < kc; ++z) s += p[(int64_t)z * n];
    Out[o] = from_f32<TO>(s);
  }
}

static hipError_t launch_igemm_kc(const Variant& v, const void* In, const void* Ker, void* Out,
                                  const ConvArgs& a, int64_t lds_bytes, hipStream_t stream,
                                  int kc, int cs, bool split) {
  switch (v.id) {
#define CNN_CASE(id, dt, wm, wn, mb, nb, tc) \
  case id:                                   \
    return launch_one<dt, wm, wn, mb, nb, tc>(In, Ker, Out, a, lds_bytes, stream, kc, cs, split);
    CNN_IGEMM_VARIANTS(CNN_CASE)
#undef CNN_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_igemm(const Variant& v, const void* In, const void* Ker, void* Out,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  return launch_igemm_kc(v, In, Ker, Out, a, lds_bytes, stream, 1, a.Nc, false);
}

int64_t splitc_slice_channels(int64_t Nc, int64_t tc, int64_t kc) {
  const int64_t stages = (Nc + tc - 1) / tc;
  return (stages + kc - 1) / kc * tc;
}

hipError_t launch_splitc_reduce(const float* Part, void* Out, int kc, int64_t n, int dtype,
                                hipStream_t stream) {
  // One wave per workgroup: a small Out (25k elements for a batch-1 7x7
  // layer) then spreads its loads over every CU rather than a hundred
  // (0.05 us less on that layer's 7.4).
  int64_t blocks = (n + 63) / 64;
  if (blocks > 8192) blocks = 8192;  // grid-stride loop covers the rest
  if (dtype == CNN_BF16_OBF16)
    hipLaunchKernelGGL(splitc_reduce<bf16_t>, dim3((unsigned)blocks), dim3(64), 0, stream,
                       Part, (bf16_t*)Out, kc, n);
  else
    hipLaunchKernelGGL(splitc_reduce<float>, dim3((unsigned)blocks), dim3(64), 0, stream,
                       Part, (float*)Out, kc, n);
  return hipGetLastError();
}

hipError_t launch_splitc(const Variant& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, int kc, int dtype,
                         hipStream_t stream) {
  const int cs = (int)splitc_slice_channels(a.Nc, v.tc, kc);
  hipError_t e = launch_igemm_kc(v, In, Ker, ws, a, lds_bytes, stream, kc, cs, true);
  if (e != hipSuccess) return e;
  return launch_splitc_reduce((const float*)ws, Out, kc, a.out_total, dtype, stream);
}

}  // namespace cnnlib

// Channel-slice kernel: the paper's Case 2 (Sec. 2.1, W_c < N_c, the partial
// Outs summed at the end as in Sec. 2.3) for layers whose output is too
// small to occupy the chip with whole-channel tiles -- the deep layers of a
// network at batch 1, where a 7x7 output has 49 positions and Ker (Nk x Nc
// x taps) is nearly all of the traffic.
//
// Workgroup (tile, z) owns 32 output features x 64 consecutive outputs of the
// flattened (b, w, h) index (the paper's composite T_bhw) and the channels
// [z*cs, z*cs + cs) of slice z, in stages of TC = 16, 32, 64 or 128
// channels.  A stage issues all of its global loads before it waits on any:
// the tile's Ker rows (32 features x TC channels x all taps, 16-byte loads of
// the rows as they lie, one feature's 8 channels per thread) and the halo'd
// In slab of the tile ((position, 8-channel group) tasks spread over all
// threads: with one position's groups per thread, 81 threads issued every
// load of the 7x7 layer's slab, 0.18 us slower).  The stage therefore costs
// one memory latency rather than one per tap or channel group.  Both then go to LDS in (tap, channel) order:
//   Ker [tap][c/8][k (+1)][8]    an A operand (8 channels of one feature at
//                                one tap) is one 16-byte read; one pad
//                                vector per 32 features keeps the four
//                                channel groups a thread quad writes off
//                                one bank;
//   In  [position][c/8 (+1)][8]  a B operand (8 channels of one position) is
//                                one 16-byte read; one pad vector per
//                                position spreads 32 lanes over the banks.
// Ker is transposed in registers: a thread's loads hold 8 channels x T taps
// of one feature, from which it assembles each tap's 8 channels.
//
// GEMM view of a stage: D[k][p] += sum over (tap, c) of Ker[k][c][tap] *
// In[c][pos(p) + off(tap)] on v_mfma_f32_32x32x16_bf16, a K-step being one
// tap x 16 channels.  The workgroup has two waves per K group -- outputs
// 0-31 and 32-63 -- and TC / 16 K groups (two for TC = 16), each taking
// every (TC/16)-th K-step; the groups' accumulators are added through LDS
// (always in group order), and the slice's fp32 partial tile goes to slice
// z of the workspace.  On the batch-1 512-channel 3x3 layer TC = 32 (256
// workgroups) measured fastest: TC = 16 doubles the partials, TC = 64
// halves the workgroups.  The ordered reduce of the kc slices
// (splitc_reduce) then writes Out, so the result does not depend on which
// workgroup finishes first.
//
// Workspace-free instantiations:
//   atomic (MODE 1, fp32 Out): a fill kernel zeroes Out, then every slice
//     adds its partial tile into Out with fp32 atomic adds.  The sum is then
//     formed in the order the workgroups arrive, so the last bits of Out may
//     differ from call to call (integer-valued sums excepted: they are exact
//     in any order);
//   direct (MODE 2, any Out type): one slice (kc = 1) of 128-channel stages
//     on 1024-thread workgroups (eight K groups), each workgroup walking all
//     channels of its tile and writing Out itself, in a fixed order.
#include "internal.h"
#include "common.h"

namespace cnnlib {

namespace {

constexpr int kTK = 32;          // output features per tile (one MFMA block of rows)
constexpr int kTP = 64;          // outputs per tile (two MFMA blocks of columns)
constexpr int kKS = kTK + 1;     // LDS vectors per (tap, channel group) of Ker (one pad)

__device__ __forceinline__ f32x16_t mfma_bf16(const u32x4_t& a, const u32x4_t& b,
                                              const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Halfword e of a run of 16-byte vectors (e a compile-time constant after
// unrolling).
template <int N>
__device__ __forceinline__ uint32_t half_at(const u32x4_t (&v)[N], int e) {
  const uint32_t d = v[e >> 3][(e >> 1) & 3];
  return (e & 1) ? (d >> 16) : (d & 0xffffu);
}

}  // namespace

// Waves of a workgroup with stages of TC channels: two per K group, TC / 16
// K groups (two for TC = 16, whose groups alternate taps).
template <int TC> struct CsliceShape {
  static constexpr int NK = TC >= 32 ? TC / 16 : 2;  // K groups
  static constexpr int NT = 128 * NK;                // threads
};

// MODE 0: fp32 partial tiles to slice z of Dst (the workspace); 1: fp32
// atomic adds into Dst (Out, zeroed); 2: TO values into Dst (Out), kc = 1.
template <int NR, int NS, int TC, int MODE, typename TO>
__global__ __launch_bounds__(CsliceShape<TC>::NT) void conv_cslice(const bf16_t* __restrict__ In,
                                                   const bf16_t* __restrict__ Ker,
                                                   void* __restrict__ Dst, ConvArgs a, int cs,
                                                   FastDiv dv_nxny) {
  constexpr int T = NR * NS;
  constexpr int kTC = TC;          // channels per stage (16, 32, 64 or 128)
  constexpr int kCG = kTC / 8;     // 8-channel groups per stage
  constexpr int kIPV = kCG + 1;    // 16-byte vectors per In position in LDS (one pad)
  constexpr int NK = CsliceShape<TC>::NK, NT = CsliceShape<TC>::NT;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* kl = reinterpret_cast<u32x4_t*>(smem);  // [T][kCG][kKS]
  u32x4_t* il = kl + T * kCG * kKS;                 // [position][kIPV]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, half = lane >> 5;
  const int pb = wave & 1, kh = wave >> 1;

  const int pt = (int)blockIdx.x / a.n_ktiles;
  const int kt = (int)blockIdx.x - pt * a.n_ktiles;
  const int p0 = pt * kTP, k0 = kt * kTK;
  const int plast = min(p0 + kTP, a.npix) - 1;

  // Input rows of the tile: flattened (b, x) rows G0 .. G0 + S - 1, all Ny
  // columns; its positions are consecutive in the flattened (b, x, y) index.
  const int b0 = p0 / a.hw, w0 = (p0 - b0 * a.hw) / a.Nh;
  const int b1 = plast / a.hw, w1 = (plast - b1 * a.hw) / a.Nh;
  const int G0 = b0 * a.Nx + a.sw * w0;
  const int SNt = (b1 * a.Nx + a.sw * w1 + NR - G0) * a.Ny;
  const int gpos0 = G0 * a.Ny;

  // This lane's output (column l32 of block pb): the LDS position of its
  // (0, 0) tap and the Out offset of its k = 0 plane.  Outputs past the end
  // read the last valid one's inputs and are not stored.
  const int p = p0 + pb * 32 + l32;
  const bool pval = p <= plast;
  int pix;
  int64_t obase;
  {
    const int pc = pval ? p : plast;
    const int b = pc / a.hw, q = pc - b * a.hw;
    const int w = q / a.Nh, h = q - w * a.Nh;
    pix = (b * a.Nx + a.sw * w - G0) * a.Ny + a.sh * h;
    obase = (int64_t)b * a.Nk * a.hw + q;
  }

  // Ker task of this thread (threads 0 .. 4*TC - 1): feature k0 + kk, its
  // channel group kcg of every stage.  Features past Nk stage nothing; their
  // LDS rows feed only accumulator rows that are not stored.
  const int kk = tid / kCG, kcg = tid % kCG;
  const bool ktask = tid < kTK * kCG && k0 + kk < a.Nk;
  const bf16_t* krow = Ker + ((int64_t)min(k0 + kk, a.Nk - 1) * a.Nc + 8 * kcg) * T;

  f32x16_t acc;
#pragma unroll
  for (int j = 0; j < 16; ++j) acc[j] = 0.f;

  const int c_begin = (int)blockIdx.y * cs;
  const int c_end = min(a.Nc, c_begin + cs);
  for (int c0 = c_begin; c0 < c_end; c0 += kTC) {
    const int ncg = min(kTC, c_end - c0) >> 3;  // even (Nc and cs are multiples of 16)
    static_assert(kTC == 16 || kTC == 32 || kTC == 64 || kTC == 128,
                  "stages of 16, 32, 64 or 128 channels");
    // Every global load of the stage, Ker first.
    u32x4_t kr[T];
    const bool kload = ktask && kcg < ncg;
    if (kload) {
      const u32x4_t* src = reinterpret_cast<const u32x4_t*>(krow + (int64_t)c0 * T);
#pragma unroll
      for (int t = 0; t < T; ++t) kr[t] = src[t];
    }
    // (position, group) tasks, positions fastest: idx = g * SNt + pos.
    const int ntask = SNt * kCG;
    for (int base = 0; base < ntask; base += 2 * NT) {
      uint32_t iv[2][8];
      int tpos[2], tg[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const int idx = base + m * NT + tid;
        tg[m] = idx / SNt;
        tpos[m] = idx - tg[m] * SNt;
        if (idx < ntask && tg[m] < ncg) {
          const int gp = gpos0 + tpos[m];
          const int b = fdiv(gp, dv_nxny);
          const bf16_t* src = In + (int64_t)b * a.in_img + (int64_t)(c0 + 8 * tg[m]) * a.nxny +
                              (gp - b * a.nxny);
#pragma unroll
          for (int i = 0; i < 8; ++i) iv[m][i] = src[(int64_t)i * a.nxny];
        }
      }
#pragma unroll
      for (int m = 0; m < 2; ++m)
        if (base + m * NT + tid < ntask && tg[m] < ncg) {
          u32x4_t v;
#pragma unroll
          for (int q = 0; q < 4; ++q) v[q] = iv[m][2 * q] | (iv[m][2 * q + 1] << 16);
          il[tpos[m] * kIPV + tg[m]] = v;
        }
    }
    if (kload) {
      // kr holds channels 8*kcg .. 8*kcg + 7 x taps 0 .. T-1 as (c, tap),
      // tap fastest; tap t's 8 channels are halfwords c*T + t.
#pragma unroll
      for (int t = 0; t < T; ++t) {
        u32x4_t v;
#pragma unroll
        for (int m = 0; m < 4; ++m)
          v[m] = half_at(kr, 2 * m * T + t) | (half_at(kr, (2 * m + 1) * T + t) << 16);
        kl[(t * kCG + kcg) * kKS + kk] = v;
      }
    }
    __syncthreads();

    // K-steps j = (tap t, 16-channel block cb), t-major over the stage's
    // nb blocks; K group kh takes the steps with j % NK == kh (with full
    // stages: cb == kh).
    const int nb = ncg >> 1;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int toff = (t / NS) * a.Ny + (t % NS);
#pragma unroll
      for (int cb = 0; cb < kCG / 2; ++cb) {
        const bool mine = cb < nb && (t * nb + cb) % NK == kh;
        if (mine) {
          const u32x4_t av = kl[(t * kCG + 2 * cb + half) * kKS + l32];
          const u32x4_t bv = il[(pix + toff) * kIPV + 2 * cb + half];
          acc = mfma_bf16(av, bv, acc);
        }
      }
    }
    __syncthreads();  // the stage's LDS fully read before the next overwrites it
  }

  // The K groups' sum (groups 1 .. NK-1 hand theirs to group 0, which adds
  // them in group order), then the slice's partial tile.  Register j of a
  // 32x32 accumulator holds row 8*(j/4) + 4*half + j%4 (the feature) of
  // column l32 (the output).  (Staging the tile's block in LDS to store
  // whole lines, written through or not, measured slower than these direct
  // stores, which overlap other workgroups' work.)
  float* red = reinterpret_cast<float*>(smem);  // [NK - 1][2][16][64]
  if (kh > 0) {
#pragma unroll
    for (int j = 0; j < 16; ++j) red[(((kh - 1) * 2 + pb) * 16 + j) * 64 + lane] = acc[j];
  }
  __syncthreads();
  if (kh == 0) {
    float* dst = static_cast<float*>(Dst) + (MODE == 0 ? (int64_t)blockIdx.y * a.out_total : 0);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int k = k0 + 8 * (j >> 2) + 4 * half + (j & 3);
      float v = acc[j];
#pragma unroll
      for (int g = 1; g < NK; ++g) v += red[(((g - 1) * 2 + pb) * 16 + j) * 64 + lane];
      if (pval && k < a.Nk) {
        if constexpr (MODE == 1)
          unsafeAtomicAdd(dst + obase + (int64_t)k * a.hw, v);  // hardware fp32 add
        else if constexpr (MODE == 2)
          static_cast<TO*>(Dst)[obase + (int64_t)k * a.hw] = from_f32<TO>(v);
        else
          dst[obase + (int64_t)k * a.hw] = v;
      }
    }
  }
}

// ---- instantiation table ------------------------------------------------
// X(id, dtype, Nr, Ns, tc, mode): mode 0 (partials and the ordered reduce)
// is the same kernel for both bf16 dtypes (the reduce writes the Out type);
// mode 1 (atomic sums) needs fp32 Out; mode 2 (direct, kc = 1) writes the
// dtype's Out type.
#define CNN_CSLICE_VARIANTS(X)           \
  X(2500, CNN_BF16, 3, 3, 32, 0)         \
  X(2501, CNN_BF16_OBF16, 3, 3, 32, 0)   \
  X(2502, CNN_BF16, 1, 1, 32, 0)         \
  X(2503, CNN_BF16_OBF16, 1, 1, 32, 0)   \
  X(2504, CNN_BF16, 3, 3, 16, 0)         \
  X(2505, CNN_BF16_OBF16, 3, 3, 16, 0)   \
  X(2506, CNN_BF16, 3, 3, 64, 0)         \
  X(2507, CNN_BF16_OBF16, 3, 3, 64, 0)   \
  X(2508, CNN_BF16, 3, 3, 32, 1)         \
  X(2509, CNN_BF16, 1, 1, 32, 1)         \
  X(2510, CNN_BF16, 3, 3, 128, 2)        \
  X(2511, CNN_BF16_OBF16, 3, 3, 128, 2)

static const VariantC kVariantsC[] = {
#define CNN_ROW(id, dt, nr, ns, tc, mode) {id, dt, kTK, kTP, tc, nr, ns, mode},
    CNN_CSLICE_VARIANTS(CNN_ROW)
#undef CNN_ROW
};

const VariantC* variants_cslice(int* count) {
  *count = (int)(sizeof(kVariantsC) / sizeof(kVariantsC[0]));
  return kVariantsC;
}

int64_t cslice_lds_bytes(const VariantC& v, int64_t slab_rows, int64_t Ny) {
  const int64_t cg = v.tc / 8;  // Ker [tap][cg][tk + 1] and In [position][cg + 1] vectors
  const int64_t b = 16 * ((int64_t)v.nr * v.ns * cg * kKS + slab_rows * Ny * (cg + 1));
  const int64_t red = 4 * ((v.tc >= 32 ? v.tc / 16 : 2) - 1) * 2 * 16 * 64;  // K groups' exchange
  return b > red ? b : red;
}

bool cslice_fits(const VariantC& v, const cnn_problem& p) {
  const int64_t Nx = p.sw * (p.Nw - 1) + p.Nr, Ny = p.sh * (p.Nh - 1) + p.Ns;
  return p.Nr == v.nr && p.Ns == v.ns && p.Nc % 16 == 0 &&
         p.Nb * Nx * Ny < (1LL << 31);  // flattened (b, x, y) positions divided by fdiv
}

__global__ __launch_bounds__(256) void cslice_zero(float* __restrict__ Out, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n; o += stride) Out[o] = 0.f;
}

// Out element type of an instantiation: fp32 except the direct form of
// the bf16-Out dtype.
template <int DT, int MODE> struct CsliceOut { typedef float T; };
template <> struct CsliceOut<CNN_BF16_OBF16, 2> { typedef bf16_t T; };

// dst: the partial slices (mode 0), or Out itself (mode 1: zeroed first;
// mode 2: written once).
template <int NR, int NS, int TC, int MODE, typename TO>
static hipError_t launch_one_c(const void* In, const void* Ker, void* dst, const ConvArgs& a,
                               int64_t lds, int kc, int cs, hipStream_t stream) {
  auto kern = conv_cslice<NR, NS, TC, MODE, TO>;
  if (lds > 64 * 1024) {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  if (MODE == 1) {
    int64_t blocks = (a.out_total + 255) / 256;
    if (blocks > 2048) blocks = 2048;  // grid-stride loop covers the rest
    hipLaunchKernelGGL(cslice_zero, dim3((unsigned)blocks), dim3(256), 0, stream, (float*)dst,
                       a.out_total);
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid, (unsigned)kc), dim3(CsliceShape<TC>::NT),
                     (unsigned)lds,
                     stream, (const bf16_t*)In, (const bf16_t*)Ker, dst, a, cs,
                     make_fastdiv((uint32_t)a.nxny));
  return hipGetLastError();
}

hipError_t launch_cslice(const VariantC& v, const void* In, const void* Ker, void* Out, void* ws,
                         const ConvArgs& a, int64_t lds_bytes, int kc, int dtype,
                         hipStream_t stream) {
  const int cs = (int)splitc_slice_channels(a.Nc, v.tc, kc);
  hipError_t e;
  switch (v.id) {
#define CNN_CASE(id, dt, nr, ns, tc, mode)                                              \
  case id:                                                                               \
    e = launch_one_c<nr, ns, tc, mode, CsliceOut<dt, mode>::T>(In, Ker, mode ? Out : ws, a, \
                                                               lds_bytes, kc, cs, stream); \
    break;
    CNN_CSLICE_VARIANTS(CNN_CASE)
#undef CNN_CASE
    default:
      return hipErrorInvalidValue;
  }
  if (e != hipSuccess || v.mode) return e;
  return launch_splitc_reduce((const float*)ws, Out, kc, a.out_total, dtype, stream);
}

}  // namespace cnnlib

// Implicit-GEMM convolution on bf16 MFMA, wide staging + software pipeline
// (gfx950).
//
// Tile schedule as conv_igemm (paper Sec. 2.1 / Listing 3 with W_c = N_c):
// a workgroup keeps a tk x tp Out tile in accumulators and walks the input
// features tc at a time.  Per c stage:
//
// * Ker: the repacked Ker block (pack_ker_bf16: the LDS image
//   [tap][c/8][k][8] of every (k tile, c stage)) is copied with 16-byte
//   global->LDS DMA.
// * In: a work item is eight consecutive slab positions of eight channels.
//   Each channel's eight positions are one 16-byte load at whatever 2-byte
//   alignment the row has (the memory system splits unaligned accesses), so
//   a wave-wide load moves 1 KiB.  The 8x8 block of bf16 is transposed in
//   registers (v_perm) into eight [8 channels] vectors and written to LDS.
//   Octets that cross an image's end are loaded element by element.
// * LDS layout of the transposed In: [c/8][slot][8] with
//   slot(pos) = pos ^ ((pos >> 3) & 7): an item's eight vectors then fall
//   in eight different 16-byte bank groups (no write conflicts), and a
//   half-wave's 32 consecutive positions still cover four whole 128-byte
//   lines (no read conflicts).
// * Both LDS tiles are double-buffered, one barrier per stage.  The global
//   loads of stage i+1 are issued a few at a time between the K-steps of
//   stage i, and the MFMA operands of K-step t+1 are read from LDS before
//   the MFMAs of step t issue (scheduling fences keep that order), so
//   neither memory latency nor a full memory queue stalls the MFMA stream.
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

#define LDS_PTR4(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc4(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

__device__ __forceinline__ int swz(int pos) { return pos ^ ((pos >> 3) & 7); }

template <typename TO, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int MAXI>
__global__ __launch_bounds__(256) void conv_igemm4(const bf16_t* __restrict__ In,
                                                   const u32x4_t* __restrict__ Kp,
                                                   TO* __restrict__ Out, ConvArgs a,
                                                   int blk_vecs) {
  constexpr int TK = 32 * WM * MB;
  constexpr int TP = 32 * WN * NB;
  constexpr int G = TC / 8;
  constexpr int KSTEPS = G / 2;
  static_assert(WM * WN == 4, "four waves");
  static_assert(TC % 16 == 0, "whole MFMA K-steps per stage");
  const int Nr = NR > 0 ? NR : a.Nr;
  const int Ns = NS > 0 ? NS : a.Ns;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int SN8 = (a.slab_max * a.Ny + 7) & ~7;       // swizzled slots per channel group
  u32x4_t* inbuf = reinterpret_cast<u32x4_t*>(smem);  // [2][G][SN8]
  u32x4_t* kerbuf = inbuf + 2 * G * SN8;              // [2][blk_vecs]

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
  const int b0 = p0 / a.hw, w0 = (p0 - b0 * a.hw) / a.Nh;
  const int b1 = plast / a.hw, w1 = (plast - b1 * a.hw) / a.Nh;
  const int G0 = b0 * a.Nx + a.sw * w0;
  const int S = b1 * a.Nx + a.sw * w1 + Nr - G0;
  const int SNt = S * a.Ny;
  const int NO = (SNt + 7) >> 3;  // octets per channel group

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
    pix[nb] = (b * a.Nx + a.sw * w - G0) * a.Ny + a.sh * h;
    obyte[nb] = (uint32_t)(((int64_t)(b - b0) * a.Nk * a.hw + q) * (int64_t)sizeof(TO));
  }

  // Items: (channel group g, octet m).  Offsets are bytes from the
  // descriptor base for channel 0; an octet that leaves its image plane is
  // marked for element-wise loading.
  const int64_t base_el = ((int64_t)b0 * a.in_img) & ~(int64_t)7;
  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc4(In + base_el, (a.in_total - base_el) * 2);
  const int gpos0 = G0 * a.Ny;
  uint32_t it_off[MAXI];
  int it_g[MAXI], it_m[MAXI], it_slot[MAXI];
  bool it_ok[MAXI], it_edge[MAXI];
#pragma unroll
  for (int j = 0; j < MAXI; ++j) {
    const int item = tid + 256 * j;
    it_ok[j] = item < G * NO;
    const int it = it_ok[j] ? item : 0;
    const int g = it / NO;
    const int m = it - g * NO;
    const int gp = gpos0 + 8 * m;
    const int b = gp / a.nxny;
    const int r0 = gp - b * a.nxny;
    it_g[j] = g;
    it_m[j] = m;
    it_slot[j] = g * SN8 + 8 * m;
    it_off[j] = (uint32_t)(((int64_t)b * a.in_img - base_el + r0) * 2);
    it_edge[j] = r0 + 8 > a.nxny;  // the octet leaves its image plane
  }

  uint32_t pre[MAXI][8][4];
  // One 16-byte In load: item j, channel i of stage base c0.
  auto load_one = [&](int c0, int j, int i) __attribute__((always_inline)) {
    const int c = c0 + 8 * it_g[j] + i;
    const bool cv = c < a.Nc;
    const uint32_t co = (uint32_t)((int64_t)(cv ? c : 0) * a.nxny * 2);
    u32x4_t v = __builtin_bit_cast(
        u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(in_rsrc, it_off[j] + co, 0, 0));
#pragma unroll
    for (int d = 0; d < 4; ++d) pre[j][i][d] = cv ? v[d] : 0u;
  };
  auto load_edges = [&](int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < MAXI; ++j) {
      if (it_edge[j] && it_ok[j]) {
        const int gp0 = gpos0 + 8 * it_m[j];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int c = c0 + 8 * it_g[j] + i;
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            uint32_t lohi[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
              const int pos = 8 * it_m[j] + 2 * d + e;
              const int gp = gp0 + 2 * d + e;
              const int b = gp / a.nxny;
              const int r0 = gp - b * a.nxny;
              const bool ok = c < a.Nc && pos < SNt;
              const uint32_t off =
                  (uint32_t)(((int64_t)b * a.in_img - base_el + (int64_t)(ok ? c : 0) * a.nxny + r0) * 2);
              const uint32_t val = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, off, 0, 0);
              lohi[e] = ok ? val : 0u;
            }
            pre[j][i][d] = lohi[0] | (lohi[1] << 16);
          }
        }
      }
    }
  };
  auto load_in = [&](int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < MAXI; ++j)
#pragma unroll
      for (int i = 0; i < 8; ++i) load_one(c0, j, i);
    load_edges(c0);
  };
  auto write_in = [&](u32x4_t* buf) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < MAXI; ++j) {
      if (it_ok[j]) {
        const uint32_t(&oct)[8][4] = pre[j];
        const int m7 = it_m[j] & 7;  // the swizzle of position 8m + p is p ^ (m mod 8)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          u32x4_t lo, hi;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            lo[k] = __builtin_amdgcn_perm(oct[2 * k + 1][q], oct[2 * k][q], 0x05040100u);
            hi[k] = __builtin_amdgcn_perm(oct[2 * k + 1][q], oct[2 * k][q], 0x07060302u);
          }
          buf[it_slot[j] + ((2 * q) ^ m7)] = lo;
          buf[it_slot[j] + ((2 * q + 1) ^ m7)] = hi;
        }
      }
    }
  };
  const int n_cc = (a.Nc + TC - 1) / TC;
  auto dma_ker = [&](int cc, u32x4_t* dst) __attribute__((always_inline)) {
    const u32x4_t* src = Kp + ((int64_t)kt * n_cc + cc) * blk_vecs;
    for (int v0 = wave * 64; v0 < blk_vecs; v0 += 256)
      __builtin_amdgcn_global_load_lds(src + v0 + lane, LDS_PTR4(void, dst + v0), 16, 0, 0);
  };
  // DMA instruction q (compile-time) of a Ker block of NDK*256 vectors.
  auto dma_one = [&](int cc, u32x4_t* dst, int q) __attribute__((always_inline)) {
    const u32x4_t* src = Kp + ((int64_t)kt * n_cc + cc) * blk_vecs;
    const int v0 = 256 * q + 64 * wave;
    __builtin_amdgcn_global_load_lds(src + v0 + lane, LDS_PTR4(void, dst + v0), 16, 0, 0);
  };
  // Workgroups start their walk over c at different stages (the tile index
  // mod the stage count), so concurrently running tiles read different Ker
  // blocks rather than all hitting the same L2 lines.

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
    const u32x4_t* ib = inbuf + buf * G * SN8;
    const u32x4_t* kb = kerbuf + buf * blk_vecs;
    u32x4_t* next_kb = kerbuf + (buf ^ 1) * blk_vecs;
    const bool more = cc + 1 < n_cc;
    const int next = more ? cc + 1 : 0;
    write_in(inbuf + buf * G * SN8);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    const u32x4_t* abase = kb + (wm * MB) * 32 + l32;
    auto load_ops = [&](int step, u32x4_t (&av)[MB], u32x4_t (&bv)[NB]) {
      const int tap = step / KSTEPS;
      const int j = step - tap * KSTEPS;
      const int rr = tap / Ns;
      const int ss = tap - rr * Ns;
      const int grp = 2 * j + half;
      const int toff = rr * a.Ny + ss;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) av[mb] = abase[(tap * G + grp) * TK + mb * 32];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) bv[nb] = ib[grp * SN8 + swz(pix[nb] + toff)];
    };
    auto mfmas = [&](const u32x4_t (&av)[MB], const u32x4_t (&bv)[NB]) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, av[mb]), __builtin_bit_cast(bf16x8_t, bv[nb]),
              acc[mb][nb], 0, 0, 0);
    };
    if constexpr (NR > 0 && NS > 0) {
      // The next stage's global loads (NDK Ker DMA instructions, then 8
      // In loads per item) are spread over the K-steps, after each step's
      // MFMAs: a load that must wait for queue space then stalls only
      // itself, never the MFMA stream.
      constexpr int STEPS = NR * NS * KSTEPS;
      constexpr int NDK = (NR * NS * G * TK + 255) / 256;
      constexpr int NLOADS = NDK + 8 * MAXI;
      constexpr int PER = (NLOADS + STEPS - 1) / STEPS;
      u32x4_t A[2][MB], B[2][NB];
      load_ops(0, A[0], B[0]);
#pragma unroll
      for (int st = 0; st < STEPS; ++st) {
        if (st + 1 < STEPS) load_ops(st + 1, A[(st + 1) & 1], B[(st + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        mfmas(A[st & 1], B[st & 1]);
        __builtin_amdgcn_sched_barrier(0);
        if (more) {
#pragma unroll
          for (int q = st * PER; q < (st + 1) * PER && q < NLOADS; ++q) {
            if (q < NDK) {
              dma_one(next, next_kb, q);
            } else {
              const int j = (q - NDK) / 8, i = (q - NDK) % 8;
              load_one(next * TC, j, i);
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if (more) load_edges(next * TC);
    } else {
      if (more) {
        dma_ker(next, next_kb);
        load_in(next * TC);
      }
      const int steps = Nr * Ns * KSTEPS;
      for (int st = 0; st < steps; ++st) {
        u32x4_t A[MB], B[NB];
        load_ops(st, A, B);
        mfmas(A, B);
      }
    }
  }

  const __amdgpu_buffer_rsrc_t out_rsrc =
      rsrc4(Out + (int64_t)b0 * a.Nk * a.hw,
            (a.out_total - (int64_t)b0 * a.Nk * a.hw) * (int64_t)sizeof(TO));
  const uint32_t half_off = (uint32_t)(4 * half * a.hw * (int)sizeof(TO));
  const bool k_full = k0 + TK <= a.Nk;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int kw = k0 + (wm * MB + mb) * 32 + 8 * (j >> 2) + (j & 3);
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
// (id, dtype, WM, WN, MB, NB, TC, NR, NS, MAXI): tk = 32*WM*MB,
// tp = 32*WN*NB; MAXI In items per thread (tc/8 * ceil(S*Ny/8) <= 256*MAXI).
#define CNN_IGEMM4_VARIANTS(X)                        \
  X(800, CNN_BF16, 1, 4, 2, 2, 16, 3, 3, 1)           \
  X(801, CNN_BF16, 1, 4, 2, 2, 32, 3, 3, 2)           \
  X(802, CNN_BF16, 2, 2, 2, 4, 16, 3, 3, 2)           \
  X(803, CNN_BF16, 2, 2, 2, 2, 16, 3, 3, 1)           \
  X(810, CNN_BF16, 4, 1, 2, 4, 32, 1, 1, 1)           \
  X(811, CNN_BF16, 2, 2, 2, 4, 32, 1, 1, 1)           \
  X(812, CNN_BF16, 4, 1, 2, 4, 64, 1, 1, 1)           \
  X(820, CNN_BF16, 1, 4, 2, 2, 16, 0, 0, 2)           \
  X(900, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 1)     \
  X(901, CNN_BF16_OBF16, 1, 4, 2, 2, 32, 3, 3, 2)     \
  X(902, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 2)     \
  X(903, CNN_BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 1)     \
  X(910, CNN_BF16_OBF16, 4, 1, 2, 4, 32, 1, 1, 1)     \
  X(911, CNN_BF16_OBF16, 2, 2, 2, 4, 32, 1, 1, 1)     \
  X(912, CNN_BF16_OBF16, 4, 1, 2, 4, 64, 1, 1, 1)     \
  X(920, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 0, 0, 2)

static const Variant4 kVariants4[] = {
#define CNN_ROW4(id, dt, wm, wn, mb, nb, tc, nr, ns, maxi) \
  {id, dt, 32 * (wm) * (mb), 32 * (wn) * (nb), tc, 16 * (mb) * (nb), nr, ns, maxi},
    CNN_IGEMM4_VARIANTS(CNN_ROW4)
#undef CNN_ROW4
};

const Variant4* variants4(int* count) {
  *count = (int)(sizeof(kVariants4) / sizeof(kVariants4[0]));
  return kVariants4;
}

int64_t igemm4_blk_vecs(const Variant4& v, int64_t RS) {
  return (RS * (v.tc / 8) * v.tk + 255) / 256 * 256;
}

int64_t igemm4_lds_bytes(const Variant4& v, int64_t slab_rows, int64_t Ny, int64_t RS) {
  const int64_t sn8 = (slab_rows * Ny + 7) / 8 * 8;
  return 2 * ((v.tc / 8) * sn8 + igemm4_blk_vecs(v, RS)) * 16;
}

bool igemm4_fits(const Variant4& v, const cnn_problem& p, int64_t slab_rows) {
  if (v.nr > 0 && (v.nr != p.Nr || v.ns != p.Ns)) return false;
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  return (v.tc / 8) * ((slab_rows * Ny + 7) / 8) <= 256LL * v.maxi;
}

int64_t igemm4_ws_bytes(const Variant4& v, const cnn_problem& p) {
  const int64_t n_kt = (p.Nk + v.tk - 1) / v.tk, n_cc = (p.Nc + v.tc - 1) / v.tc;
  return n_kt * n_cc * igemm4_blk_vecs(v, p.Nr * p.Ns) * 16;
}

template <int DT, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int MAXI>
static hipError_t launch_one4(const void* In, const void* Ker, void* Out, void* ws,
                              const ConvArgs& a, int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  constexpr int TK = 32 * WM * MB;
  const int64_t RS = (int64_t)a.Nr * a.Ns;
  const int64_t blk = (RS * (TC / 8) * TK + 255) / 256 * 256;
  const int64_t n_cc = (a.Nc + TC - 1) / TC;
  const int64_t total = (int64_t)a.n_ktiles * n_cc * blk;
  int64_t pgrid = (total + 255) / 256;
  if (pgrid > 4096) pgrid = 4096;
  hipLaunchKernelGGL(pack_ker_bf16, dim3((unsigned)pgrid), dim3(256), 0, stream,
                     (const bf16_t*)Ker, (u32x4_t*)ws, a, TK, TC, (int)blk, total);
  auto kern = conv_igemm4<TO, WM, WN, MB, NB, TC, NR, NS, MAXI>;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(256), (unsigned)lds, stream,
                     (const bf16_t*)In, (const u32x4_t*)ws, (TO*)Out, a, (int)blk);
  return hipGetLastError();
}

hipError_t launch_igemm4(const Variant4& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASE4(id, dt, wm, wn, mb, nb, tc, nr, ns, maxi) \
  case id:                                                  \
    return launch_one4<dt, wm, wn, mb, nb, tc, nr, ns, maxi>(In, Ker, Out, ws, a, lds_bytes, stream);
    CNN_IGEMM4_VARIANTS(CNN_CASE4)
#undef CNN_CASE4
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

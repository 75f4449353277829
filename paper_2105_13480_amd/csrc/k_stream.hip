// Persistent, streaming implicit-GEMM convolution (bf16 MFMA, gfx950).
//
// The tile schedule of Sec. 2.1 / Listing 3 (W_c = N_c: a workgroup keeps a
// tk x tp Out tile in accumulators and walks the input features tc at a
// time), run by persistent workgroups: the grid fills the machine's
// workgroup slots once and each workgroup walks a contiguous range of
// tiles (the P processors of Eq. (2), each with its share of the tiles).
// The (tile, c stage) sequence of a workgroup is one software pipeline:
//
// * the loads of stage i+1 -- of the same tile, or the first stage of the
//   next tile -- are issued before the MFMAs of stage i;
// * a tile's Out stores are issued and left to drain while the next tile's
//   stages run: barriers wait for LDS only (s_waitcnt lgkmcnt(0)), never for
//   outstanding stores, and every In load is consumed by a register read
//   that the compiler guards with an exact vmcnt wait;
// * Ker: raw rows (each feature's tc channels x all taps, contiguous in
//   memory) copied by 16-byte buffer->LDS DMA, one padding chunk per row so
//   the A-operand reads of 8 consecutive features hit distinct banks.  When
//   the whole Ker fits (one k tile), it is copied once per workgroup and
//   stays resident (KRES); otherwise each stage's block is streamed;
// * In: the tile's halo'd slab (whole input rows) staged through registers
//   as dword pairs of one channel, transposed with v_perm into 8-channel
//   16-byte vectors [c/8][position][8] (the MFMA B operand).
// A operands are built from the raw Ker rows with v_perm per tap.
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

namespace {

#define LDS_PTR_S(T, p) ((__attribute__((address_space(3))) T*)(p))

enum { kPairAligned = 0, kPairFunnel = 1, kPairElement = 2 };

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_t(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

__device__ __forceinline__ void dma16_t(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR_S(void, lds), 16, voff, 0, 0, 0);
#endif
}

// LDS barrier: wait for this wave's LDS operations, then s_barrier.  The
// memory clobber keeps the compiler from moving memory accesses across it;
// outstanding global loads and stores are not waited for.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace

// Per-tile geometry (one pair slot per thread).
struct StreamGeo {
  int p0, plast, b0, G0, kt;
  int path;
  int pdst;         // LDS position of the thread's pair (a padding slot if none)
  uint32_t voff, voff2;
  int pix[4];
  uint32_t obyte[4];
};

template <typename TO, int WM, int WN, int MB, int NB, int TC, int NR, int NS, bool KRES>
__global__ __launch_bounds__(64 * WM * WN) void conv_stream(const bf16_t* __restrict__ In,
                                                            const bf16_t* __restrict__ Ker,
                                                            TO* __restrict__ Out, ConvArgs a) {
  constexpr int NT = 64 * WM * WN;
  constexpr int TK = 32 * WM * MB;
  constexpr int G = TC / 8;
  constexpr int KSTEPS = G / 2;
  constexpr int RS = NR * NS;
  constexpr int RC = (RS * TC / 8) | 1;              // Ker row chunks (odd)
  constexpr int KVECS = (TK * RC + 63) / 64 * 64;    // Ker vectors per stage
  static_assert(TC % 16 == 0 && NB <= 4, "whole K-steps; at most 4 blocks per wave");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int SN = ((a.slab_max * a.Ny + 1) & ~1) + 2;  // + one padding pair per group
  u32x4_t* inbuf = reinterpret_cast<u32x4_t*>(smem);  // [2][G][SN]
  u32x4_t* kbuf = inbuf + 2 * G * SN;                  // [KRES ? n_cc : 2][KVECS]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, half = lane >> 5;
  const int n_cc = (a.Nc + TC - 1) / TC;

  // This workgroup's tiles: a contiguous range, XCD-aware (neighbouring
  // tiles share halo rows and Ker in the same L2).
  const int n_tiles = a.n_ptiles * a.n_ktiles;
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int t_begin = (int)((int64_t)L * n_tiles / gridDim.x);
  const int t_end = (int)((int64_t)(L + 1) * n_tiles / gridDim.x);
  if (t_begin >= t_end) return;

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_t(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t ker_rsrc = rsrc_t(Ker, (int64_t)a.Nk * a.Nc * RS * 2);

  auto geometry = [&](int t, StreamGeo& g) __attribute__((always_inline)) {
    const int pt = t / a.n_ktiles;
    g.kt = t - pt * a.n_ktiles;
    g.p0 = pt * a.tp;
    g.plast = min(g.p0 + a.tp, a.npix) - 1;
    g.b0 = g.p0 / a.hw;
    const int w0 = (g.p0 - g.b0 * a.hw) / a.Nh;
    const int b1 = g.plast / a.hw, w1 = (g.plast - b1 * a.hw) / a.Nh;
    g.G0 = g.b0 * a.Nx + a.sw * w0;
    const int S = b1 * a.Nx + a.sw * w1 + NR - g.G0;
    const int SNt = S * a.Ny;
    const int npairs = (SNt + 1) >> 1;
    // pair loads: dword-aligned in every channel plane, or a funnel shift,
    // or two 16-bit loads where a pair straddles an image
    const int64_t img0 = (int64_t)g.b0 * a.in_img;
    g.path = ((a.Ny & 1) == 0 && (img0 & 1) == 0 && (a.nxny & 1) == 0) ? kPairAligned
                                                                        : kPairFunnel;
    if (g.path == kPairFunnel) {
      for (int b = g.b0 + 1; b <= b1; ++b)
        if ((((int64_t)b * a.Nx - g.G0) * a.Ny) & 1) g.path = kPairElement;
    }
    const bool valid = tid < npairs;
    const int pos = 2 * (valid ? tid : 0);
    g.pdst = valid ? pos : SN - 2;
    const int gp = g.G0 * a.Ny + pos;
    const int b = gp / a.nxny;
    const int r0 = gp - b * a.nxny;
    g.voff = (uint32_t)(((int64_t)b * a.in_img + r0) * 2);
    const int b2 = (r0 + 1 == a.nxny) ? b + 1 : b;
    const int r2 = (r0 + 1 == a.nxny) ? 0 : r0 + 1;
    g.voff2 = (uint32_t)(((int64_t)b2 * a.in_img + r2) * 2);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int p = g.p0 + (wn * NB + nb) * 32 + l32;
      const int pc = p <= g.plast ? p : g.plast;
      const int bb = pc / a.hw;
      const int q = pc - bb * a.hw;
      const int w = q / a.Nh;
      const int h = q - w * a.Nh;
      g.pix[nb] = (bb * a.Nx + a.sw * w - g.G0) * a.Ny + a.sh * h;
      g.obyte[nb] = (uint32_t)(((int64_t)bb * a.Nk * a.hw + q) * (int64_t)sizeof(TO));
    }
  };

  // In: channel q of the stage at c0 for the thread's pair.
  uint32_t pre[G][8];
  auto load_in = [&](const StreamGeo& g, int c0) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 8 * G; ++q) {
      const int c = c0 + q;
      if (c < a.Nc) {
        const uint32_t so = (uint32_t)((int64_t)c * a.nxny * 2);
        uint32_t v;
        if (g.path == kPairAligned) {
          v = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, g.voff, so, 0);
        } else if (g.path == kPairFunnel) {
          const uint32_t t = g.voff + (so & 2u);
          const uint32_t lo_off = t & ~3u;
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, lo_off, so & ~3u, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b32(in_rsrc, lo_off + 4, so & ~3u, 0);
          v = __builtin_amdgcn_alignbit(hi, lo, (t & 2u) * 8u);
        } else {
          const uint32_t lo = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, g.voff, so, 0);
          const uint32_t hi = __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, g.voff2, so, 0);
          v = lo | (hi << 16);
        }
        pre[q >> 3][q & 7] = v;
      } else {
        pre[q >> 3][q & 7] = 0u;
      }
    }
  };
  // Every thread writes (threads without a pair write the padding slot), so
  // each wave's vmcnt wait covers all of its loads and DMA of the stage.
  auto write_in = [&](u32x4_t* buf, const StreamGeo& g) __attribute__((always_inline)) {
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      u32x4_t lo, hi;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        lo[i] = __builtin_amdgcn_perm(pre[gg][2 * i + 1], pre[gg][2 * i], 0x05040100u);
        hi[i] = __builtin_amdgcn_perm(pre[gg][2 * i + 1], pre[gg][2 * i], 0x07060302u);
      }
      buf[gg * SN + g.pdst] = lo;
      buf[gg * SN + g.pdst + 1] = hi;
    }
  };
  // Ker stage cc of k tile kt into dst: slot v is feature kt*TK + v / RC,
  // chunk v % RC of its run (chunks past RS*TC/8 are padding).
  auto dma_ker = [&](int kt, int cc, u32x4_t* dst) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < (KVECS + NT - 1) / NT; ++j) {
      if (NT * j + wave * 64 < KVECS) {
        const int v = tid + NT * j;
        const int kk = v / RC;
        const int part = v - kk * RC;
        const uint32_t off = (uint32_t)((((int64_t)(kt * TK + kk) * a.Nc + cc * TC) * RS) * 2 +
                                        16 * part);
        dma16_t(ker_rsrc, dst + NT * j + wave * 64, off);
      }
    }
  };

  f32x16_t acc[MB][NB];
  StreamGeo cur, nxt;
  geometry(t_begin, cur);
  if constexpr (KRES) {
    for (int cc = 0; cc < n_cc; ++cc) dma_ker(0, cc, kbuf + cc * KVECS);
  } else {
    dma_ker(cur.kt, 0, kbuf);
  }
  load_in(cur, 0);
  int buf = 0;

  for (int t = t_begin; t < t_end; ++t) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;
    const int k0 = cur.kt * TK;

    for (int cc = 0; cc < n_cc; ++cc) {
      u32x4_t* ib = inbuf + buf * G * SN;
      const u32x4_t* kb = KRES ? kbuf + cc * KVECS : kbuf + buf * KVECS;
      write_in(ib, cur);
      lds_barrier();
      // next stage: this tile's stage cc+1, or the next tile's first stage
      if (cc + 1 < n_cc) {
        if constexpr (!KRES) dma_ker(cur.kt, cc + 1, kbuf + (buf ^ 1) * KVECS);
        load_in(cur, (cc + 1) * TC);
      } else if (t + 1 < t_end) {
        geometry(t + 1, nxt);
        if constexpr (!KRES) dma_ker(nxt.kt, 0, kbuf + (buf ^ 1) * KVECS);
        load_in(nxt, 0);
      }
      // MFMAs of stage cc
      constexpr int RSD = RS * 4;
#pragma unroll
      for (int j = 0; j < KSTEPS; ++j) {
        const int grp = 2 * j + half;
        // whole group in range (Nc % 8 == 0); masked, not branched on
        const uint32_t gmask = cc * TC + 8 * grp < a.Nc ? ~0u : 0u;
        uint32_t raw[MB][RSD];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const u32x4_t* src = kb + ((wm * MB + mb) * 32 + l32) * RC + grp * RS;
#pragma unroll
          for (int q = 0; q < RS; ++q) {
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
                const int e0 = (2 * i) * RS + tap, e1 = e0 + RS;
                const uint32_t sel = ((e0 & 1) ? 0x0302u : 0x0100u) |
                                     ((e1 & 1) ? 0x07060000u : 0x05040000u);
                av[mb][i] = __builtin_amdgcn_perm(raw[mb][e1 >> 1], raw[mb][e0 >> 1], sel);
              }
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) bv[nb] = ib[grp * SN + cur.pix[nb] + toff];
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
      buf ^= 1;
    }

    // Epilogue: register j of a 32x32 accumulator holds feature
    // 8*(j/4) + 4*half + j%4 of output l32; stores are left to drain.
    const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_t(Out, a.out_total * (int64_t)sizeof(TO));
    const uint32_t half_off = (uint32_t)(4 * half * a.hw * (int)sizeof(TO));
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int kw = k0 + (wm * MB + mb) * 32 + 8 * (j >> 2) + (j & 3);
        // rows past Nk: an offset beyond the descriptor's range drops the store
        const bool kv = kw + 4 * half < a.Nk;
        const uint32_t so = (uint32_t)kw * (uint32_t)a.hw * (uint32_t)sizeof(TO);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const uint32_t vo = kv ? cur.obyte[nb] + half_off + so : 0x80000000u;
          if constexpr (sizeof(TO) == 4) {
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[mb][nb][j]), out_rsrc, vo,
                                                  0, 0);
          } else {
            __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc[mb][nb][j]), out_rsrc, vo,
                                                  0, 0);
          }
        }
      }
    }
    cur = nxt;
  }
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, WM, WN, MB, NB, TC, NR, NS, KRES): tk = 32*WM*MB, largest
// tile tp = 32*WN*NB, 64*WM*WN threads; KRES keeps all of Ker in LDS
// (needs Nk <= tk).
#define CNN_STREAM_VARIANTS(X)                            \
  X(1300, CNN_BF16, 1, 8, 2, 1, 16, 3, 3, 1)              \
  X(1310, CNN_BF16, 2, 4, 2, 1, 16, 3, 3, 0)              \
  X(1400, CNN_BF16_OBF16, 1, 8, 2, 1, 16, 3, 3, 1)        \
  X(1410, CNN_BF16_OBF16, 2, 4, 2, 1, 16, 3, 3, 0)

static const VariantT kVariantsT[] = {
#define CNN_ROWT(id, dt, wm, wn, mb, nb, tc, nr, ns, kres) \
  {id, dt, 32 * (wm) * (mb), 32 * (wn) * (nb), tc, 16 * (mb) * (nb), nr, ns, 64 * (wm) * (wn), kres},
    CNN_STREAM_VARIANTS(CNN_ROWT)
#undef CNN_ROWT
};

const VariantT* variants_stream(int* count) {
  *count = (int)(sizeof(kVariantsT) / sizeof(kVariantsT[0]));
  return kVariantsT;
}

int64_t stream_lds_bytes(const VariantT& v, const cnn_problem& p, int64_t slab_rows) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t sn = (slab_rows * Ny + 1) / 2 * 2 + 2;
  const int64_t rc = (v.nr * v.ns * v.tc / 8) | 1;
  const int64_t kvecs = (v.tk * rc + 63) / 64 * 64;
  const int64_t n_cc = (p.Nc + v.tc - 1) / v.tc;
  return (2 * (v.tc / 8) * sn + (v.kres ? n_cc : 2) * kvecs) * 16;
}

template <int DT, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int KRES>
static hipError_t launch_t(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                           int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  auto kern = conv_stream<TO, WM, WN, MB, NB, TC, NR, NS, (KRES != 0)>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(64 * WM * WN), (unsigned)lds, stream,
                     (const bf16_t*)In, (const bf16_t*)Ker, (TO*)Out, a);
  return hipGetLastError();
}

hipError_t launch_stream(const VariantT& v, const void* In, const void* Ker, void* Out,
                         const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASET(id, dt, wm, wn, mb, nb, tc, nr, ns, kres) \
  case id:                                                  \
    return launch_t<dt, wm, wn, mb, nb, tc, nr, ns, kres>(In, Ker, Out, a, lds_bytes, stream);
    CNN_STREAM_VARIANTS(CNN_CASET)
#undef CNN_CASET
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

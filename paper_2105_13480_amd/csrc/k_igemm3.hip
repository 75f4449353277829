// Implicit-GEMM convolution on bf16 MFMA with DMA staging (gfx950).
//
// Tile schedule as conv_igemm (paper Sec. 2.1 / Listing 3 with W_c = N_c):
// a workgroup keeps a tk x tp Out tile in accumulators and walks the input
// features tc at a time.  Data movement per c stage:
//
// * Ker: the call's repacked Ker (pack_ker_bf16, the exact LDS image
//   [tap][c/8][k][8] of every (k tile, c stage) block) is copied with
//   16-byte buffer->LDS DMA (buffer_load_dwordx4 ... lds).
// * In: every input row of the halo'd slab is copied in its natural layout
//   with the same 16-byte DMA: the 16-byte-aligned blocks that cover the
//   row, so any row alignment and image boundary is handled by the copy
//   itself; reads past the tensor end are range-checked to zero.  One LDS
//   pass then transposes the copy into [c/8][position][8] (eight channels
//   per 16-byte vector, the MFMA B operand).
// * The DMA of stage i+2 is in flight while stage i is transposed and
//   multiplied: a ring of NBUF copy buffers, and per-thread DMA counts fixed
//   at compile time so `s_waitcnt vmcnt` can wait for exactly one stage.
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

#define LDS_PTR3(T, p) ((__attribute__((address_space(3))) T*)(p))

// s_waitcnt immediate that waits until at most n vector-memory operations
// are outstanding and does not wait on LDS/scalar or export counters
// (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8], vmcnt[5:4] at 15:14).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 16-byte buffer -> LDS copy: lane i's 16 bytes at voff + soff land at
// lds + 16 i (lds is wave-uniform).  Out-of-range reads give zeros.  The
// builtin exists only for the device target; clang's host pass (which never
// runs device code) would otherwise reject the enclosing kernel template.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff,
                                      uint32_t soff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR3(void, lds), 16, voff, soff, 0, 0);
#endif
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc3(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

template <typename TO, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int NBUF,
          int NDI, int NDK, int MPOS>
__global__ __launch_bounds__(256) void conv_igemm3(const bf16_t* __restrict__ In,
                                                   const u32x4_t* __restrict__ Kp,
                                                   TO* __restrict__ Out, ConvArgs a, int nbr) {
  constexpr int TK = 32 * WM * MB;
  constexpr int TP = 32 * WN * NB;
  constexpr int G = TC / 8;
  constexpr int KSTEPS = G / 2;
  constexpr int BLK = 256 * NDK;   // Ker vectors per stage
  constexpr int NAT = 256 * NDI;   // natural-copy blocks per stage
  static_assert(WM * WN == 4, "four waves");
  static_assert(TC % 16 == 0, "whole MFMA K-steps per stage");
  static_assert(NBUF >= 2 && NBUF <= 3, "ring of two or three stages");
  const int Nr = NR > 0 ? NR : a.Nr;
  const int Ns = NS > 0 ? NS : a.Ns;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int SN = a.slab_max * a.Ny;                       // positions per channel group
  u32x4_t* tbuf = reinterpret_cast<u32x4_t*>(smem);       // [G][SN] transposed In
  u32x4_t* natbuf = tbuf + G * SN;                        // [NBUF][NAT] natural In copies
  u32x4_t* kerbuf = natbuf + NBUF * NAT;                  // [NBUF][BLK] Ker blocks

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
  const int rb = S * nbr;         // natural-copy blocks per channel (this tile)
  const int nat_n = TC * rb;      // natural-copy blocks per stage (this tile)

  // Output side (as conv_igemm2): clamped lanes recompute and rewrite the
  // tile's last output, so stores need no pixel mask.
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

  // Natural-copy DMA: block f = tid + 256 j of a stage is (channel f / rb,
  // slab row (f % rb) / nbr, block f % nbr); its source offset (bytes, from
  // the tile's first image, channel c0 excluded) is fixed for the tile.
  // Descriptor base: the tile's first image, rounded down to 8 elements so
  // that 16-byte blocks relative to it are 16-byte aligned in memory.
  const int64_t base_el = ((int64_t)b0 * a.in_img) & ~(int64_t)7;
  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc3(In + base_el, (a.in_total - base_el) * 2);
  uint32_t dma_off[NDI];
#pragma unroll
  for (int j = 0; j < NDI; ++j) {
    int f = tid + 256 * j;
    f = f < nat_n ? f : nat_n - 1;  // surplus lanes repeat the last block
    const int cl = f / rb;
    const int rem = f - cl * rb;
    const int row = rem / nbr;
    const int blk = rem - row * nbr;
    const int gr = G0 + row;
    const int b = gr / a.Nx;
    const int x = gr - b * a.Nx;
    const int64_t row_el = (int64_t)b * a.in_img - base_el + (int64_t)cl * a.nxny + (int64_t)x * a.Ny;
    dma_off[j] = (uint32_t)(((row_el & ~(int64_t)7) + 8 * blk) * 2);
  }
  // Transpose side: position pos = tid + 256 m of the slab reads natural
  // element (row * nbr * 8 + y + shift) of its channel's copy, where
  // shift = (row start element) mod 8 = (rs + c * Nx * Ny) mod 8.
  int t_base[MPOS], t_rs[MPOS];
  bool t_ok[MPOS];
#pragma unroll
  for (int m = 0; m < MPOS; ++m) {
    const int pos = tid + 256 * m;
    t_ok[m] = pos < SNt;
    const int pp = t_ok[m] ? pos : 0;
    const int row = pp / a.Ny;
    const int y = pp - row * a.Ny;
    const int gr = G0 + row;
    const int b = gr / a.Nx;
    const int x = gr - b * a.Nx;
    t_base[m] = row * nbr * 8 + y;
    t_rs[m] = (int)(((int64_t)b * a.in_img - base_el + (int64_t)x * a.Ny) & 7);
  }

  const int n_cc = (a.Nc + TC - 1) / TC;
  const __amdgpu_buffer_rsrc_t ker_rsrc =
      rsrc3(Kp, (int64_t)a.n_ktiles * n_cc * BLK * 16);
  auto issue_dma = [&](int cc, int slot) {
    const uint32_t so_in = (uint32_t)((int64_t)cc * TC * a.nxny * 2);
    u32x4_t* nat = natbuf + slot * NAT;
#pragma unroll
    for (int j = 0; j < NDI; ++j)
      dma16(in_rsrc, nat + 256 * j + 64 * wave, dma_off[j], so_in);
    const uint32_t so_k = (uint32_t)(((int64_t)kt * n_cc + cc) * BLK * 16);
    u32x4_t* kb = kerbuf + slot * BLK;
#pragma unroll
    for (int j = 0; j < NDK; ++j)
      dma16(ker_rsrc, kb + 256 * j + 64 * wave, (uint32_t)(256 * j + tid) * 16u, so_k);
  };
  // All of a thread's reads first (unconditional, straight-line), then its
  // writes: reads and writes share the LDS array, so interleaving them -- or
  // branching per element -- would serialize every read.  Channels past Nc
  // are read anyway (in-range LDS) and masked to zero.
  auto transpose = [&](int cc, int slot) __attribute__((always_inline)) {
    const uint16_t* nat = reinterpret_cast<const uint16_t*>(natbuf + slot * NAT);
    const int c0 = cc * TC;
    uint32_t e[G][MPOS][8];
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int cl = 8 * g + i;  // channel within the stage (the DMA offsets' channel)
        const uint32_t keep = c0 + cl < a.Nc ? 0xffffu : 0u;
        const uint32_t cm = (uint32_t)(((int64_t)cl * a.nxny) & 7);
#pragma unroll
        for (int m = 0; m < MPOS; ++m) {
          const int idx = cl * rb * 8 + t_base[m] + (int)((t_rs[m] + cm) & 7u);
          e[g][m][i] = (uint32_t)nat[idx] & keep;
        }
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int m = 0; m < MPOS; ++m) {
        if (t_ok[m]) {
          u32x4_t v;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = e[g][m][2 * i] | (e[g][m][2 * i + 1] << 16);
          tbuf[g * SN + tid + 256 * m] = v;
        }
      }
    }
  };

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;

  issue_dma(0, 0);
  if (NBUF == 3 && n_cc > 1) issue_dma(1, 1);
  for (int cc = 0; cc < n_cc; ++cc) {
    const int slot = cc % NBUF;
    if (NBUF == 3 && cc + 1 < n_cc)
      wait_vmcnt<NDI + NDK>();  // stage cc landed; stage cc+1 may still be in flight
    else
      wait_vmcnt<0>();
    __syncthreads();  // stage cc visible; every wave finished compute(cc-1)
    if (NBUF == 3) {
      if (cc + 2 < n_cc) issue_dma(cc + 2, (cc + 2) % 3);
    } else {
      if (cc + 1 < n_cc) issue_dma(cc + 1, (cc + 1) & 1);
    }
    transpose(cc, slot);
    __syncthreads();  // transposed In complete
    const u32x4_t* kb = kerbuf + slot * BLK;
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
        for (int nb = 0; nb < NB; ++nb) bv[nb] = tbuf[grp * SN + pix[nb] + toff];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, av[mb]), __builtin_bit_cast(bf16x8_t, bv[nb]),
                acc[mb][nb], 0, 0, 0);
      }
    };
    if constexpr (NR > 0 && NS > 0) {
#pragma unroll
      for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int s = 0; s < NS; ++s) tap_step(r, s);
    } else {
      for (int r = 0; r < Nr; ++r)
        for (int s = 0; s < Ns; ++s) tap_step(r, s);
    }
  }

  const __amdgpu_buffer_rsrc_t out_rsrc =
      rsrc3(Out + (int64_t)b0 * a.Nk * a.hw,
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
// (id, dtype, WM, WN, MB, NB, TC, NR, NS, NBUF, NDI, NDK, MPOS):
// tk = 32*WM*MB, tp = 32*WN*NB; NDI/NDK DMA instructions per thread per
// stage (In natural copy: tc*S*nbr <= 256*NDI blocks; Ker: exactly
// 256*NDK vectors); MPOS transposed positions per thread (S*Ny <= 256*MPOS).
#define CNN_IGEMM3_VARIANTS(X)                                  \
  X(600, CNN_BF16, 1, 4, 2, 2, 16, 3, 3, 3, 6, 5, 3)            \
  X(602, CNN_BF16, 2, 2, 2, 2, 16, 3, 3, 2, 7, 9, 3)            \
  X(603, CNN_BF16, 2, 2, 2, 4, 16, 3, 3, 2, 6, 9, 3)            \
  X(610, CNN_BF16, 1, 4, 2, 2, 16, 0, 0, 3, 4, 1, 2)            \
  X(611, CNN_BF16, 2, 2, 2, 4, 16, 0, 0, 3, 4, 2, 2)            \
  X(612, CNN_BF16, 4, 1, 2, 4, 16, 0, 0, 3, 4, 2, 2)            \
  X(613, CNN_BF16, 1, 4, 2, 1, 16, 0, 0, 2, 6, 13, 4)           \
  X(700, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 3, 3, 3, 6, 5, 3)      \
  X(702, CNN_BF16_OBF16, 2, 2, 2, 2, 16, 3, 3, 2, 7, 9, 3)      \
  X(703, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 3, 3, 2, 6, 9, 3)      \
  X(710, CNN_BF16_OBF16, 1, 4, 2, 2, 16, 0, 0, 3, 4, 1, 2)      \
  X(711, CNN_BF16_OBF16, 2, 2, 2, 4, 16, 0, 0, 3, 4, 2, 2)      \
  X(712, CNN_BF16_OBF16, 4, 1, 2, 4, 16, 0, 0, 3, 4, 2, 2)      \
  X(713, CNN_BF16_OBF16, 1, 4, 2, 1, 16, 0, 0, 2, 6, 13, 4)

static const Variant3 kVariants3[] = {
#define CNN_ROW3(id, dt, wm, wn, mb, nb, tc, nr, ns, nbuf, ndi, ndk, mpos) \
  {id, dt, 32 * (wm) * (mb), 32 * (wn) * (nb), tc, 16 * (mb) * (nb), nr, ns, nbuf, ndi, ndk, mpos},
    CNN_IGEMM3_VARIANTS(CNN_ROW3)
#undef CNN_ROW3
};

const Variant3* variants3(int* count) {
  *count = (int)(sizeof(kVariants3) / sizeof(kVariants3[0]));
  return kVariants3;
}

int64_t igemm3_blocks_per_row(int64_t Ny) { return (Ny + 7 + 7) / 8; }

int64_t igemm3_lds_bytes(const Variant3& v, int64_t slab_rows, int64_t Ny) {
  return ((v.tc / 8) * slab_rows * Ny + (int64_t)v.nbuf * 256 * (v.ndi + v.ndk)) * 16;
}

bool igemm3_fits(const Variant3& v, const cnn_problem& p, int64_t slab_rows) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t RS = p.Nr * p.Ns;
  if (v.nr > 0 && (v.nr != p.Nr || v.ns != p.Ns)) return false;
  if ((int64_t)v.tc * slab_rows * igemm3_blocks_per_row(Ny) > 256LL * v.ndi) return false;
  if (RS * (v.tc / 8) * v.tk > 256LL * v.ndk) return false;
  if (slab_rows * Ny > 256LL * v.mpos) return false;
  return true;
}

int64_t igemm3_ws_bytes(const Variant3& v, const cnn_problem& p) {
  const int64_t n_kt = (p.Nk + v.tk - 1) / v.tk, n_cc = (p.Nc + v.tc - 1) / v.tc;
  return n_kt * n_cc * 256LL * v.ndk * 16;
}

template <int DT, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int NBUF, int NDI,
          int NDK, int MPOS>
static hipError_t launch_one3(const void* In, const void* Ker, void* Out, void* ws,
                              const ConvArgs& a, int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  constexpr int TK = 32 * WM * MB;
  const int64_t n_cc = (a.Nc + TC - 1) / TC;
  const int64_t blk = 256LL * NDK;
  const int64_t total = (int64_t)a.n_ktiles * n_cc * blk;
  int64_t pgrid = (total + 255) / 256;
  if (pgrid > 4096) pgrid = 4096;
  hipLaunchKernelGGL(pack_ker_bf16, dim3((unsigned)pgrid), dim3(256), 0, stream,
                     (const bf16_t*)Ker, (u32x4_t*)ws, a, TK, TC, (int)blk, total);
  auto kern = conv_igemm3<TO, WM, WN, MB, NB, TC, NR, NS, NBUF, NDI, NDK, MPOS>;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(256), (unsigned)lds, stream,
                     (const bf16_t*)In, (const u32x4_t*)ws, (TO*)Out, a,
                     (int)igemm3_blocks_per_row(a.Ny));
  return hipGetLastError();
}

hipError_t launch_igemm3(const Variant3& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASE3(id, dt, wm, wn, mb, nb, tc, nr, ns, nbuf, ndi, ndk, mpos)                 \
  case id:                                                                                  \
    return launch_one3<dt, wm, wn, mb, nb, tc, nr, ns, nbuf, ndi, ndk, mpos>(In, Ker, Out, ws, \
                                                                            a, lds_bytes, stream);
    CNN_IGEMM3_VARIANTS(CNN_CASE3)
#undef CNN_CASE3
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

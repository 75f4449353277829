// Persistent, streaming implicit-GEMM convolution (bf16 MFMA, gfx950).
//
// The tile schedule of Sec. 2.1 / Listing 3 (W_c = N_c: a workgroup keeps a
// tk x tp Out tile in accumulators and walks the input features tc at a
// time), run by persistent workgroups: the grid fills the machine's
// workgroup slots once and each workgroup walks a contiguous range of
// tiles (the P processors of Eq. (2), each with its share of the tiles).
// The (tile, c stage) sequence of a workgroup is one software pipeline:
//
// * In: every input row of the stage's halo'd slab is copied in its
//   natural layout by 16-byte buffer->LDS DMA (the 16-byte-aligned blocks
//   covering the row, so any row alignment is handled by the copy) into a
//   two-slot ring; the copy of stage i+1 -- of the same tile, or the first
//   stage of the next tile -- is in flight while stage i is transposed and
//   multiplied.  One LDS pass (all reads, then all writes) transposes the
//   copy into 8-channel 16-byte vectors [c/8][position][8], the MFMA B
//   operand.
// * Ker, when the whole Ker fits (one k tile, KRES): loaded once per
//   workgroup with aligned 16-byte loads (a feature's 8 channels x all taps
//   are one contiguous 16*RS-byte run) and written to LDS already in MFMA
//   A-operand order [stage][tap][c/8][feature][8]: one 16-byte read per
//   operand, no per-stage work.  Otherwise: raw rows streamed per stage by
//   the same DMA as In (one padding chunk per row so the A-operand reads of
//   8 consecutive features hit distinct banks), A operands built per tap
//   with v_perm.
// * A tile's Out stores are left to drain under the next tile: barriers
//   wait for LDS only, and the wait for a stage's DMA counts the stores
//   issued after it (vector memory operations complete in issue order).
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

namespace {

#define LDS_PTR_S(T, p) ((__attribute__((address_space(3))) T*)(p))

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

// Wait until at most N vector memory operations of this wave are pending.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

}  // namespace

// Per-tile geometry.
template <int NB, int MPOS>
struct StreamGeo {
  int p0, plast, b0, G0, S, kt;
  int t_base[MPOS];  // natural-copy element of each transposed position (shift excluded)
  int t_rs[MPOS];    // (row start element) mod 8, channel 0
  int pix[NB];       // slab position of each lane's output
  uint32_t obyte[NB];
};

template <typename TO, int WM, int WN, int MB, int NB, int TC, int NR, int NS, bool KRES,
          int MPOS, int NDMA>
__global__ __launch_bounds__(64 * WM * WN) void conv_stream(const bf16_t* __restrict__ In,
                                                            const bf16_t* __restrict__ Ker,
                                                            TO* __restrict__ Out, ConvArgs a,
                                                            int nbr) {
  constexpr int NT = 64 * WM * WN;
  constexpr int TK = 32 * WM * MB;
  constexpr int G = TC / 8;
  constexpr int KSTEPS = G / 2;
  constexpr int RS = NR * NS;
  constexpr int RC = (RS * TC / 8) | 1;              // Ker row chunks (odd)
  constexpr int KVECS = (TK * RC + 63) / 64 * 64;    // Ker vectors per stage
  constexpr int NATV = NT * NDMA;                    // natural-copy vectors per ring slot
  constexpr int NSTORE = MB * 16 * NB;               // store instructions per lane per tile
  static_assert(TC % 16 == 0 && NB <= 4, "whole K-steps; at most 4 blocks per wave");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int SN = a.slab_max * a.Ny;                   // transposed positions per group
  u32x4_t* natbuf = reinterpret_cast<u32x4_t*>(smem);  // [2][NATV] natural copies
  u32x4_t* tbuf = natbuf + 2 * NATV;                   // [G][SN] transposed In
  u32x4_t* kbuf = tbuf + G * SN;  // KRES: [n_cc][RS][G][TK] packed; else [2][KVECS] raw rows

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

  auto geometry = [&](int t, StreamGeo<NB, MPOS>& g) __attribute__((always_inline)) {
    const int pt = t / a.n_ktiles;
    g.kt = t - pt * a.n_ktiles;
    g.p0 = pt * a.tp;
    g.plast = min(g.p0 + a.tp, a.npix) - 1;
    g.b0 = g.p0 / a.hw;
    const int w0 = (g.p0 - g.b0 * a.hw) / a.Nh;
    const int b1 = g.plast / a.hw, w1 = (g.plast - b1 * a.hw) / a.Nh;
    g.G0 = g.b0 * a.Nx + a.sw * w0;
    g.S = b1 * a.Nx + a.sw * w1 + NR - g.G0;
#pragma unroll
    for (int m = 0; m < MPOS; ++m) {
      const int pos = min(tid + NT * m, g.S * a.Ny - 1);  // past the slab: repeat the last
      const int row = pos / a.Ny;
      const int y = pos - row * a.Ny;
      const int gr = g.G0 + row;
      const int b = gr / a.Nx;
      const int x = gr - b * a.Nx;
      g.t_base[m] = row * nbr * 8 + y;
      g.t_rs[m] = (int)(((int64_t)b * a.in_img + (int64_t)x * a.Ny) & 7);
    }
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

  // Natural copy of stage cc of tile g into ring slot dst: block f = tid +
  // NT*j is (channel f / (S*nbr), slab row, 16-byte block of the row);
  // blocks past the stage repeat its last block (their slots are unused).
  auto dma_in = [&](const StreamGeo<NB, MPOS>& g, int cc, u32x4_t* dst)
                    __attribute__((always_inline)) {
    const int nblk = TC * g.S * nbr;
    const int c0 = cc * TC;
#pragma unroll
    for (int j = 0; j < NDMA; ++j) {
      const int f = min(tid + NT * j, nblk - 1);
      const int cl = f / (g.S * nbr);
      const int rem = f - cl * (g.S * nbr);
      const int row = rem / nbr;
      const int blk = rem - row * nbr;
      const int gr = g.G0 + row;
      const int b = gr / a.Nx;
      const int x = gr - b * a.Nx;
      const int c = min(c0 + cl, a.Nc - 1);  // channels past Nc: zeroed when transposed
      const int64_t e = (int64_t)b * a.in_img + (int64_t)c * a.nxny + (int64_t)x * a.Ny;
      dma16_t(in_rsrc, dst + NT * j + wave * 64, (uint32_t)(((e & ~(int64_t)7) + 8 * blk) * 2));
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
  // Natural copy (slot src) -> tbuf: all reads first, then all writes.
  auto transpose = [&](const StreamGeo<NB, MPOS>& g, int cc, const u32x4_t* src)
                       __attribute__((always_inline)) {
    const uint16_t* nat = reinterpret_cast<const uint16_t*>(src);
    const int c0 = cc * TC;
    const int cstride = g.S * nbr * 8;
    const uint32_t cs0 = (uint32_t)(((int64_t)c0 * a.nxny) & 7);
    uint32_t e[G][MPOS][8];
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int cl = 8 * gg + i;
        const uint32_t keep = c0 + cl < a.Nc ? 0xffffu : 0u;
        const uint32_t cm = cs0 + (uint32_t)(((int64_t)cl * a.nxny) & 7);
#pragma unroll
        for (int m = 0; m < MPOS; ++m) {
          const int idx = cl * cstride + g.t_base[m] + (int)((g.t_rs[m] + cm) & 7u);
          e[gg][m][i] = (uint32_t)nat[idx] & keep;
        }
      }
    }
    const int snt = g.S * a.Ny;
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
#pragma unroll
      for (int m = 0; m < MPOS; ++m) {
        if (tid + NT * m < snt) {
          u32x4_t v;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = e[gg][m][2 * i] | (e[gg][m][2 * i + 1] << 16);
          tbuf[gg * SN + tid + NT * m] = v;
        }
      }
    }
  };

  f32x16_t acc[MB][NB];
  StreamGeo<NB, MPOS> cur, nxt;
  geometry(t_begin, cur);
  if constexpr (KRES) {
    // (stage, group, feature) triples, two per thread per round; a group's
    // run starts at element (k*Nc + c)*RS with c % 8 == 0, Nc % 8 == 0, so
    // it is 16-byte aligned and RS 16-byte loads cover it.
    const int ntr = n_cc * G * TK;
    for (int t0 = 0; t0 < ntr; t0 += 2 * NT) {
      u32x4_t run[2][RS];
      bool ok[2];
      int dst[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int tr = t0 + tid + NT * u;
        ok[u] = tr < ntr;
        const int trc = ok[u] ? tr : 0;
        const int kk = trc % TK;
        const int g = (trc / TK) % G;
        const int cc = trc / (TK * G);
        const int c = cc * TC + 8 * g;
        ok[u] = ok[u] && c < a.Nc;  // groups past Nc stay zero
        dst[u] = (cc * RS * G + g) * TK + kk;
        const uint32_t off = (uint32_t)((((int64_t)kk * a.Nc + c) * RS) * 2);
#pragma unroll
        for (int q = 0; q < RS; ++q)
          run[u][q] = __builtin_bit_cast(
              u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ker_rsrc, off + 16 * q, 0, 0));
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (t0 + tid + NT * u < ntr) {
#pragma unroll
          for (int tap = 0; tap < RS; ++tap) {
            u32x4_t v;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int e0 = (2 * i) * RS + tap, e1 = e0 + RS;
              const uint32_t sel = ((e0 & 1) ? 0x0302u : 0x0100u) |
                                   ((e1 & 1) ? 0x07060000u : 0x05040000u);
              const uint32_t w1 = run[u][(e1 >> 1) >> 2][(e1 >> 1) & 3];
              const uint32_t w0 = run[u][(e0 >> 1) >> 2][(e0 >> 1) & 3];
              v[i] = ok[u] ? __builtin_amdgcn_perm(w1, w0, sel) : 0u;
            }
            kbuf[dst[u] + tap * G * TK] = v;
          }
        }
      }
    }
  } else {
    dma_ker(cur.kt, 0, kbuf);
  }
  dma_in(cur, 0, natbuf);
  int slot = 0;
  bool stores_pending = false;  // the previous stage ended a tile

  for (int t = t_begin; t < t_end; ++t) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[mb][nb][j] = 0.f;
    const int k0 = cur.kt * TK;

    for (int cc = 0; cc < n_cc; ++cc) {
      // this wave's DMA of the stage has landed (its later tile stores may not)
      if (stores_pending)
        wait_vm<(NSTORE < 63 ? NSTORE : 63)>();
      else
        wait_vm<0>();
      stores_pending = false;
      lds_barrier();  // every wave's DMA landed; every wave done with tbuf
      // next stage's copies: this tile's stage cc+1, or the next tile's first
      if (cc + 1 < n_cc) {
        if constexpr (!KRES) dma_ker(cur.kt, cc + 1, kbuf + (slot ^ 1) * KVECS);
        dma_in(cur, cc + 1, natbuf + (slot ^ 1) * NATV);
      } else if (t + 1 < t_end) {
        geometry(t + 1, nxt);
        if constexpr (!KRES) dma_ker(nxt.kt, 0, kbuf + (slot ^ 1) * KVECS);
        dma_in(nxt, 0, natbuf + (slot ^ 1) * NATV);
      }
      transpose(cur, cc, natbuf + slot * NATV);
      lds_barrier();  // tbuf complete
      const u32x4_t* kb = kbuf + slot * KVECS;
      constexpr int RSD = RS * 4;
      if constexpr (KRES) {
#pragma unroll
        for (int j = 0; j < KSTEPS; ++j) {
          const int grp = 2 * j + half;
          const u32x4_t* ka = kbuf + ((cc * RS) * G + grp) * TK + wm * MB * 32 + l32;
#pragma unroll
          for (int r = 0; r < NR; ++r) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
              const int tap = r * NS + s;
              const int toff = r * a.Ny + s;
              u32x4_t av[MB], bv[NB];
#pragma unroll
              for (int mb = 0; mb < MB; ++mb) av[mb] = ka[tap * G * TK + mb * 32];
#pragma unroll
              for (int nb = 0; nb < NB; ++nb) bv[nb] = tbuf[grp * SN + cur.pix[nb] + toff];
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
      } else
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
            for (int nb = 0; nb < NB; ++nb) bv[nb] = tbuf[grp * SN + cur.pix[nb] + toff];
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
      slot ^= 1;
    }

    // Epilogue: register j of a 32x32 accumulator holds feature
    // 8*(j/4) + 4*half + j%4 of output l32.  Every lane issues exactly
    // NSTORE stores (rows past Nk get an offset beyond the descriptor's
    // range, which drops them), so the next stage's wait can count them.
    const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_t(Out, a.out_total * (int64_t)sizeof(TO));
    const uint32_t half_off = (uint32_t)(4 * half * a.hw * (int)sizeof(TO));
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int kw = k0 + (wm * MB + mb) * 32 + 8 * (j >> 2) + (j & 3);
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
    asm volatile("" ::: "memory");  // the stores stay ahead of the next wait
    stores_pending = true;
    cur = nxt;
  }
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, WM, WN, MB, NB, TC, NR, NS, KRES, MPOS, NDMA): tk = 32*WM*MB,
// largest tile tp = 32*WN*NB, 64*WM*WN threads; KRES keeps all of Ker in
// LDS (needs Nk <= tk); MPOS transposed positions per thread (S*Ny <=
// threads*MPOS); NDMA natural-copy blocks per thread (tc*S*nbr <=
// threads*NDMA, nbr = (Ny+14)/8).
#define CNN_STREAM_VARIANTS(X)                                  \
  X(1300, CNN_BF16, 2, 4, 1, 2, 16, 3, 3, 1, 1, 2)              \
  X(1310, CNN_BF16, 2, 4, 2, 1, 16, 3, 3, 0, 2, 3)              \
  X(1400, CNN_BF16_OBF16, 2, 4, 1, 2, 16, 3, 3, 1, 1, 2)        \
  X(1410, CNN_BF16_OBF16, 2, 4, 2, 1, 16, 3, 3, 0, 2, 3)

static const VariantT kVariantsT[] = {
#define CNN_ROWT(id, dt, wm, wn, mb, nb, tc, nr, ns, kres, mpos, ndma)                 \
  {id, dt, 32 * (wm) * (mb), 32 * (wn) * (nb), tc, 16 * (mb) * (nb), nr, ns, 64 * (wm) * (wn), \
   kres, mpos, ndma},
    CNN_STREAM_VARIANTS(CNN_ROWT)
#undef CNN_ROWT
};

const VariantT* variants_stream(int* count) {
  *count = (int)(sizeof(kVariantsT) / sizeof(kVariantsT[0]));
  return kVariantsT;
}

int64_t stream_nbr(const cnn_problem& p) { return (p.sh * (p.Nh - 1) + p.Ns + 14) / 8; }

int64_t stream_lds_bytes(const VariantT& v, const cnn_problem& p, int64_t slab_rows) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  const int64_t rc = (v.nr * v.ns * v.tc / 8) | 1;
  const int64_t kvecs = (v.tk * rc + 63) / 64 * 64;
  const int64_t n_cc = (p.Nc + v.tc - 1) / v.tc;
  const int64_t natv = (int64_t)v.threads * v.ndma;
  const int64_t ker = v.kres ? n_cc * v.nr * v.ns * (v.tc / 8) * v.tk : 2 * kvecs;
  return (2 * natv + (v.tc / 8) * slab_rows * Ny + ker) * 16;
}

bool stream_fits(const VariantT& v, const cnn_problem& p, int64_t slab_rows) {
  const int64_t Ny = p.sh * (p.Nh - 1) + p.Ns;
  return slab_rows * Ny <= (int64_t)v.threads * v.mpos &&
         v.tc * slab_rows * stream_nbr(p) <= (int64_t)v.threads * v.ndma;
}

template <int DT, int WM, int WN, int MB, int NB, int TC, int NR, int NS, int KRES, int MPOS,
          int NDMA>
static hipError_t launch_t(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                           int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  auto kern = conv_stream<TO, WM, WN, MB, NB, TC, NR, NS, (KRES != 0), MPOS, NDMA>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void*)kern,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int nbr = (a.Ny + 14) / 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(64 * WM * WN), (unsigned)lds, stream,
                     (const bf16_t*)In, (const bf16_t*)Ker, (TO*)Out, a, nbr);
  return hipGetLastError();
}

hipError_t launch_stream(const VariantT& v, const void* In, const void* Ker, void* Out,
                         const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASET(id, dt, wm, wn, mb, nb, tc, nr, ns, kres, mpos, ndma)                        \
  case id:                                                                                    \
    return launch_t<dt, wm, wn, mb, nb, tc, nr, ns, kres, mpos, ndma>(In, Ker, Out, a, lds_bytes, \
                                                                      stream);
    CNN_STREAM_VARIANTS(CNN_CASET)
#undef CNN_CASET
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

// 1x1, stride-1 convolution as a per-pixel GEMM (bf16 MFMA, gfx950).
//
// With Nr = Ns = 1 and unit strides, In[b][c][w][h] and Out[b][k][w][h]
// share the flattened pixel index p = (b, w, h): Out[k][p] = sum_c Ker[k][c]
// * In[c][p] (Eq. (1) with Nr = Ns = 1: no halo).  A workgroup owns a tile of
// tp consecutive pixels by tk output features and walks the input features
// tc at a time (Listing 3 with W_c = N_c):
//
// * In: per stage, the tile's tc channel rows [c][p] in their natural layout,
//   4 pixels (8 bytes) per load, so a load never crosses an image (Nh*Nw and
//   the tile start are multiples of 4).  The MFMA A operand (pixels x 8
//   channels) is read straight from those rows by the transposing LDS read
//   (ds_read_b64_tr_b16): no transpose pass.
// * Ker: per stage, the tk rows [k][c] of tc channels, 16-byte loads; a row
//   segment is the MFMA B operand as it lies (8 consecutive channels).
// * Both are double-buffered in LDS: the next stage's loads are in flight
//   (in registers) while the current stage is multiplied.
// * D[feature][pixel] (Ker as the A operand): a lane ends with one pixel of
//   16 features; each 4-byte store instruction writes 32 consecutive pixels
//   of two features (whole 128-byte rows: faster than 16-byte stores of
//   32-byte pieces of 32 feature rows).
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

namespace {

typedef short s16x4_g __attribute__((ext_vector_type(4)));
#define LDS_PTR_G(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ u32x2_t read_tr16_g(const bf16_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(
      u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR_G(s16x4_g, const_cast<bf16_t*>(p))));
#else
  (void)p;
  return u32x2_t{0u, 0u};
#endif
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_g(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// Wait for this wave's LDS operations, then s_barrier; outstanding global
// loads and stores are not waited for.
__device__ __forceinline__ void lds_barrier_g() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace

// Cache policy of the staged Out stores: sc1, write through to memory
// (device scope).  Measured on whole-line 16-byte stores at the end of a
// tile: 38.2 -> 36.5-37.1 us (ring) and 47.9 -> 47.1 us (stride 2); on
// stores of partial lines, or stores interleaved with other workgroups'
// products, it lost.
constexpr int kStoreThrough = 16;

// TO: Out element type.  WP x WK waves: WP pixel groups of MBP 32-pixel
// blocks, WK feature groups of NBK 32-feature blocks.  TC: channels per stage.
// S2: strides 2 and 2 (Out pixel (w, h) reads In (2w, 2h)): a 4-pixel chunk
// is the even elements of one unaligned 16-byte load (8 input columns),
// picked with v_perm when the chunk is written to LDS; chunks never cross
// an output row (Nh % 4 == 0).
template <typename TO, int WP, int WK, int MBP, int NBK, int TC, bool S2>
__global__ __launch_bounds__(64 * WP * WK) void conv_gemm1(const bf16_t* __restrict__ In,
                                                          const bf16_t* __restrict__ Ker,
                                                          TO* __restrict__ Out, ConvArgs a) {
  constexpr int NT = 64 * WP * WK;
  constexpr int TPMAX = 32 * WP * MBP;   // pixels per tile (at most)
  constexpr int TK = 32 * WK * NBK;      // features per tile
  constexpr int RSI = TPMAX + 16;        // LDS In row (pixels): +32 bytes, distinct banks per channel
  constexpr int RSK = TC + 8;            // LDS Ker row (channels): +16 bytes, conflict-free B reads
  constexpr int IN_ELEMS = TC * RSI;
  constexpr int KER_ELEMS = TK * RSK;
  constexpr int NQ = TPMAX / 4;          // 4-pixel chunks per channel row
  constexpr int NIN = (TC * NQ + NT - 1) / NT;          // In chunks per thread per stage
  constexpr int NKER = (TK * (TC / 8) + NT - 1) / NT;   // Ker blocks per thread per stage
  constexpr int KSTEPS = TC / 16;
  static_assert(TC % 16 == 0, "whole K-steps");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  bf16_t* in_lds = reinterpret_cast<bf16_t*>(smem);            // [2][TC][RSI]
  bf16_t* ker_lds = in_lds + 2 * IN_ELEMS;                      // [2][TK][RSK]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wp = wave / WK, wk = wave % WK;
  const int l32 = lane & 31, half = lane >> 5;

  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int pt = tile / a.n_ktiles;
  const int kt = tile - pt * a.n_ktiles;
  const int p0 = pt * a.tp;
  const int tp = min(a.tp, a.npix - p0);  // pixels of this tile (a multiple of 4)
  const int k0 = kt * TK;
  const int n_st = (a.Nc + TC - 1) / TC;

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_g(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t ker_rsrc = rsrc_g(Ker, (int64_t)a.Nk * a.Nc * 2);
  const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_g(Out, a.out_total * (int64_t)sizeof(TO));

  // Per-thread load slots (fixed over the stages): In chunk f = (channel
  // f / NQ, pixels 4*(f % NQ) .. +3); Ker block g = (feature g / (TC/8),
  // channels 8*(g % (TC/8)) .. +7).  Invalid slots load nothing useful and
  // write zeros (a mask), so every load is issued and every wait is exact.
  int in_off[NIN];        // element offset of the chunk's pixel, channel 0
  int in_c[NIN];          // channel within the stage
  uint32_t in_ok[NIN];    // ~0 if the chunk's pixels are in the tile
  int in_dst[NIN];
#pragma unroll
  for (int j = 0; j < NIN; ++j) {
    const int f = min(tid + NT * j, TC * NQ - 1);
    const int c = f / NQ, q = f % NQ;
    const int p = p0 + 4 * q;
    const bool ok = tid + NT * j < TC * NQ && 4 * q < tp;
    const int pc = ok ? p : p0;
    const int b = pc / a.hw;
    if constexpr (S2) {
      const int rem = pc - b * a.hw, w = rem / a.Nh;
      in_off[j] = b * (int)a.in_img + 2 * w * a.Ny + 2 * (rem - w * a.Nh);
    } else {
      in_off[j] = b * (int)a.in_img + (pc - b * a.hw);  // < in_total < 2^30
    }
    in_c[j] = c;
    in_ok[j] = ok ? ~0u : 0u;
    in_dst[j] = c * RSI + 4 * q;
  }
  int ker_off[NKER];
  int ker_c[NKER];
  bool ker_ok[NKER];
  int ker_dst[NKER];
#pragma unroll
  for (int j = 0; j < NKER; ++j) {
    const int g = min(tid + NT * j, TK * (TC / 8) - 1);
    const int n = g / (TC / 8), cb = g % (TC / 8);
    ker_ok[j] = tid + NT * j < TK * (TC / 8) && k0 + n < a.Nk;
    ker_off[j] = (k0 + n) * a.Nc + 8 * cb;  // (features past Nk masked)
    ker_c[j] = 8 * cb;
    ker_dst[j] = n * RSK + 8 * cb;
  }

  typedef typename std::conditional<S2, u32x4_t, u32x2_t>::type vin_t;
  vin_t vin[NIN];
  u32x4_t vker[NKER];
  // S2: the range check drops a whole dword that straddles the end of In;
  // the only needed element such a dword can hold is In's last, loaded once
  // and patched in when its chunk is written.
  const uint32_t in_last =
      S2 ? __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, (uint32_t)((a.in_total - 1) * 2), 0, 0) : 0u;
  auto load_stage = [&](int s) __attribute__((always_inline)) {
    const int c0 = s * TC;
#pragma unroll
    for (int j = 0; j < NIN; ++j) {
      const int c = min(c0 + in_c[j], a.Nc - 1);
      if constexpr (S2)
        vin[j] = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                         in_rsrc, (uint32_t)((in_off[j] + c * a.nxny) * 2), 0, 0));
      else
        vin[j] = __builtin_bit_cast(
            u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(
                         in_rsrc, (uint32_t)((in_off[j] + c * a.hw) * 2), 0, 0));
    }
#pragma unroll
    for (int j = 0; j < NKER; ++j) {
      const int c = min(c0 + ker_c[j], a.Nc - 8);
      vker[j] = __builtin_bit_cast(
          u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                       ker_rsrc, (uint32_t)((ker_off[j] - ker_c[j] + c) * 2), 0, 0));
    }
  };
  auto write_stage = [&](int s, int buf) __attribute__((always_inline)) {
    const int c0 = s * TC;
    bf16_t* ib = in_lds + buf * IN_ELEMS;
    bf16_t* kb = ker_lds + buf * KER_ELEMS;
#pragma unroll
    for (int j = 0; j < NIN; ++j) {
      const uint32_t keep = (c0 + in_c[j] < a.Nc) ? in_ok[j] : 0u;
      u32x2_t v;
      if constexpr (S2) {
        v = u32x2_t{__builtin_amdgcn_perm(vin[j][1], vin[j][0], 0x05040100u),
                    __builtin_amdgcn_perm(vin[j][3], vin[j][2], 0x05040100u)};
        const int d = (int)(a.in_total - 1) - (in_off[j] + min(c0 + in_c[j], a.Nc - 1) * a.nxny);
        if (d >= 0 && d < 8 && (d & 1) == 0) {  // rare: In's last element, kept element d/2
          const int kq = d >> 1;
          const uint32_t w = v[kq >> 1];
          v[kq >> 1] = (kq & 1) ? ((w & 0xffffu) | (in_last << 16)) : ((w & 0xffff0000u) | in_last);
        }
      } else {
        v = vin[j];
      }
      if (tid + NT * j < TC * NQ)
        *reinterpret_cast<u32x2_t*>(ib + in_dst[j]) = u32x2_t{v[0] & keep, v[1] & keep};
    }
#pragma unroll
    for (int j = 0; j < NKER; ++j) {
      const uint32_t keep = (ker_ok[j] && c0 + ker_c[j] < a.Nc) ? ~0u : 0u;
      if (tid + NT * j < TK * (TC / 8))
        *reinterpret_cast<u32x4_t*>(kb + ker_dst[j]) =
            u32x4_t{vker[j][0] & keep, vker[j][1] & keep, vker[j][2] & keep, vker[j][3] & keep};
    }
  };

  // A operand lane offsets (transposing read, as in the row kernel): lane i
  // of 16-lane group G supplies channel 8*(G/2) + i/4 (+4 for the second
  // read), pixels 16*(G%2) + 4*(i%4) of the 32-pixel block.
  const int G = lane >> 4, li = lane & 15;
  const int aoff0 = (8 * (G >> 1) + (li >> 2)) * RSI + 16 * (G & 1) + 4 * (li & 3) +
                    32 * (wp * MBP);
  const int aoff1 = aoff0 + 4 * RSI;
  const int boff = (wk * NBK * 32 + l32) * RSK + 8 * half;

  f32x16_t acc[MBP][NBK];
#pragma unroll
  for (int mb = 0; mb < MBP; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mb][nb][e] = 0.f;

  load_stage(0);
  write_stage(0, 0);
  lds_barrier_g();
  for (int s = 0; s < n_st; ++s) {
    const int buf = s & 1;
    if (s + 1 < n_st) load_stage(s + 1);
    const bf16_t* ib = in_lds + buf * IN_ELEMS;
    const bf16_t* kb = ker_lds + buf * KER_ELEMS;
    // K-steps of 16 channels, operands one step ahead
    auto read_ops = [&](int ks, u32x4_t (&A)[MBP], u32x4_t (&B)[NBK])
                        __attribute__((always_inline)) {
#pragma unroll
      for (int mb = 0; mb < MBP; ++mb) {
        const u32x2_t lo = read_tr16_g(ib + ks * 16 * RSI + aoff0 + 32 * mb);
        const u32x2_t hi = read_tr16_g(ib + ks * 16 * RSI + aoff1 + 32 * mb);
        A[mb] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
      }
#pragma unroll
      for (int nb = 0; nb < NBK; ++nb)
        B[nb] = *reinterpret_cast<const u32x4_t*>(kb + boff + nb * 32 * RSK + ks * 16);
    };
    u32x4_t A[2][MBP], B[2][NBK];
    read_ops(0, A[0], B[0]);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if (ks + 1 < KSTEPS) read_ops(ks + 1, A[(ks + 1) & 1], B[(ks + 1) & 1]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mb = 0; mb < MBP; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBK; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, B[ks & 1][nb]), __builtin_bit_cast(bf16x8_t, A[ks & 1][mb]),
              acc[mb][nb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (s + 1 < n_st) write_stage(s + 1, buf ^ 1);
    lds_barrier_g();
  }

  // Epilogue: D[feature][pixel] (Ker is the A operand) -- register j of
  // block (mb, nb) holds pixel 32*(wp*MBP + mb) + l32 of the tile, feature
  // k0 + 32*(wk*NBK + nb) + 8(j/4) + 4*half + j%4.
  if constexpr (sizeof(TO) == 4 && 32 * NBK * TPMAX * 4 <= (2 * IN_ELEMS + 2 * KER_ELEMS) * 2) {
    // fp32 Out of a tile inside one image: each feature's tp outputs are one
    // run of tp/4 16-byte units; the runs go through LDS one wk group
    // (32*NBK features) at a time and leave as 16-byte stores of
    // consecutive units.
    const int bi = p0 / a.hw;
    if (a.tp % 4 == 0 && a.hw % 4 == 0 && (p0 + tp - 1) / a.hw == bi) {
      float* stg = reinterpret_cast<float*>(smem);
      const int upf = tp / 4;  // units per feature
      const int nt_q = NT / upf, nt_r = NT - (NT / upf) * upf;
      const int64_t run0 = (int64_t)bi * a.Nk * a.hw + (p0 - bi * a.hw);
#pragma unroll
      for (int rho = 0; rho < WK; ++rho) {
        if (rho > 0) lds_barrier_g();  // the previous round's reads are done
        if (wk == rho) {
#pragma unroll
          for (int mb = 0; mb < MBP; ++mb) {
            const int q = 32 * (wp * MBP + mb) + l32;
            if (q < tp) {
#pragma unroll
              for (int nb = 0; nb < NBK; ++nb)
#pragma unroll
                for (int j = 0; j < 16; ++j)
                  stg[(32 * nb + 8 * (j >> 2) + 4 * half + (j & 3)) * tp + q] = acc[mb][nb][j];
            }
          }
        }
        lds_barrier_g();
        const int f0 = k0 + 32 * NBK * rho;
        const int nf = min(32 * NBK, a.Nk - f0);
        const int units = nf > 0 ? nf * upf : 0;
        const u32x4_t* src = reinterpret_cast<const u32x4_t*>(stg);
        // unit u = fl * upf + pc, stepped by NT without a division per unit
        int fl = tid / upf, pc = tid - (tid / upf) * upf;
        for (int u = tid; u < units; u += NT) {
          const uint32_t off = (uint32_t)((run0 + (int64_t)(f0 + fl) * a.hw) * 4) + 16u * (uint32_t)pc;
          __builtin_amdgcn_raw_buffer_store_b128(src[u], out_rsrc, off, 0, kStoreThrough);
          fl += nt_q;
          pc += nt_r;
          if (pc >= upf) {
            pc -= upf;
            ++fl;
          }
        }
      }
      return;
    }
  }
  // (otherwise each 4-byte store instruction writes 32 consecutive pixels of
  // two features)
#pragma unroll
  for (int mb = 0; mb < MBP; ++mb) {
    const int q = 32 * (wp * MBP + mb) + l32;  // pixel within the tile
    const int p = p0 + (q < tp ? q : 0);
    const int b = p / a.hw;
    const int64_t pix = (int64_t)b * a.Nk * a.hw + (p - b * a.hw);
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb) {
      const int nblk = k0 + 32 * (wk * NBK + nb) + 4 * half;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int n = nblk + 8 * (j >> 2) + (j & 3);
        const uint32_t vo = (n < a.Nk && q < tp)
                                ? (uint32_t)((pix + (int64_t)n * a.hw) * (int64_t)sizeof(TO))
                                : 0x80000000u;
        if constexpr (sizeof(TO) == 4)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[mb][nb][j]), out_rsrc, vo, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc[mb][nb][j]), out_rsrc, vo, 0, 0);
      }
    }
  }
}

// 16-byte buffer -> LDS copy: lane i's 16 bytes land at lds + 16 i (lds
// wave-uniform); out-of-range reads give zeros.
__device__ __forceinline__ void dma16_g(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR_G(void, lds), 16, voff, 0, 0, 0);
#else
  (void)r;
  (void)lds;
  (void)voff;
#endif
}

// The eight transposing reads of a K-step's A operands (four 32-pixel
// blocks, rows r0 and r1 = r0 + 4 channels) in one block that also waits for
// them.  As inline assembly they carry no memory operands the compiler could
// match against the buffer->LDS copies in flight, so it adds no wait for
// those copies (it would wait for all of them before a transposing-read
// builtin); the values are defined only once the block's own wait is done.
__device__ __forceinline__ void read_a4_tr(const bf16_t* r0, const bf16_t* r1, u32x4_t (&A)[4]) {
#if defined(__HIP_DEVICE_COMPILE__)
  const uint32_t p0 = (uint32_t)(uintptr_t)LDS_PTR_G(bf16_t, const_cast<bf16_t*>(r0));
  const uint32_t p1 = (uint32_t)(uintptr_t)LDS_PTR_G(bf16_t, const_cast<bf16_t*>(r1));
  u32x2_t l0, h0, l1, h1, l2, h2, l3, h3;
  asm volatile(
      "ds_read_b64_tr_b16 %0, %8\n\t"
      "ds_read_b64_tr_b16 %1, %9\n\t"
      "ds_read_b64_tr_b16 %2, %8 offset:64\n\t"
      "ds_read_b64_tr_b16 %3, %9 offset:64\n\t"
      "ds_read_b64_tr_b16 %4, %8 offset:128\n\t"
      "ds_read_b64_tr_b16 %5, %9 offset:128\n\t"
      "ds_read_b64_tr_b16 %6, %8 offset:192\n\t"
      "ds_read_b64_tr_b16 %7, %9 offset:192\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(l0), "=&v"(h0), "=&v"(l1), "=&v"(h1), "=&v"(l2), "=&v"(h2), "=&v"(l3), "=&v"(h3)
      : "v"(p0), "v"(p1)
      : "memory");
  A[0] = u32x4_t{l0[0], l0[1], h0[0], h0[1]};
  A[1] = u32x4_t{l1[0], l1[1], h1[0], h1[1]};
  A[2] = u32x4_t{l2[0], l2[1], h2[0], h2[1]};
  A[3] = u32x4_t{l3[0], l3[1], h3[0], h3[1]};
#else
  (void)r0;
  (void)r1;
  for (int i = 0; i < 4; ++i) A[i] = u32x4_t{0u, 0u, 0u, 0u};
#endif
}

// Stride 1 with tiles of whole images (tp = Nw*Nh <= 32*WP*MBP): both
// operands are copied by 16-byte buffer->LDS DMA into a ring of DEPTH stages
// of TC = 32 channels, DEPTH-1 stages ahead of the products, with no
// register staging.  Stage layout in 16-byte units:
// * Ker: TK features x 4 chunks of 8 channels; chunk j of feature k at unit
//   4k + (j ^ ((k >> 2) & 3)), so the 16 lanes reading one chunk index of 16
//   consecutive features hit 16 distinct bank groups;
// * In: TC channel rows of RU units (8 pixels each, RU = ceil(hw/8) made
//   odd, so consecutive rows start in different banks), read by the
//   transposing LDS read as in conv_gemm1.
// Every wave issues NDMA copies per stage (lanes past the data read out of
// range and write zeros inside the stage), so each wait counts exactly.
template <typename TO, int WP, int WK, int MBP, int NBK, int TC, int DEPTH>
__global__ __launch_bounds__(64 * WP * WK) void conv_gemm1d(const bf16_t* __restrict__ In,
                                                           const bf16_t* __restrict__ Ker,
                                                           TO* __restrict__ Out, ConvArgs a) {
  constexpr int NT = 64 * WP * WK;
  constexpr int TPMAX = 32 * WP * MBP;
  constexpr int TK = 32 * WK * NBK;
  static_assert(TC == 32, "the Ker swizzle assumes 4 chunks per feature");
  static_assert(MBP == 4, "read_a4_tr reads four pixel blocks");
  constexpr int KER_UNITS = TK * 4;
  static_assert(KER_UNITS % 64 == 0, "a wave's copy is all Ker or all In");
  constexpr int RU_MAX = ((TPMAX - 8) / 8) | 1;  // whole images of at most TPMAX - 8 pixels
  constexpr int NDMA = (KER_UNITS + TC * RU_MAX + NT - 1) / NT;  // copies per thread per stage
  constexpr int STAGE = NDMA * NT;                                // units per stage
  constexpr int KSTEPS = TC / 16;

  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* ring = reinterpret_cast<u32x4_t*>(smem);  // [DEPTH][STAGE]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wvu = __builtin_amdgcn_readfirstlane(wave);
  const int wp = wave / WK, wk = wave % WK;
  const int l32 = lane & 31, half = lane >> 5;

  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int b = tile / a.n_ktiles;  // a tile is image b
  const int kt = tile - b * a.n_ktiles;
  const int k0 = kt * TK;
  const int hw = a.hw;
  const int RU = ((hw + 7) / 8) | 1;
  const int RSI = 8 * RU;  // In row stride in LDS (elements)
  const int n_st = (a.Nc + TC - 1) / TC;

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_g(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t ker_rsrc = rsrc_g(Ker, (int64_t)a.Nk * a.Nc * 2);
  const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_g(Out, a.out_total * (int64_t)sizeof(TO));

  // Copy slot j of this thread: unit NT*j + tid of every stage.
  int d_base[NDMA];  // element offset at channel offset 0 of the stage
  int d_ch[NDMA];    // channel (within the stage) of the unit's first element
  bool d_ok[NDMA];
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int u = NT * j + tid;
    if (u < KER_UNITS) {
      const int k = u >> 2, ch = (u & 3) ^ ((k >> 2) & 3);
      d_ok[j] = k0 + k < a.Nk;
      d_base[j] = (k0 + k) * a.Nc + 8 * ch;
      d_ch[j] = 8 * ch;
    } else {
      const int v = u - KER_UNITS, c = v / RU, q = v - (v / RU) * RU;
      d_ok[j] = c < TC && 8 * q < hw;
      d_base[j] = (b * a.Nc + c) * hw + 8 * q;
      d_ch[j] = c;
    }
  }
  auto issue = [&](int s) __attribute__((always_inline)) {
    u32x4_t* dst = ring + (s % DEPTH) * STAGE;
    const int c0 = s * TC;
#pragma unroll
    for (int j = 0; j < NDMA; ++j) {
      const bool ok = d_ok[j] && s < n_st && c0 + d_ch[j] < a.Nc;
      if (NT * j + 64 * wvu < KER_UNITS)  // wave-uniform
        dma16_g(ker_rsrc, dst + NT * j + 64 * wvu,
                ok ? (uint32_t)((d_base[j] + c0) * 2) : 0x80000000u);
      else
        dma16_g(in_rsrc, dst + NT * j + 64 * wvu,
                ok ? (uint32_t)((d_base[j] + c0 * hw) * 2) : 0x80000000u);
    }
  };

  // A operand (In rows, transposing read) and B operand (Ker chunks) offsets.
  const int G = lane >> 4, li = lane & 15;
  const int aoff0 = (8 * (G >> 1) + (li >> 2)) * RSI + 16 * (G & 1) + 4 * (li & 3) +
                    32 * (wp * MBP);
  const int aoff1 = aoff0 + 4 * RSI;
  int bunit[NBK][KSTEPS];
#pragma unroll
  for (int nb = 0; nb < NBK; ++nb)
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      const int kf = 32 * (wk * NBK + nb) + l32;
      bunit[nb][ks] = 4 * kf + ((2 * ks + half) ^ ((kf >> 2) & 3));
    }

  f32x16_t acc[MBP][NBK];
#pragma unroll
  for (int mb = 0; mb < MBP; ++mb)
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mb][nb][e] = 0.f;
  // whether this wave's last pixel block holds a pixel of the image (the
  // one that whole images of fewer than TPMAX - 32 pixels leave empty); if
  // not, its products (padding, never stored) are skipped
  const bool last_live = __builtin_amdgcn_readfirstlane(32 * (wp * MBP + MBP - 1) < hw ? 1 : 0) != 0;

#pragma unroll
  for (int s = 0; s < DEPTH - 1; ++s) issue(s);
  for (int s = 0; s < n_st; ++s) {
    // this wave's copies of stage s have landed (the DEPTH-2 later stages'
    // may be in flight), then every wave's have
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(NDMA * (DEPTH - 2)) : "memory");
    issue(s + DEPTH - 1);  // into the buffer every wave finished with in step s-1
    const u32x4_t* kb = ring + (s % DEPTH) * STAGE;
    const bf16_t* ib = reinterpret_cast<const bf16_t*>(kb + KER_UNITS);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      u32x4_t A[MBP], B[NBK];
#pragma unroll
      for (int nb = 0; nb < NBK; ++nb) B[nb] = kb[bunit[nb][ks]];
      read_a4_tr(ib + ks * 16 * RSI + aoff0, ib + ks * 16 * RSI + aoff1, A);
#pragma unroll
      for (int mb = 0; mb < MBP; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBK; ++nb)
          if (mb + 1 < MBP || last_live)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, B[nb]), __builtin_bit_cast(bf16x8_t, A[mb]),
                acc[mb][nb], 0, 0, 0);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the trailing (empty) copies

  // The tile's Out (image b, features k0 .. k0+TK-1, all hw pixels) is one
  // contiguous run; it goes through LDS in rounds of 128 features (the
  // waves with wk in {2 rho, 2 rho + 1}) and leaves as 16-byte stores of
  // consecutive units (4 fp32 or 8 bf16 values), whole cache lines but at
  // the run's two ends -- when the run starts and ends on 16-byte
  // boundaries (always for fp32; for bf16 unless hw and the feature count
  // are odd multiples of 4 and 2), else through the stores below.
  constexpr int EPU = 16 / (int)sizeof(TO);  // Out values per 16-byte unit
  if constexpr (128 * TPMAX * (int)sizeof(TO) <= DEPTH * STAGE * 16) {
    const bool whole_units = ((int64_t)b * a.Nk + k0) * hw % EPU == 0 &&
                             (a.Nk - k0 >= TK || (int64_t)(a.Nk - k0) * hw % EPU == 0);
    if (whole_units) {
      TO* stg = reinterpret_cast<TO*>(smem);
      constexpr int WPR = 128 / (32 * NBK);  // wk values per round
      static_assert(WK % WPR == 0, "whole rounds");
#pragma unroll
      for (int rho = 0; rho < WK / WPR; ++rho) {
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");  // LDS free
        if (wk / WPR == rho) {
#pragma unroll
          for (int mb = 0; mb < MBP; ++mb) {
            const int q = 32 * (wp * MBP + mb) + l32;
            if (q < hw) {
#pragma unroll
              for (int nb = 0; nb < NBK; ++nb)
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                  const int fl = 32 * ((wk % WPR) * NBK + nb) + 8 * (j >> 2) + 4 * half + (j & 3);
                  stg[fl * hw + q] = from_f32<TO>(acc[mb][nb][j]);
                }
            }
          }
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        const int f0 = k0 + 128 * rho;  // first feature of the round
        const int nf = min(128, a.Nk - f0);
        const int units = nf > 0 ? nf * hw / EPU : 0;
        const uint32_t base = (uint32_t)(((int64_t)b * a.Nk + f0) * hw * (int64_t)sizeof(TO));
        const u32x4_t* src = reinterpret_cast<const u32x4_t*>(stg);
        // whole lines, stored through to memory (sc1): they drain during the
        // kernel instead of waiting, dirty in the L2, for its end
        for (int u = tid; u < units; u += NT)
          __builtin_amdgcn_raw_buffer_store_b128(src[u], out_rsrc,
                                                 base + 16u * (uint32_t)u, 0, kStoreThrough);
      }
      return;
    }
  }

  // Epilogue as in conv_gemm1: a lane holds pixel q of 16 features.
#pragma unroll
  for (int mb = 0; mb < MBP; ++mb) {
    const int q = 32 * (wp * MBP + mb) + l32;
    const int64_t pix = (int64_t)b * a.Nk * hw + (q < hw ? q : 0);
#pragma unroll
    for (int nb = 0; nb < NBK; ++nb) {
      const int nblk = k0 + 32 * (wk * NBK + nb) + 4 * half;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int n = nblk + 8 * (j >> 2) + (j & 3);
        const uint32_t vo = (n < a.Nk && q < hw)
                                ? (uint32_t)((pix + (int64_t)n * hw) * (int64_t)sizeof(TO))
                                : 0x80000000u;
        if constexpr (sizeof(TO) == 4)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[mb][nb][j]), out_rsrc, vo, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc[mb][nb][j]), out_rsrc, vo, 0, 0);
      }
    }
  }
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, WP, WK, MBP, NBK, TC, mode): tk = 32*WK*NBK, tp <= 32*WP*MBP,
// 64*WP*WK threads; mode 0: stride 1, 1: strides 2 and 2, 2: stride 1 with
// whole-image tiles through the DMA ring (conv_gemm1d, four stages).
#define CNN_GEMM1_VARIANTS(X)                  \
  X(1700, CNN_BF16, 2, 4, 4, 2, 64, 0)         \
  X(1701, CNN_BF16, 4, 2, 2, 2, 64, 0)         \
  X(1702, CNN_BF16, 2, 4, 4, 2, 32, 1)         \
  X(1709, CNN_BF16, 2, 4, 4, 2, 32, 2)         \
  X(1800, CNN_BF16_OBF16, 2, 4, 4, 2, 64, 0)   \
  X(1801, CNN_BF16_OBF16, 4, 2, 2, 2, 64, 0)   \
  X(1802, CNN_BF16_OBF16, 2, 4, 4, 2, 32, 1)   \
  X(1809, CNN_BF16_OBF16, 2, 4, 4, 2, 32, 2)

static const VariantG kVariantsG[] = {
#define CNN_GV(id, dt, wp, wk, mbp, nbk, tc, s2) \
  {id, dt, 32 * wk * nbk, 32 * wp * mbp, tc, 64 * wp * wk, 16 * mbp * nbk, s2},
    CNN_GEMM1_VARIANTS(CNN_GV)
#undef CNN_GV
};

const VariantG* variants_gemm1(int* count) {
  *count = (int)(sizeof(kVariantsG) / sizeof(kVariantsG[0]));
  return kVariantsG;
}

int64_t gemm1_lds_bytes(const VariantG& v) {
  if (v.s2 == 2) {  // a ring of 4 stages of NDMA*threads units
    const int64_t ndma =
        (v.tk * 4 + (int64_t)v.tc * (((v.tp - 8) / 8) | 1) + v.threads - 1) / v.threads;
    return 4 * ndma * v.threads * 16;
  }
  return 2 * ((int64_t)v.tc * (v.tp + 16) + (int64_t)v.tk * (v.tc + 8)) * 2;
}

bool gemm1_fits(const VariantG& v, const cnn_problem& p, int64_t tp) {
  if (v.s2 == 2)  // whole-image tiles
    return p.Nr == 1 && p.Ns == 1 && p.sw == 1 && p.sh == 1 && p.Nc % 8 == 0 &&
           (p.Nw * p.Nh) % 4 == 0 && p.Nw * p.Nh <= v.tp - 8 && tp == p.Nw * p.Nh;
  if (v.s2 == 1)
    return p.Nr == 1 && p.Ns == 1 && p.sw == 2 && p.sh == 2 && p.Nc % 8 == 0 && p.Nh % 4 == 0 &&
           tp % 4 == 0 && tp >= 4;
  return p.Nr == 1 && p.Ns == 1 && p.sw == 1 && p.sh == 1 && p.Nc % 8 == 0 &&
         (p.Nw * p.Nh) % 4 == 0 && tp % 4 == 0 && tp >= 4;
}

template <typename TO, int WP, int WK, int MBP, int NBK, int TC, int S2>
struct Gemm1Kernel {
  static constexpr auto fn = conv_gemm1<TO, WP, WK, MBP, NBK, TC, S2 == 1>;
};
template <typename TO, int WP, int WK, int MBP, int NBK, int TC>
struct Gemm1Kernel<TO, WP, WK, MBP, NBK, TC, 2> {
  static constexpr auto fn = conv_gemm1d<TO, WP, WK, MBP, NBK, TC, 4>;
};

template <int DT, int WP, int WK, int MBP, int NBK, int TC, int S2>
static hipError_t launch_g(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                           int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  auto kern = Gemm1Kernel<TO, WP, WK, MBP, NBK, TC, S2>::fn;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(64 * WP * WK), (unsigned)lds, stream,
                     (const bf16_t*)In, (const bf16_t*)Ker, (TO*)Out, a);
  return hipGetLastError();
}

hipError_t launch_gemm1(const VariantG& v, const void* In, const void* Ker, void* Out,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASEG(id, dt, wp, wk, mbp, nbk, tc, s2) \
  case id:                                         \
    return launch_g<dt, wp, wk, mbp, nbk, tc, s2>(In, Ker, Out, a, lds_bytes, stream);
    CNN_GEMM1_VARIANTS(CNN_CASEG)
#undef CNN_CASEG
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

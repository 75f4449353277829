// Stride-2 convolution over bands of whole output rows (bf16 MFMA, gfx950).
//
// Out[b][k][w][h] = sum_{c,r,s} In[b][c][2w+r][2h+s] * Ker[k][c][r][s]
// (Eq. (1)'s problem with sigma_w = sigma_h = 2).  A workgroup owns a band of
// L whole output rows of one image by TK = 256 output features and walks the
// input features 16 at a time (Listing 3 with W_c = N_c); each 16-channel
// chunk is taken in Nr stages, one stencil row r per stage.
//
// * In: per chunk, the band's 2(L-1)+Nr input rows, 16-byte loads of 8
//   columns of one channel (rows start at any element; the loads are
//   unaligned).  Registers transpose four channels x eight columns into
//   MFMA-ready units of channels, split by column parity: unit (g, row, i)
//   holds the 8 channels of group g at column 2i, unit (g, row, 32 + i) at
//   column 2i+1.  Tap s of output position h reads unit s/2 + h (s even)
//   or 32 + (s-1)/2 + h (s odd): for every tap the 32 positions of a row are
//   32 consecutive 16-byte units, read with ds_read_b128.
// * Ker: repacked once per call into the B-operand image of every (k tile,
//   chunk, stencil row) slice, [s][g][k][8 channels]; a stage copies the
//   next stage's slice (24 KB for 3x3) straight into LDS with 16-byte
//   buffer->LDS loads, one contiguous kilobyte per wave instruction.
// * Buffers: Ker slices four deep (the copy for stage t + 3 is issued in
//   stage t; stage t's last K-step already reads stage t + 1's operands), In
//   two deep by chunk (the next chunk's loads are issued in a chunk's first
//   stage and written during its second); copies, loads, In writes and
//   operand reads are issued between the K-steps' products; one barrier per
//   stage.
// * Waves: waves w and w+4 (one SIMD) take features 64*(w%4) .. +63 (two
//   32-feature blocks) x the band's L rows, half of the (row, block) pairs
//   each, with the same straight-line code for odd L too.  A 32-position
//   MFMA block is one output row (Nh <= 32).
// * D[feature][position] (Ker is the A operand): a lane ends with one
//   position of 16 features, written as 4-byte (2-byte) stores; each store
//   instruction writes whole rows (Nh positions) of two features, which
//   measured faster than 16-byte stores of 32-byte pieces of 32 rows.
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

namespace {

#define LDS_PTR_Q(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_q(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// 16-byte buffer -> LDS copy: lane i's 16 bytes land at lds + 16 i (lds
// wave-uniform).
__device__ __forceinline__ void dma16_q(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR_Q(void, lds), 16, voff, 0, 0, 0);
#else
  (void)r;
  (void)lds;
  (void)voff;
#endif
}

// f(integral_constant<int, I>) for I = B .. E-1, in order.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>());
    static_for<B + 1, E>(f);
  }
}

}  // namespace

// TO: Out element type.  NR x NS stencil, stride 2 both ways; L output rows
// per band.
template <typename TO, int NR, int NS, int L, int NWV>
__global__ __launch_bounds__(64 * NWV) void conv_srows(const bf16_t* __restrict__ In,
                                                  const u32x4_t* __restrict__ Kp,
                                                  TO* __restrict__ Out, ConvArgs a,
                                                  int blk_vecs) {
  constexpr int NT = 64 * NWV;
  constexpr bool SPLIT = NWV == 8;  // two waves per feature pair (rows split)
  constexpr int TK = 256;
  constexpr int SR = NR >= 2 ? 2 * (L - 1) + NR : L;  // slab rows held per chunk
  constexpr int SX = NR >= 2 ? 1 : 2;                 // input rows per slab row
  constexpr int RW = SPLIT ? (L + 1) / 2 : L;         // rows per wave
  constexpr int NI = 2 * SR * 8 * 2;                  // In items per chunk
  constexpr int NIPT = (NI + NT - 1) / NT;            // items per thread
  constexpr int IN_UNITS = 2 * SR * 64;               // 16-byte units per In buffer
  constexpr int KER_UNITS = NS * 2 * TK;              // per Ker buffer (one stencil row)
  constexpr int NDK = KER_UNITS / NT;                 // copies per thread per stage
  static_assert(NWV == 4 || NWV == 8, "one or two waves per feature pair");
  static_assert(L >= 2 && RW <= (SPLIT ? 4 : 8), "rows per wave");
  static_assert(NR >= 2, "In loads one stage ahead of their LDS writes");
  static_assert(NS <= 3 && NR <= 3, "taps within one 64-unit row");
  static_assert(KER_UNITS % NT == 0, "whole copies");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* kbuf = reinterpret_cast<u32x4_t*>(smem);  // [4][NS][2][TK]
  u32x4_t* ibuf = kbuf + 4 * KER_UNITS;              // [2][2][SR][64]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int fp = wave & 3;   // feature pair
  const int rg = SPLIT ? wave >> 2 : 0;  // row group
  const int l32 = lane & 31, half = lane >> 5;

  const int n_bands = a.Nw / L;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int band = tile / a.n_ktiles;
  const int kt = tile - band * a.n_ktiles;
  const int b = band / n_bands;
  const int w0 = (band - b * n_bands) * L;
  const int k0 = kt * TK;
  const int n_cc = a.Nc / 16;

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_q(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t kp_rsrc =
      rsrc_q(Kp, (int64_t)a.n_ktiles * n_cc * blk_vecs * 16);
  const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_q(Out, a.out_total * (int64_t)sizeof(TO));

  // ---- In layout: unit u (0..63) of a slab row holds column 2u (u < 32) or
  // 2(u-32)+1; within each aligned group of 4 units it sits at slot
  // swz(u) = 4 (u/4) + (u%4 + 2 ((u/16) % 2) + row % 2) % 4.  The rotation
  // makes the 8-byte writes of a half wave (blocks b8 and b8 + 4, rows j and
  // j + 1) cover all 64 banks, while any 32 consecutive units -- an operand
  // read, whose partial end groups are 8 groups apart and rotate alike --
  // still fall in distinct banks.
  // ---- In items: (g, slab row j, 8-column block b8, channel half hc); an
  // item is four 16-byte loads (channels 8g + 4hc + 0..3 of the chunk).
  // The range check drops a whole dword that straddles the end of In; the
  // only element such a dword can hold is In's last, loaded once and
  // patched in when the item is written.
  const uint32_t in_last =
      __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, (uint32_t)((a.in_total - 1) * 2), 0, 0);
  int in_e[NIPT];    // element offset of the item's channel 8g + 4hc of chunk 0
  int in_dst[NIPT];  // unit of its first even column (+ 8 bytes for hc = 1)
  int in_hc[NIPT];
  int in_rot[NIPT];  // the block's slot rotation (swz)
  bool in_ok[NIPT];
#pragma unroll
  for (int j = 0; j < NIPT; ++j) {
    const int t = tid + NT * j;
    const int tt = t < NI ? t : NI - 1;
    const int hc = tt & 1, b8 = (tt >> 1) & 7, gj = tt >> 4;
    const int g = gj / SR, jr = gj - g * SR;
    const int x = 2 * w0 + jr * SX;
    in_e[j] = (int)((int64_t)b * a.in_img) + (8 * g + 4 * hc) * a.nxny + x * a.Ny + 8 * b8;
    in_dst[j] = (g * SR + jr) * 64 + 4 * b8;
    in_hc[j] = hc;
    in_rot[j] = 2 * ((b8 >> 2) & 1) + (jr & 1);
    in_ok[j] = t < NI;
  }
  u32x4_t vin[NIPT][4];
  auto load_in_part = [&](int cc, int k0_, int k1_) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < NIPT; ++j)
#pragma unroll
      for (int k = k0_; k < k1_; ++k)
        vin[j][k] = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                         in_rsrc, (uint32_t)((in_e[j] + (16 * cc + k) * a.nxny) * 2), 0, 0));
  };
  // Write steps [i0_, i1_) of the items' units: step i writes column pair i
  // of the block, units 4 b8 + i (even column) and 32 + 4 b8 + i (odd
  // column), 8 bytes each, at their swizzled slots (swz below).
  auto write_in_part = [&](int cc, u32x4_t* dstb, int i0_, int i1_) __attribute__((always_inline)) {
    char* base = reinterpret_cast<char*>(dstb);
#pragma unroll
    for (int j = 0; j < NIPT; ++j) {
      if (!in_ok[j]) continue;
      u32x4_t v[4] = {vin[j][0], vin[j][1], vin[j][2], vin[j][3]};
      // the last-element patch (one item of the whole tensor)
      const int d0 = (int)(a.in_total - 1) - (in_e[j] + 16 * cc * a.nxny);
      if (d0 >= 0 && d0 < 3 * a.nxny + 8) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int d = d0 - k * a.nxny;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const uint32_t lo = d == 2 * i ? ((v[k][i] & 0xffff0000u) | in_last) : v[k][i];
            v[k][i] = d == 2 * i + 1 ? ((lo & 0xffffu) | (in_last << 16)) : lo;
          }
        }
      }
      char* p = base + in_dst[j] * 16 + 8 * in_hc[j];
#pragma unroll
      for (int i = i0_; i < i1_; ++i) {
        const int slot = 16 * ((i + in_rot[j]) & 3);
        const u32x2_t ev = {__builtin_amdgcn_perm(v[1][i], v[0][i], 0x05040100u),
                            __builtin_amdgcn_perm(v[3][i], v[2][i], 0x05040100u)};
        *reinterpret_cast<u32x2_t*>(p + slot) = ev;
        if (NS > 1) {
          const u32x2_t od = {__builtin_amdgcn_perm(v[1][i], v[0][i], 0x07060302u),
                              __builtin_amdgcn_perm(v[3][i], v[2][i], 0x07060302u)};
          *reinterpret_cast<u32x2_t*>(p + 16 * 32 + slot) = od;
        }
      }
    }
  };
  auto write_in = [&](int cc, u32x4_t* dstb) __attribute__((always_inline)) {
    write_in_part(cc, dstb, 0, 4);
  };
  // Ker slice (chunk cc, stencil row r) -> a Ker buffer, in NDK pieces of
  // one 16-byte copy per thread
  auto copy_ker_piece = [&](int cc, int r, u32x4_t* dst, int j) __attribute__((always_inline)) {
    const uint32_t base = (uint32_t)((kt * n_cc + cc) * blk_vecs + r * KER_UNITS);
    dma16_q(kp_rsrc, dst + NT * j + 64 * wave, (base + NT * j + tid) * 16u);
  };
  auto copy_ker = [&](int cc, int r, u32x4_t* dst) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < NDK; ++j) copy_ker_piece(cc, r, dst, j);
  };

  // Rows and feature blocks of a wave (the two waves of a SIMD, w and w+4,
  // together cover the band's L rows x the feature pair's two blocks):
  //   even L: wave w+4*q takes rows q*L/2 + i, both blocks;
  //   odd L = 2m+1: wave w takes rows i = 0..m with block 0 and rows 0..m-1
  //   with block 1; wave w+4 takes rows L-1-i with block 1 and rows L-1-i,
  //   i < m, with block 0.  Row m is split between them by block, so both
  //   run the same 2*RW - 1 products per K-step, straight-line.
  constexpr bool ODD = SPLIT && (L & 1) != 0;
  const int row0 = rg == 0 ? 0 : (ODD ? L - 1 : L / 2);  // band row of i = 0 (rg = 0: 4 waves)
  const int rdir = (rg == 1 && ODD) ? -1 : 1;
  const int nbf = (rg == 1 && ODD) ? 1 : 0;               // block of the first B operand
  auto has_second = [](int i) { return !ODD || i < RW - 1; };
  // Operand offsets (units): A = In unit (half, slab row, position l32);
  // B = Ker unit (s, half, feature 64 fp + 32 nb + l32).
  const int a_off = half * SR * 64;
  // swizzled unit offset of this lane's position for tap s and row parity
  auto swz = [](int u, int par) { return (u & ~3) | (((u & 3) + 2 * ((u >> 4) & 1) + par) & 3); };
  int a_sw[NS][2];
#pragma unroll
  for (int s_ = 0; s_ < NS; ++s_)
#pragma unroll
    for (int par = 0; par < 2; ++par)
      a_sw[s_][par] = swz(((s_ & 1) ? 32 + (s_ >> 1) : (s_ >> 1)) + l32, par);
  const int b_first = half * TK + 64 * fp + 32 * nbf + l32;
  const int b_second = half * TK + 64 * fp + 32 * (1 - nbf) + l32;

  f32x16_t acc[RW][2];
#pragma unroll
  for (int i = 0; i < RW; ++i)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][nb][e] = 0.f;

  // Operand registers of two consecutive K-steps (parity p): A[p][i] = In
  // unit of row i, B[p][q] = Ker unit of the wave's first / second block.
  u32x4_t A[2][RW], B[2][2];
  auto read_a = [&](const u32x4_t* ib, int r, int s, int i) __attribute__((always_inline)) {
    const int jr = (2 * (row0 + rdir * i) + r) / SX;
    return ib[a_off + jr * 64 + a_sw[s][jr & 1]];
  };
  auto read_b = [&](const u32x4_t* kb, int s, int q) __attribute__((always_inline)) {
    return kb[s * 2 * TK + (q ? b_second : b_first)];
  };

  // One stage (stencil row r of the chunk in ib, Ker slice kb): the
  // products of NS K-steps from operand parity P, whose step-0 operands are
  // already in registers.  Each next step's operands -- in the last step,
  // those of the next stage's first step (nib, nkb, nr), whose data landed
  // before the previous barrier -- are read between the products, one row
  // ahead of their use, so no stage starts on a cold LDS read.  mem(slot)
  // issues this stage's share of the copies and loads for later stages
  // (slot 0 first, slot s + 1 after K-step s's products).
  auto stage = [&](auto PC, const u32x4_t* ib, const u32x4_t* kb, int r, const u32x4_t* nib,
                   const u32x4_t* nkb, int nr, auto mem) __attribute__((always_inline)) {
    constexpr int P = decltype(PC)::value;
    mem(0);
    __builtin_amdgcn_sched_barrier(0);
    static_for<0, NS>([&](auto SC) {
      constexpr int st = decltype(SC)::value;
      constexpr int cu = (P + st) & 1, nx = cu ^ 1;
#pragma unroll
      for (int i = 0; i < RW; ++i) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
          if (q == 0 || has_second(i))
            acc[i][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8_t, B[cu][q]), __builtin_bit_cast(bf16x8_t, A[cu][i]),
                acc[i][q], 0, 0, 0);
        if (i == 0) {
          B[nx][0] = st + 1 < NS ? read_b(kb, st + 1, 0) : read_b(nkb, 0, 0);
          B[nx][1] = st + 1 < NS ? read_b(kb, st + 1, 1) : read_b(nkb, 0, 1);
        }
        A[nx][i] = st + 1 < NS ? read_a(ib, r, st + 1, i) : read_a(nib, nr, 0, i);
        __builtin_amdgcn_sched_barrier(0);
      }
      mem(st + 1);
      __builtin_amdgcn_sched_barrier(0);
    });
  };

  // ---- prologue: chunk 0's rows and the first three Ker slices.  Ker is
  // four slices deep: stage t reads buffer t % 4 and, in its last K-step,
  // buffer (t + 1) % 4; the copy for stage t + 3 is issued during stage t
  // and waited for at the end of stage t + 1.
  copy_ker(0, 0, kbuf);
#pragma unroll
  for (int t = 1; t < 3; ++t) copy_ker(min(t / NR, n_cc - 1), t % NR, kbuf + t * KER_UNITS);
  load_in_part(0, 0, 4);
  write_in(0, ibuf);
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  B[0][0] = read_b(kbuf, 0, 0);
  B[0][1] = read_b(kbuf, 0, 1);
#pragma unroll
  for (int i = 0; i < RW; ++i) A[0][i] = read_a(ibuf, 0, 0, i);

  int kcur = 0;  // Ker buffer of the current stage
  for (int cc = 0; cc < n_cc; ++cc) {
    const int cn = cc + 1 < n_cc ? cc + 1 : cc;  // (the last chunk reloads itself)
    const u32x4_t* ib = ibuf + (cc & 1) * IN_UNITS;
    static_for<0, NR>([&](auto RC) {
      constexpr int r = decltype(RC)::value;
      const u32x4_t* kb = kbuf + kcur * KER_UNITS;
      const int k1 = (kcur + 1) & 3, k3 = (kcur + 3) & 3;
      // stage + 3: (cc3, r3), clamped to the last chunk (a redundant copy)
      const int cc3 = min(cc + (r + 3) / NR, n_cc - 1), r3 = (r + 3) % NR;
      auto mem = [&](int slot) __attribute__((always_inline)) {
        if (r == 0 && slot == 0) load_in_part(cn, 0, 2);
        if (r == 0 && slot == 1) load_in_part(cn, 2, 4);
        if (r == NR - 2 && slot == 1) write_in_part(cn, ibuf + ((cc + 1) & 1) * IN_UNITS, 0, 2);
        if (r == NR - 2 && slot == 2) write_in_part(cn, ibuf + ((cc + 1) & 1) * IN_UNITS, 2, 4);
#pragma unroll
        for (int j = 0; j < NDK; ++j)
          if (slot == 1 + (j * NS) / NDK) copy_ker_piece(cc3, r3, kbuf + k3 * KER_UNITS, j);
      };
      // the next stage: (cc, r + 1), or (cc + 1, 0) from the other In buffer
      const u32x4_t* nib = r + 1 < NR ? ib : ibuf + ((cc + 1) & 1) * IN_UNITS;
      stage(std::integral_constant<int, (r * NS) & 1>(), ib, kb, r, nib, kbuf + k1 * KER_UNITS,
            (r + 1) % NR, mem);
      __builtin_amdgcn_sched_barrier(0);
      // the copy issued a stage ago (for stage + 2) has landed; this stage's
      // copies may stay in flight.  Copies into LDS complete in issue order
      // among themselves, but a load into registers issued after a copy may
      // complete before it.  So the wait is stated over copies alone: each
      // wave issued NDK copies after the ones waited for, and while any
      // earlier copy is outstanding, so are those NDK, so vmcnt <= NDK
      // implies the earlier copies are done, whatever In loads (issued in
      // stage 0 of each chunk) are still in flight.
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(NDK) : "memory");
      kcur = k1;
    });
    if constexpr (((NR * NS) & 1) != 0) {
      // a chunk has an odd number of K-steps: the next chunk's first
      // operands were read into parity 1
#pragma unroll
      for (int i = 0; i < RW; ++i) A[0][i] = A[1][i];
      B[0][0] = B[1][0];
      B[0][1] = B[1][1];
    }
  }

  // ---- epilogue: register j of block (i, q) holds position l32 of output
  // row w0 + row0 + rdir*i, feature k0 + 64 fp + 32 (q ? 1 - nbf : nbf) +
  // 8 (j/4) + 4 half + j%4.
  // (byte offsets: the lane's part once per block, plus the wave-uniform
  // steps of feature and row; lanes past Nh or Nk store out of range)
  const int kl = l32 < a.Nh ? a.Nk - 4 * half : -1;  // valid: first feature + step < kl
  const uint32_t hw_b = (uint32_t)(a.Nw * a.Nh * (int)sizeof(TO)), nh_b = (uint32_t)(a.Nh * (int)sizeof(TO));
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int fb = k0 + 64 * fp + 32 * (q ? 1 - nbf : nbf);  // the block's first feature (half 0)
    const uint32_t vo_q =
        (uint32_t)(((((int64_t)b * a.Nk + fb + 4 * half) * a.Nw + w0 + row0) * a.Nh + l32) *
                   (int64_t)sizeof(TO));
#pragma unroll
    for (int i = 0; i < RW; ++i) {
      if (q == 1 && !has_second(i)) continue;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int f = 8 * (j >> 2) + (j & 3);
        const uint32_t vo = fb + f < kl ? vo_q + (uint32_t)f * hw_b + (uint32_t)(rdir * i) * nh_b
                                        : 0x80000000u;
        if constexpr (sizeof(TO) == 4)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[i][q][j]), out_rsrc, vo, 0, 0);
        else
          __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc[i][q][j]), out_rsrc, vo, 0, 0);
      }
    }
  }
}

// ---- raw-Ker form -------------------------------------------------------------
// conv_srows2: the same bands, In staging and operand layout, with two
// differences.  Ker is read in its raw layout ([k][c][r][s]: a feature's 16
// channels x RS taps of a chunk are one 32*RS-byte run) and repacked on
// chip, so no workspace is needed; and the workgroup's 256 features are two
// tiles of 128 taken one after the other, with two accumulator sets, so the
// first tile's Out rows are stored while the second tile is multiplied (one
// row per chunk over the second tile's first L chunks, which needs at least
// L chunks: Nc >= 16 L) and only the second tile's drain remains after the
// last product.  Four waves (one per SIMD): wave w takes features
// 32w .. 32w+31 of the tile for all L rows of the band.
// * Ker, per chunk: the raw runs of the tile's 128 features are copied by
//   16-byte buffer->LDS DMA into a raw buffer (one contiguous kilobyte per
//   wave instruction); thread (k, g) = (tid/2, tid%2) reads its feature's
//   8-channel run (RS units, conflict free) back into registers and, one
//   stage ahead of its use (two stages before it is read), writes the three
//   B-operand units of a stencil row -- [s][g][k] planes of 132 units, so
//   the two g planes of 8 consecutive lanes' writes start 16 banks apart
//   (measured faster than 136) -- into that row's slot.
// * Schedule of chunk x (global over both tiles; stage r = stencil row r):
//   stage 0 packs slot 2 for (x, 2) and writes In(x+1) from registers;
//   stage 1 loads In(x+2) into them, reads back raw(x+1) and packs slot 0
//   for (x+1, 0); stage 2 copies raw(x+2) by DMA and packs slot 1 for
//   (x+1, 1).  In the second tile's first L chunks, stages 1 and 2 also
//   store one row of the first tile.  One barrier per stage; the one ending
//   stage 0 waits for all the wave's vector-memory work (the raw copies into
//   LDS are not ordered with the In loads in the wait counter).
// * With one wave per SIMD, a wave stalled on issue leaves its SIMD's MFMA
//   idle: every piece of this memory work is issued singly between two of
//   the stage's products (a stage's pieces spread evenly over its NS*L
//   products), so the vector-memory and LDS queues never hold a burst.
// * The range check drops a whole dword that straddles the end of In, and
//   the loads start at any element: In's last element, loaded once, is
//   written into its LDS unit after the item holding it (a masked 2-byte
//   write per item and chunk; the other lanes write a scratch area).
template <typename TO, int NR, int NS, int L>
__global__ __launch_bounds__(256) void conv_srows2(const bf16_t* __restrict__ In,
                                                   const bf16_t* __restrict__ Ker,
                                                   TO* __restrict__ Out, ConvArgs a) {
  constexpr int NT = 256;
  constexpr int TKT = 128;                 // features per tile
  constexpr int RS = NR * NS;
  constexpr int SR = 2 * (L - 1) + NR;     // slab rows held per chunk
  constexpr int NI = 2 * SR * 8 * 2;       // In items per chunk
  constexpr int NIPT = (NI + NT - 1) / NT; // items per thread
  constexpr int IN_UNITS = 2 * SR * 64;    // 16-byte units per In buffer
  constexpr int RAW_UNITS = TKT * 2 * RS;  // raw Ker of a chunk: 128 x 16 channels x RS
  constexpr int NDMA = RAW_UNITS / NT;     // raw copies per thread per chunk
  constexpr int PST = TKT + 4;             // B-operand plane stride (units)
  constexpr int SLOT = NS * 2 * PST;       // units per stage slot
  constexpr int NQ = NS * L;               // products per wave per stage
  constexpr int NSTO = 16;                 // Out stores per row
  constexpr int NSH = NSTO / 2;            // of them in each of stages 1 and 2
  constexpr int SCRATCH_OFF = (NR * SLOT + RAW_UNITS + 2 * IN_UNITS) * 16;  // bytes
  static_assert(RAW_UNITS % NT == 0, "whole copies");
  static_assert(NR == 3 && NS <= 3, "one slot per stencil row, taps within one 64-unit row");
  static_assert(L >= 1 && L <= 7, "rows per band (two accumulator sets)");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* kslot = reinterpret_cast<u32x4_t*>(smem);  // [NR][NS][2][PST]
  u32x4_t* raw = kslot + NR * SLOT;                    // [RAW_UNITS]
  u32x4_t* ibuf = raw + RAW_UNITS;                     // [2][2][SR][64]
  // (then a 2 KiB scratch area: writes of lanes without an item)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // (wave-uniform)
  const int l32 = lane & 31, half = lane >> 5;

  const int n_bands = a.Nw / L;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int band = tile / a.n_ktiles;
  const int kt = tile - band * a.n_ktiles;  // 256-feature range
  const int b = band / n_bands;
  const int w0 = (band - b * n_bands) * L;
  const int n_cc = a.Nc / 16;
  const int nt = a.Nk - kt * 256 > TKT ? 2 : 1;  // tiles of 128 features in the range
  const int n_gc = nt * n_cc;                    // chunks the workgroup walks

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_q(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t ker_rsrc = rsrc_q(Ker, (int64_t)a.Nk * a.Nc * RS * 2);
  const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_q(Out, a.out_total * (int64_t)sizeof(TO));

  // ---- In items and layout: as conv_srows (slot rotation swz below).  An
  // item is (g, slab row j, 8-column block b8, channel half hc): four 16-byte
  // loads (channels 8g + 4hc + 0..3 of the chunk); lanes past the last item
  // load a duplicate and write it to the scratch area.
  const uint32_t in_last =
      __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, (uint32_t)((a.in_total - 1) * 2), 0, 0);
  int in_e[NIPT];    // element offset of the item's channel 8g + 4hc of chunk 0
  int in_lds[NIPT];  // LDS byte offset in buffer 0 of its first even column (+ 8 for hc = 1)
  int in_buf[NIPT];  // bytes from buffer 0 to buffer 1 (0 for scratch writes)
  int in_rot[NIPT];  // the block's slot rotation
  int last_c[NIPT];  // channel index (within the item, + 16 cc) of In's last element, or -1000
  int last_o[NIPT];  // its LDS byte offset from the item's channel-0 position
#pragma unroll
  for (int j = 0; j < NIPT; ++j) {
    const int t = tid + NT * j;
    const bool ok = t < NI;
    const int tt = ok ? t : NI - 1;
    const int hc = tt & 1, b8 = (tt >> 1) & 7, gj = tt >> 4;
    const int g = gj / SR, jr = gj - g * SR;
    const int x = 2 * w0 + jr;
    in_e[j] = (int)((int64_t)b * a.in_img) + (8 * g + 4 * hc) * a.nxny + x * a.Ny + 8 * b8;
    in_rot[j] = 2 * ((b8 >> 2) & 1) + (jr & 1);
    in_lds[j] = ok ? (int)((ibuf - kslot) * 16) + ((g * SR + jr) * 64 + 4 * b8) * 16 + 8 * hc
                   : SCRATCH_OFF + 16 * lane;
    in_buf[j] = ok ? IN_UNITS * 16 : 0;
    const int col = a.Ny - 1 - 8 * b8;
    const bool holds = ok && b == a.Nb - 1 && x == a.Nx - 1 && col >= 0 && col < 8;
    last_c[j] = holds ? a.Nc - 1 - 8 * g - 4 * hc : -1000;
    last_o[j] = ((col & 1) ? 16 * 32 : 0) + 16 * (((col >> 1) + in_rot[j]) & 3);
  }
  u32x4_t vin[NIPT][4];  // the In chunk the next stage 0 writes
  auto load_in_one = [&](int cc, int j, int k) __attribute__((always_inline)) {
    vin[j][k] = __builtin_bit_cast(
        u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                     in_rsrc, (uint32_t)((in_e[j] + (16 * cc + k) * a.nxny) * 2), 0, 0));
  };
  // Step i of item j: column pair i of its block, units 4 b8 + i (even
  // column) and 32 + 4 b8 + i (odd column), 8 bytes each, at their
  // swizzled slots.
  auto write_in_step = [&](int par, int j, int i) __attribute__((always_inline)) {
    char* p = smem + in_lds[j] + par * in_buf[j];
    const int slot = 16 * ((i + in_rot[j]) & 3);
    const u32x4_t* v = vin[j];
    const u32x2_t ev = {__builtin_amdgcn_perm(v[1][i], v[0][i], 0x05040100u),
                        __builtin_amdgcn_perm(v[3][i], v[2][i], 0x05040100u)};
    *reinterpret_cast<u32x2_t*>(p + slot) = ev;
    if (NS > 1) {
      const u32x2_t od = {__builtin_amdgcn_perm(v[1][i], v[0][i], 0x07060302u),
                          __builtin_amdgcn_perm(v[3][i], v[2][i], 0x07060302u)};
      *reinterpret_cast<u32x2_t*>(p + 16 * 32 + slot) = od;
    }
  };
  auto write_last = [&](int par, int cc, int j) __attribute__((always_inline)) {
    const int ch = last_c[j] - 16 * cc;  // 0..3 when this item holds the element
    const int off = (unsigned)ch < 4u ? in_lds[j] + par * in_buf[j] + last_o[j] + 2 * ch
                                      : SCRATCH_OFF + 2 * lane;
    *reinterpret_cast<uint16_t*>(smem + off) = (uint16_t)in_last;
  };
  // the second tile walks the chunks in reverse: its first chunks are the
  // ones the first tile read last, still in the L2
  auto cc_of = [&](int x) { return x < n_cc ? x : 2 * n_cc - 1 - x; };

  // ---- Ker: raw copies, read-back, repack.
  uint32_t raw_src[NDMA];  // byte offset of this thread's pieces, feature base 0, chunk 0
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int p = j * NT + tid;
    const int k = p / (2 * RS), q = p - k * 2 * RS;
    raw_src[j] = (uint32_t)(k * a.Nc * RS * 2 + 16 * q);
  }
  auto raw_base = [&](int x) {
    const int kb = kt * 256 + (x < n_cc ? 0 : TKT);
    return (uint32_t)((kb * a.Nc + 16 * cc_of(x)) * RS * 2);
  };
  auto copy_raw_one = [&](uint32_t base, int j) __attribute__((always_inline)) {
    dma16_q(ker_rsrc, raw + j * NT + 64 * wave, base + raw_src[j]);
  };
  u32x4_t run[RS];
  auto read_run_one = [&](int q) __attribute__((always_inline)) { run[q] = raw[tid * RS + q]; };
  const int pk = tid >> 1, pg = tid & 1;
  // Slot of stencil row R, tap s: unit (s, g, k) = channels 8g .. 8g+7 of
  // feature k at tap (R, s), from the run's elements (8g + i) * RS + R NS + s.
  auto pack_tap = [&](int R, int s_) __attribute__((always_inline)) {
    const int tap = R * NS + s_;
    u32x4_t v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e0 = (2 * i) * RS + tap, e1 = e0 + RS;
      const uint32_t sel =
          ((e0 & 1) ? 0x0302u : 0x0100u) | ((e1 & 1) ? 0x07060000u : 0x05040000u);
      v[i] = __builtin_amdgcn_perm(run[(e1 >> 1) >> 2][(e1 >> 1) & 3],
                                   run[(e0 >> 1) >> 2][(e0 >> 1) & 3], sel);
    }
    kslot[R * SLOT + (s_ * 2 + pg) * PST + pk] = v;
  };

  // ---- operands: A = Ker unit (s, half, feature 32 wave + l32) of a slot;
  // B = In unit of band row i for stencil row r, tap s (as conv_srows).
  auto swz = [](int u, int par) { return (u & ~3) | (((u & 3) + 2 * ((u >> 4) & 1) + par) & 3); };
  int a_sw[NS][2];
#pragma unroll
  for (int s_ = 0; s_ < NS; ++s_)
#pragma unroll
    for (int par = 0; par < 2; ++par)
      a_sw[s_][par] = swz(((s_ & 1) ? 32 + (s_ >> 1) : (s_ >> 1)) + l32, par);
  const int ka_off = half * PST + 32 * wave + l32;
  const int ib_off = half * SR * 64;
  auto read_ka = [&](int r, int s_) __attribute__((always_inline)) {
    return kslot[r * SLOT + s_ * 2 * PST + ka_off];
  };
  auto read_ib = [&](const u32x4_t* ib, int r, int s_, int i) __attribute__((always_inline)) {
    const int jr = 2 * i + r;
    return ib[ib_off + jr * 64 + a_sw[s_][jr & 1]];
  };

  f32x16_t acc[2][L];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int i = 0; i < L; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[t][i][e] = 0.f;

  // ---- Out: register j of (tile t, row i) is position l32 of output row
  // w0 + i, feature kt*256 + 128 t + 32 wave + 4 half + 8 (j/4) + j%4.  The
  // lane's part of the offset is one register; the rest (tile, row,
  // register) is wave-uniform and goes in the scalar offset.  Stores of
  // features past Nk or positions past Nh get an out-of-range lane offset.
  const int nhw = a.Nw * a.Nh;
  const uint32_t lane_off = (uint32_t)((4 * half * nhw + l32) * (int)sizeof(TO));
  const int feat_lane = kt * 256 + 32 * wave + 4 * half;  // + 128 t + 8 (j/4) + j%4
  const uint32_t lo = l32 < a.Nh ? lane_off : 0x80000000u;
  auto store_one = [&](const f32x16_t& v, int t, int i, int j) __attribute__((always_inline)) {
    // (b, first feature of the wave's block, row w0 + i): wave-uniform,
    // computed at the store (the empty asm keeps the compiler from hoisting
    // every row's and register's offset out of the loop into registers)
    uint32_t row_off = (uint32_t)(((((int64_t)b * a.Nk + kt * 256 + TKT * t + 32 * wave) * a.Nw +
                                    w0 + i) * a.Nh) * (int64_t)sizeof(TO));
    asm volatile("" : "+s"(row_off));
    const int dj = 8 * (j >> 2) + (j & 3);
    const uint32_t vo = dj < a.Nk - (feat_lane + TKT * t) ? lo : 0x80000000u;
    const uint32_t so = row_off + (uint32_t)(dj * nhw * (int)sizeof(TO));
    if constexpr (sizeof(TO) == 4)
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[j]), out_rsrc, vo, so, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(v[j]), out_rsrc, vo, so, 0);
  };

  u32x4_t KA[2], IB[2][L];
  // One stage (stencil row r of the chunk in ib) into accumulator set TL:
  // NS K-steps from operand parity P, whose step-0 operands are in
  // registers; each next step's operands -- in the last step, those of the
  // next stage (slot nr_, buffer nib) -- are read between the products.
  // mem(q) (q = 1 .. NQ, compile-time) issues the memory work placed after
  // product q.
  auto stage = [&](auto PC, auto TC, int r, const u32x4_t* ib, int nr_, const u32x4_t* nib,
                   auto mem) __attribute__((always_inline)) {
    constexpr int P = decltype(PC)::value;
    constexpr int TL = decltype(TC)::value;
    static_for<0, NS>([&](auto SC) {
      constexpr int st = decltype(SC)::value;
      constexpr int cu = (P + st) & 1, nx = cu ^ 1;
      static_for<0, L>([&](auto IC) {
        constexpr int i = decltype(IC)::value;
        acc[TL][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, KA[cu]), __builtin_bit_cast(bf16x8_t, IB[cu][i]),
            acc[TL][i], 0, 0, 0);
        if (i == 0) KA[nx] = st + 1 < NS ? read_ka(r, st + 1) : read_ka(nr_, 0);
        IB[nx][i] = st + 1 < NS ? read_ib(ib, r, st + 1, i) : read_ib(nib, nr_, 0, i);
        mem(std::integral_constant<int, st * L + i + 1>());
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  };
  // The pieces of a stage's memory work, numbered 0 .. W-1 in issue order,
  // go after products 1 + floor(w NQ / W): product q takes pieces
  // [ceil((q-1) W / NQ), ceil(q W / NQ)).
  auto spread = [&](auto QC, auto WC, auto piece) __attribute__((always_inline)) {
    constexpr int q = decltype(QC)::value, W = decltype(WC)::value;
    static_for<((q - 1) * W + NQ - 1) / NQ, (q * W + NQ - 1) / NQ>(piece);
  };

  // One chunk x into accumulator set TL; SROW >= 0: also store row SROW of
  // the first tile (acc[0][SROW]) during stages 1 and 2.
  auto chunk = [&](auto TC, auto SC, int x) __attribute__((always_inline)) {
    constexpr int SROW = decltype(SC)::value;
    constexpr int NST = SROW >= 0 ? NSH : 0;  // stores per stage (1 and 2)
    const int x1 = min(x + 1, n_gc - 1), x2 = min(x + 2, n_gc - 1);
    const int c1 = cc_of(x1), c2 = cc_of(x2);
    const int par = (x + 1) & 1;  // In buffer of chunk x + 1
    const u32x4_t* ib = ibuf + (x & 1) * IN_UNITS;
    const u32x4_t* ibn = ibuf + par * IN_UNITS;
    // stage 0: the three taps of slot 2, then the item steps and
    // last-element writes of In(x+1) (5 per item), late in the stage (their
    // registers were loaded in the previous chunk's stage 1)
    stage(std::integral_constant<int, 0>(), TC, 0, ib, 1, ib, [&](auto QC) __attribute__((always_inline)) {
      spread(QC, std::integral_constant<int, 5 * NIPT + NS>(), [&](auto WC) __attribute__((always_inline)) {
        constexpr int w = decltype(WC)::value;
        if constexpr (w < NS) {
          pack_tap(2, w);
        } else {
          constexpr int v = w - NS;
          if constexpr (v % 5 < 4) write_in_step(par, v / 5, v % 5);
          else write_last(par, c1, v / 5);
        }
      });
    });
    // raw(x+1), copied during the previous chunk's stage 2, has landed.
    // (The copies into LDS are not counted in issue order with loads into
    // registers: waiting for fewer than all would not cover them.)
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    // stage 1: In(x+2) loads, raw(x+1) read-backs and stores 0 .. NST-1 in
    // turn (the loads first: they have until the next chunk's stage 0);
    // then the taps of slot 0 for (x+1, 0)
    stage(std::integral_constant<int, (NS & 1)>(), TC, 1, ib, 2, ib, [&](auto QC) __attribute__((always_inline)) {
      constexpr int NL = 4 * NIPT;        // In loads
      static_assert(NL <= RS && (NST == 0 || NST == NL), "stage-1 groups");
      constexpr int G = NST > 0 ? 3 : 2;  // group g: load g, read-back g (, store g)
      spread(QC, std::integral_constant<int, RS + NL + NST + NS>(), [&](auto WC) __attribute__((always_inline)) {
        constexpr int w = decltype(WC)::value;
        if constexpr (w < G * NL) {
          constexpr int g = w / G, e = w % G;
          if constexpr (e == 0) load_in_one(c2, g / 4, g % 4);
          else if constexpr (e == 1) read_run_one(g);
          else store_one(acc[0][SROW < 0 ? 0 : SROW], 0, SROW, g);
        } else if constexpr (w < G * NL + RS - NL) {
          read_run_one(NL + w - G * NL);
        } else {
          pack_tap(0, w - G * NL - (RS - NL));
        }
      });
    });
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    // stage 2: raw(x+2) copies interleaved with stores NST .. 2 NST-1, then
    // the taps of slot 1 for (x+1, 1)
    const uint32_t rb = raw_base(x2);
    stage(std::integral_constant<int, ((2 * NS) & 1)>(), TC, 2, ib, 0, ibn, [&](auto QC) __attribute__((always_inline)) {
      spread(QC, std::integral_constant<int, NDMA + NST + NS>(), [&](auto WC) __attribute__((always_inline)) {
        constexpr int w = decltype(WC)::value;
        if constexpr (w < 2 * NST) {
          if constexpr (w % 2 == 0) copy_raw_one(rb, w / 2);
          else store_one(acc[0][SROW < 0 ? 0 : SROW], 0, SROW, NST + w / 2);
        } else if constexpr (w < NDMA + NST) {
          copy_raw_one(rb, w - NST);
        } else {
          pack_tap(1, w - NDMA - NST);
        }
      });
    });
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if constexpr (((NR * NS) & 1) != 0) {
      // a chunk has an odd number of K-steps: the next chunk's first
      // operands were read into parity 1
      KA[0] = KA[1];
#pragma unroll
      for (int i = 0; i < L; ++i) IB[0][i] = IB[1][i];
    }
  };

  // ---- prologue: In(0) and raw(0) in, slots 0 and 1 packed, In(1) loads
  // and raw(1) copies in flight.
  {
#pragma unroll
    for (int j = 0; j < NIPT; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) load_in_one(0, j, k);
    const uint32_t rb0 = raw_base(0);
#pragma unroll
    for (int j = 0; j < NDMA; ++j) copy_raw_one(rb0, j);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
    for (int j = 0; j < NIPT; ++j) {
#pragma unroll
      for (int i = 0; i < 4; ++i) write_in_step(0, j, i);
      write_last(0, 0, j);
    }
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
    for (int q = 0; q < RS; ++q) read_run_one(q);
#pragma unroll
    for (int s_ = 0; s_ < NS; ++s_) pack_tap(0, s_);
#pragma unroll
    for (int s_ = 0; s_ < NS; ++s_) pack_tap(1, s_);
    const int c1 = cc_of(min(1, n_gc - 1));
#pragma unroll
    for (int j = 0; j < NIPT; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) load_in_one(c1, j, k);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    const uint32_t rb1 = raw_base(min(1, n_gc - 1));
#pragma unroll
    for (int j = 0; j < NDMA; ++j) copy_raw_one(rb1, j);
    KA[0] = read_ka(0, 0);
#pragma unroll
    for (int i = 0; i < L; ++i) IB[0][i] = read_ib(ibuf, 0, 0, i);
  }

  using NOSTORE = std::integral_constant<int, -1>;
  for (int x = 0; x < n_cc; ++x) chunk(std::integral_constant<int, 0>(), NOSTORE(), x);
  if (nt == 2) {
    // the second tile: its first L chunks store the first tile's rows
    // (Nc >= 16 L), the rest store nothing
    static_for<0, L>([&](auto JC) {
      chunk(std::integral_constant<int, 1>(), JC, n_cc + decltype(JC)::value);
    });
    for (int x = n_cc + L; x < n_gc; ++x) chunk(std::integral_constant<int, 1>(), NOSTORE(), x);
    // ---- epilogue: the second tile's rows
#pragma unroll
    for (int i = 0; i < L; ++i)
#pragma unroll
      for (int j = 0; j < NSTO; ++j) store_one(acc[1][i], 1, i, j);
  } else {
#pragma unroll
    for (int i = 0; i < L; ++i)
#pragma unroll
      for (int j = 0; j < NSTO; ++j) store_one(acc[0][i], 0, i, j);
  }
}

// ---- register-Ker form ---------------------------------------------------------
// conv_srows3: the same bands, In staging and operand layout as conv_srows,
// with Ker's B operands loaded from the packed image (the workspace, read
// through the L2) straight into registers instead of through LDS.  Every
// global access is then a load into registers or a store: no copy into LDS
// has to be waited for, so no stage ends on a wait for vector memory, and
// the In loads of a chunk, issued a whole chunk before their rows are
// written into LDS, stay in flight across stage boundaries.  LDS holds only
// the two In buffers.
// * Waves: four, one per SIMD; wave w takes features 64w .. 64w+63 (two
//   32-feature blocks) for all L rows of the band, accumulators in AGPRs.
// * Ker: stencil row r's three B-operand units of a block (one per tap, 16
//   bytes per lane, a wave's load of one unit reads 512 contiguous bytes
//   per channel group) live in register set r; after the products of tap s
//   of (chunk, r), the set's tap-s units are reloaded for (chunk + 1, r),
//   three stages ahead.
// * In: the next chunk's rows are written item by item in stages 0 (item
//   0) and 1 (item 1); each item's loads for the chunk after follow its
//   writes.  Barriers after stage 1 (the next chunk's rows are complete)
//   and after stage 2 (this chunk's rows are no longer read).
template <typename TO, int NR, int NS, int L>
__global__ __launch_bounds__(256) void conv_srows3(const bf16_t* __restrict__ In,
                                                   const u32x4_t* __restrict__ Kp,
                                                   TO* __restrict__ Out, ConvArgs a,
                                                   int blk_vecs) {
  constexpr int NT = 256;
  constexpr int TK = 256;
  constexpr int SR = 2 * (L - 1) + NR;      // slab rows held per chunk
  constexpr int NI = 2 * SR * 8 * 2;        // In items per chunk
  constexpr int NIPT = (NI + NT - 1) / NT;  // items per thread
  constexpr int IN_UNITS = 2 * SR * 64;     // 16-byte units per In buffer
  constexpr int KER_UNITS = NS * 2 * TK;    // units of one stencil row's slice
  constexpr int NQ = NS * L;                // product pairs per wave per stage
  constexpr int SCRATCH_OFF = 2 * IN_UNITS * 16;  // bytes
  static_assert(NR == 3 && NS <= 3, "one register set per stencil row, taps within one 64-unit row");
  static_assert(NIPT == 2, "two In items per thread: one written in stage 0, one in stage 1");
  static_assert(L >= 1 && L <= 7, "rows per band");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* ibuf = reinterpret_cast<u32x4_t*>(smem);  // [2][2][SR][64]
  // (then a 2 KiB scratch area: writes of lanes without an item)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // (wave-uniform)
  const int l32 = lane & 31, half = lane >> 5;

  const int n_bands = a.Nw / L;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int band = tile / a.n_ktiles;
  const int kt = tile - band * a.n_ktiles;
  const int b = band / n_bands;
  const int w0 = (band - b * n_bands) * L;
  const int k0 = kt * TK;
  const int n_cc = a.Nc / 16;

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_q(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t kp_rsrc =
      rsrc_q(Kp, (int64_t)a.n_ktiles * n_cc * blk_vecs * 16);
  const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_q(Out, a.out_total * (int64_t)sizeof(TO));

  // ---- In items and layout: as conv_srows2 (lanes past the last item load
  // a duplicate and write it to the scratch area).
  const uint32_t in_last =
      __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, (uint32_t)((a.in_total - 1) * 2), 0, 0);
  int in_e[NIPT];    // element offset of the item's channel 8g + 4hc of chunk 0
  int in_lds[NIPT];  // LDS byte offset in buffer 0 of its first even column (+ 8 for hc = 1)
  int in_buf[NIPT];  // bytes from buffer 0 to buffer 1 (0 for scratch writes)
  int in_rot[NIPT];  // the block's slot rotation
  int last_c[NIPT];  // channel index (within the item, + 16 cc) of In's last element, or -1000
  int last_o[NIPT];  // its LDS byte offset from the item's channel-0 position
#pragma unroll
  for (int j = 0; j < NIPT; ++j) {
    const int t = tid + NT * j;
    const bool ok = t < NI;
    const int tt = ok ? t : NI - 1;
    const int hc = tt & 1, b8 = (tt >> 1) & 7, gj = tt >> 4;
    const int g = gj / SR, jr = gj - g * SR;
    const int x = 2 * w0 + jr;
    in_e[j] = (int)((int64_t)b * a.in_img) + (8 * g + 4 * hc) * a.nxny + x * a.Ny + 8 * b8;
    in_rot[j] = 2 * ((b8 >> 2) & 1) + (jr & 1);
    in_lds[j] = ok ? ((g * SR + jr) * 64 + 4 * b8) * 16 + 8 * hc : SCRATCH_OFF + 16 * lane;
    in_buf[j] = ok ? IN_UNITS * 16 : 0;
    const int col = a.Ny - 1 - 8 * b8;
    const bool holds = ok && b == a.Nb - 1 && x == a.Nx - 1 && col >= 0 && col < 8;
    last_c[j] = holds ? a.Nc - 1 - 8 * g - 4 * hc : -1000;
    last_o[j] = ((col & 1) ? 16 * 32 : 0) + 16 * (((col >> 1) + in_rot[j]) & 3);
  }
  u32x4_t vin[NIPT][4];  // In rows of the chunk after the next, until written
  auto load_in_one = [&](int cc, int j, int k) __attribute__((always_inline)) {
    vin[j][k] = __builtin_bit_cast(
        u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(
                     in_rsrc, (uint32_t)((in_e[j] + (16 * cc + k) * a.nxny) * 2), 0, 0));
  };
  auto write_in_from = [&](const u32x4_t* v, int par, int j, int i) __attribute__((always_inline)) {
    char* p = smem + in_lds[j] + par * in_buf[j];
    const int slot = 16 * ((i + in_rot[j]) & 3);
    const u32x2_t ev = {__builtin_amdgcn_perm(v[1][i], v[0][i], 0x05040100u),
                        __builtin_amdgcn_perm(v[3][i], v[2][i], 0x05040100u)};
    *reinterpret_cast<u32x2_t*>(p + slot) = ev;
    if (NS > 1) {
      const u32x2_t od = {__builtin_amdgcn_perm(v[1][i], v[0][i], 0x07060302u),
                          __builtin_amdgcn_perm(v[3][i], v[2][i], 0x07060302u)};
      *reinterpret_cast<u32x2_t*>(p + 16 * 32 + slot) = od;
    }
  };
  auto write_in_step = [&](int par, int j, int i) __attribute__((always_inline)) {
    write_in_from(vin[j], par, j, i);
  };
  auto write_last = [&](int par, int cc, int j) __attribute__((always_inline)) {
    const int ch = last_c[j] - 16 * cc;  // 0..3 when this item holds the element
    const int off = (unsigned)ch < 4u ? in_lds[j] + par * in_buf[j] + last_o[j] + 2 * ch
                                      : SCRATCH_OFF + 2 * lane;
    *reinterpret_cast<uint16_t*>(smem + off) = (uint16_t)in_last;
  };

  // ---- operands: A = Ker unit (tap s, channel group half, feature
  // 64 wave + 32 nb + l32) from the packed image; B = In unit of band row i
  // for stencil row r, tap s (as conv_srows).
  auto swz = [](int u, int par) { return (u & ~3) | (((u & 3) + 2 * ((u >> 4) & 1) + par) & 3); };
  int a_sw[NS][2];
#pragma unroll
  for (int s_ = 0; s_ < NS; ++s_)
#pragma unroll
    for (int par = 0; par < 2; ++par)
      a_sw[s_][par] = swz(((s_ & 1) ? 32 + (s_ >> 1) : (s_ >> 1)) + l32, par);
  const int ib_off = half * SR * 64;
  auto read_ib = [&](const u32x4_t* ib, int r, int s_, int i) __attribute__((always_inline)) {
    const int jr = 2 * i + r;
    return ib[ib_off + jr * 64 + a_sw[s_][jr & 1]];
  };
  const uint32_t kb_lane = (uint32_t)((half * TK + 64 * wave + l32) * 16);
  auto load_k = [&](int cc, int r, int s_, int nb) __attribute__((always_inline)) {
    const uint32_t base = (uint32_t)(((kt * n_cc + cc) * blk_vecs + r * KER_UNITS + s_ * 2 * TK +
                                      32 * nb) * 16);
    return __builtin_bit_cast(u32x4_t,
                              __builtin_amdgcn_raw_buffer_load_b128(kp_rsrc, kb_lane, base, 0));
  };

  f32x16_t acc[L][2];
#pragma unroll
  for (int i = 0; i < L; ++i)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][nb][e] = 0.f;

  u32x4_t KB[NR][NS][2];  // B-operand units: set r = stencil row r of the current chunk
  u32x4_t IB[2][L];       // In operands of two consecutive K-steps
  // One stage (chunk cc, stencil row R, In buffer ib): NS K-steps from
  // operand parity P, whose step-0 In operands are in registers; each next
  // step's In operands -- in the last step, those of the next stage (row
  // nr_, buffer nib) -- are read between the products; after tap s's
  // products, set R's tap-s units are reloaded for chunk ccn.  mem(q)
  // (q = 1 .. NQ, compile-time) issues the memory work placed after
  // product pair q.
  auto stage = [&](auto PC, auto RC, const u32x4_t* ib, int nr_, const u32x4_t* nib, int ccn,
                   auto mem) __attribute__((always_inline)) {
    constexpr int P = decltype(PC)::value;
    constexpr int R = decltype(RC)::value;
    static_for<0, NS>([&](auto SC) {
      constexpr int st = decltype(SC)::value;
      constexpr int cu = (P + st) & 1, nx = cu ^ 1;
      static_for<0, L>([&](auto IC) {
        constexpr int i = decltype(IC)::value;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[i][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, KB[R][st][nb]), __builtin_bit_cast(bf16x8_t, IB[cu][i]),
              acc[i][nb], 0, 0, 0);
        IB[nx][i] = st + 1 < NS ? read_ib(ib, R, st + 1, i) : read_ib(nib, nr_, 0, i);
        mem(std::integral_constant<int, st * L + i + 1>());
        __builtin_amdgcn_sched_barrier(0);
      });
      KB[R][st][0] = load_k(ccn, R, st, 0);
      KB[R][st][1] = load_k(ccn, R, st, 1);
      __builtin_amdgcn_sched_barrier(0);
    });
  };
  // The pieces of a stage's memory work, numbered 0 .. W-1 in issue order,
  // go after product pairs 1 + floor(w NQ / W).
  auto spread = [&](auto QC, auto WC, auto piece) __attribute__((always_inline)) {
    constexpr int q = decltype(QC)::value, W = decltype(WC)::value;
    static_for<((q - 1) * W + NQ - 1) / NQ, (q * W + NQ - 1) / NQ>(piece);
  };
  // item j of In(c1) into buffer par (four steps and the last element),
  // then its loads of In(c2)
  auto in_piece = [&](int j, int w, int par, int c1, int c2) __attribute__((always_inline)) {
    if (w < 4) write_in_step(par, j, w);
    else if (w == 4) write_last(par, c1, j);
    else load_in_one(c2, j, w - 5);
  };

  // ---- prologue: In(0) written, In(1) loads in flight, the B operands of
  // chunk 0 loaded.  In(0) goes through registers of its own, so In(1)'s
  // loads are issued with it; stencil row 0's B loads go before In(1)'s and
  // the other rows' after, so the loop's first waits match its steady state.
  {
    u32x4_t v0[NIPT][4];
#pragma unroll
    for (int j = 0; j < NIPT; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        load_in_one(0, j, k);
        v0[j][k] = vin[j][k];
      }
#pragma unroll
    for (int s_ = 0; s_ < NS; ++s_)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) KB[0][s_][nb] = load_k(0, 0, s_, nb);
    const int c1 = min(1, n_cc - 1);
#pragma unroll
    for (int j = 0; j < NIPT; ++j)
#pragma unroll
      for (int k = 0; k < 4; ++k) load_in_one(c1, j, k);
#pragma unroll
    for (int r = 1; r < NR; ++r)
#pragma unroll
      for (int s_ = 0; s_ < NS; ++s_)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) KB[r][s_][nb] = load_k(0, r, s_, nb);
#pragma unroll
    for (int j = 0; j < NIPT; ++j) {
#pragma unroll
      for (int i = 0; i < 4; ++i) write_in_from(v0[j], 0, j, i);
      write_last(0, 0, j);
    }
  }
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
  for (int i = 0; i < L; ++i) IB[0][i] = read_ib(ibuf, 0, 0, i);

  for (int cc = 0; cc + 1 < n_cc; ++cc) {
    const int c1 = cc + 1, c2 = min(cc + 2, n_cc - 1);
    const int par = (cc + 1) & 1;  // In buffer of chunk cc + 1
    const u32x4_t* ib = ibuf + (cc & 1) * IN_UNITS;
    const u32x4_t* ibn = ibuf + par * IN_UNITS;
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    // stage 0: item 0 of In(cc+1), then its loads of In(cc+2)
    stage(std::integral_constant<int, 0>(), I0(), ib, 1, ib, c1, [&](auto QC) __attribute__((always_inline)) {
      spread(QC, std::integral_constant<int, 9>(), [&](auto WC) __attribute__((always_inline)) {
        in_piece(0, decltype(WC)::value, par, c1, c2);
      });
    });
    // stage 1: item 1
    stage(std::integral_constant<int, (NS & 1)>(), I1(), ib, 2, ib, c1, [&](auto QC) __attribute__((always_inline)) {
      spread(QC, std::integral_constant<int, 9>(), [&](auto WC) __attribute__((always_inline)) {
        in_piece(1, decltype(WC)::value, par, c1, c2);
      });
    });
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    // stage 2: the next chunk's first In operands come from its buffer
    stage(std::integral_constant<int, ((2 * NS) & 1)>(), I2(), ib, 0, ibn, c1, [&](auto QC) __attribute__((always_inline)) {
      (void)QC;
    });
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if constexpr (((NR * NS) & 1) != 0) {
#pragma unroll
      for (int i = 0; i < L; ++i) IB[0][i] = IB[1][i];
    }
  }

  // ---- the last chunk, band row by band row: all NR x NS taps of row i
  // (every stencil row's B operands are in registers, the chunk's In in its
  // buffer), then row i's Out, whose stores drain while the later rows are
  // multiplied.  Register j of block (i, nb) holds position l32 of output
  // row w0 + i, feature k0 + 64 wave + 32 nb + 8 (j/4) + 4 half + j%4.
  // Out byte offsets: this lane's part (feature k0 + 64 wave + 4 half, band
  // row 0, position l32) is formed once; a store adds the wave-uniform part
  // of its feature step f = 32 nb + 8 (j/4) + j%4 and band row i.  Lanes past
  // Nh or Nk store out of range (dropped).
  // valid feature steps of this lane: f < kl (none past Nh)
  const int kl = l32 < a.Nh ? a.Nk - (k0 + 64 * wave) - 4 * half : -1;
  const uint32_t vo_lane =
      (uint32_t)(((((int64_t)b * a.Nk + k0 + 64 * wave + 4 * half) * a.Nw + w0) * a.Nh + l32) *
                 (int64_t)sizeof(TO));
  const uint32_t hw_b = (uint32_t)(a.Nw * a.Nh * (int)sizeof(TO)), nh_b = (uint32_t)(a.Nh * (int)sizeof(TO));
  auto store_row = [&](int i, int q) __attribute__((always_inline)) {
    const int nb = q >> 4, j = q & 15;
    const int f = 32 * nb + 8 * (j >> 2) + (j & 3);
    const uint32_t vo = f < kl ? vo_lane + (uint32_t)f * hw_b + (uint32_t)i * nh_b : 0x80000000u;
    if constexpr (sizeof(TO) == 4)
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[i][nb][j]), out_rsrc, vo, 0, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(acc[i][nb][j]), out_rsrc, vo, 0, 0);
  };
  {
    constexpr int T = NR * NS;
    const u32x4_t* ib = ibuf + ((n_cc - 1) & 1) * IN_UNITS;
    u32x4_t AT[2][T];  // In operands of a band row's taps
#pragma unroll
    for (int t = 0; t < T; ++t) AT[0][t] = read_ib(ib, t / NS, t % NS, 0);
    static_for<0, L>([&](auto IC) {
      constexpr int i = decltype(IC)::value;
      static_for<0, T>([&](auto TC) {
        constexpr int t = decltype(TC)::value;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[i][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, KB[t / NS][t % NS][nb]),
              __builtin_bit_cast(bf16x8_t, AT[i & 1][t]), acc[i][nb], 0, 0, 0);
        if constexpr (i + 1 < L) AT[(i + 1) & 1][t] = read_ib(ib, t / NS, t % NS, i + 1);
        if constexpr (i > 0) {
          // row i-1's 32 stores, spread over row i's T steps
          static_for<(t * 32 + T - 1) / T, ((t + 1) * 32 + T - 1) / T>([&](auto QC) {
            store_row(i - 1, decltype(QC)::value);
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    });
#pragma unroll
    for (int q = 0; q < 32; ++q) store_row(L - 1, q);
  }
}

// ---- Ker repack --------------------------------------------------------------
// Slice image of every (k tile, 16-channel chunk): unit
// ((kt*n_cc + cc)*blk_vecs + (tap*2 + g)*TK + kk) holds channels
// 16cc + 8g .. +7 of feature kt*TK + kk at tap (zero for features past Nk),
// so the stage of stencil row r copies units r*NS*2*TK .. +NS*2*TK of its
// block.  One thread per (k tile, chunk, g, kk): its feature's 8 channels x
// RS taps are one 16-byte-aligned run of RS 16-byte blocks, transposed in
// registers (v_perm) into RS units.
template <int RS>
__global__ __launch_bounds__(64) void pack_ker_srows(const bf16_t* __restrict__ Ker,
                                                      u32x4_t* __restrict__ P, ConvArgs a,
                                                      int blk_vecs) {
  constexpr int TK = 256;
  const int n_cc = a.Nc / 16;
  const int t = blockIdx.x * 64 + threadIdx.x;
  if (t >= a.n_ktiles * n_cc * 2 * TK) return;
  const int kk = t % TK, g = (t / TK) & 1, blk = t / (2 * TK);
  const int kt = blk / n_cc, cc = blk - kt * n_cc;
  const int k = kt * TK + kk;
  const bool ok = k < a.Nk;
  u32x4_t run[RS];
  const u32x4_t* src =
      reinterpret_cast<const u32x4_t*>(Ker + ((int64_t)(ok ? k : 0) * a.Nc + 16 * cc + 8 * g) * RS);
#pragma unroll
  for (int q = 0; q < RS; ++q) run[q] = src[q];
  u32x4_t* dst = P + (int64_t)blk * blk_vecs + g * TK + kk;
#pragma unroll
  for (int tap = 0; tap < RS; ++tap) {
    u32x4_t v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e0 = (2 * i) * RS + tap, e1 = e0 + RS;
      const uint32_t sel =
          ((e0 & 1) ? 0x0302u : 0x0100u) | ((e1 & 1) ? 0x07060000u : 0x05040000u);
      const uint32_t w1 = run[(e1 >> 1) >> 2][(e1 >> 1) & 3];
      const uint32_t w0 = run[(e0 >> 1) >> 2][(e0 >> 1) & 3];
      v[i] = ok ? __builtin_amdgcn_perm(w1, w0, sel) : 0u;
    }
    dst[tap * 2 * TK] = v;
  }
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, NR, NS, L, waves, form): tk = 256, tc = 16, bands of L output
// rows; form 1 = conv_srows (Ker repacked into a workspace by a second
// kernel, copied into LDS), form 2 = conv_srows2 (raw Ker, repacked on
// chip, no workspace), form 3 = conv_srows3 (the workspace's B operands
// loaded into registers).
// (Four waves -- one per feature pair, all L rows, accumulators in AGPRs --
// time the same as eight for conv_srows on the 3x3 stride-2 layer, so only
// eight are built of that form.)
#define CNN_SROWS_VARIANTS(X)             \
  X(1900, CNN_BF16, 3, 3, 7, 8, 1)        \
  X(1901, CNN_BF16, 3, 3, 4, 8, 1)        \
  X(2000, CNN_BF16_OBF16, 3, 3, 7, 8, 1)  \
  X(2001, CNN_BF16_OBF16, 3, 3, 4, 8, 1)  \
  X(2300, CNN_BF16, 3, 3, 7, 4, 3)        \
  X(2301, CNN_BF16, 3, 3, 4, 4, 3)        \
  X(2400, CNN_BF16_OBF16, 3, 3, 7, 4, 3)  \
  X(2401, CNN_BF16_OBF16, 3, 3, 4, 4, 3)  \
  X(2100, CNN_BF16, 3, 3, 7, 4, 2)        \
  X(2101, CNN_BF16, 3, 3, 4, 4, 2)        \
  X(2200, CNN_BF16_OBF16, 3, 3, 7, 4, 2)  \
  X(2201, CNN_BF16_OBF16, 3, 3, 4, 4, 2)

// acc: fp32 accumulators per lane (form 1, 8 waves: 2 RW - 1 blocks for
// odd L, else 2 RW; form 2, 4 waves: two sets of L blocks; 16 each)
static const VariantQ kVariantsQ[] = {
#define CNN_QV(id, dt, nr, ns, l, nw, form)                                            \
  {id, dt, 256, nr, ns, l, nw,                                                         \
   form == 2 ? 32 * l : (nw == 8 ? 32 * ((l + 1) / 2) - 16 * (l & 1) : 32 * l), form},
    CNN_SROWS_VARIANTS(CNN_QV)
#undef CNN_QV
};

const VariantQ* variants_srows(int* count) {
  *count = (int)(sizeof(kVariantsQ) / sizeof(kVariantsQ[0]));
  return kVariantsQ;
}

int64_t srows_slab_rows(const VariantQ& v) {
  return v.nr >= 2 ? 2 * (v.L - 1) + v.nr : v.L;
}

int64_t srows_lds_bytes(const VariantQ& v) {
  if (v.form == 3)  // two In buffers, scratch
    return 2 * 2 * srows_slab_rows(v) * 64 * 16 + 2048;
  if (v.form == 2)  // stencil-row slots, the raw chunk, two In buffers, scratch
    return ((int64_t)v.nr * v.ns * 2 * (128 + 4) + 128 * 2 * v.nr * v.ns +
            2 * 2 * srows_slab_rows(v) * 64) * 16 + 2048;
  return (4 * (int64_t)v.ns * 2 * v.tk + 2 * 2 * srows_slab_rows(v) * 64) * 16;
}

int64_t srows_blk_vecs(const VariantQ& v) {
  const int64_t n = (int64_t)v.nr * v.ns * 2 * v.tk;
  return (n + 255) / 256 * 256;
}

int64_t srows_ws_bytes(const VariantQ& v, const cnn_problem& p) {
  if (v.form == 2) return 0;
  return ((p.Nk + v.tk - 1) / v.tk) * (p.Nc / 16) * srows_blk_vecs(v) * 16;
}

bool srows_fits(const VariantQ& v, const cnn_problem& p) {
  const int64_t Ny = 2 * (p.Nh - 1) + p.Ns;
  // (the raw-Ker form stores the first tile's L rows during the second
  // tile's first L chunks: Nc >= 16 L)
  return p.sw == 2 && p.sh == 2 && p.Nr == v.nr && p.Ns == v.ns && p.Nc % 16 == 0 &&
         p.Nh <= 32 && Ny <= 64 && p.Nw % v.L == 0 && (v.form != 2 || p.Nc >= 16 * v.L);
}

template <int DT, int NR, int NS, int L, int NWV, int FORM>
static hipError_t launch_q(const void* In, const void* Ker, void* Out, void* ws, const ConvArgs& a,
                           int64_t lds, hipStream_t stream, const VariantQ& v) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  if constexpr (FORM == 2) {
    (void)ws;
    (void)v;
    auto kern = conv_srows2<TO, NR, NS, L>;
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(256), (unsigned)lds, stream,
                       (const bf16_t*)In, (const bf16_t*)Ker, (TO*)Out, a);
    return hipGetLastError();
  } else if constexpr (FORM == 3) {
    const int blk = (int)srows_blk_vecs(v);
    const int64_t threads = (int64_t)a.n_ktiles * (a.Nc / 16) * 2 * 256;
    hipLaunchKernelGGL(pack_ker_srows<NR * NS>, dim3((unsigned)((threads + 63) / 64)), dim3(64),
                       0, stream, (const bf16_t*)Ker, (u32x4_t*)ws, a, blk);
    auto kern = conv_srows3<TO, NR, NS, L>;
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(256), (unsigned)lds, stream,
                       (const bf16_t*)In, (const u32x4_t*)ws, (TO*)Out, a, blk);
    return hipGetLastError();
  } else {
    const int blk = (int)srows_blk_vecs(v);
    const int64_t threads = (int64_t)a.n_ktiles * (a.Nc / 16) * 2 * 256;
    hipLaunchKernelGGL(pack_ker_srows<NR * NS>, dim3((unsigned)((threads + 63) / 64)), dim3(64),
                       0, stream, (const bf16_t*)Ker, (u32x4_t*)ws, a, blk);
    auto kern = conv_srows<TO, NR, NS, L, NWV>;
    {
      const hipError_t e = allow_max_lds((const void*)kern);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(64 * NWV), (unsigned)lds, stream,
                       (const bf16_t*)In, (const u32x4_t*)ws, (TO*)Out, a, blk);
    return hipGetLastError();
  }
}

hipError_t launch_srows(const VariantQ& v, const void* In, const void* Ker, void* Out, void* ws,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASEQ(id, dt, nr, ns, l, nw, form) \
  case id:                                    \
    return launch_q<dt, nr, ns, l, nw, form>(In, Ker, Out, ws, a, lds_bytes, stream, v);
    CNN_SROWS_VARIANTS(CNN_CASEQ)
#undef CNN_CASEQ
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

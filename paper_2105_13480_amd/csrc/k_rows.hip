// Row-streaming convolution: Ker-stationary, stride 1 (bf16 MFMA, gfx950).
//
// One workgroup per tile of the flattened output index, the tile being L
// whole output rows of one image (a band) by tk = 64 output features, all
// Nc input features at once (Listing 3 with W_c = N_c and the Ker tile
// resident).  The whole Ker tile is packed into LDS once, in MFMA operand
// order; input rows then stream through a ring of LDS row buffers.  The
// band is walked in groups of WR output rows (one per wave pair): while a
// group is multiplied, the rows the next group adds are loaded, and the
// group's Out rows are stored as soon as they are complete, so the stores
// of one group drain under the next.
//
// The product is D[position][feature] = In-row x Ker (A = In, B = Ker):
// * In operands come straight from the natural row layout [c][position]
//   by the transposing LDS read (ds_read_b64_tr_b16): in each 16-lane
//   group, lane 4v+q supplies the 8-byte chunk (channel v, positions
//   4q..4q+3) and lane j receives position j of the four channels.  No
//   transpose pass, no per-element gathers.
// * The horizontal taps s are not applied by shifting the reads (chunks
//   must stay 8-byte aligned): tap s accumulates into its own accumulator
//   at the unshifted input position p, and Out[h] = sum_s acc_s[h + s] is
//   formed once per row.  In a 32x32 D block, lane l holds positions
//   8g + 4*(l/32) + i (register 4g + i), so h + s is either a register of
//   the same lane or of the partner lane l ^ 32 (one ds_bpermute).
//   Positions past the input row are padding: they only feed acc_s at
//   positions >= Ny, which no stored output reads.
// * Stores: each lane holds 4 consecutive outputs of one feature, written
//   as one 16-byte (fp32) or 8-byte (bf16) store.
#include <type_traits>

#include "internal.h"
#include "common.h"

namespace cnnlib {

namespace {

typedef short s16x4_t __attribute__((ext_vector_type(4)));
#define LDS_PTR_R(T, p) ((__attribute__((address_space(3))) T*)(p))

__device__ __forceinline__ u32x2_t read_tr16(const bf16_t* p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(
      u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR_R(s16x4_t, const_cast<bf16_t*>(p))));
#else
  (void)p;
  return u32x2_t{0u, 0u};
#endif
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_r(const void* base, int64_t bytes) {
  bytes = (bytes + 3) & ~(int64_t)3;
  const int32_t n = bytes > 0x7ffffffcLL ? 0x7ffffffc : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// 16-byte buffer -> LDS copy: lane i's 16 bytes land at lds + 16 i (lds
// wave-uniform); out-of-range reads give zeros.
__device__ __forceinline__ void dma16_r(__amdgpu_buffer_rsrc_t r, void* lds, uint32_t voff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, LDS_PTR_R(void, lds), 16, voff, 0, 0, 0);
#else
  (void)r;
  (void)lds;
  (void)voff;
#endif
}

// Wait for this wave's LDS operations, then s_barrier; outstanding global
// loads and stores are not waited for.
__device__ __forceinline__ void lds_barrier_r() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace

// TO: Out element type.  NR x NS: stencil.  WAVES: waves per workgroup, in
// pairs; the two waves of a pair take 32 features each and the same RPW
// output rows, so a group is WR = RPW * WAVES/2 output rows.  MB:
// 32-position blocks per row (Ny <= 32*MB).  NCG: 16-channel groups (Nc
// rounded up to 16 is 16*NCG, the tail zero).  VEC (Nh % 4 == 0): a group's
// Out rows are written as 16-byte (8-byte) chunks spread over the next
// group's products; otherwise element by element at the end of the group.
template <typename TO, int NR, int NS, int WAVES, int RPW, int MB, int NCG, bool VEC>
__global__ __launch_bounds__(64 * WAVES) void conv_rows(const bf16_t* __restrict__ In,
                                                       const bf16_t* __restrict__ Ker,
                                                       TO* __restrict__ Out, ConvArgs a, int L,
                                                       int n_bands) {
  constexpr int NT = 64 * WAVES;
  constexpr int WR = RPW * WAVES / 2;
  constexpr int TK = 64;
  constexpr int RS = NR * NS;
  constexpr int RSTR = 32 * MB;        // row buffer: positions per channel
  constexpr int BPC = RSTR / 8;        // 16-byte blocks per channel row
  constexpr int NRING = 2 * WR + NR - 1;
  constexpr int ncp = 16 * NCG;
  constexpr int row_elems = ncp * RSTR;
  constexpr int row_blocks = ncp * BPC;
  constexpr int NLD = (WR * row_blocks + NT - 1) / NT;             // blocks per thread per group
  constexpr int NINIT = ((WR + NR - 1) * row_blocks + NT - 1) / NT;  // first group's
  constexpr int NTRIP = NCG * 2 * TK;                               // Ker (group, half, feature)
  constexpr int KPT = (NTRIP + NT - 1) / NT;
  constexpr int NQ = RPW + NR - 1;     // input rows a wave reads per group
  // RAWST: the ring holds the raw Ker tile (all copies of whole 16-byte
  // chunks), so the set-up copies it there with buffer->LDS DMA and repacks
  // it from LDS; B-operand planes then get 2 units of padding (PST) so the
  // repack's writes spread over the banks.
  constexpr int KCH = (TK * ncp * RS / 8 + NT - 1) / NT;  // DMA copies per thread (at most)
  constexpr bool RAWST = NRING * row_elems * 2 >= KCH * NT * 16;
  constexpr int PST = RAWST ? TK + 2 : TK;  // B-operand plane stride (units)
  static_assert(NS <= 4, "a tap shift crosses at most into the partner lane");
  static_assert(WAVES % 2 == 0, "waves come in feature pairs");

  extern __shared__ __attribute__((aligned(16))) char smem[];
  u32x4_t* kbuf = reinterpret_cast<u32x4_t*>(smem);  // [NCG][RS][2][PST] B operands
  bf16_t* rows = reinterpret_cast<bf16_t*>(kbuf + NCG * RS * 2 * PST);  // [NRING][ncp][RSTR]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wp = wave >> 1, wk = wave & 1;
  const int l32 = lane & 31, half = lane >> 5;

  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int band = tile / a.n_ktiles;
  const int kt = tile - band * a.n_ktiles;
  const int b = band / n_bands;
  const int y0 = (band - b * n_bands) * L;
  const int y1 = min(y0 + L, a.Nw);
  const int Lb = y1 - y0;
  const int k0 = kt * TK;

  const __amdgpu_buffer_rsrc_t in_rsrc = rsrc_r(In, a.in_total * 2);
  const __amdgpu_buffer_rsrc_t ker_rsrc = rsrc_r(Ker, (int64_t)a.Nk * a.Nc * RS * 2);
  const __amdgpu_buffer_rsrc_t out_rsrc = rsrc_r(Out, a.out_total * (int64_t)sizeof(TO));
  const int64_t in_b = (int64_t)b * a.in_img;

  // Input row blocks: block f of rows [xa, ...) is (row xa + f / row_blocks,
  // channel, 16-byte block); channels past Nc are zero.  Rows start at any
  // element: the 16-byte loads are unaligned, the LDS rows aligned.  The
  // range check drops a whole dword that straddles the end of In; the only
  // element of In such a dword can hold is the last one, which is loaded
  // once and patched in.  Nothing touches a loaded block before it is
  // written to LDS (the fix-up code travels beside it), so every load of a
  // batch stays in flight.
  const uint32_t in_last =
      __builtin_amdgcn_raw_buffer_load_b16(in_rsrc, (uint32_t)((a.in_total - 1) * 2), 0, 0);
  // fix-up code: -2 zero block (channel past Nc), 0..7 In's last element at
  // that position, -1 as loaded
  auto load_block = [&](int xa, int f, int& fix) __attribute__((always_inline)) -> u32x4_t {
    const int rr = f / row_blocks;
    const int rem = f - rr * row_blocks;
    const int c = rem / BPC;
    const int blk = rem - c * BPC;
    const int x = xa + rr;
    const bool ok = c < a.Nc;
    const int64_t e = in_b + (int64_t)(ok ? c : 0) * a.nxny + (int64_t)x * a.Ny + 8 * blk;
    const int64_t d = a.in_total - 1 - e;
    fix = !ok ? -2 : (d >= 0 && d < 8) ? (int)d : -1;
    return __builtin_bit_cast(
        u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(in_rsrc, (uint32_t)(e * 2), 0, 0));
  };
  // Write a block to its ring slot: zeroing a channel past Nc is a mask;
  // the last-element patch is rare (one block of the whole tensor), so it
  // rewrites the block behind a branch.
  auto put_block = [&](u32x4_t* dst, u32x4_t v, int fix) __attribute__((always_inline)) {
    const uint32_t keep = fix == -2 ? 0u : ~0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] &= keep;
    *dst = v;
    if (fix >= 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t lo = fix == 2 * i ? ((v[i] & 0xffff0000u) | in_last) : v[i];
        v[i] = fix == 2 * i + 1 ? ((lo & 0xffffu) | (in_last << 16)) : lo;
      }
      *dst = v;
    }
  };
  auto store_block = [&](int xa, int f, u32x4_t v, int fix) __attribute__((always_inline)) {
    const int rr = f / row_blocks;
    const int rem = f - rr * row_blocks;
    const int slot = (xa + rr - y0) % NRING;
    put_block(reinterpret_cast<u32x4_t*>(rows + slot * row_elems) + rem, v, fix);
  };

  // Rows group gi adds beyond group gi-1's: [new_lo(gi), new_lo(gi) + new_n(gi)).
  const int n_groups = (Lb + WR - 1) / WR;
  auto new_lo = [&](int gi) { return y0 + min(gi * WR, Lb) + NR - 1; };
  auto new_n = [&](int gi) { return gi < n_groups ? min((gi + 1) * WR, Lb) - min(gi * WR, Lb) : 0; };
  u32x4_t pre[NLD];  // the next group's new rows, loaded a group ahead
  int fixp[NLD];

  // ---- set-up: the Ker tile and the first group's rows, all loads in
  // flight together.  Ker goes to LDS packed as B operands: vector
  // ((cg*RS + tap)*2 + g)*TK + kk holds channels 16cg + 8g .. +7 of feature
  // k0 + kk at tap (a feature's 8 channels x all taps are one 16-byte-aligned
  // run of RS 16-byte blocks).
  if constexpr (RAWST) {
    // The tile's raw rows Ker[k0 .. k0+63][Nc][RS] are one contiguous run
    // of 16-byte chunks: copied into the ring by DMA, one kilobyte per wave
    // instruction (features past Nk read as zeros).
    {
      char* raw = reinterpret_cast<char*>(rows);
      const int nch = TK * a.Nc * RS / 8;
      const uint32_t kbase = (uint32_t)(k0 * a.Nc * RS * 2);
      for (int q = 0; q * NT < nch; ++q)
        dma16_r(ker_rsrc, raw + (NT * q + 64 * wave) * 16, kbase + (uint32_t)(NT * q + tid) * 16u);
    }
    // the copies have landed in every wave; the first group's rows are
    // requested only then (a wait covering the copies would otherwise
    // cover them too: copies into LDS are not counted in issue order with
    // loads into registers), and arrive while the tile is repacked
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    const int nb0 = (min(WR, Lb) + NR - 1) * row_blocks;
    u32x4_t v0[NINIT];
    int fix0[NINIT];
#pragma unroll
    for (int j = 0; j < NINIT; ++j) v0[j] = load_block(y0, min(tid + NT * j, nb0 - 1), fix0[j]);
    // Repack: item (octet j, feature kk), j fastest, so a 16-lane group
    // reads 8 octets of 2 features (runs 144 bytes / a feature apart: distinct
    // banks) and writes 8 consecutive planes at 2 features (plane stride PST
    // = TK + 2: distinct banks).
    {
      const char* raw = reinterpret_cast<const char*>(rows);
      constexpr int NJ = 2 * NCG;  // 8-channel octets per feature
#pragma unroll
      for (int u = 0; u < KPT; ++u) {
        const int tr = tid + NT * u;
        if (tr >= NTRIP) continue;
        const int j = tr % NJ, kk = tr / NJ;
        const int c = 8 * j;
        const bool ok = c < a.Nc && k0 + kk < a.Nk;
        const u32x4_t* rp =
            reinterpret_cast<const u32x4_t*>(raw + (ok ? (kk * a.Nc + c) * RS * 2 : 0));
        u32x4_t run[RS];
#pragma unroll
        for (int q = 0; q < RS; ++q) run[q] = rp[q];
        const int dst = ((j >> 1) * RS * 2 + (j & 1)) * PST + kk;
#pragma unroll
        for (int tap = 0; tap < RS; ++tap) {
          u32x4_t v;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int e0 = (2 * i) * RS + tap, e1 = e0 + RS;
            const uint32_t sel = ((e0 & 1) ? 0x0302u : 0x0100u) |
                                 ((e1 & 1) ? 0x07060000u : 0x05040000u);
            const uint32_t w1 = run[(e1 >> 1) >> 2][(e1 >> 1) & 3];
            const uint32_t w0 = run[(e0 >> 1) >> 2][(e0 >> 1) & 3];
            v[i] = ok ? __builtin_amdgcn_perm(w1, w0, sel) : 0u;
          }
          kbuf[dst + tap * 2 * PST] = v;
        }
      }
    }
    // every wave is done with the raw tile before rows overwrite it
    lds_barrier_r();
#pragma unroll
    for (int j = 0; j < NINIT; ++j) {
      const int f = tid + NT * j;
      if (f < nb0) store_block(y0, f, v0[j], fix0[j]);
    }
  } else   {
    u32x4_t run[KPT][RS];
    bool ok[KPT];
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int tr = tid + NT * u;
      const int trc = tr < NTRIP ? tr : 0;
      const int kk = trc % TK;
      const int g = (trc / TK) & 1;
      const int cg = trc / (2 * TK);
      const int c = 16 * cg + 8 * g;
      ok[u] = tr < NTRIP && c < a.Nc && k0 + kk < a.Nk;
      const uint32_t off = ok[u] ? (uint32_t)(((k0 + kk) * a.Nc + c) * RS * 2) : 0u;
#pragma unroll
      for (int q = 0; q < RS; ++q)
        run[u][q] = __builtin_bit_cast(
            u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(ker_rsrc, off + 16 * q, 0, 0));
    }
    // (loads are unconditional -- clamped to a block of the set -- so all
    // stay in flight; only the LDS writes are guarded)
    const int nb0 = (min(WR, Lb) + NR - 1) * row_blocks;
    u32x4_t v0[NINIT];
    int fix0[NINIT];
#pragma unroll
    for (int j = 0; j < NINIT; ++j) v0[j] = load_block(y0, min(tid + NT * j, nb0 - 1), fix0[j]);
#pragma unroll
    for (int u = 0; u < KPT; ++u) {
      const int tr = tid + NT * u;
      if (tr < NTRIP) {
        const int kk = tr % TK;
        const int g = (tr / TK) & 1;
        const int cg = tr / (2 * TK);
        const int dst = (cg * RS * 2 + g) * TK + kk;
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
          kbuf[dst + tap * 2 * TK] = v;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NINIT; ++j) {
      const int f = tid + NT * j;
      if (f < nb0) store_block(y0, f, v0[j], fix0[j]);
    }
  }
  __syncthreads();
  // The second group's rows are requested only now, so that they do not
  // compete with the first group's for HBM; they are written to the ring in
  // the second half of the first group's steps.
#pragma unroll
  for (int j = 0; j < NLD; ++j)
    pre[j] = load_block(new_lo(1), max(0, min(tid + NT * j, new_n(1) * row_blocks - 1)), fixp[j]);

  // In operand lane offsets (elements within a 16-channel group of a row):
  // lane i of 16-lane group G supplies channel 8*(G/2) + i/4 (+4 for the
  // second read), positions 16*(G%2) + 4*(i%4).
  const int G = lane >> 4, li = lane & 15;
  const int aoff0 = (8 * (G >> 1) + (li >> 2)) * RSTR + 16 * (G & 1) + 4 * (li & 3);
  const int aoff1 = aoff0 + 4 * RSTR;
  const u32x4_t* kwave = kbuf + half * PST + wk * 32 + l32;

  const int n = k0 + wk * 32 + l32;  // this lane's output feature
  const bool nv = n < a.Nk;

  f32x16_t acc[RPW][NS][MB];

  // VEC: the previous group's Out rows, pending: chunk c of row j holds
  // positions 32*(c/4) + 8*(c%4) + 4*half .. +3 of feature n.  Every chunk is
  // always issued (invalid ones at an offset past the range check, which
  // drops them), so each group issues the same stores on every path.
  constexpr int NCHUNK = 4 * MB;
  constexpr int SOW = sizeof(TO) == 4 ? 16 : 8;  // pending words per block (fp32 or packed bf16)
  uint32_t so[RPW][MB][SOW];
  uint32_t s_orow[RPW];
  bool s_on[RPW];
#pragma unroll
  for (int j = 0; j < RPW; ++j) s_on[j] = false;
  auto store_chunk = [&](int j, int c) __attribute__((always_inline)) {
    const int mb = c / 4, g = c % 4;
    const int p0 = 32 * mb + 8 * g + 4 * half;
    const uint32_t vo =
        (s_on[j] && p0 < a.Nh) ? (s_orow[j] + p0) * (uint32_t)sizeof(TO) : 0x80000000u;
    if constexpr (sizeof(TO) == 4) {
      const u32x4_t v = {so[j][mb][4 * g], so[j][mb][4 * g + 1], so[j][mb][4 * g + 2],
                         so[j][mb][4 * g + 3]};
      __builtin_amdgcn_raw_buffer_store_b128(v, out_rsrc, vo, 0, 0);
    } else {
      const u32x2_t v = {so[j][mb][2 * g], so[j][mb][2 * g + 1]};
      __builtin_amdgcn_raw_buffer_store_b64(v, out_rsrc, vo, 0, 0);
    }
  };

  // A SIMD issues the MFMAs of its older wave first, so the second half of
  // the workgroup would finish each group's products last and alone; it
  // takes the higher issue priority during the products instead (measured
  // faster than equal priority and than alternating it step by step).
  const bool hiw = __builtin_amdgcn_readfirstlane(threadIdx.x) >= NT / 2;
  for (int gi = 0; gi < n_groups; ++gi) {

    // this wave's first output row, relative to y0; rows past the band are
    // computed too (from stale ring rows, in bounds) and not stored: every
    // wave runs the same straight-line code, so the waits count exactly (a
    // wave without a row shares its SIMD with one that has a row)
    const int yrel = gi * WR + wp * RPW;
    {
#pragma unroll
      for (int j = 0; j < RPW; ++j)
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[j][s][mb][e] = 0.f;

      // Step (cg, q): input row q of this wave (q = 0 .. RPW+NR-2) feeds
      // output row j through tap r = q - j: one In operand per position
      // block, the Ker operands of the taps it meets.  The operands of step
      // t+1 are read before the products of step t, and scheduling barriers
      // keep them there, so each product waits only for reads issued a whole
      // step earlier.
      constexpr int NSTEP = NCG * NQ;
      auto read_step = [&](int t, u32x4_t (&A)[MB], u32x4_t (&B)[NR][NS])
                           __attribute__((always_inline)) {
        const int cg = t / NQ, q = t % NQ;
        const bf16_t* rp = rows + ((yrel + q) % NRING) * row_elems + cg * 16 * RSTR;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const u32x2_t lo = read_tr16(rp + aoff0 + 32 * mb);
          const u32x2_t hi = read_tr16(rp + aoff1 + 32 * mb);
          A[mb] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
        }
        const u32x4_t* kp = kwave + cg * RS * 2 * PST;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          bool used = false;
#pragma unroll
          for (int j = 0; j < RPW; ++j) used |= (q - j == r);
          if (!used) continue;  // compile-time
#pragma unroll
          for (int s = 0; s < NS; ++s) B[r][s] = kp[(r * NS + s) * 2 * PST];
        }
      };
      auto multiply_step = [&](int t, const u32x4_t (&A)[MB], const u32x4_t (&B)[NR][NS])
                               __attribute__((always_inline)) {
        const int q = t % NQ;
#pragma unroll
        for (int j = 0; j < RPW; ++j) {
          const int r = q - j;
          if (r < 0 || r >= NR) continue;  // compile-time
#pragma unroll
          for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int mb = 0; mb < MB; ++mb)
              acc[j][s][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  __builtin_bit_cast(bf16x8_t, A[mb]), __builtin_bit_cast(bf16x8_t, B[r][s]),
                  acc[j][s][mb], 0, 0, 0);
        }
      };
      // (VEC: the previous group's chunks go out a few per step)
      constexpr int CPS = (RPW * NCHUNK + NSTEP - 1) / NSTEP;
      // The next group's rows (loaded a group ago) go to ring slots no wave
      // reads in this group, one block per step between the products of the
      // group's second half.
      const int nb_next = new_n(gi + 1) * row_blocks;
      u32x4_t A[2][MB], B[2][NR][NS];
      read_step(0, A[0], B[0]);
      if (hiw) __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int t = 0; t < NSTEP; ++t) {
        if (t + 1 < NSTEP) read_step(t + 1, A[(t + 1) & 1], B[(t + 1) & 1]);
        __builtin_amdgcn_sched_barrier(0);
        multiply_step(t, A[t & 1], B[t & 1]);
        if constexpr (VEC) {
#pragma unroll
          for (int k = 0; k < CPS; ++k) {
            const int c = t * CPS + k;
            if (c < RPW * NCHUNK) store_chunk(c / NCHUNK, c % NCHUNK);
          }
        }
#pragma unroll
        for (int j = 0; j < NLD; ++j) {
          if (NSTEP / 2 + (j * (NSTEP - NSTEP / 2)) / NLD != t) continue;  // compile-time
          const int f = tid + NT * j;
          if (f < nb_next) store_block(new_lo(gi + 1), f, pre[j], fixp[j]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      __builtin_amdgcn_s_setprio(0);
    }

    // Then the loads of the group after it are issued, before this group's
    // stores.  Every batch is issued and consumed whole, past the last group
    // too (clamped, in-range loads whose blocks are not written), so the
    // code is straight-line and each wait counts exactly the loads it needs.
#pragma unroll
    for (int j = 0; j < NLD; ++j)
      pre[j] = load_block(new_lo(gi + 2),
                          max(0, min(tid + NT * j, new_n(gi + 2) * row_blocks - 1)), fixp[j]);

#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      if constexpr (VEC) s_on[j] = false;
      if (yrel + j >= Lb) continue;  // wave-uniform
      // Out[h] = sum_s acc_s[h + s]; register 4g + i of block mb holds
      // position 32mb + 8g + 4*half + i.
      float o[MB][16];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int e = 0; e < 16; ++e) o[mb][e] = acc[j][0][mb][e];
#pragma unroll
      for (int s = 1; s < NS; ++s) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
#pragma unroll
            for (int i = 0; i + s < 4; ++i) o[mb][4 * g + i] += acc[j][s][mb][4 * g + i + s];
            // i + s >= 4: position 32mb + 8g + 4*half + i + s lies in the
            // partner half: half 0 takes register (mb, g, i') of lane l+32,
            // half 1 takes register (next 8-group, i') of lane l-32.  One
            // v_permlane32_swap of (mine, next) moves mine's upper half to
            // the lower lanes of its second result and next's lower half to
            // the upper lanes of its first.
#pragma unroll
            for (int ip = 0; ip < s; ++ip) {
              const int ng = g + 1 < 4 ? g + 1 : 0;
              const int nmb = g + 1 < 4 ? mb : mb + 1;
              const float mine = acc[j][s][mb][4 * g + ip];
              const float next = nmb < MB ? acc[j][s][nmb < MB ? nmb : 0][4 * ng + ip] : 0.f;
              const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mine),
                                                               __float_as_uint(next), false, false);
              o[mb][4 * g + ip + 4 - s] += __uint_as_float(half ? sw[0] : sw[1]);
            }
          }
        }
      }

      const int y = y0 + yrel + j;
      const uint32_t orow =
          (uint32_t)((((int64_t)b * a.Nk + (nv ? n : 0)) * a.Nw + y) * a.Nh);  // elements
      if constexpr (VEC) {
        s_on[j] = nv;
        s_orow[j] = orow;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int w = 0; w < SOW; ++w) {
            if constexpr (sizeof(TO) == 4)
              so[j][mb][w] = __float_as_uint(o[mb][w]);
            else
              so[j][mb][w] = (uint32_t)from_f32<bf16_t>(o[mb][2 * w]) |
                             ((uint32_t)from_f32<bf16_t>(o[mb][2 * w + 1]) << 16);
          }
        continue;  // written during the next group (or after the last)
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          if (32 * mb + 8 * g >= a.Nh) continue;  // wave-uniform
          const int p0 = 32 * mb + 8 * g + 4 * half;
          {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const uint32_t vo =
                  (nv && p0 + i < a.Nh) ? (orow + p0 + i) * (uint32_t)sizeof(TO) : 0x80000000u;
              if constexpr (sizeof(TO) == 4)
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(o[mb][4 * g + i]), out_rsrc,
                                                      vo, 0, 0);
              else
                __builtin_amdgcn_raw_buffer_store_b16(from_f32<bf16_t>(o[mb][4 * g + i]),
                                                      out_rsrc, vo, 0, 0);
            }
          }
        }
      }
    }
    lds_barrier_r();  // next group's rows written; every wave done with this group's
  }
  if constexpr (VEC) {
#pragma unroll
    for (int c = 0; c < RPW * NCHUNK; ++c) store_chunk(c / NCHUNK, c % NCHUNK);
  }
}

// ---- instantiation table ----------------------------------------------------
// (id, dtype, NR, NS, WAVES, RPW, MB, NCG): tk = 64, 64*WAVES threads,
// WR = RPW*WAVES/2 output rows per group.  Where several fit, the lowest id
// is taken: the 32-position rows come first.
#define CNN_ROWS_VARIANTS(X)                     \
  X(1500, CNN_BF16, 3, 3, 8, 1, 1, 4)            \
  X(1501, CNN_BF16, 3, 3, 8, 1, 1, 2)            \
  X(1502, CNN_BF16, 3, 3, 8, 1, 2, 4)            \
  X(1503, CNN_BF16, 3, 3, 8, 1, 2, 2)            \
  X(1504, CNN_BF16, 1, 1, 8, 1, 2, 4)            \
  X(1600, CNN_BF16_OBF16, 3, 3, 8, 1, 1, 4)      \
  X(1601, CNN_BF16_OBF16, 3, 3, 8, 1, 1, 2)      \
  X(1602, CNN_BF16_OBF16, 3, 3, 8, 1, 2, 4)      \
  X(1603, CNN_BF16_OBF16, 3, 3, 8, 1, 2, 2)      \
  X(1604, CNN_BF16_OBF16, 1, 1, 8, 1, 2, 4)

static const VariantR kVariantsR[] = {
#define CNN_ROWV(id, dt, nr, ns, waves, rpw, mb, ncg) \
  {id, dt, 64, nr, ns, rpw * waves / 2, mb, waves, ncg, 16 * mb * ns * rpw},
    CNN_ROWS_VARIANTS(CNN_ROWV)
#undef CNN_ROWV
};

const VariantR* variants_rows(int* count) {
  *count = (int)(sizeof(kVariantsR) / sizeof(kVariantsR[0]));
  return kVariantsR;
}

int64_t rows_ncp(const cnn_problem& p) { return (p.Nc + 15) / 16 * 16; }

int64_t rows_lds_bytes(const VariantR& v, const cnn_problem& p) {
  // (the kernel's NCG fixes ncp; RAWST and PST as in conv_rows)
  const int64_t ncp = 16 * v.ncg, nt = 64 * v.waves, rs = v.nr * v.ns;
  const int64_t ring = (2 * v.wr + v.nr - 1) * ncp * 32 * v.mb * 2;
  const int64_t kch = (v.tk * ncp * rs / 8 + nt - 1) / nt;
  const int64_t pst = ring >= kch * nt * 16 ? v.tk + 2 : v.tk;
  const int64_t ker = (ncp / 16) * rs * 2 * pst * 16;
  return ker + ring;
}

bool rows_fits(const VariantR& v, const cnn_problem& p) {
  if (v.nr != p.Nr || v.ns != p.Ns || p.sw != 1 || p.sh != 1 || p.Nc % 8 != 0) return false;
  if (rows_ncp(p) != 16 * v.ncg) return false;
  return p.Nh + p.Ns - 1 <= 32 * v.mb;
}

template <int DT, int NR, int NS, int WAVES, int RPW, int MB, int NCG>
static hipError_t launch_r(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                           int64_t lds, hipStream_t stream) {
  typedef typename std::conditional<DT == CNN_BF16, float, bf16_t>::type TO;
  // 16-byte Out chunks need rows of a multiple of 4 outputs
  auto kern = (a.Nh & 3) == 0 ? conv_rows<TO, NR, NS, WAVES, RPW, MB, NCG, true>
                              : conv_rows<TO, NR, NS, WAVES, RPW, MB, NCG, false>;
  {
    const hipError_t e = allow_max_lds((const void*)kern);
    if (e != hipSuccess) return e;
  }
  const int L = a.tp / a.Nh;
  const int n_bands = a.Nw / L;
  hipLaunchKernelGGL(kern, dim3((unsigned)a.grid), dim3(64 * WAVES), (unsigned)lds, stream,
                     (const bf16_t*)In, (const bf16_t*)Ker, (TO*)Out, a, L, n_bands);
  return hipGetLastError();
}

hipError_t launch_rows(const VariantR& v, const void* In, const void* Ker, void* Out,
                       const ConvArgs& a, int64_t lds_bytes, hipStream_t stream) {
  switch (v.id) {
#define CNN_CASER(id, dt, nr, ns, waves, rpw, mb, ncg) \
  case id:                                            \
    return launch_r<dt, nr, ns, waves, rpw, mb, ncg>(In, Ker, Out, a, lds_bytes, stream);
    CNN_ROWS_VARIANTS(CNN_CASER)
#undef CNN_CASER
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace cnnlib

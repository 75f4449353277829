/*
 * cnn.h -- C ABI of the MI355X (gfx950) CNN forward contraction library
 * (libcnn_mi355x.so).
 *
 * The operation (paper Sec. 1, the CNN equation; Listing 1 with strides):
 *
 *   Out[b][k][w][h] = sum_{c<Nc} sum_{r<Nr} sum_{s<Ns}
 *                       In[b][c][sw*w + r][sh*h + s] * Ker[k][c][r][s]
 *
 * b < Nb batch, k < Nk output feature, c < Nc input feature, w < Nw and
 * h < Nh output pixel, r < Nr and s < Ns stencil tap, sw / sh the strides
 * sigma_w / sigma_h.  It is a cross-correlation (no kernel flip) with no
 * padding ("valid"): In has exactly Nx = sw*(Nw-1)+Nr rows and
 * Ny = sh*(Nh-1)+Ns columns per channel.
 *
 * Layout: every tensor is dense and row-major in the index order above
 * (last index fastest): In[Nb][Nc][Nx][Ny], Ker[Nk][Nc][Nr][Ns],
 * Out[Nb][Nk][Nw][Nh].  No strides, no padding arguments.
 *
 * Ownership: the caller owns all three buffers, which are device pointers
 * on the current HIP device.  The library keeps no pointer after a call,
 * never writes In or Ker, and fully overwrites Out (its prior contents do
 * not matter; only the atomic-sum channel split reads it, after zeroing
 * it).  Out must not overlap In or Ker.
 *
 * Streams: every compute call is asynchronous on `stream` (a hipStream_t
 * passed as void*; NULL is the null stream).  There is no implicit
 * synchronisation; a kernel fault surfaces at the caller's next
 * synchronisation on that stream.
 *
 * Errors: every function returns a cnn_status (0 = success, negative =
 * error).  Arguments are validated before any HIP call, so an error return
 * guarantees nothing was launched.  cnn_last_error() returns a per-thread
 * message describing the most recent failure.  No C++ exception crosses
 * this interface.
 *
 * Thread safety: all functions are reentrant; calls may be made from several
 * host threads at once.
 */
#ifndef CNN_MI355X_H
#define CNN_MI355X_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CNN_ABI_VERSION 2

/* Element types of (In, Ker) -> Out.  Accumulation is always fp32. */
typedef enum cnn_dtype {
  CNN_F32 = 0,        /* In, Ker, Out float32                              */
  CNN_BF16 = 1,       /* In, Ker bfloat16; Out float32                     */
  CNN_BF16_OBF16 = 2  /* In, Ker bfloat16; Out bfloat16 (round to nearest even) */
} cnn_dtype;

typedef enum cnn_status {
  CNN_OK = 0,
  CNN_E_NULL = -1,         /* a required pointer argument is NULL                  */
  CNN_E_SHAPE = -2,        /* a size < 1 or a stride < 1                           */
  CNN_E_DTYPE = -3,        /* unknown dtype                                        */
  CNN_E_OVERFLOW = -4,     /* an element count does not fit the kernels' indexing  */
  CNN_E_ALIAS = -5,        /* Out overlaps In or Ker                               */
  CNN_E_UNSUPPORTED = -6,  /* requested kernel / tiling does not exist or does not fit */
  CNN_E_HIP = -7,          /* a HIP runtime call failed (see cnn_last_error)       */
  CNN_E_PLAN = -8          /* plan does not belong to this problem / dtype         */
} cnn_status;

/* Problem sizes in the paper's notation (Sec. 1). */
typedef struct cnn_problem {
  int64_t Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh;
} cnn_problem;

/* A box tiling (Listing 2): tile sizes of the b, k, c, w, h loops. */
typedef struct cnn_tiles {
  int64_t Tb, Tk, Tc, Tw, Th;
} cnn_tiles;

/* Kernel families. */
typedef enum cnn_kernel {
  CNN_K_AUTO = 0,     /* let cnn_plan choose                                          */
  CNN_K_DIRECT = 1,   /* one thread per output, fp32 FMA; any shape (correctness path)  */
  CNN_K_IGEMM = 2,    /* implicit GEMM on MFMA, LDS-staged halo'd In slab + Ker tile,
                         element-wise staging (any dtype; fallback of CNN_K_IGEMM_PIPE) */
  CNN_K_POINTWISE = 3,/* 1x1 stencils, any stride, bf16, Nc % 8 == 0: the inputs of the
                         tile's outputs gathered (no halo, no unused rows), 64 channels
                         per stage, raw Ker rows as in CNN_K_IGEMM_RAWK              */
  CNN_K_SMALLC = 4,   /* few input channels, wide stencils (Ns <= 8, ceil(Nc*Nr/2) <= 24),
                         bf16: K = flattened (c, r, s), the Ker image and the tile's
                         halo'd slab in LDS, workgroups walking runs of tiles; tc of
                         its plans is Nc; variants 1003 and 1103 have the 3-channel
                         7x7 stride-2 stencil compiled in                            */
  CNN_K_IGEMM_PIPE = 5,/* implicit GEMM, bf16: repacked Ker streamed by DMA, In staged
                         through registers, both double-buffered in LDS               */
  CNN_K_IGEMM_DMA = 6,/* implicit GEMM, bf16: Ker and the natural In rows both copied
                         by 16-byte DMA into a ring of LDS buffers, In transposed in LDS */
  CNN_K_IGEMM_WIDE = 7,/* implicit GEMM, bf16: In staged as 8x8 (position x channel)
                         blocks of 16-byte loads transposed in registers, swizzled LDS,
                         MFMA operands prefetched one K-step ahead                  */
  CNN_K_IGEMM_RAWK = 8,/* as CNN_K_IGEMM_PIPE for fixed 3x3 / 1x1 stencils, Nc % 8 == 0:
                         raw Ker rows copied by DMA, MFMA operands built in registers,
                         no repack and no workspace                                 */
                      /* 9: not used                                                  */
  CNN_K_ROWS = 10,    /* stride-1 row streaming, bf16: tiles are whole output rows
                         of one image (tp = L*Nh, L dividing Nw) by 64 features;
                         the Ker tile resident in LDS, input rows streamed through
                         a ring of row buffers and read with transposing LDS
                         reads; fixed 3x3 or 1x1, Nc % 8 == 0, Ny <= 64; tc of
                         its plans is Nc                                          */
  CNN_K_GEMM1 = 11,   /* 1x1 layers as a per-pixel GEMM, bf16: In channel rows
                         read by transposing LDS reads, Ker rows as they lie,
                         both double-buffered in LDS (or, for whole-image tiles
                         at stride 1, copied by DMA into a four-stage ring);
                         Nc % 8 == 0, tp a multiple of 4; strides 1 (Nw*Nh % 4
                         == 0) or 2 and 2 (Nh % 4 == 0: 4 output pixels = the
                         even half of 8 input columns)                         */
  CNN_K_SROWS = 12,   /* stride-2 layers over bands of whole output rows, bf16:
                         256 features x L rows per workgroup, In rows split by
                         column parity into MFMA-ready LDS units, one stencil
                         row of Ker per stage.  Three forms (cnn_variants):
                         Ker repacked per call into the workspace and copied
                         by DMA (8 waves, one tile of 256 features); the same
                         workspace read straight into the B-operand
                         registers (4 waves, one tile of 256 features, LDS
                         for In only); or raw Ker rows copied by DMA and
                         repacked in registers on chip, no workspace (4
                         waves, two tiles of 128 features in turn, the first
                         tile's Out written while the second computes); fixed
                         3x3, Nc % 16 == 0,
                         Nh <= 32, Ny <= 64, L | Nw; tp of its plans is L*Nh
                         (cnn_plan_tiles: tp = L*Nh, or 0 for any L)           */
  CNN_K_SPLITC = 13,  /* the paper's Case 2 (Sec. 2.1, W_c < N_c; the partial Outs
                         reduced at the end, Sec. 2.3) on one GPU: the
                         channel loop split over kc workgroup slices
                         (plan.kc); each slice writes fp32 partial sums to the
                         workspace, a second kernel adds the kc slices in slice
                         order and writes Out.  For shapes with few output
                         tiles and many channels.  Two kernels: the
                         CNN_K_IGEMM tiles (same tk/tp/tc and instantiations;
                         any dtype and stencil), and the channel-slice kernel
                         (tk 32, tp 64, tc 16/32/64 channels per stage, bf16,
                         3x3 or 1x1, Nc % 16 == 0), which issues a stage's
                         loads all at once.  Its atomic-sum instantiations
                         (cnn_variant_t.mode = 1; fp32 Out) need no
                         workspace: Out is zeroed, then every slice adds its
                         partial tile into Out with fp32 atomic adds, so the
                         summation order -- and the last bits of Out -- may
                         vary from call to call.  Its direct instantiations
                         (mode = 2; 3x3, either Out type; kc = 1) need none
                         either: one slice of 128-channel stages per
                         1024-thread workgroup writes Out in a fixed order */
  CNN_K_AUTO_NO_WORKSPACE = 14 /* (cnn_plan_tiles only) the model's choice among the
                         plans that need no workspace: the plan cnn_fwd runs
                         when no cnn_plan_find result is cached              */
} cnn_kernel;

/*
 * Machine budget the tile selector works against: the per-processor fast
 * memory M of Eq. (1), split into the two stores a CU really has.
 */
typedef struct cnn_budget {
  int64_t cus;          /* compute units (the paper's P processors)                 */
  int64_t lds_bytes;    /* LDS per CU (holds the In and Ker tiles)                  */
  int64_t acc_regs;     /* fp32 accumulator registers per lane for the Out tile     */
  int64_t wg_per_cu;    /* workgroups the selector plans to keep resident per CU    */
} cnn_budget;

/*
 * An execution plan.  Produced by cnn_plan (automatic choice) or
 * cnn_plan_tiles (a requested tiling); consumed by cnn_fwd_plan.
 *
 * Tiles: a workgroup computes tk output features for tp consecutive outputs
 * of the flattened (b, w, h) index (the paper's composite T_bhw), looping
 * over all Nc input features tc at a time (Listing 3 with W_c = N_c).
 */
typedef struct cnn_plan_t {
  cnn_problem prob;     /* problem the plan was made for                            */
  int32_t dtype;        /* cnn_dtype                                                */
  int32_t kernel;       /* cnn_kernel (never CNN_K_AUTO in a finished plan)         */
  int32_t variant;      /* internal kernel instantiation id                         */
  int32_t kc;           /* CNN_K_SPLITC: channel slices (the paper's P_c), 1 ..
                           ceil(Nc/tc); slice z takes channels [z*cs, z*cs + cs),
                           cs = ceil(ceil(Nc/tc)/kc)*tc; a caller may change it
                           and must then set ws_bytes = 4*kc*Nb*Nk*Nw*Nh (0
                           for the atomic-sum instantiations; the direct ones
                           take kc = 1 and no workspace only).
                           cnn_plan_tiles picks the smallest kc with no empty
                           slice that gives at least two workgroups per CU,
                           else ceil(Nc/tc).  0 for the other kernels.        */
  int64_t tk;           /* output features per workgroup (T_k)                      */
  int64_t tp;           /* outputs of the flattened (b,w,h) index per workgroup     */
  int64_t tc;           /* input features per LDS stage (T_c)                       */
  int64_t grid;         /* workgroups launched                                      */
  int64_t lds_bytes;    /* LDS per workgroup                                        */
  int64_t slab_rows;    /* max input rows a workgroup stages (halo included)        */
  int64_t ws_bytes;     /* device workspace the plan needs (repacked Ker, or the
                           fp32 partial Outs of CNN_K_SPLITC), which the caller
                           passes to cnn_fwd_plan_ws; 0 for most plans        */
  double eq1_elems[3];  /* Eq. (1) terms Out, Ker, In for this tiling (elements)    */
  double eq1_bytes;     /* the same, weighted by element size, summed               */
  double compulsory_bytes; /* |In read| + |Ker| + |Out|, each once                  */
  double flops;         /* 2 Nb Nk Nc Nr Ns Nw Nh                                   */
  double mfma_flops;    /* flops the workgroups' MFMA tiles issue (tile and
                           channel-stage padding included)                    */
  double hbm_bytes;     /* predicted HBM bytes: Eq. (3) at the XCD / L2 level
                           (cnn_hbm_bytes with 8 XCDs of 4 MiB L2)            */
  double model_us;      /* the selector's predicted kernel time (microseconds):
                           the slowest of the MFMA work, the Eq. (1) traffic
                           and the HBM traffic of the busiest CU's tiles, at
                           rates measured on MI355X, plus the family's fixed
                           costs (see cnn_plan)                               */
} cnn_plan_t;

/*
 * Out = conv(In, Ker) on `stream` (the CNN equation of Sec. 1, scheduled as
 * Listing 3 of Sec. 2).  Uses the plan cached for (problem, dtype, current
 * device): the fastest workspace-free plan of an earlier cnn_plan_find,
 * else cnn_plan's choice (computed on the first call and cached).  Only
 * plans that need no workspace are ever used here, so cnn_fwd allocates no
 * device memory, never synchronises, and may be captured into a HIP graph.
 * For layers with few outputs and many channels that plan may be the
 * atomic-sum channel split (CNN_K_SPLITC, fp32 Out), whose summation order
 * and hence last bits vary between calls; run a CNN_K_SPLITC plan with a
 * workspace (cnn_fwd_plan_ws) for a fixed order.
 * See the file header for layouts.  Errors: CNN_E_NULL, CNN_E_SHAPE,
 * CNN_E_DTYPE, CNN_E_OVERFLOW, CNN_E_ALIAS, CNN_E_HIP.
 */
int cnn_fwd(const void* In, const void* Ker, void* Out,
            int64_t Nb, int64_t Nc, int64_t Nk, int64_t Nw, int64_t Nh,
            int64_t Nr, int64_t Ns, int64_t sw, int64_t sh,
            int dtype, void* stream);

/*
 * Tile-size selection (Sec. 2, Eq. (1); Eq. (3) one level up).  Lists every
 * tiling the kernels implement whose footprint (LDS tiles and accumulators,
 * the two halves of the paper's fast memory M) fits the budget, prices each
 * with its MFMA work, its Eq. (1) bytes (slab form) per channel stage and
 * the two-level HBM bytes (Eq. (3) over the 8 XCDs, plan.hbm_bytes),
 * converts them into a time with per-family rates measured on MI355X
 * (plan.model_us), and returns the candidate of least time; candidates
 * within 2 % of it are ranked by fewer HBM bytes, then fewer Eq. (1) bytes,
 * then the lower instantiation id.  The choice may need a workspace
 * (plan.ws_bytes > 0: run it with cnn_fwd_plan_ws); cnn_fwd runs the best
 * candidate that needs none (cnn_plan_tiles with CNN_K_AUTO_NO_WORKSPACE,
 * or cnn_plan_lookup).  budget == NULL queries the current HIP device.
 * Writes *plan.  Errors: CNN_E_NULL, CNN_E_SHAPE, CNN_E_DTYPE,
 * CNN_E_OVERFLOW, CNN_E_HIP (device query failed).
 */
int cnn_plan(const cnn_problem* prob, int dtype, const cnn_budget* budget,
             cnn_plan_t* plan);

/*
 * The candidates cnn_plan ranks (and cnn_plan_find times), each a complete
 * plan with its model fields: writes min(*count, cap) of them to out (out
 * may be NULL when cap is 0) and sets *count to the number of candidates.
 * Errors: CNN_E_NULL (count NULL, or out NULL with cap > 0), as cnn_plan.
 */
int cnn_plan_candidates(const cnn_problem* prob, int dtype, const cnn_budget* budget,
                        cnn_plan_t* out, int cap, int* count);

/*
 * The kernel instantiations the library holds (its compile-time tilings),
 * for tests and tuning tools.  Writes min(*count, cap) entries to out (out
 * may be NULL when cap is 0); *count = how many exist.  Host only.
 * Errors: CNN_E_NULL.
 */
typedef struct cnn_variant_t {
  int32_t kernel;       /* cnn_kernel family                                      */
  int32_t variant;      /* instantiation id (cnn_plan_t.variant)                  */
  int32_t dtype;        /* cnn_dtype                                              */
  int32_t nr, ns;       /* compile-time stencil, 0 = any                          */
  int32_t mode;         /* CNN_K_GEMM1: 0 stride 1, 1 strides 2, 2 whole-image
                           DMA ring; CNN_K_SROWS: output rows per band;
                           CNN_K_ROWS: 32-position blocks per input row;
                           CNN_K_SPLITC: 1 for the atomic-sum and 2 for the
                           direct (both workspace-free) channel-slice
                           instantiations; else 0                        */
  int64_t tk;           /* output features per workgroup                          */
  int64_t tp;           /* largest tile of outputs, 0 where the problem sets it   */
  int64_t tc;           /* input channels per stage, 0 = all; CNN_K_ROWS: the
                           channel count rounded up to 16 it is built for       */
} cnn_variant_t;

int cnn_variants(cnn_variant_t* out, int cap, int* count);

/*
 * Empirical selection among the candidates of cnn_plan_candidates (every
 * tiling whose footprint fits the current device's budget): after about
 * 0.2 s of warm-up runs (clocks up from idle), runs each on the caller's
 * buffers on `stream`, times it with HIP events (one untimed run, then 3-20
 * timed runs; a candidate faster than 50 us a run is timed again as a
 * replay of those runs captured into a HIP graph on a private stream, so
 * that launch overhead does not rank short kernels), times the candidates
 * within 25 % of the fastest (at most six) again over three interleaved
 * rounds of 10-100 runs, and returns the one with the fastest round in
 * *plan (that round's mean time in *best_ms when best_ms is not NULL).  The winner may need a
 * workspace (plan->ws_bytes > 0, run it with cnn_fwd_plan_ws); the fastest
 * candidate that needs none is cached for (problem, dtype, device), so
 * later cnn_fwd calls use it.  Candidates that need a workspace are timed
 * with one this call allocates and frees before it returns (the only device
 * allocation the library makes).  In and Ker are only read; Out is
 * overwritten and on success holds the result of the returned plan.
 * Blocks until the timing runs finish; cannot be called while `stream` is
 * being captured (CNN_E_UNSUPPORTED).  Other errors as cnn_fwd.
 */
int cnn_plan_find(const void* In, const void* Ker, void* Out,
                  const cnn_problem* prob, int dtype, void* stream,
                  cnn_plan_t* plan, double* best_ms);

/*
 * The plan cnn_fwd would use for (prob, dtype) on the current device
 * (cached winner of cnn_plan_find, else cnn_plan's choice).  Errors:
 * CNN_E_NULL, CNN_E_SHAPE, CNN_E_DTYPE, CNN_E_OVERFLOW, CNN_E_HIP.
 */
int cnn_plan_lookup(const cnn_problem* prob, int dtype, cnn_plan_t* plan);

/*
 * Build the plan for a requested kernel family and tiling (tests, tuning).
 * kernel = CNN_K_DIRECT ignores tk/tp/tc.  Returns CNN_E_UNSUPPORTED when
 * no instantiation implements (kernel, tk, tp, tc) for this dtype or its
 * LDS footprint exceeds the budget.  budget == NULL queries the device.
 */
int cnn_plan_tiles(const cnn_problem* prob, int dtype, int kernel,
                   int64_t tk, int64_t tp, int64_t tc,
                   const cnn_budget* budget, cnn_plan_t* plan);

/*
 * Out = conv(In, Ker) with an explicit plan.  The plan's problem and dtype
 * must equal (*prob, dtype), and its tiling must be one the library makes
 * for that problem (geometry, LDS size and the byte ranges its kernel
 * addresses), else CNN_E_PLAN.  A plan that needs a workspace
 * (plan->ws_bytes > 0) returns CNN_E_UNSUPPORTED: run it with
 * cnn_fwd_plan_ws.  Allocates nothing.  Other errors as cnn_fwd.
 */
int cnn_fwd_plan(const void* In, const void* Ker, void* Out,
                 const cnn_problem* prob, int dtype, const cnn_plan_t* plan,
                 void* stream);

/*
 * As cnn_fwd_plan, with a caller-provided device workspace of ws_bytes
 * bytes (at least plan->ws_bytes, 16-byte aligned; NULL allowed when
 * plan->ws_bytes is 0): the repacked Ker of the packed-Ker families, or
 * the kc fp32 partial Outs of CNN_K_SPLITC.  The library keeps no pointer to
 * it after the call returns, but the kernels queued on `stream` use it
 * until they finish: it must not be freed or used by another call that may
 * run concurrently before then.  Allocates nothing, so it may be captured
 * into a HIP graph.  Errors: as cnn_fwd_plan, and CNN_E_NULL /
 * CNN_E_SHAPE if the workspace is missing, too small or misaligned.
 */
int cnn_fwd_plan_ws(const void* In, const void* Ker, void* Out,
                    const cnn_problem* prob, int dtype, const cnn_plan_t* plan,
                    void* workspace, int64_t ws_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid allocation): cnn_fwd_plan_ws with the
 * library's own device scratch of CNN_STATIC_SCRATCH_BYTES (8 MiB) in place
 * of a caller workspace.  Allocates nothing: the scratch is a static device
 * array that each GPU the library runs on holds until the process ends.
 * All calls on one GPU share it, so calls whose kernels may overlap on that
 * GPU (on different streams, or from several host threads) race and must
 * be ordered by the caller; consecutive calls on one stream are safe.  A
 * plan needing more than the scratch holds returns CNN_E_UNSUPPORTED
 * before any HIP call (use cnn_fwd_plan_ws).  Other errors as cnn_fwd_plan.
 */
#define CNN_STATIC_SCRATCH_BYTES (8LL << 20)

int cnn_fwd_plan_static(const void* In, const void* Ker, void* Out,
                        const cnn_problem* prob, int dtype, const cnn_plan_t* plan,
                        void* stream);

/*
 * Eq. (1) of the paper for a box tiling, in elements: terms[0] = Out
 * written once, terms[1] = Ker re-read per (b, w, h) tile, terms[2] = In
 * (with halo) re-read per k tile.  halo_mode 0 = the formula as printed
 * (real division, halo sigma*T + R - 1); 1 = exact (tile counts rounded up,
 * edge tiles clipped, halo sigma*(T-1) + R).  *footprint (may be NULL)
 * receives the left side of the Eq. (1) capacity constraint in elements,
 * in the same halo mode.  Errors: CNN_E_NULL, CNN_E_SHAPE.
 */
int cnn_eq1_cost(const cnn_problem* prob, const cnn_tiles* tiles, int halo_mode,
                 double terms[3], double* footprint);

/*
 * Eq. (1) terms (elements) of the composite tiling a plan uses: tp
 * consecutive outputs of the flattened (b, w, h) index by tk features, each
 * tile staging whole input rows.  Errors: CNN_E_NULL, CNN_E_SHAPE.
 */
int cnn_slab_cost(const cnn_problem* prob, int64_t tk, int64_t tp, double terms[3]);

/*
 * Closed-form optimum of the relaxed tiling problem, Eq. (4) of Sec. 2.1,
 * for P processors with M elements of fast memory each (host only, no HIP
 * call).  capacity_mode 0 takes M_L = M (the costs are then lower bounds for
 * any valid tiles); 1 takes M_L = M - (1/2) 3K (sqrt(9K^2 + 4M) - 3K),
 * K = sqrt(sw sh Nr Ns), for which the tiles are valid for Eq. (3).  With
 * V = Nk Nc Nbhw / P and Q = Nr Ns sw sh (Nbhw = Nb Nw Nh), the Table 1 row:
 *   1: Nk Nbhw / P >= M_L (Case 1a, W_c = N_c): Eq. (6),
 *      Tk = sqrt(M_L sw sh / (Nr Ns)), Tbhw = sqrt(M_L Nr Ns / (sw sh));
 *   2: M_L >= V^(2/3) Q^(1/3) (Case 2a, W_c < N_c): Eq. (8),
 *      Tk = (V / (Nr Ns))^(1/3) (sw sh)^(2/3), Tbhw = (V / (sw sh))^(1/3) (Nr Ns)^(2/3);
 *   3: otherwise (Case 2b, W_c < N_c): Eq. (9), the Case 1a tiles.
 * Tiles are real-valued; costs are elements moved per processor.  Errors:
 * CNN_E_NULL, CNN_E_SHAPE (a problem size below 1, P < 1, M <= 0 or a
 * capacity_mode other than 0 and 1).
 */
typedef struct cnn_closed_form_t {
  double M_L;           /* capacity of the relaxed problem                         */
  double Tk, Tbhw;      /* the row's optimal tile sizes                            */
  double cost;          /* the row's cost (Table 1)                                */
  int32_t row;          /* Table 1 row, 1 .. 3                                     */
  int32_t split_c;      /* 1 when the optimum has W_c < N_c (rows 2 and 3)         */
} cnn_closed_form_t;

int cnn_closed_form(const cnn_problem* prob, double P, double M, int capacity_mode,
                    cnn_closed_form_t* out);

/*
 * Eq. (3) of Sec. 2.1 one level up, for a plan: its workgroup tiles split
 * over `xcds` processors (the XCDs, each with an L2 of l2_bytes) the way the
 * kernels assign them -- XCD x runs the x-th of `xcds` contiguous runs of
 * the tile index (tile = pixel tile * ceil(Nk/tk) + k tile).  Each XCD reads
 * from HBM each input row its tiles read (all channels and columns) once,
 * and each Ker
 * tile its run meets once if those Ker tiles fit its L2 beside the largest
 * slab, else once per tile; Out is written once.  terms[0] = Out bytes
 * written (plus, for CNN_K_SPLITC, the fp32 partial Outs written and read
 * once), terms[1] = Ker bytes read, terms[2] = In bytes read.  A model for
 * the HBM counters, not a measurement; host only.  Errors: CNN_E_NULL,
 * CNN_E_SHAPE (xcds or l2_bytes below 1, a bad problem), CNN_E_DTYPE,
 * CNN_E_PLAN (the direct kernel's plan, or tk or tp below 1).
 */
int cnn_hbm_bytes(const cnn_plan_t* plan, int64_t xcds, int64_t l2_bytes, double terms[3]);

/* Budget of HIP device `device` (CU count, LDS per CU, accumulator regs). */
int cnn_device_budget(int device, cnn_budget* budget);

/* Static description of a status code. */
const char* cnn_strerror(int status);

/* Per-thread message of the most recent failing call ("" if none). */
const char* cnn_last_error(void);

/* CNN_ABI_VERSION of the loaded library. */
int cnn_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CNN_MI355X_H */

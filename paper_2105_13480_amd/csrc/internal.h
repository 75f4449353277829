// Internal declarations shared by the library's host code and kernels.
// Nothing here is part of the public ABI (include/cnn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cnn.h"

namespace cnnlib {

// Element size in bytes of In/Ker and of Out for a cnn_dtype.
inline int in_bytes(int dtype) { return dtype == CNN_F32 ? 4 : 2; }
inline int out_bytes(int dtype) { return dtype == CNN_BF16_OBF16 ? 2 : 4; }

// Arguments of every convolution kernel.  Sizes that the validation step
// bounds below 2^31 are int32; offsets into whole tensors are int64.
struct ConvArgs {
  int32_t Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh, Nx, Ny;
  int32_t hw;          // Nw*Nh outputs per (b, k) plane
  int32_t npix;        // Nb*Nw*Nh outputs of the flattened (b, w, h) index
  int32_t nxny;        // Nx*Ny input elements per (b, c) plane
  int64_t in_img;      // Nc*Nx*Ny input elements per image
  int64_t in_total;    // Nb*Nc*Nx*Ny
  int64_t out_total;   // Nb*Nk*Nw*Nh
  // tiling (implicit-GEMM kernels)
  int32_t tp, tk, tc;  // outputs, features, channels per workgroup tile / stage
  int32_t n_ptiles;    // ceil(npix / tp)
  int32_t n_ktiles;    // ceil(Nk / tk)
  int32_t slab_max;    // max input rows (flattened (b, x)) one tile stages
  int32_t grid;        // workgroups launched
};

// A kernel instantiation the selector may choose.
struct Variant {
  int32_t id;
  int32_t kernel;   // cnn_kernel
  int32_t dtype;    // cnn_dtype
  int32_t tk, tp, tc;
  int32_t threads;  // workgroup size
  int32_t acc;      // fp32 accumulators per lane
};

// Variant table (defined next to the kernels) and its size.
const Variant* variants(int* count);

// A pipelined implicit-GEMM instantiation (bf16 In/Ker, packed Ker).
struct Variant2 {
  int32_t id;
  int32_t dtype;    // CNN_BF16 or CNN_BF16_OBF16
  int32_t tk, tp, tc;
  int32_t acc;      // fp32 accumulators per lane
  int32_t nr, ns;   // compile-time stencil (0 = any)
  int32_t maxp;     // slab position pairs per thread: ceil(S*Ny/2) <= 256*maxp
  int32_t rawk;     // 1: stages raw Ker rows (needs Nc % 8 == 0), no repack / workspace
  int32_t pw;       // 1: 1x1 gather -- stages the tile's outputs' inputs, any stride
};
const Variant2* variants2(int* count);
int v2_family(const Variant2& v);
int64_t igemm2_blk_vecs(const Variant2& v, int64_t RS);
int64_t igemm2_lds_bytes(const Variant2& v, int64_t slab_rows, int64_t Ny, int64_t RS,
                         int64_t tp);
int64_t igemm2_ws_bytes(const Variant2& v, const cnn_problem& p);

// LDS bytes an implicit-GEMM variant needs for a given slab height.
int64_t igemm_lds_bytes(const Variant& v, int64_t slab_rows, int64_t Ny, int64_t RS);

// Max input rows any composite tile of `tp` outputs stages.
int64_t slab_rows_max(const cnn_problem& p, int64_t tp);

// A DMA-staged implicit-GEMM instantiation (bf16 In/Ker, packed Ker).
struct Variant3 {
  int32_t id;
  int32_t dtype;
  int32_t tk, tp, tc;
  int32_t acc;
  int32_t nr, ns;   // compile-time stencil (0 = any)
  int32_t nbuf;     // copy buffers in the DMA ring (2 or 3)
  int32_t ndi, ndk; // DMA instructions per thread per stage (In copy, Ker)
  int32_t mpos;     // transposed positions per thread (slab positions <= 256*mpos)
};
const Variant3* variants3(int* count);
int64_t igemm3_lds_bytes(const Variant3& v, int64_t slab_rows, int64_t Ny);
int64_t igemm3_ws_bytes(const Variant3& v, const cnn_problem& p);
bool igemm3_fits(const Variant3& v, const cnn_problem& p, int64_t slab_rows);

// A wide-staging, software-pipelined instantiation (bf16, packed Ker).
struct Variant4 {
  int32_t id;
  int32_t dtype;
  int32_t tk, tp, tc;
  int32_t acc;
  int32_t nr, ns;   // compile-time stencil (0 = any)
  int32_t maxi;     // In items per thread: tc/8 * ceil(S*Ny/8) <= 256*maxi
};
const Variant4* variants4(int* count);
int64_t igemm4_lds_bytes(const Variant4& v, int64_t slab_rows, int64_t Ny, int64_t RS);
int64_t igemm4_ws_bytes(const Variant4& v, const cnn_problem& p);
bool igemm4_fits(const Variant4& v, const cnn_problem& p, int64_t slab_rows);
hipError_t launch_igemm4(const Variant4& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

// A few-channel, wide-stencil instantiation (bf16): K = flattened (c, r, s8).
struct VariantS {
  int32_t id;
  int32_t dtype;
  int32_t tk, tp;   // tk = 64; tp = largest tile
  int32_t ks;       // K-steps held in registers: ceil(Nc*Nr/2) <= ks
  int32_t acc;
  int32_t nc, nr, ns, st;  // stencil compiled in (Nc, Nr, Ns, both strides), 0 for any
};
const VariantS* variants_smallc(int* count);
bool smallc_stencil_ok(const VariantS& v, const cnn_problem& p);  // the problem fits a fixed stencil
int64_t smallc_lds_bytes(const VariantS& v, const cnn_problem& p, int64_t slab_rows);
hipError_t launch_smallc(const VariantS& v, const void* In, const void* Ker, void* Out,
                         const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

// A row-streaming instantiation (bf16, stride 1, fixed stencil): tk = 64,
// tiles of whole output rows, Ker resident.
struct VariantR {
  int32_t id;
  int32_t dtype;
  int32_t tk;
  int32_t nr, ns;  // compile-time stencil
  int32_t wr;      // output rows per group
  int32_t mb;      // 32-position blocks per input row: Ny <= 32*mb
  int32_t waves;   // waves per workgroup (two per group of rows)
  int32_t ncg;     // 16-channel groups: Nc rounded up to 16 is 16*ncg
  int32_t acc;
};
const VariantR* variants_rows(int* count);
int64_t rows_lds_bytes(const VariantR& v, const cnn_problem& p);
bool rows_fits(const VariantR& v, const cnn_problem& p);
hipError_t launch_rows(const VariantR& v, const void* In, const void* Ker, void* Out,
                       const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

// A 1x1 stride-1 GEMM instantiation (bf16): tk features x up to tp pixels,
// tc channels per stage.
struct VariantG {
  int32_t id;
  int32_t dtype;
  int32_t tk, tp, tc;  // tp = largest tile
  int32_t threads;
  int32_t acc;
  int32_t s2;          // 0: stride 1; 1: strides 2 and 2 (gathers the even input rows
                       // and columns); 2: stride 1, whole-image tiles (at most
                       // tp - 8 pixels), operands copied by DMA into a ring of 4
                       // stages
};
const VariantG* variants_gemm1(int* count);
int64_t gemm1_lds_bytes(const VariantG& v);
bool gemm1_fits(const VariantG& v, const cnn_problem& p, int64_t tp);
hipError_t launch_gemm1(const VariantG& v, const void* In, const void* Ker, void* Out,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

// A stride-2 row-band instantiation (bf16, fixed stencil): tk = 256, bands
// of L whole output rows (Nh <= 32), 16 channels per chunk, packed Ker.
struct VariantQ {
  int32_t id;
  int32_t dtype;
  int32_t tk;
  int32_t nr, ns;  // compile-time stencil
  int32_t L;       // output rows per band
  int32_t waves;   // 4 or 8
  int32_t acc;     // fp32 accumulators per lane
  int32_t form;    // 1: packed Ker in a workspace, via LDS; 2: raw Ker repacked on chip;
                   // 3: packed Ker in a workspace, B operands in registers
};
const VariantQ* variants_srows(int* count);
int64_t srows_slab_rows(const VariantQ& v);
int64_t srows_lds_bytes(const VariantQ& v);
int64_t srows_ws_bytes(const VariantQ& v, const cnn_problem& p);
bool srows_fits(const VariantQ& v, const cnn_problem& p);
hipError_t launch_srows(const VariantQ& v, const void* In, const void* Ker, void* Out, void* ws,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

// Ker repack for the pipelined kernels (defined with conv_igemm2).
__global__ void pack_ker_bf16(const uint16_t* __restrict__ Ker, uint32_t __attribute__((ext_vector_type(4)))* __restrict__ P,
                              ConvArgs a, int TK, int TC, int blk_vecs, int64_t total_vecs);

// Byte ranges a family addresses with 32-bit buffer offsets (below 2 GiB):
// the images a tile of up to tp outputs touches (plus tc_extra channels of
// one more image), Ker rows of the raw-Ker families, whole tensors (In and
// Ker below in_limit), the few-channel and stride-2 row-band families.
bool ranges_ok_tile(const cnn_problem& p, int dtype, int64_t tp, int64_t tc_extra);
bool ranges_ok_rawk(const cnn_problem& p);
bool ranges_ok_whole(const cnn_problem& p, int dtype, int64_t in_limit);
bool ranges_ok_smallc(const VariantS& v, const cnn_problem& p, int dtype);
bool ranges_ok_srows(const VariantQ& v, const cnn_problem& p, int dtype);

// Records a failure message for cnn_last_error(); returns status.
int set_error(int status, const char* msg);

// cnn_fwd_plan_ws; with `dry` = true every argument and plan check and no
// HIP call (a NULL workspace then stands for one of ws_bytes bytes).
int fwd_plan_checked(const void* In, const void* Ker, void* Out, const cnn_problem* prob,
                     int dtype, const cnn_plan_t* plan, void* workspace, int64_t ws_bytes,
                     void* stream, bool dry);

// Lets `kernel` use up to 160 KiB of dynamic LDS on the current device.
// The attribute is set once per (kernel, device); later calls return at
// once.  Thread safe.
hipError_t allow_max_lds(const void* kernel);
// Compute units of the current device (cached per device; 256 if the query fails).
int device_cus();

// Launchers (asynchronous; return hipGetLastError()).
hipError_t launch_direct(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                         int dtype, hipStream_t stream);
hipError_t launch_igemm(const Variant& v, const void* In, const void* Ker, void* Out,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);
// Two-level (XCD, L2) HBM bytes of a plan (host).
void hbm_terms(const cnn_plan_t& pl, int64_t xcds, int64_t l2, double terms[3]);

// Table 1 optimum of Eq. (4) (host).
void closed_form(const cnn_problem& p, double P, double M, int capacity_mode,
                 cnn_closed_form_t* out);

// Split channels: conv_igemm over kc channel slices of
// splitc_slice_channels(Nc, tc, kc) channels each, fp32 partials in `ws`
// (kc * out_total floats), then their sum in slice order into Out.
int64_t splitc_slice_channels(int64_t Nc, int64_t tc, int64_t kc);
hipError_t launch_splitc(const Variant& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, int kc, int dtype,
                         hipStream_t stream);
// Out[o] = the sum over the kc fp32 partial Outs Part[z][o], z in order,
// converted to the Out type of `dtype` (n = |Out| elements).
hipError_t launch_splitc_reduce(const float* Part, void* Out, int kc, int64_t n, int dtype,
                                hipStream_t stream);

// A channel-slice instantiation (bf16, fixed stencil): tiles of tk = 32
// features x tp = 64 outputs over one slice of the channels, tc = 32
// channels per stage, every load of a stage in flight at once; fp32 partial
// tiles in the workspace, then the ordered reduce (mode 0); fp32 atomic
// adds into Out after a zero fill (mode 1: no workspace, fp32 Out only); or
// one slice (kc = 1) of 128-channel stages writing Out directly (mode 2: no
// workspace, any Out type).  A CNN_K_SPLITC family member beside the
// CNN_K_IGEMM split form.
struct VariantC {
  int32_t id;
  int32_t dtype;
  int32_t tk, tp, tc;
  int32_t nr, ns;  // compile-time stencil
  int32_t mode;    // 0 partials + reduce; 1 atomic sums into Out (order varies); 2 direct, kc = 1
};
const VariantC* variants_cslice(int* count);
int64_t cslice_lds_bytes(const VariantC& v, int64_t slab_rows, int64_t Ny);
bool cslice_fits(const VariantC& v, const cnn_problem& p);  // stencil, Nc % 16, index range
hipError_t launch_cslice(const VariantC& v, const void* In, const void* Ker, void* Out, void* ws,
                         const ConvArgs& a, int64_t lds_bytes, int kc, int dtype,
                         hipStream_t stream);
hipError_t launch_igemm3(const Variant3& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);
// Runs the pipelined kernel; non-raw-Ker variants first pack Ker into `ws`
// (igemm2_ws_bytes).
hipError_t launch_igemm2(const Variant2& v, const void* In, const void* Ker, void* Out,
                         void* ws, const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

}  // namespace cnnlib

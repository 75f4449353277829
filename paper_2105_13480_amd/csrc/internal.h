// Internal declarations shared by the library's host code and kernels.
// Nothing here is part of the public ABI (include/cnn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cnn.h"

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

// LDS bytes an implicit-GEMM variant needs for a given slab height.
int64_t igemm_lds_bytes(const Variant& v, int64_t slab_rows, int64_t Ny, int64_t RS);

// Max input rows any composite tile of `tp` outputs stages.
int64_t slab_rows_max(const cnn_problem& p, int64_t tp);

// Launchers (asynchronous; return hipGetLastError()).
hipError_t launch_direct(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                         int dtype, hipStream_t stream);
hipError_t launch_igemm(const Variant& v, const void* In, const void* Ker, void* Out,
                        const ConvArgs& a, int64_t lds_bytes, hipStream_t stream);

}  // namespace cnnlib

// Direct convolution: one thread per output, fp32 fused multiply-add over
// (c, r, s) in the order of the paper's Listing 1.  Handles every shape the
// ABI accepts; it is the correctness path and the fallback for problems
// whose input rows do not fit an LDS slab.
#include "internal.h"
#include "common.h"

namespace cnnlib {

template <typename TI, typename TO>
__global__ __launch_bounds__(256) void conv_direct(const TI* __restrict__ In,
                                                   const TI* __restrict__ Ker,
                                                   TO* __restrict__ Out, ConvArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int RS = a.Nr * a.Ns;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < a.out_total; o += stride) {
    const int h = (int)(o % a.Nh);
    const int w = (int)((o / a.Nh) % a.Nw);
    const int64_t bk = o / a.hw;
    const int k = (int)(bk % a.Nk);
    const int b = (int)(bk / a.Nk);
    const TI* in_b = In + (int64_t)b * a.in_img + (int64_t)(a.sw * w) * a.Ny + a.sh * h;
    const TI* ker_k = Ker + (int64_t)k * a.Nc * RS;
    float acc = 0.f;
    for (int c = 0; c < a.Nc; ++c) {
      const TI* in_c = in_b + (int64_t)c * a.nxny;
      const TI* ker_c = ker_k + c * RS;
      for (int r = 0; r < a.Nr; ++r)
        for (int s = 0; s < a.Ns; ++s)
          acc = __builtin_fmaf(to_f32(in_c[r * a.Ny + s]), to_f32(ker_c[r * a.Ns + s]), acc);
    }
    Out[o] = from_f32<TO>(acc);
  }
}

hipError_t launch_direct(const void* In, const void* Ker, void* Out, const ConvArgs& a,
                         int dtype, hipStream_t stream) {
  const int threads = 256;
  int64_t blocks = (a.out_total + threads - 1) / threads;
  if (blocks > 65536) blocks = 65536;  // grid-stride loop covers the rest
  dim3 g((unsigned)blocks), b(threads);
  switch (dtype) {
    case CNN_F32:
      hipLaunchKernelGGL((conv_direct<float, float>), g, b, 0, stream,
                         (const float*)In, (const float*)Ker, (float*)Out, a);
      break;
    case CNN_BF16:
      hipLaunchKernelGGL((conv_direct<bf16_t, float>), g, b, 0, stream,
                         (const bf16_t*)In, (const bf16_t*)Ker, (float*)Out, a);
      break;
    default:
      hipLaunchKernelGGL((conv_direct<bf16_t, bf16_t>), g, b, 0, stream,
                         (const bf16_t*)In, (const bf16_t*)Ker, (bf16_t*)Out, a);
      break;
  }
  return hipGetLastError();
}

}  // namespace cnnlib

// The shared dense branch MLP(x) of Eq. 7 as a SwiGLU block: two projections run on the logit
// GEMM kernels (gate and up rows in one GEMM into an fp32 buffer, then the down projection
// added into y), and this elementwise step between them: a = silu(g) * u, stored in the
// layer's dtype so that the down projection runs on MFMA for bf16.
#include "device_common.hpp"
#include "internal.hpp"

namespace omnimoe {
namespace {

// Four features per thread: h row t holds the d_ff gate values then the d_ff up values.
template <bool BF16>
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ h, void* a,
                                                     int64_t T, int d_ff) {
  const int q = d_ff / 4;
  const int64_t n = T * q;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256) {
    const int64_t t = i / q;
    const int f = (int)(i - t * q) * 4;
    const float4 g = *(const float4*)(h + t * 2 * d_ff + f);
    const float4 u = *(const float4*)(h + t * 2 * d_ff + d_ff + f);
    const float r0 = activation(1, g.x) * u.x, r1 = activation(1, g.y) * u.y;
    const float r2 = activation(1, g.z) * u.z, r3 = activation(1, g.w) * u.w;
    if constexpr (BF16) {
      uint2 o;
      o.x = (uint32_t)bf16_rne(r0) | ((uint32_t)bf16_rne(r1) << 16);
      o.y = (uint32_t)bf16_rne(r2) | ((uint32_t)bf16_rne(r3) << 16);
      *(uint2*)((uint16_t*)a + t * d_ff + f) = o;
    } else {
      *(float4*)((float*)a + t * d_ff + f) = make_float4(r0, r1, r2, r3);
    }
  }
}

}  // namespace

hipError_t launch_swiglu(int64_t T, int d_ff, bool bf16, const float* h, void* a,
                         hipStream_t st) {
  const int64_t n = T * (d_ff / 4);
  if (n == 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (bf16)
    hipLaunchKernelGGL(swiglu_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, h, a, T,
                       d_ff);
  else
    hipLaunchKernelGGL(swiglu_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, h, a, T,
                       d_ff);
  return hipGetLastError();
}

}  // namespace omnimoe

// Grouped value heads (Sec. 3.5, App. C.1): q, k, the log-decay and b of a key
// head are shared by the G value heads of its group, so their gradients are
// the sums of the per-value-head contributions, which the fp32 chunk backward
// leaves in fp32 on the value-head axis (the bf16 one adds them up itself).
// One thread per 4 consecutive outputs; the G partials are added in a fixed
// order (deterministic).

#include "gdr2_kernels.hpp"

namespace gdr2 {

__device__ __forceinline__ void store4(float* p, const float4& x) { *reinterpret_cast<float4*>(p) = x; }
__device__ __forceinline__ void store4(bf16_t* p, const float4& x) {
  bf16_t t[4];
  put(&t[0], x.x);
  put(&t[1], x.y);
  put(&t[2], x.z);
  put(&t[3], x.w);
  *reinterpret_cast<uint2*>(p) = make_uint2((uint32_t)t[0].x | ((uint32_t)t[1].x << 16),
                                            (uint32_t)t[2].x | ((uint32_t)t[3].x << 16));
}

template <typename TOut>
__global__ __launch_bounds__(256) void group_reduce_kernel(const float* __restrict__ P, TOut* __restrict__ out,
                                                           size_t n4, int Hk, int G, int D) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const size_t e = 4 * i;  // output element (r * Hk + h) * D + c
    const size_t c = e % D, rh = e / D;
    // partial of value head h * G + j at row r: ((r * Hk + h) * G + j) * D + c
    const float* src = P + rh * G * D + c;
    float4 acc = ld4(src);
    for (int j = 1; j < G; ++j) {
      const float4 x = ld4(src + (size_t)j * D);
      acc.x += x.x;
      acc.y += x.y;
      acc.z += x.z;
      acc.w += x.w;
    }
    store4(out + e, acc);
  }
}

template <typename TOut>
hipError_t launch_group_reduce(const float* P, TOut* out, size_t rows, int Hk, int G, int D, hipStream_t st) {
  const size_t n4 = rows * Hk * (size_t)D / 4;
  const size_t blocks = (n4 + 255) / 256;
  dim3 grid((unsigned)(blocks < 16384 ? blocks : 16384));
  if (n4 == 0) return hipSuccess;
  hipLaunchKernelGGL((group_reduce_kernel<TOut>), grid, dim3(256), 0, st, P, out, n4, Hk, G, D);
  return hipGetLastError();
}

template hipError_t launch_group_reduce<float>(const float*, float*, size_t, int, int, int, hipStream_t);
template hipError_t launch_group_reduce<bf16_t>(const float*, bf16_t*, size_t, int, int, int, hipStream_t);

}  // namespace gdr2

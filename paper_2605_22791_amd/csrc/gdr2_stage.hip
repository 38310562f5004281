// Backward of the fused input stage (App. C.1, App. D.2), after the chunk
// backward has left the gradients of the normalised q, k and the per-workgroup
// sums of the decay-parameter gradients.
//
// Normalisation VJP: y = rinv x with rinv = (sum x^2 + eps)^(-1/2) has
//     dx = rinv (dy - y <y, dy>),
// which needs a whole row of dy; DK / 8 consecutive lanes own one row (8
// channels each, 16-byte accesses) and reduce <y, dy> by shuffles.  dy comes
// in fp32 (rounded once, after the VJP): for grouped value heads the sum of the
// G per-value-head partials, added here in a fixed order.
//
// Decay parameters: ddelta and da are sums over every (token, value head) of
// the partials the chunk backward wrote per workgroup; they are added in two
// deterministic passes (slot ranges in parallel, then the ranges).

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK>
__global__ __launch_bounds__(256) void norm_vjp_kernel(NormVjpArgs a) {
  constexpr int LPR = DK / 8, RPB = 256 / LPR;  // lanes per row, rows per block pass
  const int z = blockIdx.y;  // 0: q, 1: k
  const bf16_t* X = a.x[z];
  const float* RI = a.rinv[z];
  const int tid = threadIdx.x, lr = tid % LPR, c0 = 8 * lr;
  const size_t nrows = a.rows * (size_t)a.Hk;
  // every lane of a row takes the same trips through this loop (R is shared)
  for (size_t R = (size_t)blockIdx.x * RPB + tid / LPR; R < nrows; R += (size_t)gridDim.x * RPB) {
    const float ri = RI[R];
    float x[8], dy[8];
    unpack8(ldg16(X + R * DK + c0), x);
    const float* p = a.P[z] + (size_t)a.G * R * DK + c0;
    ldf8(p, dy);
    for (int j = 1; j < a.G; ++j) {
      float t[8];
      ldf8(p + (size_t)j * DK, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) dy[e] += t[e];
    }
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      x[e] *= ri;  // y
      dot += x[e] * dy[e];
    }
#pragma unroll
    for (int o = 1; o < LPR; o <<= 1) dot += __shfl_xor(dot, o);
    float dx[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) dx[e] = ri * (dy[e] - x[e] * dot);
    sts16(a.dx[z] + R * DK + c0, __builtin_bit_cast(u4v, round8(dx)));
  }
}

template <int DK>
hipError_t launch_norm_vjp(const NormVjpArgs& a, hipStream_t st) {
  constexpr int RPB = 256 / (DK / 8);
  const size_t nrows = a.rows * (size_t)a.Hk;
  if (nrows == 0) return hipSuccess;
  const size_t blocks = (nrows + RPB - 1) / RPB;
  dim3 grid((unsigned)(blocks < 32768 ? blocks : 32768), 2);
  hipLaunchKernelGGL((norm_vjp_kernel<DK>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template hipError_t launch_norm_vjp<64>(const NormVjpArgs&, hipStream_t);
template hipError_t launch_norm_vjp<128>(const NormVjpArgs&, hipStream_t);

// out[(z * Hk + hk) * D + c] = sum over slots s of split z (and m < M) of
// P[((s * Hk + hk) * M + m) * D + c]; block (hk, 64-channel group, split z),
// four parts of 64 threads interleaved over the slots, combined in order.
__global__ __launch_bounds__(256) void param_reduce_kernel(const float* __restrict__ P, float* __restrict__ out,
                                                           int nslots, int Hk, int M, int D, int per) {
  __shared__ float red[4][64];
  const int hk = blockIdx.x, cl = threadIdx.x & 63, part = threadIdx.x >> 6, z = blockIdx.z;
  const int c = blockIdx.y * 64 + cl;
  const int s0 = z * per, s1 = min(nslots, s0 + per);
  float acc = 0.f;
  if (c < D) {
    for (int s = s0 + part; s < s1; s += 4) {
      const float* p = P + (((size_t)s * Hk + hk) * M) * D + c;
      for (int m = 0; m < M; ++m) acc += p[(size_t)m * D];
    }
  }
  red[part][cl] = acc;
  __syncthreads();
  if (part == 0 && c < D) out[((size_t)z * Hk + hk) * D + c] = ((red[0][cl] + red[1][cl]) + red[2][cl]) + red[3][cl];
}

hipError_t launch_param_reduce_pass(const float* P, float* out, int nslots, int Hk, int M, int D, int splits,
                                    hipStream_t st) {
  const int per = (nslots + splits - 1) / splits;
  dim3 grid(Hk, (D + 63) / 64, splits);
  hipLaunchKernelGGL(param_reduce_kernel, grid, dim3(256), 0, st, P, out, nslots, Hk, M, D, per);
  return hipGetLastError();
}

}  // namespace gdr2

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

// ---- fp32 problems: the stage as its own passes around the fp32 operator ----
// Forward: rows of q (z = 0) and k (z = 1) normalised, y = x rinv, with rinv
// kept; z = 2 forms g = -exp(a) softplus(f + delta).  DK / 4 lanes per row.
template <int DK>
__global__ __launch_bounds__(256) void stage_fwd_f32_kernel(StageF32Args a) {
  constexpr int LPR = DK / 4, RPB = 256 / LPR;
  const int z = blockIdx.y, tid = threadIdx.x, lr = tid % LPR, c0 = 4 * lr;
  const size_t nrows = a.rows * (size_t)a.Hk;
  for (size_t R = (size_t)blockIdx.x * RPB + tid / LPR; R < nrows; R += (size_t)gridDim.x * RPB) {
    const size_t o = R * DK + c0;
    if (z < 2) {
      const float4 x = ld4((z == 0 ? a.q : a.k) + o);
      float ss = x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
#pragma unroll
      for (int m = 1; m < LPR; m <<= 1) ss += __shfl_xor(ss, m);
      const float ri = inv_norm(ss, a.eps);
      *reinterpret_cast<float4*>((z == 0 ? a.qn : a.kn) + o) = make_float4(x.x * ri, x.y * ri, x.z * ri, x.w * ri);
      if (lr == 0) (z == 0 ? a.rq : a.rk)[R] = ri;
    } else {
      const int hk = (int)(R % a.Hk);
      const float A = expf(a.a_log[hk]);
      const float4 f = ld4(a.f + o), dl = ld4(a.delta + (size_t)hk * DK + c0);
      *reinterpret_cast<float4*>(a.g + o) = make_float4(decay_act(f.x, dl.x, A), decay_act(f.y, dl.y, A),
                                                        decay_act(f.z, dl.z, A), decay_act(f.w, dl.w, A));
    }
  }
}

// Backward: z = 0, 1: dx = rinv (dy - y <y, dy>) from the fp32 gradients of the
// normalised q, k; z = 2: df = dg * (-exp(a) sigmoid(f + delta)) and, per row,
// sum_c dg * g into pa (the partials of da).
template <int DK>
__global__ __launch_bounds__(256) void stage_bwd_f32_kernel(StageF32Args a) {
  constexpr int LPR = DK / 4, RPB = 256 / LPR;
  const int z = blockIdx.y, tid = threadIdx.x, lr = tid % LPR, c0 = 4 * lr;
  const size_t nrows = a.rows * (size_t)a.Hk;
  for (size_t R = (size_t)blockIdx.x * RPB + tid / LPR; R < nrows; R += (size_t)gridDim.x * RPB) {
    const size_t o = R * DK + c0;
    if (z < 2) {
      const float ri = (z == 0 ? a.rq : a.rk)[R];
      const float4 x = ld4((z == 0 ? a.q : a.k) + o), dy = ld4((z == 0 ? a.dqn : a.dkn) + o);
      const float y[4] = {x.x * ri, x.y * ri, x.z * ri, x.w * ri};
      float dot = y[0] * dy.x + y[1] * dy.y + y[2] * dy.z + y[3] * dy.w;
#pragma unroll
      for (int m = 1; m < LPR; m <<= 1) dot += __shfl_xor(dot, m);
      *reinterpret_cast<float4*>((z == 0 ? a.dq : a.dk) + o) =
          make_float4(ri * (dy.x - y[0] * dot), ri * (dy.y - y[1] * dot), ri * (dy.z - y[2] * dot),
                      ri * (dy.w - y[3] * dot));
    } else {
      const int hk = (int)(R % a.Hk);
      const float A = expf(a.a_log[hk]);
      const float4 f = ld4(a.f + o), dl = ld4(a.delta + (size_t)hk * DK + c0), dg = ld4(a.dg + o);
      const float x[4] = {f.x + dl.x, f.y + dl.y, f.z + dl.z, f.w + dl.w}, d[4] = {dg.x, dg.y, dg.z, dg.w};
      float df[4], pa = 0.f;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        df[e] = d[e] * (-A * sigmoid_f(x[e]));
        pa += d[e] * (-A * softplus_f(x[e]));
      }
      *reinterpret_cast<float4*>(a.df + o) = make_float4(df[0], df[1], df[2], df[3]);
#pragma unroll
      for (int m = 1; m < LPR; m <<= 1) pa += __shfl_xor(pa, m);
      if (lr == 0) a.pa[R] = pa;
    }
  }
}

template <int DK>
hipError_t launch_stage_f32(const StageF32Args& a, bool backward, hipStream_t st) {
  constexpr int RPB = 256 / (DK / 4);
  const size_t nrows = a.rows * (size_t)a.Hk;
  if (nrows == 0) return hipSuccess;
  const size_t blocks = (nrows + RPB - 1) / RPB;
  dim3 grid((unsigned)(blocks < 32768 ? blocks : 32768), 3);
  if (backward)
    hipLaunchKernelGGL((stage_bwd_f32_kernel<DK>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((stage_fwd_f32_kernel<DK>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template hipError_t launch_stage_f32<64>(const StageF32Args&, bool, hipStream_t);
template hipError_t launch_stage_f32<128>(const StageF32Args&, bool, hipStream_t);

}  // namespace gdr2

// Recurrent (token-by-token) GDR-2 forward for decoding, App. C.5.
//
// One workgroup per (batch, head), or per (sequence, head) of a packed batch
// (App. C.6: the same cumulative-length layout as the chunk kernels).  The fp32 state (DK x DV) stays in registers
// for all T tokens of the call: each thread owns RPG rows x 4 columns.  Per token
//     Sbar = Diag(exp g) S,  r = Sbar^T (b*k),  S = Sbar + k (w*v - r)^T,
//     o    = scale * S^T q = scale * (Sbar^T q + (w*v - r) (k . q)),
// so S is read and written once per call; the column sums r and Sbar^T q are
// reduced across the row groups through LDS in a fixed order.
//
// Fused input stage (a.st.a_log set; App. C.1, App. D.2): q and k are the raw
// projections, L2-normalised per token in fp32 and rounded to the operand
// dtype, as the chunk path does; the log-decay is -exp(a) softplus(f + delta)
// from the decay projection f.

#include "gdr2_kernels.hpp"

namespace gdr2 {

// x rounded to the operand dtype (nearest, ties to even)
template <typename TIn>
__device__ __forceinline__ float round_as(float x);
template <>
__device__ __forceinline__ float round_as<float>(float x) { return x; }
template <>
__device__ __forceinline__ float round_as<bf16_t>(float x) {
  bf16_t t;
  put(&t, x);
  return to_f(t);
}

template <int DK, int DV, typename TIn, bool FUSED>
__global__ __launch_bounds__(256) void recurrent_kernel(RecurArgs<TIn> a) {
  constexpr int NTHR = 256;
  constexpr int CG = DV / 4;        // column groups of 4
  constexpr int RG = NTHR / CG;     // row groups
  constexpr int RPG = DK / RG;      // rows per thread
  static_assert(NTHR % CG == 0 && DK % RG == 0, "thread split");
  static_assert(DK <= NTHR, "one key channel per thread");
  const int seq = blockIdx.x;
  const int bb = seq / a.H, h = seq % a.H;
  const int tid = threadIdx.x, cg = tid % CG, rg = tid / CG;
  const int T = a.T, H = a.H;

  __shared__ float sAl[DK], sE[DK], sK[DK], sQ[DK], sZ[DV];
  __shared__ float redR[RG * DV], redP[RG * DV];
  __shared__ float sRes[DV], sP[DV];
  __shared__ float sKQ[NTHR / 64], sKK[NTHR / 64], sQQ[NTHR / 64];

  float* Sg = a.S + (size_t)seq * DK * DV;
  float4 S[RPG];
#pragma unroll
  for (int i = 0; i < RPG; ++i) S[i] = ld4(Sg + (rg * RPG + i) * DV + 4 * cg);

  // tokens of this sequence: bb's T tokens, or cu[bb] .. cu[bb+1) of a packed batch (clamped into [0, T])
  int t0 = 0, t1 = T;
  size_t rbase = (size_t)bb * T;
  if (a.cu != nullptr) {
    t0 = min(max(a.cu[bb], 0), T);
    t1 = min(max(a.cu[bb + 1], t0), T);
    rbase = 0;
  }
  const int HK = H / a.G, hk = h / a.G;  // key side (q, k, g, b) on the H / G key heads
  const float Adec = FUSED ? expf(a.st.a_log[hk]) : 0.f;
  for (int t = t0; t < t1; ++t) {
    const size_t row = (rbase + t) * H + h, rowk = (rbase + t) * HK + hk;
    // thread c < DK holds key channel c of this token (DK <= NTHR)
    const int c = tid;
    float kv = 0.f, qv = 0.f, bv = 0.f, kq = 0.f;
    if (c < DK) {
      kv = to_f(a.k[rowk * DK + c]);
      qv = to_f(a.q[rowk * DK + c]);
      bv = to_f(a.b[rowk * DK + c]);
      const float gv = a.g[rowk * DK + c];
      sAl[c] = expf(FUSED ? decay_act(gv, a.st.delta[(size_t)hk * DK + c], Adec) : gv);
      if constexpr (!FUSED) {
        sK[c] = kv;
        sQ[c] = qv;
        sE[c] = bv * kv;
        kq = kv * qv;
      }
    }
    for (int v = tid; v < DV; v += NTHR) sZ[v] = to_f(a.w[row * DV + v]) * to_f(a.v[row * DV + v]);
    if constexpr (FUSED) {
      // fused stage: sums of squares over the row, then y = x (sum x^2 + eps)^(-1/2) in the operand dtype
      float kk = kv * kv, qq = qv * qv;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        kk += __shfl_xor(kk, m);
        qq += __shfl_xor(qq, m);
      }
      if ((tid & 63) == 0) {
        sKK[tid >> 6] = kk;
        sQQ[tid >> 6] = qq;
      }
      __syncthreads();
      float sk = 0.f, sq = 0.f;
#pragma unroll
      for (int w2 = 0; w2 < NTHR / 64; ++w2) {
        sk += sKK[w2];
        sq += sQQ[w2];
      }
      kv = round_as<TIn>(kv * inv_norm(sk, a.st.eps));
      qv = round_as<TIn>(qv * inv_norm(sq, a.st.eps));
      if (c < DK) {
        sK[c] = kv;
        sQ[c] = qv;
        sE[c] = bv * kv;
        kq = kv * qv;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) kq += __shfl_xor(kq, m);
    if ((tid & 63) == 0) sKQ[tid >> 6] = kq;
    __syncthreads();

    float4 pr = make_float4(0.f, 0.f, 0.f, 0.f), pp = pr;
#pragma unroll
    for (int i = 0; i < RPG; ++i) {
      const int c = rg * RPG + i;
      const float al = sAl[c], e = sE[c], q = sQ[c];
      S[i].x *= al; S[i].y *= al; S[i].z *= al; S[i].w *= al;
      pr.x += S[i].x * e; pr.y += S[i].y * e; pr.z += S[i].z * e; pr.w += S[i].w * e;
      pp.x += S[i].x * q; pp.y += S[i].y * q; pp.z += S[i].z * q; pp.w += S[i].w * q;
    }
    *reinterpret_cast<float4*>(redR + rg * DV + 4 * cg) = pr;
    *reinterpret_cast<float4*>(redP + rg * DV + 4 * cg) = pp;
    __syncthreads();
    for (int v = tid; v < DV; v += NTHR) {
      float r = 0.f, p = 0.f;
      for (int g2 = 0; g2 < RG; ++g2) {
        r += redR[g2 * DV + v];
        p += redP[g2 * DV + v];
      }
      const float res = sZ[v] - r;
      sRes[v] = res;
      sP[v] = p;
    }
    __syncthreads();
    float kqa = 0.f;
#pragma unroll
    for (int w2 = 0; w2 < NTHR / 64; ++w2) kqa += sKQ[w2];
    const float4 res = ld4(sRes + 4 * cg);
#pragma unroll
    for (int i = 0; i < RPG; ++i) {
      const float kc = sK[rg * RPG + i];
      S[i].x += kc * res.x; S[i].y += kc * res.y; S[i].z += kc * res.z; S[i].w += kc * res.w;
    }
    for (int v = tid; v < DV; v += NTHR) put(a.o + row * DV + v, a.scale * (sP[v] + sRes[v] * kqa));
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < RPG; ++i) *reinterpret_cast<float4*>(Sg + (rg * RPG + i) * DV + 4 * cg) = S[i];
}

template <int DK, int DV, typename TIn>
hipError_t launch_recurrent(const RecurArgs<TIn>& a, int B, hipStream_t st) {
  if (a.st.a_log != nullptr)
    hipLaunchKernelGGL((recurrent_kernel<DK, DV, TIn, true>), dim3(B * a.H), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((recurrent_kernel<DK, DV, TIn, false>), dim3(B * a.H), dim3(256), 0, st, a);
  return hipGetLastError();
}

#define GDR2_INST_REC(DK, DV, TIN) \
  template hipError_t launch_recurrent<DK, DV, TIN>(const RecurArgs<TIN>&, int, hipStream_t);

GDR2_INST_REC(64, 64, float)
GDR2_INST_REC(64, 128, float)
GDR2_INST_REC(128, 64, float)
GDR2_INST_REC(128, 128, float)
GDR2_INST_REC(64, 64, bf16_t)
GDR2_INST_REC(64, 128, bf16_t)
GDR2_INST_REC(128, 64, bf16_t)
GDR2_INST_REC(128, 128, bf16_t)

}  // namespace gdr2

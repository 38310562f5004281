// Device-side building blocks shared by the GDR-2 kernels (gfx950 / CDNA4).
//
// Chunk geometry: C = 64 tokens per chunk (App. C.2), split into four 16-row
// blocks that match the 16x16 MFMA tiles.  Inside a chunk every decay ratio
// gamma_r / gamma_s = exp(G_r - G_s) (r >= s, App. A.1) is formed as a product
// of three factors that are each bounded, so no intermediate overflows even
// when the chunk's total decay is far below fp32's exp range:
//
//   exp(G_r - G_s) = exp(G_r - G_p(i)) * exp(G_p(i) - G_e(j)) * exp(G_e(j) - G_s)
//                    \_ left, <= 1 _/   \____ bridge d_ij ____/  \_ right, <= 1 _/
//
// with r in block i, s in block j <= i, p(i) = 16 i the first row of block i
// and e(j) = 16 j + 15 the last row of block j.  For j < i the bridge is <= 1;
// for j == i it is >= 1 and bounded by the decay accumulated inside one block.
// When that exceeds kDiagLimit (a decay below e^-60 within 15 tokens, far
// outside ordinary inputs) the diagonal block is computed element by element
// instead (kernels check the per-block `unsafe` flag).  The paper does not
// prescribe a stabilisation; this one is this library's.

#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gdr2 {

constexpr int CH = 64;            // chunk length C
constexpr int LD64 = CH + 4;      // LDS row stride of 64-wide fp32 tiles
constexpr float kDiagLimit = 60.f;

typedef float f4 __attribute__((ext_vector_type(4)));

// raw bfloat16 storage
struct bf16_t {
  uint16_t x;
};

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  // v_mfma_f32_16x16x4_f32: D(16x16) += A(16x4) B(4x16), one block.
  // lane l supplies A[l%16][l/16] and B[l/16][l%16]; D[4*(l/16)+i][l%16] -> c[i].
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(bf16_t x) { return __uint_as_float(((uint32_t)x.x) << 16); }

__device__ __forceinline__ void put(float* p, float x) { *p = x; }
__device__ __forceinline__ void put(bf16_t* p, float x) {
  uint32_t u = __float_as_uint(x);
  uint16_t r;
  if ((u & 0x7fffffffu) > 0x7f800000u) {
    r = 0x7fc0;  // quiet NaN
  } else {
    u += 0x7fffu + ((u >> 16) & 1u);  // round to nearest even
    r = (uint16_t)(u >> 16);
  }
  p->x = r;
}

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4(const bf16_t* p) {
  uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}
// ld4 / to_f of a token row that may lie past a partial chunk's end (then 0)
template <typename T>
__device__ __forceinline__ float4 ld4z(const T* p, bool ok) {
  return ok ? ld4(p) : make_float4(0.f, 0.f, 0.f, 0.f);
}
template <typename T>
__device__ __forceinline__ float to_fz(const T* p, bool ok) {
  return ok ? to_f(*p) : 0.f;
}
__device__ __forceinline__ float f4at(const float4& v, int u) {
  return u == 0 ? v.x : (u == 1 ? v.y : (u == 2 ? v.z : v.w));
}

__device__ __forceinline__ int pair_index(int i, int j) { return (i * (i + 1)) / 2 + j; }

// ---- fused input stage (App. C.1, App. D.1 - D.2) ---------------------------
// Both on the transcendental unit (v_exp_f32 = 2^x, v_log_f32 = log2 x,
// v_rcp_f32, each within about an ulp), written so that no step loses relative
// accuracy: u = e^-|x| in (0, 1], and log1p(u) by the identity
// log1p(u) = u log(w) / (w - 1) with w = fl(1 + u) (exact to a few ulps, u
// itself when w rounds to 1), so the tiny values of very negative x keep their
// relative accuracy and large x cannot overflow.
__device__ __forceinline__ float softplus_f(float x) {
  constexpr float kL2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
  const float u = __builtin_amdgcn_exp2f(-fabsf(x) * kL2e);
  const float w = 1.f + u;
  const float l = w == 1.f ? u : __builtin_amdgcn_logf(w) * kLn2 * u * __builtin_amdgcn_rcpf(w - 1.f);
  return fmaxf(x, 0.f) + l;
}
// logistic function, the derivative of softplus: 1 / (1 + e^-x), e^x / (1 + e^x) for x < 0
__device__ __forceinline__ float sigmoid_f(float x) {
  constexpr float kL2e = 1.4426950408889634f;
  const float u = __builtin_amdgcn_exp2f(-fabsf(x) * kL2e), r = __builtin_amdgcn_rcpf(1.f + u);
  return x >= 0.f ? r : u * r;
}
// log-decay from the decay projection: g = -A softplus(f + delta), A = exp(a) of the key head
__device__ __forceinline__ float decay_act(float f, float delta, float A) { return -A * softplus_f(f + delta); }
// inverse norm of the L2 normalisation y = x (sum x^2 + eps)^(-1/2)
__device__ __forceinline__ float inv_norm(float ss, float eps) { return 1.f / sqrtf(ss + eps); }
__device__ __forceinline__ void pair_of(int p, int& i, int& j) {
  i = (p >= 6) ? 3 : (p >= 3) ? 2 : (p >= 1) ? 1 : 0;
  j = p - (i * (i + 1)) / 2;
}

// ---------------------------------------------------------------------------
// Chunk-local cumulative log-decay G_r = sum_{i<=r} g_i (eq. eq_gdn2_gamma),
// computed in fp32 from the fp32 log-decay (App. D.1).  g points at row 0,
// channel 0 of the chunk for one head; rs is the row stride in elements.
// Result in sG[r * (DK+4) + c]; rows r >= len (past a partial chunk's end)
// count as g = 0.  All threads of the block must call it.
template <int DK, int NTHR>
__device__ void chunk_cumsum(const float* __restrict__ g, size_t rs, float* sG, int tid, int len) {
  constexpr int LG = DK + 4;
  for (int e = tid; e < CH * DK / 4; e += NTHR) {
    const int r = e / (DK / 4), c4 = (e % (DK / 4)) * 4;
    const float4 x = ld4z(g + r * rs + c4, r < len);
    float* d = sG + r * LG + c4;
    d[0] = x.x; d[1] = x.y; d[2] = x.z; d[3] = x.w;
  }
  __syncthreads();
  constexpr int NSEG = NTHR / DK;
  constexpr int RPS = CH / NSEG;
  static_assert(NTHR % DK == 0 && CH % NSEG == 0, "scan split");
  const int c = tid % DK, seg = tid / DK;
  float run = 0.f;
  for (int r = seg * RPS; r < (seg + 1) * RPS; ++r) {
    run += sG[r * LG + c];
    sG[r * LG + c] = run;
  }
  __syncthreads();
  float off = 0.f;
  for (int s = 0; s < seg; ++s) off += sG[((s + 1) * RPS - 1) * LG + c];
  __syncthreads();
  if (seg > 0)
    for (int r = seg * RPS; r < (seg + 1) * RPS; ++r) sG[r * LG + c] += off;
  __syncthreads();
}

// Reference exponentials of the block factorisation: eP[i][c] = exp(G_{16i}),
// brg[pair(i,j)][c] = exp(G_{16i} - G_{16j+15}) for j <= i, eGC[c] = exp(G_63),
// unsafe[i] = 1 when block i's diagonal bridge would exceed e^kDiagLimit.
template <int DK, int NTHR>
__device__ void chunk_refs(const float* sG, float* eP, float* brg, float* eGC, int* unsafe,
                           int tid) {
  constexpr int LG = DK + 4;
  for (int e = tid; e < 4 * DK; e += NTHR) {
    const int i = e / DK, c = e % DK;
    eP[i * DK + c] = expf(sG[(16 * i) * LG + c]);
  }
  for (int e = tid; e < 10 * DK; e += NTHR) {
    const int p = e / DK, c = e % DK;
    int i, j;
    pair_of(p, i, j);
    const float d = sG[(16 * i) * LG + c] - sG[(16 * j + 15) * LG + c];
    brg[p * DK + c] = expf(d);
    if (i == j && d > kDiagLimit) unsafe[i] = 1;
  }
  for (int c = tid; c < DK; c += NTHR) eGC[c] = expf(sG[(CH - 1) * LG + c]);
  __syncthreads();
}

// ---------------------------------------------------------------------------
// 16x16 tile of  sum_c L[16i+m][c] * d[c] * R[16j+n][c]  on MFMA (fp32).
// L, R: LDS tiles with row stride DK+4; d: bridge vector (length DK).
// The k index c is permuted so that each lane reads 4 consecutive channels.
template <int DK>
__device__ __forceinline__ f4 gram_tile(const float* L, const float* R, const float* d, int i,
                                        int j, int lane) {
  constexpr int LS = DK + 4;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  const float* pa = L + (16 * i + (lane & 15)) * LS + 4 * (lane >> 4);
  const float* pb = R + (16 * j + (lane & 15)) * LS + 4 * (lane >> 4);
  const float* pd = d + 4 * (lane >> 4);
#pragma unroll 4
  for (int kk = 0; kk < DK; kk += 16) {
    const float4 a = ld4(pa + kk), b = ld4(pb + kk), s = ld4(pd + kk);
    acc = mfma4(a.x * s.x, b.x, acc);
    acc = mfma4(a.y * s.y, b.y, acc);
    acc = mfma4(a.z * s.z, b.z, acc);
    acc = mfma4(a.w * s.w, b.w, acc);
  }
  return acc;
}

// Diagonal 16x16 tile computed element by element (used only for an unsafe
// block): out[m][n] = sum_c X[r][c] * k[s][c] * exp(G_r - G_s), r = 16i+m,
// s = 16i+n, for r >= s (strict when `strict`), else 0.  X = b*k (Gram T) or
// q (scores).  Reads the raw inputs; G differences are accumulated locally
// from g so they never leave the block.  Rows >= len read as zero.
template <int DK, typename TIn>
__device__ f4 diag_tile_direct(const TIn* __restrict__ x1, const TIn* __restrict__ x2,
                               const TIn* __restrict__ k, const float* __restrict__ g,
                               size_t rs, int i, int lane, bool strict, int len) {
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  const int n = lane & 15, mb = 4 * (lane >> 4);
  const int s = 16 * i + n;
  for (int c = 0; c < DK; ++c) {
    float run = 0.f, Gs = 0.f, Gr[4] = {0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < 16; ++t) {
      run += to_fz(g + (16 * i + t) * rs + c, 16 * i + t < len);
      if (t == n) Gs = run;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (t == mb + u) Gr[u] = run;
    }
    const float ks = to_fz(k + s * rs + c, s < len);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int m = mb + u;
      if (m > n || (!strict && m == n)) {
        const int r = 16 * i + m;
        float xv = to_fz(x1 + r * rs + c, r < len);
        if (x2) xv *= to_fz(x2 + r * rs + c, r < len);
        acc[u] += xv * ks * expf(Gr[u] - Gs);
      }
    }
  }
  return acc;
}

// ---------------------------------------------------------------------------
// A = (I + T)^{-1} for the strictly lower 64x64 T (eq. eq_gdn2_wy_matrix),
// in IEEE fp32 (App. D.4).  Blocked forward substitution: the four 16x16
// diagonal blocks are inverted by one wave (lane = column), then the
// off-diagonal blocks follow by block distance:
//     A_ij = -A_ii * sum_{j <= k < i} T_ik A_kj .
// sT, sA: row stride LD64.  sM: scratch of 3*256 floats.
template <int NTHR>
__device__ void wy_solve(const float* sT, float* sA, float* sM, int tid) {
  if (tid < 64) {
    const int blk = tid >> 4, c = tid & 15;
    float x[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float acc = (r == c) ? 1.f : 0.f;
#pragma unroll
      for (int s = 0; s < r; ++s) acc -= sT[(16 * blk + r) * LD64 + 16 * blk + s] * x[s];
      x[r] = acc;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) sA[(16 * blk + r) * LD64 + 16 * blk + c] = x[r];
  }
  for (int e = tid; e < CH * CH; e += NTHR) {
    const int r = e / CH, s = e % CH;
    if ((s >> 4) > (r >> 4)) sA[r * LD64 + s] = 0.f;
  }
  __syncthreads();
  for (int dist = 1; dist <= 3; ++dist) {
    const int nb = 4 - dist;
    for (int e = tid; e < nb * 256; e += NTHR) {
      const int j = e >> 8, i = j + dist, r = (e & 255) >> 4, c = e & 15;
      float acc = 0.f;
      for (int s = 16 * j; s < 16 * i; ++s)
        acc += sT[(16 * i + r) * LD64 + s] * sA[s * LD64 + 16 * j + c];
      sM[e] = acc;
    }
    __syncthreads();
    for (int e = tid; e < nb * 256; e += NTHR) {
      const int j = e >> 8, i = j + dist, r = (e & 255) >> 4, c = e & 15;
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < 16; ++u)
        acc += sA[(16 * i + r) * LD64 + 16 * i + u] * sM[(e & ~255) + u * 16 + c];
      sA[(16 * i + r) * LD64 + 16 * j + c] = -acc;
    }
    __syncthreads();
  }
}

}  // namespace gdr2

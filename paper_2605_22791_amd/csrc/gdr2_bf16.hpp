// bf16 matrix-core building blocks for gfx950 (CDNA4).
//
// Every contraction of the bf16 path runs on v_mfma_f32_16x16x32_bf16
// (16x16 output tile, K = 32, fp32 accumulate).  Operand fragment of one lane
// l (g = l / 16, r16 = l % 16):
//     A operand  A[m = r16][k = 8g + e], e = 0..7       (8 bf16)
//     B operand  B[k = 8g + e][n = r16]
//     C / D      C[4g + u][n = r16], u = 0..3           (4 fp32)
// Any permutation of k shared by A and B gives the same product.
//
// Products that must be fp32-accurate split each operand x into
// hi = bf16(x) and lo = bf16(x - hi) (16 significant bits together) and sum
// hi*hi + hi*lo + lo*hi (the bfloat16 split of Henry, Tang and Heinecke,
// ARITH 2019); an operand that is exactly bf16 (a raw input) has lo = 0 and
// drops its pass.
//
// Transposed fragments come from row-major bf16 tiles in LDS through the
// gfx950 transpose load ds_read_b64_tr_b16: inside each group of 16 lanes,
// output lane j, element i is element (j % 4) of the 8 bytes addressed by
// lane 4i + j/4.  Pointing lane 4i + q of group G at X[k0 + 8G + i][n0 + 4q]
// (and then at row + 4) therefore yields X[k0 + 8G + e][n0 + j], e = 0..7:
// the B fragment of a row-major X[k][n], or equally the A fragment of X^T.

#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdr2 {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf4 __attribute__((ext_vector_type(4)));
// 16 raw bytes as a native vector (HIP's uint4 is a struct, whose copies go
// through memory and keep staging arrays out of registers)
typedef unsigned u4v __attribute__((ext_vector_type(4)));

#define GDR2_LDS __attribute__((address_space(3)))

// Decay bookkeeping in base 2: G2 = log2(e) * G, factors 2^(G2_r - G2_s).
constexpr float kLog2e = 1.4426950408889634f;
// a diagonal block whose internal decay exceeds e^60 is formed element by element
constexpr float kDiagLimit2 = 60.f * kLog2e;

// 2^x on the transcendental unit (v_exp_f32)
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

struct Fr {  // split operand fragment
  bf8 hi, lo;
};

__device__ __forceinline__ f4 f4zero() { return f4{0.f, 0.f, 0.f, 0.f}; }

__device__ __forceinline__ f4 mma(bf8 a, bf8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// hi*hi + hi*lo + lo*hi
__device__ __forceinline__ f4 mma3(const Fr& a, const Fr& b, f4 c) {
  c = mma(a.lo, b.hi, c);
  c = mma(a.hi, b.lo, c);
  return mma(a.hi, b.hi, c);
}
// a split, b exact bf16
__device__ __forceinline__ f4 mma2a(const Fr& a, bf8 b, f4 c) {
  c = mma(a.lo, b, c);
  return mma(a.hi, b, c);
}
// a exact bf16, b split
__device__ __forceinline__ f4 mma2b(bf8 a, const Fr& b, f4 c) {
  c = mma(a, b.lo, c);
  return mma(a, b.hi, c);
}

__device__ __forceinline__ bf8 round8(const float (&x)[8]) {
  bf8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (__bf16)x[e];
  return r;
}
__device__ __forceinline__ Fr split8(const float (&x)[8]) {
  Fr f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const __bf16 h = (__bf16)x[e];
    f.hi[e] = h;
    f.lo[e] = (__bf16)(x[e] - (float)h);
  }
  return f;
}
__device__ __forceinline__ bf8 neg8(bf8 x) {
  uint4 u = __builtin_bit_cast(uint4, x);
  u.x ^= 0x80008000u;
  u.y ^= 0x80008000u;
  u.z ^= 0x80008000u;
  u.w ^= 0x80008000u;
  return __builtin_bit_cast(bf8, u);
}
__device__ __forceinline__ void unpack8(bf8 x, float (&o)[8]) {
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (float)x[e];
}
__device__ __forceinline__ void unpack8(u4v u, float (&o)[8]) { unpack8(__builtin_bit_cast(bf8, u), o); }
__device__ __forceinline__ u4v ldg16(const void* p) { return *reinterpret_cast<const u4v*>(p); }
__device__ __forceinline__ void sts16(void* p, u4v x) { *reinterpret_cast<u4v*>(p) = x; }

// 16-byte LDS / global accessors
__device__ __forceinline__ bf8 ld8(const __bf16* p) { return *reinterpret_cast<const bf8*>(p); }
__device__ __forceinline__ void st8(__bf16* p, bf8 x) { *reinterpret_cast<bf8*>(p) = x; }
__device__ __forceinline__ void ldf8(const float* p, float (&o)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
// four consecutive bf16 (8 bytes)
__device__ __forceinline__ void st4(__bf16* p, float a, float b, float c, float d) {
  bf4 v;
  v[0] = (__bf16)a; v[1] = (__bf16)b; v[2] = (__bf16)c; v[3] = (__bf16)d;
  *reinterpret_cast<bf4*>(p) = v;
}
// split four consecutive values into hi and lo planes
__device__ __forceinline__ void st4split(__bf16* phi, __bf16* plo, const f4& x) {
  bf4 h, l;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const __bf16 t = (__bf16)x[u];
    h[u] = t;
    l[u] = (__bf16)(x[u] - (float)t);
  }
  *reinterpret_cast<bf4*>(phi) = h;
  *reinterpret_cast<bf4*>(plo) = l;
}

// Transposed fragment of a row-major bf16 LDS tile X (row stride ld elements):
// lane (G, j) receives X[k0 + 8G + e][n0 + j], e = 0..7.  ld and n0 must be
// multiples of 4.
__device__ __forceinline__ bf8 ld_tr8(const __bf16* X, int ld, int k0, int n0, int lane) {
  const int G = lane >> 4, s = lane & 15;
  const __bf16* p0 = X + (k0 + 8 * G + (s >> 2)) * ld + n0 + 4 * (s & 3);
  const __bf16* p1 = p0 + 4 * ld;
  const bf4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((GDR2_LDS bf4*)(p0));
  const bf4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((GDR2_LDS bf4*)(p1));
  bf8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}

// Transposed fragment from two per-lane addresses: p0 points at the 4
// consecutive elements (row 8G + i, cols 4q..4q+3) that lane 4i + q of group
// G contributes for rows 0..3 of its group, p1 at rows 4..7.  Used where the
// source tile is stored in fragment order rather than row-major.
__device__ __forceinline__ bf8 ld_tr8p(const __bf16* p0, const __bf16* p1) {
  const bf4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((GDR2_LDS bf4*)(p0));
  const bf4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((GDR2_LDS bf4*)(p1));
  bf8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}

// v_mfma_f32_16x16x4_f32: lane l supplies A[l%16][l/16] and B[l/16][l%16].
__device__ __forceinline__ f4 mfma_f32(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

}  // namespace gdr2

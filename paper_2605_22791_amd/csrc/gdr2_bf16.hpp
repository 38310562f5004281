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

// 4 x 4 transpose inside each quad of lanes (lanes 4m + j, j = 0..3): on entry
// lane j holds v[u] = M[j][u], on exit v[k] = M[k][j].  Two stages of 2 x 2
// block swaps with DPP quad permutations (xor 1, then xor 2).
__device__ __forceinline__ float dpp_quad(float x, int ctrl_xor) {
  const int v = __float_as_int(x);
  return __int_as_float(ctrl_xor == 1 ? __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false)
                                      : __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
}
__device__ __forceinline__ void quad_transpose(float (&v)[4], int j) {
  {
    const bool odd = (j & 1) != 0;
    const float a = dpp_quad(odd ? v[0] : v[1], 1), b = dpp_quad(odd ? v[2] : v[3], 1);
    if (odd) {
      v[0] = a;
      v[2] = b;
    } else {
      v[1] = a;
      v[3] = b;
    }
  }
  {
    const bool hi = (j & 2) != 0;
    const float a = dpp_quad(hi ? v[0] : v[2], 2), b = dpp_quad(hi ? v[1] : v[3], 2);
    if (hi) {
      v[0] = a;
      v[1] = b;
    } else {
      v[2] = a;
      v[3] = b;
    }
  }
}

// ---- chunk states between the scans and the chunk backward -----------------
// The bf16 path keeps the chunk-start states h_n (forward scan) and the
// gradients dh_n of the chunk-end states (reverse scan) for the chunk backward
// in fp16 with one power-of-two scale per 16 x 32 block (16 key rows, 32 value
// columns): the block's largest magnitude m is mapped into [2^14, 2^15), so no
// value overflows fp16 and every value within 2^28 of m keeps fp16's 11
// significant bits.  The state recursions themselves stay in fp32; only the
// copies the chunk backward reads are rounded (relative 2^-12 per element,
// against the bf16 rounding 2^-9 of the operator's outputs).
//   H16 (Dk x Dv)            fp16 rows, each 32-value group in the permuted K order
//                            (store_state_f16), per chunk-head
//   HSC (Dk / 16, Dv / 32)   fp32 inverse scales (x = fp16 value * HSC)
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
// 16 x 16 x 32 product of fp16 fragments, fp32 accumulation: the products of
// fp16 values are exact in fp32
__device__ __forceinline__ f4 mma_f16(f16x8 a, f16x8 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Largest value over the wave (x >= 0): DPP steps inside each 16-lane row
// (quad swaps, then the half-row and row mirrors), then the four row maxima
// read as scalars.
template <int CTRL>
__device__ __forceinline__ float dppf(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dppf<0xB1>(x));   // quad_perm [1, 0, 3, 2]
  x = fmaxf(x, dppf<0x4E>(x));   // quad_perm [2, 3, 0, 1]
  x = fmaxf(x, dppf<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dppf<0x140>(x));  // row_mirror
  const int b = __float_as_int(x);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(b, 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(b, 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(b, 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(b, 48));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}
// The value the same lane holds in the partner 16-lane row: rows 2k and 2k + 1
// (row_partner16), rows k and k + 2 (row_partner32), from one v_permlane16_swap
// / v_permlane32_swap of the value with itself (VALU, no LDS round trip).  odd:
// the lane's row is odd; upper: its row is 2 or 3.
__device__ __forceinline__ float row_partner16(float x, bool odd) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(odd ? r[0] : r[1]);
}
__device__ __forceinline__ float row_partner32(float x, bool upper) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(upper ? r[0] : r[1]);
}
// 4 x 4 transpose across the four 16-lane rows, lane by lane: on entry row R
// holds v[u] = M[R][u], on exit v[u] = M[u][R].  permlane16_swap(a, b) trades
// a's odd rows for b's even rows, permlane32_swap(a, b) a's rows 2, 3 for b's
// rows 0, 1.
__device__ __forceinline__ void row_transpose4(f4& v) {
  auto sw16 = [](float& a, float& b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  };
  auto sw32 = [](float& a, float& b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  };
  float x0 = v[0], x1 = v[1], x2 = v[2], x3 = v[3];
  sw16(x0, x1);
  sw16(x2, x3);
  sw32(x0, x2);
  sw32(x1, x3);
  v[0] = x0, v[1] = x1, v[2] = x2, v[3] = x3;
}
// Sum over the 16 lanes of each row (every lane gets it): quad swaps, then the
// half-row and row mirrors; with HALF, over each 8-lane half-row instead.
template <bool HALF = false>
__device__ __forceinline__ float row_sum(float x) {
  x += dppf<0xB1>(x);   // quad_perm [1, 0, 3, 2]
  x += dppf<0x4E>(x);   // quad_perm [2, 3, 0, 1]
  x += dppf<0x141>(x);  // row_half_mirror
  if constexpr (!HALF) x += dppf<0x140>(x);  // row_mirror
  return x;
}
// Power-of-two exponent that maps the block maximum m >= 0 into [2^14, 2^15)
// (0 for m = 0 or a non-finite m, whose values then pass through unscaled).
__device__ __forceinline__ int state_shift(float m) {
  if (!(m > 0.f) || !(m <= 3.0e38f)) return 0;
  int e;
  (void)frexpf(m, &e);  // m = f 2^e, f in [0.5, 1)
  const int sh = 15 - e;
  return sh < -120 ? -120 : (sh > 120 ? 120 : sh);
}
// The wave's state tiles s[t] are an MFMA accumulator layout: lane (g, r16)
// holds rows 4 g + u of the wave's 16 key rows, column 16 t + r16 of its
// columns; value blocks t, t + 1 share one scale (TPW even).
// state_shifts: the scale exponent of each of the wave's TPW / 2 blocks.
template <int TPW>
__device__ __forceinline__ void state_shifts(const f4 (&s)[TPW], int (&sh)[TPW / 2]) {
  static_assert(TPW % 2 == 0, "pairs of 16-column tiles per scale block");
#pragma unroll
  for (int t2 = 0; t2 < TPW; t2 += 2) {
    float mx = 0.f;
#pragma unroll
    for (int t = t2; t < t2 + 2; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) mx = fmaxf(mx, fabsf(s[t][u]));
    sh[t2 / 2] = state_shift(wave_max(mx));
  }
}
// store_state_f16: the tiles as fp16 with their scales, each 32-column group
// in the permuted K order of the fragments (columns 4 m + e and 16 + 4 m + e,
// e = 0..3, side by side at 8 m + e and 8 m + 4 + e).  h0 points at the wave's
// first row and column in the chunk's H16 (row stride ld; the column a multiple
// of 32), sc at its first block's scale; tiles 2 t2 and 2 t2 + 1 form 32-column
// block t2.  A quad transpose gives each lane four consecutive columns of one
// row from both tiles of a block: one 16-byte store.
template <int TPW>
__device__ __forceinline__ void store_state_f16(const f4 (&s)[TPW], const int (&sh)[TPW / 2], _Float16* h0, int ld,
                                                float* sc, int lane) {
  static_assert(TPW % 2 == 0, "whole 32-column blocks");
  const int g = lane >> 4, r16 = lane & 15, m = r16 >> 2, j = r16 & 3;
#pragma unroll
  for (int t2 = 0; t2 < TPW / 2; ++t2) {
    const float f = ldexpf(1.f, sh[t2]);
    float v0[4] = {s[2 * t2][0] * f, s[2 * t2][1] * f, s[2 * t2][2] * f, s[2 * t2][3] * f};
    float v1[4] = {s[2 * t2 + 1][0] * f, s[2 * t2 + 1][1] * f, s[2 * t2 + 1][2] * f, s[2 * t2 + 1][3] * f};
    quad_transpose(v0, j);
    quad_transpose(v1, j);
    const f16x8 hv = {(_Float16)v0[0], (_Float16)v0[1], (_Float16)v0[2], (_Float16)v0[3],
                      (_Float16)v1[0], (_Float16)v1[1], (_Float16)v1[2], (_Float16)v1[3]};
    *reinterpret_cast<f16x8*>(h0 + (size_t)(4 * g + j) * ld + 32 * t2 + 8 * m) = hv;
  }
  // every lane writes the (wave-uniform) scales: no branch around the store
#pragma unroll
  for (int t2 = 0; t2 < TPW / 2; ++t2) sc[t2] = ldexpf(1.f, -sh[t2]);
}
// store_tile_f16: one 16 x 16 accumulator tile (lane (g, r16) holds rows
// 4 g + u, column r16) as a 512-byte fp16 block of 16 x 16 x 16 operand
// fragments, scaled by 2^sh (sh = state_shift of the tile's largest
// magnitude): lane l's 8 bytes hold column l % 16 (the fragment's row or
// column) and rows 4 (l / 16) + u (its K elements).  Lane 0 writes the inverse
// scale to *sc.
__device__ __forceinline__ void store_tile_f16(const f4& x, int sh, _Float16* blk, float* sc, int lane) {
  const float f = ldexpf(1.f, sh);
  const f16x4 v = {(_Float16)(x[0] * f), (_Float16)(x[1] * f), (_Float16)(x[2] * f), (_Float16)(x[3] * f)};
  *reinterpret_cast<f16x4*>(blk + 4 * lane) = v;
  if (lane == 0) *sc = ldexpf(1.f, -sh);
}
__device__ __forceinline__ int tile_shift(const f4& x) {
  return state_shift(wave_max(fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3])))));
}
// store_frag_f16: a 16 x 32 tile held as two MFMA accumulator tiles (s[0]:
// columns 0..15, s[1]: columns 16..31; lane (g, r16) holds rows 4 g + u,
// column r16) as one fp16 permuted fragment block (1 KB, the layout of
// gdr2_kernels.hpp's permuted blocks: lane l holds row l % 16 and columns
// 4 (l / 16) + e, 16 + 4 (l / 16) + e), scaled by 2^sh.  After a quad
// transpose each lane holds four consecutive columns of one row from either
// tile, which are exactly the two halves of one fragment lane's 16 bytes.
__device__ __forceinline__ void store_frag_f16(const f4 (&s)[2], int sh, _Float16* blk, int lane) {
  const int g = lane >> 4, r16 = lane & 15, m = r16 >> 2, j = r16 & 3;
  const float f = ldexpf(1.f, sh);
  float v0[4] = {s[0][0] * f, s[0][1] * f, s[0][2] * f, s[0][3] * f};
  float v1[4] = {s[1][0] * f, s[1][1] * f, s[1][2] * f, s[1][3] * f};
  quad_transpose(v0, j);
  quad_transpose(v1, j);
  const f16x8 hv = {(_Float16)v0[0], (_Float16)v0[1], (_Float16)v0[2], (_Float16)v0[3],
                    (_Float16)v1[0], (_Float16)v1[1], (_Float16)v1[2], (_Float16)v1[3]};
  // row 4 g + j, column group m -> fragment lane (m, 4 g + j)
  *reinterpret_cast<f16x8*>(blk + 8 * (16 * m + 4 * g + j)) = hv;
}
// One lane's fp16 fragment (8 values), scaled back and split hi / lo.
__device__ __forceinline__ Fr frag_f16_split(u4v raw, float inv) {
  const f16x8 h = __builtin_bit_cast(f16x8, raw);
  float x[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (float)h[e] * inv;
  return split8(x);
}

// Eight consecutive values of one row of a stored state, back in fp32.
__device__ __forceinline__ void load_state8(u4v raw, float inv, float (&x)[8]) {
  const f16x8 h = __builtin_bit_cast(f16x8, raw);
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (float)h[e] * inv;
}

// v_mfma_f32_16x16x4_f32: lane l supplies A[l%16][l/16] and B[l/16][l%16].
__device__ __forceinline__ f4 mfma_f32(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

}  // namespace gdr2

// Chunk-parallel backward of the bf16 path (gfx950), App. B.2 - B.5 in one
// kernel: one 4-wave workgroup per chunk-head, two workgroups per CU.
//
// Per chunk it reads the chunk-start state h = S_0 and the gradient dh of the
// chunk-end state (fp16 [Dk][Dv] with block scales and each 32-value group in
// the permuted K order, store_state_f16), R (fp16 fragment blocks with block
// scales, store_frag_f16) from the scan, dR from the reverse scan and
// A = (I + T)^{-1} from the intra-chunk recompute (16 x 16 blocks: dR split
// bf16, A fp16 with block scales, store_tile_f16), and q, k, v, b, w, g, dO.
//
// Because R = A (Z - Ebar h) (App. A.2), the gate-aware WY VJP of App. B.2
// needs neither dA nor dY:
//     dZ = A^T dR                         (dv = dZ * w, dw = dZ * v)
//     dT = -tril(dZ R^T, -1)              (= -tril(A^T dA A^T, -1))
//     dEbar_WY = A^T dY = -dZ h^T
//     dA_qk = tril(scale dO R^T)
// and App. B.3 - B.5 become, with dEg = dEbar * gamma, dKg = dKbar / gamma,
// factors 2^(G2_r - G2_s) for r >= s and X1 = dZ h^T, X2 = dO h^T, X3 = R dh^T:
//     dEg_r = -gamma_r X1_r + sum_{s<r}  dT[r][s] k_s 2^(G2_r - G2_s)
//     dq_r  = scale gamma_r X2_r + sum_{s<=r} dA_qk[r][s] k_s 2^(G2_r - G2_s)
//     dKg_s = sum_{r>s} dT[r][s] (b k)_r 2^(G2_r - G2_s)
//             + sum_{r>=s} dA_qk[r][s] q_r 2^(G2_r - G2_s) + tail_s X3_s
//     db = dEg k,  dk = dEg b + dKg,  dG = dq q - dKg k + dEg b k
//     dG_{C-1} += gamma_C rowsum(dh * h) + sum_r X3_r k_r tail_r
//     dlog_alpha = reverse cumulative sum of dG over the chunk
// (tail_r = gamma_C / gamma_r).
//
// X3 is formed from the fp16 copies of R and dh as they are stored (their
// products are exact in fp32); X1 and X2 from the split h.
//
// Work split: wave i owns the 16 chunk rows of block i: its dZ rows, the dT /
// dA_qk tiles (i, j <= i) and every output tile (i, key block).  The key
// blocks run in a loop; each stages its h and dh rows, its G2, k, b, q columns
// and the decay-scaled operands of the decay products in LDS while the next
// block's loads are in flight.  dT and dA_qk live in LDS transposed ([s][r],
// split hi/lo) so that both the row-r and the column-s operands of the decay
// products are plain or transposed reads.  Cross-lane sums (the staging's
// prefix sums over a block's rows, the dh.h row sums, the dG suffix sums) use
// DPP moves inside 16-lane rows and the permlane swaps across rows, never an
// LDS round trip.  The outputs leave as whole 128-byte row lines (bf16 dq, dk,
// db of four key blocks, fp32 ones of two), and workgroups take the key heads
// fastest in launch order, so that the resident ones share token rows.
//
// Decay factors (App. D.4 / the forward kernels), with 16-row blocks j and
// G2f_j, G2l_j the cumulative log2-decay at their first and last rows: for the
// products over s <= r of row block i the factor 2^(G2_r - G2_s) is
//     2^(G2_r - G2f_i) * 2^(G2f_i - G2l_j) * 2^(G2l_j - G2_s)        (s in block j),
// the last part inside the operand k_s eR_s, which is the same for every row
// block and is built once per key block, the middle one applied to block j's
// 16-deep product, the first one after the sum.  The products over r >= s of
// key-row block i use b_r k_r eL_r and q_r eL_r with eL_r = 2^(G2_r - G2f_j)
// and the block factor 2^(G2f_j - G2l_i).  Every part is <= 1 except a
// diagonal block's factor, bounded by one block's decay; a diagonal block
// whose decay exceeds e^60 is formed element by element.
//
// Precision: every product is fp32-accurate on its operands (split hi/lo; dO
// is exact bf16; X3 and the dT / dA_qk tiles multiply fp16 operands exactly:
// the stored copies of R and dh, and dZ split in fp16 hi / lo under a
// power-of-two scale, which keeps 22 bits relative to the wave's largest dZ).
//
// Fused input stage (FUSED; App. C.1, App. D.2): q and k arrive raw and are
// normalised as they are staged, with the inverse norms the forward kept; the
// log-decay is formed from the decay projection f on staging, and the stored
// gradient is df = dg * (-exp(a) sigmoid(f + delta)) instead of dg, with the
// per-workgroup sums that give ddelta and da.  dq and dk remain the gradients
// of the normalised q, k: the normalisation VJP needs whole rows and follows in
// its own kernel.

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

// LDS layouts.  The 16-byte pieces of a row are permuted by an XOR with a
// function of the row, chosen so that every access of the key-block loop is
// free of bank conflicts on gfx950: a 16-byte read serves 16 lanes per cycle
// over 64 banks (the two lane quads of each half wave with even, then odd,
// quad-index parity), 8-byte reads 32 lanes over 64 banks, and 4-byte accesses
// and all writes 32 banks.  Every element of an array is addressed through its
// function below, writes and reads alike.
//   dT^T, dA_qk^T planes [64][LP] bf16:   8-element pieces ^ ((r >> 3) & 1)                   (LP = 80)
//                                         8-element pieces ^ ((r & 7) ^ ((r >> 3) & 1))       (LP = 64)
//   log2-decay sums [16][80] fp32:        4-element pieces ^ (((r >> 2) & 1) ^ (((r >> 2) & 3) << 1))
//   k, b, q columns [16][64] bf16:        8-element pieces ^ ((r >> 1) & 7)
//   h (bf16 hi / lo), dh (fp16) rows [16][DV + 16]:  8-element pieces ^ (r & 1)
//   decay-scaled operands [64][16] bf16 hi / lo (rows s, key channels): plain
// Among the conflict-free choices these keep the loop's addresses few: most
// accesses differ from another by a lane-independent constant.  The padded
// planes (LP = 80) need 8 KB more than LP = 64, which the fused stage's
// tables leave no room for.  Consecutive planes and k / b / q arrays sit 16
// bytes further apart than their size: reads of the same element in two of
// them are then not paired into one ds_read2st64_b64, whose halves are served
// like 8-byte writes (32 banks, 16 lanes per cycle) and conflict here.
template <int LP>
__device__ __forceinline__ int plane_ix(int r, int c) {
  const int f = LP == 80 ? ((r >> 3) & 1) : ((r & 7) ^ ((r >> 3) & 1));
  return r * LP + ((((c >> 3) ^ f) << 3) | (c & 7));
}
constexpr int kTabLd = 80;
__device__ __forceinline__ int tab_ix(int r, int c) {
  return r * kTabLd + ((((c >> 2) ^ ((r >> 2) & 1) ^ (((r >> 2) & 3) << 1)) << 2) | (c & 3));
}
__device__ __forceinline__ int col_ix(int r, int c) { return r * 64 + ((((c >> 3) ^ ((r >> 1) & 7)) << 3) | (c & 7)); }
template <int LH>
__device__ __forceinline__ int row_ix(int r, int c) {
  return r * LH + ((((c >> 3) ^ (r & 1)) << 3) | (c & 7));
}

template <int DK, int DV, bool FUSED>
struct BChunkCfg {
  static constexpr int NTHR = 256;
  static constexpr int NCB = DK / 16, NVB = DV / 16, KV = DV / 32;
  static constexpr int LP = FUSED ? 64 : 80;  // dT^T / dA_qk^T plane rows (plane_ix)
  static constexpr int LH = DV + 16;          // h (bf16 hi, lo) and dh (fp16) rows of a key block [16][LH] (row_ix)
  // region 1: dR (fragment blocks, prologue) -> dT^T / dA_qk^T planes
  static constexpr int SZ_DR = (int)WsBf16::dr(DV), SZ_AM = (int)WsBf16::am();
  static constexpr int OFF_T = 0;
  static constexpr int PSZ = 64 * LP + 8;  // one plane, elements
  static constexpr int CSZ = 16 * 64 + 8;  // one k / b / q array, elements
  static constexpr int SZ_T = 4 * PSZ * 2;
  // region 2: A (fragment blocks, prologue) -> the staged key block
  static constexpr int OFF_S = OFF_T + SZ_T;
  static constexpr int SZ_TAB = 16 * kTabLd * 4;
  static constexpr int OFF_G = OFF_S;            // in-block log2-decay sums [16][64] fp32 (tab_ix)
  static constexpr int OFF_XO = OFF_G + SZ_TAB;  // k eR, b k eL, q eL, hi / lo [6][64][16] bf16
  static constexpr int OFF_X = OFF_XO + 6 * 64 * 16 * 2;  // k, b, q columns [16][64] bf16 (col_ix)
  static constexpr int OFF_H = OFF_X + 3 * CSZ * 2;
  static constexpr int OFF_END_S = OFF_H + 3 * 16 * LH * 2;
  // small exchange arrays
  static constexpr int OFF_BK = OFF_END_S;              // block totals / first rows [2][4][16]
  static constexpr int OFF_HH = OFF_BK + 2 * 4 * 16 * 4;  // rowsum(dh * h)      [2][16]
  static constexpr int OFF_BT = OFF_HH + 2 * 16 * 4;      // dG block totals     [2][4][16]
  static constexpr int OFF_TL = OFF_BT + 2 * 4 * 16 * 4;  // tail-key sums       [2][4][16]
  static constexpr int LDS_BASE = OFF_TL + 2 * 4 * 16 * 4;
  // fused stage: f + delta of the staged key block [16][64] (tab_ix), the decay
  // bias of the key head [DK], the inverse norms of the chunk's q and k rows [2][64]
  static constexpr int OFF_XS = LDS_BASE;
  static constexpr int OFF_DL = OFF_XS + SZ_TAB;
  static constexpr int OFF_RN = OFF_DL + DK * 4;
  static constexpr int LDS = FUSED ? OFF_RN + 2 * 64 * 4 : LDS_BASE;
  // prologue: dR into region 1, A then R (fp16 fragment blocks) into region 2, by
  // direct global -> LDS loads of 1 KB per wave instruction
  static constexpr int SZ_R = (int)WsBf16::rs(DV);
  static constexpr int OFF_R = OFF_S + SZ_AM;
  static constexpr int NKB = (SZ_DR + SZ_AM + SZ_R) / 1024;
  static_assert(SZ_DR <= SZ_T && SZ_AM + SZ_R <= OFF_END_S - OFF_S, "prologue operands fit their regions");
  static_assert(NKB % (NTHR / 64) == 0 && SZ_DR % 1024 == 0 && SZ_AM % 1024 == 0, "whole blocks per wave");
  static_assert(LDS <= 80 * 1024, "two workgroups per CU");
  static_assert(16 * DV / 8 <= NTHR, "one 16-byte piece of h / dh per thread");
};

// 16 x 16 x 16 products on split operands (lane l: row / column l % 16, K
// elements 4 (l / 16) + e): one decay-scaled key block per K-step
struct Fr4 {
  bf4 hi, lo;
};
typedef short s4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f4 mma16(bf4 a, bf4 b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s4v, a), __builtin_bit_cast(s4v, b), c, 0, 0, 0);
}
// the cross terms first, as in mma3
__device__ __forceinline__ f4 mma3_16(const Fr4& a, const Fr4& b, f4 c) {
  c = mma16(a.lo, b.hi, c);
  c = mma16(a.hi, b.lo, c);
  return mma16(a.hi, b.hi, c);
}
__device__ __forceinline__ bf4 ld_tr4(const __bf16* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((GDR2_LDS bf4*)(p));
}

__device__ __forceinline__ bf8 cat8(bf4 x, bf4 y) {
  bf8 r;
  r[0] = x[0]; r[1] = x[1]; r[2] = x[2]; r[3] = x[3];
  r[4] = y[0]; r[5] = y[1]; r[6] = y[2]; r[7] = y[3];
  return r;
}
__device__ __forceinline__ float4 ldg_f4(const float* p) { return *reinterpret_cast<const float4*>(p); }
typedef unsigned u2v __attribute__((ext_vector_type(2)));
// (x, y | z, w) -> one permlane16 swap of x with z and of y with w: between
// "8 consecutive values at 32 p + {0, 16, 8, 24}[g]" and "4 values at 32 p + 4 g
// then 4 at 32 p + 16 + 4 g" (g: the lane's 16-lane row), in either direction
__device__ __forceinline__ u4v unswap_pair(u4v x) {
  const auto r0 = __builtin_amdgcn_permlane16_swap(x[0], x[2], false, false);
  const auto r1 = __builtin_amdgcn_permlane16_swap(x[1], x[3], false, false);
  return u4v{r0[0], r1[0], r0[1], r1[1]};
}
// An empty asm that reads and rewrites x: the loads that produced x have
// completed there.  One vmcnt counts loads and stores in issue order, and a
// wait for a load that has stores of a path-dependent count behind it becomes
// vmcnt(0); settling the prefetched operands before a key block's stores keeps
// the later waits for them from waiting for those stores too.
__device__ __forceinline__ void settle(float& x) { asm volatile("" : "+v"(x)::"memory"); }
__device__ __forceinline__ void settle(u4v& x) { asm volatile("" : "+v"(x)::"memory"); }
__device__ __forceinline__ void settle(bf4& x) {
  u2v u = __builtin_bit_cast(u2v, x);
  asm volatile("" : "+v"(u)::"memory");
  x = __builtin_bit_cast(bf4, u);
}
__device__ __forceinline__ void settle(float4& x) {
  f4 u = __builtin_bit_cast(f4, x);
  asm volatile("" : "+v"(u)::"memory");
  x = __builtin_bit_cast(float4, u);
}
// four consecutive outputs of one row: 8-byte bf16 or 16-byte fp32 store
__device__ __forceinline__ void store_row4(__bf16* p, const float (&v)[4]) {
  *reinterpret_cast<bf4*>(p) = bf4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
}
__device__ __forceinline__ void store_row4(float* p, const float (&v)[4]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
}
// four outputs as bf16, packed for a later 8-byte store
__device__ __forceinline__ uint2 pack_bf4(const float (&v)[4]) {
  return __builtin_bit_cast(uint2, bf4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]});
}
__device__ __forceinline__ void add_row4(const float* p, float (&v)[4]) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  v[0] += x.x;
  v[1] += x.y;
  v[2] += x.z;
  v[3] += x.w;
}

// element j (0..3) of four per-block values, j lane-dependent
__device__ __forceinline__ float pick4(const float (&x)[4], int j) {
  return j == 0 ? x[0] : (j == 1 ? x[1] : (j == 2 ? x[2] : x[3]));
}

template <int DK, int DV, bool FUSED>
__global__ __launch_bounds__(256, 2) void bchunk_bf16_kernel(BChunkBf16Args a) {
  using C = BChunkCfg<DK, DV, FUSED>;
  constexpr int NCB = C::NCB, NVB = C::NVB, KV = C::KV, NKB = C::NKB;
  constexpr int LH = C::LH, LP = C::LP;

  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* sTh = reinterpret_cast<__bf16*>(smem + C::OFF_T);  // dT^T [s][r]
  __bf16* sTl = sTh + C::PSZ;
  __bf16* sAh = sTl + C::PSZ;  // dA_qk^T [s][r]
  __bf16* sAl = sAh + C::PSZ;
  const unsigned char* sDR = smem + C::OFF_T;  // prologue: dR fragment blocks
  const unsigned char* sAm = smem + C::OFF_S;  // prologue: A fragment blocks
  const unsigned char* sR = smem + C::OFF_R;   // prologue: R, fp16 fragment blocks [row block][KV]
  float* sG = reinterpret_cast<float*>(smem + C::OFF_G);    // in-block cumsum of log2-decay [c][s]
  // decay-scaled operands of the products over the key block, split hi / lo, [s][c]:
  // k_s eR_s (eR_s = 2^(G2 at the last row of s's 16-row block - G2_s)), b_r k_r eL_r
  // and q_r eL_r (eL_r = 2^(G2_r - G2 at the first row of r's block))
  __bf16* sXh = reinterpret_cast<__bf16*>(smem + C::OFF_XO);
  __bf16* sXl = sXh + 64 * 16;
  __bf16* sBh = sXl + 64 * 16;
  __bf16* sBl = sBh + 64 * 16;
  __bf16* sQh = sBl + 64 * 16;
  __bf16* sQl = sQh + 64 * 16;
  __bf16* sKc = reinterpret_cast<__bf16*>(smem + C::OFF_X);  // k [c][s]
  __bf16* sBc = sKc + C::CSZ;
  __bf16* sQc = sBc + C::CSZ;
  __bf16* sHh = reinterpret_cast<__bf16*>(smem + C::OFF_H);  // h [c][v], permuted K order
  __bf16* sHl = sHh + 16 * LH;
  _Float16* sD16 = reinterpret_cast<_Float16*>(sHl + 16 * LH);  // dh [c][v] as stored: fp16, permuted K order
  float* sBK = reinterpret_cast<float*>(smem + C::OFF_BK);  // [0]: block totals, [1]: first rows
  float* sHH = reinterpret_cast<float*>(smem + C::OFF_HH);
  float* sBT = reinterpret_cast<float*>(smem + C::OFF_BT);
  float* sTL = reinterpret_cast<float*>(smem + C::OFF_TL);
  float* sXS = reinterpret_cast<float*>(smem + C::OFF_XS);  // fused stage: f + delta [c][s]
  float* sDL = reinterpret_cast<float*>(smem + C::OFF_DL);  // fused stage: delta [c]
  float* sRN = reinterpret_cast<float*>(smem + C::OFF_RN);  // fused stage: 1/||q||, 1/||k|| [2][64]

  // the wave index as a scalar: branches on the row block are uniform
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r16 = lane & 15;
  const bool podd = (g & 1) != 0, pup = g >= 2;  // the lane's 16-lane row: odd; 2 or 3
  ChunkPos cp;
  // the grid covers the key heads; this launch takes value head gj of each group
  // workgroups in launch order take the key heads fastest, then the chunks: the
  // ones resident together read and write neighbouring parts of the same token rows
  const int lin = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int bx = (lin / gridDim.y) % gridDim.x, by = lin % gridDim.y, bz = lin / (gridDim.y * gridDim.x);
  const int h = by * a.G + a.gj, H = a.H;
  // fused stage: this workgroup's slot of the decay-parameter partials
  const size_t pslot = ((size_t)(bz * gridDim.x + bx) * H + h) * 4 + wave;
  if (!chunk_pos(a.vl, bx, h, bz, a.T, H, a.NT, cp)) {
    if constexpr (FUSED) {  // an unused slot of a packed grid adds zeros
      for (int c = lane; c < DK; c += 64) a.PD[pslot * DK + c] = 0.f;
      if (lane == 0) a.PA[pslot] = 0.f;
    }
    return;
  }
  const size_t ch = cp.ch, row0 = cp.row0;
  const size_t kch = key_ch(a.vl, ch, a.H, a.G, a.NT);  // the key head's chunk (A)
  // Rows in use.  Loads read in-range rows only (rows past a partial chunk's
  // end re-read its last row); g, k and dO of those rows are then taken as
  // zero, which makes every term they could add to a valid row vanish (their
  // dT, dA_qk, dR and dG are zero), and their outputs are not written.
  const int len = cp.len;
  // key-side inputs (q, k, g, b) and gradients live on the H / G key heads
  // (value head h reads key head h / G); the fused stage keeps dq, dk in fp32
  // (partq; one rounding after its normalisation VJP)
  const int HK = H / a.G, hk = by;
  const bool partq = a.Pq != nullptr;
  const int gmode = a.gmode;  // 0: direct, 1 / 2 / 3: first / middle / last value head of a group
  const size_t KST = (size_t)HK * DK, VST = (size_t)H * DV;  // token strides
  const size_t kb0 = row0 * KST + (size_t)hk * DK, vb0 = row0 * VST + (size_t)h * DV;
  const size_t ko0 = kb0;  // key-side outputs
  const int i = wave;  // the row block this wave owns

  // per-chunk bases (uniform) and 32-bit lane offsets: KST = (H / G) Dk, VST = H Dv
  const __bf16* Qp = reinterpret_cast<const __bf16*>(a.q) + kb0;
  const __bf16* Kp = reinterpret_cast<const __bf16*>(a.k) + kb0;
  const __bf16* Bp = reinterpret_cast<const __bf16*>(a.b) + kb0;
  const float* Gp0 = a.g + kb0;
  __bf16* dQp = reinterpret_cast<__bf16*>(a.dq) + ko0;
  __bf16* dKp = reinterpret_cast<__bf16*>(a.dk) + ko0;
  __bf16* dBp = reinterpret_cast<__bf16*>(a.db) + ko0;
  float* pQp = partq ? a.Pq + ko0 : nullptr;
  float* pKp = partq ? a.Pk + ko0 : nullptr;
  float* dGp = a.dg + ko0;
  const __bf16* Vp = reinterpret_cast<const __bf16*>(a.v) + vb0;
  const __bf16* Wp = reinterpret_cast<const __bf16*>(a.w) + vb0;
  const __bf16* dOp = reinterpret_cast<const __bf16*>(a.dout) + vb0;
  __bf16* dVp = reinterpret_cast<__bf16*>(a.dv) + vb0;
  __bf16* dWp = reinterpret_cast<__bf16*>(a.dw) + vb0;
  const _Float16* Hc = a.Hs + ch * DK * DV;
  const _Float16* DHc = a.DH + ch * DK * DV;
  const float* Hscc = a.Hsc + ch * (WsBf16::hsc(DK, DV) / 4);
  const float* DHscc = a.DHsc + ch * (WsBf16::hsc(DK, DV) / 4);
  const _Float16* Rc = a.Rs + ch * (WsBf16::rs(DV) / 2);
  const float* Rscc = a.Rsc + ch * (WsBf16::rsc(DV) / 4);
  const int kst = HK * DK, kso = kst, vst = H * DV;

  // staging role: chunk row grow (block = wave), channels 16 cb + 4 cq + (0..3)
  const int rl = lane >> 2, cq = lane & 3, grow = 16 * wave + rl;
  const bool grin = grow < len;
  const int growc = min(grow, len - 1);
  // h / dh staging role: row hc of the key block, 16-byte piece hv / 8 (the fp16
  // copies keep each 32-value group in the permuted K order, so a piece is one
  // lane's fragment run: values 32 p + 4 q + (0..3) and 32 p + 16 + 4 q + (0..3))
  const int hc = (8 * tid) / DV, hv = (8 * tid) % DV;
  const bool hact = tid < 2 * DV;
  // Per-lane bases of the swizzled LDS accesses (element offsets; each equals
  // its index function, with the per-step part a compile-time offset):
  //   aH + 32 p              = row_ix(r16, 32 p + 8 g)                   h, dh fragments
  //   aHs                    = row_ix(hc, hv)                            h, dh staging
  //   aTr + 16 LP j          = plane_ix(16 j + 4 g + r16 / 4, 16 i + 4 (r16 % 4))   transposed plane reads
  //   aP3 + 16 j             = plane_ix(16 i + r16, 16 j + 4 g)          plane rows (LP = 80)
  //   aXr + 256 j            = (16 j + 4 g + r16 / 4) * 16 + 4 (r16 % 4)   decay-scaled operands, transposed
  //   aXs                    = grow * 16 + 4 cq                          their staging
  //   aE                     = tab_ix(r16, 16 i + 4 g),  aTs + 80 u = tab_ix(4 cq + u, 16 i + rl)
  //   aK4                    = col_ix(r16, 16 i + 4 g),  aKs[u / 2] + 64 (u % 2) = col_ix(4 cq + u, 16 i + rl)
  const int fT = ((r16 >> 2) & 1) ^ (((r16 >> 2) & 3) << 1), fTs = (cq & 1) ^ ((cq & 3) << 1);
  const int fK = (r16 >> 1) & 7;
  const int aH = r16 * LH + 8 * (g ^ (r16 & 1));
  const int aHs = hc * LH + 8 * ((hv >> 3) ^ (hc & 1));
  const int aTr = plane_ix<LP>(4 * g + (r16 >> 2), 16 * i + 4 * (r16 & 3));
  const int aP3 = plane_ix<LP>(16 * i + r16, 4 * g);
  const int aXr = (4 * g + (r16 >> 2)) * 16 + 4 * (r16 & 3);
  const int aXs = grow * 16 + 4 * cq;
  const int aE = r16 * kTabLd + 4 * ((4 * i + g) ^ fT);
  const int aTs = 4 * cq * kTabLd + 4 * ((4 * i + (rl >> 2)) ^ fTs) + (rl & 3);
  const int aK4 = r16 * 64 + 8 * ((2 * i + (g >> 1)) ^ fK) + 4 * (g & 1);
  const int aKs[2] = {4 * cq * 64 + 8 * ((2 * i + (rl >> 3)) ^ ((2 * cq) & 7)) + (rl & 7),
                      (4 * cq + 2) * 64 + 8 * ((2 * i + (rl >> 3)) ^ ((2 * cq + 1) & 7)) + (rl & 7)};
  // fused stage: exp(a) of the key head; its decay bias and the chunk's inverse
  // norms go to LDS (visible after the barrier that follows the prologue)
  float Adec = 0.f;
  if constexpr (FUSED) {
    Adec = expf(a.st.a_log[hk]);
    if (tid < DK) sDL[tid] = a.st.delta[(size_t)hk * DK + tid];
    if (tid < 128) {
      const float* rn = tid < 64 ? a.st.RQ : a.st.RK;
      sRN[tid] = rn[(row0 + min(tid & 63, len - 1)) * HK + hk];
    }
  }

  // ---- loads in flight from the start: dR and A (cooperative), this wave's dO
  // rows and the operands of key block 0
  {
    // wave w moves the 1 KB blocks w, w + 4, ... of dR | A | R straight into LDS
    const unsigned char* DRc = reinterpret_cast<const unsigned char*>(a.DR) + ch * WsBf16::dr(DV);
    const unsigned char* Amc = reinterpret_cast<const unsigned char*>(a.Am) + kch * WsBf16::am();  // A: per key head
    const unsigned char* Rcb = reinterpret_cast<const unsigned char*>(Rc);
#pragma unroll
    for (int m = 0; m < NKB / 4; ++m) {
      const int off = 1024 * (4 * m + wave);
      const unsigned char* src;
      unsigned char* dst;
      if (off < C::SZ_DR) {
        src = DRc + off;
        dst = smem + C::OFF_T + off;
      } else if (off < C::SZ_DR + C::SZ_AM) {
        // A's 1 KB pieces 4 and 6 hold tiles (sb, rb) = (2, 0..1) and (3, 0..1),
        // above the diagonal: not stored, never read
        if (off - C::SZ_DR == 4096 || off - C::SZ_DR == 6144) continue;
        src = Amc + (off - C::SZ_DR);
        dst = smem + C::OFF_S + (off - C::SZ_DR);
      } else {
        src = Rcb + (off - C::SZ_DR - C::SZ_AM);
        dst = smem + C::OFF_R + (off - C::SZ_DR - C::SZ_AM);
      }
      __builtin_amdgcn_global_load_lds((void*)(src + 16 * lane), (GDR2_LDS void*)dst, 16, 0, 0);
    }
  }
  // A's block scales (key block i, row block rb) in lanes rb < 4
  const float ascl = lane < 4 ? a.Amsc[kch * (WsBf16::amsc() / 4) + 4 * i + lane] : 0.f;
  // R's block scales: lane j * KV + p holds that of row block j, value block p
  const float rscl = lane < 4 * KV ? Rscc[lane] : 0.f;
  const auto rsc = [&](int blk) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(rscl), blk)); };
  // dO rows of block i as fragments (values 32 p + 4 g .. and 32 p + 16 + 4 g ..):
  // one 16-byte load of 8 consecutive values at 32 p + {0, 16, 8, 24}[g] and one
  // permlane swap per dword, which puts the two 4-value pieces where they belong
  // (the same swap, applied twice, is the identity)
  const int goff = 8 * (((g & 1) << 1) | (g >> 1));
  bf8 dof[KV];
#pragma unroll
  for (int p = 0; p < KV; ++p) {
    const int o = (min(16 * i + r16, len - 1)) * vst + 32 * p + goff;
    dof[p] = __builtin_bit_cast(bf8, unswap_pair(*reinterpret_cast<const u4v*>(dOp + o)));
  }
  float4 pg;
  u4v ph, pd;     // 8 fp16 values of h and dh
  float psh, psd;  // their inverse scales
  float pds;       // lane p < KV: the scale of dh's value block p (key block of the prefetch)
  float dscl;      //   the same for the staged key block
  bf4 pk, pb, pq;
  // q, k, b, g of two key blocks are fetched together (they share cache lines);
  // the second block's values wait in registers for the next prefetch
  float4 pg2;
  bf4 pk2, pb2, pq2;
#define GDR2_PREFETCH(CB)                                                                  \
  {                                                                                        \
    if (((CB) & 1) == 0) {                                                                 \
      const int o_ = growc * kst + 16 * (CB) + 4 * cq;                                     \
      pg = ldg_f4(Gp0 + o_);                                                               \
      pk = *reinterpret_cast<const bf4*>(Kp + o_);                                         \
      pb = *reinterpret_cast<const bf4*>(Bp + o_);                                         \
      pq = *reinterpret_cast<const bf4*>(Qp + o_);                                         \
      pg2 = ldg_f4(Gp0 + o_ + 16);                                                         \
      pk2 = *reinterpret_cast<const bf4*>(Kp + o_ + 16);                                   \
      pb2 = *reinterpret_cast<const bf4*>(Bp + o_ + 16);                                   \
      pq2 = *reinterpret_cast<const bf4*>(Qp + o_ + 16);                                   \
    } else {                                                                               \
      pg = pg2;                                                                            \
      pk = pk2;                                                                            \
      pb = pb2;                                                                            \
      pq = pq2;                                                                            \
    }                                                                                      \
    if (hact) {                                                                            \
      const int so_ = (16 * (CB) + hc) * DV + hv;                                          \
      ph = ldg16(Hc + so_);                                                                \
      pd = ldg16(DHc + so_);                                                               \
      psh = Hscc[(CB) * (DV / 32) + hv / 32];                                              \
      psd = DHscc[(CB) * (DV / 32) + hv / 32];                                             \
    }                                                                                      \
    pds = lane < KV ? DHscc[(CB) * KV + lane] : 0.f;                                       \
  }
  // Writes key block CB's staged operands (parity PAR for the small arrays):
  // in-block cumulative sums of the log2-decay, the block totals and first
  // rows, the decay-scaled operands, k / b / q columns, h / dh rows,
  // rowsum(dh * h).
#define GDR2_STAGE(PAR, CBS)                                                               \
  {                                                                                        \
    const int cbs_ = (CBS);                                                                \
    if constexpr (FUSED) {                                                                 \
      const float4 dl_ = *reinterpret_cast<const float4*>(sDL + 16 * cbs_ + 4 * cq);       \
      const float x_[4] = {pg.x + dl_.x, pg.y + dl_.y, pg.z + dl_.z, pg.w + dl_.w};        \
      const float rq_ = sRN[grow], rk_ = sRN[64 + grow];                                   \
      _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                   \
        sXS[aTs + kTabLd * u_] = x_[u_];                                                   \
        pk[u_] = (__bf16)((float)pk[u_] * rk_);                                            \
        pq[u_] = (__bf16)((float)pq[u_] * rq_);                                            \
      }                                                                                    \
      pg = make_float4(-Adec * softplus_f(x_[0]), -Adec * softplus_f(x_[1]),               \
                       -Adec * softplus_f(x_[2]), -Adec * softplus_f(x_[3]));              \
    }                                                                                      \
    if (!grin) {                                                                           \
      pg = make_float4(0.f, 0.f, 0.f, 0.f);                                                \
      pk = bf4{};                                                                          \
    }                                                                                      \
    float x_[4] = {pg.x * kLog2e, pg.y * kLog2e, pg.z * kLog2e, pg.w * kLog2e};            \
    /* inclusive sums over the block's 16 rows (lanes 4 rl + cq), with the first  */     \
    /* row's value f_ and the total l_: DPP shifts by 4 and 8 lanes inside each    */     \
    /* 16-lane row, the row totals spread over the row by rotations, then the     */     \
    /* earlier rows' totals from the partner rows (no LDS round trips)             */     \
    float fs_[4], ls_[4];                                                                  \
    _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                     \
      float x1_ = x_[u_];                                                                  \
      float f1_ = lane < 4 ? x1_ : 0.f;                                                    \
      x1_ += dppf<0x114>(x1_); /* row_shr:4 */                                             \
      x1_ += dppf<0x118>(x1_); /* row_shr:8 */                                             \
      float t1_ = (rl & 3) == 3 ? x1_ : 0.f;                                               \
      t1_ += dppf<0x124>(t1_); /* row_ror:4 */                                             \
      t1_ += dppf<0x128>(t1_); /* row_ror:8 */                                             \
      f1_ += dppf<0x124>(f1_);                                                             \
      f1_ += dppf<0x128>(f1_);                                                             \
      const float p1_ = row_partner16(t1_, podd);                                          \
      const float s1_ = t1_ + p1_;                                                         \
      const float q1_ = row_partner32(s1_, pup);                                           \
      x_[u_] = x1_ + (podd ? p1_ : 0.f) + (pup ? q1_ : 0.f);                               \
      ls_[u_] = s1_ + q1_;                                                                 \
      f1_ += row_partner16(f1_, podd);                                                     \
      fs_[u_] = f1_ + row_partner32(f1_, pup);                                             \
    }                                                                                      \
    f4 xk_, xb_, xq_;                                                                      \
    _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                     \
      const float f_ = fs_[u_], l_ = ls_[u_];                                              \
      sG[aTs + kTabLd * u_] = x_[u_];                                                      \
      const float el_ = ex2(x_[u_] - f_), er_ = ex2(l_ - x_[u_]);                          \
      const float kv_ = (float)pk[u_];                                                     \
      xk_[u_] = kv_ * er_;                                                                 \
      xb_[u_] = (float)pb[u_] * kv_ * el_;                                                 \
      xq_[u_] = (float)pq[u_] * el_;                                                       \
      if (rl == 15) sBK[(0 * 4 + wave) * 16 + 4 * cq + u_] = x_[u_];                       \
      if (rl == 0) sBK[(1 * 4 + wave) * 16 + 4 * cq + u_] = x_[u_];                        \
      const int ac_ = aKs[u_ >> 1] + 64 * (u_ & 1);                                        \
      sKc[ac_] = pk[u_];                                                                   \
      sBc[ac_] = pb[u_];                                                                   \
      sQc[ac_] = pq[u_];                                                                   \
    }                                                                                      \
    st4split(sXh + aXs, sXl + aXs, xk_);                                                   \
    st4split(sBh + aXs, sBl + aXs, xb_);                                                   \
    st4split(sQh + aXs, sQl + aXs, xq_);                                                   \
    if (hact) {                                                                            \
      float hx_[8], dx_[8];                                                                \
      load_state8(ph, psh, hx_);                                                           \
      load_state8(pd, psd, dx_);                                                           \
      const Fr hf_ = split8(hx_);                                                          \
      st8(sHh + aHs, hf_.hi);                                                              \
      st8(sHl + aHs, hf_.lo);                                                              \
      sts16(sD16 + aHs, pd);                                                               \
      float hh_ = hx_[0] * dx_[0];                                                         \
      _Pragma("unroll") for (int e_ = 1; e_ < 8; ++e_) hh_ += hx_[e_] * dx_[e_];           \
      hh_ = row_sum<DV == 64>(hh_); /* the DV / 8 lanes of row hc */                     \
      if ((tid % (DV / 8)) == 0) sHH[(PAR) * 16 + hc] = hh_;                               \
    }                                                                                      \
    dscl = pds;                                                                            \
  }
  // v, w for dv / dw, in flight across the barrier
  bf4 vvr[NVB], wwr[NVB];
#pragma unroll
  for (int p2 = 0; p2 < NVB / 2; ++p2) {
    const int o = min(16 * i + r16, len - 1) * vst + 32 * p2 + goff;
    const u4v xv = unswap_pair(*reinterpret_cast<const u4v*>(Vp + o));
    const u4v xw = unswap_pair(*reinterpret_cast<const u4v*>(Wp + o));
    vvr[2 * p2] = __builtin_bit_cast(bf4, u2v{xv[0], xv[1]});
    vvr[2 * p2 + 1] = __builtin_bit_cast(bf4, u2v{xv[2], xv[3]});
    wwr[2 * p2] = __builtin_bit_cast(bf4, u2v{xw[0], xw[1]});
    wwr[2 * p2 + 1] = __builtin_bit_cast(bf4, u2v{xw[2], xw[3]});
  }
  __syncthreads();  // dR, A and R are in LDS (the barrier waits for the direct loads)
  // key block 0's operands, in flight while the prologue computes
  GDR2_PREFETCH(0)

  // ---- dZ^T = dR^T A for the key rows s of block i: lane gets
  //      dZ[s = 16 i + r16][v = 16 vb + 4 g + u];  dv = dZ * w, dw = dZ * v.
  //      16-deep products over the chunk-row blocks rb >= i (A is lower
  //      triangular).  A's fp16 copy, scaled back by its power-of-two block
  //      scale, splits exactly into bf16 hi and lo (11 significant bits).
  f4 zacc[NVB];
  {
    Fr4 af[4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      if (rb < i) continue;
      const f16x4 a16 = *reinterpret_cast<const f16x4*>(sAm + (4 * i + rb) * 512 + 8 * lane);
      const float s = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ascl), rb));
      f4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = (float)a16[e] * s;
      bf4 hi, lo;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        hi[e] = (__bf16)x[e];
        lo[e] = (__bf16)(x[e] - (float)hi[e]);
      }
      af[rb].hi = hi;
      af[rb].lo = lo;
    }
    // chunk-row block outer and each of the three passes across the value
    // blocks: consecutive products are independent
#pragma unroll
    for (int vb = 0; vb < NVB; ++vb) zacc[vb] = f4zero();
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
      if (rb < i) continue;
      Fr4 rf[NVB];
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb) {
        rf[vb].hi = *reinterpret_cast<const bf4*>(sDR + (4 * vb + rb) * 1024 + 8 * lane);
        rf[vb].lo = *reinterpret_cast<const bf4*>(sDR + (4 * vb + rb) * 1024 + 512 + 8 * lane);
      }
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb) zacc[vb] = mma16(rf[vb].lo, af[rb].hi, zacc[vb]);
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb) zacc[vb] = mma16(rf[vb].hi, af[rb].lo, zacc[vb]);
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb) zacc[vb] = mma16(rf[vb].hi, af[rb].hi, zacc[vb]);
    }
  }
  // value blocks in pairs: one permlane swap per dword turns the lane's two
  // 4-value pieces (columns 32 p + 4 g .., 32 p + 16 + 4 g ..) into 8
  // consecutive values of its row, at 32 p + {0, 16, 8, 24}[g], so that each
  // lane stores 16 bytes per pair
  static_assert(NVB % 2 == 0, "value blocks in pairs");
#pragma unroll
  for (int p2 = 0; p2 < NVB / 2; ++p2) {
    u2v av[2], aw[2];
#pragma unroll
    for (int h2 = 0; h2 < 2; ++h2) {
      const int vb = 2 * p2 + h2;
      bf4 odv, odw;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        odv[u] = (__bf16)(zacc[vb][u] * (float)wwr[vb][u]);
        odw[u] = (__bf16)(zacc[vb][u] * (float)vvr[vb][u]);
      }
      av[h2] = __builtin_bit_cast(u2v, odv);
      aw[h2] = __builtin_bit_cast(u2v, odw);
    }
    const u4v sv = unswap_pair(u4v{av[0][0], av[0][1], av[1][0], av[1][1]});
    const u4v sw = unswap_pair(u4v{aw[0][0], aw[0][1], aw[1][0], aw[1][1]});
    const int o = (16 * i + r16) * vst + 32 * p2 + goff;
    if (16 * i + r16 < len) {
      *reinterpret_cast<u4v*>(dVp + o) = sv;
      *reinterpret_cast<u4v*>(dWp + o) = sw;
    }
  }
  // dZ, dO and R rows of block i as A operands over the values, permuted K:
  // K-step p holds values 32 p + 4 g + (0..3) and 32 p + 16 + 4 g + (0..3).
  // zf (split bf16) serves the key-block loop; for the tiles below dZ is also
  // split into fp16 hi / lo and dO converted to fp16, each under one
  // power-of-two scale for the wave (the largest magnitude into [2^14, 2^15)),
  // so that the tiles multiply R's stored fp16 copy directly.
  Fr zf[KV];
  u4v rfr16[KV];  // R rows of block i, fp16 as stored (scale rsc(i * KV + p))
  f16x8 zh16[KV], zl16[KV], do16[KV];
  float zmx = 0.f, omx = 0.f;
  if (16 * i + r16 >= len) {
#pragma unroll
    for (int p = 0; p < KV; ++p) dof[p] = bf8{};
  }
#pragma unroll
  for (int vb = 0; vb < NVB; ++vb)
#pragma unroll
    for (int u = 0; u < 4; ++u) zmx = fmaxf(zmx, fabsf(zacc[vb][u]));
#pragma unroll
  for (int p = 0; p < KV; ++p)
#pragma unroll
    for (int e = 0; e < 8; ++e) omx = fmaxf(omx, fabsf((float)dof[p][e]));
  const int zsh = state_shift(wave_max(zmx)), osh = state_shift(wave_max(omx));
  const float zs = ldexpf(1.f, zsh), os = ldexpf(1.f, osh);
  const float izs = ldexpf(1.f, -zsh), ios = ldexpf(1.f, -osh);
#pragma unroll
  for (int p = 0; p < KV; ++p) {
    float x[8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      x[u] = zacc[2 * p][u];
      x[4 + u] = zacc[2 * p + 1][u];
    }
    zf[p] = split8(x);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float y = x[e] * zs;
      zh16[p][e] = (_Float16)y;
      zl16[p][e] = (_Float16)(y - (float)zh16[p][e]);
      do16[p][e] = (_Float16)((float)dof[p][e] * os);
    }
    rfr16[p] = *reinterpret_cast<const u4v*>(sR + (i * KV + p) * 1024 + 16 * lane);
  }

  // ---- dT = -tril(dZ R^T, -1) and dA_qk = tril(scale dO R^T), tiles (i, j <= i),
  //      stored transposed: plane[s][r].  The R rows of block j are the fp16
  //      fragment blocks in LDS; every product is exact (fp16 operands), each
  //      K-step scaled by R's block scale and the wave's dZ / dO scale.  The
  //      tiles of one K-step are formed together (independent products).  They
  //      stay in registers until every wave is done with dR (region 1, which
  //      the planes take over) and with A and R (region 2, which key block 0
  //      takes over), so dZ and the tiles run without a barrier between them.
  f4 ta[4], aa[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) ta[j] = aa[j] = f4zero();
#pragma unroll
  for (int p = 0; p < KV; ++p) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j > i) break;
      const f16x8 rv = __builtin_bit_cast(
          f16x8, j == i ? rfr16[p] : *reinterpret_cast<const u4v*>(sR + (j * KV + p) * 1024 + 16 * lane));
      const f4 t = mma_f16(zl16[p], rv, mma_f16(zh16[p], rv, f4zero()));
      const f4 t2 = mma_f16(do16[p], rv, f4zero());
      const float rs = rsc(j * KV + p), cz = rs * izs, co = rs * ios;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ta[j][u] += t[u] * cz;
        aa[j][u] += t2[u] * co;
      }
    }
  }
  __syncthreads();  // dR, A and R are dead: the planes and key block 0 go over them
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j > i) break;
    const int s = 16 * j + r16;
    const int rr = 16 * i + 4 * g;
    f4 tv, av;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      tv[u] = (rr + u > s) ? -ta[j][u] : 0.f;
      av[u] = (rr + u >= s) ? a.scale * aa[j][u] : 0.f;
    }
    const int at = plane_ix<LP>(s, rr);
    st4split(sTh + at, sTl + at, tv);
    st4split(sAh + at, sAl + at, av);
  }
  GDR2_STAGE(0, 0)
  __syncthreads();

  const float scale = a.scale;
  float pa_acc = 0.f;  // fused stage: sum of dg * g over this lane's outputs
  // outputs leave as whole 128-byte row lines where they can: with bf16 dq, dk,
  // db the row pieces of three key blocks wait in registers (packed bf16) for the
  // fourth; fp32 outputs (dg, and the fp32 partial or group sums) wait one block.
  // Stored one 16-key block at a time, the pieces of a line would be written some
  // microseconds apart, and the L2 often writes such a line back in parts.
  static_assert(NCB % 4 == 0, "key blocks leave in fours");
  const bool narrow = !FUSED && gmode == 0 && !partq;  // dq, dk, db all bf16
  // narrow: blocks cb & 3 < 3 as bf16 (q, k, b); wide: the even block's fp32 q, k, b
  // in the first twelve words
  uint2 wn[9];
  float wq[4], wk[4], wb[4];  // fused stage: the even block's q, k, b
  float wg[4];                // dg of the even block
#pragma unroll 1
  for (int cb = 0; cb < NCB; ++cb) {
    const int par = cb & 1;
    if (cb + 1 < NCB) GDR2_PREFETCH(cb + 1)
    const int c = 16 * cb + r16;  // this lane's key channel in every output tile

    // X1 = dZ h^T, X2 = dO h^T, X3 = R dh^T   (rows 16 i + 4 g + u, key c).
    // X3 multiplies the fp16 copies of R and dh directly (exact products), one
    // K-step per 32-value block, each scaled by the two blocks' scales.
    f4 x1 = f4zero(), x2 = f4zero(), x3 = f4zero();
#pragma unroll
    for (int p = 0; p < KV; ++p) {
      Fr hf;
      hf.hi = ld8(sHh + aH + 32 * p);
      hf.lo = ld8(sHl + aH + 32 * p);
      const f16x8 d16 = *reinterpret_cast<const f16x8*>(sD16 + aH + 32 * p);
      x1 = mma3(zf[p], hf, x1);
      x2 = mma2b(dof[p], hf, x2);
      const f4 t = mma_f16(__builtin_bit_cast(f16x8, rfr16[p]), d16, f4zero());
      const float sp = rsc(i * KV + p) * __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dscl), p));
#pragma unroll
      for (int u = 0; u < 4; ++u) x3[u] += t[u] * sp;
    }

    // G2 at the first (G2f) and last (G2l) row of every 16-row block, channel c
    float G2f[4], G2l[4];
    {
      float run = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        G2f[j] = run + sBK[(4 + j) * 16 + r16];
        run += sBK[j * 16 + r16];
        G2l[j] = run;
      }
    }
    const float G2fi = pick4(G2f, i), G2li = pick4(G2l, i);
    // a diagonal block whose decay exceeds e^60 anywhere in this key block is formed element by element
    const bool uns = __ballot(G2fi - G2li > kDiagLimit2) != 0ull;

    // P1 = dT (k 2^(G2_p - G2_s)),  P2 = dA_qk (k 2^(G2_p - G2_s)),  p = 16 i, s <= 16 i + 15:
    // per key-row block j <= i one 16-deep step on the shared operand k eR, whose
    // product takes the block factor 2^(G2f_i - G2l_j)
    f4 p1 = f4zero(), p2 = f4zero();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j > i) break;
      if (j == i && uns) continue;
      Fr4 xf, tf, af;
      xf.hi = ld_tr4(sXh + aXr + 256 * j);
      xf.lo = ld_tr4(sXl + aXr + 256 * j);
      // dT, dA_qk rows of block i, keys of block j: transposed reads of the planes
      const int t0 = aTr + 16 * LP * j;
      tf.hi = ld_tr4(sTh + t0);
      tf.lo = ld_tr4(sTl + t0);
      af.hi = ld_tr4(sAh + t0);
      af.lo = ld_tr4(sAl + t0);
      const float br = ex2(G2fi - pick4(G2l, j));
      const f4 t1 = mma3_16(tf, xf, f4zero()), t2 = mma3_16(af, xf, f4zero());
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        p1[u] += br * t1[u];
        p2[u] += br * t2[u];
      }
    }
    // P3 = dT^T ((b k) 2^(G2_r - G2_e)) + dA_qk^T (q 2^(G2_r - G2_e)),  e = 16 i + 15, r >= 16 i:
    // per row block j >= i one 16-deep step on the shared operands b k eL and q eL,
    // the product taking 2^(G2f_j - G2l_i)
    f4 p3 = f4zero();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (j < i || (j == i && uns)) continue;
      Fr4 bf, qf, tf, af;
      bf.hi = ld_tr4(sBh + aXr + 256 * j);
      bf.lo = ld_tr4(sBl + aXr + 256 * j);
      qf.hi = ld_tr4(sQh + aXr + 256 * j);
      qf.lo = ld_tr4(sQl + aXr + 256 * j);
      const int at = LP == 80 ? aP3 + 16 * j : plane_ix<LP>(16 * i + r16, 16 * j + 4 * g);
      tf.hi = *reinterpret_cast<const bf4*>(sTh + at);
      tf.lo = *reinterpret_cast<const bf4*>(sTl + at);
      af.hi = *reinterpret_cast<const bf4*>(sAh + at);
      af.lo = *reinterpret_cast<const bf4*>(sAl + at);
      const float br = ex2(pick4(G2f, j) - G2li);
      const f4 t = mma3_16(af, qf, mma3_16(tf, bf, f4zero()));
#pragma unroll
      for (int u = 0; u < 4; ++u) p3[u] += br * t[u];
    }

    // ---- elementwise chain (App. B.4) on rows rb + u, key c:
    // gamma_r = eL_r 2^(G2f_i),  tail_r = eR_r 2^(G2_{C-1} - G2l_i)
    const int rb = 16 * i + 4 * g;
    const int ae = aE, ak = aK4;
    // eL_r, eR_r of the lane's rows from the in-block sums (as staged)
    const float4 G4 = *reinterpret_cast<const float4*>(sG + ae);
    const float gf = sBK[(4 + i) * 16 + r16], gl = sBK[i * 16 + r16];
    const float elv[4] = {ex2(G4.x - gf), ex2(G4.y - gf), ex2(G4.z - gf), ex2(G4.w - gf)};
    const float erv[4] = {ex2(gl - G4.x), ex2(gl - G4.y), ex2(gl - G4.z), ex2(gl - G4.w)};
    const bf4 k4 = *reinterpret_cast<const bf4*>(sKc + ak);
    const bf4 b4 = *reinterpret_cast<const bf4*>(sBc + ak);
    const bf4 q4 = *reinterpret_cast<const bf4*>(sQc + ak);
    float4 xs4 = make_float4(0.f, 0.f, 0.f, 0.f);  // fused stage: f + delta of rows rb + u, key c
    if constexpr (FUSED) xs4 = *reinterpret_cast<const float4*>(sXS + ae);
    const float gam0 = ex2(G2fi), tb = ex2(G2l[3] - G2li);
    float dgl[4], tailp = 0.f;
    float oq[4], ok[4], ob[4];  // dq, dk, db of rows rb + u, key c
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float lf = elv[u], rf = erv[u], gam = lf * gam0, tl = rf * tb;
      const float kv = (float)k4[u], bv = (float)b4[u], qv = (float)q4[u];
      float dEg = lf * p1[u] - gam * x1[u];
      float dq = scale * gam * x2[u] + lf * p2[u];
      float dKg = rf * p3[u] + tl * x3[u];
      if (uns) {
        // diagonal block element by element (in-block sums of the log2-decay):
        // every factor has exponent <= 0
        const int r = rb + u;
        const float G = sG[tab_ix(r16, r)];
#pragma unroll 1
        for (int s = 16 * i; s < 16 * i + 16; ++s) {
          const float Gs = sG[tab_ix(r16, s)];
          const int as = col_ix(r16, s);
          const float ks = (float)sKc[as];
          if (s <= r) {
            const float e = ex2(G - Gs);
            const int sr = plane_ix<LP>(s, r);
            const float dTv = (s < r) ? (float)sTh[sr] + (float)sTl[sr] : 0.f;
            const float dAv = (float)sAh[sr] + (float)sAl[sr];
            dEg += dTv * ks * e;
            dq += dAv * ks * e;
          }
          if (s >= r) {
            const float e = ex2(Gs - G);
            const int rs = plane_ix<LP>(r, s);
            const float dTv = (s > r) ? (float)sTh[rs] + (float)sTl[rs] : 0.f;
            const float dAv = (float)sAh[rs] + (float)sAl[rs];
            dKg += (dTv * (float)sBc[as] * ks + dAv * (float)sQc[as]) * e;
          }
        }
      }
      oq[u] = dq;
      ok[u] = dEg * bv + dKg;
      ob[u] = dEg * kv;
      dgl[u] = dq * qv - dKg * kv + dEg * bv * kv;
      tailp += x3[u] * kv * tl;
    }
    // outputs leave as row pieces: after a transpose inside each quad of lanes,
    // lane (g, 4 m + j) holds row 16 i + 4 g + j, keys 16 cb + 4 m .. + 3
    const int jq = r16 & 3, orow = 16 * i + 4 * g + jq;
    const int oo = orow * kso + 16 * cb + 4 * (r16 >> 2);
    quad_transpose(oq, jq);
    quad_transpose(ok, jq);
    quad_transpose(ob, jq);
    // the next block's operands (prefetched at the top of this one) have arrived
    // long before this point: settle them ahead of this block's stores (on every
    // path, the last block's too, so that no later wait sees them as pending)
    settle(pg), settle(pk), settle(pb), settle(pq);
    settle(pg2), settle(pk2), settle(pb2), settle(pq2);
    settle(ph), settle(pd), settle(psh), settle(psd), settle(pds);
    auto emit_qkb = [&](int o, const float(&xq)[4], const float(&xk)[4], const float(&xb)[4]) {
      const size_t ao = ko0 + o;
      float vq[4], vk[4], vb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) vq[u] = xq[u], vk[u] = xk[u], vb[u] = xb[u];
      if (gmode >= 2) {  // the earlier value heads' sums
        add_row4(a.Aq + ao, vq);
        add_row4(a.Ak + ao, vk);
        add_row4(a.Ab + ao, vb);
      }
      if (gmode == 1 || gmode == 2) {
        store_row4(a.Aq + ao, vq);
        store_row4(a.Ak + ao, vk);
        store_row4(a.Ab + ao, vb);
      } else {
        if (partq) {
          store_row4(pQp + o, vq);
          store_row4(pKp + o, vk);
        } else {
          store_row4(dQp + o, vq);
          store_row4(dKp + o, vk);
        }
        store_row4(dBp + o, vb);
      }
    };
    if (narrow) {
      const uint2 pq = pack_bf4(oq), pk = pack_bf4(ok), pb = pack_bf4(ob);
      switch (cb & 3) {  // uniform; constant register indices
        case 0: wn[0] = pq, wn[1] = pk, wn[2] = pb; break;
        case 1: wn[3] = pq, wn[4] = pk, wn[5] = pb; break;
        case 2: wn[6] = pq, wn[7] = pk, wn[8] = pb; break;
        default:
          if (orow < len) {
#pragma unroll
            for (int t = 0; t < 3; ++t) {
              const int o = oo - 16 * (3 - t);
              *reinterpret_cast<uint2*>(dQp + o) = wn[3 * t];
              *reinterpret_cast<uint2*>(dKp + o) = wn[3 * t + 1];
              *reinterpret_cast<uint2*>(dBp + o) = wn[3 * t + 2];
            }
            *reinterpret_cast<uint2*>(dQp + oo) = pq;
            *reinterpret_cast<uint2*>(dKp + oo) = pk;
            *reinterpret_cast<uint2*>(dBp + oo) = pb;
          }
      }
    } else if (FUSED) {
      if (par != 0 && orow < len) {
        emit_qkb(oo - 16, wq, wk, wb);
        emit_qkb(oo, oq, ok, ob);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) wq[u] = oq[u], wk[u] = ok[u], wb[u] = ob[u];
    } else if (par == 0) {
#pragma unroll
      for (int u = 0; u < 4; u += 2) {
        wn[u / 2] = uint2{__float_as_uint(oq[u]), __float_as_uint(oq[u + 1])};
        wn[2 + u / 2] = uint2{__float_as_uint(ok[u]), __float_as_uint(ok[u + 1])};
        wn[4 + u / 2] = uint2{__float_as_uint(ob[u]), __float_as_uint(ob[u + 1])};
      }
    } else if (orow < len) {
#pragma unroll
      for (int u = 0; u < 4; u += 2) {
        wq[u] = __uint_as_float(wn[u / 2].x), wq[u + 1] = __uint_as_float(wn[u / 2].y);
        wk[u] = __uint_as_float(wn[2 + u / 2].x), wk[u + 1] = __uint_as_float(wn[2 + u / 2].y);
        wb[u] = __uint_as_float(wn[4 + u / 2].x), wb[u + 1] = __uint_as_float(wn[4 + u / 2].y);
      }
      emit_qkb(oo - 16, wq, wk, wb);
      emit_qkb(oo, oq, ok, ob);
    }
    // reverse cumulative sum of dG: within the lane, over the lane groups, then blocks
    const float s3 = dgl[3], s2 = s3 + dgl[2], s1 = s2 + dgl[1], s0 = s1 + dgl[0];
    float y = s0;
    {
      // suffix over the four lane groups g (16-lane rows): pair sums, then the other pair
      const float py = y + row_partner16(y, podd);
      const float qy = row_partner32(py, pup);
      y = (podd ? y : py) + (pup ? 0.f : qy);
    }
    float tp = tailp;
    tp += row_partner16(tp, podd);
    tp += row_partner32(tp, pup);
    if (g == 0) {
      sBT[(par * 4 + i) * 16 + r16] = y;
      sTL[(par * 4 + i) * 16 + r16] = tp;
    }
    const float gamC = ex2(G2l[3]);
    __syncthreads();
    // gamma_C d gamma_C joins row C - 1, hence every row's suffix sum
    float off = gamC * sHH[par * 16 + r16] + (y - s0);
#pragma unroll
    for (int i2 = 0; i2 < 4; ++i2) {
      off += sTL[(par * 4 + i2) * 16 + r16];
      if (i2 > i) off += sBT[(par * 4 + i2) * 16 + r16];
    }
    auto emit_g = [&](float(&v)[4]) {
      auto one = [&](int o, const float(&y)[4]) {
        float x[4] = {y[0], y[1], y[2], y[3]};
        if (gmode >= 2) add_row4(a.Ag + ko0 + o, x);
        store_row4((gmode == 1 || gmode == 2) ? a.Ag + ko0 + o : dGp + o, x);
      };
      if (par != 0 && orow < len) {
        one(oo - 16, wg);
        one(oo, v);
      }
      // held unconditionally (an odd block's copy is not used): a branch here
      // would let the compiler merge it with the stores above and keep wg in memory
#pragma unroll
      for (int u = 0; u < 4; ++u) wg[u] = v[u];
    };
    if constexpr (FUSED) {
      // df = dg * dg/df, dg/df = -exp(a) sigmoid(f + delta); partial sums for ddelta and da
      const float dgv[4] = {s0 + off, s1 + off, s2 + off, s3 + off};
      const float xv[4] = {xs4.x, xs4.y, xs4.z, xs4.w};
      float pdc = 0.f, dfv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        dfv[u] = dgv[u] * (-Adec * sigmoid_f(xv[u]));
        if (rb + u < len) {
          pdc += dfv[u];
          pa_acc += dgv[u] * (-Adec * softplus_f(xv[u]));
        }
      }
      quad_transpose(dfv, jq);
      emit_g(dfv);
      pdc += row_partner16(pdc, podd);
      pdc += row_partner32(pdc, pup);
      if (g == 0) a.PD[pslot * DK + 16 * cb + r16] = pdc;
    } else {
      float dgv[4] = {s0 + off, s1 + off, s2 + off, s3 + off};
      quad_transpose(dgv, jq);
      emit_g(dgv);
    }
    if (cb + 1 < NCB) GDR2_STAGE(par ^ 1, cb + 1)
    __syncthreads();
  }
  if constexpr (FUSED) {
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) pa_acc += __shfl_xor(pa_acc, o);
    if (lane == 0) a.PA[pslot] = pa_acc;
  }
#undef GDR2_PREFETCH
#undef GDR2_STAGE
}

template <int DK, int DV, bool FUSED>
hipError_t launch_bchunk_bf16_t(const BChunkBf16Args& a, hipStream_t st) {
  using C = BChunkCfg<DK, DV, FUSED>;
  constexpr int lds = C::LDS;
  const void* fn = reinterpret_cast<const void*>(&bchunk_bf16_kernel<DK, DV, FUSED>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  if (e != hipSuccess) return e;
  dim3 grid(a.vl.ct0 ? a.vl.ncmax : a.NT, a.H / a.G, a.vl.ct0 ? 1 : a.B);
  hipLaunchKernelGGL((bchunk_bf16_kernel<DK, DV, FUSED>), grid, dim3(C::NTHR), lds, st, a);
  return hipGetLastError();
}

template <int DK, int DV>
hipError_t launch_bchunk_bf16(const BChunkBf16Args& a, hipStream_t st) {
  return a.st.a_log != nullptr ? launch_bchunk_bf16_t<DK, DV, true>(a, st)
                               : launch_bchunk_bf16_t<DK, DV, false>(a, st);
}

template hipError_t launch_bchunk_bf16<64, 64>(const BChunkBf16Args&, hipStream_t);
template hipError_t launch_bchunk_bf16<64, 128>(const BChunkBf16Args&, hipStream_t);
template hipError_t launch_bchunk_bf16<128, 64>(const BChunkBf16Args&, hipStream_t);
template hipError_t launch_bchunk_bf16<128, 128>(const BChunkBf16Args&, hipStream_t);

}  // namespace gdr2

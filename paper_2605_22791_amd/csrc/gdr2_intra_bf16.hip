// Intra-chunk kernel of the bf16 path (gfx950): one 4-wave workgroup per
// key-head chunk, two workgroups per CU (grouped value heads share everything
// but U, which is formed for each value head of the group).  Per chunk of
// C = 64 tokens it forms
//
//   G2 = log2(e) * cumsum(g)                          eq. eq_gdn2_gamma (fp32)
//   Q_g = q * gamma,  Ktail^T = (k * gamma_C / gamma)^T    eqs. eq_gdn2_gate_matrices,
//                                                     eq_gdn2_chunk_state
//   T = tril(Ebar Kbar^T, -1), A_qk = tril(Q_g Kbar^T)     eqs. eq_gdn2_wy_matrix,
//                                                     eq_gdn2_chunk_scores
//   A = (I + T)^{-1}                                  fp32 (App. D.4)
//   Y = A Ebar,  U = A (W * V)                        eq. eq_gdn2_wy_aux
//
// and writes Y, Q_g, A_qk, Ktail^T, U and gamma_C to the workspace in MFMA
// fragment order (layout in gdr2_kernels.hpp) for the state scan; the
// backward's recompute also keeps A itself (split hi/lo).
//
// Precision: every product is fp32-accurate (split hi/lo operands: T, the
// solve, A in Y and U, A_qk, Q_g, Ktail, Ebar, Z); Y is stored in bf16.
//
// Decay factors are 2^(G2_r - G2_s) for r >= s, formed relative to the first
// row p = 16 i of the row block i of r: 2^(G2_r - G2_p) * 2^(G2_p - G2_s); the
// first factor is <= 1, the second <= 1 outside the diagonal block and bounded
// by one block's decay inside it.  A diagonal block whose internal decay
// exceeds e^60 is formed element by element.
//
// T and A_qk are computed transposed (rows = keys) so that each lane's four
// outputs are consecutive keys of one query row: T goes to LDS as float4 rows
// and A_qk / Y land directly in the permuted fragment order.
//
// Fused input stage (FUSED; App. C.1, App. D.2): q and k arrive raw and are
// L2-normalised in registers as they are loaded (the lanes holding one row
// reduce its sum of squares by shuffles), and the log-decay is formed in fp32
// from the decay projection as -exp(a) softplus(f + delta) before the
// cumulative sum, so the normalised tensors and g never exist in HBM.  The
// inverse norms go to the workspace for the backward.

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK, int DV>
struct IntraCfg {
  static constexpr int NTHR = 256;
  static constexpr int KS = DK / 32, NCB = DK / 16, NVB = DV / 16;
  static constexpr int LG = DK + 8;    // G2 fp32 [64][LG]
  static constexpr int LE = DK + 8;    // Ebar hi/lo bf16 [64][LE] (over G2)
  static constexpr int LVW = DV + 8;   // v, w bf16 [64][LVW] (over Ebar)
  static constexpr int LKB = DK + 8;   // k bf16 [64][LKB]
  static constexpr int LTA = 64 + 4;   // T -> A fp32 [64][LTA]
  static constexpr int SZ_G = 64 * LG * 4, SZ_E = 2 * 64 * LE * 2, SZ_VW = 2 * 64 * LVW * 2;
  static constexpr int SZ_X = SZ_G > SZ_E ? (SZ_G > SZ_VW ? SZ_G : SZ_VW) : (SZ_E > SZ_VW ? SZ_E : SZ_VW);
  static constexpr int OFF_X = 0;
  static constexpr int OFF_K = SZ_X;
  static constexpr int OFF_TA = OFF_K + 64 * LKB * 2;
  static constexpr int OFF_MISC = OFF_TA + 64 * LTA * 4;
  static constexpr int OFF_RQ = OFF_MISC + 16;  // fused stage: inverse norms of the q rows [64]
  // A split hi / lo, bf16 [64][LA]: hi over the k tile (dead by then), lo after the rest
  static constexpr int LA = 64 + 8;
  static constexpr int OFF_AL = OFF_RQ + 64 * 4;
  static constexpr int LDS = OFF_AL + 64 * LA * 2;
  static_assert(64 * LA * 2 <= 64 * LKB * 2, "A hi plane fits the k tile");
  static_assert(LDS <= 80 * 1024, "two workgroups per CU");
};

// T / A_qk tiles per wave: (row block i of queries, column block j of keys)
// encoded as 4 * i + j; -1 marks "no tile".  The A_qk tiles above the
// diagonal are written as zeros (they share fragment blocks with causal tiles).
__device__ __forceinline__ int tile_of(int wave, int t) {
  // w0: (0,0) (1,0) (1,1)   w1: (2,0) (2,1) (2,2)   w2: (3,0) (3,1)   w3: (3,2) (3,3)
  switch (wave) {
    case 0: return t == 0 ? 0 : (t == 1 ? 4 : 5);
    case 1: return 8 + t;
    case 2: return t < 2 ? 12 + t : -1;
    default: return t < 2 ? 14 + t : -1;
  }
}
// A_qk tiles above the diagonal that share fragment blocks with causal tiles,
// written as zeros: (0,1) and (2,3).  (0,2) (0,3) (1,2) (1,3) make up two whole
// blocks, which are not stored.
__device__ __forceinline__ int zero_tile(int z) { return z == 0 ? 1 : 11; }

template <int DK, int DV, bool FUSED>
__global__ __launch_bounds__(256, 2) void intra_bf16_kernel(IntraBf16Args a) {
  using C = IntraCfg<DK, DV>;
  constexpr int KS = C::KS, NCB = C::NCB, NVB = C::NVB;
  constexpr int LG = C::LG, LE = C::LE, LVW = C::LVW, LKB = C::LKB, LTA = C::LTA, LA = C::LA;

  extern __shared__ __align__(16) unsigned char smem[];
  float* sG = reinterpret_cast<float*>(smem + C::OFF_X);
  __bf16* sEhi = reinterpret_cast<__bf16*>(smem + C::OFF_X);
  __bf16* sElo = sEhi + 64 * LE;
  __bf16* sV = reinterpret_cast<__bf16*>(smem + C::OFF_X);
  __bf16* sW = sV + 64 * LVW;
  __bf16* sK = reinterpret_cast<__bf16*>(smem + C::OFF_K);
  float* sTA = reinterpret_cast<float*>(smem + C::OFF_TA);
  int* unsafe = reinterpret_cast<int*>(smem + C::OFF_MISC);
  float* sRQ = reinterpret_cast<float*>(smem + C::OFF_RQ);
  __bf16* sAh = reinterpret_cast<__bf16*>(smem + C::OFF_K);  // A hi (after the k tile is dead)
  __bf16* sAl = reinterpret_cast<__bf16*>(smem + C::OFF_AL);  // A lo

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  // one workgroup per key-head chunk: the key-side tiles (everything but U) are
  // shared by the G value heads of the group; U is formed for each of them
  const int H = a.H, HK = H / a.G, hk = blockIdx.y;
  ChunkPos cp;
  if (!chunk_pos(a.vl, blockIdx.x, hk, blockIdx.z, a.T, HK, a.NT, cp)) return;
  const size_t ch = cp.ch;  // key-head chunk
  // Rows in use.  Every load below reads an in-range row (rows past a partial
  // chunk's end re-read its last row); g, k and v of those rows are then taken
  // as zero, which makes their T / A_qk entries, Ebar, Z, Ktail and decay
  // vanish, so they add nothing to the valid rows or the state.  Their q, b and
  // w only reach outputs of those rows, which nobody reads.
  const int len = cp.len;
  const u4v z16 = {0u, 0u, 0u, 0u};

  const __bf16* Q = reinterpret_cast<const __bf16*>(a.q);
  const __bf16* K = reinterpret_cast<const __bf16*>(a.k);
  const __bf16* Vg = reinterpret_cast<const __bf16*>(a.v);
  const __bf16* Bg = reinterpret_cast<const __bf16*>(a.b);
  const __bf16* Wg = reinterpret_cast<const __bf16*>(a.w);
  const size_t row0 = cp.row0;
  // key-side tensors (q, k, g, b) on the H / G key heads; v, w of value head hv
  auto kofs = [&](int r) -> size_t { return (row0 + min(r, len - 1)) * ((size_t)HK * DK) + (size_t)hk * DK; };
  auto vofs = [&](int hv, int r) -> size_t {
    return (row0 + min(r, len - 1)) * ((size_t)H * DV) + (size_t)hv * DV;
  };

  // ---- loads: g in scan layout (NG rows of 4 channels per thread), k
  constexpr int GCG = DK / 4, GSEG = 256 / GCG, NG = 64 / GSEG;
  constexpr int NKC = DK / 32;  // 16-byte chunks of k per thread
  const int gcg = tid % GCG, gsg = tid / GCG;
  float4 gr[NG];
#pragma unroll
  for (int m = 0; m < NG; ++m) gr[m] = *reinterpret_cast<const float4*>(a.g + kofs(NG * gsg + m) + 4 * gcg);
  // fused stage: decay bias of this thread's 4 channels and exp(a) of the key head
  float4 dlt = make_float4(0.f, 0.f, 0.f, 0.f);
  float Adec = 0.f;
  if constexpr (FUSED) {
    dlt = *reinterpret_cast<const float4*>(a.st.delta + (size_t)hk * DK + 4 * gcg);
    Adec = expf(a.st.a_log[hk]);
  }
  constexpr bool wr_norm = FUSED;
  u4v kst[NKC];
#pragma unroll
  for (int m = 0; m < NKC; ++m) {
    const int e = tid + 256 * m, r = e / (DK / 8), c8 = (e % (DK / 8)) * 8;
    kst[m] = ldg16(K + kofs(r) + c8);
  }
  // q and b rows of the row blocks whose T / A_qk tiles this wave forms (wave 0:
  // blocks 0 and 1, wave 1: block 2, waves 2 and 3: block 3), as K-step
  // fragments (row 16 rb + r16, channels 32 p + 8 g ..): the same registers
  // feed Q_g and Ebar, so each row of q and b is fetched once per wave that needs it
  const int rbA = wave == 0 ? 0 : (wave == 1 ? 2 : 3);
  u4v qreg[2][KS], breg[2][KS];
#pragma unroll
  for (int p = 0; p < KS; ++p) {
    qreg[0][p] = ldg16(Q + kofs(16 * rbA + r16) + 32 * p + 8 * g);
    breg[0][p] = ldg16(Bg + kofs(16 * rbA + r16) + 32 * p + 8 * g);
  }
  if (wave == 0) {
#pragma unroll
    for (int p = 0; p < KS; ++p) {
      qreg[1][p] = ldg16(Q + kofs(16 + r16) + 32 * p + 8 * g);
      breg[1][p] = ldg16(Bg + kofs(16 + r16) + 32 * p + 8 * g);
    }
  } else {
#pragma unroll
    for (int p = 0; p < KS; ++p) qreg[1][p] = breg[1][p] = u4v{0u, 0u, 0u, 0u};
  }

  // ---- G2 = log2(e) * cumsum(g): in-register segment scans + segment offsets
  if (tid < 4) unsafe[tid] = 0;
  {
    float4* tot = reinterpret_cast<float4*>(sTA);  // scratch before T exists
    float4 run = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int m = 0; m < NG; ++m) {
      if constexpr (FUSED) {
        gr[m].x = decay_act(gr[m].x, dlt.x, Adec);
        gr[m].y = decay_act(gr[m].y, dlt.y, Adec);
        gr[m].z = decay_act(gr[m].z, dlt.z, Adec);
        gr[m].w = decay_act(gr[m].w, dlt.w, Adec);
      }
      if (NG * gsg + m >= len) gr[m] = make_float4(0.f, 0.f, 0.f, 0.f);
      run.x += gr[m].x * kLog2e; run.y += gr[m].y * kLog2e;
      run.z += gr[m].z * kLog2e; run.w += gr[m].w * kLog2e;
      gr[m] = run;
    }
    tot[gsg * GCG + gcg] = run;
    if constexpr (FUSED) {
      // k rows: the DK / 8 consecutive lanes holding a row reduce its sum of squares
#pragma unroll
      for (int m = 0; m < NKC; ++m) {
        const int e = tid + 256 * m, r = e / (DK / 8);
        float kf[8];
        unpack8(kst[m], kf);
        float ss = 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u) ss += kf[u] * kf[u];
        ss = row_sum<DK == 64>(ss);  // the DK / 8 lanes of row r
        const float rk = inv_norm(ss, a.st.eps);
#pragma unroll
        for (int u = 0; u < 8; ++u) kf[u] *= rk;
        kst[m] = __builtin_bit_cast(u4v, round8(kf));
        if (wr_norm && a.st.RK != nullptr && (e % (DK / 8)) == 0 && r < len)
          a.st.RK[(row0 + r) * HK + hk] = rk;
      }
    }
#pragma unroll
    for (int m = 0; m < NKC; ++m) {
      const int e = tid + 256 * m, r = e / (DK / 8), c8 = (e % (DK / 8)) * 8;
      sts16(sK + r * LKB + c8, r < len ? kst[m] : z16);
    }
    __syncthreads();
    float4 off = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s = 0; s < gsg; ++s) {
      const float4 t4 = tot[s * GCG + gcg];
      off.x += t4.x; off.y += t4.y; off.z += t4.z; off.w += t4.w;
    }
#pragma unroll
    for (int m = 0; m < NG; ++m)
      *reinterpret_cast<float4*>(sG + (NG * gsg + m) * LG + 4 * gcg) =
          make_float4(gr[m].x + off.x, gr[m].y + off.y, gr[m].z + off.z, gr[m].w + off.w);
    __syncthreads();
  }
  for (int e = tid; e < 4 * DK; e += 256) {
    const int i = e / DK, c = e % DK;
    if (sG[(16 * i) * LG + c] - sG[(16 * i + 15) * LG + c] > kDiagLimit2) unsafe[i] = 1;
  }
  for (int c = tid; c < DK; c += 256) a.GC[ch * (WsBf16::gc(DK) / 4) + c] = ex2(sG[(CH - 1) * LG + c]);
  if constexpr (FUSED) {
    // q rows: the four lane groups of a row reduce its sum of squares
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      if (sl == 1 && wave != 0) continue;
      float qf[KS][8];
      float ss = 0.f;
#pragma unroll
      for (int p = 0; p < KS; ++p) {
        unpack8(qreg[sl][p], qf[p]);
#pragma unroll
        for (int u = 0; u < 8; ++u) ss += qf[p][u] * qf[p][u];
      }
      ss += row_partner16(ss, (g & 1) != 0);
      ss += row_partner32(ss, g >= 2);
      const float rq = inv_norm(ss, a.st.eps);
#pragma unroll
      for (int p = 0; p < KS; ++p) {
#pragma unroll
        for (int u = 0; u < 8; ++u) qf[p][u] *= rq;
        qreg[sl][p] = __builtin_bit_cast(u4v, round8(qf[p]));
      }
      const int row = 16 * (sl == 0 ? rbA : 1) + r16;
      if (g == 0 && !(sl == 0 && wave == 3)) {  // wave 3 holds a copy of wave 2's rows
        sRQ[row] = rq;
        if (wr_norm && a.st.RQ != nullptr && row < len) a.st.RQ[(row0 + row) * HK + hk] = rq;
      }
    }
  }
  for (int e = tid; e < 6 * 256; e += 256) {  // upper blocks of T/A (the region held scratch)
    const int blk = e >> 8, rr = (e & 255) >> 4, cc = e & 15;
    const int bi = blk < 3 ? 0 : (blk < 5 ? 1 : 2);
    const int bj = blk < 3 ? blk + 1 : (blk < 5 ? blk - 1 : 3);
    sTA[(16 * bi + rr) * LTA + 16 * bj + cc] = 0.f;
  }
  __syncthreads();

  // ---- Q_g (standard fragments) and Ktail^T (standard fragments, via transposed k)
  {
    unsigned char* Qo = a.Qg + ch * WsBf16::qg(DK);
    // row block rb (K-steps kb) from the q fragments; wave 3 holds a copy of block 3
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      if (sl == 0 ? wave == 3 : wave != 0) continue;
      const int rb = sl == 0 ? rbA : 1;
#pragma unroll
      for (int kb = 0; kb < KS; ++kb) {
        const int r = 16 * rb + r16, c0 = 32 * kb + 8 * g, blk = rb * KS + kb;
        float Gr[8], qf[8], x[8];
        ldf8(sG + r * LG + c0, Gr);
        unpack8(qreg[sl][kb], qf);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = qf[e] * ex2(Gr[e]);
        const Fr f = split8(x);
        st8(reinterpret_cast<__bf16*>(Qo + blk * 2048 + 16 * lane), f.hi);
        st8(reinterpret_cast<__bf16*>(Qo + blk * 2048 + 1024 + 16 * lane), f.lo);
      }
    }
    unsigned char* Ko = a.KtT + ch * WsBf16::ktt(DK);
    for (int blk = wave; blk < NCB * 2; blk += 4) {
      const int cb = blk >> 1, kb = blk & 1;
      const int c = 16 * cb + r16;
      float kf[8], x[8];
      unpack8(ld_tr8(sK, LKB, 32 * kb, 16 * cb, lane), kf);  // k[32 kb + 8 g + e][c]
      const float GC2 = sG[(CH - 1) * LG + c];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = kf[e] * ex2(GC2 - sG[(32 * kb + 8 * g + e) * LG + c]);
      const Fr f = split8(x);
      st8(reinterpret_cast<__bf16*>(Ko + blk * 2048 + 16 * lane), f.hi);
      st8(reinterpret_cast<__bf16*>(Ko + blk * 2048 + 1024 + 16 * lane), f.lo);
    }
  }

  // ---- T^T and A_qk^T tiles: D[s][r] = sum_c RK_s[c] * {LE, LQ}_r[c]
  {
    unsigned char* Ao = a.Aqk + ch * WsBf16::aqk();
#pragma unroll 1
    for (int t = 0; t < 3; ++t) {
      const int code = tile_of(wave, t);
      if (code < 0) continue;
      const int i = code >> 2, j = code & 3;
      const int r = 16 * i + r16;  // query row of this lane's outputs
      f4 accT = f4zero(), accA = f4zero();
      if (unsafe[i] && i == j) {
        // element by element: every factor 2^(G2_r - G2_s) with r >= s is <= 1
#pragma unroll 1
        for (int u = 0; u < 4; ++u) {
          const int s = 16 * j + 4 * g + u;
          float tt = 0.f, ta = 0.f;
          if (r >= s) {
#pragma unroll 1
            for (int c = 0; c < DK; ++c) {
              const float e = ex2(sG[r * LG + c] - sG[s * LG + c]) * (float)sK[s * LKB + c];
              tt += (float)Bg[kofs(r) + c] * (float)sK[r * LKB + c] * e;
              if constexpr (FUSED)
                ta += (float)(__bf16)((float)Q[kofs(r) + c] * sRQ[r]) * e;
              else
                ta += (float)Q[kofs(r) + c] * e;
            }
          }
#pragma unroll
          for (int uu = 0; uu < 4; ++uu)
            if (uu == u) {
              accT[uu] = tt;
              accA[uu] = ta;
            }
        }
      } else {
        const int s = 16 * j + r16;  // key row supplied by this lane (A operand)
        const bool sec = i == 1;        // wave 0's second row block
#pragma unroll
        for (int p = 0; p < KS; ++p) {
          const int c0 = 32 * p + 8 * g;
          float Gs[8], Gr[8], Gp[8], ks[8], kr[8], br[8], qr[8];
          ldf8(sG + s * LG + c0, Gs);
          ldf8(sG + r * LG + c0, Gr);
          ldf8(sG + (16 * i) * LG + c0, Gp);
          unpack8(ld8(sK + s * LKB + c0), ks);
          unpack8(ld8(sK + r * LKB + c0), kr);
          unpack8(sec ? breg[1][p] : breg[0][p], br);
          unpack8(sec ? qreg[1][p] : qreg[0][p], qr);
          float rk[8], le[8], lq[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            rk[e] = ks[e] * ex2(Gp[e] - Gs[e]);
            const float f = ex2(Gr[e] - Gp[e]);
            le[e] = br[e] * kr[e] * f;
            lq[e] = qr[e] * f;
          }
          const Fr rkf = split8(rk);
          accT = mma3(rkf, split8(le), accT);
          accA = mma3(rkf, split8(lq), accA);
        }
      }
      // lane holds T[r][s0 + u] and A_qk[r][s0 + u], s0 = 16 j + 4 g
      const int s0 = 16 * j + 4 * g;
      float4 tv;
      tv.x = (r > s0 + 0) ? accT[0] : 0.f;
      tv.y = (r > s0 + 1) ? accT[1] : 0.f;
      tv.z = (r > s0 + 2) ? accT[2] : 0.f;
      tv.w = (r > s0 + 3) ? accT[3] : 0.f;
      *reinterpret_cast<float4*>(sTA + r * LTA + s0) = tv;
      f4 av;
#pragma unroll
      for (int u = 0; u < 4; ++u) av[u] = (r >= s0 + u) ? accA[u] : 0.f;
      const size_t off = (size_t)(i * 2 + (j >> 1)) * 2048 + 16 * lane + 8 * (j & 1);
      st4split(reinterpret_cast<__bf16*>(Ao + off), reinterpret_cast<__bf16*>(Ao + off + 1024), av);
    }
    // zero A_qk tiles above the diagonal that share fragment blocks with causal
    // tiles, (0,1) and (2,3); the blocks of query rows 0..31 and keys 32..63 are
    // all zero and are neither written nor read (the scans skip them)
    if (wave < 2) {
      const int i = zero_tile(wave) >> 2, j = zero_tile(wave) & 3;
      const size_t off = (size_t)(i * 2 + (j >> 1)) * 2048 + 16 * lane + 8 * (j & 1);
      st4split(reinterpret_cast<__bf16*>(Ao + off), reinterpret_cast<__bf16*>(Ao + off + 1024), f4zero());
    }
  }
  __syncthreads();

  // ---- A = (I + T)^{-1} in place, fp32: diagonal blocks by forward
  // substitution (lane = column), then the off-diagonal blocks row block by
  // row block:  A_ij = -A_ii * sum_{j <= k < i} T_ik A_kj
  if (wave == 0) {
    const int blk = lane >> 4, cc = lane & 15;
    float x[16];
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const float* trow = sTA + (16 * blk + rr) * LTA + 16 * blk;
      float a0 = (rr == cc) ? 1.f : 0.f, a1 = 0.f;
#pragma unroll
      for (int s = 0; s + 1 < rr; s += 2) {
        a0 -= trow[s] * x[s];
        a1 -= trow[s + 1] * x[s + 1];
      }
      if (rr & 1) a0 -= trow[rr - 1] * x[rr - 1];
      x[rr] = a0 + a1;
    }
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) sTA[(16 * blk + rr) * LTA + 16 * blk + cc] = x[rr];
  }
  // v, w of the group's first value head for U = A Z, loaded while the solve runs
  constexpr int NVC = DV / 32;  // 16-byte chunks of v (and of w) per thread
  const int h0 = hk * a.G;
  u4v vst[NVC], wst[NVC];
#pragma unroll
  for (int m = 0; m < NVC; ++m) {
    const int e = tid + 256 * m, r = e / (DV / 8), c8 = (e % (DV / 8)) * 8;
    vst[m] = ldg16(Vg + vofs(h0, r) + c8);
    wst[m] = ldg16(Wg + vofs(h0, r) + c8);
  }
  __syncthreads();
#pragma unroll 1
  for (int i = 1; i < 4; ++i) {
    f4 res = f4zero();
    if (wave < i) {
      const int j = wave;
      f4 M = f4zero();
      for (int kb = j; kb < i; ++kb) {
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const int kk = 16 * kb + 4 * st + g;
          M = mfma_f32(sTA[(16 * i + r16) * LTA + kk], sTA[kk * LTA + 16 * j + r16], M);
        }
      }
      // B operand of the next product: lane (g, r16) takes element g of lane
      // (st, r16)'s accumulator for K-step st, a 4 x 4 transpose across the
      // 16-lane rows (two stages of 2 x 2 swaps with the permlane swaps)
      row_transpose4(M);
#pragma unroll
      for (int st = 0; st < 4; ++st)
        res = mfma_f32(sTA[(16 * i + r16) * LTA + 16 * i + 4 * st + g], M[st], res);
    }
    __syncthreads();
    if (wave < i) {
#pragma unroll
      for (int u = 0; u < 4; ++u) sTA[(16 * i + 4 * g + u) * LTA + 16 * wave + r16] = -res[u];
    }
    __syncthreads();
  }

  // ---- A for the backward: fp16 16 x 16 blocks (key s block, chunk row r block)
  //      with one scale each, the B operand of the chunk backward's dR^T A
  if (a.Am) {
    _Float16* Ao = a.Am + ch * (WsBf16::am() / 2);
    float* Asc = a.Amsc + ch * (WsBf16::amsc() / 4);
#pragma unroll
    for (int blk = wave; blk < 16; blk += 4) {
      const int sb = blk >> 2, rb = blk & 3;
      if (rb < sb) continue;  // above the diagonal: zero, neither stored nor read
      f4 x;  // A[r = 16 rb + 4 g + e][s = 16 sb + r16]
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = sTA[(16 * rb + 4 * g + e) * LTA + 16 * sb + r16];
      store_tile_f16(x, tile_shift(x), Ao + blk * 256, Asc + blk, lane);
    }
  }

  // ---- Ebar = b * k * gamma (split) over the G2 region
  // (rows of the wave's row blocks, from the b fragments; wave 3 has none of its own)
  {
    Fr ef[2][KS];
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      if (sl == 0 ? wave == 3 : wave != 0) continue;
      const int r = 16 * (sl == 0 ? rbA : 1) + r16;
#pragma unroll
      for (int p = 0; p < KS; ++p) {
        const int c0 = 32 * p + 8 * g;
        float Gv[8], kf[8], bf[8], x[8];
        ldf8(sG + r * LG + c0, Gv);
        unpack8(ld8(sK + r * LKB + c0), kf);
        unpack8(breg[sl][p], bf);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = bf[e] * kf[e] * ex2(Gv[e]);
        ef[sl][p] = split8(x);
      }
    }
    __syncthreads();
#pragma unroll
    for (int sl = 0; sl < 2; ++sl) {
      if (sl == 0 ? wave == 3 : wave != 0) continue;
      const int r = 16 * (sl == 0 ? rbA : 1) + r16;
#pragma unroll
      for (int p = 0; p < KS; ++p) {
        st8(sEhi + r * LE + 32 * p + 8 * g, ef[sl][p].hi);
        st8(sElo + r * LE + 32 * p + 8 * g, ef[sl][p].lo);
      }
    }
    // A split once into bf16 hi / lo planes (the k tile is dead): the Y and U
    // products read their A fragments from there (row r, 16 values per thread)
    {
      const int r = tid >> 2, c0 = 16 * (tid & 3);
      float x[8];
#pragma unroll
      for (int h8 = 0; h8 < 2; ++h8) {
        ldf8(sTA + r * LTA + c0 + 8 * h8, x);
        const Fr f = split8(x);
        st8(sAh + r * LA + c0 + 8 * h8, f.hi);
        st8(sAl + r * LA + c0 + 8 * h8, f.lo);
      }
    }
    __syncthreads();
  }

  // ---- Y^T tiles: D[c][r] = sum_s Ebar[s][c] A[r][s]  -> permuted fragments of Y
  {
    unsigned char* Yo = a.Y + ch * WsBf16::y(DK);
#pragma unroll 1
    for (int cb = wave; cb < NCB; cb += 4) {
      Fr ef[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        ef[kb].hi = ld_tr8(sEhi, LE, 32 * kb, 16 * cb, lane);
        ef[kb].lo = ld_tr8(sElo, LE, 32 * kb, 16 * cb, lane);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f4 acc = f4zero();
#pragma unroll
        for (int kb = 0; kb <= (i >> 1); ++kb) {
          Fr af;
          af.hi = ld8(sAh + (16 * i + r16) * LA + 32 * kb + 8 * g);
          af.lo = ld8(sAl + (16 * i + r16) * LA + 32 * kb + 8 * g);
          acc = mma3(ef[kb], af, acc);
        }
        st4(reinterpret_cast<__bf16*>(Yo + (size_t)(i * KS + (cb >> 1)) * 1024 + 16 * lane + 8 * (cb & 1)), acc[0],
            acc[1], acc[2], acc[3]);
      }
    }
  }
  // ---- U = A (W * V) for every value head of the group: fp32 accumulator tiles
#pragma unroll 1
  for (int j = 0; j < a.G; ++j) {
    if (j > 0) {
#pragma unroll
      for (int m = 0; m < NVC; ++m) {
        const int e = tid + 256 * m, r = e / (DV / 8), c8 = (e % (DV / 8)) * 8;
        vst[m] = ldg16(Vg + vofs(h0 + j, r) + c8);
        wst[m] = ldg16(Wg + vofs(h0 + j, r) + c8);
      }
    }
    __syncthreads();  // Ebar (then the previous value head's v, w) is dead; the region takes v and w
#pragma unroll
    for (int m = 0; m < NVC; ++m) {
      const int e = tid + 256 * m, r = e / (DV / 8), c8 = (e % (DV / 8)) * 8;
      sts16(sV + r * LVW + c8, r < len ? vst[m] : u4v{0u, 0u, 0u, 0u});
      sts16(sW + r * LVW + c8, wst[m]);
    }
    __syncthreads();
    {
      float* Uo = a.U + value_ch(a.vl, blockIdx.x, h0 + j, blockIdx.z, H, a.NT) * (WsBf16::u(DV) / 4);
      constexpr int VPW = NVB / 4;  // value blocks per wave
#pragma unroll 1
      for (int t = 0; t < VPW; ++t) {
        const int vb = wave * VPW + t;
        Fr zf[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          float vf[8], wf[8], z[8];
          unpack8(ld_tr8(sV, LVW, 32 * kb, 16 * vb, lane), vf);
          unpack8(ld_tr8(sW, LVW, 32 * kb, 16 * vb, lane), wf);
#pragma unroll
          for (int e = 0; e < 8; ++e) z[e] = vf[e] * wf[e];
          zf[kb] = split8(z);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f4 acc = f4zero();
#pragma unroll
          for (int kb = 0; kb <= (i >> 1); ++kb) {
            Fr af;
            af.hi = ld8(sAh + (16 * i + r16) * LA + 32 * kb + 8 * g);
            af.lo = ld8(sAl + (16 * i + r16) * LA + 32 * kb + 8 * g);
            acc = mma3(af, zf[kb], acc);
          }
          *reinterpret_cast<f4*>(Uo + ((size_t)(vb * 4 + i) * 64 + lane) * 4) = acc;
        }
      }
    }
  }
}

template <int DK, int DV, bool FUSED>
hipError_t launch_intra_bf16_t(const IntraBf16Args& a, hipStream_t st) {
  using C = IntraCfg<DK, DV>;
  const void* fn = reinterpret_cast<const void*>(&intra_bf16_kernel<DK, DV, FUSED>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  dim3 grid(a.vl.ct0 ? a.vl.ncmax : a.NT, a.H / a.G, a.vl.ct0 ? 1 : a.B);
  hipLaunchKernelGGL((intra_bf16_kernel<DK, DV, FUSED>), grid, dim3(C::NTHR), C::LDS, st, a);
  return hipGetLastError();
}

template <int DK, int DV>
hipError_t launch_intra_bf16(const IntraBf16Args& a, hipStream_t st) {
  return a.st.a_log != nullptr ? launch_intra_bf16_t<DK, DV, true>(a, st) : launch_intra_bf16_t<DK, DV, false>(a, st);
}

template hipError_t launch_intra_bf16<64, 64>(const IntraBf16Args&, hipStream_t);
template hipError_t launch_intra_bf16<64, 128>(const IntraBf16Args&, hipStream_t);
template hipError_t launch_intra_bf16<128, 64>(const IntraBf16Args&, hipStream_t);
template hipError_t launch_intra_bf16<128, 128>(const IntraBf16Args&, hipStream_t);

}  // namespace gdr2

// Fused chunkwise forward of the bf16 path (gfx950): one workgroup per
// (sequence, head, 64-wide value slice) walks the chunks in order and, per
// chunk of C = 64 tokens, does all of
//
//   G  = cumsum(g)                                  eq. eq_gdn2_gamma (fp32)
//   T  = tril(Ebar Kbar^T, -1), A_qk = tril(Q_g Kbar^T)   eqs. eq_gdn2_gate_matrices,
//                                                   eq_gdn2_wy_matrix, eq_gdn2_chunk_scores
//   A  = (I + T)^{-1}                               fp32 (App. D.4)
//   Y  = A Ebar,  U = A (W*V)                       eq. eq_gdn2_wy_aux
//   R  = U - Y S,  O = Q_g S + A_qk R               eq. eq_gdn2_chunk_output
//   S <- Diag(gamma_C) S + Ktail^T R                eq. eq_gdn2_chunk_state
//
// with the state slice S (Dk x 64, fp32) resident in registers as MFMA
// accumulators and its bf16 hi/lo copy in LDS.  Nothing goes through HBM but
// the inputs, the output and (for the backward recompute) the chunk states.
// The two value slices of one head run on the same XCD so that their shared
// key-side reads hit one L2.
//
// Precision (bf16 MFMA, fp32 accumulate): T and the A side of Y, U use one
// bf16 pass (the solve itself is fp32); Y is kept in bf16 and Y S uses the
// bf16 part of S; every other product is split so that it is fp32-accurate.
//
// The cumulative decay is kept in base 2 (G2 = G * log2(e)) so that every decay
// factor is one v_exp_f32.  Decay ratios gamma_r / gamma_s (r >= s) are formed
// relative to the first row
// p = 16 i of the 16-row block i of r:  exp(G_r - G_p) * exp(G_p - G_s), both
// factors <= 1 except inside the diagonal block, where the second is bounded by
// the decay of one block; a diagonal block whose internal decay exceeds
// e^kDiagLimit is computed element by element instead.

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK, int DV>
struct ScanCfg {
  static constexpr int NTHR = 512;
  static constexpr int DVS = DV < 64 ? DV : 64;  // value columns per workgroup
  static constexpr int NS = DV / DVS;            // value slices per head
  static constexpr int KS = DK / 32;             // K = 32 steps over the key dim
  static constexpr int NCB = DK / 16;            // 16-wide key blocks
  static constexpr int NVB = DVS / 16;           // 16-wide value blocks
  static constexpr int TPW = NCB * NVB / 8;      // state tiles per wave
  // LDS row strides (elements)
  static constexpr int LSS = DK + 8;    // S hi/lo   [DVS][LSS] bf16
  static constexpr int LG = DK + 4;     // G         [64][LG]   fp32
  static constexpr int LKB = DK + 16;   // k, b      [64][LKB]  bf16
  static constexpr int LVW = DVS + 16;  // v, w      [64][LVW]  bf16
  static constexpr int LTA = 64 + 4;    // T -> A    [64][LTA]  fp32
  static constexpr int LAQ = 64 + 8;    // A_qk hi/lo [64][LAQ] bf16
  static constexpr int LR = 64 + 8;     // R hi/lo   [DVS][LR]  bf16 (in the G region)
  static constexpr int LYT = 64 + 16;   // Y^T       [DK][LYT]  bf16 (in the k, b region)
  // byte offsets
  static constexpr int OFF_S = 0;
  static constexpr int SZ_S = 2 * DVS * LSS * 2;
  static constexpr int OFF_G = OFF_S + SZ_S;
  static constexpr int SZ_G = 64 * LG * 4;
  static constexpr int OFF_KB = OFF_G + SZ_G;
  static constexpr int SZ_KB = 2 * 64 * LKB * 2;
  static constexpr int OFF_VW = OFF_KB + SZ_KB;
  static constexpr int SZ_VW = 2 * 64 * LVW * 2;
  static constexpr int OFF_TA = OFF_VW + SZ_VW;
  static constexpr int SZ_TA = 64 * LTA * 4;
  static constexpr int OFF_AQ = OFF_TA + SZ_TA;
  static constexpr int SZ_AQ = 2 * 64 * LAQ * 2;
  // R and Y^T reuse the G and k, b regions when those are large enough (Dk = 128)
  static constexpr int SZ_R = 2 * DVS * LR * 2;
  static constexpr int SZ_YT = DK * LYT * 2;
  static constexpr bool R_IN_G = SZ_R <= SZ_G;
  static constexpr bool YT_IN_KB = SZ_YT <= SZ_KB;
  static constexpr int OFF_X = OFF_AQ + SZ_AQ;
  static constexpr int OFF_R = R_IN_G ? OFF_G : OFF_X;
  static constexpr int OFF_YT = YT_IN_KB ? OFF_KB : OFF_X + (R_IN_G ? 0 : SZ_R);
  static constexpr int OFF_MISC = OFF_X + (R_IN_G ? 0 : SZ_R) + (YT_IN_KB ? 0 : SZ_YT);
  static constexpr int LDS = OFF_MISC + 16;
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(TPW >= 1 && NVB % 2 == 0, "wave split");
};

// T / A_qk tiles (i, j <= i) per wave: row block, first column block, count.
__device__ __forceinline__ void tile_set(int wave, int& i, int& j0, int& n) {
  switch (wave) {
    case 0: i = 0; j0 = 0; n = 1; break;
    case 1: i = 1; j0 = 0; n = 2; break;
    case 2: i = 2; j0 = 0; n = 2; break;
    case 3: i = 2; j0 = 2; n = 1; break;
    default: i = 3; j0 = wave - 4; n = 1; break;
  }
}

template <int DK, int DV, bool WITH_O, bool STORE_H>
__global__ __launch_bounds__(512) void fwd_scan_kernel(ScanFwdArgs a) {
  using C = ScanCfg<DK, DV>;
  constexpr int DVS = C::DVS, NS = C::NS, KS = C::KS, NCB = C::NCB, NVB = C::NVB, TPW = C::TPW;
  constexpr int LSS = C::LSS, LG = C::LG, LKB = C::LKB, LVW = C::LVW, LTA = C::LTA;
  constexpr int LAQ = C::LAQ, LR = C::LR, LYT = C::LYT;
  constexpr int NG = DK / 32, NKB = DK / 64, NVW = DVS / 64;  // 16-byte staging chunks per thread

  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* sShi = reinterpret_cast<__bf16*>(smem + C::OFF_S);
  __bf16* sSlo = sShi + DVS * LSS;
  float* sG = reinterpret_cast<float*>(smem + C::OFF_G);
  __bf16* sRhi = reinterpret_cast<__bf16*>(smem + C::OFF_R);
  __bf16* sRlo = sRhi + DVS * LR;
  __bf16* sK = reinterpret_cast<__bf16*>(smem + C::OFF_KB);
  __bf16* sB = sK + 64 * LKB;
  __bf16* sYT = reinterpret_cast<__bf16*>(smem + C::OFF_YT);
  __bf16* sV = reinterpret_cast<__bf16*>(smem + C::OFF_VW);
  __bf16* sW = sV + 64 * LVW;
  float* sTA = reinterpret_cast<float*>(smem + C::OFF_TA);
  __bf16* sAqhi = reinterpret_cast<__bf16*>(smem + C::OFF_AQ);
  __bf16* sAqlo = sAqhi + 64 * LAQ;
  int* unsafe = reinterpret_cast<int*>(smem + C::OFF_MISC);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  const int T = a.T, H = a.H, NT = a.NT;

  // workgroup -> (sequence, value slice); the slices of one sequence share an XCD
  const int nseq = a.B * H;
  int seq, slice;
  if (NS > 1 && (nseq & 7) == 0) {
    const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
    seq = (j / NS) * 8 + xcd;
    slice = j % NS;
  } else {
    seq = blockIdx.x / NS;
    slice = blockIdx.x % NS;
  }
  const int bb = seq / H, h = seq % H;
  const int v0 = slice * DVS;

  const __bf16* Q = reinterpret_cast<const __bf16*>(a.q);
  const __bf16* K = reinterpret_cast<const __bf16*>(a.k);
  const __bf16* Vg = reinterpret_cast<const __bf16*>(a.v);
  const __bf16* Bg = reinterpret_cast<const __bf16*>(a.b);
  const __bf16* Wg = reinterpret_cast<const __bf16*>(a.w);
  __bf16* O = reinterpret_cast<__bf16*>(a.o);
  const size_t rs = (size_t)H * DK, rsv = (size_t)H * DV;
  auto kofs = [&](int n, int r) -> size_t {
    return ((size_t)bb * T + (size_t)n * 64 + r) * rs + (size_t)h * DK;
  };
  auto vofs = [&](int n, int r) -> size_t {
    return ((size_t)bb * T + (size_t)n * 64 + r) * rsv + (size_t)h * DV + v0;
  };

  // ---- staging of one chunk's inputs.  g stays in registers and is scanned
  // there (thread: NG consecutive rows of 4 channels); k, b go to LDS at the end
  // of the previous chunk; v, w are loaded at the start of the chunk and stored
  // to LDS just before their use.
  constexpr int GCG = DK / 4;     // 4-channel groups of g
  constexpr int GSEG = 512 / GCG; // row segments of g (NG rows each)
  static_assert(GSEG * NG == 64, "g staging covers the chunk");
  const int gcg = tid % GCG, gsg = tid / GCG;
  float4 stg_g[NG];
  uint4 stg_k[NKB], stg_b[NKB], stg_v[NVW], stg_w[NVW];
  auto load_g = [&](int n) {
#pragma unroll
    for (int m = 0; m < NG; ++m)
      stg_g[m] = *reinterpret_cast<const float4*>(a.g + kofs(n, NG * gsg + m) + 4 * gcg);
  };
  auto load_kb = [&](int n) {
#pragma unroll
    for (int m = 0; m < NKB; ++m) {
      const int e = tid + 512 * m, r = e / (DK / 8), c8 = (e % (DK / 8)) * 8;
      stg_k[m] = *reinterpret_cast<const uint4*>(K + kofs(n, r) + c8);
      stg_b[m] = *reinterpret_cast<const uint4*>(Bg + kofs(n, r) + c8);
    }
  };
  auto store_kb = [&]() {
#pragma unroll
    for (int m = 0; m < NKB; ++m) {
      const int e = tid + 512 * m, r = e / (DK / 8), c8 = (e % (DK / 8)) * 8;
      *reinterpret_cast<uint4*>(sK + r * LKB + c8) = stg_k[m];
      *reinterpret_cast<uint4*>(sB + r * LKB + c8) = stg_b[m];
    }
  };
  auto load_vw = [&](int n) {
#pragma unroll
    for (int m = 0; m < NVW; ++m) {
      const int e = tid + 512 * m, r = e / (DVS / 8), c8 = (e % (DVS / 8)) * 8;
      stg_v[m] = *reinterpret_cast<const uint4*>(Vg + vofs(n, r) + c8);
      stg_w[m] = *reinterpret_cast<const uint4*>(Wg + vofs(n, r) + c8);
    }
  };
  auto store_vw = [&]() {
#pragma unroll
    for (int m = 0; m < NVW; ++m) {
      const int e = tid + 512 * m, r = e / (DVS / 8), c8 = (e % (DVS / 8)) * 8;
      *reinterpret_cast<uint4*>(sV + r * LVW + c8) = stg_v[m];
      *reinterpret_cast<uint4*>(sW + r * LVW + c8) = stg_w[m];
    }
  };

  // ---- per-wave roles
  int iT, jT0, nTt;
  tile_set(wave, iT, jT0, nTt);   // T / A_qk tiles
  const int iO = wave >> 1;       // row block of the R, U and O tiles
  const int vbO = (wave & 1) * (NVB / 2);
  const int cs = wave % NCB;      // key block of the state tiles and of Y
  const int sv0 = (wave / NCB) * TPW;

  // query fragments (rows of blocks iT and iO, all key steps), loaded while G is formed
  uint4 qT[KS], qO[KS];
  auto load_q = [&](int n) {
#pragma unroll
    for (int p = 0; p < KS; ++p) {
      qT[p] = *reinterpret_cast<const uint4*>(Q + kofs(n, 16 * iT + r16) + 32 * p + 8 * g);
      if (WITH_O) qO[p] = *reinterpret_cast<const uint4*>(Q + kofs(n, 16 * iO + r16) + 32 * p + 8 * g);
    }
  };

  // ---- state: S tiles (key block cs, value blocks sv0..) as fp32 accumulators
  f4 sreg[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int vb = sv0 + t;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = 16 * cs + 4 * g + u, v = 16 * vb + r16;
      sreg[t][u] = a.S0 ? a.S0[((size_t)seq * DK + c) * DV + v0 + v] : 0.f;
    }
    st4split(sShi + (16 * vb + r16) * LSS + 16 * cs + 4 * g, sSlo + (16 * vb + r16) * LSS + 16 * cs + 4 * g,
             sreg[t]);
  }
  // upper (j > i) blocks of T/A and A_qk stay zero for the whole call
  for (int e = tid; e < 6 * 256; e += 512) {
    const int blk = e >> 8, rr = (e & 255) >> 4, cc = e & 15;
    const int bi = blk < 3 ? 0 : (blk < 5 ? 1 : 2);
    const int bj = blk < 3 ? blk + 1 : (blk < 5 ? blk - 1 : 3);
    sTA[(16 * bi + rr) * LTA + 16 * bj + cc] = 0.f;
    sAqhi[(16 * bi + rr) * LAQ + 16 * bj + cc] = (__bf16)0.f;
    sAqlo[(16 * bi + rr) * LAQ + 16 * bj + cc] = (__bf16)0.f;
  }
  load_g(0);
  load_kb(0);
  store_kb();
  __syncthreads();

  for (int n = 0; n < NT; ++n) {
    const size_t ch = (size_t)seq * NT + n;
    // ---------------- P1: G2 = log2(e) * cumsum(g), block safety flags
    load_q(n);
    if (tid < 4) unsafe[tid] = 0;
    {
      float4* tot = reinterpret_cast<float4*>(sV);  // segment totals (v, w region is free here)
      float4 run = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int m = 0; m < NG; ++m) {
        run.x += stg_g[m].x * kLog2e; run.y += stg_g[m].y * kLog2e;
        run.z += stg_g[m].z * kLog2e; run.w += stg_g[m].w * kLog2e;
        stg_g[m] = run;
      }
      tot[gsg * GCG + gcg] = run;
      __syncthreads();
      float4 off = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s2 = 0; s2 < gsg; ++s2) {
        const float4 t4 = tot[s2 * GCG + gcg];
        off.x += t4.x; off.y += t4.y; off.z += t4.z; off.w += t4.w;
      }
#pragma unroll
      for (int m = 0; m < NG; ++m) {
        const float4 v4 = make_float4(stg_g[m].x + off.x, stg_g[m].y + off.y, stg_g[m].z + off.z,
                                      stg_g[m].w + off.w);
        *reinterpret_cast<float4*>(sG + (NG * gsg + m) * LG + 4 * gcg) = v4;
      }
      __syncthreads();
      for (int e = tid; e < 4 * DK; e += 512) {
        const int i = e / DK, cc = e % DK;
        if (sG[(16 * i) * LG + cc] - sG[(16 * i + 15) * LG + cc] > kDiagLimit2) unsafe[i] = 1;
      }
      __syncthreads();
    }

    // ---------------- P2: O^T partial = S^T Q_g^T, then the T and A_qk tiles
    f4 accO[NVB / 2];
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) accO[t] = f4zero();
    if (WITH_O) {
      const int r = 16 * iO + r16;
#pragma unroll
      for (int p = 0; p < KS; ++p) {
        const int c0 = 32 * p + 8 * g;
        float Gr[8], qf[8], qg[8];
        ldf8(sG + r * LG + c0, Gr);
        unpack8(qO[p], qf);
#pragma unroll
        for (int e = 0; e < 8; ++e) qg[e] = qf[e] * ex2(Gr[e]);
        const Fr qgf = split8(qg);
#pragma unroll
        for (int t = 0; t < NVB / 2; ++t) {
          const int vb = vbO + t;
          Fr sf;
          sf.hi = ld8(sShi + (16 * vb + r16) * LSS + c0);
          sf.lo = ld8(sSlo + (16 * vb + r16) * LSS + c0);
          accO[t] = mma3(sf, qgf, accO[t]);
        }
      }
    }
    {
      const bool diag_direct = unsafe[iT] != 0;
      const int rA = 16 * iT + r16;
#pragma unroll 1
      for (int t = 0; t < nTt; ++t) {
        const int j = jT0 + t;
        f4 accT = f4zero(), accA = f4zero();
        if (diag_direct && j == iT) {
          // element by element: every factor 2^(G2_r - G2_s) with r >= s is <= 1
          const int s = 16 * iT + r16;
#pragma unroll 1
          for (int u = 0; u < 4; ++u) {
            const int r = 16 * iT + 4 * g + u;
            float tt = 0.f, ta = 0.f;
            if (r >= s) {
#pragma unroll 1
              for (int c = 0; c < DK; ++c) {
                const float e = ex2(sG[r * LG + c] - sG[s * LG + c]) * (float)sK[s * LKB + c];
                tt += (float)sB[r * LKB + c] * (float)sK[r * LKB + c] * e;
                ta += (float)Q[kofs(n, r) + c] * e;
              }
            }
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) {
              if (uu == u) {
                accT[uu] = tt;
                accA[uu] = ta;
              }
            }
          }
        } else {
          const int sR_ = 16 * j + r16;
#pragma unroll 2
          for (int p = 0; p < KS; ++p) {
            const int c0 = 32 * p + 8 * g;
            float Gr[8], Gp[8], Gs[8], kf[8], bf[8], qf[8], ks[8];
            ldf8(sG + rA * LG + c0, Gr);
            ldf8(sG + (16 * iT) * LG + c0, Gp);
            ldf8(sG + sR_ * LG + c0, Gs);
            unpack8(ld8(sK + rA * LKB + c0), kf);
            unpack8(ld8(sB + rA * LKB + c0), bf);
            unpack8(ld8(sK + sR_ * LKB + c0), ks);
            unpack8(qT[p], qf);
            float le[8], lq[8], rk[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float f = ex2(Gr[e] - Gp[e]);
              le[e] = bf[e] * kf[e] * f;
              lq[e] = qf[e] * f;
              rk[e] = ks[e] * ex2(Gp[e] - Gs[e]);
            }
            const Fr rkf = split8(rk);
            accT = mma(round8(le), rkf.hi, accT);
            accA = mma3(split8(lq), rkf, accA);
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = 16 * iT + 4 * g + u, s = 16 * j + r16;
          sTA[r * LTA + s] = (r > s) ? accT[u] : 0.f;
          const float av = (r >= s) ? accA[u] : 0.f;
          const __bf16 hv = (__bf16)av;
          sAqhi[r * LAQ + s] = hv;
          sAqlo[r * LAQ + s] = (__bf16)(av - (float)hv);
        }
      }
    }
    __syncthreads();

    // ---------------- P3: A = (I + T)^{-1} in place, fp32
    load_vw(n);
    if (wave == 0) {
      const int blk = lane >> 4, cc = lane & 15;
      float x[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float* trow = sTA + (16 * blk + r) * LTA + 16 * blk;
        float a0 = (r == cc) ? 1.f : 0.f, a1 = 0.f;
#pragma unroll
        for (int s = 0; s + 1 < r; s += 2) {
          a0 -= trow[s] * x[s];
          a1 -= trow[s + 1] * x[s + 1];
        }
        if (r & 1) a0 -= trow[r - 1] * x[r - 1];
        x[r] = a0 + a1;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) sTA[(16 * blk + r) * LTA + 16 * blk + cc] = x[r];
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
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const int src = r16 + 16 * st;
          const float m0 = __shfl(M[0], src), m1 = __shfl(M[1], src);
          const float m2 = __shfl(M[2], src), m3 = __shfl(M[3], src);
          const float mv = g == 0 ? m0 : (g == 1 ? m1 : (g == 2 ? m2 : m3));
          res = mfma_f32(sTA[(16 * i + r16) * LTA + 16 * i + 4 * st + g], mv, res);
        }
      }
      __syncthreads();
      if (wave < i) {
#pragma unroll
        for (int u = 0; u < 4; ++u) sTA[(16 * i + 4 * g + u) * LTA + 16 * wave + r16] = -res[u];
      }
      __syncthreads();
    }

    // ---------------- P4: Ktail and Ebar fragments (from G, k, b), then
    // Y = A Ebar straight to LDS as Y^T (bf16) and U = A Z into the R tiles
    store_vw();
    Fr ktf[2], ebf[2];
    float gamC[4];
    {
      const int c = 16 * cs + r16;
      const float GCc = sG[(CH - 1) * LG + c];
#pragma unroll
      for (int u = 0; u < 4; ++u) gamC[u] = ex2(sG[(CH - 1) * LG + 16 * cs + 4 * g + u]);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        float kf[8], Gs[8], kt[8];
        unpack8(ld_tr8(sK, LKB, 32 * kb, 16 * cs, lane), kf);
#pragma unroll
        for (int e = 0; e < 8; ++e) Gs[e] = sG[(32 * kb + 8 * g + e) * LG + c];
#pragma unroll
        for (int e = 0; e < 8; ++e) kt[e] = kf[e] * ex2(GCc - Gs[e]);
        ktf[kb] = split8(kt);
        if (wave < NCB) {
          float bf[8], eb[8];
          unpack8(ld_tr8(sB, LKB, 32 * kb, 16 * cs, lane), bf);
#pragma unroll
          for (int e = 0; e < 8; ++e) eb[e] = bf[e] * kf[e] * ex2(Gs[e]);
          ebf[kb] = split8(eb);
        }
      }
    }
    __syncthreads();  // G, k and b are dead from here on (their regions take R and Y^T)
    if (n + 1 < NT) {
      load_g(n + 1);
      load_kb(n + 1);
    }
    if (wave < NCB) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f4 acc = f4zero();
#pragma unroll
        for (int kb = 0; kb <= (i >> 1); ++kb) {
          float av[8];
          ldf8(sTA + (16 * i + r16) * LTA + 32 * kb + 8 * g, av);
          acc = mma2b(round8(av), ebf[kb], acc);
        }
        st4(sYT + (16 * cs + r16) * LYT + 16 * i + 4 * g, acc[0], acc[1], acc[2], acc[3]);
      }
    }
    f4 racc[NVB / 2];
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) racc[t] = f4zero();
#pragma unroll
    for (int kb = 0; kb <= (iO >> 1); ++kb) {
      float av[8];
      ldf8(sTA + (16 * iO + r16) * LTA + 32 * kb + 8 * g, av);
      const bf8 ah = round8(av);
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const int vb = vbO + t;
        float vf[8], wf[8], z[8];
        unpack8(ld_tr8(sV, LVW, 32 * kb, 16 * vb, lane), vf);
        unpack8(ld_tr8(sW, LVW, 32 * kb, 16 * vb, lane), wf);
#pragma unroll
        for (int e = 0; e < 8; ++e) z[e] = vf[e] * wf[e];
        racc[t] = mma2b(ah, split8(z), racc[t]);
      }
    }
    __syncthreads();

    // ---------------- P5: R = U - Y S
#pragma unroll
    for (int p = 0; p < KS; ++p) {
      const bf8 yf = neg8(ld_tr8(sYT, LYT, 32 * p, 16 * iO, lane));
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const int vb = vbO + t;
        racc[t] = mma(yf, ld8(sShi + (16 * vb + r16) * LSS + 32 * p + 8 * g), racc[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) {
      const int vb = vbO + t;
      st4split(sRhi + (16 * vb + r16) * LR + 16 * iO + 4 * g, sRlo + (16 * vb + r16) * LR + 16 * iO + 4 * g,
               racc[t]);
      if (STORE_H) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          a.Rs[(ch * CH + 16 * iO + 4 * g + u) * DV + v0 + 16 * vb + r16] = racc[t][u];
      }
    }
    __syncthreads();

    // ---------------- P6: O^T += R^T A_qk^T; S <- Diag(gamma_C) S + Ktail^T R
    if (WITH_O) {
#pragma unroll
      for (int kb = 0; kb <= (iO >> 1); ++kb) {
        Fr af;
        af.hi = ld8(sAqhi + (16 * iO + r16) * LAQ + 32 * kb + 8 * g);
        af.lo = ld8(sAqlo + (16 * iO + r16) * LAQ + 32 * kb + 8 * g);
#pragma unroll
        for (int t = 0; t < NVB / 2; ++t) {
          const int vb = vbO + t;
          Fr rf;
          rf.hi = ld8(sRhi + (16 * vb + r16) * LR + 32 * kb + 8 * g);
          rf.lo = ld8(sRlo + (16 * vb + r16) * LR + 32 * kb + 8 * g);
          accO[t] = mma3(rf, af, accO[t]);
        }
      }
      const float sc = a.scale;
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const int vb = vbO + t;
        st4(O + vofs(n, 16 * iO + r16) + 16 * vb + 4 * g, sc * accO[t][0], sc * accO[t][1], sc * accO[t][2],
            sc * accO[t][3]);
      }
    }
    if (STORE_H) {
#pragma unroll
      for (int t = 0; t < TPW; ++t)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          a.Hs[(ch * DK + 16 * cs + 4 * g + u) * DV + v0 + 16 * (sv0 + t) + r16] = sreg[t][u];
    }
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) sreg[t][u] *= gamC[u];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        const int vb = sv0 + t;
        Fr rf;
        rf.hi = ld8(sRhi + (16 * vb + r16) * LR + 32 * kb + 8 * g);
        rf.lo = ld8(sRlo + (16 * vb + r16) * LR + 32 * kb + 8 * g);
        sreg[t] = mma3(ktf[kb], rf, sreg[t]);
      }
    }
    __syncthreads();

    // ---------------- P7: new S to LDS; next chunk's inputs to LDS
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int vb = sv0 + t;
      st4split(sShi + (16 * vb + r16) * LSS + 16 * cs + 4 * g, sSlo + (16 * vb + r16) * LSS + 16 * cs + 4 * g,
               sreg[t]);
    }
    if (n + 1 < NT) store_kb();
    __syncthreads();
  }

  if (a.ST) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        a.ST[((size_t)seq * DK + 16 * cs + 4 * g + u) * DV + v0 + 16 * (sv0 + t) + r16] = sreg[t][u];
  }
}

template <int DK, int DV, bool WITH_O, bool STORE_H>
hipError_t launch_fwd_scan(const ScanFwdArgs& a, hipStream_t st) {
  using C = ScanCfg<DK, DV>;
  const void* fn = reinterpret_cast<const void*>(&fwd_scan_kernel<DK, DV, WITH_O, STORE_H>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  dim3 grid(a.B * a.H * C::NS);
  hipLaunchKernelGGL((fwd_scan_kernel<DK, DV, WITH_O, STORE_H>), grid, dim3(C::NTHR), C::LDS, st, a);
  return hipGetLastError();
}

#define GDR2_INST_SCAN(DK, DV)                                                           \
  template hipError_t launch_fwd_scan<DK, DV, true, false>(const ScanFwdArgs&, hipStream_t); \
  template hipError_t launch_fwd_scan<DK, DV, false, true>(const ScanFwdArgs&, hipStream_t);

GDR2_INST_SCAN(64, 64)
GDR2_INST_SCAN(64, 128)
GDR2_INST_SCAN(128, 64)
GDR2_INST_SCAN(128, 128)

}  // namespace gdr2

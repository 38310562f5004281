// Chunk-parallel backward of the bf16 path (gfx950), App. B.2 - B.5 in one
// kernel: one 4-wave workgroup per chunk-head, two workgroups per CU.
//
// Per chunk it reads the chunk-start state h = S_0 and the gradient dh of the
// chunk-end state (fp32 [Dk][Dv]), R (fp32 [C][Dv]) from the recompute scan, dR
// from the reverse scan and A = (I + T)^{-1} from the intra-chunk recompute
// (both split bf16 fragment blocks), and q, k, v, b, w, g, dO.
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
// Work split: wave i owns the 16 chunk rows of block i: its dZ rows, the dT /
// dA_qk tiles (i, j <= i) and every output tile (i, key block).  The key
// blocks run in a loop; each stages its h and dh rows and its G2, k, b, q
// columns in LDS while the next block's loads are in flight.  dT and dA_qk
// live in LDS transposed ([s][r], split hi/lo) so that both the row-r and the
// column-s operands of the decay products are plain or transposed reads.
//
// Decay factors (App. D.4 / the forward kernels): for the products over s <= r
// of row block i the factor is split at p = 16 i, 2^(G2_r - G2_p) after the
// product and 2^(G2_p - G2_s) inside the operand; for the products over r >= s
// of key-row block i it is split at e = 16 i + 15.  Both inner factors are <= 1
// outside the diagonal block and bounded by one block's decay inside it; a
// diagonal block whose decay exceeds e^60 is formed element by element.
//
// Precision: every product is fp32-accurate (split hi/lo; dO is exact bf16).

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK, int DV>
struct BChunkCfg {
  static constexpr int NTHR = 256;
  static constexpr int NCB = DK / 16, NVB = DV / 16, KV = DV / 32;
  static constexpr int LT = 64 + 8;   // dT^T, dA_qk^T planes, bf16 [64][LT]
  static constexpr int LGT = 64 + 4;  // G2 columns of a key block, fp32 [16][LGT]
  static constexpr int LXT = 64 + 8;  // k, b, q columns of a key block, bf16 [16][LXT]
  static constexpr int LH = DV + 8;   // h, dh rows of a key block, bf16 hi/lo [16][LH]
  static constexpr int OFF_T = 0;
  static constexpr int OFF_G = OFF_T + 4 * 64 * LT * 2;
  static constexpr int OFF_X = OFF_G + 16 * LGT * 4;
  static constexpr int OFF_H = OFF_X + 3 * 16 * LXT * 2;
  static constexpr int OFF_HH = OFF_H + 4 * 16 * LH * 2;  // rowsum(dh * h)      [2][16]
  static constexpr int OFF_BT = OFF_HH + 2 * 16 * 4;      // dG block totals     [2][4][16]
  static constexpr int OFF_TL = OFF_BT + 2 * 4 * 16 * 4;  // tail-key sums       [2][4][16]
  static constexpr int OFF_GT = OFF_TL + 2 * 4 * 16 * 4;  // G2 wave totals      [4][DK]
  static constexpr int OFF_U = OFF_GT + 4 * DK * 4;       // unsafe diagonal flags [4]
  static constexpr int LDS = OFF_U + 16;
  static_assert(LDS <= 80 * 1024, "two workgroups per CU");
  static_assert(16 * DV / 8 <= NTHR, "one 8-value piece of h / dh per thread");
};

// eight bf16 of a row: elements 0..3 at p, 4..7 at p + 16 (the permuted K order)
__device__ __forceinline__ bf8 ld_p8(const __bf16* p) {
  const bf4 x = *reinterpret_cast<const bf4*>(p);
  const bf4 y = *reinterpret_cast<const bf4*>(p + 16);
  bf8 r;
  r[0] = x[0]; r[1] = x[1]; r[2] = x[2]; r[3] = x[3];
  r[4] = y[0]; r[5] = y[1]; r[6] = y[2]; r[7] = y[3];
  return r;
}
__device__ __forceinline__ bf8 ldg_bf8(const unsigned char* p) { return *reinterpret_cast<const bf8*>(p); }
__device__ __forceinline__ float4 ldg_f4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ Fr split_f44(const float4& x, const float4& y) {
  const float v[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
  return split8(v);
}

template <int DK, int DV>
__global__ __launch_bounds__(256, 2) void bchunk_bf16_kernel(BChunkBf16Args a) {
  using C = BChunkCfg<DK, DV>;
  constexpr int NCB = C::NCB, NVB = C::NVB, KV = C::KV;
  constexpr int LT = C::LT, LGT = C::LGT, LXT = C::LXT, LH = C::LH;

  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* sTh = reinterpret_cast<__bf16*>(smem + C::OFF_T);  // dT^T [s][r]
  __bf16* sTl = sTh + 64 * LT;
  __bf16* sAh = sTl + 64 * LT;  // dA_qk^T [s][r]
  __bf16* sAl = sAh + 64 * LT;
  float* sG = reinterpret_cast<float*>(smem + C::OFF_G);     // G2 [c][s]
  __bf16* sKc = reinterpret_cast<__bf16*>(smem + C::OFF_X);  // k [c][s]
  __bf16* sBc = sKc + 16 * LXT;
  __bf16* sQc = sBc + 16 * LXT;
  __bf16* sHh = reinterpret_cast<__bf16*>(smem + C::OFF_H);  // h [c][v]
  __bf16* sHl = sHh + 16 * LH;
  __bf16* sDh = sHl + 16 * LH;  // dh [c][v]
  __bf16* sDl = sDh + 16 * LH;
  float* sHH = reinterpret_cast<float*>(smem + C::OFF_HH);
  float* sBT = reinterpret_cast<float*>(smem + C::OFF_BT);
  float* sTL = reinterpret_cast<float*>(smem + C::OFF_TL);
  float* sGT = reinterpret_cast<float*>(smem + C::OFF_GT);
  int* unsafe = reinterpret_cast<int*>(smem + C::OFF_U);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  const int n = blockIdx.x, h = blockIdx.y, bb = blockIdx.z;
  const int T = a.T, H = a.H, NT = a.NT;
  const size_t ch = ((size_t)bb * H + h) * NT + n;
  const size_t row0 = (size_t)bb * T + (size_t)n * CH;
  const size_t KST = (size_t)H * DK, VST = (size_t)H * DV;
  const size_t kb0 = row0 * KST + (size_t)h * DK, vb0 = row0 * VST + (size_t)h * DV;
  const int i = wave;  // the row block this wave owns

  const __bf16* Qp = reinterpret_cast<const __bf16*>(a.q);
  const __bf16* Kp = reinterpret_cast<const __bf16*>(a.k);
  const __bf16* Vp = reinterpret_cast<const __bf16*>(a.v);
  const __bf16* Bp = reinterpret_cast<const __bf16*>(a.b);
  const __bf16* Wp = reinterpret_cast<const __bf16*>(a.w);
  const __bf16* dOp = reinterpret_cast<const __bf16*>(a.dout);
  __bf16* dQp = reinterpret_cast<__bf16*>(a.dq);
  __bf16* dKp = reinterpret_cast<__bf16*>(a.dk);
  __bf16* dVp = reinterpret_cast<__bf16*>(a.dv);
  __bf16* dBp = reinterpret_cast<__bf16*>(a.db);
  __bf16* dWp = reinterpret_cast<__bf16*>(a.dw);

  // staging role: chunk row grow, channels 16 cb + 4 cq + (0..3) of key block cb
  const int rl = lane >> 2, cq = lane & 3, grow = 16 * wave + rl;
  // h / dh staging role: row hc of the key block, values hv .. hv + 7
  const int hc = (8 * tid) / DV, hv = (8 * tid) % DV;
  const bool hact = tid < 2 * DV;

  // ---- loads: g (all key blocks) and the staging operands of key block 0
  float4 G2v[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) G2v[cb] = ldg_f4(a.g + kb0 + grow * KST + 16 * cb + 4 * cq);
  bf4 pk, pb, pq;
  float4 ph0, ph1, pd0, pd1;
#define GDR2_PREFETCH(CB)                                                                  \
  {                                                                                        \
    const size_t o_ = kb0 + grow * KST + 16 * (CB) + 4 * cq;                               \
    pk = *reinterpret_cast<const bf4*>(Kp + o_);                                           \
    pb = *reinterpret_cast<const bf4*>(Bp + o_);                                           \
    pq = *reinterpret_cast<const bf4*>(Qp + o_);                                           \
    if (hact) {                                                                            \
      const size_t so_ = (ch * DK + 16 * (CB) + hc) * DV + hv;                             \
      ph0 = ldg_f4(a.Hs + so_);                                                            \
      ph1 = ldg_f4(a.Hs + so_ + 4);                                                        \
      pd0 = ldg_f4(a.DH + so_);                                                            \
      pd1 = ldg_f4(a.DH + so_ + 4);                                                        \
    }                                                                                      \
  }
  // writes the staged operands of key block CB into LDS (rowsum(dh * h) into parity PAR)
#define GDR2_STAGE(CB, PAR)                                                                \
  {                                                                                        \
    float4 gs_ = G2v[0];                                                                   \
    _Pragma("unroll") for (int m_ = 1; m_ < NCB; ++m_) if (m_ == (CB)) gs_ = G2v[m_];      \
    sG[(4 * cq + 0) * LGT + grow] = gs_.x;                                                 \
    sG[(4 * cq + 1) * LGT + grow] = gs_.y;                                                 \
    sG[(4 * cq + 2) * LGT + grow] = gs_.z;                                                 \
    sG[(4 * cq + 3) * LGT + grow] = gs_.w;                                                 \
    _Pragma("unroll") for (int u_ = 0; u_ < 4; ++u_) {                                     \
      sKc[(4 * cq + u_) * LXT + grow] = pk[u_];                                            \
      sBc[(4 * cq + u_) * LXT + grow] = pb[u_];                                            \
      sQc[(4 * cq + u_) * LXT + grow] = pq[u_];                                            \
    }                                                                                      \
    if (hact) {                                                                            \
      const Fr hf_ = split_f44(ph0, ph1), df_ = split_f44(pd0, pd1);                       \
      st8(sHh + hc * LH + hv, hf_.hi);                                                     \
      st8(sHl + hc * LH + hv, hf_.lo);                                                     \
      st8(sDh + hc * LH + hv, df_.hi);                                                     \
      st8(sDl + hc * LH + hv, df_.lo);                                                     \
      float hh_ = ph0.x * pd0.x + ph0.y * pd0.y + ph0.z * pd0.z + ph0.w * pd0.w +          \
                  ph1.x * pd1.x + ph1.y * pd1.y + ph1.z * pd1.z + ph1.w * pd1.w;           \
      _Pragma("unroll") for (int o_ = DV / 16; o_ >= 1; o_ >>= 1) hh_ += __shfl_xor(hh_, o_); \
      if ((tid % (DV / 8)) == 0) sHH[(PAR) * 16 + hc] = hh_;                               \
    }                                                                                      \
  }
  GDR2_PREFETCH(0)

  // ---- dZ^T = dR^T A for the key rows s of block i: lane gets
  //      dZ[s = 16 i + r16][v = 16 vb + 4 g + u]
  const int kbl = i >> 1;  // first 32-row block of r with A[r][s] != 0
  f4 zacc[NVB];
  {
    const unsigned char* Ab = a.Am + ch * WsBf16::am();
    const unsigned char* Rb = a.DR + ch * WsBf16::dr(DV);
    Fr af[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      af[kb].hi = ldg_bf8(Ab + (2 * i + kb) * 2048 + 16 * lane);
      af[kb].lo = ldg_bf8(Ab + (2 * i + kb) * 2048 + 1024 + 16 * lane);
    }
#pragma unroll
    for (int vb = 0; vb < NVB; ++vb) {
      zacc[vb] = f4zero();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        if (kb < kbl) continue;
        Fr rf;
        rf.hi = ldg_bf8(Rb + (2 * vb + kb) * 2048 + 16 * lane);
        rf.lo = ldg_bf8(Rb + (2 * vb + kb) * 2048 + 1024 + 16 * lane);
        zacc[vb] = mma3(rf, af[kb], zacc[vb]);
      }
    }
  }
  // dv = dZ * w, dw = dZ * v
  {
    const int s = 16 * i + r16;
#pragma unroll
    for (int vb = 0; vb < NVB; ++vb) {
      const size_t o = vb0 + (size_t)s * VST + 16 * vb + 4 * g;
      const bf4 vv = *reinterpret_cast<const bf4*>(Vp + o);
      const bf4 ww = *reinterpret_cast<const bf4*>(Wp + o);
      bf4 odv, odw;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        odv[u] = (__bf16)(zacc[vb][u] * (float)ww[u]);
        odw[u] = (__bf16)(zacc[vb][u] * (float)vv[u]);
      }
      *reinterpret_cast<bf4*>(dVp + o) = odv;
      *reinterpret_cast<bf4*>(dWp + o) = odw;
    }
  }
  // dZ, dO and R rows of block i as A operands over the values, permuted K:
  // K-step p holds values 32 p + 4 g + (0..3) and 32 p + 16 + 4 g + (0..3)
  Fr zf[KV], rfr[KV];
  bf8 dof[KV];
  {
    const int r = 16 * i + r16;
#pragma unroll
    for (int p = 0; p < KV; ++p) {
      float x[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        x[u] = zacc[2 * p][u];
        x[4 + u] = zacc[2 * p + 1][u];
      }
      zf[p] = split8(x);
      dof[p] = ld_p8(dOp + vb0 + (size_t)r * VST + 32 * p + 4 * g);
      const float* rp = a.Rs + (ch * CH + r) * DV + 32 * p + 4 * g;
      rfr[p] = split_f44(ldg_f4(rp), ldg_f4(rp + 16));
    }
  }

  // ---- dT = -tril(dZ R^T, -1) and dA_qk = tril(scale dO R^T), tiles (i, j <= i),
  //      stored transposed: plane[s][r]
#pragma unroll 1
  for (int j = 0; j <= i; ++j) {
    const int s = 16 * j + r16;
    f4 ta = f4zero(), aa = f4zero();
#pragma unroll
    for (int p = 0; p < KV; ++p) {
      const float* rp = a.Rs + (ch * CH + s) * DV + 32 * p + 4 * g;
      const Fr rj = split_f44(ldg_f4(rp), ldg_f4(rp + 16));
      ta = mma3(zf[p], rj, ta);
      aa = mma2b(dof[p], rj, aa);
    }
    const int rr = 16 * i + 4 * g;
    f4 tv, av;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      tv[u] = (rr + u > s) ? -ta[u] : 0.f;
      av[u] = (rr + u >= s) ? a.scale * aa[u] : 0.f;
    }
    st4split(sTh + s * LT + rr, sTl + s * LT + rr, tv);
    st4split(sAh + s * LT + rr, sAl + s * LT + rr, av);
  }
  // tiles (0,1) and (2,3) above the diagonal share 32-wide operand steps with causal tiles
  if (i == 0 || i == 2) {
    const int s = 16 * (i + 1) + r16, rr = 16 * i + 4 * g;
    st4split(sTh + s * LT + rr, sTl + s * LT + rr, f4zero());
    st4split(sAh + s * LT + rr, sAl + s * LT + rr, f4zero());
  }

  // ---- G2 = log2(e) cumsum(g): scan over the wave's 16 rows, then wave offsets
  {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      G2v[cb].x *= kLog2e; G2v[cb].y *= kLog2e; G2v[cb].z *= kLog2e; G2v[cb].w *= kLog2e;
    }
#pragma unroll
    for (int off = 4; off < 64; off <<= 1) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        const float x0 = __shfl_up(G2v[cb].x, off), x1 = __shfl_up(G2v[cb].y, off);
        const float x2 = __shfl_up(G2v[cb].z, off), x3 = __shfl_up(G2v[cb].w, off);
        if (lane >= off) {
          G2v[cb].x += x0; G2v[cb].y += x1; G2v[cb].z += x2; G2v[cb].w += x3;
        }
      }
    }
    // block i's internal decay G2[16 i] - G2[16 i + 15] (offsets cancel)
    bool bad = false;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const float y0 = __shfl(G2v[cb].x, cq), y1 = __shfl(G2v[cb].y, cq);
      const float y2 = __shfl(G2v[cb].z, cq), y3 = __shfl(G2v[cb].w, cq);
      if (rl == 15)
        bad = bad || (y0 - G2v[cb].x > kDiagLimit2) || (y1 - G2v[cb].y > kDiagLimit2) ||
              (y2 - G2v[cb].z > kDiagLimit2) || (y3 - G2v[cb].w > kDiagLimit2);
    }
    const unsigned long long m = __ballot(bad);
    if (lane == 0) unsafe[wave] = (m != 0ull) ? 1 : 0;
    if (rl == 15) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) *reinterpret_cast<float4*>(sGT + wave * DK + 16 * cb + 4 * cq) = G2v[cb];
    }
  }
  __syncthreads();
  for (int w2 = 0; w2 < wave; ++w2) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const float4 t4 = *reinterpret_cast<const float4*>(sGT + w2 * DK + 16 * cb + 4 * cq);
      G2v[cb].x += t4.x; G2v[cb].y += t4.y; G2v[cb].z += t4.z; G2v[cb].w += t4.w;
    }
  }
  const bool uns = unsafe[i] != 0;
  GDR2_STAGE(0, 0)
  __syncthreads();

  const float scale = a.scale;
#pragma unroll 1
  for (int cb = 0; cb < NCB; ++cb) {
    const int par = cb & 1;
    if (cb + 1 < NCB) GDR2_PREFETCH(cb + 1)
    const int c = 16 * cb + r16;  // this lane's key channel in every output tile

    // X1 = dZ h^T, X2 = dO h^T, X3 = R dh^T   (rows 16 i + 4 g + u, key c)
    f4 x1 = f4zero(), x2 = f4zero(), x3 = f4zero();
#pragma unroll
    for (int p = 0; p < KV; ++p) {
      Fr hf, df;
      hf.hi = ld_p8(sHh + r16 * LH + 32 * p + 4 * g);
      hf.lo = ld_p8(sHl + r16 * LH + 32 * p + 4 * g);
      df.hi = ld_p8(sDh + r16 * LH + 32 * p + 4 * g);
      df.lo = ld_p8(sDl + r16 * LH + 32 * p + 4 * g);
      x1 = mma3(zf[p], hf, x1);
      x2 = mma2b(dof[p], hf, x2);
      x3 = mma3(rfr[p], df, x3);
    }

    const float* gcol = sG + r16 * LGT;
    const float Gp = gcol[16 * i], Ge = gcol[16 * i + 15], GCl = gcol[CH - 1];

    // P1 = dT (k 2^(G2_p - G2_s)),  P2 = dA_qk (k 2^(G2_p - G2_s)),  s <= 16 i + 15
    f4 p1 = f4zero(), p2 = f4zero();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb > kbl) break;
      const int s0 = 32 * kb + 8 * g;
      float Gs[8], ks[8], x[8];
      ldf8(gcol + s0, Gs);
      unpack8(ld8(sKc + r16 * LXT + s0), ks);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int s = s0 + e;
        const bool ok = (s < 16 * i + 16) && !(uns && s >= 16 * i);
        x[e] = ok ? ks[e] * ex2(Gp - Gs[e]) : 0.f;
      }
      const Fr kf = split8(x);
      Fr tf, af;
      tf.hi = ld_tr8(sTh, LT, 32 * kb, 16 * i, lane);
      tf.lo = ld_tr8(sTl, LT, 32 * kb, 16 * i, lane);
      af.hi = ld_tr8(sAh, LT, 32 * kb, 16 * i, lane);
      af.lo = ld_tr8(sAl, LT, 32 * kb, 16 * i, lane);
      p1 = mma3(tf, kf, p1);
      p2 = mma3(af, kf, p2);
    }
    // P3 = dT^T ((b k) 2^(G2_r - G2_e)) + dA_qk^T (q 2^(G2_r - G2_e)),  r >= 16 i
    f4 p3 = f4zero();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb < kbl) continue;
      const int r0 = 32 * kb + 8 * g;
      float Gr[8], kr[8], br[8], qr[8], lb[8], lq[8];
      ldf8(gcol + r0, Gr);
      unpack8(ld8(sKc + r16 * LXT + r0), kr);
      unpack8(ld8(sBc + r16 * LXT + r0), br);
      unpack8(ld8(sQc + r16 * LXT + r0), qr);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int r = r0 + e;
        const bool ok = (r >= 16 * i) && !(uns && r < 16 * i + 16);
        const float f = ex2(Gr[e] - Ge);
        lb[e] = ok ? br[e] * kr[e] * f : 0.f;
        lq[e] = ok ? qr[e] * f : 0.f;
      }
      Fr tf, af;
      tf.hi = ld8(sTh + (16 * i + r16) * LT + r0);
      tf.lo = ld8(sTl + (16 * i + r16) * LT + r0);
      af.hi = ld8(sAh + (16 * i + r16) * LT + r0);
      af.lo = ld8(sAl + (16 * i + r16) * LT + r0);
      p3 = mma3(tf, split8(lb), p3);
      p3 = mma3(af, split8(lq), p3);
    }

    // ---- elementwise chain (App. B.4) on rows rb + u, key c
    const int rb = 16 * i + 4 * g;
    float Gr4[4];
    {
      const float4 t4 = *reinterpret_cast<const float4*>(gcol + rb);
      Gr4[0] = t4.x; Gr4[1] = t4.y; Gr4[2] = t4.z; Gr4[3] = t4.w;
    }
    const bf4 k4 = *reinterpret_cast<const bf4*>(sKc + r16 * LXT + rb);
    const bf4 b4 = *reinterpret_cast<const bf4*>(sBc + r16 * LXT + rb);
    const bf4 q4 = *reinterpret_cast<const bf4*>(sQc + r16 * LXT + rb);
    float dgl[4], tailp = 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float G = Gr4[u];
      const float gam = ex2(G), lf = ex2(G - Gp), rf = ex2(Ge - G), tl = ex2(GCl - G);
      const float kv = (float)k4[u], bv = (float)b4[u], qv = (float)q4[u];
      float dEg = lf * p1[u] - gam * x1[u];
      float dq = scale * gam * x2[u] + lf * p2[u];
      float dKg = rf * p3[u] + tl * x3[u];
      if (uns) {
        // diagonal block element by element: every factor has exponent <= 0
        const int r = rb + u;
#pragma unroll 1
        for (int s = 16 * i; s < 16 * i + 16; ++s) {
          const float Gs = gcol[s];
          const float ks = (float)sKc[r16 * LXT + s];
          if (s <= r) {
            const float e = ex2(G - Gs);
            const float dTv = (s < r) ? (float)sTh[s * LT + r] + (float)sTl[s * LT + r] : 0.f;
            const float dAv = (float)sAh[s * LT + r] + (float)sAl[s * LT + r];
            dEg += dTv * ks * e;
            dq += dAv * ks * e;
          }
          if (s >= r) {
            const float e = ex2(Gs - G);
            const float dTv = (s > r) ? (float)sTh[r * LT + s] + (float)sTl[r * LT + s] : 0.f;
            const float dAv = (float)sAh[r * LT + s] + (float)sAl[r * LT + s];
            dKg += (dTv * (float)sBc[r16 * LXT + s] * ks + dAv * (float)sQc[r16 * LXT + s]) * e;
          }
        }
      }
      const size_t o = kb0 + (size_t)(rb + u) * KST + c;
      dQp[o] = (__bf16)dq;
      dKp[o] = (__bf16)(dEg * bv + dKg);
      dBp[o] = (__bf16)(dEg * kv);
      dgl[u] = dq * qv - dKg * kv + dEg * bv * kv;
      tailp += x3[u] * kv * tl;
    }
    // reverse cumulative sum of dG: within the lane, over the lane groups, then blocks
    const float s3 = dgl[3], s2 = s3 + dgl[2], s1 = s2 + dgl[1], s0 = s1 + dgl[0];
    float y = s0;
    {
      const float t1 = __shfl_down(y, 16);
      if (g < 3) y += t1;
      const float t2 = __shfl_down(y, 32);
      if (g < 2) y += t2;
    }
    float tp = tailp;
    tp += __shfl_xor(tp, 16);
    tp += __shfl_xor(tp, 32);
    if (g == 0) {
      sBT[(par * 4 + i) * 16 + r16] = y;
      sTL[(par * 4 + i) * 16 + r16] = tp;
    }
    const float gamC = ex2(GCl);
    __syncthreads();
    // gamma_C d gamma_C joins row C - 1, hence every row's suffix sum
    float off = gamC * sHH[par * 16 + r16] + (y - s0);
#pragma unroll
    for (int i2 = 0; i2 < 4; ++i2) {
      off += sTL[(par * 4 + i2) * 16 + r16];
      if (i2 > i) off += sBT[(par * 4 + i2) * 16 + r16];
    }
    a.dg[kb0 + (size_t)(rb + 0) * KST + c] = s0 + off;
    a.dg[kb0 + (size_t)(rb + 1) * KST + c] = s1 + off;
    a.dg[kb0 + (size_t)(rb + 2) * KST + c] = s2 + off;
    a.dg[kb0 + (size_t)(rb + 3) * KST + c] = s3 + off;
    if (cb + 1 < NCB) GDR2_STAGE(cb + 1, par ^ 1)
    __syncthreads();
  }
#undef GDR2_PREFETCH
#undef GDR2_STAGE
}

template <int DK, int DV>
hipError_t launch_bchunk_bf16(const BChunkBf16Args& a, hipStream_t st) {
  using C = BChunkCfg<DK, DV>;
  const void* fn = reinterpret_cast<const void*>(&bchunk_bf16_kernel<DK, DV>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  dim3 grid(a.NT, a.H, a.B);
  hipLaunchKernelGGL((bchunk_bf16_kernel<DK, DV>), grid, dim3(C::NTHR), C::LDS, st, a);
  return hipGetLastError();
}

template hipError_t launch_bchunk_bf16<64, 64>(const BChunkBf16Args&, hipStream_t);
template hipError_t launch_bchunk_bf16<64, 128>(const BChunkBf16Args&, hipStream_t);
template hipError_t launch_bchunk_bf16<128, 64>(const BChunkBf16Args&, hipStream_t);
template hipError_t launch_bchunk_bf16<128, 128>(const BChunkBf16Args&, hipStream_t);

}  // namespace gdr2

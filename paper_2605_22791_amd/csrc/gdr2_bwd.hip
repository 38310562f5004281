// Backward kernels of the chunkwise WY GDR-2 operator (gfx950), App. B / App. C.3.
//
//   bwd_state  reverse inter-chunk scan (state and output paths, App. B.1):
//                dR_n  = scale * Aqk^T dO_n + Ktail dS_{n+1}
//                dS_n  = Diag(gamma_C) dS_{n+1} + scale * Qg^T dO_n - Y^T dR_n
//              one workgroup per (value slice, head, batch), dS slice in LDS.
//   bwd_wy     the gate-aware WY vector-Jacobian product (App. B.2, the
//              method-specific step): dA_qk, dY = -dR S0^T, dZ = A^T dR (-> dw,
//              dv), dEbar = A^T dY, dA = dR Z^T + dY Ebar^T with the gates inside
//              the products, dT = -tril(A^T dA A^T, -1).
//   bwd_intra  the score / Gram / tail-key VJPs and the elementwise decay chain
//              (App. B.3 - B.5): dq, dk, db and dlog_alpha by a reverse
//              cumulative sum over the chunk.
//
// Every gamma^{-1} of App. B is paired with a gamma of the same channel so that
// only ratios exp(G_r - G_s), r >= s, appear; they are formed with the block
// factorisation described in gdr2_device.hpp.  Writing dEg = dEbar*gamma,
// dKg = dKbar/gamma and dq = dQg*gamma, App. B.4 becomes
//     db = dEg*k,  dk = dEg*b + dKg,  dG = dq*q - dKg*k + dEg*b*k,
// and d gamma_C (App. B.1, B.3) is added to the last row of dG (gamma_C is
// gamma at row C) before the reverse cumulative sum.

#include "gdr2_kernels.hpp"

namespace gdr2 {

// ---------------------------------------------------------------------------
template <int DK, int DV, int DVS, typename TIn>
__global__ __launch_bounds__(256) void bwd_state_kernel(BwdStateArgs<TIn> a) {
  constexpr int NTHR = 256, NW = 4;
  constexpr int LSS = DVS + 4;
  constexpr int NVB = DVS / 16;
  const int vs = blockIdx.x, h = blockIdx.y, bb = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int T = a.T, H = a.H, NT = a.NT;
  const int v0 = vs * DVS;
  const size_t seq = (size_t)scan_pair(a.vl, bb * H + h, H);  // (sequence, head) pair
  const ScanRange rng = scan_range(a.vl, (int)seq, H, NT);

  __shared__ float sdS[DK * LSS];
  __shared__ float sdO[CH * LSS];
  __shared__ float sdR[CH * LSS];

  for (int e = tid; e < DK * DVS; e += NTHR) {
    const int c = e / DVS, v = e % DVS;
    sdS[c * LSS + v] = a.dST ? a.dST[(seq * DK + c) * DV + v0 + v] : 0.f;
  }
  __syncthreads();

  for (int n = rng.c1 - 1; n >= rng.c0; --n) {
    const size_t ch = rng.chs + n;
    const float* Qg = a.Qg + ch * CH * DK;
    const float* Kt = a.Kt + ch * CH * DK;
    const float* Y = a.Y + ch * CH * DK;
    const float* Aqk = a.Aqk + ch * CH * CH;
    const float* GC = a.GC + ch * DK;
    size_t orow0;
    int olen;
    scan_rows(a.vl, (int)seq, H, T, n, orow0, olen);

    for (int e = tid; e < CH * DVS; e += NTHR) {
      const int r = e / DVS, v = e % DVS;
      sdO[r * LSS + v] = a.scale * to_fz(a.dout + ((orow0 + r) * H + h) * DV + v0 + v, r < olen);
    }
    {
      float* DHn = a.DH + ch * DK * DV;
      for (int e = tid; e < DK * DVS; e += NTHR) {
        const int c = e / DVS, v = e % DVS;
        DHn[c * DV + v0 + v] = sdS[c * LSS + v];
      }
    }
    __syncthreads();

    // dR = Aqk^T dO + Ktail dS   (wave -> row block of dR)
    {
      const int i = wave;
      f4 acc[NVB];
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb) acc[vb] = f4{0.f, 0.f, 0.f, 0.f};
      for (int kk = 16 * i; kk < CH; kk += 4) {
        const int r = kk + lg;
        const float av = Aqk[r * CH + 16 * i + lr];
#pragma unroll
        for (int vb = 0; vb < NVB; ++vb) acc[vb] = mfma4(av, sdO[r * LSS + 16 * vb + lr], acc[vb]);
      }
      const float* pk = Kt + (16 * i + lr) * DK + 4 * lg;
      for (int kk = 0; kk < DK; kk += 16) {
        const float4 kt = ld4(pk + kk);
        const int c0 = kk + 4 * lg;
#pragma unroll
        for (int vb = 0; vb < NVB; ++vb) {
          acc[vb] = mfma4(kt.x, sdS[(c0 + 0) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(kt.y, sdS[(c0 + 1) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(kt.z, sdS[(c0 + 2) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(kt.w, sdS[(c0 + 3) * LSS + 16 * vb + lr], acc[vb]);
        }
      }
      float* DRn = a.DR + ch * CH * DV;
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = 16 * i + 4 * lg + u;
          sdR[r * LSS + 16 * vb + lr] = acc[vb][u];
          DRn[r * DV + v0 + 16 * vb + lr] = acc[vb][u];
        }
    }
    __syncthreads();

    // dS <- Diag(gamma_C) dS + Qg^T dO - Y^T dR
    constexpr int NTILE = (DK / 16) * NVB;
    constexpr int TPW = (NTILE + NW - 1) / NW;
    f4 nacc[TPW];
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
      const int t = wave + q * NW;
      if (t < NTILE) {
        const int cb = t / NVB, vb = t % NVB;
        f4 acc;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = 16 * cb + 4 * lg + u;
          acc[u] = GC[c] * sdS[c * LSS + 16 * vb + lr];
        }
        for (int kk = 0; kk < CH; kk += 4) {
          const int r = kk + lg;
          acc = mfma4(Qg[r * DK + 16 * cb + lr], sdO[r * LSS + 16 * vb + lr], acc);
          acc = mfma4(-Y[r * DK + 16 * cb + lr], sdR[r * LSS + 16 * vb + lr], acc);
        }
        nacc[q] = acc;
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < TPW; ++q) {
      const int t = wave + q * NW;
      if (t < NTILE) {
        const int cb = t / NVB, vb = t % NVB;
#pragma unroll
        for (int u = 0; u < 4; ++u) sdS[(16 * cb + 4 * lg + u) * LSS + 16 * vb + lr] = nacc[q][u];
      }
    }
    __syncthreads();
  }
  if (a.dS0) {
    for (int e = tid; e < DK * DVS; e += NTHR) {
      const int c = e / DVS, v = e % DVS;
      a.dS0[(seq * DK + c) * DV + v0 + v] = sdS[c * LSS + v];
    }
  }
}

// ---------------------------------------------------------------------------
// Gate-aware WY VJP.  Writes dv, dw (final), and per chunk-head workspace:
//   DAqk (64x64) = tril(scale dO R^T),  DT (64x64) strict lower,
//   DEg (64xDK)  = (A^T dY) * gamma  with dY = -dR S0^T.
template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(512) void bwd_wy_kernel(BwdChunkArgs<TIn> a) {
  constexpr int NTHR = 512, NW = 8;
  constexpr int LS = DK + 4;
  ChunkPos cp;
  if (!chunk_pos(a.vl, blockIdx.x, blockIdx.y, blockIdx.z, a.T, a.H, a.NT, cp)) return;
  const int h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int H = a.H;
  const size_t rs = (size_t)(H / a.G) * DK, rsv = (size_t)H * DV;  // key side on the H / G key heads
  const size_t row0 = cp.row0;
  const int len = cp.len;  // rows in use: the rest read as zero and are not written
  const size_t kbase = row0 * rs + (size_t)(h / a.G) * DK;
  const size_t vbase = row0 * rsv + (size_t)h * DV;
  const size_t ch = cp.ch;

  extern __shared__ float smem[];
  float* sR0 = smem;                // G, later X = A^T dA (LD64)
  float* sLe = sR0 + CH * LS;       // b*k*exp(G_r - G_p)
  float* sRk = sLe + CH * LS;       // k*exp(G_e - G_s); later solve scratch, then dY
  float* sTd = sRk + CH * LS;       // T, later dA (LD64)
  float* sA = sTd + CH * LD64;      // A (LD64)
  float* eP = sA + CH * LD64;
  float* brg = eP + 4 * DK;
  float* eGC = brg + 10 * DK;
  int* unsafe = reinterpret_cast<int*>(eGC + DK);
  float* sG = sR0;
  float* sX = sR0;
  float* sdY = sRk;

  const float* Hn = a.Hs + ch * DK * DV;
  const float* Rn = a.Rs + ch * CH * DV;
  const float* DRn = a.DR + ch * CH * DV;
  float* DAqk = a.DAqk + ch * CH * CH;
  float* DT = a.DT + ch * CH * CH;
  float* DEg = a.DEg + ch * CH * DK;

  if (tid < 4) unsafe[tid] = 0;
  chunk_cumsum<DK, NTHR>(a.g + kbase, rs, sG, tid, len);
  chunk_refs<DK, NTHR>(sG, eP, brg, eGC, unsafe, tid);
  for (int e = tid; e < CH * DK / 4; e += NTHR) {
    const int r = e / (DK / 4), c4 = (e % (DK / 4)) * 4, i = r >> 4;
    const float4 kk = ld4z(a.k + kbase + r * rs + c4, r < len);
    const float4 bv = ld4z(a.b + kbase + r * rs + c4, r < len);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c4 + u;
      const float G = sG[r * LS + c];
      const float kv = f4at(kk, u);
      sLe[r * LS + c] = f4at(bv, u) * kv * expf(G - sG[(16 * i) * LS + c]);
      sRk[r * LS + c] = kv * expf(sG[(16 * i + 15) * LS + c] - G);
    }
  }
  __syncthreads();

  // T tiles (10) into sTd, and the 16 tiles of dA_qk = tril(scale dO R^T)
  for (int it = wave; it < 26; it += NW) {
    if (it < 10) {
      int i, j;
      pair_of(it, i, j);
      const f4 acc = (i == j && unsafe[i])
                         ? diag_tile_direct<DK, TIn>(a.b + kbase, a.k + kbase, a.k + kbase,
                                                     a.g + kbase, rs, i, lane, true, len)
                         : gram_tile<DK>(sLe, sRk, brg + pair_index(i, j) * DK, i, j, lane);
      const int s = 16 * j + lr;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = 16 * i + 4 * lg + u;
        sTd[r * LD64 + s] = (r > s) ? acc[u] : 0.f;
      }
    } else {
      const int i = (it - 10) >> 2, j = (it - 10) & 3;
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      if (j <= i) {
        const TIn* pd = a.dout + vbase + (16 * i + lr) * rsv + 4 * lg;
        const bool pdin = 16 * i + lr < len;
        const float* pr = Rn + (16 * j + lr) * DV + 4 * lg;
        for (int kk = 0; kk < DV; kk += 16) {
          const float4 dv4 = ld4z(pd + kk, pdin), r4 = ld4(pr + kk);
          acc = mfma4(dv4.x, r4.x, acc);
          acc = mfma4(dv4.y, r4.y, acc);
          acc = mfma4(dv4.z, r4.z, acc);
          acc = mfma4(dv4.w, r4.w, acc);
        }
      }
      const int s = 16 * j + lr;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = 16 * i + 4 * lg + u;
        DAqk[r * CH + s] = (r >= s) ? a.scale * acc[u] : 0.f;
      }
    }
  }
  __syncthreads();

  wy_solve<NTHR>(sTd, sA, sRk, tid);  // sRk is dead after T; used as scratch

  // dY = -dR S0^T  (64 x DK) into sdY
  for (int it = wave; it < 4 * (DK / 16); it += NW) {
    const int i = it / (DK / 16), cb = it % (DK / 16);
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    const float* pa = DRn + (16 * i + lr) * DV + 4 * lg;
    const float* pb = Hn + (16 * cb + lr) * DV + 4 * lg;
    for (int kk = 0; kk < DV; kk += 16) {
      const float4 x = ld4(pa + kk), y = ld4(pb + kk);
      acc = mfma4(-x.x, y.x, acc);
      acc = mfma4(-x.y, y.y, acc);
      acc = mfma4(-x.z, y.z, acc);
      acc = mfma4(-x.w, y.w, acc);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) sdY[(16 * i + 4 * lg + u) * LS + 16 * cb + lr] = acc[u];
  }
  __syncthreads();

  // dZ = A^T dR (-> dw = dZ*v, dv = dZ*w) and dEg = (A^T dY) * gamma
  for (int it = wave; it < 4 * (DV / 16) + 4 * (DK / 16); it += NW) {
    const bool isZ = it < 4 * (DV / 16);
    const int idx = isZ ? it : it - 4 * (DV / 16);
    const int NB = isZ ? DV / 16 : DK / 16;
    const int i = idx / NB, cb = idx % NB;
    const int col = 16 * cb + lr;
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int kk = 16 * i; kk < CH; kk += 4) {
      const int r = kk + lg;
      const float av = sA[r * LD64 + 16 * i + lr];
      const float bv = isZ ? DRn[r * DV + col] : sdY[r * LS + col];
      acc = mfma4(av, bv, acc);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int s = 16 * i + 4 * lg + u;
      if (isZ) {
        const size_t off = vbase + s * rsv + col;
        if (s < len) {
          put(a.dw + off, acc[u] * to_f(a.v[off]));
          put(a.dv + off, acc[u] * to_f(a.w[off]));
        }
      } else {
        DEg[s * DK + col] = acc[u] * expf(sG[s * LS + col]);
      }
    }
  }
  __syncthreads();  // sG and T dead from here on

  // dA = dR Z^T + dY Ebar^T, strictly lower part, into sTd
  for (int it = wave; it < 16; it += NW) {
    const int i = it >> 2, j = it & 3;
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    if (j <= i) {
      const float* pa = DRn + (16 * i + lr) * DV + 4 * lg;
      const TIn* pw = a.w + vbase + (16 * j + lr) * rsv + 4 * lg;
      const TIn* pv = a.v + vbase + (16 * j + lr) * rsv + 4 * lg;
      const bool jin = 16 * j + lr < len;
      for (int kk = 0; kk < DV; kk += 16) {
        const float4 x = ld4(pa + kk), w4 = ld4z(pw + kk, jin), v4 = ld4z(pv + kk, jin);
        acc = mfma4(x.x, w4.x * v4.x, acc);
        acc = mfma4(x.y, w4.y * v4.y, acc);
        acc = mfma4(x.z, w4.z * v4.z, acc);
        acc = mfma4(x.w, w4.w * v4.w, acc);
      }
      const float* py = sdY + (16 * i + lr) * LS + 4 * lg;
      const float* pe = sLe + (16 * j + lr) * LS + 4 * lg;
      const float* pp = eP + j * DK + 4 * lg;
      for (int kk = 0; kk < DK; kk += 16) {
        const float4 x = ld4(py + kk), e4 = ld4(pe + kk), p4 = ld4(pp + kk);
        acc = mfma4(x.x, e4.x * p4.x, acc);
        acc = mfma4(x.y, e4.y * p4.y, acc);
        acc = mfma4(x.z, e4.z * p4.z, acc);
        acc = mfma4(x.w, e4.w * p4.w, acc);
      }
    }
    const int s = 16 * j + lr;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 16 * i + 4 * lg + u;
      sTd[r * LD64 + s] = (r > s) ? acc[u] : 0.f;
    }
  }
  __syncthreads();

  // X = A^T dA, lower tiles
  for (int it = wave; it < 10; it += NW) {
    int i, j;
    pair_of(it, i, j);
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int kk = 16 * i; kk < CH; kk += 4) {
      const int p = kk + lg;
      acc = mfma4(sA[p * LD64 + 16 * i + lr], sTd[p * LD64 + 16 * j + lr], acc);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) sX[(16 * i + 4 * lg + u) * LD64 + 16 * j + lr] = acc[u];
  }
  __syncthreads();

  // dT = -tril(X A^T, -1)
  for (int it = wave; it < 16; it += NW) {
    const int i = it >> 2, j = it & 3;
    f4 acc = {0.f, 0.f, 0.f, 0.f};
    if (j <= i) {
      for (int kb = 0; kb <= j; ++kb) {
        const float4 x = ld4(sX + (16 * i + lr) * LD64 + 16 * kb + 4 * lg);
        const float4 y = ld4(sA + (16 * j + lr) * LD64 + 16 * kb + 4 * lg);
        acc = mfma4(x.x, y.x, acc);
        acc = mfma4(x.y, y.y, acc);
        acc = mfma4(x.z, y.z, acc);
        acc = mfma4(x.w, y.w, acc);
      }
    }
    const int s = 16 * j + lr;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 16 * i + 4 * lg + u;
      DT[r * CH + s] = (r > s) ? -acc[u] : 0.f;
    }
  }
}

// ---------------------------------------------------------------------------
// Intra-chunk VJP and decay chain: dq, dk, db, dlog_alpha.
template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(512) void bwd_intra_kernel(BwdChunkArgs<TIn> a) {
  constexpr int NTHR = 512, NW = 8;
  constexpr int LS = DK + 4;
  constexpr int NCB = DK / 16;
  constexpr int NITEM = 4 * NCB;
  constexpr int IPW = NITEM / NW;
  constexpr int NSPLIT = NTHR / DK;
  static_assert(NITEM % NW == 0, "items per wave");
  ChunkPos cp;
  if (!chunk_pos(a.vl, blockIdx.x, blockIdx.y, blockIdx.z, a.T, a.H, a.NT, cp)) return;
  const int h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int H = a.H;
  const size_t rs = (size_t)(H / a.G) * DK, rsv = (size_t)H * DV;  // key side on the H / G key heads
  const size_t row0 = cp.row0;
  const int len = cp.len;  // rows in use: the rest read as zero and are not written
  const size_t kbase = row0 * rs + (size_t)(h / a.G) * DK;
  // key-side gradients: with grouped value heads (G > 1) this value head's
  // contribution goes, on the value-head axis, to the fp32 partials the group
  // reduction sums
  const size_t rso = a.G > 1 ? (size_t)H * DK : rs;
  const size_t kobase = a.G > 1 ? row0 * rso + (size_t)h * DK : kbase;
  const size_t vbase = row0 * rsv + (size_t)h * DV;
  const size_t ch = cp.ch;

  extern __shared__ float smem[];
  float* sG = smem;
  float* sLe = sG + CH * LS;
  float* sLq = sLe + CH * LS;
  float* sRk = sLq + CH * LS;
  float* eP = sRk + CH * LS;
  float* brg = eP + 4 * DK;
  float* eGC = brg + 10 * DK;
  float* colp = eGC + DK;          // [4 row blocks][4 lane groups][DK]
  float* dgp = colp + 16 * DK;     // [DK][NSPLIT]
  int* unsafe = reinterpret_cast<int*>(dgp + DK * NSPLIT);
  float* sdG = sLq;                // reused after the item loop

  const float* Hn = a.Hs + ch * DK * DV;
  const float* DHn = a.DH + ch * DK * DV;
  const float* Rn = a.Rs + ch * CH * DV;
  const float* DAqk = a.DAqk + ch * CH * CH;
  const float* DT = a.DT + ch * CH * CH;
  const float* DEg = a.DEg + ch * CH * DK;

  if (tid < 4) unsafe[tid] = 0;
  chunk_cumsum<DK, NTHR>(a.g + kbase, rs, sG, tid, len);
  chunk_refs<DK, NTHR>(sG, eP, brg, eGC, unsafe, tid);
  for (int e = tid; e < CH * DK / 4; e += NTHR) {
    const int r = e / (DK / 4), c4 = (e % (DK / 4)) * 4, i = r >> 4;
    const float4 kk = ld4z(a.k + kbase + r * rs + c4, r < len);
    const float4 bv = ld4z(a.b + kbase + r * rs + c4, r < len);
    const float4 qq = ld4z(a.q + kbase + r * rs + c4, r < len);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c4 + u;
      const float G = sG[r * LS + c];
      const float lf = expf(G - sG[(16 * i) * LS + c]);
      const float kv = f4at(kk, u);
      sLe[r * LS + c] = f4at(bv, u) * kv * lf;
      sLq[r * LS + c] = f4at(qq, u) * lf;
      sRk[r * LS + c] = kv * expf(sG[(16 * i + 15) * LS + c] - G);
    }
  }
  // state part of d gamma_C: rowsum(dS_C * S0) per key channel
  for (int e = tid; e < DK * NSPLIT; e += NTHR) {
    const int c = e / NSPLIT, part = e % NSPLIT;
    float acc = 0.f;
    for (int v = part * (DV / NSPLIT); v < (part + 1) * (DV / NSPLIT); ++v)
      acc += DHn[c * DV + v] * Hn[c * DV + v];
    dgp[c * NSPLIT + part] = acc;
  }
  __syncthreads();

  float keep[IPW][4];
#pragma unroll
  for (int q = 0; q < IPW; ++q) {
    const int it = wave + q * NW;
    const int i = it / NCB, cb = it % NCB;
    const int c = 16 * cb + lr;
    f4 P1 = {0.f, 0.f, 0.f, 0.f}, P2 = P1, P3 = P1, dQs = P1, dKt = P1;
    const bool diag_direct = unsafe[i] != 0;
    // P1 / P2: sum_{s<=r} M[r][s] k_s exp(G_r - G_s), without the left factor
    for (int j = 0; j <= i; ++j) {
      if (j == i && diag_direct) break;
      const float d = brg[pair_index(i, j) * DK + c];
      const float4 mt = ld4(DT + (16 * i + lr) * CH + 16 * j + 4 * lg);
      const float4 mq = ld4(DAqk + (16 * i + lr) * CH + 16 * j + 4 * lg);
      const int s0 = 16 * j + 4 * lg;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float bv = sRk[(s0 + u) * LS + c] * d;
        P1 = mfma4(f4at(mt, u), bv, P1);
        P2 = mfma4(f4at(mq, u), bv, P2);
      }
    }
    // P3: sum_{r>=s} (dT[r][s] (b k)_r + dAqk[r][s] q_r) exp(G_r - G_s), without the right factor
    for (int i2 = i; i2 < 4; ++i2) {
      if (i2 == i && diag_direct) continue;
      const float d = brg[pair_index(i2, i) * DK + c];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = 16 * i2 + 4 * lg + u;
        P3 = mfma4(DT[r * CH + 16 * i + lr], sLe[r * LS + c] * d, P3);
        P3 = mfma4(DAqk[r * CH + 16 * i + lr], sLq[r * LS + c] * d, P3);
      }
    }
    // dQs = dO S0^T and dKt = R dS_C^T
    {
      const TIn* pd = a.dout + vbase + (16 * i + lr) * rsv + 4 * lg;
      const bool pdin = 16 * i + lr < len;
      const float* pr = Rn + (16 * i + lr) * DV + 4 * lg;
      const float* ph = Hn + (16 * cb + lr) * DV + 4 * lg;
      const float* pdh = DHn + (16 * cb + lr) * DV + 4 * lg;
      for (int kk = 0; kk < DV; kk += 16) {
        const float4 x = ld4z(pd + kk, pdin), y = ld4(ph + kk);
        const float4 rr = ld4(pr + kk), z = ld4(pdh + kk);
        dQs = mfma4(x.x, y.x, dQs);
        dQs = mfma4(x.y, y.y, dQs);
        dQs = mfma4(x.z, y.z, dQs);
        dQs = mfma4(x.w, y.w, dQs);
        dKt = mfma4(rr.x, z.x, dKt);
        dKt = mfma4(rr.y, z.y, dKt);
        dKt = mfma4(rr.z, z.z, dKt);
        dKt = mfma4(rr.w, z.w, dKt);
      }
    }
    float tailpart = 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 16 * i + 4 * lg + u;
      const float G = sG[r * LS + c];
      const float lf = expf(G - sG[(16 * i) * LS + c]);
      const float rf = expf(sG[(16 * i + 15) * LS + c] - G);
      const float gam = expf(G);
      const float tail = expf(sG[(CH - 1) * LS + c] - G);
      const size_t off = kbase + r * rs + c, offo = kobase + r * rso + c;
      const bool rin = r < len;
      const float kv = to_fz(a.k + off, rin), bv = to_fz(a.b + off, rin), qv = to_fz(a.q + off, rin);
      float dEg = DEg[r * DK + c] + lf * P1[u];
      float dq = a.scale * gam * dQs[u] + lf * P2[u];
      float dKg = rf * P3[u] + tail * dKt[u];
      if (diag_direct) {
        for (int s = 16 * i; s < 16 * i + 16; ++s) {
          const size_t so = kbase + s * rs + c;
          const float Gs = sG[s * LS + c];
          if (s <= r) {
            const float e = expf(G - Gs);   // r >= s: <= 1
            const float ks = to_fz(a.k + so, s < len);
            if (s < r) dEg += DT[r * CH + s] * ks * e;
            dq += DAqk[r * CH + s] * ks * e;
          }
          if (s >= r) {
            const float e = expf(Gs - G);   // s >= r: <= 1
            if (s > r) dKg += DT[s * CH + r] * to_fz(a.b + so, s < len) * to_fz(a.k + so, s < len) * e;
            dKg += DAqk[s * CH + r] * to_fz(a.q + so, s < len) * e;
          }
        }
      }
      if (rin) {
        put(a.db + offo, dEg * kv);
        put(a.dk + offo, dEg * bv + dKg);
        put(a.dq + offo, dq);
      }
      keep[q][u] = dq * qv - dKg * kv + dEg * bv * kv;
      tailpart += dKt[u] * kv * tail;
    }
    colp[(i * 4 + lg) * DK + c] = tailpart;
  }
  __syncthreads();  // every read of sLq / sRk / sLe is done

#pragma unroll
  for (int q = 0; q < IPW; ++q) {
    const int it = wave + q * NW;
    const int i = it / NCB, cb = it % NCB;
#pragma unroll
    for (int u = 0; u < 4; ++u) sdG[(16 * i + 4 * lg + u) * LS + 16 * cb + lr] = keep[q][u];
  }
  __syncthreads();
  // d gamma_C * gamma_C joins the last row of dG
  for (int c = tid; c < DK; c += NTHR) {
    float st = 0.f;
    for (int p = 0; p < NSPLIT; ++p) st += dgp[c * NSPLIT + p];
    float tl = 0.f;
    for (int p = 0; p < 16; ++p) tl += colp[p * DK + c];
    sdG[(CH - 1) * LS + c] += eGC[c] * st + tl;
  }
  __syncthreads();
  // dlog_alpha_i = sum_{r >= i} dG_r (eq. eq_app_dg_reverse_cumsum), segmented scan
  {
    constexpr int NSEG = NTHR / DK;
    constexpr int RPS = CH / NSEG;
    const int c = tid % DK, seg = tid / DK;
    float run = 0.f;
    for (int r = (seg + 1) * RPS - 1; r >= seg * RPS; --r) {
      run += sdG[r * LS + c];
      sdG[r * LS + c] = run;
    }
    __syncthreads();
    float off = 0.f;
    for (int s = seg + 1; s < NSEG; ++s) off += sdG[(s * RPS) * LS + c];
    __syncthreads();
    for (int r = seg * RPS; r < (seg + 1) * RPS; ++r)
      if (r < len) a.dg[kobase + r * rso + c] = sdG[r * LS + c] + off;
  }
}

// ---------------------------------------------------------------------------
template <int DK, int DV, typename TIn>
hipError_t launch_bwd_state(const BwdStateArgs<TIn>& a, int B, hipStream_t st) {
  constexpr int DVS = 32;
  dim3 grid(DV / DVS, a.H, B);
  hipLaunchKernelGGL((bwd_state_kernel<DK, DV, DVS, TIn>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int DK, int DV, typename TIn>
hipError_t launch_bwd_wy(const BwdChunkArgs<TIn>& a, int B, hipStream_t st) {
  constexpr size_t lds = sizeof(float) * (3 * CH * (DK + 4) + 2 * CH * LD64 + 15 * DK) + 4 * sizeof(int);
  hipError_t e = hipFuncSetAttribute((const void*)bwd_wy_kernel<DK, DV, TIn>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(a.vl.ct0 ? a.vl.ncmax : a.NT, a.H, a.vl.ct0 ? 1 : B);
  hipLaunchKernelGGL((bwd_wy_kernel<DK, DV, TIn>), grid, dim3(512), lds, st, a);
  return hipGetLastError();
}

template <int DK, int DV, typename TIn>
hipError_t launch_bwd_intra(const BwdChunkArgs<TIn>& a, int B, hipStream_t st) {
  constexpr int NSPLIT = 512 / DK;
  constexpr size_t lds = sizeof(float) * (4 * CH * (DK + 4) + 15 * DK + 16 * DK + DK * NSPLIT) + 4 * sizeof(int);
  hipError_t e = hipFuncSetAttribute((const void*)bwd_intra_kernel<DK, DV, TIn>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(a.vl.ct0 ? a.vl.ncmax : a.NT, a.H, a.vl.ct0 ? 1 : B);
  hipLaunchKernelGGL((bwd_intra_kernel<DK, DV, TIn>), grid, dim3(512), lds, st, a);
  return hipGetLastError();
}

#define GDR2_INST_BWD(DK, DV, TIN)                                                                \
  template hipError_t launch_bwd_state<DK, DV, TIN>(const BwdStateArgs<TIN>&, int, hipStream_t); \
  template hipError_t launch_bwd_wy<DK, DV, TIN>(const BwdChunkArgs<TIN>&, int, hipStream_t);    \
  template hipError_t launch_bwd_intra<DK, DV, TIN>(const BwdChunkArgs<TIN>&, int, hipStream_t);

GDR2_INST_BWD(64, 64, float)
GDR2_INST_BWD(64, 128, float)
GDR2_INST_BWD(128, 64, float)
GDR2_INST_BWD(128, 128, float)
GDR2_INST_BWD(64, 64, bf16_t)
GDR2_INST_BWD(64, 128, bf16_t)
GDR2_INST_BWD(128, 64, bf16_t)
GDR2_INST_BWD(128, 128, bf16_t)

}  // namespace gdr2

// Forward kernels of the chunkwise WY GDR-2 operator (gfx950).
//
//   fwd_intra  one workgroup per (chunk, head, batch): the decay scan, the
//              gate-absorbed tiles, the Gram T and scores A_qk on MFMA, the
//              fp32 WY solve and the auxiliaries Y = A Ebar, U = A (W*V)
//              (Sec. 3.3; App. A; App. C.2: the intra-chunk products, the WY
//              solve and the construction of the auxiliaries).
//   fwd_state  one workgroup per (value slice, head, batch): the sequential
//              inter-chunk recurrence (eq. eq_gdn2_chunk_state) with the fp32
//              state slice resident in LDS, fused with the chunk output
//              (eq. eq_gdn2_chunk_output).  Columns of S evolve independently,
//              so the value axis is split across workgroups.

#include "gdr2_kernels.hpp"

namespace gdr2 {

// ---------------------------------------------------------------------------
// fwd_intra.  Workspace written per chunk-head `ch`:
//   Y[ch]   (64 x DK)  Y = A Ebar,   Ebar = gamma*(b*k)
//   U[ch]   (64 x DV)  U = A Z,      Z = w*v
//   Kt[ch]  (64 x DK)  Ktail rows (gamma_C / gamma_r) * k_r
//   Qg[ch]  (64 x DK)  gamma_r * q_r
//   Aqk[ch] (64 x 64)  causal scores, zero above the diagonal
//   GC[ch]  (DK)       gamma_C
template <int DK, int DV, typename TIn>
__global__ __launch_bounds__(512) void fwd_intra_kernel(IntraArgs<TIn> a) {
  constexpr int NTHR = 512;
  constexpr int LS = DK + 4;
  ChunkPos cp;
  if (!chunk_pos(a.vl, blockIdx.x, blockIdx.y, blockIdx.z, a.T, a.H, a.NT, cp)) return;
  const int h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = a.H;
  const size_t rs = (size_t)(H / a.G) * DK, rsv = (size_t)H * DV;  // key side on the H / G key heads
  const size_t row0 = cp.row0;
  const int len = cp.len;  // rows in use: the rest read as zero and are not written
  const size_t kbase = row0 * rs + (size_t)(h / a.G) * DK;
  const size_t vbase = row0 * rsv + (size_t)h * DV;
  const size_t ch = cp.ch;

  extern __shared__ float smem[];
  float* sR0 = smem;                      // G (64 x LS), later T (64 x LD64)
  float* sLe = sR0 + CH * LS;             // b*k*exp(G_r - G_p)
  float* sLq = sLe + CH * LS;             // q*exp(G_r - G_p); later Z and solve scratch
  float* sRk = sLq + CH * LS;             // k*exp(G_e - G_s)
  float* sA = sRk + CH * LS;              // A (64 x LD64)
  float* eP = sA + CH * LD64;             // 4 x DK
  float* brg = eP + 4 * DK;               // 10 x DK
  float* eGC = brg + 10 * DK;             // DK
  int* unsafe = reinterpret_cast<int*>(eGC + DK);
  float* sG = sR0;
  float* sT = sR0;

  if (tid < 4) unsafe[tid] = 0;
  chunk_cumsum<DK, NTHR>(a.g + kbase, rs, sG, tid, len);
  chunk_refs<DK, NTHR>(sG, eP, brg, eGC, unsafe, tid);

  // gate-absorbed tiles; Qg and Ktail go straight to the workspace
  float* Qg = a.Qg + ch * CH * DK;
  float* Kt = a.Kt + ch * CH * DK;
  for (int e = tid; e < CH * DK / 4; e += NTHR) {
    const int r = e / (DK / 4), c4 = (e % (DK / 4)) * 4, i = r >> 4;
    const float4 kk = ld4z(a.k + kbase + r * rs + c4, r < len);
    const float4 bv = ld4z(a.b + kbase + r * rs + c4, r < len);
    const float4 qq = ld4z(a.q + kbase + r * rs + c4, r < len);
    float4 qg, kt;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c4 + u;
      const float G = sG[r * LS + c];
      const float lf = expf(G - sG[(16 * i) * LS + c]);
      const float rf = expf(sG[(16 * i + 15) * LS + c] - G);
      const float kv = f4at(kk, u), qv = f4at(qq, u);
      sLe[r * LS + c] = f4at(bv, u) * kv * lf;
      sLq[r * LS + c] = qv * lf;
      sRk[r * LS + c] = kv * rf;
      const float gq = qv * expf(G), gk = kv * expf(sG[(CH - 1) * LS + c] - G);
      if (u == 0) { qg.x = gq; kt.x = gk; }
      if (u == 1) { qg.y = gq; kt.y = gk; }
      if (u == 2) { qg.z = gq; kt.z = gk; }
      if (u == 3) { qg.w = gq; kt.w = gk; }
    }
    *reinterpret_cast<float4*>(Qg + r * DK + c4) = qg;
    *reinterpret_cast<float4*>(Kt + r * DK + c4) = kt;
  }
  for (int c = tid; c < DK; c += NTHR) a.GC[ch * DK + c] = eGC[c];
  __syncthreads();  // sG dead from here on; region reused for T

  // T (strict lower) and A_qk (lower incl. diagonal): 10 + 10 tiles of 16x16
  float* Aqk = a.Aqk + ch * CH * CH;
  for (int it = wave; it < 20; it += NTHR / 64) {
    const bool isT = it < 10;
    int i, j;
    pair_of(isT ? it : it - 10, i, j);
    f4 acc;
    if (i == j && unsafe[i]) {
      acc = isT ? diag_tile_direct<DK, TIn>(a.b + kbase, a.k + kbase, a.k + kbase, a.g + kbase, rs, i, lane, true, len)
                : diag_tile_direct<DK, TIn>(a.q + kbase, nullptr, a.k + kbase, a.g + kbase, rs, i, lane, false, len);
    } else {
      acc = gram_tile<DK>(isT ? sLe : sLq, sRk, brg + pair_index(i, j) * DK, i, j, lane);
    }
    const int ccol = 16 * j + (lane & 15);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 16 * i + 4 * (lane >> 4) + u;
      if (isT) {
        sT[r * LD64 + ccol] = (r > ccol) ? acc[u] : 0.f;
      } else {
        Aqk[r * CH + ccol] = (r >= ccol) ? acc[u] : 0.f;
      }
    }
  }
  // zero the strictly-upper score tiles
  for (int e = tid; e < CH * CH; e += NTHR) {
    const int r = e / CH, s = e % CH;
    if ((s >> 4) > (r >> 4)) Aqk[r * CH + s] = 0.f;
  }
  __syncthreads();

  wy_solve<NTHR>(sT, sA, sLq, tid);  // sLq is free: used as solve scratch

  // Z = w * v into the sLq region (row stride DV + 4)
  float* sZ = sLq;
  constexpr int LZ = DV + 4;
  for (int e = tid; e < CH * DV / 4; e += NTHR) {
    const int r = e / (DV / 4), c4 = (e % (DV / 4)) * 4;
    const float4 wv = ld4z(a.w + vbase + r * rsv + c4, r < len);
    const float4 vv = ld4z(a.v + vbase + r * rsv + c4, r < len);
    float* d = sZ + r * LZ + c4;
    d[0] = wv.x * vv.x; d[1] = wv.y * vv.y; d[2] = wv.z * vv.z; d[3] = wv.w * vv.w;
  }
  __syncthreads();

  // Y = A Ebar (Ebar = Le * eP[block]) and U = A Z, lower-triangular A
  float* Yo = a.Y + ch * CH * DK;
  float* Uo = a.U + ch * CH * DV;
  constexpr int NCB = DK / 16 + DV / 16;
  for (int it = wave; it < NCB; it += NTHR / 64) {
    const bool isY = it < DK / 16;
    const int cb = isY ? it : it - DK / 16;
    const int col = 16 * cb + (lane & 15);
    for (int i = 0; i < 4; ++i) {
      f4 acc = {0.f, 0.f, 0.f, 0.f};
      const float* pa = sA + (16 * i + (lane & 15)) * LD64 + 4 * (lane >> 4);
      for (int kb = 0; kb <= i; ++kb) {
        const float4 av = ld4(pa + 16 * kb);
        const int s0 = 16 * kb + 4 * (lane >> 4);
        float bv[4];
        if (isY) {
          const float ep = eP[kb * DK + col];
#pragma unroll
          for (int u = 0; u < 4; ++u) bv[u] = sLe[(s0 + u) * LS + col] * ep;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) bv[u] = sZ[(s0 + u) * LZ + col];
        }
        acc = mfma4(av.x, bv[0], acc);
        acc = mfma4(av.y, bv[1], acc);
        acc = mfma4(av.z, bv[2], acc);
        acc = mfma4(av.w, bv[3], acc);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = 16 * i + 4 * (lane >> 4) + u;
        if (isY)
          Yo[r * DK + col] = acc[u];
        else
          Uo[r * DV + col] = acc[u];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fwd_state: S (DK x DVS slice, fp32, LDS) carried across chunks.  Per chunk:
//   R   = U - Y S                         (eq. eq_app_residual_matrix)
//   O   = scale * (Qg S + Aqk R)          (eq. eq_app_chunk_output)  [WITH_O]
//   S  <- Diag(gamma_C) S + Ktail^T R     (eq. eq_app_chunk_state)
// With STORE_H the chunk-start states h_n and R are kept for the backward.
template <int DK, int DV, int DVS, typename TIn, bool WITH_O, bool STORE_H>
__global__ __launch_bounds__(256) void fwd_state_kernel(StateArgs<TIn> a) {
  constexpr int NTHR = 256, NW = 4;
  constexpr int LSS = DVS + 4;
  constexpr int NVB = DVS / 16;
  const int vs = blockIdx.x, h = blockIdx.y, bb = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = a.T, H = a.H, NT = a.NT;
  const int v0 = vs * DVS;
  const size_t seq = (size_t)scan_pair(a.vl, bb * H + h, H);  // (sequence, head) pair
  const ScanRange rng = scan_range(a.vl, (int)seq, H, NT);

  __shared__ float sS[DK * LSS];
  __shared__ float sR[CH * LSS];

  for (int e = tid; e < DK * DVS; e += NTHR) {
    const int c = e / DVS, v = e % DVS;
    sS[c * LSS + v] = a.S0 ? a.S0[(seq * DK + c) * DV + v0 + v] : 0.f;
  }
  __syncthreads();

  const int lr = lane & 15, lg = lane >> 4;
  for (int n = rng.c0; n < rng.c1; ++n) {
    const size_t ch = rng.chs + n;
    const float* Y = a.Y + ch * CH * DK;
    const float* U = a.U + ch * CH * DV;
    const float* Kt = a.Kt + ch * CH * DK;
    const float* GC = a.GC + ch * DK;

    if (STORE_H) {
      float* Hn = a.Hs + ch * DK * DV;
      for (int e = tid; e < DK * DVS; e += NTHR) {
        const int c = e / DVS, v = e % DVS;
        Hn[c * DV + v0 + v] = sS[c * LSS + v];
      }
    }
    // R = U - Y S : wave -> row block, all value tiles of the slice
    {
      const int i = wave;
      f4 acc[NVB];
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          acc[vb][u] = U[(16 * i + 4 * lg + u) * DV + v0 + 16 * vb + lr];
      const float* py = Y + (16 * i + lr) * DK + 4 * lg;
      for (int kk = 0; kk < DK; kk += 16) {
        const float4 y = ld4(py + kk);
        const int c0 = kk + 4 * lg;
#pragma unroll
        for (int vb = 0; vb < NVB; ++vb) {
          acc[vb] = mfma4(-y.x, sS[(c0 + 0) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(-y.y, sS[(c0 + 1) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(-y.z, sS[(c0 + 2) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(-y.w, sS[(c0 + 3) * LSS + 16 * vb + lr], acc[vb]);
        }
      }
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = 16 * i + 4 * lg + u;
          sR[r * LSS + 16 * vb + lr] = acc[vb][u];
          if (STORE_H) a.Rs[ch * CH * DV + r * DV + v0 + 16 * vb + lr] = acc[vb][u];
        }
    }
    __syncthreads();

    if (WITH_O) {
      const float* Qg = a.Qg + ch * CH * DK;
      const float* Aqk = a.Aqk + ch * CH * CH;
      const int i = wave;
      f4 acc[NVB];
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb) acc[vb] = f4{0.f, 0.f, 0.f, 0.f};
      const float* pq = Qg + (16 * i + lr) * DK + 4 * lg;
      for (int kk = 0; kk < DK; kk += 16) {
        const float4 qv = ld4(pq + kk);
        const int c0 = kk + 4 * lg;
#pragma unroll
        for (int vb = 0; vb < NVB; ++vb) {
          acc[vb] = mfma4(qv.x, sS[(c0 + 0) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(qv.y, sS[(c0 + 1) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(qv.z, sS[(c0 + 2) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(qv.w, sS[(c0 + 3) * LSS + 16 * vb + lr], acc[vb]);
        }
      }
      const float* pa = Aqk + (16 * i + lr) * CH + 4 * lg;
      for (int kb = 0; kb <= i; ++kb) {
        const float4 av = ld4(pa + 16 * kb);
        const int s0 = 16 * kb + 4 * lg;
#pragma unroll
        for (int vb = 0; vb < NVB; ++vb) {
          acc[vb] = mfma4(av.x, sR[(s0 + 0) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(av.y, sR[(s0 + 1) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(av.z, sR[(s0 + 2) * LSS + 16 * vb + lr], acc[vb]);
          acc[vb] = mfma4(av.w, sR[(s0 + 3) * LSS + 16 * vb + lr], acc[vb]);
        }
      }
      size_t orow0;
      int olen;
      scan_rows(a.vl, (int)seq, H, T, n, orow0, olen);
#pragma unroll
      for (int vb = 0; vb < NVB; ++vb)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = 16 * i + 4 * lg + u;
          if (r < olen) put(a.o + ((orow0 + r) * H + h) * DV + v0 + 16 * vb + lr, a.scale * acc[vb][u]);
        }
    }

    // S <- Diag(gamma_C) S + Ktail^T R : tiles over (key block, value block)
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
          acc[u] = GC[c] * sS[c * LSS + 16 * vb + lr];
        }
        for (int kk = 0; kk < CH; kk += 4) {
          const int r = kk + lg;
          acc = mfma4(Kt[r * DK + 16 * cb + lr], sR[r * LSS + 16 * vb + lr], acc);
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
        for (int u = 0; u < 4; ++u) sS[(16 * cb + 4 * lg + u) * LSS + 16 * vb + lr] = nacc[q][u];
      }
    }
    __syncthreads();
  }
  if (a.ST) {
    for (int e = tid; e < DK * DVS; e += NTHR) {
      const int c = e / DVS, v = e % DVS;
      a.ST[(seq * DK + c) * DV + v0 + v] = sS[c * LSS + v];
    }
  }
}

// ---------------------------------------------------------------------------
template <int DK, int DV, typename TIn>
hipError_t launch_fwd_intra(const IntraArgs<TIn>& a, int B, hipStream_t st) {
  constexpr size_t lds = sizeof(float) * (4 * CH * (DK + 4) + CH * LD64 + 15 * DK) + 4 * sizeof(int);
  // Z (row stride DV+4) reuses the dead sLq + sRk regions
  static_assert(CH * (DV + 4) <= 2 * CH * (DK + 4), "Z tile fits the freed regions");
  static_assert(CH * LD64 <= CH * (DK + 4), "T tile fits the G region");
  hipError_t e = hipFuncSetAttribute((const void*)fwd_intra_kernel<DK, DV, TIn>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(a.vl.ct0 ? a.vl.ncmax : a.NT, a.H, a.vl.ct0 ? 1 : B);
  hipLaunchKernelGGL((fwd_intra_kernel<DK, DV, TIn>), grid, dim3(512), lds, st, a);
  return hipGetLastError();
}

template <int DK, int DV, typename TIn, bool WITH_O, bool STORE_H>
hipError_t launch_fwd_state(const StateArgs<TIn>& a, int B, hipStream_t st) {
  constexpr int DVS = 32;
  dim3 grid(DV / DVS, a.H, B);
  hipLaunchKernelGGL((fwd_state_kernel<DK, DV, DVS, TIn, WITH_O, STORE_H>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

#define GDR2_INST_FWD(DK, DV, TIN)                                                          \
  template hipError_t launch_fwd_intra<DK, DV, TIN>(const IntraArgs<TIN>&, int, hipStream_t); \
  template hipError_t launch_fwd_state<DK, DV, TIN, true, false>(const StateArgs<TIN>&, int,  \
                                                                 hipStream_t);               \
  template hipError_t launch_fwd_state<DK, DV, TIN, false, true>(const StateArgs<TIN>&, int,  \
                                                                 hipStream_t);               \
  template hipError_t launch_fwd_state<DK, DV, TIN, true, true>(const StateArgs<TIN>&, int,   \
                                                                hipStream_t);

GDR2_INST_FWD(64, 64, float)
GDR2_INST_FWD(64, 128, float)
GDR2_INST_FWD(128, 64, float)
GDR2_INST_FWD(128, 128, float)
GDR2_INST_FWD(64, 64, bf16_t)
GDR2_INST_FWD(64, 128, bf16_t)
GDR2_INST_FWD(128, 64, bf16_t)
GDR2_INST_FWD(128, 128, bf16_t)

}  // namespace gdr2

// Segment chaining of the sequence-parallel state scans (gfx950).
//
// The chunk recursion of the state (eq. eq_gdn2_chunk_state with R from
// eq. eq_app_residual_matrix) is affine in the state:
//     S_{n+1} = (Diag(gamma_C) - Ktail^T Y) S_n + Ktail^T U,
// so a segment of chunks maps its start state X to M X + N, where M is the
// product of the chunk transitions (obtained by scanning identity columns with
// U = 0) and N the segment's end state from a zero start.  The reverse scan of
// the gradient is affine the same way (App. B.1).  This kernel walks the
// segments of each sequence in order (forward) or backwards (reverse),
// X <- M_k X + N_k, and writes the value entering every segment; the segments
// are then re-scanned in parallel from those values.  With no input a chunk's
// reverse step, dS <- Diag(gamma_C) dS - Y^T (Ktail dS), is the transpose of
// its forward step, so the reverse chain of a square state can use the
// forward's maps as M_k^T (transpose_m).
//
// One 4-wave workgroup per (sequence, 64-wide value slice).  X lives in fp32
// MFMA accumulators and, for the product, as a split bf16 copy X^T in LDS;
// M_k X is fp32-accurate (split hi/lo, three passes).

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK, int DV>
__global__ __launch_bounds__(256) void segcombine_kernel(SegCombineArgs a) {
  constexpr int DVS = 64, NCB = DK / 16, KS = DK / 32;
  constexpr int CPW = NCB / 4;  // key blocks of X per wave
  constexpr int LX = DK + 8;    // X^T hi / lo, bf16 [DVS][LX]
  static_assert(NCB % 4 == 0 && DV % DVS == 0, "tiling");
  __shared__ __align__(16) __bf16 sXh[DVS * LX];
  __shared__ __align__(16) __bf16 sXl[DVS * LX];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  const int seq = blockIdx.x, v0 = blockIdx.y * DVS;
  const int nseg = a.nseg;

  // lane holds X[c][v] for c = 16 cb + 4 g + u (cb = CPW * wave + c'), v = v0 + 16 vb + r16
  f4 x[CPW][4];
#pragma unroll
  for (int cc = 0; cc < CPW; ++cc)
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = 16 * (CPW * wave + cc) + 4 * g + u, v = v0 + 16 * vb + r16;
        x[cc][vb][u] = a.X0 ? a.X0[((size_t)seq * DK + c) * DV + v] : 0.f;
      }

#pragma unroll 1
  for (int step = 0; step < nseg; ++step) {
    const int k = a.reverse ? nseg - 1 - step : step;
    const size_t sk = (size_t)seq * nseg + k;
    float* xs = a.Xs + sk * DK * DV;
#pragma unroll
    for (int cc = 0; cc < CPW; ++cc)
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          xs[(size_t)(16 * (CPW * wave + cc) + 4 * g + u) * DV + v0 + 16 * vb + r16] = x[cc][vb][u];
    if (step == nseg - 1) break;

    __syncthreads();  // the previous step's readers of X^T are done
#pragma unroll
    for (int cc = 0; cc < CPW; ++cc)
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) {
        const int off = (16 * vb + r16) * LX + 16 * (CPW * wave + cc) + 4 * g;
        st4split(sXh + off, sXl + off, x[cc][vb]);
      }
    __syncthreads();

    // X <- M_k X + N_k
    const float* M = a.M + sk * DK * DK;
    const float* N = a.N + sk * DK * DV;
#pragma unroll
    for (int cc = 0; cc < CPW; ++cc)
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          x[cc][vb][u] = N[(size_t)(16 * (CPW * wave + cc) + 4 * g + u) * DV + v0 + 16 * vb + r16];
#pragma unroll
    for (int p = 0; p < KS; ++p) {
      Fr xf[4];
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) {
        xf[vb].hi = ld8(sXh + (16 * vb + r16) * LX + 32 * p + 8 * g);
        xf[vb].lo = ld8(sXl + (16 * vb + r16) * LX + 32 * p + 8 * g);
      }
#pragma unroll
      for (int cc = 0; cc < CPW; ++cc) {
        float m[8];
        const int mr = 16 * (CPW * wave + cc) + r16, mc = 32 * p + 8 * g;
        if (a.transpose_m) {
#pragma unroll
          for (int e = 0; e < 8; ++e) m[e] = M[(size_t)(mc + e) * DK + mr];
        } else {
          ldf8(M + (size_t)mr * DK + mc, m);
        }
        const Fr mf = split8(m);
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) x[cc][vb] = mma3(mf, xf[vb], x[cc][vb]);
      }
    }
  }
}

template <int DK, int DV>
hipError_t launch_segcombine(const SegCombineArgs& a, hipStream_t st) {
  dim3 grid(a.nseq, DV / 64);
  hipLaunchKernelGGL((segcombine_kernel<DK, DV>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template hipError_t launch_segcombine<64, 64>(const SegCombineArgs&, hipStream_t);
template hipError_t launch_segcombine<64, 128>(const SegCombineArgs&, hipStream_t);
template hipError_t launch_segcombine<128, 64>(const SegCombineArgs&, hipStream_t);
template hipError_t launch_segcombine<128, 128>(const SegCombineArgs&, hipStream_t);

}  // namespace gdr2

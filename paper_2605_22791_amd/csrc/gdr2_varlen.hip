// Chunk table of packed variable-length calls (App. C.6): every sequence of a
// packed batch is cut into chunks of its own (C = 64 tokens, the last one
// partial), so that the state restarts at each sequence boundary.  One
// 1024-thread workgroup: a block-wide exclusive scan of the per-sequence chunk
// counts gives coff, then each thread writes the entries of its sequences, and
// a counting sort orders the sequences longest first for the scans.

#include "gdr2_kernels.hpp"

namespace gdr2 {

__global__ __launch_bounds__(1024) void varlen_table_kernel(const int* cu, int nseq, int T, int ncmax, int* coff,
                                                            int* ct0, int* clen, int* sorder) {
  constexpr int NTHR = 1024;
  constexpr int NBIN = 4096;  // chunk counts >= NBIN - 1 share the first bin
  __shared__ int sc[NTHR];
  __shared__ int carry;
  __shared__ int hist[NBIN];
  const int tid = threadIdx.x;
  if (tid == 0) carry = 0;
  __syncthreads();
  // coff[s] = number of chunks before sequence s (clamped to ncmax)
  for (int base = 0; base < nseq; base += NTHR) {
    const int s = base + tid;
    int n = 0;
    if (s < nseq) {
      const int t0 = min(max(cu[s], 0), T);
      const int t1 = min(max(cu[s + 1], t0), T);
      n = (t1 - t0 + CH - 1) / CH;
    }
    sc[tid] = n;
    __syncthreads();
    for (int o = 1; o < NTHR; o <<= 1) {
      const int y = tid >= o ? sc[tid - o] : 0;
      __syncthreads();
      sc[tid] += y;
      __syncthreads();
    }
    const int c = carry;
    if (s < nseq) coff[s] = min(c + sc[tid] - n, ncmax);
    __syncthreads();
    if (tid == NTHR - 1) carry = min(c + sc[NTHR - 1], ncmax);
    __syncthreads();
  }
  if (tid == 0) coff[nseq] = carry;
  __syncthreads();
  for (int s = tid; s < nseq; s += NTHR) {
    const int t0 = min(max(cu[s], 0), T);
    const int t1 = min(max(cu[s + 1], t0), T);
    const int c0 = coff[s], c1 = s + 1 < nseq ? coff[s + 1] : carry;
    for (int c = c0; c < c1; ++c) {
      const int t = t0 + (c - c0) * CH;
      ct0[c] = t;
      clen[c] = min(CH, t1 - t);
    }
  }
  // scan order: counting sort by decreasing chunk count (bin NBIN-1-count);
  // the order within a bin is whatever the LDS atomics give -- it only decides
  // when a scan starts, never what it computes
  for (int i = tid; i < NBIN; i += NTHR) hist[i] = 0;
  __syncthreads();
  auto bin_of = [&](int s) {
    const int c1 = s + 1 < nseq ? coff[s + 1] : carry;
    return NBIN - 1 - min(c1 - coff[s], NBIN - 1);
  };
  for (int s = tid; s < nseq; s += NTHR) atomicAdd(&hist[bin_of(s)], 1);
  __syncthreads();
  if (tid == 0) {  // exclusive prefix over the bins
    int run = 0;
    for (int i = 0; i < NBIN; ++i) {
      const int x = hist[i];
      hist[i] = run;
      run += x;
    }
  }
  __syncthreads();
  for (int s = tid; s < nseq; s += NTHR) sorder[atomicAdd(&hist[bin_of(s)], 1)] = s;
}

hipError_t launch_varlen_table(const int* cu, int nseq, int T, int ncmax, int* coff, int* ct0, int* clen,
                               int* sorder, hipStream_t st) {
  hipLaunchKernelGGL(varlen_table_kernel, dim3(1), dim3(1024), 0, st, cu, nseq, T, ncmax, coff, ct0, clen, sorder);
  return hipGetLastError();
}

}  // namespace gdr2

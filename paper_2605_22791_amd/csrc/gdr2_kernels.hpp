// Internal launch interface between the C ABI (gdr2_api.hip) and the kernels.
#pragma once

#include "gdr2_device.hpp"

namespace gdr2 {

// Arguments of the intra-chunk forward kernel.  Inputs use the operator's
// token-major layouts; outputs are per-chunk-head workspace tiles, chunk-head
// index ch = (b * H + h) * NT + n.
template <typename TIn>
struct IntraArgs {
  const TIn* q;
  const TIn* k;
  const TIn* v;
  const float* g;
  const TIn* b;
  const TIn* w;
  float* Y;
  float* U;
  float* Kt;
  float* Qg;
  float* Aqk;
  float* GC;
  int T, H, NT;
};

// Arguments of the sequential forward state kernel.
template <typename TIn>
struct StateArgs {
  const float* Y;
  const float* U;
  const float* Kt;
  const float* Qg;
  const float* Aqk;
  const float* GC;
  const float* S0;  // nullable
  float* ST;        // nullable
  TIn* o;           // written when the output is fused in
  float* Hs;        // chunk-start states (backward recompute)
  float* Rs;        // R per chunk (backward recompute)
  int T, H, NT;
  float scale;
};

// Reverse state scan of the backward (App. B.1).
template <typename TIn>
struct BwdStateArgs {
  const float* Qg;
  const float* Kt;
  const float* Y;
  const float* Aqk;
  const float* GC;
  const TIn* dout;
  const float* dST;  // nullable
  float* dS0;        // nullable
  float* DH;         // gradient of each chunk's end state
  float* DR;         // dR per chunk
  int T, H, NT;
  float scale;
};

// Chunk-parallel backward kernels (App. B.2 - B.5).
template <typename TIn>
struct BwdChunkArgs {
  const TIn* q;
  const TIn* k;
  const TIn* v;
  const float* g;
  const TIn* b;
  const TIn* w;
  const TIn* dout;
  const float* Hs;
  const float* DH;
  const float* Rs;
  const float* DR;
  float* DAqk;
  float* DT;
  float* DEg;
  TIn* dq;
  TIn* dk;
  TIn* dv;
  TIn* db;
  TIn* dw;
  float* dg;
  int T, H, NT;
  float scale;
};

// One recurrent (decode) call over T tokens, state updated in place.
template <typename TIn>
struct RecurArgs {
  const TIn* q;
  const TIn* k;
  const TIn* v;
  const float* g;
  const TIn* b;
  const TIn* w;
  float* S;
  TIn* o;
  int T, H;
  float scale;
};

// Fused chunkwise scan of the bf16 path: intra-chunk WY products and the
// inter-chunk state recurrence in one kernel, sequential over chunks.
struct ScanFwdArgs {
  const bf16_t* q;
  const bf16_t* k;
  const bf16_t* v;
  const float* g;
  const bf16_t* b;
  const bf16_t* w;
  const float* S0;  // nullable
  float* ST;        // nullable
  bf16_t* o;        // written when the output is fused in
  float* Hs;        // chunk-start states (backward recompute)
  float* Rs;        // R per chunk (backward recompute)
  int B, T, H, NT;
  float scale;
};

template <int DK, int DV, bool WITH_O, bool STORE_H>
hipError_t launch_fwd_scan(const ScanFwdArgs& a, hipStream_t st);

template <int DK, int DV, typename TIn>
hipError_t launch_fwd_intra(const IntraArgs<TIn>& a, int B, hipStream_t st);
template <int DK, int DV, typename TIn, bool WITH_O, bool STORE_H>
hipError_t launch_fwd_state(const StateArgs<TIn>& a, int B, hipStream_t st);
template <int DK, int DV, typename TIn>
hipError_t launch_bwd_state(const BwdStateArgs<TIn>& a, int B, hipStream_t st);
template <int DK, int DV, typename TIn>
hipError_t launch_bwd_wy(const BwdChunkArgs<TIn>& a, int B, hipStream_t st);
template <int DK, int DV, typename TIn>
hipError_t launch_bwd_intra(const BwdChunkArgs<TIn>& a, int B, hipStream_t st);
template <int DK, int DV, typename TIn>
hipError_t launch_recurrent(const RecurArgs<TIn>& a, int B, hipStream_t st);

}  // namespace gdr2

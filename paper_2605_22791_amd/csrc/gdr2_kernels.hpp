// Internal launch interface between the C ABI (gdr2_api.hip) and the kernels.
#pragma once

#include "gdr2_device.hpp"

namespace gdr2 {

// Token placement of the chunks.  Fixed-length calls: sequence bb holds T
// tokens in NT = ceil(T / C) chunks (the last one partial when C does not
// divide T) and chunk-head ch = (bb * H + h) * NT + n.  Packed variable-length
// calls (App. C.6): B = 1, sequence s holds tokens cu[s] .. cu[s+1) and its
// chunks are entries coff[s] .. coff[s+1) of a table built on the device from
// cu_seqlens (first token ct0, rows clen <= C); ch = h * ncmax + c.  Rows of a
// partial chunk past its length read as zero (log-decay 0) and are never
// written: they add nothing to the chunk's products, its decay or the state.
struct Varlen {
  const int* cu = nullptr;    // cu_seqlens (nseq + 1); null: fixed-length call
  const int* coff = nullptr;  // first chunk of every sequence; coff[nseq] = chunks in use
  const int* ct0 = nullptr;   // first token of every chunk
  const int* clen = nullptr;  // rows of every chunk (1 .. C)
  const int* sorder = nullptr;  // sequences by decreasing chunk count: the order the scans take them in
  int nseq = 0, ncmax = 0;    // sequences; chunk slots (grid and workspace extent)
};

// Entry i of a chunk table.  The tables are written before any kernel that
// reads them starts and never while it runs, so they are read through the
// constant address space: with a uniform index that is a scalar load, which
// the kernels' waits for their vector loads (the next chunk's operands, counted
// in issue order) do not have to wait behind.
__device__ __forceinline__ int ld_table(const int* p, int i) {
  return ((const __attribute__((address_space(4))) int*)p)[i];
}

// Scanned pair (sequence, head) of a scan workgroup's index q: for packed
// calls the sequences are taken longest first, so that the longest scans start
// with the grid and the short ones fill in behind them.
__device__ __forceinline__ int scan_pair(const Varlen& vl, int q, int H) {
  return vl.sorder != nullptr ? ld_table(vl.sorder, q / H) * H + q % H : q;
}

struct ChunkPos {
  size_t row0;  // token row of the chunk's first row (row = b * T + t)
  int len;      // rows in use
  size_t ch;    // chunk-head index
};

// Chunk x of a chunk-parallel grid (x < NT resp. ncmax, y = h, z = bb);
// false for the unused tail of a packed grid (uniform per workgroup).
__device__ __forceinline__ bool chunk_pos(const Varlen& vl, int x, int h, int bb, int T, int H, int NT,
                                          ChunkPos& p) {
  if (vl.ct0 != nullptr) {
    if (x >= ld_table(vl.coff, vl.nseq)) return false;
    p.row0 = (size_t)ld_table(vl.ct0, x);
    p.len = ld_table(vl.clen, x);
    p.ch = (size_t)h * vl.ncmax + x;
  } else {
    p.row0 = (size_t)bb * T + (size_t)x * CH;
    p.len = min(CH, T - x * CH);
    p.ch = ((size_t)bb * H + h) * NT + x;
  }
  return true;
}

// Chunk index of chunk x of value head hv: the per-value-head workspace tiles
// (U, the states, R, dR) of grouped problems whose key-side tiles are indexed
// by the key head (chunk_pos with the key heads).
__device__ __forceinline__ size_t value_ch(const Varlen& vl, int x, int hv, int bb, int H, int NT) {
  return vl.ct0 != nullptr ? (size_t)hv * vl.ncmax + x : ((size_t)bb * H + hv) * NT + x;
}
// Key-head chunk of value-head chunk ch = value_ch(x, hv, ...) (G value heads per key head).
__device__ __forceinline__ size_t key_ch(const Varlen& vl, size_t ch, int H, int G, int NT) {
  if (G == 1) return ch;
  if (vl.ct0 != nullptr) {
    const size_t hv = ch / vl.ncmax;
    return (hv / G) * vl.ncmax + ch % vl.ncmax;
  }
  const size_t bh = ch / NT, bb = bh / H, hv = bh % H;
  return (bb * (H / G) + hv / G) * NT + ch % NT;
}

// Chunks of the scanned pair q = s * H + h (sequence s, head h): ch = chs + c
// for c in [c0, c1).
struct ScanRange {
  size_t chs;
  int c0, c1;
};
__device__ __forceinline__ ScanRange scan_range(const Varlen& vl, int q, int H, int NT) {
  if (vl.coff != nullptr) return {(size_t)(q % H) * vl.ncmax, ld_table(vl.coff, q / H), ld_table(vl.coff, q / H + 1)};
  return {(size_t)q * NT, 0, NT};
}
// First token row and rows in use of chunk c of the scanned pair q.
__device__ __forceinline__ void scan_rows(const Varlen& vl, int q, int H, int T, int c, size_t& row0, int& len) {
  if (vl.ct0 != nullptr) {
    row0 = (size_t)ld_table(vl.ct0, c);
    len = ld_table(vl.clen, c);
  } else {
    row0 = (size_t)(q / H) * T + (size_t)c * CH;
    len = min(CH, T - c * CH);
  }
}

// Fused input stage (App. C.1, App. D.2), active when a_log is set: q and k
// are the raw projections and are L2-normalised per (token, key head) on load,
// y = x (sum x^2 + eps)^(-1/2), rounded to bf16 as the operands of the bf16
// path; g holds the decay projection f, and the log-decay is formed on load in
// fp32 as -exp(a_log[hk]) softplus(f + delta[hk][c]).  The intra-chunk kernel
// writes the inverse norms to RQ / RK ((rows, H / G) fp32, nullable) for the
// backward, which reads them there.
struct Stage {
  const float* a_log = nullptr;  // (H / G) decay magnitude per key head
  const float* delta = nullptr;  // (H / G, Dk) decay bias per key channel
  float eps = 0.f;
  float* RQ = nullptr;
  float* RK = nullptr;
};

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
  Varlen vl{};
  int G = 1;  // grouped value heads: H value heads share H / G key heads (q, k, g, b)
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
  Varlen vl{};
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
  Varlen vl{};
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
  Varlen vl{};
  int G = 1;  // grouped value heads (as in IntraArgs); G > 1: dq, dk, db, dg are per-value-head partials
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
  const int* cu = nullptr;  // packed sequences: tokens cu[s] .. cu[s+1) of sequence s (B = 1)
  int G = 1;                // grouped value heads (as in IntraArgs)
  Stage st{};               // fused input stage (RQ, RK unused)
};

// ---------------------------------------------------------------------------
// bf16 path workspace: per chunk-head ch (C = 64 tokens of one head), every
// tile is stored in MFMA fragment order so that a wave loads a 16 x 32
// operand block as one contiguous kilobyte (16 bytes per lane):
//   standard fragment block (row R, key K):  lane l holds R = l % 16,
//       K = 8 (l / 16) + e, e = 0..7;
//   permuted fragment block:                 lane l holds R = l % 16,
//       K = 4 (l / 16) + e (e < 4) and K = 16 + 4 (l / 16) + (e - 4) (e >= 4).
// Split operands store the hi block and then the lo block (2 KB per block).
//   Y    (64 x Dk)  bf16, permuted,  blocks [row block 4][key block Dk/32]
//   Qg   (64 x Dk)  bf16 hi/lo, standard, blocks [4][Dk/32]
//   Aqk  (64 x 64)  bf16 hi/lo, permuted, blocks [4][2] (causal, zeros above)
//   KtT  (Dk x 64)  Ktail^T, bf16 hi/lo, standard, blocks [Dk/16][2]
//   U    (64 x Dv)  fp32 accumulator tiles [Dv/16][4] x (64 lanes x 4):
//                   lane l holds U[16 i + 4 (l / 16) + u][16 vb + l % 16]
//   GC   (Dk)       gamma_C, fp32
// and, for the backward:
//   Hs, DH (Dk x Dv) chunk-start states and chunk-end state gradients, fp16 rows with
//                   each 32-value group in the permuted K order and one scale per
//                   16 x 32 block (store_state_f16 in gdr2_bf16.hpp)
//   Rs   (64 x Dv)  R, fp16 permuted blocks [row block 4][value block Dv/32] with one
//                   scale per block (store_frag_f16): the R operands of the chunk backward
//   Am   (64 x 64)  A = (I + T)^{-1}, fp16 16 x 16 blocks [key s block 4][row r block 4] with
//                   one scale per block (store_tile_f16; lane l: s = l % 16, r = 4 (l / 16) + e):
//                   the B operand of the 16-deep fp16 products dR^T A
//   DR   (64 x Dv)  dR, bf16 hi/lo 16 x 16 blocks [value block Dv/16][row block 4] (hi 512
//                   bytes, then lo; lane l: value l % 16, chunk row 4 (l / 16) + e): the A
//                   operand of the 16-deep products dR^T A
struct WsBf16 {
  static constexpr size_t y(int dk) { return (size_t)4 * (dk / 32) * 1024; }
  static constexpr size_t qg(int dk) { return (size_t)4 * (dk / 32) * 2048; }
  static constexpr size_t aqk() { return (size_t)8 * 2048; }
  static constexpr size_t ktt(int dk) { return (size_t)(dk / 16) * 2 * 2048; }
  static constexpr size_t u(int dv) { return (size_t)(dv / 16) * 4 * 1024; }
  static constexpr size_t gc(int dk) { return (size_t)((dk * 4 + 255) / 256) * 256; }
  // A of the backward: fp16 16 x 16 blocks (512 bytes) and one fp32 scale per block;
  // dR: split bf16 16 x 16 blocks (1 KB)
  static constexpr size_t am() { return (size_t)16 * 512; }
  static constexpr size_t amsc() { return (size_t)16 * 4; }
  static constexpr size_t dr(int dv) { return (size_t)(dv / 16) * 4 * 1024; }
  // chunk states of the backward: fp16 (Dk x Dv) and one fp32 scale per 16 x 32 block
  static constexpr size_t hs(int dk, int dv) { return (size_t)dk * dv * 2; }
  static constexpr size_t hsc(int dk, int dv) { return (size_t)(dk / 16) * (dv / 32) * 4; }
  // R of the backward: fp16 permuted fragment blocks [row block 4][value block Dv/32]
  // (1 KB each) and one fp32 scale per block
  static constexpr size_t rs(int dv) { return (size_t)4 * (dv / 32) * 1024; }
  static constexpr size_t rsc(int dv) { return (size_t)4 * (dv / 32) * 4; }
};

struct IntraBf16Args {
  const bf16_t* q;
  const bf16_t* k;
  const bf16_t* v;
  const float* g;
  const bf16_t* b;
  const bf16_t* w;
  unsigned char* Y;
  unsigned char* Qg;
  unsigned char* Aqk;
  unsigned char* KtT;
  float* U;
  float* GC;
  _Float16* Am;  // nullable: A for the backward (WsBf16::am, with Amsc)
  int B, T, H, NT;
  Varlen vl{};
  // grouped value heads: H value heads share H / G key heads (q, k, g, b); the
  // kernel runs per key-head chunk and writes Y, Q_g, A_qk, K_tail, gamma_C and A
  // once there (chunk_pos over the key heads) and U for each value head (value_ch)
  int G = 1;
  Stage st{};
  float* Amsc = nullptr;  // the inverse scales of Am's blocks
};

// Sequence-parallel scans: with nseg > 1 every sequence is cut into nseg
// segments of seg_len chunks and each workgroup scans one segment of one
// sequence alone, from a given start state.  A pass with kScanNoInput (U = 0,
// resp. dO = 0) and kScanEye (identity start columns) yields a segment's
// transition matrix; the segment-combine kernel then chains the segments.
enum ScanFlags : int { kScanNoInput = 1, kScanEye = 2 };

struct ScanArgs {
  const unsigned char* Y;
  const unsigned char* Qg;
  const unsigned char* Aqk;
  const unsigned char* KtT;
  const float* U;
  const float* GC;
  const float* S0;  // nullable
  float* ST;        // nullable
  bf16_t* o;        // written when the output is fused in
  _Float16* Hs;     // chunk-start states for the backward, fp16 (store_state_f16 layout)
  _Float16* Rs;     // R per chunk for the backward, fp16 fragment blocks (WsBf16::rs)
  int B, T, H, NT;
  float scale;
  float* Hsc = nullptr;          // their inverse scales (WsBf16::hsc per chunk-head)
  float* Rsc = nullptr;          // R's inverse scales (WsBf16::rsc per chunk-head)
  int nseg = 1, seg_len = 0;     // segments per sequence and their length in chunks (0: NT)
  const float* S0seg = nullptr;  // nullable: start state of every segment (B*H*nseg, Dk, DV)
  float* STseg = nullptr;        // nullable: end state of every segment (B*H*nseg, Dk, DV)
  int flags = 0;                 // ScanFlags
  Varlen vl{};
  int G = 1;                     // value heads per key head: Y, Q_g, A_qk, K_tail, gamma_C per key head
  float* STseg_m = nullptr;      // the map pass (Dk = DV): M of every segment (B*H*nseg, Dk, Dk)
};

struct BScanArgs {
  const unsigned char* Y;
  const unsigned char* Qg;
  const unsigned char* Aqk;
  const unsigned char* KtT;
  const float* GC;
  const bf16_t* dout;
  const float* dST;  // nullable
  float* dS0;        // nullable
  _Float16* DH;      // nullable: gradient of each chunk's end state, fp16 (store_state_f16 layout)
  __bf16* DR;        // nullable: dR per chunk, split bf16 16 x 16 blocks (WsBf16::dr)
  int B, T, H, NT;
  float scale;
  float* DHsc = nullptr;           // the inverse scales of DH
  int nseg = 1, seg_len = 0;       // as in ScanArgs; the scan runs from a segment's end to its start
  const float* dSseg_in = nullptr; // nullable: gradient at the end of every segment (B*H*nseg, Dk, DV)
  float* dSseg_out = nullptr;      // nullable: gradient at the start of every segment
  int flags = 0;                   // ScanFlags (kScanNoInput: dO = 0)
  Varlen vl{};
  int G = 1;                       // as in ScanArgs
};

// Chaining of segment maps: X <- M_k X + N_k over the segments of each sequence
// (forward: k = 0, 1, ..., Xs[0] = X0; reverse: k = nseg-1, ..., Xs[nseg-1] = X0).
// Xs[k] receives the value entering segment k.  M: (nseq*nseg, Dk, Dk),
// N, Xs: (nseq*nseg, Dk, DV), X0: (nseq, Dk, DV) or null (zero); fp32.
struct SegCombineArgs {
  const float* M;
  const float* N;
  const float* X0;
  float* Xs;
  int nseq, nseg;
  int reverse;
  int transpose_m = 0;  // use M_k^T (the reverse chain with the forward's maps, Dk = DV)
};

// Chunk-parallel backward of the bf16 path (App. B.2 - B.5).
struct BChunkBf16Args {
  const bf16_t* q;
  const bf16_t* k;
  const bf16_t* v;
  const float* g;
  const bf16_t* b;
  const bf16_t* w;
  const bf16_t* dout;
  const _Float16* Hs;       // chunk-start states, fp16 (store_state_f16 layout)
  const _Float16* DH;       // gradients of the chunk-end states, fp16
  const _Float16* Rs;       // R per chunk, fp16 fragment blocks (WsBf16::rs)
  const __bf16* DR;         // dR, split bf16 16 x 16 blocks (WsBf16::dr)
  const _Float16* Am;       // A, fp16 16 x 16 blocks (WsBf16::am)
  bf16_t* dq;
  bf16_t* dk;
  bf16_t* dv;
  bf16_t* db;
  bf16_t* dw;
  float* dg;
  int B, T, H, NT;
  float scale;
  const float* Hsc = nullptr;   // inverse scales of Hs and DH (WsBf16::hsc per chunk-head)
  const float* DHsc = nullptr;
  const float* Rsc = nullptr;   // inverse scales of Rs (WsBf16::rsc per chunk-head)
  const float* Amsc = nullptr;  // inverse scales of Am (WsBf16::amsc per key-head chunk)
  Varlen vl{};
  // grouped value heads: H value heads share H / G key heads.  With G > 1 the
  // kernel is launched once per value head of every group (gj = 0 .. G - 1, in
  // order; the grid covers the key heads) and the key-side gradients add up in
  // fp32 on the key-head axis in Aq, Ak, Ab, Ag ((rows, H / G, Dk) each): gmode
  // 1 stores the first value head's, 2 adds the next, 3 adds the last and
  // writes the outputs (gmode 0: G = 1, outputs written directly).  The sums
  // run in the order of the value heads, so the result is deterministic.
  int G = 1;
  int gj = 0, gmode = 0;
  float* Aq = nullptr;
  float* Ak = nullptr;
  float* Ab = nullptr;
  float* Ag = nullptr;
  // Pq, Pk set: dq, dk leave in fp32 there (key-head axis) instead of in the
  // output dtype (the fused stage's normalisation VJP reads them)
  float* Pq = nullptr;
  float* Pk = nullptr;
  // fused input stage: q, k raw (normalised with the stored inverse norms), g
  // holds f and dg receives df = dg * dg/df; dq and dk stay the gradients of the
  // normalised q, k (the normalisation VJP follows in its own kernel).  Per
  // workgroup (chunk slot s = z * gridDim.x + x, value head h, wave i) PD gets
  // sum_rows df over each key channel and PA sum_{rows, channels} dg * g:
  // PD ((s * H + h) * 4 + i) * Dk + c, PA (s * H + h) * 4 + i.
  Stage st{};
  float* PD = nullptr;
  float* PA = nullptr;
};

template <int DK, int DV>
hipError_t launch_intra_bf16(const IntraBf16Args& a, hipStream_t st);
template <int DK, int DV>
hipError_t launch_bscan_bf16(const BScanArgs& a, hipStream_t st);
template <int DK, int DV, bool WITH_O, bool STORE_H>
hipError_t launch_scan_bf16(const ScanArgs& a, hipStream_t st);
// both segment maps of the sequence-parallel forward scan in one launch (Dk = Dv = D):
// N into a.STseg, M into a.STseg_m
template <int D>
hipError_t launch_scan_map_bf16(const ScanArgs& a, hipStream_t st);
template <int DK, int DV>
hipError_t launch_bchunk_bf16(const BChunkBf16Args& a, hipStream_t st);
template <int DK, int DV>
hipError_t launch_segcombine(const SegCombineArgs& a, hipStream_t st);

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

// Grouped value heads: out[r, h, c] = sum_{j < G} P[r, h * G + j, c] for rows
// r < rows, key heads h < Hk, channels c < D (P fp32 on the value-head axis).
template <typename TOut>
hipError_t launch_group_reduce(const float* P, TOut* out, size_t rows, int Hk, int G, int D, hipStream_t st);

// Normalisation VJP of the fused stage (App. D.2): for rows r < rows, key
// heads hk < Hk, dx = rinv (dy - y <y, dy>), y = rinv x, with x the raw q or
// k (bf16), rinv its stored inverse norm and dy the gradient of the normalised
// tensor, the sum of the G fp32 partials P[r, hk * G + j, :] (G = 1: the fp32
// gradient itself).  Two tensors (q, k) per launch.
struct NormVjpArgs {
  const bf16_t* x[2];
  const float* rinv[2];
  const float* P[2];
  bf16_t* dx[2];
  size_t rows;
  int Hk, G;
};
template <int DK>
hipError_t launch_norm_vjp(const NormVjpArgs& a, hipStream_t st);

// The fused stage of fp32 problems as passes around the fp32 operator: rows
// r < rows of the H_k = Hk key heads, (rows, Hk, DK) fp32 tensors.
// Forward: qn, kn = normalised q, k (inverse norms to rq, rk), g from f.
// Backward: dq, dk from the gradients dqn, dkn of the normalised tensors;
// df from dg, and pa[r * Hk + h] = sum_c dg * g (the per-row partials of da).
struct StageF32Args {
  const float* q;
  const float* k;
  const float* f;
  const float* a_log;
  const float* delta;
  float eps;
  float* qn;
  float* kn;
  float* g;
  float* rq;
  float* rk;
  const float* dqn;
  const float* dkn;
  const float* dg;
  float* dq;
  float* dk;
  float* df;
  float* pa;
  size_t rows;
  int Hk;
};
template <int DK>
hipError_t launch_stage_f32(const StageF32Args& a, bool backward, hipStream_t st);

// Sums of the per-workgroup partials of the decay parameters, one pass:
// out[(z * Hk + hk) * D + c] = sum over the slots s of range z (nslots cut into
// `splits` ranges) and m < M of P[((s * Hk + hk) * M + m) * D + c].  A second
// pass with nslots = splits, M = 1, splits = 1 adds the ranges.
hipError_t launch_param_reduce_pass(const float* P, float* out, int nslots, int Hk, int M, int D, int splits,
                                    hipStream_t st);

// Builds the chunk table of a packed call (Varlen) from cu_seqlens: lengths
// are clamped into [0, T] and the chunk count to ncmax, so malformed offsets
// cannot lead to accesses outside the tensors or the workspace; and the scan
// order of the sequences (decreasing chunk count).
hipError_t launch_varlen_table(const int* cu, int nseq, int T, int ncmax, int* coff, int* ct0, int* clen,
                               int* sorder, hipStream_t st);

}  // namespace gdr2

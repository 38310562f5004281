// C ABI of the GDR-2 operator: argument validation, workspace layout and the
// launch sequence.  Every check runs before the first HIP call; on an error
// nothing is enqueued.  See include/gdr2.h for the contract.

#include "../../include/gdr2.h"

#include <cmath>
#include <type_traits>
#include <cstdlib>
#include <vector>

#include "gdr2_kernels.hpp"

using namespace gdr2;

namespace {

constexpr size_t kAlign = 256;

size_t round_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kMaxSeqs = 1 << 24;  // sequences of one packed call

// nseq > 0: a packed variable-length call of nseq sequences (B must be 1).
gdr2_status check_problem(const gdr2_problem* p, bool chunked, int nseq = 0) {
  if (p == nullptr) return GDR2_EINVAL;
  if (p->B <= 0 || p->T <= 0 || p->H <= 0 || p->Dk <= 0 || p->Dv <= 0) return GDR2_EINVAL;
  if (!std::isfinite(p->scale)) return GDR2_EINVAL;
  if (p->dtype != GDR2_BF16 && p->dtype != GDR2_FP32) return GDR2_EINVAL;
  if (nseq < 0 || (nseq > 0 && p->B != 1)) return GDR2_EINVAL;
  if (p->Hv < 0 || (p->Hv > 0 && p->Hv % p->H != 0)) return GDR2_EINVAL;
  if ((p->Dk != 64 && p->Dk != 128) || (p->Dv != 64 && p->Dv != 128)) return GDR2_EUNSUPPORTED;
  if (chunked && p->chunk != CH) return GDR2_EUNSUPPORTED;
  if (nseq > kMaxSeqs) return GDR2_EUNSUPPORTED;
  const double Hv = p->Hv > 0 ? p->Hv : p->H;
  const double rows = (double)p->B * (double)p->T * Hv;
  const int dmax = p->Dk > p->Dv ? p->Dk : p->Dv;
  if (rows * dmax >= 2147483648.0) return GDR2_EUNSUPPORTED;
  const double states = nseq > 0 ? (double)nseq : (double)p->B;
  if (states * Hv * (double)p->Dk * p->Dv >= 2147483648.0) return GDR2_EUNSUPPORTED;
  return GDR2_OK;
}

// The problem seen from the value heads: every kernel runs per value head
// (H := Hv) and reads the key-side tensors q, k, g, b at key head h / G.
gdr2_problem value_view(const gdr2_problem* p) {
  gdr2_problem v = *p;
  v.H = p->Hv > 0 ? p->Hv : p->H;
  v.Hv = 0;
  return v;
}
int group_of(const gdr2_problem* p) { return p->Hv > 0 ? p->Hv / p->H : 1; }

// Chunks per sequence of a fixed-length call (the last one partial when 64 does not divide T).
int chunks_per_seq(const gdr2_problem* p) { return (p->T + CH - 1) / CH; }
// Chunk slots of a packed call: sum_s ceil(L_s / 64) <= floor(T / 64) + nseq.
int varlen_slots(const gdr2_problem* p, int nseq) { return p->T / CH + nseq; }

// Workspace regions, chunk-head major: ch = (b*H + h)*NT + n (fixed length) or
// h*slots + c (packed; see Varlen in gdr2_kernels.hpp).  The bf16
// path uses the fragment-order regions of WsBf16 (gdr2_kernels.hpp) plus fp32
// chunk states and R for the backward; the fp32 path uses fp32 tiles.
struct Layout {
  size_t Y, U, Kt, Qg, Aqk, GC;          // fp32 forward tiles
  size_t Hs, Rs, DH, DR, DAqk, DT, DEg;  // backward extras
  size_t Hsc, DHsc, Rsc;                 // bf16 backward: scales of the fp16 chunk states and R
  size_t bY, bQ, bA, bK, bU, bG;         // bf16 forward (fragment order)
  size_t bDR, bAm, bAmsc;                // bf16 backward extras (dR split, A fp16 with scales)
  size_t sM, sN, sX;                     // segment maps and entry states (sequence-parallel scans)
  int nseg, seg_len;
  size_t vcoff, vct0, vclen, vsord;      // chunk table and scan order of a packed call (int32)
  size_t pQ, pK, pB, pG;                 // grouped value heads: fp32 key-side gradient partials
  size_t RQ, RK;                         // fused stage: inverse norms of q, k rows (rows, Hk)
  size_t PD, PA, PT;                     // fused backward: decay-parameter partials, range sums
  size_t fQ, fK, fG, fdQ, fdK, fdG;      // fused stage of fp32 problems: its outputs and their gradients
  size_t total;
};

constexpr int kParamSplits = 64;  // slot ranges of the first decay-parameter reduction pass

// Sequence-parallel scans (bf16 path).  The state scans run one workgroup per
// (sequence, 64-wide value slice); when there are too few of those to occupy
// the chip and the sequences are long, every sequence is cut into segments
// that are scanned side by side (segment maps, then a short chain over the
// segments, then the segments again from their true start states).  Segments
// are doubled while the scan grid stays within one workgroup per compute unit
// and a segment keeps at least 8 chunks.  The rule depends on the problem's
// shape alone, so a problem always runs the same schedule (and rounds the same
// way).
void scan_segments(const gdr2_problem* p, int& nseg, int& seg_len) {
  const int NT = chunks_per_seq(p);
  const long long slices = (long long)p->B * p->H * (p->Dv / 64);
  int n = 1;
  if (p->dtype == GDR2_BF16 && slices < 128 && NT >= 16) {
    while (slices * n * 2 <= 256 && n * 2 * 8 <= NT) n *= 2;
  }
  seg_len = (NT + n - 1) / n;
  nseg = (NT + seg_len - 1) / seg_len;
}

// p: the value view (value_view); G > 1 adds the backward's group partials;
// fused adds the fused stage's regions (bwd: saving forward and backward).
Layout layout(const gdr2_problem* p, bool bwd, int nseq = 0, int G = 1, bool fused = false) {
  const size_t NC = nseq > 0 ? (size_t)p->H * varlen_slots(p, nseq) : (size_t)p->B * p->H * chunks_per_seq(p);
  const size_t Dk = p->Dk, Dv = p->Dv;
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t floats) {
    const size_t at = off;
    off += round_up(floats * sizeof(float));
    return at;
  };
  if (p->dtype == GDR2_BF16) {
    auto takeb = [&](size_t bytes) {
      const size_t at = off;
      off += round_up(bytes);
      return at;
    };
    // the key-side tiles (all but U) once per key-head chunk: shared by the G value heads
    const size_t NCk = NC / G;
    L.bY = takeb(NCk * WsBf16::y(p->Dk));
    L.bQ = takeb(NCk * WsBf16::qg(p->Dk));
    L.bA = takeb(NCk * WsBf16::aqk());
    L.bK = takeb(NCk * WsBf16::ktt(p->Dk));
    L.bU = takeb(NC * WsBf16::u(p->Dv));
    L.bG = takeb(NCk * WsBf16::gc(p->Dk));
  } else {
    L.Y = take(NC * CH * Dk);
    L.U = take(NC * CH * Dv);
    L.Kt = take(NC * CH * Dk);
    L.Qg = take(NC * CH * Dk);
    L.Aqk = take(NC * CH * CH);
    L.GC = take(NC * Dk);
  }
  if (bwd && p->dtype == GDR2_BF16) {
    // fp16 chunk states with their block scales (store_state_f16), fp32 R
    auto takeb = [&](size_t bytes) {
      const size_t at = off;
      off += round_up(bytes);
      return at;
    };
    L.Hs = takeb(NC * WsBf16::hs(p->Dk, p->Dv));
    L.Hsc = takeb(NC * WsBf16::hsc(p->Dk, p->Dv));
    L.Rs = takeb(NC * WsBf16::rs(p->Dv));
    L.Rsc = takeb(NC * WsBf16::rsc(p->Dv));
    L.DH = takeb(NC * WsBf16::hs(p->Dk, p->Dv));
    L.DHsc = takeb(NC * WsBf16::hsc(p->Dk, p->Dv));
  } else if (bwd) {
    L.Hs = take(NC * Dk * Dv);
    L.Rs = take(NC * CH * Dv);
    L.DH = take(NC * Dk * Dv);
  }
  if (bwd) {
    if (p->dtype == GDR2_BF16) {
      // dR (split bf16) and A (fp16 with block scales) for the chunk-parallel backward
      L.bDR = off;
      off += round_up(NC * WsBf16::dr(p->Dv));
      L.bAm = off;
      off += round_up(NC / G * WsBf16::am());  // A per key-head chunk
      L.bAmsc = off;
      off += round_up(NC / G * WsBf16::amsc());
    } else {
      L.DR = take(NC * CH * Dv);
      L.DAqk = take(NC * CH * CH);
      L.DT = take(NC * CH * CH);
      L.DEg = take(NC * CH * Dk);
    }
  }
  if (nseq > 0) {
    // packed calls scan every sequence whole (their lengths differ)
    L.nseg = 1;
    L.seg_len = 0;
    const size_t slots = (size_t)varlen_slots(p, nseq);
    L.vcoff = take((size_t)nseq + 1);
    L.vct0 = take(slots);
    L.vclen = take(slots);
    L.vsord = take((size_t)nseq);
  } else {
    scan_segments(p, L.nseg, L.seg_len);
  }
  const bool fbf16 = fused && p->dtype == GDR2_BF16;  // stage inside the bf16 kernels
  if (bwd && (G > 1 || fbf16)) {
    // fp32 key-side gradients: bf16 problems sum a group's value heads in them
    // on the key-head axis (and the fused stage keeps dq, dk there for its VJP,
    // which rounds once); fp32 problems keep one partial per value head
    const size_t heads = p->dtype == GDR2_BF16 ? (size_t)(p->H / G) : (size_t)p->H;
    const size_t n = (size_t)p->B * p->T * heads * Dk;
    L.pQ = take(n);
    L.pK = take(n);
    if (G > 1) {
      L.pB = take(n);
      L.pG = take(n);
    }
  }
  if (fbf16 && bwd) {
    const size_t rows = (size_t)p->B * p->T, Hk = (size_t)(p->H / G);
    const size_t nslots = nseq > 0 ? (size_t)varlen_slots(p, nseq) : (size_t)p->B * chunks_per_seq(p);
    L.RQ = take(rows * Hk);
    L.RK = take(rows * Hk);
    L.PD = take(nslots * p->H * 4 * Dk);
    L.PA = take(nslots * p->H * 4);
    L.PT = take((size_t)kParamSplits * Hk * (Dk + 1));
  }
  if (L.nseg > 1) {
    const size_t nvs = (size_t)p->B * p->H * L.nseg;
    L.sM = take(nvs * Dk * Dk);
    L.sN = take(nvs * Dk * Dv);
    L.sX = take(nvs * Dk * Dv);
  }
  if (fused && p->dtype == GDR2_FP32) {
    // fp32 problems run the stage as passes of its own around the fp32 operator:
    // its outputs (and, for the backward, their gradients) follow everything the
    // operator itself uses, so the operator's layout is a prefix of this one
    const size_t n = (size_t)p->B * p->T * (size_t)(p->H / G);
    L.fQ = take(n * Dk);
    L.fK = take(n * Dk);
    L.fG = take(n * Dk);
    L.RQ = take(n);
    L.RK = take(n);
    if (bwd) {
      L.fdQ = take(n * Dk);
      L.fdK = take(n * Dk);
      L.fdG = take(n * Dk);
      L.PA = take(n);
      L.PT = take((size_t)kParamSplits * (p->H / G) * (Dk + 1));
    }
  }
  L.total = off;
  return L;
}

template <typename T>
T* at(void* ws, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Everything a run needs about the chunking: the workspace layout, chunks per
// sequence (fixed length) or chunk slots (packed), the number of scanned
// sequences and, for packed calls, the device chunk table.
struct Geo {
  Layout L;
  int NT;
  int nscan;
  Varlen vl;
  int G;  // value heads per key head
  Stage st;  // fused input stage (st.a_log null: off); RQ / RK set when the layout has them
};

// p: the value view; G: value heads per key head; stage: the fused stage or null
Geo make_geo(const gdr2_problem* p, bool bwd, int nseq, const int* cu, void* ws, int grp = 1,
             const gdr2_stage* stage = nullptr) {
  Geo G{};
  G.G = grp;
  G.L = layout(p, bwd, nseq, grp, stage != nullptr);
  if (stage != nullptr) {
    G.st.a_log = stage->a_log;
    G.st.delta = stage->delta;
    G.st.eps = stage->eps;
    if (bwd) {
      G.st.RQ = at<float>(ws, G.L.RQ);
      G.st.RK = at<float>(ws, G.L.RK);
    }
  }
  if (nseq > 0) {
    G.NT = varlen_slots(p, nseq);
    G.nscan = nseq;
    G.vl.cu = cu;
    G.vl.coff = at<int>(ws, G.L.vcoff);
    G.vl.ct0 = at<int>(ws, G.L.vct0);
    G.vl.clen = at<int>(ws, G.L.vclen);
    G.vl.sorder = at<int>(ws, G.L.vsord);
    G.vl.nseq = nseq;
    G.vl.ncmax = G.NT;
  } else {
    G.NT = chunks_per_seq(p);
    G.nscan = p->B;
  }
  return G;
}

// Builds the chunk table of a packed call in the workspace (no-op otherwise).
hipError_t build_table(const gdr2_problem* p, const Geo& G, hipStream_t st) {
  if (G.vl.cu == nullptr) return hipSuccess;
  return launch_varlen_table(G.vl.cu, G.vl.nseq, p->T, G.vl.ncmax, const_cast<int*>(G.vl.coff),
                             const_cast<int*>(G.vl.ct0), const_cast<int*>(G.vl.clen),
                             const_cast<int*>(G.vl.sorder), st);
}

bool debug_sync() {
  static const bool on = [] {
    const char* e = std::getenv("GDR2_DEBUG_SYNC");
    return e != nullptr && e[0] == '1';
  }();
  return on;
}

gdr2_status hip_status(hipError_t e, hipStream_t st) {
  if (e != hipSuccess) return GDR2_EHIP;
  if (debug_sync()) {
    if (hipStreamSynchronize(st) != hipSuccess) return GDR2_EHIP;
    if (hipGetLastError() != hipSuccess) return GDR2_EHIP;
  }
  return GDR2_OK;
}

// ---- measurement support ---------------------------------------------------
// When a thread enables it, every kernel launch that thread makes is bracketed
// by two hipEvents on the launch stream; gdr2_profile_collect() waits for them
// and returns accumulated milliseconds and launch counts per kernel.  The state
// is per calling thread and is only touched while profiling is on.
struct ProfState {
  bool on = false;
  struct Pending {
    int id;
    hipEvent_t a, b;
  };
  std::vector<Pending> pending;
  std::vector<hipEvent_t> pool;
  double ms[GDR2_NUM_KERNELS] = {};
  long long launches[GDR2_NUM_KERNELS] = {};
};
thread_local ProfState g_prof;

hipEvent_t prof_event() {
  if (!g_prof.pool.empty()) {
    hipEvent_t e = g_prof.pool.back();
    g_prof.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <class F>
hipError_t timed(int id, hipStream_t st, F&& launch) {
  if (!g_prof.on) return launch();
  hipEvent_t a = prof_event(), b = prof_event();
  if (a == nullptr || b == nullptr) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, st);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, st);
  if (e != hipSuccess) return e;
  g_prof.pending.push_back({id, a, b});
  return hipSuccess;
}

// ---- grouped value heads of fp32 problems: sum each key head's G partials into
// dq, dk, db, dlog_alpha (p: the value view, so the key heads are p->H / G)
template <typename TIn>
hipError_t group_reduce(const gdr2_problem* p, const Geo& G, const Layout& L, void* ws, void* dq, void* dk,
                        void* db, float* dg, hipStream_t st) {
  const size_t rows = (size_t)p->B * p->T;
  const int Hk = p->H / G.G;
  hipError_t e = hipSuccess;
  if (dq != nullptr)
    e = launch_group_reduce<TIn>(at<float>(ws, L.pQ), static_cast<TIn*>(dq), rows, Hk, G.G, p->Dk, st);
  if (e == hipSuccess && dk != nullptr)
    e = launch_group_reduce<TIn>(at<float>(ws, L.pK), static_cast<TIn*>(dk), rows, Hk, G.G, p->Dk, st);
  if (e == hipSuccess) e = launch_group_reduce<TIn>(at<float>(ws, L.pB), static_cast<TIn*>(db), rows, Hk, G.G, p->Dk, st);
  if (e == hipSuccess) e = launch_group_reduce<float>(at<float>(ws, L.pG), dg, rows, Hk, G.G, p->Dk, st);
  return e;
}

// ---- fused stage, backward tail: the normalisation VJP of q and k (from the
// gradients of the normalised tensors in dq, dk, or in the group partials) and
// the two-pass sums of the decay-parameter partials into ddelta and da
template <int DK>
hipError_t stage_bwd(const gdr2_problem* p, const Geo& G, void* ws, const void* q, const void* k, void* dq,
                     void* dk, float* da, float* ddelta, hipStream_t st) {
  const Layout& L = G.L;
  const int Hk = p->H / G.G;
  NormVjpArgs na{};
  na.x[0] = static_cast<const bf16_t*>(q);
  na.x[1] = static_cast<const bf16_t*>(k);
  na.rinv[0] = G.st.RQ;
  na.rinv[1] = G.st.RK;
  na.P[0] = at<float>(ws, L.pQ);  // summed over the group already (key-head axis)
  na.P[1] = at<float>(ws, L.pK);
  na.dx[0] = static_cast<bf16_t*>(dq);
  na.dx[1] = static_cast<bf16_t*>(dk);
  na.rows = (size_t)p->B * p->T;
  na.Hk = Hk;
  na.G = 1;
  hipError_t e = launch_norm_vjp<DK>(na, st);
  if (e != hipSuccess) return e;
  const int nslots = G.vl.ct0 != nullptr ? G.vl.ncmax : p->B * G.NT;
  const int splits = nslots < kParamSplits ? nslots : kParamSplits;
  float* PT = at<float>(ws, L.PT);
  float* PT1 = PT + (size_t)kParamSplits * Hk * DK;
  e = launch_param_reduce_pass(at<float>(ws, L.PD), PT, nslots, Hk, 4 * G.G, DK, splits, st);
  if (e == hipSuccess) e = launch_param_reduce_pass(PT, ddelta, splits, Hk, 1, DK, 1, st);
  if (e == hipSuccess) e = launch_param_reduce_pass(at<float>(ws, L.PA), PT1, nslots, Hk, 4 * G.G, 1, splits, st);
  if (e == hipSuccess) e = launch_param_reduce_pass(PT1, da, splits, Hk, 1, 1, 1, st);
  return e;
}

// ---- state scans of the bf16 path, sequential or sequence-parallel ---------
// Forward: segment maps N (zero start) and M (identity start, no input), the
// chain X_k entering every segment, then `last` scans every segment from X_k
// (it writes the output and, if asked, the chunk states, R and S_T).
template <int DK, int DV, class Last>
hipError_t scan_fwd_bf16(const ScanArgs& sa, const Layout& L, void* ws, Last&& last, hipStream_t st) {
  if (L.nseg == 1) return last(sa);
  ScanArgs pn = sa;
  pn.S0 = nullptr;
  pn.ST = nullptr;
  pn.o = nullptr;
  pn.Hs = nullptr;
  pn.Rs = nullptr;
  pn.nseg = L.nseg;
  pn.seg_len = L.seg_len;
  pn.STseg = at<float>(ws, L.sN);
  hipError_t e;
  if constexpr (DK == DV) {
    // N and M in one launch: each map's full width in one workgroup
    pn.STseg_m = at<float>(ws, L.sM);
    e = launch_scan_map_bf16<DK>(pn, st);
  } else {
    e = launch_scan_bf16<DK, DV, false, false>(pn, st);
    if (e != hipSuccess) return e;
    ScanArgs pm = pn;
    pm.U = nullptr;
    pm.flags = kScanNoInput | kScanEye;
    pm.STseg = at<float>(ws, L.sM);
    e = launch_scan_bf16<DK, DK, false, false>(pm, st);
  }
  if (e != hipSuccess) return e;
  const SegCombineArgs ca{at<float>(ws, L.sM), at<float>(ws, L.sN), sa.S0, at<float>(ws, L.sX),
                          sa.B * sa.H, L.nseg, 0};
  e = launch_segcombine<DK, DV>(ca, st);
  if (e != hipSuccess) return e;
  ScanArgs p3 = sa;
  p3.nseg = L.nseg;
  p3.seg_len = L.seg_len;
  p3.S0seg = at<float>(ws, L.sX);
  return last(p3);
}

// Reverse: the same steps from the segment ends, then every segment again
// from the gradient at its end (writing dH, dR and dS0).  For a square state
// the reverse segment maps are the transposes of the forward ones, which the
// forward phase of this backward (or the saving forward) left in sM: the map
// pass of the reverse scan is then skipped.
template <int DK, int DV>
hipError_t scan_bwd_bf16(const BScanArgs& ba, const Layout& L, void* ws, hipStream_t st) {
  if (L.nseg == 1) return launch_bscan_bf16<DK, DV>(ba, st);
  BScanArgs pn = ba;
  pn.dST = nullptr;
  pn.dS0 = nullptr;
  pn.DH = nullptr;
  pn.DR = nullptr;
  pn.nseg = L.nseg;
  pn.seg_len = L.seg_len;
  pn.dSseg_out = at<float>(ws, L.sN);
  hipError_t e = launch_bscan_bf16<DK, DV>(pn, st);
  if (e != hipSuccess) return e;
  if constexpr (DK != DV) {
    BScanArgs pm = pn;
    pm.dout = nullptr;
    pm.flags = kScanNoInput | kScanEye;
    pm.dSseg_out = at<float>(ws, L.sM);
    e = launch_bscan_bf16<DK, DK>(pm, st);
    if (e != hipSuccess) return e;
  }
  SegCombineArgs ca{at<float>(ws, L.sM), at<float>(ws, L.sN), ba.dST, at<float>(ws, L.sX),
                    ba.B * ba.H, L.nseg, 1};
  ca.transpose_m = DK == DV;
  e = launch_segcombine<DK, DV>(ca, st);
  if (e != hipSuccess) return e;
  BScanArgs p3 = ba;
  p3.nseg = L.nseg;
  p3.seg_len = L.seg_len;
  p3.dSseg_in = at<float>(ws, L.sX);
  return launch_bscan_bf16<DK, DV>(p3, st);
}

// ---- dispatch over (Dk, Dv) ------------------------------------------------
template <template <int, int, typename> class F, typename TIn, typename... A>
hipError_t dispatch(int Dk, int Dv, A&&... args) {
  if (Dk == 64 && Dv == 64) return F<64, 64, TIn>::run(args...);
  if (Dk == 64 && Dv == 128) return F<64, 128, TIn>::run(args...);
  if (Dk == 128 && Dv == 64) return F<128, 64, TIn>::run(args...);
  return F<128, 128, TIn>::run(args...);
}

template <int DK, int DV, typename TIn>
struct FwdRun {
  // save: also leave A, the chunk-start states and R in the workspace (backward layout)
  static hipError_t run(const gdr2_problem* p, const void* q, const void* k, const void* v,
                        const float* g, const void* b, const void* w, const float* S0, void* o,
                        float* ST, void* ws, bool save, const Geo& G, hipStream_t st) {
    const Layout& L = G.L;
    const int NT = G.NT;
    if (std::is_same<TIn, bf16_t>::value) {
      // bf16: chunk-parallel intra-chunk kernel, then the state scan with the output
      IntraBf16Args ia{static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                       static_cast<const bf16_t*>(v), g, static_cast<const bf16_t*>(b),
                       static_cast<const bf16_t*>(w), at<unsigned char>(ws, L.bY),
                       at<unsigned char>(ws, L.bQ), at<unsigned char>(ws, L.bA),
                       at<unsigned char>(ws, L.bK), at<float>(ws, L.bU), at<float>(ws, L.bG),
                       save ? at<_Float16>(ws, L.bAm) : nullptr, p->B, p->T, p->H, NT};
      ia.Amsc = save ? at<float>(ws, L.bAmsc) : nullptr;
      ia.vl = G.vl;
      ia.G = G.G;
      ia.st = G.st;
      hipError_t e = timed(GDR2_K_FWD_INTRA, st, [&] { return launch_intra_bf16<DK, DV>(ia, st); });
      if (e != hipSuccess) return e;
      ScanArgs sa{ia.Y, ia.Qg, ia.Aqk, ia.KtT, ia.U, ia.GC, S0, ST, static_cast<bf16_t*>(o),
                  save ? at<_Float16>(ws, L.Hs) : nullptr, save ? at<_Float16>(ws, L.Rs) : nullptr,
                  G.nscan, p->T, p->H, NT, p->scale};
      sa.Hsc = save ? at<float>(ws, L.Hsc) : nullptr;
      sa.Rsc = save ? at<float>(ws, L.Rsc) : nullptr;
      sa.vl = G.vl;
      sa.G = G.G;
      return timed(GDR2_K_FWD_STATE, st, [&] {
        return scan_fwd_bf16<DK, DV>(sa, L, ws, [&](const ScanArgs& x) {
          return save ? launch_scan_bf16<DK, DV, true, true>(x, st) : launch_scan_bf16<DK, DV, true, false>(x, st);
        }, st);
      });
    }
    IntraArgs<TIn> ia{static_cast<const TIn*>(q), static_cast<const TIn*>(k),
                      static_cast<const TIn*>(v), g, static_cast<const TIn*>(b),
                      static_cast<const TIn*>(w), at<float>(ws, L.Y), at<float>(ws, L.U),
                      at<float>(ws, L.Kt), at<float>(ws, L.Qg), at<float>(ws, L.Aqk),
                      at<float>(ws, L.GC), p->T, p->H, NT};
    ia.vl = G.vl;
    ia.G = G.G;
    hipError_t e = timed(GDR2_K_FWD_INTRA, st, [&] { return launch_fwd_intra<DK, DV, TIn>(ia, p->B, st); });
    if (e != hipSuccess) return e;
    StateArgs<TIn> sa{ia.Y, ia.U, ia.Kt, ia.Qg, ia.Aqk, ia.GC, S0, ST, static_cast<TIn*>(o),
                      save ? at<float>(ws, L.Hs) : nullptr, save ? at<float>(ws, L.Rs) : nullptr,
                      p->T, p->H, NT, p->scale};
    sa.vl = G.vl;
    return timed(GDR2_K_FWD_STATE, st, [&] {
      return save ? launch_fwd_state<DK, DV, TIn, true, true>(sa, G.nscan, st)
                  : launch_fwd_state<DK, DV, TIn, true, false>(sa, G.nscan, st);
    });
  }
};

template <int DK, int DV, typename TIn>
struct BwdRun {
  // saved: the workspace holds what a saving forward left there; skip the recompute
  static hipError_t run(const gdr2_problem* p, const void* q, const void* k, const void* v,
                        const float* g, const void* b, const void* w, const float* S0,
                        const void* dout, const float* dST, void* dq, void* dk, void* dv,
                        float* dg, void* db, void* dw, float* dS0, void* ws, bool saved, const Geo& G,
                        float* da, float* ddelta, hipStream_t st) {
    const Layout& L = G.L;
    const int NT = G.NT;
    const bool fused = G.st.a_log != nullptr;
    hipError_t e = hipSuccess;
    if (std::is_same<TIn, bf16_t>::value) {
      IntraBf16Args ia{static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                       static_cast<const bf16_t*>(v), g, static_cast<const bf16_t*>(b),
                       static_cast<const bf16_t*>(w), at<unsigned char>(ws, L.bY),
                       at<unsigned char>(ws, L.bQ), at<unsigned char>(ws, L.bA),
                       at<unsigned char>(ws, L.bK), at<float>(ws, L.bU), at<float>(ws, L.bG),
                       at<_Float16>(ws, L.bAm), p->B, p->T, p->H, NT};
      ia.Amsc = at<float>(ws, L.bAmsc);
      ia.vl = G.vl;
      ia.G = G.G;
      ia.st = G.st;
      if (!saved) {
        // recompute: intra-chunk tiles (with A), then the forward scan storing the chunk states and R
        e = timed(GDR2_K_BWD_RECOMPUTE_INTRA, st, [&] { return launch_intra_bf16<DK, DV>(ia, st); });
        if (e != hipSuccess) return e;
        ScanArgs sa{ia.Y, ia.Qg, ia.Aqk, ia.KtT, ia.U, ia.GC, S0, nullptr, nullptr, at<_Float16>(ws, L.Hs),
                    at<_Float16>(ws, L.Rs), G.nscan, p->T, p->H, NT, p->scale};
        sa.Hsc = at<float>(ws, L.Hsc);
        sa.Rsc = at<float>(ws, L.Rsc);
        sa.vl = G.vl;
        sa.G = G.G;
        e = timed(GDR2_K_BWD_RECOMPUTE_STATE, st, [&] {
          return scan_fwd_bf16<DK, DV>(sa, L, ws, [&](const ScanArgs& x) {
            return launch_scan_bf16<DK, DV, false, true>(x, st);
          }, st);
        });
        if (e != hipSuccess) return e;
      }
      BScanArgs ba{ia.Y, ia.Qg, ia.Aqk, ia.KtT, ia.GC, static_cast<const bf16_t*>(dout), dST, dS0,
                   at<_Float16>(ws, L.DH), at<__bf16>(ws, L.bDR), G.nscan, p->T, p->H, NT, p->scale};
      ba.DHsc = at<float>(ws, L.DHsc);
      ba.vl = G.vl;
      ba.G = G.G;
      e = timed(GDR2_K_BWD_STATE, st, [&] { return scan_bwd_bf16<DK, DV>(ba, L, ws, st); });
      if (e != hipSuccess) return e;
      // the WY VJP and the intra-chunk VJP in one chunk-parallel kernel
      BChunkBf16Args ca{static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                        static_cast<const bf16_t*>(v), g, static_cast<const bf16_t*>(b),
                        static_cast<const bf16_t*>(w), static_cast<const bf16_t*>(dout), at<_Float16>(ws, L.Hs),
                        at<_Float16>(ws, L.DH), at<_Float16>(ws, L.Rs), at<__bf16>(ws, L.bDR),
                        at<_Float16>(ws, L.bAm), static_cast<bf16_t*>(dq), static_cast<bf16_t*>(dk),
                        static_cast<bf16_t*>(dv), static_cast<bf16_t*>(db), static_cast<bf16_t*>(dw), dg,
                        p->B, p->T, p->H, NT, p->scale};
      ca.Hsc = at<float>(ws, L.Hsc);
      ca.DHsc = at<float>(ws, L.DHsc);
      ca.Rsc = at<float>(ws, L.Rsc);
      ca.Amsc = at<float>(ws, L.bAmsc);
      ca.vl = G.vl;
      ca.G = G.G;
      if (G.G > 1) {  // the group's key-side gradients add up on the key-head axis
        ca.Aq = at<float>(ws, L.pQ);
        ca.Ak = at<float>(ws, L.pK);
        ca.Ab = at<float>(ws, L.pB);
        ca.Ag = at<float>(ws, L.pG);
      }
      if (fused) {
        ca.st = G.st;
        ca.PD = at<float>(ws, L.PD);
        ca.PA = at<float>(ws, L.PA);
        ca.Pq = at<float>(ws, L.pQ);
        ca.Pk = at<float>(ws, L.pK);
      }
      e = timed(GDR2_K_BWD_INTRA, st, [&] {
        // one launch per value head of the groups, in order (G = 1: one launch)
        hipError_t r = hipSuccess;
        for (int j = 0; j < G.G && r == hipSuccess; ++j) {
          ca.gj = j;
          ca.gmode = G.G == 1 ? 0 : (j == 0 ? 1 : (j + 1 < G.G ? 2 : 3));
          r = launch_bchunk_bf16<DK, DV>(ca, st);
        }
        return r;
      });
      if (e != hipSuccess || !fused) return e;
      return timed(GDR2_K_STAGE_BWD, st, [&] { return stage_bwd<DK>(p, G, ws, q, k, dq, dk, da, ddelta, st); });
    }
    IntraArgs<TIn> ia{static_cast<const TIn*>(q), static_cast<const TIn*>(k),
                      static_cast<const TIn*>(v), g, static_cast<const TIn*>(b),
                      static_cast<const TIn*>(w), at<float>(ws, L.Y), at<float>(ws, L.U),
                      at<float>(ws, L.Kt), at<float>(ws, L.Qg), at<float>(ws, L.Aqk),
                      at<float>(ws, L.GC), p->T, p->H, NT};
    ia.vl = G.vl;
    ia.G = G.G;
    StateArgs<TIn> sa{ia.Y, ia.U, ia.Kt, ia.Qg, ia.Aqk, ia.GC, S0, nullptr, nullptr,
                      at<float>(ws, L.Hs), at<float>(ws, L.Rs), p->T, p->H, NT, p->scale};
    sa.vl = G.vl;
    if (!saved) {
      e = timed(GDR2_K_BWD_RECOMPUTE_INTRA, st, [&] { return launch_fwd_intra<DK, DV, TIn>(ia, p->B, st); });
      if (e != hipSuccess) return e;
      e = timed(GDR2_K_BWD_RECOMPUTE_STATE, st,
                [&] { return launch_fwd_state<DK, DV, TIn, false, true>(sa, G.nscan, st); });
      if (e != hipSuccess) return e;
    }
    BwdStateArgs<TIn> ba{ia.Qg, ia.Kt, ia.Y, ia.Aqk, ia.GC, static_cast<const TIn*>(dout), dST,
                         dS0, at<float>(ws, L.DH), at<float>(ws, L.DR), p->T, p->H, NT, p->scale};
    ba.vl = G.vl;
    e = timed(GDR2_K_BWD_STATE, st, [&] { return launch_bwd_state<DK, DV, TIn>(ba, G.nscan, st); });
    if (e != hipSuccess) return e;
    BwdChunkArgs<TIn> ca{static_cast<const TIn*>(q), static_cast<const TIn*>(k),
                         static_cast<const TIn*>(v), g, static_cast<const TIn*>(b),
                         static_cast<const TIn*>(w), static_cast<const TIn*>(dout),
                         sa.Hs, ba.DH, sa.Rs, ba.DR, at<float>(ws, L.DAqk), at<float>(ws, L.DT),
                         at<float>(ws, L.DEg), static_cast<TIn*>(dq), static_cast<TIn*>(dk),
                         static_cast<TIn*>(dv), static_cast<TIn*>(db), static_cast<TIn*>(dw), dg,
                         p->T, p->H, NT, p->scale};
    ca.vl = G.vl;
    ca.G = G.G;
    e = timed(GDR2_K_BWD_WY, st, [&] { return launch_bwd_wy<DK, DV, TIn>(ca, p->B, st); });
    if (e != hipSuccess) return e;
    if (G.G > 1) {  // the key-side gradients of each value head go to the fp32 partials
      ca.dq = reinterpret_cast<TIn*>(at<float>(ws, L.pQ));
      ca.dk = reinterpret_cast<TIn*>(at<float>(ws, L.pK));
      ca.db = reinterpret_cast<TIn*>(at<float>(ws, L.pB));
      ca.dg = at<float>(ws, L.pG);
    }
    return timed(GDR2_K_BWD_INTRA, st, [&] {
      hipError_t r = launch_bwd_intra<DK, DV, TIn>(ca, p->B, st);
      if (r == hipSuccess && G.G > 1) r = group_reduce<TIn>(p, G, L, ws, dq, dk, db, dg, st);
      return r;
    });
  }
};

template <int DK, int DV, typename TIn>
struct RecRun {
  static hipError_t run(const gdr2_problem* p, const void* q, const void* k, const void* v,
                        const float* g, const void* b, const void* w, float* S, void* o, const int* cu,
                        int nseq, int grp, const gdr2_stage* stage, hipStream_t st) {
    RecurArgs<TIn> ra{static_cast<const TIn*>(q), static_cast<const TIn*>(k),
                      static_cast<const TIn*>(v), g, static_cast<const TIn*>(b),
                      static_cast<const TIn*>(w), S, static_cast<TIn*>(o), p->T, p->H, p->scale};
    ra.cu = cu;
    ra.G = grp;
    if (stage != nullptr) {
      ra.st.a_log = stage->a_log;
      ra.st.delta = stage->delta;
      ra.st.eps = stage->eps;
    }
    const int nb = cu != nullptr ? nseq : p->B;
    return timed(GDR2_K_RECURRENT, st, [&] { return launch_recurrent<DK, DV, TIn>(ra, nb, st); });
  }
};

bool all_ok(std::initializer_list<const void*> req) {
  for (const void* x : req)
    if (x == nullptr || !aligned16(x)) return false;
  return true;
}

bool opt_ok(std::initializer_list<const void*> opt) {
  for (const void* x : opt)
    if (x != nullptr && !aligned16(x)) return false;
  return true;
}

bool cu_ok(const int32_t* cu) { return cu != nullptr && (reinterpret_cast<uintptr_t>(cu) & 3u) == 0; }

// The fused stage's parameters: a_log 4-byte aligned, delta 16-byte aligned, eps finite and >= 0.
bool stage_ok(const gdr2_stage* s) {
  if (s == nullptr || s->a_log == nullptr || s->delta == nullptr) return false;
  if ((reinterpret_cast<uintptr_t>(s->a_log) & 3u) != 0 || !aligned16(s->delta)) return false;
  return std::isfinite(s->eps) && s->eps >= 0.f;
}

}  // namespace

extern "C" {

gdr2_status gdr2_chunk_workspace_bytes(const gdr2_problem* p, int for_backward, size_t* bytes) {
  if (bytes == nullptr) return GDR2_EINVAL;
  const gdr2_status s = check_problem(p, true);
  if (s != GDR2_OK) return s;
  const gdr2_problem pv = value_view(p);
  *bytes = layout(&pv, for_backward != 0, 0, group_of(p)).total;
  return GDR2_OK;
}

namespace {

// A call with the fused stage checks it (both dtypes: the bf16 chunk path fuses
// the stage into its kernels, fp32 problems run it as passes of its own).
gdr2_status check_stage(const gdr2_problem*, const gdr2_stage* stage, bool) {
  if (stage == nullptr) return GDR2_OK;
  if (!stage_ok(stage)) return GDR2_EINVAL;
  return GDR2_OK;
}

// The stage's passes for fp32 problems (p: the value view).
StageF32Args stage_f32_args(const gdr2_problem* p, const Layout& L, void* ws, const gdr2_stage* stage, int G,
                            const void* q, const void* k, const float* f) {
  StageF32Args s{};
  s.q = static_cast<const float*>(q);
  s.k = static_cast<const float*>(k);
  s.f = f;
  s.a_log = stage->a_log;
  s.delta = stage->delta;
  s.eps = stage->eps;
  s.qn = at<float>(ws, L.fQ);
  s.kn = at<float>(ws, L.fK);
  s.g = at<float>(ws, L.fG);
  s.rq = at<float>(ws, L.RQ);
  s.rk = at<float>(ws, L.RK);
  s.rows = (size_t)p->B * p->T;
  s.Hk = p->H / G;
  return s;
}

hipError_t launch_stage(const gdr2_problem* p, const StageF32Args& s, bool backward, hipStream_t st) {
  return p->Dk == 64 ? launch_stage_f32<64>(s, backward, st) : launch_stage_f32<128>(s, backward, st);
}

// nseq > 0 (with cu): packed variable-length call
// stage: the fused input stage (log_alpha then holds the decay projection f) or null
gdr2_status chunk_fwd(const gdr2_problem* p, const int32_t* cu, int nseq, const void* q, const void* k,
                      const void* v, const float* log_alpha, const void* b, const void* w, const float* S0,
                      void* o, float* S_T, void* ws, size_t ws_bytes, bool save, hipStream_t stream,
                      const gdr2_stage* stage = nullptr) {
  gdr2_status s = check_problem(p, true, nseq);
  if (s != GDR2_OK) return s;
  s = check_stage(p, stage, true);
  if (s != GDR2_OK) return s;
  if (!all_ok({q, k, v, log_alpha, b, w, o, ws}) || !opt_ok({S0, S_T})) return GDR2_EINVAL;
  if (nseq > 0 && !cu_ok(cu)) return GDR2_EINVAL;
  const gdr2_problem pv = value_view(p);
  const Geo G = make_geo(&pv, save, nseq, cu, ws, group_of(p), stage);
  if (ws_bytes < G.L.total) return GDR2_EWORKSPACE;
  if (stage != nullptr && p->dtype == GDR2_FP32) {
    // normalised q, k and g into the workspace, then the fp32 operator on them
    const StageF32Args sa = stage_f32_args(&pv, G.L, ws, stage, G.G, q, k, log_alpha);
    hipError_t e = timed(GDR2_K_STAGE_FWD, stream, [&] { return launch_stage(&pv, sa, false, stream); });
    if (e != hipSuccess) return hip_status(e, stream);
    return chunk_fwd(p, cu, nseq, sa.qn, sa.kn, v, sa.g, b, w, S0, o, S_T, ws, ws_bytes, save, stream);
  }
  hipError_t e = build_table(&pv, G, stream);
  if (e != hipSuccess) return GDR2_EHIP;
  if (p->dtype == GDR2_BF16)
    e = dispatch<FwdRun, bf16_t>(p->Dk, p->Dv, &pv, q, k, v, log_alpha, b, w, S0, o, S_T, ws, save, G, stream);
  else
    e = dispatch<FwdRun, float>(p->Dk, p->Dv, &pv, q, k, v, log_alpha, b, w, S0, o, S_T, ws, save, G, stream);
  return hip_status(e, stream);
}

// stage: the fused input stage (log_alpha holds f, dlog_alpha receives df; da
// and ddelta receive the parameter gradients) or null
gdr2_status chunk_bwd(const gdr2_problem* p, const int32_t* cu, int nseq, const void* q, const void* k,
                      const void* v, const float* log_alpha, const void* b, const void* w, const float* S0,
                      const void* dout, const float* dS_T, void* dq, void* dk, void* dv,
                      float* dlog_alpha, void* db, void* dw, float* dS0, void* ws, size_t ws_bytes,
                      bool saved, hipStream_t stream, const gdr2_stage* stage = nullptr, float* da = nullptr,
                      float* ddelta = nullptr) {
  gdr2_status s = check_problem(p, true, nseq);
  if (s != GDR2_OK) return s;
  s = check_stage(p, stage, true);
  if (s != GDR2_OK) return s;
  if (!all_ok({q, k, v, log_alpha, b, w, dout, dq, dk, dv, dlog_alpha, db, dw, ws}) ||
      !opt_ok({S0, dS_T, dS0}))
    return GDR2_EINVAL;
  if (stage != nullptr && (da == nullptr || (reinterpret_cast<uintptr_t>(da) & 3u) != 0 || !all_ok({ddelta})))
    return GDR2_EINVAL;
  if (nseq > 0 && !cu_ok(cu)) return GDR2_EINVAL;
  const gdr2_problem pv = value_view(p);
  const Geo G = make_geo(&pv, true, nseq, cu, ws, group_of(p), stage);
  if (ws_bytes < G.L.total) return GDR2_EWORKSPACE;
  if (stage != nullptr && p->dtype == GDR2_FP32) {
    // the stage again (normalised q, k, g), the fp32 operator's backward into the
    // workspace, then the stage's VJPs and the decay-parameter sums
    StageF32Args sa = stage_f32_args(&pv, G.L, ws, stage, G.G, q, k, log_alpha);
    sa.dqn = at<float>(ws, G.L.fdQ);
    sa.dkn = at<float>(ws, G.L.fdK);
    sa.dg = at<float>(ws, G.L.fdG);
    sa.dq = static_cast<float*>(dq);
    sa.dk = static_cast<float*>(dk);
    sa.df = dlog_alpha;
    sa.pa = at<float>(ws, G.L.PA);
    hipError_t e = timed(GDR2_K_STAGE_FWD, stream, [&] { return launch_stage(&pv, sa, false, stream); });
    if (e != hipSuccess) return hip_status(e, stream);
    const gdr2_status r = chunk_bwd(p, cu, nseq, sa.qn, sa.kn, v, sa.g, b, w, S0, dout, dS_T, at<float>(ws, G.L.fdQ),
                                    at<float>(ws, G.L.fdK), dv, at<float>(ws, G.L.fdG), db, dw, dS0, ws, ws_bytes,
                                    saved, stream);
    if (r != GDR2_OK) return r;
    e = timed(GDR2_K_STAGE_BWD, stream, [&] {
      hipError_t x = launch_stage(&pv, sa, true, stream);
      const int Hk = pv.H / G.G, nrow = pv.B * pv.T, splits = nrow < kParamSplits ? nrow : kParamSplits;
      float* PT = at<float>(ws, G.L.PT);
      float* PT1 = PT + (size_t)kParamSplits * Hk * pv.Dk;
      if (x == hipSuccess) x = launch_param_reduce_pass(sa.df, PT, nrow, Hk, 1, pv.Dk, splits, stream);
      if (x == hipSuccess) x = launch_param_reduce_pass(PT, ddelta, splits, Hk, 1, pv.Dk, 1, stream);
      if (x == hipSuccess) x = launch_param_reduce_pass(sa.pa, PT1, nrow, Hk, 1, 1, splits, stream);
      if (x == hipSuccess) x = launch_param_reduce_pass(PT1, da, splits, Hk, 1, 1, 1, stream);
      return x;
    });
    return hip_status(e, stream);
  }
  hipError_t e = build_table(&pv, G, stream);
  if (e != hipSuccess) return GDR2_EHIP;
  if (p->dtype == GDR2_BF16)
    e = dispatch<BwdRun, bf16_t>(p->Dk, p->Dv, &pv, q, k, v, log_alpha, b, w, S0, dout, dS_T, dq,
                                 dk, dv, dlog_alpha, db, dw, dS0, ws, saved, G, da, ddelta, stream);
  else
    e = dispatch<BwdRun, float>(p->Dk, p->Dv, &pv, q, k, v, log_alpha, b, w, S0, dout, dS_T, dq,
                                dk, dv, dlog_alpha, db, dw, dS0, ws, saved, G, da, ddelta, stream);
  return hip_status(e, stream);
}

gdr2_status recurrent(const gdr2_problem* p, const int32_t* cu, int nseq, const void* q, const void* k,
                      const void* v, const float* log_alpha, const void* b, const void* w, float* S, void* o,
                      hipStream_t stream, const gdr2_stage* stage = nullptr) {
  gdr2_status s = check_problem(p, false, nseq);
  if (s != GDR2_OK) return s;
  s = check_stage(p, stage, false);
  if (s != GDR2_OK) return s;
  if (!all_ok({q, k, v, log_alpha, b, w, S, o})) return GDR2_EINVAL;
  if (nseq > 0 && !cu_ok(cu)) return GDR2_EINVAL;
  hipError_t e;
  const gdr2_problem pv = value_view(p);
  if (p->dtype == GDR2_BF16)
    e = dispatch<RecRun, bf16_t>(p->Dk, p->Dv, &pv, q, k, v, log_alpha, b, w, S, o, cu, nseq, group_of(p), stage,
                                 stream);
  else
    e = dispatch<RecRun, float>(p->Dk, p->Dv, &pv, q, k, v, log_alpha, b, w, S, o, cu, nseq, group_of(p), stage,
                                stream);
  return hip_status(e, stream);
}

}  // namespace

gdr2_status gdr2_chunk_fwd(const gdr2_problem* p, const void* q, const void* k, const void* v,
                           const float* log_alpha, const void* b, const void* w, const float* S0,
                           void* o, float* S_T, void* ws, size_t ws_bytes, hipStream_t stream) {
  return chunk_fwd(p, nullptr, 0, q, k, v, log_alpha, b, w, S0, o, S_T, ws, ws_bytes, false, stream);
}

gdr2_status gdr2_chunk_fwd_save(const gdr2_problem* p, const void* q, const void* k, const void* v,
                                const float* log_alpha, const void* b, const void* w, const float* S0,
                                void* o, float* S_T, void* ws, size_t ws_bytes, hipStream_t stream) {
  return chunk_fwd(p, nullptr, 0, q, k, v, log_alpha, b, w, S0, o, S_T, ws, ws_bytes, true, stream);
}

gdr2_status gdr2_chunk_bwd(const gdr2_problem* p, const void* q, const void* k, const void* v,
                           const float* log_alpha, const void* b, const void* w, const float* S0,
                           const void* dout, const float* dS_T, void* dq, void* dk, void* dv,
                           float* dlog_alpha, void* db, void* dw, float* dS0, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  return chunk_bwd(p, nullptr, 0, q, k, v, log_alpha, b, w, S0, dout, dS_T, dq, dk, dv, dlog_alpha, db, dw,
                   dS0, ws, ws_bytes, false, stream);
}

gdr2_status gdr2_chunk_bwd_saved(const gdr2_problem* p, const void* q, const void* k, const void* v,
                                 const float* log_alpha, const void* b, const void* w, const float* S0,
                                 const void* dout, const float* dS_T, void* dq, void* dk, void* dv,
                                 float* dlog_alpha, void* db, void* dw, float* dS0, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  return chunk_bwd(p, nullptr, 0, q, k, v, log_alpha, b, w, S0, dout, dS_T, dq, dk, dv, dlog_alpha, db, dw,
                   dS0, ws, ws_bytes, true, stream);
}

gdr2_status gdr2_recurrent_step(const gdr2_problem* p, const void* q, const void* k, const void* v,
                                const float* log_alpha, const void* b, const void* w, float* S,
                                void* o, hipStream_t stream) {
  return recurrent(p, nullptr, 0, q, k, v, log_alpha, b, w, S, o, stream);
}

gdr2_status gdr2_varlen_workspace_bytes(const gdr2_problem* p, int32_t n_seqs, int for_backward,
                                        size_t* bytes) {
  if (bytes == nullptr || n_seqs <= 0) return GDR2_EINVAL;
  const gdr2_status s = check_problem(p, true, n_seqs);
  if (s != GDR2_OK) return s;
  const gdr2_problem pv = value_view(p);
  *bytes = layout(&pv, for_backward != 0, n_seqs, group_of(p)).total;
  return GDR2_OK;
}

gdr2_status gdr2_chunk_fwd_varlen(const gdr2_problem* p, const int32_t* cu_seqlens, int32_t n_seqs,
                                  const void* q, const void* k, const void* v, const float* log_alpha,
                                  const void* b, const void* w, const float* S0, void* o, float* S_T, void* ws,
                                  size_t ws_bytes, int save, hipStream_t stream) {
  if (n_seqs <= 0) return GDR2_EINVAL;
  return chunk_fwd(p, cu_seqlens, n_seqs, q, k, v, log_alpha, b, w, S0, o, S_T, ws, ws_bytes, save != 0,
                   stream);
}

gdr2_status gdr2_chunk_bwd_varlen(const gdr2_problem* p, const int32_t* cu_seqlens, int32_t n_seqs,
                                  const void* q, const void* k, const void* v, const float* log_alpha,
                                  const void* b, const void* w, const float* S0, const void* dout,
                                  const float* dS_T, void* dq, void* dk, void* dv, float* dlog_alpha, void* db,
                                  void* dw, float* dS0, void* ws, size_t ws_bytes, int saved,
                                  hipStream_t stream) {
  if (n_seqs <= 0) return GDR2_EINVAL;
  return chunk_bwd(p, cu_seqlens, n_seqs, q, k, v, log_alpha, b, w, S0, dout, dS_T, dq, dk, dv, dlog_alpha, db,
                   dw, dS0, ws, ws_bytes, saved != 0, stream);
}

gdr2_status gdr2_recurrent_varlen(const gdr2_problem* p, const int32_t* cu_seqlens, int32_t n_seqs,
                                  const void* q, const void* k, const void* v, const float* log_alpha,
                                  const void* b, const void* w, float* S, void* o, hipStream_t stream) {
  if (n_seqs <= 0) return GDR2_EINVAL;
  return recurrent(p, cu_seqlens, n_seqs, q, k, v, log_alpha, b, w, S, o, stream);
}

gdr2_status gdr2_fused_workspace_bytes(const gdr2_problem* p, int32_t n_seqs, int for_backward, size_t* bytes) {
  if (bytes == nullptr || n_seqs < 0) return GDR2_EINVAL;
  const gdr2_status s = check_problem(p, true, n_seqs);
  if (s != GDR2_OK) return s;
  const gdr2_problem pv = value_view(p);
  *bytes = layout(&pv, for_backward != 0, n_seqs, group_of(p), true).total;
  return GDR2_OK;
}

gdr2_status gdr2_fused_fwd(const gdr2_problem* p, const gdr2_stage* stage, const int32_t* cu_seqlens,
                           int32_t n_seqs, const void* q, const void* k, const void* v, const float* f,
                           const void* b, const void* w, const float* S0, void* o, float* S_T, void* ws,
                           size_t ws_bytes, int save, hipStream_t stream) {
  if (stage == nullptr || n_seqs < 0) return GDR2_EINVAL;
  return chunk_fwd(p, n_seqs > 0 ? cu_seqlens : nullptr, n_seqs, q, k, v, f, b, w, S0, o, S_T, ws, ws_bytes,
                   save != 0, stream, stage);
}

gdr2_status gdr2_fused_bwd(const gdr2_problem* p, const gdr2_stage* stage, const int32_t* cu_seqlens,
                           int32_t n_seqs, const void* q, const void* k, const void* v, const float* f,
                           const void* b, const void* w, const float* S0, const void* dout, const float* dS_T,
                           void* dq, void* dk, void* dv, float* df, float* da, float* ddelta, void* db, void* dw,
                           float* dS0, void* ws, size_t ws_bytes, int saved, hipStream_t stream) {
  if (stage == nullptr || n_seqs < 0) return GDR2_EINVAL;
  return chunk_bwd(p, n_seqs > 0 ? cu_seqlens : nullptr, n_seqs, q, k, v, f, b, w, S0, dout, dS_T, dq, dk, dv, df,
                   db, dw, dS0, ws, ws_bytes, saved != 0, stream, stage, da, ddelta);
}

gdr2_status gdr2_fused_recurrent(const gdr2_problem* p, const gdr2_stage* stage, const int32_t* cu_seqlens,
                                 int32_t n_seqs, const void* q, const void* k, const void* v, const float* f,
                                 const void* b, const void* w, float* S, void* o, hipStream_t stream) {
  if (stage == nullptr || n_seqs < 0) return GDR2_EINVAL;
  return recurrent(p, n_seqs > 0 ? cu_seqlens : nullptr, n_seqs, q, k, v, f, b, w, S, o, stream, stage);
}

gdr2_status gdr2_profile_enable(int on) {
  g_prof.on = on != 0;
  return GDR2_OK;
}

gdr2_status gdr2_profile_collect(double* ms, long long* launches, int n) {
  if (ms == nullptr || launches == nullptr || n < GDR2_NUM_KERNELS) return GDR2_EINVAL;
  gdr2_status st = GDR2_OK;
  for (const auto& p : g_prof.pending) {
    float t = 0.f;
    if (hipEventSynchronize(p.b) != hipSuccess || hipEventElapsedTime(&t, p.a, p.b) != hipSuccess) {
      st = GDR2_EHIP;
    } else {
      g_prof.ms[p.id] += t;
      g_prof.launches[p.id] += 1;
    }
    g_prof.pool.push_back(p.a);
    g_prof.pool.push_back(p.b);
  }
  g_prof.pending.clear();
  for (int i = 0; i < n; ++i) {
    ms[i] = i < GDR2_NUM_KERNELS ? g_prof.ms[i] : 0.0;
    launches[i] = i < GDR2_NUM_KERNELS ? g_prof.launches[i] : 0;
  }
  for (int i = 0; i < GDR2_NUM_KERNELS; ++i) {
    g_prof.ms[i] = 0.0;
    g_prof.launches[i] = 0;
  }
  return st;
}

const char* gdr2_status_str(gdr2_status st) {
  switch (st) {
    case GDR2_OK: return "GDR2_OK";
    case GDR2_EINVAL: return "GDR2_EINVAL: invalid argument";
    case GDR2_EUNSUPPORTED: return "GDR2_EUNSUPPORTED: unsupported problem";
    case GDR2_EWORKSPACE: return "GDR2_EWORKSPACE: workspace too small";
    case GDR2_EHIP: return "GDR2_EHIP: HIP launch error";
  }
  return "GDR2_UNKNOWN";
}

}  // extern "C"

// Inter-chunk state scan of the bf16 path (gfx950): one 8-wave workgroup per
// (sequence, head, 64-wide value slice) walks the chunks in order:
//
//   R  = U - Y S                                     eq. eq_app_residual_matrix
//   O  = scale * (Q_g S + A_qk R)                    eq. eq_gdn2_chunk_output   [WITH_O]
//   S <- Diag(gamma_C) S + Ktail^T R                 eq. eq_gdn2_chunk_state
//
// reading Y, Q_g, A_qk, Ktail^T, U and gamma_C that the intra-chunk kernel
// left in fragment order.  The fp32 state slice lives in registers as MFMA
// accumulators (plus a bf16 hi/lo copy in LDS for the products that read it);
// the next chunk's operand blocks are fetched into registers in groups over
// the current chunk's step and copied to LDS at its end, with the step's own
// stores (R, O, the chunk state) behind its products.  With eight key blocks
// each wave's K_tail^T blocks (no other wave reads them) go from memory
// straight into its registers, one chunk ahead.  The two value slices of one
// head run on the same XCD so that their shared reads hit one L2.
// With STORE_H the chunk-start states (fp16 with block scales, store_state_f16)
// and R are written for the backward (alone in the backward's recompute, or
// with the output when the forward keeps them).
// With nseg > 1 each workgroup scans one segment of a sequence from a given
// start state (ScanArgs), which the sequence-parallel mode builds on.  Its
// map pass (MAP, Dk = DV) forms both segment maps in one launch: per segment
// one workgroup takes the whole value width of N (zero start, input U) and
// one the whole of M (identity start, no input), on the same XCD, so the Y
// and Ktail^T blocks of a step are read by two workgroups rather than by the
// four that two passes of 64-wide slices need.  Its Y S products use both
// parts of S, so the maps are fp32-accurate: the reverse scan chains the
// gradient with M^T (its segment map), the exact transpose of this one.
//
// Precision: Y S uses the bf16 part of S (Y itself is bf16), except in the
// map pass, which adds the lo part; every other product is split hi/lo and
// fp32-accurate.

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK, int DV, bool MAP = false>
struct ScanCfg2 {
  static constexpr int NTHR = 512;
  // MAP: two "slices" of the full width, the N map and the M map
  static constexpr int DVS = MAP ? DV : (DV < 64 ? DV : 64);
  static constexpr int NS = MAP ? 2 : DV / DVS;
  static constexpr int KS = DK / 32, NCB = DK / 16, NVB = DVS / 16;
  static constexpr int TPW = NCB * NVB / 8;  // state tiles per wave
  // S hi/lo [DVS][LSS] bf16; the map pass keeps it in the permuted K order of
  // Y's fragments, unpadded, its 16-byte pieces XOR'd with the row (map_s_ix)
  static constexpr int LSS = MAP ? DK : DK + 8;
  static constexpr int LR = 64 + 8;          // R hi/lo [DVS][LR] bf16
  // operand blocks, copied verbatim (contiguous Y | Qg | Aqk | KtT; MAP: Y | KtT;
  // KtT only without KD)
  static constexpr int SZ_Y = (int)WsBf16::y(DK), SZ_Q = MAP ? 0 : (int)WsBf16::qg(DK);
  static constexpr int SZ_A = MAP ? 0 : (int)WsBf16::aqk(), SZ_K = (int)WsBf16::ktt(DK);
  // with eight key blocks every wave's state tiles have a key block of their
  // own, so its K_tail^T blocks go from memory straight into its registers
  // (no LDS round trip); otherwise two waves share one and it is staged
  static constexpr bool KD = NCB == 8;
  static constexpr int SZ_OP = SZ_Y + SZ_Q + SZ_A + (KD ? 0 : SZ_K);
  static constexpr int NSTG = SZ_OP / (16 * NTHR);  // 16-byte chunks per thread
  static constexpr int OFF_S = 0;
  static constexpr int OFF_R = OFF_S + 2 * DVS * LSS * 2;
  static constexpr int OFF_OP = OFF_R + 2 * DVS * LR * 2;
  static constexpr int LDS = OFF_OP + SZ_OP;
  static_assert(SZ_OP % (16 * NTHR) == 0, "operand staging split");
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(TPW >= 1 && NVB % 2 == 0, "wave split");
  static_assert(!MAP || DK == DV, "map pass: square maps");
};

// Map pass: element (row v, key c) of S^T in LDS, keys in the permuted order of
// Y's fragments (4 m + e and 16 + 4 m + e side by side at 8 m + e, 8 m + 4 + e
// of each 32-key group) and the 16-byte pieces of a row XOR'd with v % 16, so
// that Y's B fragment is one 16-byte read and those reads are free of bank
// conflicts.  c4 is a multiple of 4: the 4 keys c4 .. c4 + 3 stay together.
template <int LD>
__device__ __forceinline__ int map_s_ix(int v, int c4) {
  const int a = (c4 & 31) >> 2, pos = (c4 & ~31) + (a < 4 ? 8 * a : 8 * (a - 4) + 4);
  return v * LD + ((((pos >> 3) ^ (v & 15)) << 3) | (pos & 7));
}
// its B fragment for K-step p: keys 32 p + 4 g + (0..3) and 32 p + 16 + 4 g + (0..3)
template <int LD>
__device__ __forceinline__ int map_s_frag(int v, int p, int g) {
  return v * LD + (((4 * p + g) ^ (v & 15)) << 3);
}

// B fragment of S for Y S in the permuted key order of Y's fragments:
// S[c][v] for c = k0 + 4 g + u and k0 + 16 + 4 g + u (stored [v][c]).
__device__ __forceinline__ bf8 ld_perm8(const __bf16* row, int k0, int g) {
  const bf4 a = *reinterpret_cast<const bf4*>(row + k0 + 4 * g);
  const bf4 b = *reinterpret_cast<const bf4*>(row + k0 + 16 + 4 * g);
  bf8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}

template <int DK, int DV, bool WITH_O, bool STORE_H, bool MAP>
__global__ __launch_bounds__(512) void scan_bf16_kernel(ScanArgs a) {
  static_assert(!MAP || (!WITH_O && !STORE_H), "the map pass writes the maps only");
  using C = ScanCfg2<DK, DV, MAP>;
  constexpr int DVS = C::DVS, NS = C::NS, KS = C::KS, NCB = C::NCB, NVB = C::NVB, TPW = C::TPW;
  constexpr int LSS = C::LSS, LR = C::LR, NSTG = C::NSTG;

  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* sShi = reinterpret_cast<__bf16*>(smem + C::OFF_S);
  __bf16* sSlo = sShi + DVS * LSS;
  __bf16* sRhi = reinterpret_cast<__bf16*>(smem + C::OFF_R);
  __bf16* sRlo = sRhi + DVS * LR;
  unsigned char* sOp = smem + C::OFF_OP;
  const unsigned char* sY = sOp;
  const unsigned char* sQ = sY + C::SZ_Y;
  const unsigned char* sA = sQ + C::SZ_Q;
  const unsigned char* sK = sA + C::SZ_A;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  const int T = a.T, H = a.H, NT = a.NT;

  // independent scans: (sequence, segment) pairs, vs = seq * nseg + seg
  const int nseg = a.nseg, nvirt = a.B * H * nseg;
  int vs, slice;
  if ((NS > 1 || a.G > 1) && ((nvirt / a.G) & 7) == 0) {
    // the NS value slices of the G value heads that read one key head's tiles
    // run on one XCD (consecutive blocks of an XCD), so they share its L2
    const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3, per = a.G * NS;
    const int unit = (j / per) * 8 + xcd, rem = j % per;
    const int HKs = H / a.G, qk = unit / nseg;
    vs = ((qk / HKs) * H + (qk % HKs) * a.G + rem / NS) * nseg + unit % nseg;
    slice = rem % NS;
  } else {
    vs = blockIdx.x / NS;
    slice = blockIdx.x % NS;
  }
  const int seq = scan_pair(a.vl, vs / nseg, H), seg = vs % nseg;  // (sequence, head) pair
  const ScanRange rng = scan_range(a.vl, seq, H, NT);
  const int seg_len = a.seg_len > 0 ? a.seg_len : rng.c1 - rng.c0;
  const int n0 = rng.c0 + seg * seg_len, n1 = min(rng.c1, n0 + seg_len);
  // MAP: slice 0 is the N map (input U, zero start), slice 1 the M map
  const bool no_input = MAP ? slice == 1 : (a.flags & kScanNoInput) != 0;
  const int h = seq % H;
  const int v0 = MAP ? 0 : slice * DVS;
  __bf16* O = reinterpret_cast<__bf16*>(a.o);

  // wave roles
  const int iO = wave >> 1;                 // row block of the R / O tiles
  const int vbO = (wave & 1) * (NVB / 2);   // their value blocks (slice-local)
  const int cs = wave % NCB;                // key block of the state tiles
  const int sv0 = (wave / NCB) * TPW;       // their value blocks

  // ---- operand staging (global -> registers -> LDS).  Thread t moves bytes
  // 8192 m + 16 t of the concatenated Y | Qg | Aqk | KtT blocks; every region is
  // a multiple of 8 KB, so the source region of slice m is known at compile time.
  constexpr int SLICE = 16 * C::NTHR;
  constexpr int E_Y = C::SZ_Y / SLICE, E_Q = E_Y + C::SZ_Q / SLICE, E_A = E_Q + C::SZ_A / SLICE;
  static_assert(C::SZ_Y % SLICE == 0 && C::SZ_Q % SLICE == 0 && C::SZ_A % SLICE == 0 && C::SZ_K % SLICE == 0,
                "regions are whole staging slices");
  u4v stg[NSTG];
  f4 ucur[NVB / 2], unext[NVB / 2];
  float gcur[4], gnext[4];
  const size_t chs = rng.chs;                        // value-head chunks: U, h, R
  const size_t chk = key_ch(a.vl, chs, H, a.G, NT);  // key-head chunks: Y, Q_g, A_qk, K_tail, gamma_C
  // Q_g and A_qk feed the output only: a scan without it moves Y and Ktail^T alone
#define GDR2_OP_USED(M_) (WITH_O || (M_) < E_Y || (M_) >= E_A)
// the thread's 16 bytes of slice M_ lie in A_qk's all-zero blocks (query rows
// 0..31, keys 32..63: blocks 1 and 3 of its first slice), which the intra-chunk
// kernel does not write and the output products never read (the map pass
// stages no A_qk: there E_Q is the first slice after Y)
#define GDR2_OP_ZERO(M_) (C::SZ_A > 0 && (M_) == E_Q && (tid & 128) != 0)
  static_assert(SLICE == 4 * 2048, "a staging slice is four 2 KB fragment blocks: thread t moves block t / 128");
// operand slices [M0, M1) of chunk CHX (the slices a step's products do not read are skipped)
#define GDR2_LOAD_OPS(CHX, M0, M1)                                                                           \
  _Pragma("unroll") for (int m = (M0); m < (M1) && m < NSTG; ++m) {                                      \
    if (!GDR2_OP_USED(m) || GDR2_OP_ZERO(m)) continue;                                                   \
    const unsigned char* src;                                                                            \
    if (m < E_Y)                                                                                         \
      src = a.Y + (CHX) * C::SZ_Y + m * SLICE;                                                           \
    else if (m < E_Q)                                                                                    \
      src = a.Qg + (CHX) * C::SZ_Q + (m - E_Y) * SLICE;                                                  \
    else if (m < E_A)                                                                                    \
      src = a.Aqk + (CHX) * C::SZ_A + (m - E_Q) * SLICE;                                                 \
    else                                                                                                 \
      src = a.KtT + (CHX) * C::SZ_K + (m - E_A) * SLICE;                                                 \
    stg[m] = ldg16(src + 16 * tid);                                                                      \
  }
#define GDR2_STORE_OPS()                                                                                     \
  _Pragma("unroll") for (int m = 0; m < NSTG; ++m) if (GDR2_OP_USED(m) && !GDR2_OP_ZERO(m)) sts16(sOp + m * SLICE + 16 * tid, stg[m]);
  // U tiles (value blocks vbO.., row block iO) and gamma_C rows of the state tiles
#define GDR2_LOAD_UG(CHX, CHKX, UARR, GARR)                                                                  \
  _Pragma("unroll") for (int t = 0; t < NVB / 2; ++t) {                                                  \
    const int vb_ = v0 / 16 + vbO + t;                                                                   \
    UARR[t] = no_input ? f4zero()                                                                        \
                       : *reinterpret_cast<const f4*>(a.U + (CHX) * (WsBf16::u(DV) / 4) +                \
                                                      ((size_t)(vb_ * 4 + iO) * 64 + lane) * 4);         \
  }                                                                                                      \
  _Pragma("unroll") for (int u2 = 0; u2 < 4; ++u2) GARR[u2] =                                            \
      a.GC[(CHKX) * (WsBf16::gc(DK) / 4) + 16 * cs + 4 * g + u2];

  // ---- state: identity columns, the given segment start, S0 (first segment) or zero
  const bool eye = MAP ? slice == 1 : (a.flags & kScanEye) != 0;  // (DV == DK)
  const float* init = eye ? nullptr
                          : (a.S0seg ? a.S0seg + (size_t)vs * DK * DV
                                     : ((a.S0 && seg == 0) ? a.S0 + (size_t)seq * DK * DV : nullptr));
  f4 sreg[TPW];
  if (init) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) sreg[t][u] = init[(size_t)(16 * cs + 4 * g + u) * DV + v0 + 16 * (sv0 + t) + r16];
  } else {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) sreg[t][u] = (eye && 16 * cs + 4 * g + u == v0 + 16 * (sv0 + t) + r16) ? 1.f : 0.f;
  }
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int vb = sv0 + t;
    const int so = MAP ? map_s_ix<LSS>(16 * vb + r16, 16 * cs + 4 * g) : (16 * vb + r16) * LSS + 16 * cs + 4 * g;
    st4split(sShi + so, sSlo + so, sreg[t]);
  }
  if (n0 < n1) {
    GDR2_LOAD_OPS(chk + n0, 0, NSTG)
    GDR2_LOAD_UG(chs + n0, chk + n0, ucur, gcur)
    GDR2_STORE_OPS()
  }
  __syncthreads();

  // K_tail^T blocks of the wave's key block (KD), one chunk ahead
  u4v kreg[4];
  if constexpr (C::KD) {
    if (n0 < n1) {
      const unsigned char* kp = a.KtT + (chk + n0) * C::SZ_K + cs * 2 * 2048 + 16 * lane;
#pragma unroll
      for (int q = 0; q < 4; ++q) kreg[q] = ldg16(kp + 1024 * q);
    }
  }
  for (int n = n0; n < n1; ++n) {
    const size_t ch = chs + n;
    // the next chunk's operands, fetched in groups over the step (the first
    // here, the others after R, inside the output products and after them):
    // all at once, the second wave of each SIMD waits behind the first one's
    // loads before it can start its products.  One vmcnt counts loads and
    // stores in issue order, so waiting for these also waits for every store
    // issued before them; this step's stores (R, O, h) come after the last group.
    // The last step loads its own chunk again (unused): with the same loads
    // issued on every path the compiler counts them exactly, and the state
    // update waits for its K_tail^T fragments alone, not for every load since
    const bool more = n + 1 < n1;
    const int nn = more ? n + 1 : n;
    GDR2_LOAD_OPS(chk + nn, 0, 3)
    GDR2_LOAD_UG(chs + nn, chk + nn, unext, gnext)

    // scale exponents of this chunk-start state's fp16 copy, early in the step
    // so that their cross-lane reductions overlap the products below
    int hsh[TPW / 2];
    if constexpr (STORE_H) state_shifts<TPW>(sreg, hsh);

    // ---- R = U - Y S
    f4 racc[NVB / 2];
    int rsh[1] = {0};
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) racc[t] = ucur[t];
#pragma unroll
    for (int p = 0; p < KS; ++p) {
      const bf8 yf = neg8(ld8(reinterpret_cast<const __bf16*>(sY + (iO * KS + p) * 1024 + 16 * lane)));
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const int vb = vbO + t;
        if constexpr (MAP) {
          const int sf = map_s_frag<LSS>(16 * vb + r16, p, g);
          racc[t] = mma(yf, ld8(sShi + sf), racc[t]);
          racc[t] = mma(yf, ld8(sSlo + sf), racc[t]);
        } else {
          racc[t] = mma(yf, ld_perm8(sShi + (16 * vb + r16) * LSS, 32 * p, g), racc[t]);
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) {
      const int vb = vbO + t;
      st4split(sRhi + (16 * vb + r16) * LR + 16 * iO + 4 * g, sRlo + (16 * vb + r16) * LR + 16 * iO + 4 * g,
               racc[t]);
    }
    // the fp16 copy's scale, taken here so its reduction overlaps the output products
    if constexpr (STORE_H) state_shifts<NVB / 2>(racc, rsh);
    GDR2_LOAD_OPS(chk + nn, 3, WITH_O ? 6 : 10)
    __syncthreads();

    // ---- O^T = S^T Q_g^T + R^T A_qk^T  (lane: O[16 iO + r16][16 vb + 4 g + u]);
    //      each K-step's fragments are read from LDS one step ahead
    if constexpr (WITH_O) {
      f4 accO[NVB / 2];
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) accO[t] = f4zero();
      constexpr int NKO = KS + 2;  // K-steps: KS over keys (S^T Q_g^T), then 2 over rows (R^T A_qk^T)
      Fr fa[2], fb[2][NVB / 2];
#define GDR2_O_FRAGS(P_, BUF_)                                                                            \
  {                                                                                                       \
    if ((P_) < KS) {                                                                                      \
      fa[BUF_].hi = ld8(reinterpret_cast<const __bf16*>(sQ + (iO * KS + (P_)) * 2048 + 16 * lane));      \
      fa[BUF_].lo = ld8(reinterpret_cast<const __bf16*>(sQ + (iO * KS + (P_)) * 2048 + 1024 + 16 * lane)); \
      _Pragma("unroll") for (int t = 0; t < NVB / 2; ++t) {                                               \
        const int vb = vbO + t;                                                                           \
        fb[BUF_][t].hi = ld8(sShi + (16 * vb + r16) * LSS + 32 * (P_) + 8 * g);                          \
        fb[BUF_][t].lo = ld8(sSlo + (16 * vb + r16) * LSS + 32 * (P_) + 8 * g);                          \
      }                                                                                                   \
    } else {                                                                                              \
      const int kb_ = (P_) - KS;                                                                          \
      fa[BUF_].hi = ld8(reinterpret_cast<const __bf16*>(sA + (iO * 2 + kb_) * 2048 + 16 * lane));        \
      fa[BUF_].lo = ld8(reinterpret_cast<const __bf16*>(sA + (iO * 2 + kb_) * 2048 + 1024 + 16 * lane)); \
      _Pragma("unroll") for (int t = 0; t < NVB / 2; ++t) {                                               \
        const int vb = vbO + t;                                                                           \
        fb[BUF_][t].hi = ld_perm8(sRhi + (16 * vb + r16) * LR, 32 * kb_, g);                             \
        fb[BUF_][t].lo = ld_perm8(sRlo + (16 * vb + r16) * LR, 32 * kb_, g);                             \
      }                                                                                                   \
    }                                                                                                     \
  }
      GDR2_O_FRAGS(0, 0)
#pragma unroll
      for (int p = 0; p < NKO; ++p) {
        // K-steps over rows r < 16 iO of A_qk^T are zero (causal): skip them
        const bool live = p < KS || (p - KS) <= (iO >> 1);
        const bool next = p + 1 < NKO && (p + 1 < KS || (p + 1 - KS) <= (iO >> 1));
        if (next) GDR2_O_FRAGS(p + 1, (p + 1) & 1)
        if (p == 1) GDR2_LOAD_OPS(chk + nn, 6, 8)
        if (p == 3) GDR2_LOAD_OPS(chk + nn, 8, 10)
        if (live) {
#pragma unroll
          for (int t = 0; t < NVB / 2; ++t) accO[t] = mma3(fb[p & 1][t], fa[p & 1], accO[t]);
        }
      }
#undef GDR2_O_FRAGS
      const float sc = a.scale;
      size_t orow;
      int olen;
      scan_rows(a.vl, seq, H, T, n, orow, olen);
      if (16 * iO + r16 < olen) {
        __bf16* orp = O + (orow + 16 * iO + r16) * ((size_t)H * DV) + (size_t)h * DV + v0;
#pragma unroll
        for (int t = 0; t < NVB / 2; ++t)
          st4(orp + 16 * (vbO + t) + 4 * g, sc * accO[t][0], sc * accO[t][1], sc * accO[t][2], sc * accO[t][3]);
      }
    }

    GDR2_LOAD_OPS(chk + nn, 10, NSTG)
    // ---- S <- Diag(gamma_C) S + Ktail^T R
    if constexpr (STORE_H) {
      // the chunk-start state for the backward, fp16 with its block scales
      // (from a copy: the state registers change right below)
      f4 hcopy[TPW];
#pragma unroll
      for (int t = 0; t < TPW; ++t) hcopy[t] = sreg[t];
      const int col0 = v0 + 16 * sv0;
      store_state_f16<TPW>(hcopy, hsh, a.Hs + (ch * DK + 16 * cs) * DV + col0, DV,
                           a.Hsc + ch * (WsBf16::hsc(DK, DV) / 4) + cs * (DV / 32) + col0 / 32, lane);
    }
    {
      if constexpr (MAP) {
        // the full-width map: R fragments one key-row block at a time
#pragma unroll
        for (int t = 0; t < TPW; ++t)
#pragma unroll
          for (int u = 0; u < 4; ++u) sreg[t][u] *= gcur[u];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          Fr kf, rf[TPW];
          if constexpr (C::KD) {
            kf.hi = __builtin_bit_cast(bf8, kreg[2 * kb]);
            kf.lo = __builtin_bit_cast(bf8, kreg[2 * kb + 1]);
          } else {
            kf.hi = ld8(reinterpret_cast<const __bf16*>(sK + (cs * 2 + kb) * 2048 + 16 * lane));
            kf.lo = ld8(reinterpret_cast<const __bf16*>(sK + (cs * 2 + kb) * 2048 + 1024 + 16 * lane));
          }
#pragma unroll
          for (int t = 0; t < TPW; ++t) {
            const int vb = sv0 + t;
            rf[t].hi = ld8(sRhi + (16 * vb + r16) * LR + 32 * kb + 8 * g);
            rf[t].lo = ld8(sRlo + (16 * vb + r16) * LR + 32 * kb + 8 * g);
          }
#pragma unroll
          for (int t = 0; t < TPW; ++t) sreg[t] = mma3(kf, rf[t], sreg[t]);
        }
      } else {
        Fr kf[2], rfs[2][TPW];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          if constexpr (C::KD) {
            kf[kb].hi = __builtin_bit_cast(bf8, kreg[2 * kb]);
            kf[kb].lo = __builtin_bit_cast(bf8, kreg[2 * kb + 1]);
          } else {
            kf[kb].hi = ld8(reinterpret_cast<const __bf16*>(sK + (cs * 2 + kb) * 2048 + 16 * lane));
            kf[kb].lo = ld8(reinterpret_cast<const __bf16*>(sK + (cs * 2 + kb) * 2048 + 1024 + 16 * lane));
          }
#pragma unroll
          for (int t = 0; t < TPW; ++t) {
            const int vb = sv0 + t;
            rfs[kb][t].hi = ld8(sRhi + (16 * vb + r16) * LR + 32 * kb + 8 * g);
            rfs[kb][t].lo = ld8(sRlo + (16 * vb + r16) * LR + 32 * kb + 8 * g);
          }
        }
#pragma unroll
        for (int t = 0; t < TPW; ++t)
#pragma unroll
          for (int u = 0; u < 4; ++u) sreg[t][u] *= gcur[u];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int t = 0; t < TPW; ++t) sreg[t] = mma3(kf[kb], rfs[kb][t], sreg[t]);
      }
    }
    if constexpr (C::KD) {
      const unsigned char* kp = a.KtT + (chk + nn) * C::SZ_K + cs * 2 * 2048 + 16 * lane;
#pragma unroll
      for (int q = 0; q < 4; ++q) kreg[q] = ldg16(kp + 1024 * q);
    }
    if constexpr (STORE_H) {
      // R for the backward: this wave's 16 x 32 tile as one fp16 fragment block
      static_assert(NVB / 2 == 2, "one 32-column block per wave");
      const int vblk = (v0 + 16 * vbO) / 32;
      const size_t blk = (size_t)ch * (WsBf16::rs(DV) / 1024) + (size_t)iO * (DV / 32) + vblk;
      store_frag_f16(racc, rsh[0], a.Rs + blk * 512, lane);
      if (lane == 0) a.Rsc[blk] = ldexpf(1.f, -rsh[0]);
    }
    __syncthreads();

    // ---- new S and the next chunk's operands to LDS
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int vb = sv0 + t;
      const int so = MAP ? map_s_ix<LSS>(16 * vb + r16, 16 * cs + 4 * g) : (16 * vb + r16) * LSS + 16 * cs + 4 * g;
      st4split(sShi + so, sSlo + so, sreg[t]);
    }
    if (more) {
      GDR2_STORE_OPS()
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) ucur[t] = unext[t];
#pragma unroll
      for (int u = 0; u < 4; ++u) gcur[u] = gnext[u];
    }
    __syncthreads();
  }

#undef GDR2_LOAD_OPS
#undef GDR2_STORE_OPS
#undef GDR2_OP_USED
#undef GDR2_OP_ZERO
#undef GDR2_LOAD_UG
  float* send = MAP ? (slice == 0 ? a.STseg : a.STseg_m) + (size_t)vs * DK * DV
                    : (a.STseg ? a.STseg + (size_t)vs * DK * DV
                               : ((a.ST && seg == nseg - 1) ? a.ST + (size_t)seq * DK * DV : nullptr));
  if (send) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) send[(size_t)(16 * cs + 4 * g + u) * DV + v0 + 16 * (sv0 + t) + r16] = sreg[t][u];
  }
}

template <int DK, int DV, bool WITH_O, bool STORE_H, bool MAP>
hipError_t launch_scan_bf16_t(const ScanArgs& a, hipStream_t st) {
  using C = ScanCfg2<DK, DV, MAP>;
  const void* fn = reinterpret_cast<const void*>(&scan_bf16_kernel<DK, DV, WITH_O, STORE_H, MAP>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  dim3 grid(a.B * a.H * a.nseg * C::NS);
  hipLaunchKernelGGL((scan_bf16_kernel<DK, DV, WITH_O, STORE_H, MAP>), grid, dim3(C::NTHR), C::LDS, st, a);
  return hipGetLastError();
}

template <int DK, int DV, bool WITH_O, bool STORE_H>
hipError_t launch_scan_bf16(const ScanArgs& a, hipStream_t st) {
  return launch_scan_bf16_t<DK, DV, WITH_O, STORE_H, false>(a, st);
}

template <int D>
hipError_t launch_scan_map_bf16(const ScanArgs& a, hipStream_t st) {
  return launch_scan_bf16_t<D, D, false, false, true>(a, st);
}
template hipError_t launch_scan_map_bf16<64>(const ScanArgs&, hipStream_t);
template hipError_t launch_scan_map_bf16<128>(const ScanArgs&, hipStream_t);

#define GDR2_INST_SCAN2(DK, DV)                                                          \
  template hipError_t launch_scan_bf16<DK, DV, true, false>(const ScanArgs&, hipStream_t); \
  template hipError_t launch_scan_bf16<DK, DV, false, true>(const ScanArgs&, hipStream_t); \
  template hipError_t launch_scan_bf16<DK, DV, true, true>(const ScanArgs&, hipStream_t);

// transition-matrix passes of the sequence-parallel scan (value width = Dk)
template hipError_t launch_scan_bf16<64, 64, false, false>(const ScanArgs&, hipStream_t);
template hipError_t launch_scan_bf16<128, 128, false, false>(const ScanArgs&, hipStream_t);
template hipError_t launch_scan_bf16<64, 128, false, false>(const ScanArgs&, hipStream_t);
template hipError_t launch_scan_bf16<128, 64, false, false>(const ScanArgs&, hipStream_t);

GDR2_INST_SCAN2(64, 64)
GDR2_INST_SCAN2(64, 128)
GDR2_INST_SCAN2(128, 64)
GDR2_INST_SCAN2(128, 128)

}  // namespace gdr2

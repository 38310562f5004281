// Reverse inter-chunk scan of the bf16 backward (gfx950), App. B.1: one
// 8-wave workgroup per (sequence, head, 64-wide value slice) walks the chunks
// from last to first, carrying dS (the gradient of the chunk's end state):
//
//   dR  = scale * A_qk^T dO + Ktail dS
//   dS <- Diag(gamma_C) dS + scale * Q_g^T dO - Y^T dR
//
// writing dS before each update (the gradient of that chunk's end state, fp16
// with block scales as store_state_f16 keeps it for the chunk backward), dR
// (split bf16 16 x 16 blocks), and finally dS0.
// With nseg > 1 each workgroup runs one segment of a sequence, from the
// gradient at the segment's end to the one at its start (BScanArgs).  The operands are the forward's fragment-ordered tiles
// (gdr2_kernels.hpp): the transposed fragments these products need come out
// of the same LDS blocks through ds_read_b64_tr_b16 with per-lane addresses,
// since every 4 consecutive elements of a block row are contiguous.  A
// chunk's blocks are fetched into one of two register buffers in six groups
// over the step two steps before the one that computes it, settled before
// the dR stores of the step in between (so that no later wait for them also
// waits for those stores) and copied to LDS at its end.  The passes that write
// dh and dR and those that do not (the segment maps) are separate kernels,
// and the dO rows come through a range-checked buffer load, so that every
// path issues the same loads and stores.
//
// Precision: every product is fp32-accurate (split hi/lo; dO and Y are exact
// bf16 and keep a single part).

#include "gdr2_kernels.hpp"
#include "gdr2_bf16.hpp"

namespace gdr2 {

template <int DK, int DV>
struct BScanCfg {
  static constexpr int NTHR = 512;
  static constexpr int DVS = DV < 64 ? DV : 64;
  static constexpr int NS = DV / DVS;
  static constexpr int KS = DK / 32, NCB = DK / 16, NVB = DVS / 16;
  static constexpr int TPW = NCB * NVB / 8;
  static constexpr int LSD = DK + 8;   // dS hi/lo [DVS][LSD]
  static constexpr int LDR = 64 + 8;   // dR hi/lo [DVS][LDR]
  static constexpr int LDO = DVS + 8;  // dO [64][LDO]
  static constexpr int SZ_Y = (int)WsBf16::y(DK), SZ_Q = (int)WsBf16::qg(DK);
  static constexpr int SZ_A = (int)WsBf16::aqk(), SZ_K = (int)WsBf16::ktt(DK);
  static constexpr int SZ_OP = SZ_Y + SZ_Q + SZ_A + SZ_K;
  static constexpr int SLICE = 16 * NTHR;
  static constexpr int NSTG = SZ_OP / SLICE;
  static constexpr int OFF_D = 0;
  static constexpr int OFF_R = OFF_D + 2 * DVS * LSD * 2;
  static constexpr int OFF_O = OFF_R + 2 * DVS * LDR * 2;
  static constexpr int OFF_OP = OFF_O + 64 * LDO * 2;
  static constexpr int LDS = OFF_OP + SZ_OP;
  static_assert(SZ_Y % SLICE == 0 && SZ_Q % SLICE == 0 && SZ_A % SLICE == 0 && SZ_K % SLICE == 0,
                "regions are whole staging slices");
  static_assert(64 * DVS * 2 == SLICE, "one dO chunk per thread");
  static_assert(LDS <= 160 * 1024, "LDS budget");
  static_assert(TPW >= 1 && NVB % 2 == 0, "wave split");
};

// STORE_D: the pass writes dh and dR (both set; the segment-map passes write neither)
template <int DK, int DV, bool STORE_D>
__global__ __launch_bounds__(512) void bscan_bf16_kernel(BScanArgs a) {
  using C = BScanCfg<DK, DV>;
  constexpr int DVS = C::DVS, NS = C::NS, KS = C::KS, NCB = C::NCB, NVB = C::NVB, TPW = C::TPW;
  constexpr int LSD = C::LSD, LDR = C::LDR, LDO = C::LDO, NSTG = C::NSTG, SLICE = C::SLICE;
  constexpr int E_Y = C::SZ_Y / SLICE, E_Q = E_Y + C::SZ_Q / SLICE, E_A = E_Q + C::SZ_A / SLICE;

  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* sDhi = reinterpret_cast<__bf16*>(smem + C::OFF_D);
  __bf16* sDlo = sDhi + DVS * LSD;
  __bf16* sRhi = reinterpret_cast<__bf16*>(smem + C::OFF_R);
  __bf16* sRlo = sRhi + DVS * LDR;
  __bf16* sdO = reinterpret_cast<__bf16*>(smem + C::OFF_O);
  unsigned char* sOp = smem + C::OFF_OP;
  const unsigned char* sY = sOp;
  const unsigned char* sQ = sY + C::SZ_Y;
  const unsigned char* sA = sQ + C::SZ_Q;
  const unsigned char* sK = sA + C::SZ_A;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  const int qq = r16 & 3, ii = r16 >> 2;  // transpose-load role of this lane (4 ii + qq)
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
  const bool no_input = (a.flags & kScanNoInput) != 0;
  const int h = seq % H;
  const int v0 = slice * DVS;
  const __bf16* dO = reinterpret_cast<const __bf16*>(a.dout);

  const int iO = wave >> 1;                // row block of the dR tiles
  const int vbO = (wave & 1) * (NVB / 2);  // their value blocks
  const int cs = wave % NCB;               // key block of the dS tiles
  const int sv0 = (wave / NCB) * TPW;      // their value blocks

  // ---- staging: operand blocks, the dO slice and gamma_C of a chunk, in two
  // register buffers (A, B): a chunk's values are fetched over the step two
  // steps before the one that computes it and copied to LDS at the end of the
  // step in between, so every load has a whole step to arrive
  u4v stgA[NSTG], stoA, stgB[NSTG], stoB;
  float gcur[4], gA[4], gB[4];
  static_assert(SLICE == 4 * 2048, "a staging slice is four 2 KB fragment blocks: thread t moves block t / 128");
  const size_t chs = rng.chs;                        // value-head chunks: dh, dR
  const size_t chk = key_ch(a.vl, chs, H, a.G, NT);  // key-head chunks: Y, Q_g, A_qk, K_tail, gamma_C
#define GDR2_LOAD_CHUNK(N_, STG, STO, GN)                                                                 \
  {                                                                                                    \
    GDR2_LOAD_OPS(N_, 0, NSTG, STG)                                                                    \
    GDR2_LOAD_DOG(N_, STO, GN)                                                                         \
  }
// operand slices [M0, M1) of chunk N_
#define GDR2_LOAD_OPS(N_, M0, M1, STG)                                                                    \
  {                                                                                                    \
    const size_t chx = chk + (N_);                                                                     \
    _Pragma("unroll") for (int m = (M0); m < (M1) && m < NSTG; ++m) {                                  \
      /* (without dO, Q_g and A_qk are loaded all the same, but not staged) */                      \
      if (m == E_Q && (tid & 128) != 0) continue;    /* A_qk's all-zero blocks: not stored */         \
      const unsigned char* src;                                                                        \
      if (m < E_Y)                                                                                     \
        src = a.Y + chx * C::SZ_Y + m * SLICE;                                                         \
      else if (m < E_Q)                                                                                \
        src = a.Qg + chx * C::SZ_Q + (m - E_Y) * SLICE;                                                \
      else if (m < E_A)                                                                                \
        src = a.Aqk + chx * C::SZ_A + (m - E_Q) * SLICE;                                               \
      else                                                                                             \
        src = a.KtT + chx * C::SZ_K + (m - E_A) * SLICE;                                               \
      STG[m] = ldg16(src + 16 * tid);                                                                  \
    }                                                                                                  \
  }
// chunk N_'s dO slice and gamma_C
#define GDR2_LOAD_DOG(N_, STO, GN)                                                                        \
  {                                                                                                    \
    const size_t chx = chk + (N_);                                                                     \
    const int r_ = tid / (DVS / 8), c8_ = (tid % (DVS / 8)) * 8;                                       \
    size_t orow_;                                                                                      \
    int olen_;                                                                                         \
    scan_rows(a.vl, seq, H, T, (N_), orow_, olen_);                                                    \
    /* through a buffer whose range ends with the chunk's last row (empty       */                  \
    /* without dO): rows past it read as zero, with no branch around the load  */                  \
    const unsigned pitch_ = (unsigned)(H * DV) * 2u;                                                   \
    const __amdgpu_buffer_rsrc_t orsrc_ = __builtin_amdgcn_make_buffer_rsrc(                          \
        no_input ? (void*)a.GC : (void*)(dO + orow_ * ((size_t)H * DV) + (size_t)h * DV + v0), 0,      \
        no_input ? 0u : (unsigned)(olen_ - 1) * pitch_ + DVS * 2, 0x00020000);                         \
    STO = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(                              \
        orsrc_, (unsigned)r_ * pitch_ + c8_ * 2, 0, 0));                                               \
    _Pragma("unroll") for (int u2 = 0; u2 < 4; ++u2) GN[u2] =                                          \
        a.GC[chx * (WsBf16::gc(DK) / 4) + 16 * cs + 4 * g + u2];                                       \
  }
#define GDR2_STORE_CHUNK(STG, STO, GN)                                                                   \
  {                                                                                                    \
    _Pragma("unroll") for (int m = 0; m < NSTG; ++m)                                                   \
        if ((!no_input || m < E_Y || m >= E_A) && (m != E_Q || (tid & 128) == 0))                       \
          sts16(sOp + m * SLICE + 16 * tid, STG[m]);                                                   \
    const int r_ = tid / (DVS / 8), c8_ = (tid % (DVS / 8)) * 8;                                       \
    sts16(sdO + r_ * LDO + c8_, STO);                                                                  \
    _Pragma("unroll") for (int u2 = 0; u2 < 4; ++u2) gcur[u2] = GN[u2];                                \
  }

  // ---- dS: tiles (key block cs, value blocks sv0..) as fp32 accumulators, starting
  // from identity columns, the given segment end, dS_T (last segment) or zero
  const bool eye = (a.flags & kScanEye) != 0;  // (DV == DK)
  const float* init = eye ? nullptr
                          : (a.dSseg_in ? a.dSseg_in + (size_t)vs * DK * DV
                                        : ((a.dST && seg == nseg - 1) ? a.dST + (size_t)seq * DK * DV : nullptr));
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
    st4split(sDhi + (16 * vb + r16) * LSD + 16 * cs + 4 * g, sDlo + (16 * vb + r16) * LSD + 16 * cs + 4 * g,
             sreg[t]);
  }
  if (n0 < n1) {
    // the last chunk into B and the one before it (or the first chunk again,
    // unused) into A; B goes to LDS, and A is settled here so that the loop
    // starts with no load pending (otherwise the registers the two paths into
    // the loop give the buffers differ, and the loop top waits for stale loads)
    GDR2_LOAD_CHUNK(n1 - 1, stgB, stoB, gB)
    GDR2_LOAD_CHUNK(max(n1 - 2, n0), stgA, stoA, gA)
    GDR2_STORE_CHUNK(stgB, stoB, gB)
#pragma unroll
    for (int m = 0; m < NSTG; ++m) asm volatile("" : "+v"(stgA[m])::"memory");
    asm volatile("" : "+v"(stoA)::"memory");
#pragma unroll
    for (int u = 0; u < 4; ++u) asm volatile("" : "+v"(gA[u])::"memory");
  }
  __syncthreads();

  // one step: chunk n is in LDS, chunk n - 1 in the buffer (cstg, csto, cg),
  // chunk n - 2 is fetched into the other one (nstg, nsto, ng)
  auto step = [&](const int n, u4v(&cstg)[NSTG], u4v& csto, float(&cg)[4], u4v(&nstg)[NSTG], u4v& nsto,
                  float(&ng)[4]) {
    const size_t ch = chs + n;
    // chunk n - 2's loads in six groups of two slices over the step (here,
    // inside the Ktail dS product, before and after the A_qk^T dO product, and
    // at the two K-steps of the dS update): issued all at once, the second
    // wave of each SIMD waits behind the first one's loads before it can start
    // its products.  The last two steps load the first chunk again (unused),
    // so that the same loads are issued on every path
    const int nn = max(n - 2, n0);
    GDR2_LOAD_OPS(nn, 0, 2, nstg)
    GDR2_LOAD_DOG(nn, nsto, ng)

    // scale exponents of the fp16 copy of dS, early in the step so that their
    // cross-lane reductions overlap the products below
    int dsh[TPW / 2];
    if constexpr (STORE_D) state_shifts<TPW>(sreg, dsh);

    // ---- dR = scale * A_qk^T dO + Ktail dS   (tiles: row block iO, value blocks vbO..)
    f4 racc[NVB / 2], aacc[NVB / 2];
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) {
      racc[t] = f4zero();
      aacc[t] = f4zero();
    }
#pragma unroll
    for (int p = 0; p < KS; ++p) {
      // Ktail[r][c], r = 16 iO + r16, c = 32 p + 8 g + e, from the Ktail^T blocks
      Fr kf;
      {
        const int c0 = 32 * p + 8 * g + ii;
        const int boff = ((c0 >> 4) * 2 + (iO >> 1)) * 2048 +
                         ((c0 & 15) + 16 * (2 * (iO & 1) + (qq >> 1))) * 16 + 8 * (qq & 1);
        const __bf16* p0 = reinterpret_cast<const __bf16*>(sK + boff);
        kf.hi = ld_tr8p(p0, p0 + 32);  // +4 rows of c = +4 lanes = 64 bytes
        kf.lo = ld_tr8p(p0 + 512, p0 + 512 + 32);
      }
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const int vb = vbO + t;
        Fr df;
        df.hi = ld8(sDhi + (16 * vb + r16) * LSD + 32 * p + 8 * g);
        df.lo = ld8(sDlo + (16 * vb + r16) * LSD + 32 * p + 8 * g);
        racc[t] = mma3(kf, df, racc[t]);
      }
      if (p == 1) GDR2_LOAD_OPS(nn, 2, 4, nstg)
    }
    GDR2_LOAD_OPS(nn, 4, 6, nstg)
    // (without dO the A_qk and Q_g products vanish: their tiles are not even loaded)
#pragma unroll
    for (int kb = (iO >> 1); kb < 2 && !no_input; ++kb) {
      // A_qk[i][j], i = 32 kb + 8 g + e (query), j = 16 iO + r16 (key)
      Fr af;
      {
        const int i0 = 32 * kb + 8 * g + ii;
        const int boff = ((i0 >> 4) * 2 + (iO >> 1)) * 2048 + (16 * qq + (i0 & 15)) * 16 + 8 * (iO & 1);
        const __bf16* p0 = reinterpret_cast<const __bf16*>(sA + boff);
        af.hi = ld_tr8p(p0, p0 + 32);  // +4 query rows = +4 lanes
        af.lo = ld_tr8p(p0 + 512, p0 + 512 + 32);
      }
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const int vb = vbO + t;
        aacc[t] = mma2a(af, ld_tr8(sdO, LDO, 32 * kb, 16 * vb, lane), aacc[t]);
      }
    }
    GDR2_LOAD_OPS(nn, 6, 8, nstg)
    // gradient of this chunk's end state (sreg is not updated before the barrier below)
    if constexpr (STORE_D) {
      const int col0 = v0 + 16 * sv0;
      store_state_f16<TPW>(sreg, dsh, a.DH + (ch * DK + 16 * cs) * DV + col0, DV,
                           a.DHsc + ch * (WsBf16::hsc(DK, DV) / 4) + cs * (DV / 32) + col0 / 32, lane);
    }
    const float sc = a.scale;
    f4 rkeep[NVB / 2];
#pragma unroll
    for (int t = 0; t < NVB / 2; ++t) {
      const int vb = vbO + t;
#pragma unroll
      for (int u = 0; u < 4; ++u) rkeep[t][u] = racc[t][u] + sc * aacc[t][u];
      st4split(sRhi + (16 * vb + r16) * LDR + 16 * iO + 4 * g, sRlo + (16 * vb + r16) * LDR + 16 * iO + 4 * g,
               rkeep[t]);
    }
    __syncthreads();

    // ---- dS <- Diag(gamma_C) dS + scale * Q_g^T dO - Y^T dR
    GDR2_LOAD_OPS(nn, 8, 10, nstg)
    f4 qacc[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) qacc[t] = f4zero();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if (kb == 1) GDR2_LOAD_OPS(nn, 10, NSTG, nstg)
      // Q_g[r][c], r = 32 kb + 8 g + e, c = 16 cs + r16
      Fr qf;
      bf8 yf;
      {
        const int r0 = 32 * kb + 8 * g + ii;
        const int qoff = ((r0 >> 4) * KS + (cs >> 1)) * 2048 + ((r0 & 15) + 16 * (2 * (cs & 1) + (qq >> 1))) * 16 +
                         8 * (qq & 1);
        const __bf16* p0 = reinterpret_cast<const __bf16*>(sQ + qoff);
        qf.hi = ld_tr8p(p0, p0 + 32);  // +4 rows of r = +4 lanes
        qf.lo = ld_tr8p(p0 + 512, p0 + 512 + 32);
        const int yoff = ((r0 >> 4) * KS + (cs >> 1)) * 1024 + (16 * qq + (r0 & 15)) * 16 + 8 * (cs & 1);
        const __bf16* y0 = reinterpret_cast<const __bf16*>(sY + yoff);
        yf = neg8(ld_tr8p(y0, y0 + 32));
      }
      if (!no_input) {
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
          const int vb = sv0 + t;
          qacc[t] = mma2a(qf, ld_tr8(sdO, LDO, 32 * kb, 16 * vb, lane), qacc[t]);
        }
      }
      if (kb == 0) {
#pragma unroll
        for (int t = 0; t < TPW; ++t)
#pragma unroll
          for (int u = 0; u < 4; ++u) sreg[t][u] *= gcur[u];
      }
#pragma unroll
      for (int t = 0; t < TPW; ++t) {
        const int vb = sv0 + t;
        Fr rf;
        rf.hi = ld8(sRhi + (16 * vb + r16) * LDR + 32 * kb + 8 * g);
        rf.lo = ld8(sRlo + (16 * vb + r16) * LDR + 32 * kb + 8 * g);
        sreg[t] = mma2b(yf, rf, sreg[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u) sreg[t][u] += sc * qacc[t][u];
    // dR for the chunk backward: each of the wave's 16 x 16 tiles (chunk rows
    // 16 iO .., values 16 vb ..) as one split block, lane l's four values
    // (value l % 16, rows 4 (l / 16) + u) at 8 l of the hi and lo halves.  Like
    // the dh stores, these leave after the chunk's products are issued.
    // chunk n - 1's values (fetched over the previous step) have arrived by
    // now: settle them ahead of the dR stores, on every path, so that neither
    // their copy to LDS nor the reuse of their registers waits for those
    // stores (one vmcnt counts loads and stores in issue order)
#pragma unroll
    for (int m = 0; m < NSTG; ++m) asm volatile("" : "+v"(cstg[m])::"memory");
    asm volatile("" : "+v"(csto)::"memory");
#pragma unroll
    for (int u = 0; u < 4; ++u) asm volatile("" : "+v"(cg[u])::"memory");
    if constexpr (STORE_D) {
#pragma unroll
      for (int t = 0; t < NVB / 2; ++t) {
        const size_t blk = ch * (WsBf16::dr(DV) / 1024) + (size_t)(v0 / 16 + vbO + t) * 4 + iO;
        st4split(a.DR + blk * 512 + 4 * lane, a.DR + blk * 512 + 256 + 4 * lane, rkeep[t]);
      }
    }
    __syncthreads();

#pragma unroll
    for (int t = 0; t < TPW; ++t) {
      const int vb = sv0 + t;
      st4split(sDhi + (16 * vb + r16) * LSD + 16 * cs + 4 * g, sDlo + (16 * vb + r16) * LSD + 16 * cs + 4 * g,
               sreg[t]);
    }
    if (n > n0) GDR2_STORE_CHUNK(cstg, csto, cg)
    __syncthreads();
  };
  // two steps per trip, so that the buffers trade roles without copies
  for (int n = n1 - 1; n >= n0; n -= 2) {
    step(n, stgA, stoA, gA, stgB, stoB, gB);
    if (n - 1 >= n0) step(n - 1, stgB, stoB, gB, stgA, stoA, gA);
  }
#undef GDR2_LOAD_CHUNK
#undef GDR2_LOAD_OPS
#undef GDR2_LOAD_DOG
#undef GDR2_STORE_CHUNK

  float* dstart = a.dSseg_out ? a.dSseg_out + (size_t)vs * DK * DV
                              : ((a.dS0 && seg == 0) ? a.dS0 + (size_t)seq * DK * DV : nullptr);
  if (dstart) {
#pragma unroll
    for (int t = 0; t < TPW; ++t)
#pragma unroll
      for (int u = 0; u < 4; ++u)
        dstart[(size_t)(16 * cs + 4 * g + u) * DV + v0 + 16 * (sv0 + t) + r16] = sreg[t][u];
  }
}

template <int DK, int DV, bool STORE_D>
hipError_t launch_bscan_bf16_t(const BScanArgs& a, hipStream_t st) {
  using C = BScanCfg<DK, DV>;
  const void* fn = reinterpret_cast<const void*>(&bscan_bf16_kernel<DK, DV, STORE_D>);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  dim3 grid(a.B * a.H * a.nseg * C::NS);
  hipLaunchKernelGGL((bscan_bf16_kernel<DK, DV, STORE_D>), grid, dim3(C::NTHR), C::LDS, st, a);
  return hipGetLastError();
}

template <int DK, int DV>
hipError_t launch_bscan_bf16(const BScanArgs& a, hipStream_t st) {
  if ((a.DH == nullptr) != (a.DR == nullptr)) return hipErrorInvalidValue;  // both or neither
  return a.DH ? launch_bscan_bf16_t<DK, DV, true>(a, st) : launch_bscan_bf16_t<DK, DV, false>(a, st);
}

template hipError_t launch_bscan_bf16<64, 64>(const BScanArgs&, hipStream_t);
template hipError_t launch_bscan_bf16<64, 128>(const BScanArgs&, hipStream_t);
template hipError_t launch_bscan_bf16<128, 64>(const BScanArgs&, hipStream_t);
template hipError_t launch_bscan_bf16<128, 128>(const BScanArgs&, hipStream_t);

}  // namespace gdr2

// Sequential inter-chunk state passes (gfx950) of the chunkwise gated delta
// rule (Sec. 3.3; state stored dk x dv).  One workgroup owns one (sequence,
// head, BV-wide slice of dv): the dk x BV state tile lives in the MFMA
// accumulators of its four waves (wave w owns state rows [w dk/4, (w+1) dk/4))
// and the chunks of the sequence are walked in order.  Per chunk the state
// (or its gradient) and the chunk's V' (or dV') are published to LDS as MFMA
// B operands straight from the accumulators (permuted contraction order, one
// 8-byte store per tile and lane); every A operand comes from HBM in
// fragment order (or, for raw q and k, in the same permuted order) and is
// loaded into registers one chunk ahead of its use.  Two barriers per chunk.
//
// Forward, per chunk:   V' = U~ - W~ S,   O = (diag(e^g) Q) S + P V',
//                       S <- e^{g_n} S + Kbar^T V'.
// Backward, per chunk (reverse order), dS = gradient of the exit state:
//                       dV' = P^T dO + diag(e^{g_n - g}) (K dS),
//                       dX = T^T dV',   dv = b dX,
//                       dS <- e^{g_n} dS + (e^g Q)^T dO - W~^T dV'.
#include "gdn_device.h"
#include "gdn_kernels.h"
#include "gdn_seq_common.h"

namespace gdn {


// dv slice per workgroup and the workgroups per CU the register budget is
// sized for.  The forward at dk = 256 takes 64-wide slices: every chunk moves
// about 100 KB of dk-side A operands through each workgroup's vector memory
// path, and a wider slice reuses them over twice the columns.
#ifndef GDN_FWD_BV256
#define GDN_FWD_BV256 64
#endif
#ifndef GDN_SEQ_MINB
#define GDN_SEQ_MINB 2
#endif
#ifndef GDN_SAVE_BV256
#define GDN_SAVE_BV256 32
#endif
#ifndef GDN_SAVE_MINB
#define GDN_SAVE_MINB GDN_SEQ_MINB
#endif
// L2 warm-up distance in chunks (0: none) of each state pass, where it
// measured faster.  The warm-up loads land in LDS; an earlier form that kept
// them in registers was slower wherever both were measured (its results had
// to stay live, and it spilled the reverse pass at dk 256).  At dk 256:
// saving forward 629 -> 548 us (598 through registers; distances 3 to 6
// within 4 us), 524 us when each wave also warms its own U~ tiles; reverse
// pass 645 -> 587 us (distance 2: 626, 3: 596, 5 and 6: 592).  At dk 128:
// reverse pass 736 -> 684 us (709 through registers; distance 4: 699); in
// the saving forward its lines crowd L2 (distance 1: 605 -> 631 us, 3:
// 651 us).  Recompute pass at dk 256: 444 -> 411 us (distance 3: 423).
// Measured and not kept: the plain forward at dk 256 (one round of 64-wide
// slices; within 2% at distances 3 and 4); one load per 64 bytes instead of per
// 128-byte line (slower in both passes: L2 fills whole lines); the reverse
// pass warming its own dO rows (dk 256: within noise; dk 128: 682 -> 743
// us); warming the gates and betas too (within noise); warming the chunks
// before the loop's first warm-up at the start of the workgroup (every
// workgroup starts at once: reverse pass 587 -> 611 us, recompute pass 411
// -> 504 us).
#ifndef GDN_WARM_SAVE
#define GDN_WARM_SAVE 4
#endif
#ifndef GDN_WARM_STORE
#define GDN_WARM_STORE 4
#endif
#ifndef GDN_WARM_FWD
#define GDN_WARM_FWD 0
#endif
#ifndef GDN_WARM_BWD256
#define GDN_WARM_BWD256 4
#endif
#ifndef GDN_WARM_BWD128
#define GDN_WARM_BWD128 3
#endif
#ifndef GDN_WARM_SAVE128
#define GDN_WARM_SAVE128 0
#endif
template <class E, int DK, int DV>
struct SeqCfg {
  static constexpr int BV = 32;
  static constexpr int FWD_BV = DK == 256 ? GDN_FWD_BV256 : 32;
  static constexpr int SAVE_BV = DK == 256 ? GDN_SAVE_BV256 : 32;
  static constexpr int MINB = GDN_SEQ_MINB;
  static constexpr bool B256 = sizeof(E) == 2 && DK == 256;
  static constexpr bool B128 = sizeof(E) == 2 && DK == 128;
  static constexpr int WARM_SAVE = B256 ? GDN_WARM_SAVE : B128 ? GDN_WARM_SAVE128 : 0;
  static constexpr int WARM_STORE = B256 ? GDN_WARM_STORE : 0;
  static constexpr int WARM_FWD = B256 ? GDN_WARM_FWD : 0;
  static constexpr int WARM_BWD = B256 ? GDN_WARM_BWD256 : B128 ? GDN_WARM_BWD128 : 0;
};

// ------------------------------------------------------------------ forward / recompute
// SEQ_FWD  : forward, writes O and ht.
// SEQ_STORE: backward recompute, writes each chunk's entry state and V' (in
//            MFMA fragment order over dv, for the gradient kernel).
// SEQ_SAVE : forward that also keeps what SEQ_STORE writes, for a backward
//            that skips the recompute.

template <class E, int DK, int DV, int MODE>
__global__ __launch_bounds__(256, (MODE == SEQ_SAVE ? GDN_SAVE_MINB : GDN_SEQ_MINB)) void k_fwd_seq(
    Args a) {
  using M = Mfma<E>;
  using frag = typename M::frag;
  using raw4 = typename Raw4<E>::type;
  constexpr bool OUT = MODE != SEQ_STORE, STORE = MODE != SEQ_FWD;
  // where the chunk-state and V' stores go: between the (b) products of the
  // next chunk (with O), or, without O (fewer products to hide them behind),
  // S before the (b) products and V' at the end of the chunk
  constexpr bool SPREAD = OUT;
  constexpr int BV = MODE == SEQ_FWD    ? SeqCfg<E, DK, DV>::FWD_BV
                     : MODE == SEQ_SAVE ? SeqCfg<E, DK, DV>::SAVE_BV
                                        : SeqCfg<E, DK, DV>::BV;
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDV = BV + PADE;
  constexpr int NTV = BV / 16, MTS = DK / 64;
  constexpr int NKD = DK / M::K, NKC = CH / M::K;
  __shared__ __align__(16) E sSB[DK * BV];  // S as B operands (k = d)
  __shared__ __align__(16) E sVB[CH * BV];  // V' as B operands (k = t)
  __shared__ __align__(16) E sSs[STORE ? 2 * DK * LDV : 1];  // state rows, by chunk parity
  __shared__ __align__(16) E sOut[STORE ? 2 * CH * LDV : 1];  // V' rows, by chunk parity
  __shared__ __align__(16) E sO[OUT ? CH * LDV : 1];      // O rows for the store
  using SC = SeqCfg<E, DK, DV>;
  constexpr int WARM = MODE == SEQ_SAVE ? SC::WARM_SAVE : MODE == SEQ_STORE ? SC::WARM_STORE
                                                                           : SC::WARM_FWD;
  __shared__ __align__(16) float sSink[WARM > 0 ? 64 : 1];  // warm-up loads land here

  int unit, tile;
  if (!map_unit_tile(DV / BV, a.N * a.H, unit, tile)) return;
  const int n = unit / a.H, h = unit - n * a.H, v0 = tile * BV;
  const int w = __builtin_amdgcn_readfirstlane(wave_id()), l = lane_id(), g4 = l >> 4;
  const int H = a.H;
  constexpr int FR = 64 * M::KPL;                  // elements of one fragment
  const unsigned lo = (unsigned)(l * M::KPL);      // lane offset inside a fragment
  const unsigned lc = (unsigned)(l * 4);           // lane offset inside an accumulator tile
  // the sequence: first token, length, first chunk (no per-chunk table loads)
  const int s0 = a.cu ? a.cu[n] : n * a.T;
  const int L = a.cu ? a.cu[n + 1] - s0 : a.T;
  const int c0 = seq_first_chunk(a, n), nch = (L + CH - 1) / CH;

  f32x4 S[MTS][NTV];
  const size_t sbase = ((size_t)n * H + h) * DK * DV;
#pragma unroll
  for (int i = 0; i < MTS; ++i)
#pragma unroll
    for (int j = 0; j < NTV; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
        S[i][j][e] = a.h0 ? a.h0[sbase + (size_t)d * DV + vv] : 0.f;
      }

  frag fW[NKD], fQ[NKD], fK[MTS][NKC], fP[NKC];
  raw4 uU[NTV];
  float gl = 0.f;  // g of token l of the chunk
  // Every operand is reloaded for the next chunk as soon as the current one
  // has consumed it, in the order the next chunk needs them (vector memory
  // returns in issue order): W~ and diag(e^g) Q rows of tile w after (b); U~
  // after (c); Kbar^T rows of the wave's state rows, P rows of tile w and the
  // gates after (d).  Nothing waits on a load right after issuing it.
  auto load_wq = [&](int j) {
    const E* Wp = (const E*)a.Wf + ((size_t)(c0 + j) * H + h) * CH * DK + (size_t)w * NKD * FR;
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt) fW[kt] = M::load(Wp + lo + kt * FR);
    if (OUT) {
      const E* Qp = (const E*)a.Qf + ((size_t)(c0 + j) * H + h) * CH * DK + (size_t)w * NKD * FR;
#pragma unroll
      for (int kt = 0; kt < NKD; ++kt) fQ[kt] = M::load(Qp + lo + kt * FR);
    }
  };
  auto load_u = [&](int j) {
    const E* Up = (const E*)a.Uc + ((size_t)(c0 + j) * H + h) * CH * DV +
                  ((size_t)w * (DV / 16) + v0 / 16) * 256;
#pragma unroll
    for (int jj = 0; jj < NTV; ++jj) uU[jj] = *reinterpret_cast<const raw4*>(Up + lc + jj * 256);
  };
  auto load_kp = [&](int j) {
    const size_t ch = (size_t)(c0 + j) * H + h;
    const E* Kp = (const E*)a.KbT + ch * DK * CH + (size_t)w * MTS * NKC * FR;
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) fK[i][kt] = M::load(Kp + lo + (i * NKC + kt) * FR);
    if (OUT) {
      const E* Pp = (const E*)a.Pf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) fP[kt] = M::load(Pp + lo + kt * FR);
    }
    if (a.gated) gl = a.g[ch * CH + l];
  };

  // Output pieces, 16 bytes per lane: chunk states and V' in fragment order
  // over dv (from the parity buffers sSs, sOut), O rows (this wave's, sO).
  constexpr int EPV = 16 / sizeof(E), VPR = BV / EPV;
  constexpr int PS = STORE ? DK * VPR / 256 : 0;  // state pieces per thread
  constexpr int PV = STORE ? CH * VPR / 256 : 0;  // V' pieces per thread
  constexpr int PO = 16 * VPR / 64;               // O pieces per lane
  static_assert(!STORE || (DK * VPR % 256 == 0 && CH * VPR % 256 == 0 && PS + PV <= NKD),
                "store pieces do not fit the k-steps");
  auto put_frag = [&](E* g, const E* lds, int idx) {
    const int r = idx / VPR, cv = idx - r * VPR, v = v0 + cv * EPV;
    const uint4 val = *reinterpret_cast<const uint4*>(lds + r * LDV + cv * EPV);
    if (sizeof(E) == 2) {
      const int kt = v / M::K, ln = (r & 15) + 16 * ((v % M::K) / M::KPL);
      store_stream(g + ((size_t)((r >> 4) * (DV / M::K) + kt) * 64 + ln) * M::KPL, val);
    } else {
      const E* x = reinterpret_cast<const E*>(&val);
#pragma unroll
      for (int q = 0; q < EPV; ++q) {
        const int vv = v + q, kt = vv / M::K, ln = (r & 15) + 16 * (vv % M::K);
        g[(size_t)((r >> 4) * (DV / M::K) + kt) * 64 + ln] = x[q];
      }
    }
  };
  auto put_s = [&](int i, size_t chk, int jj) {
    put_frag((E*)a.Sc + chk * DK * DV, sSs + (jj & 1) * DK * LDV, threadIdx.x + 256 * i);
  };
  auto put_v = [&](int i, size_t chk, int jj) {
    put_frag((E*)a.Vp + chk * CH * DV, sOut + (jj & 1) * CH * LDV, threadIdx.x + 256 * i);
  };
  auto put_o = [&](int jj) {
    const int st = s0 + jj * CH, ln = min(CH, L - jj * CH);
    wave_rows_out<E, BV, LDV>((E*)a.o + ((size_t)st * H + h) * DV + v0, (size_t)H * DV, sO, w, ln);
  };
  (void)PO;

  if (nch > 0) {
    load_wq(0);
    load_u(0);
    load_kp(0);
  }
  for (int j = 0; j < nch; ++j) {
    const int start = s0 + j * CH, len = min(CH, L - j * CH);
    const size_t ch = (size_t)(c0 + j) * H + h;

    // (a) publish S as B operands (and as rows for the chunk-state store)
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) {
        bfrag_put<E>(sSB, NTV, w * MTS + i, jj, S[i][jj]);
        if (STORE) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            sSs[(j & 1) * DK * LDV + (w * (DK / 4) + i * 16 + acc_row(e)) * LDV + jj * 16 +
                acc_col()] = to_e<E>(S[i][jj][e]);
        }
      }
    lds_barrier();

    // (b) W~ S and diag(e^g) Q S for the wave's 16 token rows.  The
    // outputs pending from the previous steps (this chunk's entry state, the
    // previous chunk's V' and O) are stored one piece per k-step between
    // the products, so that the CU's store path is never hit by a burst.
    if constexpr (STORE && !SPREAD)
      copy_out_frags<E, DK, BV, LDV, 256, true>((E*)a.Sc + ch * DK * DV, DV / M::K, v0,
                                                sSs + (j & 1) * DK * LDV);
    f32x4 P[NTV], Qs[NTV];
#pragma unroll
    for (int jj = 0; jj < NTV; ++jj) P[jj] = Qs[jj] = f32x4{0.f, 0.f, 0.f, 0.f};
    static_for<0, NKD>([&](auto ktc) {
      constexpr int kt = decltype(ktc)::value;
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) {
        const frag b = bfrag_get<E>(sSB, NTV, kt, jj);
        P[jj] = M::mma(fW[kt], b, P[jj]);
        if (OUT) Qs[jj] = M::mma(fQ[kt], b, Qs[jj]);
      }
      if constexpr (STORE && SPREAD) {
        if constexpr (kt < PS) put_s(kt, ch, j);
        else if constexpr (kt < PS + PV) {
          if (j > 0) put_v(kt - PS, ch - H, j - 1);
        }
      }
      if constexpr (OUT && kt == NKD - 1) {
        if (j > 0) put_o(j - 1);
      }
    });
    load_wq(min(j + 1, nch - 1));  // unconditional: keeps the load queue's shape static

    // (c) V' = U~ - W~ S
#pragma unroll
    for (int jj = 0; jj < NTV; ++jj) {
      f32x4 vp;
#pragma unroll
      for (int e = 0; e < 4; ++e) vp[e] = to_f(uU[jj][e]) - P[jj][e];
      bfrag_put<E>(sVB, NTV, w, jj, vp);
      if (STORE) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sOut[(j & 1) * CH * LDV + (w * 16 + acc_row(e)) * LDV + jj * 16 + acc_col()] =
              to_e<E>(vp[e]);
      }
    }
    load_u(min(j + 1, nch - 1));
    lds_barrier();

    // (d) S <- e^{g_n} S + Kbar^T V';  O = (diag(e^g) Q) S + P V'
    if (a.gated) {
      const float egn = __expf(__shfl(gl, CH - 1, 64));  // pads repeat g of the last token
#pragma unroll
      for (int i = 0; i < MTS; ++i)
#pragma unroll
        for (int jj = 0; jj < NTV; ++jj) S[i][jj] *= egn;
    }
    frag fKc[MTS][NKC], fPc[NKC];  // copies, so that the refills need not wait for the products
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) fKc[i][kt] = fK[i][kt];
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) fPc[kt] = fP[kt];
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) {
        const frag b = bfrag_get<E>(sVB, NTV, kt, jj);
#pragma unroll
        for (int i = 0; i < MTS; ++i) S[i][jj] = M::mma(fKc[i][kt], b, S[i][jj]);
        if (OUT) Qs[jj] = M::mma(fPc[kt], b, Qs[jj]);
      }
    load_kp(min(j + 1, nch - 1));
    if constexpr (WARM > 0) {
      const int jt = j + WARM;
      if (w == 0 && jt < nch) {
        const size_t cht = (size_t)(c0 + jt) * H + h;
        constexpr int LK = CH * DK * (int)sizeof(E), LP = CH * CH * (int)sizeof(E);
        const unsigned char* const base[4] = {
            (const unsigned char*)((const E*)a.Wf + cht * CH * DK),
            (const unsigned char*)((const E*)a.KbT + cht * DK * CH),
            (const unsigned char*)(OUT ? (const E*)a.Qf + cht * CH * DK : (const E*)a.Wf),
            (const unsigned char*)(OUT ? (const E*)a.Pf + cht * CH * CH : (const E*)a.Wf)};
        const int nbytes[4] = {LK, LK, OUT ? LK : 0, OUT ? LP : 0};
        warm_l2<4>(base, nbytes, tile, DV / BV, sSink);
      }
      if (jt < nch) {  // this wave's U~ tiles (read by this slice only)
        const unsigned char* const base[1] = {(const unsigned char*)(
            (const E*)a.Uc + ((size_t)(c0 + jt) * H + h) * CH * DV +
            ((size_t)w * (DV / 16) + v0 / 16) * 256)};
        const int nb[1] = {NTV * 256 * (int)sizeof(E)};
        warm_l2<1>(base, nb, 0, 1, sSink);
      }
    }
    if constexpr (STORE && !SPREAD)
      copy_out_frags<E, CH, BV, LDV, 256, true>((E*)a.Vp + ch * CH * DV, DV / M::K, v0,
                                                sOut + (j & 1) * CH * LDV);
    if (OUT) {  // O rows wait in LDS (this wave's rows) until the next chunk's (b)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sO[(w * 16 + acc_row(e)) * LDV + jj * 16 + acc_col()] = to_e<E>(Qs[jj][e]);
    }
  }
  if constexpr (WARM > 0) wait_vmcnt<0>();  // no LDS write in flight past the end
  // what the last chunk leaves pending
  if (nch > 0) {
    const size_t chl = (size_t)(c0 + nch - 1) * H + h;
    if constexpr (STORE && SPREAD)
      for (int i = 0; i < PV; ++i) put_v(i, chl, nch - 1);  // rows in LDS since (c)
    if constexpr (OUT) put_o(nch - 1);
  }

  if (OUT && a.ht) {
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + jj * 16 + acc_col();
          a.ht[sbase + (size_t)d * DV + vv] = S[i][jj][e];
        }
  }
}

// ------------------------------------------------------------------ backward state pass

template <class E, int DK, int DV>
__global__ __launch_bounds__(256, GDN_SEQ_MINB) void k_bwd_seq(Args a) {
  using M = Mfma<E>;
  using frag = typename M::frag;
  constexpr int BV = SeqCfg<E, DK, DV>::BV;
  constexpr int PADE = 16 / sizeof(E);
  constexpr int EPV = 16 / sizeof(E);
  constexpr int LDV = BV + PADE;
  constexpr int NTV = BV / 16, MTS = DK / 64;
  constexpr int NKD = DK / M::K, NKC = CH / M::K;
  constexpr int DOV = CH * BV / EPV / 256;  // dO vectors per thread
  static_assert(DOV >= 1, "dO tile too small for the workgroup");
  __shared__ __align__(16) E sdSB[DK * BV];     // dS as B operands (k = d)
  __shared__ __align__(16) E sdOB[2][CH * BV];  // dO as B operands (k = t), by chunk parity
  __shared__ __align__(16) E sdVB[CH * BV];     // dV' as B operands (k = t)
  __shared__ __align__(16) E sSs[DK * LDV];     // dS rows for the store
  __shared__ __align__(16) E sOut[CH * LDV];    // dX rows for the store
  __shared__ __align__(16) E sDv[CH * LDV];     // dv rows for the store (per wave)
  constexpr int WARM = SeqCfg<E, DK, DV>::WARM_BWD;
  __shared__ __align__(16) float sSink[WARM > 0 ? 64 : 1];  // warm-up loads land here

  int unit, tile;
  if (!map_unit_tile(DV / BV, a.N * a.H, unit, tile)) return;
  const int n = unit / a.H, h = unit - n * a.H, v0 = tile * BV;
  const int tid = threadIdx.x, l = lane_id(), g4 = l >> 4;
  const int w = __builtin_amdgcn_readfirstlane(wave_id());
  const int H = a.H;
  const E* dOin = (const E*)a.dO;
  constexpr int FR = 64 * M::KPL;                  // elements of one fragment
  const unsigned lo = (unsigned)(l * M::KPL);      // lane offset inside a fragment
  const int s0 = a.cu ? a.cu[n] : n * a.T;
  const int L = a.cu ? a.cu[n + 1] - s0 : a.T;
  const int c0 = seq_first_chunk(a, n), nch = (L + CH - 1) / CH;

  f32x4 dS[MTS][NTV];
  const size_t sbase = ((size_t)n * H + h) * DK * DV;
#pragma unroll
  for (int i = 0; i < MTS; ++i)
#pragma unroll
    for (int j = 0; j < NTV; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
        dS[i][j][e] = a.dht ? a.dht[sbase + (size_t)d * DV + vv] : 0.f;
      }

  frag fK[NKD], fPT[NKC], fT[NKC], fQ[MTS][NKC], fW[MTS][NKC];
  uint4 dov[DOV];
  float gl = 0.f, bl = 0.f;  // g and beta of token l of the chunk
  // Loads for the next chunk (in reverse order) are issued once the current
  // chunk has consumed the registers, in the order they are needed, and
  // unconditionally (clamped at the first chunk) so that every wait on the
  // in-order vector-memory counter stays partial.
  // First group, needed in (a)/(b): dO tile, K rows and P^T rows of tile w,
  // gates.
  auto load_first = [&](int j) {
    const int start = s0 + j * CH, len = min(CH, L - j * CH);
    const size_t ch = (size_t)(c0 + j) * H + h;
    const size_t row0 = (size_t)start * H + h;
#pragma unroll
    for (int x = 0; x < DOV; ++x) {
      const int idx = tid + x * 256, tt = idx & (CH - 1), cv = idx >> 6;
      dov[x] = *reinterpret_cast<const uint4*>(dOin + (row0 + (size_t)min(tt, len - 1) * H) * DV +
                                               v0 + cv * EPV);
      if (tt >= len) dov[x] = uint4{0u, 0u, 0u, 0u};
    }
    const E* Kp = (const E*)a.Kf + ch * CH * DK + (size_t)w * NKD * FR;
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt) fK[kt] = M::load(Kp + lo + kt * FR);
    const E* Pp = (const E*)a.PTf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) fPT[kt] = M::load(Pp + lo + kt * FR);
    if (a.gated) gl = a.g[ch * CH + l];
    bl = a.beta[row0 + (size_t)min(l, len - 1) * H];
  };
  // Second group, needed in (c): T^T rows of tile w; (e^g Q)^T and -W~^T rows
  // of the wave's state rows.
  // The same loads one fragment group at a time, issued in the loop right
  // after the last product that reads the register they refill (a refill
  // of a register that queued products still read waits for them).
  auto reload_K = [&](int j, int kt) {
    const size_t ch = (size_t)(c0 + j) * H + h;
    fK[kt] = M::load((const E*)a.Kf + ch * CH * DK + (size_t)w * NKD * FR + lo + kt * FR);
  };
  auto reload_PT = [&](int j) {
    const size_t ch = (size_t)(c0 + j) * H + h;
    const E* Pp = (const E*)a.PTf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) fPT[kt] = M::load(Pp + lo + kt * FR);
  };
  auto reload_rest = [&](int j) {  // dO tile and gates
    const int start = s0 + j * CH, len = min(CH, L - j * CH);
    const size_t ch = (size_t)(c0 + j) * H + h;
    const size_t row0 = (size_t)start * H + h;
#pragma unroll
    for (int x = 0; x < DOV; ++x) {
      const int idx = tid + x * 256, tt = idx & (CH - 1), cv = idx >> 6;
      dov[x] = *reinterpret_cast<const uint4*>(dOin + (row0 + (size_t)min(tt, len - 1) * H) * DV +
                                               v0 + cv * EPV);
      if (tt >= len) dov[x] = uint4{0u, 0u, 0u, 0u};
    }
    if (a.gated) gl = a.g[ch * CH + l];
    bl = a.beta[row0 + (size_t)min(l, len - 1) * H];
  };
  auto reload_T = [&](int j) {
    const size_t ch = (size_t)(c0 + j) * H + h;
    const E* Tp = (const E*)a.TTf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) fT[kt] = M::load(Tp + lo + kt * FR);
  };
  auto reload_QW = [&](int j, int kt) {
    const size_t ch = (size_t)(c0 + j) * H + h;
    const E* Qp = (const E*)a.QgT + ch * DK * CH + (size_t)w * MTS * NKC * FR;
    const E* Wp = (const E*)a.nWT + ch * DK * CH + (size_t)w * MTS * NKC * FR;
#pragma unroll
    for (int i = 0; i < MTS; ++i) {
      fQ[i][kt] = M::load(Qp + lo + (i * NKC + kt) * FR);
      fW[i][kt] = M::load(Wp + lo + (i * NKC + kt) * FR);
    }
  };
  auto load_second = [&](int j) {
    const size_t ch = (size_t)(c0 + j) * H + h;
    const E* Tp = (const E*)a.TTf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) fT[kt] = M::load(Tp + lo + kt * FR);
    const E* Qp = (const E*)a.QgT + ch * DK * CH + (size_t)w * MTS * NKC * FR;
    const E* Wp = (const E*)a.nWT + ch * DK * CH + (size_t)w * MTS * NKC * FR;
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) {
        fQ[i][kt] = M::load(Qp + lo + (i * NKC + kt) * FR);
        fW[i][kt] = M::load(Wp + lo + (i * NKC + kt) * FR);
      }
  };

  if (nch > 0) {
    load_first(nch - 1);
    load_second(nch - 1);
  }
  size_t prev_ch = 0;  // chunk whose dX rows wait in sOut
  for (int j = nch - 1; j >= 0; --j) {
    const int start = s0 + j * CH, len = min(CH, L - j * CH);
    const size_t ch = (size_t)(c0 + j) * H + h;
    E* sdO = sdOB[j & 1];

    // (a) publish dS (B operands and rows), dO (B operands)
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) {
        bfrag_put<E>(sdSB, NTV, w * MTS + i, jj, dS[i][jj]);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sSs[(w * (DK / 4) + i * 16 + acc_row(e)) * LDV + jj * 16 + acc_col()] =
              to_e<E>(dS[i][jj][e]);
      }
#pragma unroll
    for (int x = 0; x < DOV; ++x) {
      const int idx = tid + x * 256, tt = idx & (CH - 1), cv = idx >> 6;
      union {
        uint4 u;
        E e[EPV];
      } val;
      val.u = dov[x];
#pragma unroll
      for (int q = 0; q < EPV; ++q) sdO[bfrag_pos_t<E>(tt, cv * EPV + q, NTV)] = val.e[q];
    }
    lds_barrier();

    // (b) dV' = P^T dO + diag(e^{g_n - g}) (K dS); the stores of dS and of the
    //     previous chunk's dX rows
    copy_out_frags<E, DK, BV, LDV, 256, true>((E*)a.dSc + ch * DK * DV, DV / M::K, v0, sSs);
    if (j + 1 < nch)
      copy_out_frags<E, CH, BV, LDV, 256, true>((E*)a.dXb + prev_ch * CH * DV, DV / M::K, v0, sOut);
    f32x4 X1[NTV], X2[NTV];
#pragma unroll
    for (int jj = 0; jj < NTV; ++jj) X1[jj] = X2[jj] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int jn = max(j - 1, 0);  // the chunk whose operands are loaded next
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) X2[jj] = M::mma(fPT[kt], bfrag_get<E>(sdO, NTV, kt, jj), X2[jj]);
    reload_PT(jn);
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt) {
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) X1[jj] = M::mma(fK[kt], bfrag_get<E>(sdSB, NTV, kt, jj), X1[jj]);
      reload_K(jn, kt);
    }
    const float gn = __shfl(gl, CH - 1, 64);  // pads repeat g of the last token
    float brow[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = w * 16 + acc_row(e);
      const float gr = __shfl(gl, r, 64);  // every lane takes part in the shuffle
      const float dec = a.gated ? __expf(gn - gr) : 1.f;
      const float br = __shfl(bl, r, 64);  // every lane takes part in the shuffle
      brow[e] = r < len ? br : 0.f;
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) X1[jj][e] = dec * X1[jj][e] + X2[jj][e];
    }
#pragma unroll
    for (int jj = 0; jj < NTV; ++jj) bfrag_put<E>(sdVB, NTV, w, jj, X1[jj]);
    reload_rest(jn);
    lds_barrier();

    // (c) dX = T^T dV', dv = b dX;  dS <- e^{g_n} dS + (e^g Q)^T dO - W~^T dV'
    f32x4 dX[NTV];
#pragma unroll
    for (int jj = 0; jj < NTV; ++jj) dX[jj] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) dX[jj] = M::mma(fT[kt], bfrag_get<E>(sdVB, NTV, kt, jj), dX[jj]);
    reload_T(jn);
    if (a.gated) {
      const float egn = __expf(gn);
#pragma unroll
      for (int i = 0; i < MTS; ++i)
#pragma unroll
        for (int jj = 0; jj < NTV; ++jj) dS[i][jj] *= egn;
    }
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) {
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj) {
        const frag bo = bfrag_get<E>(sdO, NTV, kt, jj);
        const frag bv = bfrag_get<E>(sdVB, NTV, kt, jj);
#pragma unroll
        for (int i = 0; i < MTS; ++i) {
          dS[i][jj] = M::mma(fQ[i][kt], bo, dS[i][jj]);
          dS[i][jj] = M::mma(fW[i][kt], bv, dS[i][jj]);
        }
      }
      reload_QW(jn, kt);
    }
    {  // dX rows (stored with the next chunk) and dv rows (through LDS, 16 bytes per lane)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = w * 16 + acc_row(e);
#pragma unroll
        for (int jj = 0; jj < NTV; ++jj) {
          sOut[t * LDV + jj * 16 + acc_col()] = to_e<E>(dX[jj][e]);
          sDv[t * LDV + jj * 16 + acc_col()] = to_e<E>(brow[e] * dX[jj][e]);
        }
      }
      wave_rows_out<E, BV, LDV>((E*)a.dv + ((size_t)start * H + h) * DV + v0, (size_t)H * DV, sDv,
                                w, len);
    }
    prev_ch = ch;
    if constexpr (WARM > 0) {
      const int jt = j - WARM;
      if (w == 0 && jt >= 0) {
        const size_t cht = (size_t)(c0 + jt) * H + h;
        constexpr int LK = CH * DK * (int)sizeof(E), LC = CH * CH * (int)sizeof(E);
        const unsigned char* const base[5] = {
            (const unsigned char*)((const E*)a.Kf + cht * CH * DK),
            (const unsigned char*)((const E*)a.QgT + cht * DK * CH),
            (const unsigned char*)((const E*)a.nWT + cht * DK * CH),
            (const unsigned char*)((const E*)a.PTf + cht * CH * CH),
            (const unsigned char*)((const E*)a.TTf + cht * CH * CH)};
        const int nbytes[5] = {LK, LK, LK, LC, LC};
        warm_l2<5>(base, nbytes, tile, DV / BV, sSink);
      }
    }
  }
  if constexpr (WARM > 0) wait_vmcnt<0>();  // no LDS write in flight past the end
  if (nch > 0) {
    lds_barrier();
    copy_out_frags<E, CH, BV, LDV, 256, true>((E*)a.dXb + prev_ch * CH * DV, DV / M::K, v0, sOut);
  }

  if (a.dh0) {
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int jj = 0; jj < NTV; ++jj)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + jj * 16 + acc_col();
          a.dh0[sbase + (size_t)d * DV + vv] = dS[i][jj][e];
        }
  }
}

// ------------------------------------------------------------------ launchers

hipError_t launch_fwd_seq(Dt dt, int dk, int dv, int mode, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    constexpr int BV = SeqCfg<E, DK, DV>::BV, FBV = SeqCfg<E, DK, DV>::FWD_BV;
    constexpr int SBV = SeqCfg<E, DK, DV>::SAVE_BV;
    if (mode == SEQ_STORE)
      hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, SEQ_STORE>), dim3(unit_tile_grid(DV / BV, a.N * a.H)),
                         dim3(256), 0, s, a);
    else if (mode == SEQ_SAVE)
      hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, SEQ_SAVE>), dim3(unit_tile_grid(DV / SBV, a.N * a.H)),
                         dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, SEQ_FWD>), dim3(unit_tile_grid(DV / FBV, a.N * a.H)),
                         dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

hipError_t launch_bwd_seq(Dt dt, int dk, int dv, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    constexpr int BV = SeqCfg<E, DK, DV>::BV;
    const dim3 grid(unit_tile_grid(DV / BV, a.N * a.H));
    hipLaunchKernelGGL((k_bwd_seq<E, DK, DV>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

}  // namespace gdn

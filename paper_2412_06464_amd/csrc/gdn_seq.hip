// Sequential inter-chunk state passes (gfx950) of the chunkwise gated delta
// rule (Sec. 3.3; state stored dk x dv).  One workgroup owns one (sequence,
// head, BV-wide slice of dv): the dk x BV state tile lives in the MFMA
// accumulators of its four waves (wave w owns state rows [w dk/4, (w+1) dk/4))
// and the chunks of the sequence are walked in order.  Every dk-side operand
// was written by the prep kernels in MFMA fragment layout, so each wave loads
// its A fragments with coalesced 16-byte loads straight into registers, one
// chunk ahead of their use.  Only the state itself (as S^T) and the chunk's
// V' (as V'^T) pass through LDS, with two barriers per chunk.
//
// Forward, per chunk:   V' = U~ - W~ S,   O = Qeff S + P U~,
//                       S <- e^{g_n} S + Kbar^T V'.
// Backward, per chunk (reverse order), dS = gradient of the exit state:
//                       dV' = P^T dO + Kbar dS,   dX = T^T dV',   dv = b dX,
//                       dS <- e^{g_n} dS + (e^g Q)^T dO - W~^T dV'.
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {

// Workgroup id i is dispatched to XCD i % 8.  All dv slices of one
// (sequence, head) unit get ids with the same residue, so they share that
// XCD's L2 for the unit's dk-side operands.
__device__ inline bool map_unit_tile(int ntiles, int nunits, int& unit, int& tile) {
  const int id = blockIdx.x, xcd = id & 7, slot = id >> 3;
  const int ul = slot / ntiles;
  tile = slot - ul * ntiles;
  unit = ul * 8 + xcd;
  return unit < nunits;
}

inline int unit_tile_grid(int ntiles, int nunits) { return (nunits + 7) / 8 * 8 * ntiles; }

template <class E, int DK, int DV>
struct SeqCfg {
  static constexpr int BV = 32;
};

// ------------------------------------------------------------------ forward / recompute
// STORE = false: forward, writes O and ht.
// STORE = true : backward recompute, writes each chunk's entry state and V'.

template <class E, int DK, int DV, bool STORE>
__global__ __launch_bounds__(256) void k_fwd_seq(Args a) {
  using M = Mfma<E>;
  using frag = typename M::frag;
  constexpr int BV = SeqCfg<E, DK, DV>::BV;
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDK = DK + PADE, LDC = CH + PADE, LDV = BV + PADE;
  constexpr int NTV = BV / 16, MTS = DK / 64;
  constexpr int NKD = DK / M::K, NKC = CH / M::K;
  __shared__ __align__(16) E sST[BV * LDK];
  __shared__ __align__(16) E sVT[BV * LDC];
  __shared__ __align__(16) E sOut[CH * LDV];
  __shared__ __align__(16) E sSs[STORE ? DK * LDV : 1];

  int unit, tile;
  if (!map_unit_tile(DV / BV, a.N * a.H, unit, tile)) return;
  const int n = unit / a.H, h = unit - n * a.H, v0 = tile * BV;
  const int w = wave_id();
  const int H = a.H;

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

  frag fW[1][NKD], fQ[1][NKD], fK[MTS][NKC];
  f32x4 uU[NTV], uO[NTV];
  auto load_rows_side = [&](int c) {  // W~ / Qeff rows of tile w, U~ / P U~ tiles
    const size_t ch = (size_t)c * H + h;
    const E* Wp = (const E*)a.Wf + ch * CH * DK;
#pragma unroll
    for (int kk = 0; kk < NKD; ++kk) fW[0][kk] = M::load(Wp + afrag_index<E>(w, kk, DK));
    const E* Up = (const E*)a.Uc + ch * CH * DV;
#pragma unroll
    for (int j = 0; j < NTV; ++j) uU[j] = load4<E>(Up + cfrag_index(w, v0 / 16 + j, DV));
    if (!STORE) {
      const E* Qp = (const E*)a.Qf + ch * CH * DK;
#pragma unroll
      for (int kk = 0; kk < NKD; ++kk) fQ[0][kk] = M::load(Qp + afrag_index<E>(w, kk, DK));
      const E* Op = (const E*)a.Oc + ch * CH * DV;
#pragma unroll
      for (int j = 0; j < NTV; ++j) uO[j] = load4<E>(Op + cfrag_index(w, v0 / 16 + j, DV));
    }
  };
  auto load_state_side = [&](int c) {  // Kbar^T rows of the wave's state rows
    const size_t ch = (size_t)c * H + h;
    const E* Kp = (const E*)a.KbT + ch * DK * CH;
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int kk = 0; kk < NKC; ++kk) fK[i][kk] = M::load(Kp + afrag_index<E>(w * MTS + i, kk, CH));
  };

  const int c0 = a.seq_chunk0[n], c1 = a.seq_chunk0[n + 1];
  if (c0 < c1) {
    load_rows_side(c0);
    load_state_side(c0);
  }
  for (int c = c0; c < c1; ++c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const float gn = a.g[ch * CH + CH - 1];  // pads repeat g of the last token

    // (a) publish S^T (and S rows for the chunk-state store)
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        store_tile_T<E>(sST, LDK, S[i][j], w * (DK / 4) + i * 16, j * 16);
        if (STORE) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            sSs[(w * (DK / 4) + i * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] =
                to_e<E>(S[i][j][e]);
        }
      }
    lds_barrier();

    // (b) W~ S and Qeff S for the wave's 16 token rows
    if (STORE) copy_out_rows<E, DK, BV, LDV, 256>((E*)a.Sc + ch * DK * DV + v0, DV, sSs, DK);
    f32x4 P[1][NTV], Qs[1][NTV];
    zero_acc(P);
    mma_regA<E, 1, NTV, NKD>(P, fW, sST, LDK);
    if (!STORE) {
      zero_acc(Qs);
      mma_regA<E, 1, NTV, NKD>(Qs, fQ, sST, LDK);
    }

    // (c) V' = U~ - W~ S;  O = Qeff S + P U~
#pragma unroll
    for (int j = 0; j < NTV; ++j) {
      const f32x4 vp = uU[j] - P[0][j];
      store_tile_T<E>(sVT, LDC, vp, w * 16, j * 16);
      const f32x4 y = STORE ? vp : Qs[0][j] + uO[j];
#pragma unroll
      for (int e = 0; e < 4; ++e) sOut[(w * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] = to_e<E>(y[e]);
    }
    if (c + 1 < c1) load_rows_side(c + 1);
    lds_barrier();

    // (d) S <- e^{g_n} S + Kbar^T V'; write the chunk's rows out
    const float egn = __expf(gn);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) S[i][j] *= egn;
    mma_regA<E, MTS, NTV, NKC>(S, fK, sVT, LDC);
    if (c + 1 < c1) load_state_side(c + 1);
    if (STORE)
      copy_out_rows<E, CH, BV, LDV, 256>((E*)a.Vp + ch * CH * DV + v0, DV, sOut, CH);
    else
      copy_out_rows<E, CH, BV, LDV, 256>((E*)a.o + ((size_t)start * H + h) * DV + v0,
                                         (size_t)H * DV, sOut, len);
  }

  if (!STORE && a.ht) {
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
          a.ht[sbase + (size_t)d * DV + vv] = S[i][j][e];
        }
  }
}

// ------------------------------------------------------------------ backward state pass

template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void k_bwd_seq(Args a) {
  using M = Mfma<E>;
  using frag = typename M::frag;
  constexpr int BV = SeqCfg<E, DK, DV>::BV;
  constexpr int PADE = 16 / sizeof(E);
  constexpr int EPV = 16 / sizeof(E);
  constexpr int LDK = DK + PADE, LDC = CH + PADE, LDV = BV + PADE;
  constexpr int NTV = BV / 16, MTS = DK / 64;
  constexpr int NKD = DK / M::K, NKC = CH / M::K;
  constexpr int DOV = CH * BV / EPV / 256;  // dO vectors per thread
  static_assert(DOV >= 1, "dO tile too small for the workgroup");
  __shared__ __align__(16) E sdST[BV * LDK];
  __shared__ __align__(16) E sdOT[BV * LDC];
  __shared__ __align__(16) E sdVT[BV * LDC];
  __shared__ __align__(16) E sOut[CH * LDV];
  __shared__ __align__(16) E sSs[DK * LDV];
  __shared__ float sdec[CH], sb[2][CH];  // sb by chunk parity: read after the last barrier

  int unit, tile;
  if (!map_unit_tile(DV / BV, a.N * a.H, unit, tile)) return;
  const int n = unit / a.H, h = unit - n * a.H, v0 = tile * BV;
  const int tid = threadIdx.x, w = wave_id(), l = lane_id();
  const int H = a.H;
  const E* Kin = (const E*)a.k;
  const E* dOin = (const E*)a.dO;

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

  frag fK[1][NKD], fQ[MTS][NKC], fW[MTS][NKC], fT[1][NKC];
  f32x4 uD[NTV];
  uint4 dov[DOV];
  float pg = 0.f, pb = 0.f;
  auto load_chunk = [&](int c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const size_t row0 = (size_t)start * H + h;
    // raw K rows of tile w (zero beyond the chunk's length)
    const int r = w * 16 + (l & 15);
#pragma unroll
    for (int kk = 0; kk < NKD; ++kk) {
      if (r < len)
        fK[0][kk] = M::load(Kin + (row0 + (size_t)r * H) * DK + kk * M::K + (l >> 4) * M::KPL);
      else
        fK[0][kk] = typename M::frag{};
    }
    const E* Qp = (const E*)a.QgT + ch * DK * CH;
    const E* Wp = (const E*)a.nWT + ch * DK * CH;
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int kk = 0; kk < NKC; ++kk) {
        fQ[i][kk] = M::load(Qp + afrag_index<E>(w * MTS + i, kk, CH));
        fW[i][kk] = M::load(Wp + afrag_index<E>(w * MTS + i, kk, CH));
      }
    const E* Tp = (const E*)a.TT + ch * CH * CH;
#pragma unroll
    for (int kk = 0; kk < NKC; ++kk) fT[0][kk] = M::load(Tp + afrag_index<E>(w, kk, CH));
    const E* Dp = (const E*)a.dVi + ch * CH * DV;
#pragma unroll
    for (int j = 0; j < NTV; ++j) uD[j] = load4<E>(Dp + cfrag_index(w, v0 / 16 + j, DV));
#pragma unroll
    for (int x = 0; x < DOV; ++x) {
      const int idx = tid + x * 256, t = idx & (CH - 1), cv = idx >> 6;
      dov[x] = uint4{0u, 0u, 0u, 0u};
      if (t < len)
        dov[x] = *reinterpret_cast<const uint4*>(dOin + (row0 + (size_t)t * H) * DV + v0 + cv * EPV);
    }
    if (tid < CH) {
      pg = a.g[ch * CH + tid];
      pb = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
    }
  };

  const int c0 = a.seq_chunk0[n], c1 = a.seq_chunk0[n + 1];
  if (c0 < c1) load_chunk(c1 - 1);
  for (int c = c1 - 1; c >= c0; --c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const float gn = a.g[ch * CH + CH - 1];  // pads repeat g of the last token

    // (a) publish dS^T, dS rows, dO^T, gates
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        store_tile_T<E>(sdST, LDK, dS[i][j], w * (DK / 4) + i * 16, j * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sSs[(w * (DK / 4) + i * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] =
              to_e<E>(dS[i][j][e]);
      }
#pragma unroll
    for (int x = 0; x < DOV; ++x) {
      const int idx = tid + x * 256, t = idx & (CH - 1), cv = idx >> 6;
      union {
        uint4 u;
        E e[EPV];
      } val;
      val.u = dov[x];
#pragma unroll
      for (int j = 0; j < EPV; ++j) sdOT[(cv * EPV + j) * LDC + t] = val.e[j];
    }
    if (tid < CH) {
      sdec[tid] = __expf(gn - pg);
      sb[c & 1][tid] = pb;
    }
    lds_barrier();

    // (b) dV' = P^T dO + Kbar dS  (P^T dO precomputed per chunk)
    copy_out_rows<E, DK, BV, LDV, 256>((E*)a.dSc + ch * DK * DV + v0, DV, sSs, DK);
    f32x4 X[1][NTV];
    zero_acc(X);
    mma_regA<E, 1, NTV, NKD>(X, fK, sdST, LDK);
#pragma unroll
    for (int j = 0; j < NTV; ++j) {
      f32x4 y;
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = sdec[w * 16 + acc_row(e)] * X[0][j][e] + uD[j][e];
      store_tile_T<E>(sdVT, LDC, y, w * 16, j * 16);
    }
    lds_barrier();

    // (c) dX = T^T dV'; dS <- e^{g_n} dS + (e^g Q)^T dO - W~^T dV'
    f32x4 dX[1][NTV];
    zero_acc(dX);
    mma_regA<E, 1, NTV, NKC>(dX, fT, sdVT, LDC);
#pragma unroll
    for (int j = 0; j < NTV; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        sOut[(w * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] = to_e<E>(dX[0][j][e]);
    const float egn = __expf(gn);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) dS[i][j] *= egn;
    mma_regA<E, MTS, NTV, NKC>(dS, fQ, sdOT, LDC);
    mma_regA<E, MTS, NTV, NKC>(dS, fW, sdVT, LDC);
    if (c - 1 >= c0) load_chunk(c - 1);
    lds_barrier();

    // (d) dX rows (all 64) to the workspace, dv = b dX rows to the output
    copy_out_rows<E, CH, BV, LDV, 256>((E*)a.dXb + ch * CH * DV + v0, DV, sOut, CH);
    {
      constexpr int VPR = BV / EPV;
      E* gdv = (E*)a.dv + ((size_t)start * H + h) * DV + v0;
      for (int idx = tid; idx < CH * VPR; idx += 256) {
        const int t = idx / VPR, cv = idx - t * VPR;
        if (t < len) {
          union {
            uint4 u;
            E e[EPV];
          } x;
          x.u = *reinterpret_cast<const uint4*>(sOut + t * LDV + cv * EPV);
          const float b = sb[c & 1][t];
#pragma unroll
          for (int j = 0; j < EPV; ++j) x.e[j] = to_e<E>(b * to_f(x.e[j]));
          *reinterpret_cast<uint4*>(gdv + (size_t)t * H * DV + cv * EPV) = x.u;
        }
      }
    }
  }

  if (a.dh0) {
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
          a.dh0[sbase + (size_t)d * DV + vv] = dS[i][j][e];
        }
  }
}

// ------------------------------------------------------------------ launchers

hipError_t launch_fwd_seq(Dt dt, int dk, int dv, bool store, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    constexpr int BV = SeqCfg<E, DK, DV>::BV;
    const dim3 grid(unit_tile_grid(DV / BV, a.N * a.H));
    if (store)
      hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, true>), grid, dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, false>), grid, dim3(256), 0, s, a);
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

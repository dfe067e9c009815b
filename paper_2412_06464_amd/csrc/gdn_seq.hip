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
// Forward, per chunk:   V' = U~ - W~ S,   O = diag(e^g) (Q S) + P V',
//                       S <- e^{g_n} S + Kbar^T V'.
// Backward, per chunk (reverse order), dS = gradient of the exit state:
//                       dV' = P^T dO + diag(e^{g_n - g}) (K dS),
//                       dX = T^T dV',   dv = b dX,
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
// STORE = true : backward recompute, writes each chunk's entry state and V'
//                (row-major, for the gradient kernel).

template <class E, int DK, int DV, bool STORE>
__global__ __launch_bounds__(256, 2) void k_fwd_seq(Args a) {
  using M = Mfma<E>;
  using frag = typename M::frag;
  constexpr int BV = SeqCfg<E, DK, DV>::BV;
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDV = BV + PADE;
  constexpr int NTV = BV / 16, MTS = DK / 64;
  constexpr int NKD = DK / M::K, NKC = CH / M::K;
  __shared__ __align__(16) E sSB[DK * BV];  // S as B operands (k = d)
  __shared__ __align__(16) E sVB[CH * BV];  // V' as B operands (k = t)
  __shared__ __align__(16) E sSs[STORE ? DK * LDV : 1];
  __shared__ __align__(16) E sOut[STORE ? CH * LDV : 1];

  int unit, tile;
  if (!map_unit_tile(DV / BV, a.N * a.H, unit, tile)) return;
  const int n = unit / a.H, h = unit - n * a.H, v0 = tile * BV;
  const int w = __builtin_amdgcn_readfirstlane(wave_id()), l = lane_id(), g4 = l >> 4;
  const int H = a.H;
  constexpr int FR = 64 * M::KPL;                  // elements of one fragment
  const unsigned lo = (unsigned)(l * M::KPL);      // lane offset inside a fragment
  const unsigned lc = (unsigned)(l * 4);           // lane offset inside an accumulator tile
  const unsigned lq = (unsigned)((l & 15) * H * DK + 4 * g4);  // lane offset of raw q rows

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
  f32x4 uU[NTV];
  // W~ rows of tile w: needed first in a chunk, loaded a full chunk ahead
  auto load_w = [&](int c) {
    const E* Wp = (const E*)a.Wf + ((size_t)c * H + h) * CH * DK + (size_t)w * NKD * FR;
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt) fW[kt] = M::load(Wp + lo + kt * FR);
  };
  // raw q rows of tile w (permuted order of sSB), U~ tiles, Kbar^T rows of
  // the wave's state rows, P rows of tile w: loaded once the current chunk
  // has consumed its own (the register file holds one chunk of these)
  auto load_rest = [&](int c) {
    const size_t ch = (size_t)c * H + h;
    if (!STORE) {
      const int4 ci = a.info[c];
      const bool valid = w * 16 + (l & 15) < ci.z;
      const E* qrow = (const E*)a.q + ((size_t)(ci.y + w * 16) * H + h) * DK + lq;
#pragma unroll
      for (int kt = 0; kt < NKD; ++kt) fQ[kt] = load_row_perm_at<E>(qrow, kt, valid);
    }
    const E* Up = (const E*)a.Uc + ch * CH * DV + ((size_t)w * (DV / 16) + v0 / 16) * 256;
#pragma unroll
    for (int j = 0; j < NTV; ++j) uU[j] = load4<E>(Up + lc + j * 256);
    const E* Kp = (const E*)a.KbT + ch * DK * CH + (size_t)w * MTS * NKC * FR;
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) fK[i][kt] = M::load(Kp + lo + (i * NKC + kt) * FR);
    if (!STORE) {
      const E* Pp = (const E*)a.Pf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) fP[kt] = M::load(Pp + lo + kt * FR);
    }
  };

  const int c0 = a.seq_chunk0[n], c1 = a.seq_chunk0[n + 1];
  if (c0 < c1) {
    load_w(c0);
    load_rest(c0);
  }
  for (int c = c0; c < c1; ++c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const float gn = a.g[ch * CH + CH - 1];  // pads repeat g of the last token

    // (a) publish S as B operands (and as rows for the chunk-state store)
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        bfrag_put<E>(sSB, NTV, w * MTS + i, j, S[i][j]);
        if (STORE) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            sSs[(w * (DK / 4) + i * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] =
                to_e<E>(S[i][j][e]);
        }
      }
    lds_barrier();

    // (b) W~ S and Q S for the wave's 16 token rows
    if (STORE) copy_out_rows<E, DK, BV, LDV, 256>((E*)a.Sc + ch * DK * DV + v0, DV, sSs, DK);
    f32x4 P[NTV], Qs[NTV];
#pragma unroll
    for (int j = 0; j < NTV; ++j) P[j] = Qs[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        const frag b = bfrag_get<E>(sSB, NTV, kt, j);
        P[j] = M::mma(fW[kt], b, P[j]);
        if (!STORE) Qs[j] = M::mma(fQ[kt], b, Qs[j]);
      }
    if (c + 1 < c1) load_w(c + 1);

    // (c) V' = U~ - W~ S
#pragma unroll
    for (int j = 0; j < NTV; ++j) {
      const f32x4 vp = uU[j] - P[j];
      bfrag_put<E>(sVB, NTV, w, j, vp);
      if (STORE) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sOut[(w * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] = to_e<E>(vp[e]);
      }
    }
    lds_barrier();

    // (d) S <- e^{g_n} S + Kbar^T V';  O = diag(e^g) (Q S) + P V'
    const float egn = __expf(gn);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) S[i][j] *= egn;
    if (!STORE) {
      const float4 gr = *reinterpret_cast<const float4*>(a.g + ch * CH + w * 16 + 4 * g4);
      const float eg[4] = {__expf(gr.x), __expf(gr.y), __expf(gr.z), __expf(gr.w)};
#pragma unroll
      for (int j = 0; j < NTV; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) Qs[j][e] *= eg[e];
    }
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        const frag b = bfrag_get<E>(sVB, NTV, kt, j);
#pragma unroll
        for (int i = 0; i < MTS; ++i) S[i][j] = M::mma(fK[i][kt], b, S[i][j]);
        if (!STORE) Qs[j] = M::mma(fP[kt], b, Qs[j]);
      }
    if (c + 1 < c1) load_rest(c + 1);
    if (STORE) {
      copy_out_rows<E, CH, BV, LDV, 256>((E*)a.Vp + ch * CH * DV + v0, DV, sOut, CH);
    } else {
      E* orow = (E*)a.o + ((size_t)start * H + h) * DV + v0 + acc_col();
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = w * 16 + acc_row(e);
        if (t < len) {
#pragma unroll
          for (int j = 0; j < NTV; ++j) orow[(size_t)t * H * DV + j * 16] = to_e<E>(Qs[j][e]);
        }
      }
    }
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

// B-buffer position (element offset) of element (t, v) of a 64 x BV matrix
// whose B operands contract over t, in the permuted order.
template <class E> __device__ inline int bfrag_pos_t(int t, int v, int NT);
template <> __device__ inline int bfrag_pos_t<bf16>(int t, int v, int NT) {
  const int kt = t >> 5, tin = t & 31;
  const int g = (tin & 15) >> 2, j = (tin >> 4) * 4 + (tin & 3);
  return ((kt * NT + (v >> 4)) * 64 + g * 16 + (v & 15)) * 8 + j;
}
template <> __device__ inline int bfrag_pos_t<float>(int t, int v, int NT) {
  const int kt = 4 * (t >> 4) + (t & 3), g = (t & 15) >> 2;
  return (kt * NT + (v >> 4)) * 64 + g * 16 + (v & 15);
}

template <class E, int DK, int DV>
__global__ __launch_bounds__(256, 2) void k_bwd_seq(Args a) {
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

  int unit, tile;
  if (!map_unit_tile(DV / BV, a.N * a.H, unit, tile)) return;
  const int n = unit / a.H, h = unit - n * a.H, v0 = tile * BV;
  const int tid = threadIdx.x, l = lane_id(), g4 = l >> 4;
  const int w = __builtin_amdgcn_readfirstlane(wave_id());
  const int H = a.H;
  const E* dOin = (const E*)a.dO;
  constexpr int FR = 64 * M::KPL;                  // elements of one fragment
  const unsigned lo = (unsigned)(l * M::KPL);      // lane offset inside a fragment
  const unsigned lk = (unsigned)((l & 15) * H * DK + 4 * g4);  // lane offset of raw k rows

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
  // raw K rows (permuted order) and P^T rows of tile w, dO tile
  auto load_first = [&](int c) {
    const int4 ci = a.info[c];
    const size_t ch = (size_t)c * H + h;
    const size_t row0 = (size_t)ci.y * H + h;
    const bool valid = w * 16 + (l & 15) < ci.z;
    const E* krow = (const E*)a.k + ((size_t)(ci.y + w * 16) * H + h) * DK + lk;
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt) fK[kt] = load_row_perm_at<E>(krow, kt, valid);
    const E* Pp = (const E*)a.PTf + ch * CH * CH + (size_t)w * NKC * FR;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) fPT[kt] = M::load(Pp + lo + kt * FR);
#pragma unroll
    for (int x = 0; x < DOV; ++x) {
      const int idx = tid + x * 256, tt = idx & (CH - 1), cv = idx >> 6;
      dov[x] = uint4{0u, 0u, 0u, 0u};
      if (tt < ci.z)
        dov[x] = *reinterpret_cast<const uint4*>(dOin + (row0 + (size_t)tt * H) * DV + v0 + cv * EPV);
    }
  };
  // T^T rows of tile w; (e^g Q)^T and -W~^T rows of the wave's state rows
  auto load_second = [&](int c) {
    const size_t ch = (size_t)c * H + h;
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

  const int c0 = a.seq_chunk0[n], c1 = a.seq_chunk0[n + 1];
  if (c0 < c1) {
    load_first(c1 - 1);
    load_second(c1 - 1);
  }
  size_t prev_ch = 0;  // chunk whose dX rows wait in sOut
  bool pending = false;
  for (int c = c1 - 1; c >= c0; --c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const float gn = a.g[ch * CH + CH - 1];  // pads repeat g of the last token
    E* sdO = sdOB[c & 1];

    // (a) publish dS (B operands and rows), dO (B operands)
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        bfrag_put<E>(sdSB, NTV, w * MTS + i, j, dS[i][j]);
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sSs[(w * (DK / 4) + i * 16 + acc_row(e)) * LDV + j * 16 + acc_col()] =
              to_e<E>(dS[i][j][e]);
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
      for (int j = 0; j < EPV; ++j) sdO[bfrag_pos_t<E>(tt, cv * EPV + j, NTV)] = val.e[j];
    }
    lds_barrier();

    // (b) dV' = P^T dO + diag(e^{g_n - g}) (K dS); the stores of dS and of the
    //     previous chunk's dX rows
    copy_out_rows<E, DK, BV, LDV, 256>((E*)a.dSc + ch * DK * DV + v0, DV, sSs, DK);
    if (pending) copy_out_rows<E, CH, BV, LDV, 256>((E*)a.dXb + prev_ch * CH * DV + v0, DV, sOut, CH);
    f32x4 X1[NTV], X2[NTV];
#pragma unroll
    for (int j = 0; j < NTV; ++j) X1[j] = X2[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < NKD; ++kt)
#pragma unroll
      for (int j = 0; j < NTV; ++j) X1[j] = M::mma(fK[kt], bfrag_get<E>(sdSB, NTV, kt, j), X1[j]);
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int j = 0; j < NTV; ++j) X2[j] = M::mma(fPT[kt], bfrag_get<E>(sdO, NTV, kt, j), X2[j]);
    {
      const float4 gr = *reinterpret_cast<const float4*>(a.g + ch * CH + w * 16 + 4 * g4);
      const float dec[4] = {__expf(gn - gr.x), __expf(gn - gr.y), __expf(gn - gr.z),
                            __expf(gn - gr.w)};
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        f32x4 y;
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = dec[e] * X1[j][e] + X2[j][e];
        bfrag_put<E>(sdVB, NTV, w, j, y);
      }
    }
    if (c - 1 >= c0) load_first(c - 1);
    lds_barrier();

    // (c) dX = T^T dV', dv = b dX;  dS <- e^{g_n} dS + (e^g Q)^T dO - W~^T dV'
    f32x4 dX[NTV];
#pragma unroll
    for (int j = 0; j < NTV; ++j) dX[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int j = 0; j < NTV; ++j) dX[j] = M::mma(fT[kt], bfrag_get<E>(sdVB, NTV, kt, j), dX[j]);
    {
      E* dvrow = (E*)a.dv + ((size_t)start * H + h) * DV + v0 + acc_col();
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = w * 16 + acc_row(e);
        const float b = t < len ? a.beta[((size_t)start + t) * H + h] : 0.f;
#pragma unroll
        for (int j = 0; j < NTV; ++j) {
          sOut[t * LDV + j * 16 + acc_col()] = to_e<E>(dX[j][e]);
          if (t < len) dvrow[(size_t)t * H * DV + j * 16] = to_e<E>(b * dX[j][e]);
        }
      }
    }
    const float egn = __expf(gn);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) dS[i][j] *= egn;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        const frag bo = bfrag_get<E>(sdO, NTV, kt, j);
        const frag bv = bfrag_get<E>(sdVB, NTV, kt, j);
#pragma unroll
        for (int i = 0; i < MTS; ++i) {
          dS[i][j] = M::mma(fQ[i][kt], bo, dS[i][j]);
          dS[i][j] = M::mma(fW[i][kt], bv, dS[i][j]);
        }
      }
    if (c - 1 >= c0) load_second(c - 1);
    prev_ch = ch;
    pending = true;
  }
  if (pending) {
    lds_barrier();
    copy_out_rows<E, CH, BV, LDV, 256>((E*)a.dXb + prev_ch * CH * DV + v0, DV, sOut, CH);
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

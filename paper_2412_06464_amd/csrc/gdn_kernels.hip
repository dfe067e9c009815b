// HIP kernels (gfx950) of the chunkwise gated delta rule.
//
// Chunk algebra (Sec. 3.3 of the paper, state stored dk x dv, i.e. the
// transpose of the paper's dv x dk state).  For one chunk of n <= 64 tokens
// with entry state S, beta b, cumulative log gate g (Sec. 2.1 footnote:
// restarted at every chunk):
//   Gamma_ri = exp(g_r - g_i) for i <= r          (decay-aware causal mask)
//   A  = strictLower(diag(b) (Gamma * K K^T)),   T = (I + A)^-1
//   X  = diag(b) (V - diag(e^g) K S),            V' = T X
//   O  = diag(e^g) Q S + (Gamma * Q K^T) V'
//   S' = e^{g_n} S + (diag(e^{g_n - g}) K)^T V'
// V' equals the paper's  U~ - <-W S  (gated UT transform applied to the
// decayed keys and the values), written with one inverse; the intra-chunk
// output mask is Gamma (the paper prints M in the gated output equation,
// which does not reproduce the recurrence).
//
// Kernels:
//   k_chunk_table  chunk -> (sequence, first row, length) table
//   k_prep         per (chunk, head): g, Gamma*KK^T, Gamma*QK^T, T = (I+A)^-1
//   k_fwd_seq      per (sequence, head, dv tile): sequential over chunks,
//                  state tile in registers; emits O (forward) or the chunk
//                  entry states and V' (backward recompute)
//   k_bwd_seq      per (sequence, head, dv tile): reverse over chunks for the
//                  state gradient; emits dv, dX and every chunk's dS_next
//   k_grad         per (chunk, head): dq, dk, dbeta, dlog_alpha
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {

// ------------------------------------------------------------------ table

__global__ void k_chunk_table(const int32_t* cu, int N, int T, int4* info, int* seq_chunk0) {
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int n = 0; n < N; ++n) {
      seq_chunk0[n] = acc;
      const int L = cu ? cu[n + 1] - cu[n] : T;
      acc += (L + CH - 1) / CH;
    }
    seq_chunk0[N] = acc;
  }
  __syncthreads();
  for (int n = threadIdx.x; n < N; n += blockDim.x) {
    const int s = cu ? cu[n] : n * T;
    const int L = cu ? cu[n + 1] - cu[n] : T;
    const int c0 = seq_chunk0[n];
    for (int j = 0; j * CH < L; ++j) info[c0 + j] = make_int4(n, s + j * CH, min(CH, L - j * CH), 0);
  }
}

// ------------------------------------------------------------------ prep
// Grid (NC, H), 256 threads.  Writes g, Ak, Pm and Tm of one chunk-head.

template <class E, int DK>
__global__ __launch_bounds__(256) void k_prep(Args a) {
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDK = DK + PADE;
  constexpr int LDA = CH + 1;
  __shared__ __align__(16) E sK[CH * LDK];
  __shared__ __align__(16) E sQ[CH * LDK];
  __shared__ float sA[CH * LDA];
  __shared__ float sT[CH * LDA];
  __shared__ float sY[3 * 16 * 17];
  __shared__ float sg[CH], sb[CH];

  const int c = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, w = wave_id();
  const int H = a.H;
  const int4 ci = a.info[c];
  const int start = ci.y, len = ci.z;
  const size_t ch = (size_t)c * H + h;
  const size_t row0 = (size_t)start * H + h;

  stage_rows<E, CH, DK, LDK, 256>(sK, (const E*)a.k + row0 * DK, (size_t)H * DK, len);
  stage_rows<E, CH, DK, LDK, 256>(sQ, (const E*)a.q + row0 * DK, (size_t)H * DK, len);
  if (tid < CH) {
    const float la = tid < len ? a.log_alpha[row0 + (size_t)tid * H] : 0.f;
    const float g = wave_incl_scan(la);  // pads repeat g at the last token
    sg[tid] = g;
    sb[tid] = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
    a.g[ch * CH + tid] = g;
  }
  __syncthreads();

  // Gram blocks: wave w owns rows 16w..16w+15 of K K^T and Q K^T.
  f32x4 kk[1][4], qk[1][4];
  zero_acc(kk);
  zero_acc(qk);
  wave_mma_nt<E, 1, 4, DK>(kk, sK + w * 16 * LDK, LDK, sK, LDK);
  wave_mma_nt<E, 1, 4, DK>(qk, sQ + w * 16 * LDK, LDK, sK, LDK);
  float* gAk = a.Ak + ch * CH * CH;
  float* gP = a.Pm + ch * CH * CH;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = w * 16 + acc_row(e), i = j * 16 + acc_col();
      // select, never multiply by an overflowed exp above the diagonal
      const float gam = (i <= r) ? __expf(sg[r] - sg[i]) : 0.f;
      const float ak = (i < r) ? gam * kk[0][j][e] : 0.f;
      const float p = (i <= r) ? gam * qk[0][j][e] : 0.f;
      gAk[r * CH + i] = ak;
      gP[r * CH + i] = p;
      sA[r * LDA + i] = sb[r] * ak;
    }
  __syncthreads();

  // T = (I + A)^-1, A strictly lower.  Diagonal 16x16 blocks by forward
  // substitution (one column per thread), then the off-diagonal blocks in
  // order of their distance from the diagonal:
  //   T_IJ = -T_II * sum_{m=J}^{I-1} A_Im T_mJ.
  if (tid < CH) {
    const int blk = tid >> 4, j = tid & 15, o = blk * 16;
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float s = (i == j) ? 1.f : 0.f;
#pragma unroll
      for (int l = 0; l < i; ++l) s -= sA[(o + i) * LDA + o + l] * x[l];
      x[i] = s;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) sT[(o + i) * LDA + o + j] = x[i];
  }
  __syncthreads();
  for (int d = 1; d < 4; ++d) {
    const int i = tid >> 4, j = tid & 15;
    for (int J = 0; J + d < 4; ++J) {
      const int I = J + d;
      float y = 0.f;
      for (int m = J; m < I; ++m)
#pragma unroll
        for (int l = 0; l < 16; ++l)
          y += sA[(16 * I + i) * LDA + 16 * m + l] * sT[(16 * m + l) * LDA + 16 * J + j];
      sY[J * 272 + i * 17 + j] = y;
    }
    __syncthreads();
    for (int J = 0; J + d < 4; ++J) {
      const int I = J + d;
      float t = 0.f;
#pragma unroll
      for (int l = 0; l < 16; ++l) t -= sT[(16 * I + i) * LDA + 16 * I + l] * sY[J * 272 + l * 17 + j];
      sT[(16 * I + i) * LDA + 16 * J + j] = t;
    }
    __syncthreads();
  }
  float* gT = a.Tm + ch * CH * CH;
  for (int idx = tid; idx < CH * CH; idx += 256) {
    const int r = idx >> 6, i = idx & 63;
    gT[idx] = ((i >> 4) > (r >> 4)) ? 0.f : sT[r * LDA + i];
  }
}

// ------------------------------------------------------------------ forward state pass
// Grid (DV / BV, H, N), 256 threads (4 waves).  The dk x BV state tile lives
// in the MFMA accumulators: wave w owns state rows [w*DK/4, (w+1)*DK/4).
// STORE = false: forward, writes O and ht.
// STORE = true : backward recompute, writes each chunk's entry state and V'.

template <class E, int DK, int DV, int BV, bool STORE>
__global__ __launch_bounds__(256) void k_fwd_seq(Args a) {
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDK = DK + PADE;
  constexpr int LDC = CH + PADE;
  constexpr int LDV = BV + PADE;
  constexpr int NTV = BV / 16;
  constexpr int MTS = DK / 64;
  constexpr int QN = STORE ? 1 : CH;  // Q / P buffers are unused when storing
  __shared__ __align__(16) E sK[CH * LDK];
  __shared__ __align__(16) E sQ[QN * LDK];
  __shared__ __align__(16) E sKbT[DK * LDC];
  __shared__ __align__(16) E sST[BV * LDK];
  __shared__ __align__(16) E sTm[CH * LDC];
  __shared__ __align__(16) E sPm[QN * LDC];
  __shared__ __align__(16) E sXT[BV * LDC];
  __shared__ __align__(16) E sVpT[BV * LDC];
  __shared__ __align__(16) E sV[CH * LDV];
  __shared__ float sg[CH], sb[CH], sdec[CH];
  __shared__ float sgn[1];

  const int v0 = blockIdx.x * BV, h = blockIdx.y, n = blockIdx.z;
  const int tid = threadIdx.x, w = wave_id();
  const int H = a.H;
  const E* K = (const E*)a.k;
  const E* Q = (const E*)a.q;
  const E* V = (const E*)a.v;

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

  const int c0 = a.seq_chunk0[n], c1 = a.seq_chunk0[n + 1];
  for (int c = c0; c < c1; ++c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const size_t row0 = (size_t)start * H + h;

    // phase 0: stage the chunk, publish S^T
    if (tid < CH) {
      const float g = a.g[ch * CH + tid];
      const float gn = __shfl(g, len - 1, 64);
      sg[tid] = g;
      sb[tid] = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
      sdec[tid] = __expf(gn - g);
      if (tid == 0) sgn[0] = gn;
    }
    stage_rows<E, CH, DK, LDK, 256>(sK, K + row0 * DK, (size_t)H * DK, len);
    if (!STORE) stage_rows<E, CH, DK, LDK, 256>(sQ, Q + row0 * DK, (size_t)H * DK, len);
    stage_rows<E, CH, BV, LDV, 256>(sV, V + row0 * DV + v0, (size_t)H * DV, len);
    stage_mat64<E, LDC, 256, false>(sTm, a.Tm + ch * CH * CH);
    if (!STORE) stage_mat64<E, LDC, 256, false>(sPm, a.Pm + ch * CH * CH);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        store_tile_T<E>(sST, LDK, S[i][j], w * (DK / 4) + i * 16, j * 16);
        if (STORE) {
          E* gS = (E*)a.Sc + ch * DK * DV;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
            gS[(size_t)d * DV + vv] = to_e<E>(S[i][j][e]);
          }
        }
      }
    __syncthreads();

    // phase 1: decayed keys (transposed), K S and Q S, X
    stage_rows_T<E, DK, LDC, 256>(sKbT, K + row0 * DK, (size_t)H * DK, len, sdec);
    f32x4 ks[1][NTV], qs[1][NTV];
    zero_acc(ks);
    wave_mma_nt<E, 1, NTV, DK>(ks, sK + w * 16 * LDK, LDK, sST, LDK);
    if (!STORE) {
      zero_acc(qs);
      wave_mma_nt<E, 1, NTV, DK>(qs, sQ + w * 16 * LDK, LDK, sST, LDK);
    }
#pragma unroll
    for (int j = 0; j < NTV; ++j) {
      f32x4 x;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int t = w * 16 + acc_row(e), vv = j * 16 + acc_col();
        x[e] = sb[t] * (to_f(sV[t * LDV + vv]) - __expf(sg[t]) * ks[0][j][e]);
        if (!STORE) qs[0][j][e] *= __expf(sg[t]);
      }
      store_tile_T<E>(sXT, LDC, x, w * 16, j * 16);
    }
    __syncthreads();

    // phase 2: V' = T X
    f32x4 vp[1][NTV];
    zero_acc(vp);
    wave_mma_nt<E, 1, NTV, CH>(vp, sTm + w * 16 * LDC, LDC, sXT, LDC);
#pragma unroll
    for (int j = 0; j < NTV; ++j) {
      store_tile_T<E>(sVpT, LDC, vp[0][j], w * 16, j * 16);
      if (STORE) {
        E* gV = (E*)a.Vp + ch * CH * DV;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int t = w * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
          gV[(size_t)t * DV + vv] = to_e<E>(vp[0][j][e]);
        }
      }
    }
    __syncthreads();

    // phase 3: O = e^g Q S + P V'; S <- e^{g_n} S + Kbar^T V'
    if (!STORE) {
      wave_mma_nt<E, 1, NTV, CH>(qs, sPm + w * 16 * LDC, LDC, sVpT, LDC);
      E* O = (E*)a.o + row0 * DV + v0;
#pragma unroll
      for (int j = 0; j < NTV; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int t = w * 16 + acc_row(e), vv = j * 16 + acc_col();
          if (t < len) O[(size_t)t * H * DV + vv] = to_e<E>(qs[0][j][e]);
        }
    }
    const float egn = __expf(sgn[0]);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) S[i][j] *= egn;
    wave_mma_nt<E, MTS, NTV, CH>(S, sKbT + w * (DK / 4) * LDC, LDC, sVpT, LDC);
    __syncthreads();
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
// Grid (DV / BV, H, N), 256 threads.  Reverse over the chunks of a sequence,
// carrying dS (gradient of the chunk's exit state) in the accumulators:
//   dV' = P^T dO + Kbar dS,   dX = T^T dV',   dv = b dX,
//   dS <- e^{g_n} dS + (e^g Q)^T dO - (b e^g K)^T dX.

template <class E, int DK, int DV, int BV>
__global__ __launch_bounds__(256) void k_bwd_seq(Args a) {
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDK = DK + PADE;
  constexpr int LDC = CH + PADE;
  constexpr int NTV = BV / 16;
  constexpr int MTS = DK / 64;
  __shared__ __align__(16) E sK[CH * LDK];
  __shared__ __align__(16) E sQgT[DK * LDC];
  __shared__ __align__(16) E sKbT[DK * LDC];
  __shared__ __align__(16) E sdST[BV * LDK];
  __shared__ __align__(16) E sdOT[BV * LDC];
  __shared__ __align__(16) E sPT[CH * LDC];
  __shared__ __align__(16) E sTT[CH * LDC];
  __shared__ __align__(16) E sdVpT[BV * LDC];
  __shared__ __align__(16) E sdXT[BV * LDC];
  __shared__ float sb[CH], sdec[CH], seg[CH], snbeg[CH];
  __shared__ float sgn[1];

  const int v0 = blockIdx.x * BV, h = blockIdx.y, n = blockIdx.z;
  const int tid = threadIdx.x, w = wave_id();
  const int H = a.H;
  const E* K = (const E*)a.k;
  const E* Q = (const E*)a.q;
  const E* dO = (const E*)a.dO;

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

  const int c0 = a.seq_chunk0[n], c1 = a.seq_chunk0[n + 1];
  for (int c = c1 - 1; c >= c0; --c) {
    const int4 ci = a.info[c];
    const int start = ci.y, len = ci.z;
    const size_t ch = (size_t)c * H + h;
    const size_t row0 = (size_t)start * H + h;

    // phase 0
    if (tid < CH) {
      const float g = a.g[ch * CH + tid];
      const float gn = __shfl(g, len - 1, 64);
      const float b = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
      const float eg = __expf(g);
      sb[tid] = b;
      seg[tid] = eg;
      snbeg[tid] = -b * eg;
      sdec[tid] = __expf(gn - g);
      if (tid == 0) sgn[0] = gn;
    }
    stage_rows<E, CH, DK, LDK, 256>(sK, K + row0 * DK, (size_t)H * DK, len);
    stage_rows_T<E, BV, LDC, 256>(sdOT, dO + row0 * DV + v0, (size_t)H * DV, len, nullptr);
    stage_mat64<E, LDC, 256, true>(sPT, a.Pm + ch * CH * CH);
    stage_mat64<E, LDC, 256, true>(sTT, a.Tm + ch * CH * CH);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        store_tile_T<E>(sdST, LDK, dS[i][j], w * (DK / 4) + i * 16, j * 16);
        E* gdS = (E*)a.dSc + ch * DK * DV;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int d = w * (DK / 4) + i * 16 + acc_row(e), vv = v0 + j * 16 + acc_col();
          gdS[(size_t)d * DV + vv] = to_e<E>(dS[i][j][e]);
        }
      }
    __syncthreads();

    // phase 1: scaled transposed Q and K; dV' = Kbar dS + P^T dO
    stage_rows_T<E, DK, LDC, 256>(sQgT, Q + row0 * DK, (size_t)H * DK, len, seg);
    stage_rows_T<E, DK, LDC, 256>(sKbT, K + row0 * DK, (size_t)H * DK, len, snbeg);
    f32x4 dvp[1][NTV];
    zero_acc(dvp);
    wave_mma_nt<E, 1, NTV, DK>(dvp, sK + w * 16 * LDK, LDK, sdST, LDK);
#pragma unroll
    for (int j = 0; j < NTV; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) dvp[0][j][e] *= sdec[w * 16 + acc_row(e)];
    wave_mma_nt<E, 1, NTV, CH>(dvp, sPT + w * 16 * LDC, LDC, sdOT, LDC);
#pragma unroll
    for (int j = 0; j < NTV; ++j) store_tile_T<E>(sdVpT, LDC, dvp[0][j], w * 16, j * 16);
    __syncthreads();

    // phase 2: dX = T^T dV'; dv = b dX
    f32x4 dx[1][NTV];
    zero_acc(dx);
    wave_mma_nt<E, 1, NTV, CH>(dx, sTT + w * 16 * LDC, LDC, sdVpT, LDC);
    {
      E* gdv = (E*)a.dv + row0 * DV + v0;
      E* gdX = (E*)a.dXb + ch * CH * DV + v0;
#pragma unroll
      for (int j = 0; j < NTV; ++j) {
        store_tile_T<E>(sdXT, LDC, dx[0][j], w * 16, j * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int t = w * 16 + acc_row(e), vv = j * 16 + acc_col();
          gdX[(size_t)t * DV + vv] = to_e<E>(dx[0][j][e]);
          if (t < len) gdv[(size_t)t * H * DV + vv] = to_e<E>(sb[t] * dx[0][j][e]);
        }
      }
    }
    __syncthreads();

    // phase 3: dS <- e^{g_n} dS + (e^g Q)^T dO - (b e^g K)^T dX
    const float egn = __expf(sgn[0]);
#pragma unroll
    for (int i = 0; i < MTS; ++i)
#pragma unroll
      for (int j = 0; j < NTV; ++j) dS[i][j] *= egn;
    wave_mma_nt<E, MTS, NTV, CH>(dS, sQgT + w * (DK / 4) * LDC, LDC, sdOT, LDC);
    wave_mma_nt<E, MTS, NTV, CH>(dS, sKbT + w * (DK / 4) * LDC, LDC, sdXT, LDC);
    __syncthreads();
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

// ------------------------------------------------------------------ gradient kernel
// Grid (NC, H), 512 threads (8 waves).  Streams the dv dimension in tiles of
// BVG and accumulates, for the chunk:
//   Gq = dO S^T, Gk = dX S^T, Gs = V' dS_next^T       (64 x dk)
//   dO V'^T, dX V'^T                                  (64 x 64)
// then finishes
//   dQ = diag(e^g) Gq + (dP * Gamma) K
//   dK = (dP * Gamma)^T Q + diag(e^{g_n-g}) Gs - diag(b e^g) Gk + (D + D^T) K
//   dbeta_r = sum_i dA_ri Ak_ri + dX_r . V_r - e^{g_r} k_r . Gk_r
//   dg_r = e^{g_r} q_r.Gq_r - b_r e^{g_r} k_r.Gk_r - e^{g_n-g_r} k_r.Gs_r
//          + sum_i E_ri - sum_j E_jr   (+ the g_n terms on the last token)
//   dlog_alpha = reverse cumulative sum of dg inside the chunk
// with dP = lower(dO V'^T), dA = strictLower(-dX V'^T), D = diag(b)(dA*Gamma),
// E = dA * diag(b) Ak + dP * P.

template <class E, int DK, int DV, int BVG>
struct GradLds {
  static constexpr int PADE = 16 / sizeof(E);
  static constexpr int LDG = BVG + PADE;
  static constexpr int LDC = CH + PADE;
  static constexpr size_t stream_bytes = (size_t)(4 * CH * LDG + 2 * DK * LDG) * sizeof(E);
  static constexpr size_t finish_e = (size_t)(2 * DK * LDC + 3 * CH * LDC) * sizeof(E);
  static constexpr size_t finish_bytes = finish_e + 2 * CH * (CH + 1) * sizeof(float);
  static constexpr size_t bytes = stream_bytes > finish_bytes ? stream_bytes : finish_bytes;
};

template <class E, int DK, int DV, int BVG>
__global__ __launch_bounds__(512) void k_grad(Args a) {
  using L = GradLds<E, DK, DV, BVG>;
  constexpr int LDG = L::LDG, LDC = L::LDC, LDE = CH + 1;
  constexpr int NTH = 512;
  constexpr int CT = DK / 16;
  constexpr int CTW = CT >= 16 ? CT / 8 : 1;
  constexpr int WC = CT / CTW;
  constexpr int WR = 8 / WC;
  constexpr int RTW = 4 / WR;
  __shared__ __align__(16) unsigned char smem[L::bytes];
  __shared__ float sg[CH], sb[CH], seg[CH], sdec[CH], sxv[CH], sdbA[CH];
  __shared__ float sErow[CH], sEcol[CH];
  __shared__ float srow[WC][3][CH];
  __shared__ float sred[8];

  E* sdO = (E*)smem;
  E* sdX = sdO + CH * LDG;
  E* sVp = sdX + CH * LDG;
  E* sV = sVp + CH * LDG;
  E* sS = sV + CH * LDG;
  E* sdS = sS + DK * LDG;
  E* sKT = (E*)smem;
  E* sQT = sKT + DK * LDC;
  E* sM1 = sQT + DK * LDC;
  E* sM1T = sM1 + CH * LDC;
  E* sDD = sM1T + CH * LDC;
  float* sD = (float*)(smem + L::finish_e);
  float* sE = sD + CH * LDE;

  const int c = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, w = wave_id();
  const int H = a.H;
  const int4 ci = a.info[c];
  const int start = ci.y, len = ci.z;
  const size_t ch = (size_t)c * H + h;
  const size_t row0 = (size_t)start * H + h;
  const E* K = (const E*)a.k;
  const E* Q = (const E*)a.q;
  const E* V = (const E*)a.v;
  const E* dO = (const E*)a.dO;

  if (tid < CH) {
    const float g = a.g[ch * CH + tid];
    const float gn = __shfl(g, len - 1, 64);
    sg[tid] = g;
    sb[tid] = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
    seg[tid] = __expf(g);
    sdec[tid] = __expf(gn - g);
  }

  const int wc = w % WC, wr = w / WC;
  const int pm = w >> 2, prt = w & 3;
  f32x4 Gq[RTW][CTW], Gk[RTW][CTW], Gs[RTW][CTW], PA[1][4];
  zero_acc(Gq);
  zero_acc(Gk);
  zero_acc(Gs);
  zero_acc(PA);
  float sdot = 0.f, xvp = 0.f;

  for (int v0 = 0; v0 < DV; v0 += BVG) {
    stage_rows<E, CH, BVG, LDG, NTH>(sdO, dO + row0 * DV + v0, (size_t)H * DV, len);
    stage_rows<E, CH, BVG, LDG, NTH>(sV, V + row0 * DV + v0, (size_t)H * DV, len);
    stage_rows<E, CH, BVG, LDG, NTH>(sdX, (const E*)a.dXb + ch * CH * DV + v0, DV, CH);
    stage_rows<E, CH, BVG, LDG, NTH>(sVp, (const E*)a.Vp + ch * CH * DV + v0, DV, CH);
    stage_rows<E, DK, BVG, LDG, NTH>(sS, (const E*)a.Sc + ch * DK * DV + v0, DV, DK);
    stage_rows<E, DK, BVG, LDG, NTH>(sdS, (const E*)a.dSc + ch * DK * DV + v0, DV, DK);
    __syncthreads();
    const E* Arow = sdO + wr * RTW * 16 * LDG;
    const E* Brow = sS + wc * CTW * 16 * LDG;
    wave_mma_nt<E, RTW, CTW, BVG>(Gq, Arow, LDG, Brow, LDG);
    wave_mma_nt<E, RTW, CTW, BVG>(Gk, sdX + wr * RTW * 16 * LDG, LDG, Brow, LDG);
    wave_mma_nt<E, RTW, CTW, BVG>(Gs, sVp + wr * RTW * 16 * LDG, LDG,
                                  sdS + wc * CTW * 16 * LDG, LDG);
    wave_mma_nt<E, 1, 4, BVG>(PA, (pm ? sdX : sdO) + prt * 16 * LDG, LDG, sVp, LDG);
    for (int idx = tid; idx < DK * BVG; idx += NTH) {
      const int d = idx / BVG, vv = idx - d * BVG;
      sdot += to_f(sS[d * LDG + vv]) * to_f(sdS[d * LDG + vv]);
    }
    {
      const int t = tid >> 3, part = tid & 7;
#pragma unroll
      for (int vv = part * (BVG / 8); vv < (part + 1) * (BVG / 8); ++vv)
        xvp += to_f(sdX[t * LDG + vv]) * to_f(sV[t * LDG + vv]);
    }
    __syncthreads();
  }

  // reductions of <dS_next, S> and dX . V
  {
    float x = xvp;
    x += __shfl_xor(x, 1, 64);
    x += __shfl_xor(x, 2, 64);
    x += __shfl_xor(x, 4, 64);
    if ((tid & 7) == 0) sxv[tid >> 3] = x;
    float s = sdot;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) s += __shfl_xor(s, off, 64);
    if (lane_id() == 0) sred[w] = s;
  }
  stage_rows_T<E, DK, LDC, NTH>(sKT, K + row0 * DK, (size_t)H * DK, len, nullptr);
  stage_rows_T<E, DK, LDC, NTH>(sQT, Q + row0 * DK, (size_t)H * DK, len, nullptr);
  __syncthreads();

  // intra-chunk matrices
  float ea[4][4];
  {
    const float* gP = a.Pm + ch * CH * CH;
    const float* gAk = a.Ak + ch * CH * CH;
    float dbA[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = prt * 16 + acc_row(e), i = j * 16 + acc_col();
        const float gam = (i <= r) ? __expf(sg[r] - sg[i]) : 0.f;
        if (pm == 0) {
          const float dp = (i <= r) ? PA[0][j][e] : 0.f;
          const float m1 = dp * gam;
          sM1[r * LDC + i] = to_e<E>(m1);
          sM1T[i * LDC + r] = to_e<E>(m1);
          sE[r * LDE + i] = dp * gP[r * CH + i];
          ea[j][e] = 0.f;
        } else {
          const float da = (i < r) ? -PA[0][j][e] : 0.f;
          const float ak = gAk[r * CH + i];
          sD[r * LDE + i] = sb[r] * da * gam;
          ea[j][e] = da * sb[r] * ak;
          dbA[e] += da * ak;
        }
      }
    if (pm == 1) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float s = reduce16(dbA[e]);
        if (acc_col() == 0) sdbA[prt * 16 + acc_row(e)] = s;
      }
    }
  }
  // row dot products of the raw accumulators
  {
    float pq[RTW][4], pk[RTW][4], ps[RTW][4];
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pq[i][e] = pk[i][e] = ps[i][e] = 0.f;
        const int r = (wr * RTW + i) * 16 + acc_row(e);
#pragma unroll
        for (int j = 0; j < CTW; ++j) {
          const int d = (wc * CTW + j) * 16 + acc_col();
          const float qv = to_f(sQT[d * LDC + r]), kv = to_f(sKT[d * LDC + r]);
          pq[i][e] += qv * Gq[i][j][e];
          pk[i][e] += kv * Gk[i][j][e];
          ps[i][e] += kv * Gs[i][j][e];
        }
      }
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a0 = reduce16(pq[i][e]), a1 = reduce16(pk[i][e]), a2 = reduce16(ps[i][e]);
        if (acc_col() == 0) {
          const int r = (wr * RTW + i) * 16 + acc_row(e);
          srow[wc][0][r] = a0;
          srow[wc][1][r] = a1;
          srow[wc][2][r] = a2;
        }
      }
  }
  __syncthreads();
  if (pm == 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = prt * 16 + acc_row(e), i = j * 16 + acc_col();
        sE[r * LDE + i] += ea[j][e];
      }
  }
  __syncthreads();
  for (int idx = tid; idx < CH * CH; idx += NTH) {
    const int r = idx >> 6, i = idx & 63;
    sDD[r * LDC + i] = to_e<E>(sD[r * LDE + i] + sD[i * LDE + r]);
  }
  if (tid < CH) {
    float s = 0.f;
    for (int i = 0; i < CH; ++i) s += sE[tid * LDE + i];
    sErow[tid] = s;
  } else if (tid < 2 * CH) {
    const int col = tid - CH;
    float s = 0.f;
    for (int j = 0; j < CH; ++j) s += sE[j * LDE + col];
    sEcol[col] = s;
  }
  __syncthreads();

  // dQ and dK
#pragma unroll
  for (int i = 0; i < RTW; ++i)
#pragma unroll
    for (int j = 0; j < CTW; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = (wr * RTW + i) * 16 + acc_row(e);
        Gq[i][j][e] *= seg[r];
        Gk[i][j][e] = sdec[r] * Gs[i][j][e] - sb[r] * seg[r] * Gk[i][j][e];
      }
  {
    const E* Bk = sKT + wc * CTW * 16 * LDC;
    const E* Bq = sQT + wc * CTW * 16 * LDC;
    wave_mma_nt<E, RTW, CTW, CH>(Gq, sM1 + wr * RTW * 16 * LDC, LDC, Bk, LDC);
    wave_mma_nt<E, RTW, CTW, CH>(Gk, sM1T + wr * RTW * 16 * LDC, LDC, Bq, LDC);
    wave_mma_nt<E, RTW, CTW, CH>(Gk, sDD + wr * RTW * 16 * LDC, LDC, Bk, LDC);
  }
  {
    E* gdq = (E*)a.dq + row0 * DK;
    E* gdk = (E*)a.dk + row0 * DK;
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
      for (int j = 0; j < CTW; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = (wr * RTW + i) * 16 + acc_row(e);
          const int d = (wc * CTW + j) * 16 + acc_col();
          if (r < len) {
            gdq[(size_t)r * H * DK + d] = to_e<E>(Gq[i][j][e]);
            gdk[(size_t)r * H * DK + d] = to_e<E>(Gk[i][j][e]);
          }
        }
  }

  // dbeta, dg, dlog_alpha (one wave, one lane per chunk position)
  if (w == 0) {
    const int r = lane_id();
    float pq = 0.f, pk = 0.f, ps = 0.f;
#pragma unroll
    for (int x = 0; x < WC; ++x) {
      pq += srow[x][0][r];
      pk += srow[x][1][r];
      ps += srow[x][2][r];
    }
    float s_dot = 0.f;
#pragma unroll
    for (int x = 0; x < 8; ++x) s_dot += sred[x];
    const bool valid = r < len;
    const float eg = seg[r], b = sb[r], dec = sdec[r];
    float dg = eg * pq - b * eg * pk - dec * ps + sErow[r] - sEcol[r];
    const float db = sdbA[r] + sxv[r] - eg * pk;
    float tail = valid ? dec * ps : 0.f;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) tail += __shfl_xor(tail, off, 64);
    const float gn = __shfl(sg[r], len - 1, 64);
    if (r == len - 1) dg += tail + __expf(gn) * s_dot;
    if (!valid) dg = 0.f;
    // reverse inclusive scan: lane r receives sum_{r' >= r} dg_r'
    const float rev = __shfl(dg, 63 - r, 64);
    const float sc = wave_incl_scan(rev);
    const float dla = __shfl(sc, 63 - r, 64);
    if (valid) {
      a.dbeta[row0 + (size_t)r * H] = db;
      a.dlog_alpha[row0 + (size_t)r * H] = dla;
    }
  }
}

// ------------------------------------------------------------------ launchers

template <class E, int DK, int DV>
struct Cfg {
  static constexpr int BV = (sizeof(E) == 2 && DK == 256) ? 32 : 64;
  static constexpr int BVG = (sizeof(E) == 2 && DK == 256) ? 32 : 64;
};

static hipError_t table(const Args& a, hipStream_t s) {
  hipLaunchKernelGGL(k_chunk_table, dim3(1), dim3(256), 0, s, a.cu, a.N, a.T, a.info,
                     a.seq_chunk0);
  return hipGetLastError();
}

template <class E, int DK, int DV>
static hipError_t fwd_impl(const Args& a, hipStream_t s) {
  using C = Cfg<E, DK, DV>;
  hipError_t e = table(a, s);
  if (e != hipSuccess) return e;
  if (a.NC > 0) {
    hipLaunchKernelGGL((k_prep<E, DK>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, C::BV, false>), dim3(DV / C::BV, a.H, a.N), dim3(256),
                     0, s, a);
  return hipGetLastError();
}

template <class E, int DK, int DV>
static hipError_t bwd_impl(const Args& a, hipStream_t s) {
  using C = Cfg<E, DK, DV>;
  hipError_t e = table(a, s);
  if (e != hipSuccess) return e;
  if (a.NC > 0) {
    hipLaunchKernelGGL((k_prep<E, DK>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL((k_fwd_seq<E, DK, DV, C::BV, true>), dim3(DV / C::BV, a.H, a.N), dim3(256),
                     0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((k_bwd_seq<E, DK, DV, C::BV>), dim3(DV / C::BV, a.H, a.N), dim3(256), 0, s,
                     a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (a.NC > 0) {
    hipLaunchKernelGGL((k_grad<E, DK, DV, C::BVG>), dim3(a.NC, a.H), dim3(512), 0, s, a);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s) {
  if (dt == Dt::F32 && dk == 64 && dv == 64) return fwd_impl<float, 64, 64>(a, s);
  if (dt == Dt::BF16 && dk == 64 && dv == 64) return fwd_impl<bf16, 64, 64>(a, s);
  if (dt == Dt::BF16 && dk == 128 && dv == 128) return fwd_impl<bf16, 128, 128>(a, s);
  if (dt == Dt::BF16 && dk == 256 && dv == 512) return fwd_impl<bf16, 256, 512>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_bwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s) {
  if (dt == Dt::F32 && dk == 64 && dv == 64) return bwd_impl<float, 64, 64>(a, s);
  if (dt == Dt::BF16 && dk == 64 && dv == 64) return bwd_impl<bf16, 64, 64>(a, s);
  if (dt == Dt::BF16 && dk == 128 && dv == 128) return bwd_impl<bf16, 128, 128>(a, s);
  if (dt == Dt::BF16 && dk == 256 && dv == 512) return bwd_impl<bf16, 256, 512>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace gdn

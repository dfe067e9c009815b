// Parallel per-chunk preparation kernels (gfx950) of the chunkwise gated
// delta rule.  Chunk algebra (Sec. 3.3 of the paper; state stored dk x dv,
// the transpose of the paper's dv x dk state), for one chunk of n <= 64
// tokens with beta b and cumulative log gate g (restarted at every chunk,
// Sec. 2.1 footnote):
//   Gamma_ri = exp(g_r - g_i) for i <= r          (decay-aware causal mask)
//   A  = strictLower(diag(b) (Gamma * K K^T)),   T = (I + A)^-1
//   W~ = T diag(b e^g) K,   U~ = T diag(b) V       (gated UT transform)
//   P  = Gamma * Q K^T   (lower, with the diagonal)
// With these, for entry state S:  V' = U~ - W~ S,
//   O = diag(e^g) Q S + P V' = Qeff S + P U~   (Qeff = diag(e^g) Q - P W~),
//   S_next = e^{g_n} S + Kbar^T V'             (Kbar = diag(e^{g_n - g}) K).
// W~ is the paper's decayed W (decay on the left of the ungated UT
// transform) rewritten with the gated inverse: diag(e^g) (I + A_u)^-1 =
// (I + A_g)^-1 diag(e^g) when A_g = diag(e^g) A_u diag(e^-g).  The output
// mask is Gamma; the plain causal mask printed in the gated output equation
// does not reproduce the recurrence.
//
//   k_chunk_table  chunk -> (sequence, first row, length)
//   k_prep_a       g, Ak, P, T per (chunk, head)                     (fp32)
//   k_prep_w       W~, Kbar^T, and Qeff (forward) or -W~^T, (e^g Q)^T, T^T
//                  (backward) in MFMA A-fragment layout
//   k_prep_u       U~, and P U~ (forward) or P^T dO (backward) in
//                  accumulator layout, per 64-wide block of dv
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {


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
__global__ __launch_bounds__(256) void k_prep_a(Args a) {
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
  lds_barrier();

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
  lds_barrier();

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
  lds_barrier();
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
    lds_barrier();
    for (int J = 0; J + d < 4; ++J) {
      const int I = J + d;
      float t = 0.f;
#pragma unroll
      for (int l = 0; l < 16; ++l) t -= sT[(16 * I + i) * LDA + 16 * I + l] * sY[J * 272 + l * 17 + j];
      sT[(16 * I + i) * LDA + 16 * J + j] = t;
    }
    lds_barrier();
  }
  float* gT = a.Tm + ch * CH * CH;
  for (int idx = tid; idx < CH * CH; idx += 256) {
    const int r = idx >> 6, i = idx & 63;
    gT[idx] = ((i >> 4) > (r >> 4)) ? 0.f : sT[r * LDA + i];
  }
}

// ------------------------------------------------------------------ W~ and friends
// Grid (NC, H), 256 threads.

template <class E, int DK, bool FWD>
__global__ __launch_bounds__(256) void k_prep_w(Args a) {
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDK = DK + PADE;  // [64][LDK]: rows of K, Q, W~
  constexpr int LDC = CH + PADE;  // [..][LDC]: token-indexed rows
  constexpr int NCT = DK / 16;
  constexpr int XSZ = (DK * LDC > CH * LDK) ? DK * LDC : CH * LDK;
  __shared__ __align__(16) E sTe[CH * LDC];
  __shared__ __align__(16) E sPe[FWD ? CH * LDC : 1];
  __shared__ __align__(16) E sK[CH * LDK];  // K rows, later W~ rows
  __shared__ __align__(16) E sX[XSZ];       // (b e^g K)^T, later Q rows (Qeff in place)
  __shared__ __align__(16) E sWT[DK * LDC]; // W~^T
  __shared__ float sdec[CH], sbeg[CH], seg[CH];

  const int c = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, w = wave_id();
  const int H = a.H;
  const int4 ci = a.info[c];
  const int start = ci.y, len = ci.z;
  const size_t ch = (size_t)c * H + h;
  const size_t row0 = (size_t)start * H + h;
  const E* K = (const E*)a.k + row0 * DK;
  const E* Q = (const E*)a.q + row0 * DK;

  stage_rows<E, CH, DK, LDK, 256>(sK, K, (size_t)H * DK, len);
  stage_mat64<E, LDC, 256, false>(sTe, a.Tm + ch * CH * CH);
  if (FWD) stage_mat64<E, LDC, 256, false>(sPe, a.Pm + ch * CH * CH);
  if (tid < CH) {
    const float g = a.g[ch * CH + tid];
    const float gn = __shfl(g, len - 1, 64);
    const float b = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
    const float eg = __expf(g);
    seg[tid] = eg;
    sdec[tid] = __expf(gn - g);
    sbeg[tid] = b * eg;
  }
  lds_barrier();

  export_afrag<E, DK, CH, 256>((E*)a.KbT + ch * DK * CH, [&](int d, int t) {
    return sdec[t] * to_f(sK[t * LDK + d]);
  });
  for (int idx = tid; idx < DK * CH; idx += 256) {
    const int t = idx & (CH - 1), d = idx >> 6;
    sX[d * LDC + t] = to_e<E>(sbeg[t] * to_f(sK[t * LDK + d]));
  }
  lds_barrier();

  // W~ = T (b e^g K): wave w owns rows 16w..16w+15
  f32x4 W[1][NCT];
  zero_acc(W);
  wave_mma_nt<E, 1, NCT, CH>(W, sTe + w * 16 * LDC, LDC, sX, LDC);
#pragma unroll
  for (int j = 0; j < NCT; ++j) {
    store_tile_T<E>(sWT, LDC, W[0][j], w * 16, j * 16);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      sK[(w * 16 + acc_row(e)) * LDK + j * 16 + acc_col()] = to_e<E>(W[0][j][e]);
  }
  lds_barrier();
  export_afrag<E, CH, DK, 256>((E*)a.Wf + ch * CH * DK,
                               [&](int t, int d) { return to_f(sK[t * LDK + d]); });
  if (FWD) {
    stage_rows<E, CH, DK, LDK, 256>(sX, Q, (size_t)H * DK, len);
    lds_barrier();
    f32x4 Qe[1][NCT];
    zero_acc(Qe);
    wave_mma_nt<E, 1, NCT, CH>(Qe, sPe + w * 16 * LDC, LDC, sWT, LDC);
#pragma unroll
    for (int j = 0; j < NCT; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = w * 16 + acc_row(e), d = j * 16 + acc_col();
        E& x = sX[r * LDK + d];  // each lane rewrites exactly the elements it reads
        x = to_e<E>(seg[r] * to_f(x) - Qe[0][j][e]);
      }
    lds_barrier();
    export_afrag<E, CH, DK, 256>((E*)a.Qf + ch * CH * DK,
                                 [&](int t, int d) { return to_f(sX[t * LDK + d]); });
  } else {
    export_afrag<E, DK, CH, 256>((E*)a.nWT + ch * DK * CH,
                                 [&](int d, int t) { return -to_f(sWT[d * LDC + t]); });
    export_afrag<E, CH, CH, 256>((E*)a.TT + ch * CH * CH,
                                 [&](int t, int i) { return to_f(sTe[i * LDC + t]); });
    stage_rows<E, CH, DK, LDK, 256>(sX, Q, (size_t)H * DK, len);
    lds_barrier();
    export_afrag<E, DK, CH, 256>((E*)a.QgT + ch * DK * CH, [&](int d, int t) {
      return seg[t] * to_f(sX[t * LDK + d]);
    });
  }
}

// ------------------------------------------------------------------ U~ and friends
// Grid (NC, H, DV / 64), 256 threads: one 64-wide block of dv.

template <class E, int DV, bool FWD>
__global__ __launch_bounds__(256) void k_prep_u(Args a) {
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LDC = CH + PADE;
  constexpr int VB = 64;
  __shared__ __align__(16) E sTe[CH * LDC];
  __shared__ __align__(16) E sPx[CH * LDC];  // P (forward) or P^T (backward)
  __shared__ __align__(16) E sVT[VB * LDC];  // (b V)^T block
  __shared__ __align__(16) E sYT[VB * LDC];  // U~^T (forward) or dO^T (backward)
  __shared__ float sb[CH];

  const int c = blockIdx.x, h = blockIdx.y, v0 = blockIdx.z * VB;
  const int tid = threadIdx.x, w = wave_id();
  const int H = a.H;
  const int4 ci = a.info[c];
  const int start = ci.y, len = ci.z;
  const size_t ch = (size_t)c * H + h;
  const size_t row0 = (size_t)start * H + h;

  stage_mat64<E, LDC, 256, false>(sTe, a.Tm + ch * CH * CH);
  if (FWD)
    stage_mat64<E, LDC, 256, false>(sPx, a.Pm + ch * CH * CH);
  else
    stage_mat64<E, LDC, 256, true>(sPx, a.Pm + ch * CH * CH);
  if (tid < CH) sb[tid] = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
  lds_barrier();
  stage_rows_T<E, VB, LDC, 256>(sVT, (const E*)a.v + row0 * DV + v0, (size_t)H * DV, len, sb);
  if (!FWD)
    stage_rows_T<E, VB, LDC, 256>(sYT, (const E*)a.dO + row0 * DV + v0, (size_t)H * DV, len,
                                  nullptr);
  lds_barrier();
  f32x4 U[1][4];
  zero_acc(U);
  wave_mma_nt<E, 1, 4, CH>(U, sTe + w * 16 * LDC, LDC, sVT, LDC);
  E* gU = (E*)a.Uc + ch * CH * DV;
#pragma unroll
  for (int j = 0; j < 4; ++j) store4<E>(gU + cfrag_index(w, v0 / 16 + j, DV), U[0][j]);
  f32x4 Y[1][4];
  zero_acc(Y);
  if (FWD) {
#pragma unroll
    for (int j = 0; j < 4; ++j) store_tile_T<E>(sYT, LDC, U[0][j], w * 16, j * 16);
    lds_barrier();
  }
  wave_mma_nt<E, 1, 4, CH>(Y, sPx + w * 16 * LDC, LDC, sYT, LDC);
  E* gY = (E*)(FWD ? a.Oc : a.dVi) + ch * CH * DV;
#pragma unroll
  for (int j = 0; j < 4; ++j) store4<E>(gY + cfrag_index(w, v0 / 16 + j, DV), Y[0][j]);
}

// ------------------------------------------------------------------ launchers

hipError_t launch_chunk_table(const Args& a, hipStream_t s) {
  hipLaunchKernelGGL(k_chunk_table, dim3(1), dim3(256), 0, s, a.cu, a.N, a.T, a.info,
                     a.seq_chunk0);
  return hipGetLastError();
}

hipError_t launch_prep_a(Dt dt, int dk, int dv, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    hipLaunchKernelGGL((k_prep_a<E, DK>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

hipError_t launch_prep_w(Dt dt, int dk, int dv, bool fwd, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    if (fwd)
      hipLaunchKernelGGL((k_prep_w<E, DK, true>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((k_prep_w<E, DK, false>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

hipError_t launch_prep_u(Dt dt, int dk, int dv, bool fwd, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    if (fwd)
      hipLaunchKernelGGL((k_prep_u<E, DV, true>), dim3(a.NC, a.H, DV / 64), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((k_prep_u<E, DV, false>), dim3(a.NC, a.H, DV / 64), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

}  // namespace gdn

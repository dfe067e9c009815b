// Per-chunk gradient kernel (gfx950) of the chunkwise gated delta rule: the
// parallel part of the backward, given every chunk's entry state S, exit-state
// gradient dS_next, V' and dX from the two sequential passes.  The paper gives
// no backward; these are the exact reverse-mode derivatives of its chunk
// equations (Sec. 3.3, state stored dk x dv).
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {

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
    lds_barrier();
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
    lds_barrier();
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
  lds_barrier();

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
  lds_barrier();
  if (pm == 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = prt * 16 + acc_row(e), i = j * 16 + acc_col();
        sE[r * LDE + i] += ea[j][e];
      }
  }
  lds_barrier();
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
  lds_barrier();

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


hipError_t launch_grad(Dt dt, int dk, int dv, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    constexpr int BVG = (sizeof(E) == 2 && DK == 256) ? 32 : 64;
    hipLaunchKernelGGL((k_grad<E, DK, DV, BVG>), dim3(a.NC, a.H), dim3(512), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

}  // namespace gdn

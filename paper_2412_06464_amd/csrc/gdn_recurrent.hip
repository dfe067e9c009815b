// Token-by-token (recurrent) form of the gated delta rule (gfx950): the
// inference path, one token at a time (Sec. 3.1, Eq. gated_delta_rule),
// with the state stored dk x dv:
//   u = S^T k,   w = S^T q,   r = v - alpha u,
//   S <- alpha S + beta k r^T,   o = S^T q = alpha w + beta (k . q) r.
// One workgroup owns one (sequence, head, 64-wide slice of dv).  Its fp32
// state slice stays in registers from the first token to the last (thread
// (rg, cg) holds rows rg + 16 i, columns 4 cg .. 4 cg + 3), so HBM sees the
// state once in and once out whatever the number of tokens; a single decode
// step is the case T = 1.  Per token the two contractions over dk are reduced
// across the 16 row groups by shuffles inside a wave and through LDS across
// the four waves.  The state may be updated in place (h0 == ht): every
// workgroup reads its slice before it writes it and no other workgroup
// touches that slice.
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {

template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void k_recurrent(Args a) {
  constexpr int BV = 64, NR = DK / 16, NVT = DV / BV;
  __shared__ float skq[2][2][DK];      // k, q of the token, double-buffered
  __shared__ float sred[2][4][3][BV];  // per-wave partial u, w and k.q, double-buffered
  const int tid = threadIdx.x, l = lane_id(), w = wave_id();
  const int cg = tid & 15, rg = tid >> 4;
  const int unit = blockIdx.x / NVT, vt = blockIdx.x - unit * NVT;
  const int H = a.H, n = unit / H, h = unit - n * H;
  const int c0 = 4 * cg, v0 = vt * BV + c0;
  const int s0 = a.cu ? a.cu[n] : n * a.T;
  const int L = a.cu ? a.cu[n + 1] - s0 : a.T;
  const size_t sbase = ((size_t)n * H + h) * DK * DV;
  const E* Q = (const E*)a.q;
  const E* K = (const E*)a.k;
  const E* V = (const E*)a.v;
  E* O = (E*)a.o;

  f32x4 S[NR];
#pragma unroll
  for (int i = 0; i < NR; ++i)
    S[i] = a.h0 ? *reinterpret_cast<const f32x4*>(a.h0 + sbase + (size_t)(rg + 16 * i) * DV + v0)
                : f32x4{0.f, 0.f, 0.f, 0.f};

  for (int t = 0; t < L; ++t) {
    const size_t row = (size_t)(s0 + t) * H + h;
    const int buf = t & 1;
    for (int x = tid; x < DK; x += 256) {
      skq[buf][0][x] = to_f(K[row * DK + x]);
      skq[buf][1][x] = to_f(Q[row * DK + x]);
    }
    const f32x4 vv = load4<E>(V + row * DV + v0);
    const float b = a.beta[row];
    const float al = a.gated ? __expf(a.log_alpha[row]) : 1.f;
    lds_barrier();

    // partial S^T k, S^T q and k . q over this thread's rows
    float pu[4] = {0.f, 0.f, 0.f, 0.f}, pw[4] = {0.f, 0.f, 0.f, 0.f}, pkq = 0.f;
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const float kd = skq[buf][0][rg + 16 * i], qd = skq[buf][1][rg + 16 * i];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        pu[c] += kd * S[i][c];
        pw[c] += qd * S[i][c];
      }
      pkq += kd * qd;
    }
    // the wave's four row groups differ in lane bits 4 and 5
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      pu[c] += __shfl_xor(pu[c], 16, 64);
      pu[c] += __shfl_xor(pu[c], 32, 64);
      pw[c] += __shfl_xor(pw[c], 16, 64);
      pw[c] += __shfl_xor(pw[c], 32, 64);
    }
    pkq += __shfl_xor(pkq, 16, 64);
    pkq += __shfl_xor(pkq, 32, 64);
    if (l < 16) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        sred[buf][w][0][c0 + c] = pu[c];
        sred[buf][w][1][c0 + c] = pw[c];
      }
      sred[buf][w][2][c0] = pkq;
    }
    lds_barrier();

    float u[4], wq[4], kq = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c) u[c] = wq[c] = 0.f;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        u[c] += sred[buf][x][0][c0 + c];
        wq[c] += sred[buf][x][1][c0 + c];
      }
      kq += sred[buf][x][2][c0];
    }
    f32x4 r, o;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      r[c] = vv[c] - al * u[c];
      o[c] = al * wq[c] + b * kq * r[c];
    }
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      const float bk = b * skq[buf][0][rg + 16 * i];
#pragma unroll
      for (int c = 0; c < 4; ++c) S[i][c] = al * S[i][c] + bk * r[c];
    }
    if (rg == 0) store4<E>(O + row * DV + v0, o);
  }

  if (a.ht) {
#pragma unroll
    for (int i = 0; i < NR; ++i)
      *reinterpret_cast<f32x4*>(a.ht + sbase + (size_t)(rg + 16 * i) * DV + v0) = S[i];
  }
}

hipError_t launch_recurrent(Dt dt, int dk, int dv, const Args& a, hipStream_t s) {
  auto f = [&]<class E, int DK, int DV>() {
    hipLaunchKernelGGL((k_recurrent<E, DK, DV>), dim3(a.N * a.H * (DV / 64)), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

}  // namespace gdn

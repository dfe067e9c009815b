// Block prologue and epilogue of Gated DeltaNet (gfx950): the operations the
// block design wraps around the rule (Sec. 3.4 and the block-design figure).
//
// Prologue, per channel c of a [*, T, H, D] tensor (q, k: with L2; v: without):
//   u_t[c] = sum_{j < W} w[c][W-1-j] x_{t-j}[c]     (causal, depthwise, width W;
//            zero before the sequence start)
//   z_t = silu(u_t),   y_t = z_t / sqrt(|z_t|^2 + eps)   (or y_t = z_t)
// Epilogue, per (token, head) row of the output over its dv channels:
//   y = o / sqrt(mean(o^2) + eps) * w * silu(g)
// Both are memory-bound row operations.  One wave owns whole rows (the L2 and
// RMS sums are wave reductions); each lane holds D/64 consecutive channels.
// Weight gradients are reduced deterministically: per-workgroup partial sums
// in the workspace, then a fixed-order sum over the workgroups.
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {

namespace {

// N consecutive elements of one row as loaded (two 16-byte loads at most),
// and their fp32 values.
struct Raw32 {
  uint4 lo, hi;
};
template <int BYTES> struct RawT;
template <> struct RawT<32> { using type = Raw32; };
template <> struct RawT<16> { using type = uint4; };
template <> struct RawT<8> { using type = uint2; };
template <> struct RawT<4> { using type = unsigned; };
template <> struct RawT<2> { using type = unsigned short; };

template <class E, int N>
struct RowRaw {
  using T = typename RawT<N * (int)sizeof(E)>::type;
  T r;
  __device__ inline void load(const E* p) { r = *reinterpret_cast<const T*>(p); }
  __device__ inline void zero() { r = T{}; }
  __device__ inline void to_float(float (&v)[N]) const {
    union {
      T u;
      E e[N];
    } t;
    t.u = r;
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = to_f(t.e[i]);
  }
};

template <class E, int N>
struct RowPiece {
  float v[N];
  __device__ inline void load(const E* p) {
    if constexpr (N * sizeof(E) <= 16) {
      RowRaw<E, N> t;
      t.load(p);
      t.to_float(v);
    } else {
#pragma unroll
      for (int i = 0; i < N; ++i) v[i] = to_f(p[i]);
    }
  }
  __device__ inline void zero() {
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = 0.f;
  }
};

template <class E, int N>
__device__ inline void store_piece(E* p, const float (&v)[N]) {
  union {
    E e[N];
    unsigned char b[N * sizeof(E)];
  } t;
#pragma unroll
  for (int i = 0; i < N; ++i) t.e[i] = to_e<E>(v[i]);
  if constexpr (sizeof(t) == 16 || sizeof(t) == 8 || sizeof(t) == 4) {
    store_stream_small(p, t);
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) p[i] = t.e[i];
  }
}

// Sum over the 64 lanes of a wave (every lane gets it).
__device__ inline float wave_sum(float x) {
  x = reduce16(x);
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

}  // namespace

// ------------------------------------------------------------------ prologue

// One workgroup per (chunk, head); wave w owns rows 16 w .. 16 w + 15 of the
// chunk.  The three rows before each wave's first row come from the previous
// chunk of the same sequence (or are zero at the sequence start).
// D: channels of the tensor; DL: channels of one workgroup (D, or a slice of
// it when the rows need no L2 sum).
template <class E, int D, int DL>
__global__ __launch_bounds__(256) void k_conv_fwd(ConvArgs a) {
  constexpr int CPL = DL / 64, NR = 16 + 3;
  const int c = blockIdx.x, h = blockIdx.y, w = wave_id(), l = lane_id();
  const int4 ci = a.info[c];
  const int n = ci.x, start = ci.y, len = ci.z;
  const int s0 = a.cu ? a.cu[n] : n * a.T;
  const int pos0 = start - s0, r0 = 16 * w, H = a.H;
  if (r0 >= len) return;
  const int ch = blockIdx.z * DL + l * CPL;
  float wl[CPL][4];  // weight of lag j (x_{t-j}); zero for j >= W
#pragma unroll
  for (int k = 0; k < CPL; ++k)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      wl[k][j] = j < a.W ? a.w[(size_t)(h * D + ch + k) * a.W + (a.W - 1 - j)] : 0.f;
  const E* X = (const E*)a.x;
  RowRaw<E, CPL> xr[NR];  // rows r0 - 3 .. r0 + 15, all loads issued up front
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    const int r = r0 - 3 + i;
    if (pos0 + r >= 0 && r < len)
      xr[i].load(X + ((size_t)(start + r) * H + h) * D + ch);
    else
      xr[i].zero();
  }
  float xw[4][CPL];  // x_{t-3} .. x_t
#pragma unroll
  for (int i = 0; i < 3; ++i) xr[i].to_float(xw[i + 1]);
  E* Y = (E*)a.y;
#pragma unroll
  for (int i = 3; i < NR; ++i) {
    const int r = r0 - 3 + i;
    if (r >= len) break;  // uniform over the wave
#pragma unroll
    for (int q = 0; q < 3; ++q)
#pragma unroll
      for (int k = 0; k < CPL; ++k) xw[q][k] = xw[q + 1][k];
    xr[i].to_float(xw[3]);
    float z[CPL], ss = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      const float u = wl[k][0] * xw[3][k] + wl[k][1] * xw[2][k] + wl[k][2] * xw[1][k] +
                      wl[k][3] * xw[0][k];
      z[k] = u * sigmoidf(u);
      ss += z[k] * z[k];
    }
    if (a.l2) {
      const float sc = rsqrtf(wave_sum(ss) + a.eps);
#pragma unroll
      for (int k = 0; k < CPL; ++k) z[k] *= sc;
    }
    store_piece<E, CPL>(Y + ((size_t)(start + r) * H + h) * D + ch, z);
  }
}

// Backward.  Wave w owns rows 16 w .. 16 w + 15, taken in passes of RP rows.
// A pass walks its rows and the three after them (which may lie in the next
// chunk of the same sequence), recomputing du_t, so that
// dx_s = sum_j w_lag(j) du_{s+j} is complete for its own rows; dw is summed
// over own rows only.  x, du: 4-row sliding windows; raw rows prefetched.
template <class E, int D, int DL>
__global__ __launch_bounds__(256) void k_conv_bwd(ConvArgs a) {
  constexpr int CPL = DL / 64;
  constexpr int RP = 8;  // rows per pass
  constexpr int NX = RP + 6, NG = RP + 3;
  __shared__ float sdw[4][DL][4];
  const int c = blockIdx.x, h = blockIdx.y, w = wave_id(), l = lane_id();
  const int4 ci = a.info[c];
  const int n = ci.x, start = ci.y, len = ci.z;
  const int s0 = a.cu ? a.cu[n] : n * a.T;
  const int L = a.cu ? a.cu[n + 1] - s0 : a.T;
  const int pos0 = start - s0, H = a.H;
  const int cl = l * CPL, ch = blockIdx.z * DL + cl;
  float wl[CPL][4];
#pragma unroll
  for (int k = 0; k < CPL; ++k)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      wl[k][j] = j < a.W ? a.w[(size_t)(h * D + ch + k) * a.W + (a.W - 1 - j)] : 0.f;
  float dwp[CPL][4];
#pragma unroll
  for (int k = 0; k < CPL; ++k)
#pragma unroll
    for (int j = 0; j < 4; ++j) dwp[k][j] = 0.f;
  const E* X = (const E*)a.x;
  const E* DY = (const E*)a.dy;
  E* DX = (E*)a.dx;

  for (int r0 = 16 * w; r0 < 16 * w + 16 && r0 < len; r0 += RP) {
    RowRaw<E, CPL> xr[NX], gr[NG];  // x rows r0-3 .. r0+RP+2, dy rows r0 .. r0+RP+2
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const int r = r0 - 3 + i, p = pos0 + r;
      if (p >= 0 && p < L)
        xr[i].load(X + ((size_t)(start + r) * H + h) * D + ch);
      else
        xr[i].zero();
    }
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int r = r0 + i;
      if (pos0 + r < L)
        gr[i].load(DY + ((size_t)(start + r) * H + h) * D + ch);
      else
        gr[i].zero();
    }
    float xw[4][CPL], dw4[4][CPL];  // x_{t-3} .. x_t;  du_{t-3} .. du_t
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int k = 0; k < CPL; ++k) xw[q][k] = dw4[q][k] = 0.f;
#pragma unroll
    for (int i = 0; i < 3; ++i) xr[i].to_float(xw[i + 1]);
#pragma unroll
    for (int i = 0; i < NG; ++i) {
      const int r = r0 + i;
      const bool valid = pos0 + r < L;  // uniform over the wave
#pragma unroll
      for (int q = 0; q < 3; ++q)
#pragma unroll
        for (int k = 0; k < CPL; ++k) {
          xw[q][k] = xw[q + 1][k];
          dw4[q][k] = dw4[q + 1][k];
        }
      xr[i + 3].to_float(xw[3]);
      float gy[CPL], u[CPL], z[CPL], sg[CPL], ss = 0.f, zg = 0.f;
      gr[i].to_float(gy);
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        u[k] = wl[k][0] * xw[3][k] + wl[k][1] * xw[2][k] + wl[k][2] * xw[1][k] + wl[k][3] * xw[0][k];
        sg[k] = sigmoidf(u[k]);
        z[k] = u[k] * sg[k];
        ss += z[k] * z[k];
        zg += z[k] * gy[k];
      }
      float sc = 1.f, yg = 0.f;
      if (a.l2) {
        sc = rsqrtf(wave_sum(ss) + a.eps);  // 1 / |z|
        yg = wave_sum(zg) * sc;             // y . dy
      }
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const float dz = a.l2 ? (gy[k] - z[k] * sc * yg) * sc : gy[k];
        dw4[3][k] = valid ? dz * sg[k] * (1.f + u[k] * (1.f - sg[k])) : 0.f;
      }
      if (i < RP && r < len) {  // own row: dw over x_{t-j}
#pragma unroll
        for (int k = 0; k < CPL; ++k)
#pragma unroll
          for (int j = 0; j < 4; ++j) dwp[k][j] += dw4[3][k] * xw[3 - j][k];
      }
      if (i >= 3 && r - 3 < len) {  // dx of row r - 3 is complete
        float dx[CPL];
#pragma unroll
        for (int k = 0; k < CPL; ++k)
          dx[k] = wl[k][0] * dw4[0][k] + wl[k][1] * dw4[1][k] + wl[k][2] * dw4[2][k] +
                  wl[k][3] * dw4[3][k];
        store_piece<E, CPL>(DX + ((size_t)(start + r - 3) * H + h) * D + ch, dx);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < CPL; ++k)
#pragma unroll
    for (int j = 0; j < 4; ++j) sdw[w][cl + k][j] = dwp[k][j];
  __syncthreads();
  // this workgroup's partial dw[h][ch][tap], in the order of the weights
  float* part = a.part + (((size_t)c * H + h) * D + blockIdx.z * DL) * a.W;
  for (int idx = threadIdx.x; idx < DL * a.W; idx += 256) {
    const int cc = idx / a.W, tap = idx - cc * a.W, j = a.W - 1 - tap;
    part[idx] = sdw[0][cc][j] + sdw[1][cc][j] + sdw[2][cc][j] + sdw[3][cc][j];
  }
}

// out[y * M + m] = sum of in[i * M + m] over the rows i of slice y (rows
// [y * RS, (y + 1) * RS) of N), in a fixed order: thread (m, seg) sums rows
// seg, seg + 16, ... of the slice, then the 16 partial sums are added in order.
constexpr int SUM_RS = 256;  // rows per slice
__global__ __launch_bounds__(256) void k_sum_rows(const float* in, int N, int M, float* out) {
  __shared__ float s[16][17];
  const int ml = threadIdx.x & 15, seg = threadIdx.x >> 4, m = blockIdx.x * 16 + ml;
  const int i0 = blockIdx.y * SUM_RS, i1 = min(N, i0 + SUM_RS);
  float acc = 0.f;
  if (m < M)
    for (int i = i0 + seg; i < i1; i += 16) acc += in[(size_t)i * M + m];
  s[seg][ml] = acc;
  __syncthreads();
  if (seg == 0 && m < M) {
    float t = 0.f;
#pragma unroll
    for (int x = 0; x < 16; ++x) t += s[x][ml];
    out[(size_t)blockIdx.y * M + m] = t;
  }
}

// dw = sum over the N rows of part [N][M]: slices of SUM_RS rows summed in
// parallel into tmp [NS][M] (NS = slices), then the NS slice sums in order.
// tmp may be null when N <= SUM_RS.  Deterministic for a given N.
hipError_t launch_sum_rows(const float* part, int N, int M, float* tmp, float* out,
                           hipStream_t s) {
  const int NS = (N + SUM_RS - 1) / SUM_RS;
  if (NS <= 1) {
    hipLaunchKernelGGL(k_sum_rows, dim3((M + 15) / 16, 1), dim3(256), 0, s, part, N, M, out);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_sum_rows, dim3((M + 15) / 16, NS), dim3(256), 0, s, part, N, M, tmp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sum_rows, dim3((M + 15) / 16, 1), dim3(256), 0, s, tmp, NS, M, out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ epilogue

// Rows are (token, head) pairs; wave w of workgroup b owns rows
// 64 b + 16 w .. 64 b + 16 w + 15.
template <class E, int DV>
__global__ __launch_bounds__(256) void k_norm_gate_fwd(NormArgs a) {
  constexpr int CPL = DV / 64;
  const int l = lane_id(), ch = l * CPL;
  const long r0 = (long)blockIdx.x * 64 + 16 * wave_id();
  RowPiece<float, CPL> wt;
  wt.load(a.w + ch);
  // one row ahead: the next row's loads are in flight while this one computes
  const int nr = (int)min(16L, max(0L, a.rows - r0));
  RowRaw<E, CPL> on, gn;
  if (nr > 0) {
    on.load((const E*)a.o + r0 * DV + ch);
    gn.load((const E*)a.g + r0 * DV + ch);
  }
  for (int i = 0; i < nr; ++i) {
    const long r = r0 + i;
    RowPiece<E, CPL> o, g;
    on.to_float(o.v);
    gn.to_float(g.v);
    if (i + 1 < nr) {
      on.load((const E*)a.o + (r + 1) * DV + ch);
      gn.load((const E*)a.g + (r + 1) * DV + ch);
    }
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) ss += o.v[k] * o.v[k];
    const float rs = rsqrtf(wave_sum(ss) / DV + a.eps);
    float y[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) y[k] = o.v[k] * rs * wt.v[k] * (g.v[k] * sigmoidf(g.v[k]));
    store_piece<E, CPL>((E*)a.y + r * DV + ch, y);
  }
}

template <class E, int DV>
__global__ __launch_bounds__(256) void k_norm_gate_bwd(NormArgs a) {
  constexpr int CPL = DV / 64;
  __shared__ float sdw[4][DV];
  const int l = lane_id(), w = wave_id(), ch = l * CPL;
  const long r0 = (long)blockIdx.x * 64 + 16 * w;
  RowPiece<float, CPL> wt;
  wt.load(a.w + ch);
  float dwp[CPL];
#pragma unroll
  for (int k = 0; k < CPL; ++k) dwp[k] = 0.f;
  // one row ahead: the next row's loads are in flight while this one computes
  const int nr = (int)min(16L, max(0L, a.rows - r0));
  RowRaw<E, CPL> on, gn, dn;
  if (nr > 0) {
    on.load((const E*)a.o + r0 * DV + ch);
    gn.load((const E*)a.g + r0 * DV + ch);
    dn.load((const E*)a.dy + r0 * DV + ch);
  }
  for (int i = 0; i < nr; ++i) {
    const long r = r0 + i;
    RowPiece<E, CPL> o, g, dy;
    on.to_float(o.v);
    gn.to_float(g.v);
    dn.to_float(dy.v);
    if (i + 1 < nr) {
      on.load((const E*)a.o + (r + 1) * DV + ch);
      gn.load((const E*)a.g + (r + 1) * DV + ch);
      dn.load((const E*)a.dy + (r + 1) * DV + ch);
    }
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) ss += o.v[k] * o.v[k];
    const float rs = rsqrtf(wave_sum(ss) / DV + a.eps);
    float oh[CPL], doh[CPL], dg[CPL], dot = 0.f;
#pragma unroll
    for (int k = 0; k < CPL; ++k) {
      oh[k] = o.v[k] * rs;
      const float s = sigmoidf(g.v[k]), sg = g.v[k] * s;
      dg[k] = dy.v[k] * oh[k] * wt.v[k] * s * (1.f + g.v[k] * (1.f - s));
      const float da = dy.v[k] * sg;
      dwp[k] += da * oh[k];
      doh[k] = da * wt.v[k];
      dot += doh[k] * oh[k];
    }
    dot = wave_sum(dot) / DV;
    float dout[CPL];
#pragma unroll
    for (int k = 0; k < CPL; ++k) dout[k] = rs * (doh[k] - oh[k] * dot);
    store_piece<E, CPL>((E*)a.dout + r * DV + ch, dout);
    store_piece<E, CPL>((E*)a.dg + r * DV + ch, dg);
  }
#pragma unroll
  for (int k = 0; k < CPL; ++k) sdw[w][ch + k] = dwp[k];
  __syncthreads();
  for (int idx = threadIdx.x; idx < DV; idx += 256)
    a.part[(size_t)blockIdx.x * DV + idx] = sdw[0][idx] + sdw[1][idx] + sdw[2][idx] + sdw[3][idx];
}

// ------------------------------------------------------------------ launchers

#define GDN_BLOCK_DISPATCH(dt, d, f)                                                       \
  do {                                                                                     \
    if ((dt) == Dt::F32 && (d) == 64) return (f).template operator()<float, 64>();         \
    if ((dt) == Dt::F32 && (d) == 128) return (f).template operator()<float, 128>();       \
    if ((dt) == Dt::F32 && (d) == 256) return (f).template operator()<float, 256>();       \
    if ((dt) == Dt::F32 && (d) == 512) return (f).template operator()<float, 512>();       \
    if ((dt) == Dt::BF16 && (d) == 64) return (f).template operator()<__bf16, 64>();       \
    if ((dt) == Dt::BF16 && (d) == 128) return (f).template operator()<__bf16, 128>();     \
    if ((dt) == Dt::BF16 && (d) == 256) return (f).template operator()<__bf16, 256>();     \
    if ((dt) == Dt::BF16 && (d) == 512) return (f).template operator()<__bf16, 512>();     \
    return hipErrorInvalidValue;                                                           \
  } while (0)

// Rows without the L2 sum are split over workgroups of at most 256 channels.
hipError_t launch_conv_fwd(Dt dt, int d, const ConvArgs& a, hipStream_t s) {
  auto f = [&]<class E, int D>() {
    if constexpr (D > 256) {
      if (!a.l2) {
        hipLaunchKernelGGL((k_conv_fwd<E, D, 256>), dim3(a.NC, a.H, D / 256), dim3(256), 0, s, a);
        return hipGetLastError();
      }
    }
    hipLaunchKernelGGL((k_conv_fwd<E, D, D>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_BLOCK_DISPATCH(dt, d, f);
}

hipError_t launch_conv_bwd(Dt dt, int d, const ConvArgs& a, hipStream_t s) {
  auto f = [&]<class E, int D>() {
    bool split = false;
    if constexpr (D > 256) split = !a.l2;
    if constexpr (D > 256) {
      if (split)
        hipLaunchKernelGGL((k_conv_bwd<E, D, 256>), dim3(a.NC, a.H, D / 256), dim3(256), 0, s,
                           a);
    }
    if (!split) hipLaunchKernelGGL((k_conv_bwd<E, D, D>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_sum_rows(a.part, a.NC, a.H * D * a.W, a.tmp, a.dw, s);
  };
  GDN_BLOCK_DISPATCH(dt, d, f);
}

hipError_t launch_norm_gate_fwd(Dt dt, int dv, const NormArgs& a, hipStream_t s) {
  auto f = [&]<class E, int DV>() {
    hipLaunchKernelGGL((k_norm_gate_fwd<E, DV>), dim3(a.nblk), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_BLOCK_DISPATCH(dt, dv, f);
}

hipError_t launch_norm_gate_bwd(Dt dt, int dv, const NormArgs& a, hipStream_t s) {
  auto f = [&]<class E, int DV>() {
    hipLaunchKernelGGL((k_norm_gate_bwd<E, DV>), dim3(a.nblk), dim3(256), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_sum_rows(a.part, a.nblk, DV, a.tmp, a.dw, s);
  };
  GDN_BLOCK_DISPATCH(dt, dv, f);
}

}  // namespace gdn

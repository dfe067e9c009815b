// Device pieces of the fused block prologue (Sec. 3.4 and the block-design
// figure): the projections x of q, k and v pass through a short causal
// depthwise convolution and a SiLU, and q and k are then L2-normalised over
// each head's channels.  Per channel, with wl_j the weight of lag j (tap
// width-1-j of the weight row, zero for j >= width) and x zero before the
// sequence's first token:
//   u_t = sum_{j < 4} wl_j x_{t-j},   z_t = silu(u_t),
//   y_t = z_t / sqrt(|z_t|^2 + eps) (q and k),  y_t = z_t (v).
// A chunk's rows of x and the three rows before it are staged in LDS
// (staged row r holds token start - 3 + r), so row t of the chunk reads its
// four taps from staged rows t .. t + 3.  The forward (in the prep kernel)
// and the backward (in the gradient kernel) form u with the same code, in
// the same order.
#pragma once
#include "gdn_device.h"
#include "gdn_kernels.h"

namespace gdn {

constexpr int up16(int x) { return (x + 15) / 16 * 16; }

// Element q of a 16-byte group of E, as float: for bf16 the dword's low or
// high half moved to the top (no 16-bit extraction), for fp32 the dword.
template <class E> __device__ inline float elem_f(const uint4& r, int q);
template <> __device__ inline float elem_f<bf16>(const uint4& r, int q) {
  const unsigned d = q < 2 ? r.x : q < 4 ? r.y : q < 6 ? r.z : r.w;
  return __uint_as_float((q & 1) ? (d & 0xffff0000u) : (d << 16));
}
template <> __device__ inline float elem_f<float>(const uint4& r, int q) {
  return __uint_as_float(q == 0 ? r.x : q == 1 ? r.y : q == 2 ? r.z : r.w);
}

// A wave-uniform float in a scalar register (the bits, moved as an int: the
// builtin converts a float argument to int).
__device__ inline float uniform_f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, x)));
}
// A wave-uniform float4 (weights by lag of one channel) in scalar registers:
// read from LDS by every lane at the same address, then kept once per wave.
// (As vector registers, the weights of all of a lane's channels spill; read
// through the scalar cache, their waits serialise with the LDS reads.)
__device__ inline float4 uniform_weights(const float4 v) {
  return make_float4(uniform_f(v.x), uniform_f(v.y), uniform_f(v.z), uniform_f(v.w));
}

// Staging of NCOL columns of the chunk's rows of x (and the three before).
template <class E, int NCOL, int NTH>
struct ProStage {
  static constexpr int EPV = 16 / sizeof(E);      // elements per 16 bytes
  static constexpr int XR = CH + 3;               // staged rows
  static constexpr int LD = NCOL + EPV;           // row stride in elements
  static constexpr int VPR = NCOL / EPV;          // 16-byte pieces per row
  static constexpr int PIECES = XR * VPR;
  static constexpr int PPT = (PIECES + NTH - 1) / NTH;  // pieces per thread
  static constexpr int BYTES = XR * LD * (int)sizeof(E);
  static_assert(NCOL % EPV == 0, "whole 16-byte pieces");

  uint4 nxt[PPT];  // this thread's pieces, loaded ahead of the store to LDS

  // Columns col0 .. col0 + NCOL of rows start - 3 .. start + 63 of x
  // [token][H][D]; zero past the chunk's len rows and before the sequence
  // (nprev of the three earlier rows belong to it).
  __device__ void fetch(const E* X, int D, int H, int h, int start, int len, int nprev, int col0,
                        int tid) {
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
      const int idx = tid + NTH * k, r = idx / VPR, cv = idx - r * VPR;
      const int tr = r - 3;  // row within the chunk
      const bool ok = idx < PIECES && (tr >= 0 ? tr < len : -tr <= nprev);
      nxt[k] = ok ? *reinterpret_cast<const uint4*>(X + ((size_t)(start + tr) * H + h) * D +
                                                    col0 + cv * EPV)
                  : uint4{0u, 0u, 0u, 0u};
    }
  }
  __device__ void store(E* s, int tid) const {
#pragma unroll
    for (int k = 0; k < PPT; ++k) {
      const int idx = tid + NTH * k, r = idx / VPR, cv = idx - r * VPR;
      if (idx < PIECES) *reinterpret_cast<uint4*>(s + r * LD + cv * EPV) = nxt[k];
    }
  }
  // u of row t for the EPV channels at staged column cg, with the weights
  // by lag of those channels at wl[0 .. EPV) (LDS); cg and wl are the same
  // for every lane of the wave
  __device__ static void u_of(const E* s, const float4* wl, int t, int cg, float (&u)[EPV]) {
    uint4 tap[4];  // x_{t-j}: staged row t + 3 - j
#pragma unroll
    for (int j = 0; j < 4; ++j) tap[j] = *reinterpret_cast<const uint4*>(s + (t + 3 - j) * LD + cg);
#pragma unroll
    for (int q = 0; q < EPV; ++q) {
      const float4 w = uniform_weights(wl[q]);
      u[q] = w.x * elem_f<E>(tap[0], q) + w.y * elem_f<E>(tap[1], q) +
             w.z * elem_f<E>(tap[2], q) + w.w * elem_f<E>(tap[3], q);
    }
  }
};

// Weights by lag of n channels (the first n rows of w [*, width]) into
// dst[0 .. n), lag j in component j, zero past the width.
__device__ inline void pro_weights(float4* dst, const float* w, int width, int n, int tid,
                                   int nth) {
  for (int i = tid; i < n; i += nth) {
    const float* row = w + (size_t)i * width;
    float wl[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) wl[j] = j < width ? row[width - 1 - j] : 0.f;
    dst[i] = make_float4(wl[0], wl[1], wl[2], wl[3]);
  }
}

// L2 warm-up of the rows a chunk's prologue stages: one dword of every
// 128-byte line of rows start - nprev .. start + len - 1 of x (the D channels
// of head h), loaded straight into LDS (`sink`: 256 bytes that nothing reads),
// so that the slice fetches that follow find their lines in L2 instead of
// waiting on HBM one slice at a time.  As with the state passes' warm-up, the
// statement sets m0 (which the compiler never uses in these kernels: checked on
// the built code object), the compiler does not count these loads (its own
// vmcnt waits only get stricter), and the caller waits vmcnt(0) before the
// workgroup ends.  Every address lies in the sequence's rows of x.
template <class E>
__device__ inline void pro_warm(const E* X, int D, int H, int h, int start, int len, int nprev,
                                float* sink, int tid, int nth) {
  const int lpr = D * (int)sizeof(E) / 128;  // 128-byte lines per row
  const int n = (nprev + len) * lpr;
  const unsigned char* base =
      reinterpret_cast<const unsigned char*>(X + ((size_t)(start - nprev) * H + h) * D);
  const unsigned lds = (unsigned)(uintptr_t)sink;
  const unsigned rowb = (unsigned)H * (unsigned)D * (unsigned)sizeof(E);
  for (int i = tid; i < n; i += nth) {
    const int r = i / lpr;
    const unsigned off = (unsigned)r * rowb + (unsigned)(i - r * lpr) * 128u;
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2" ::"s"(lds), "v"(off),
                 "s"(base)
                 : "memory");
  }
}

// First token of the sequence of chunk table entry ci.
__device__ inline int pro_seq_start(const Args& a, int4 ci) {
  return a.cu ? a.cu[ci.x] : ci.x * a.T;
}
// One past the last token of that sequence.
__device__ inline int pro_seq_end(const Args& a, int4 ci) {
  return a.cu ? a.cu[ci.x + 1] : (ci.x + 1) * a.T;
}

}  // namespace gdn

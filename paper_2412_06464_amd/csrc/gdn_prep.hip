// Parallel per-chunk preparation (gfx950) of the chunkwise gated delta rule.
// Chunk algebra (Sec. 3.3 of the paper; state stored dk x dv, the transpose
// of the paper's dv x dk state), for one chunk of n <= 64 tokens with beta b
// and cumulative log gate g (restarted at every chunk, Sec. 2.1 footnote):
//   Gamma_ri = exp(g_r - g_i) for i <= r          (decay-aware causal mask)
//   A  = strictLower(diag(b) (Gamma * K K^T)),   T = (I + A)^-1
//   W~ = T diag(b e^g) K,   U~ = T diag(b) V       (gated UT transform)
//   P  = Gamma * Q K^T   (lower, with the diagonal)
// With these, for entry state S:  V' = U~ - W~ S,
//   O = diag(e^g) Q S + P V',   S_next = e^{g_n} S + Kbar^T V'
//   (Kbar = diag(e^{g_n - g}) K).
// W~ is the paper's decayed W (decay on the left of the ungated UT
// transform) rewritten with the gated inverse: diag(e^g) (I + A_u)^-1 =
// (I + A_g)^-1 diag(e^g) when A_g = diag(e^g) A_u diag(e^-g).  The output
// mask is Gamma; the plain causal mask printed in the gated output equation
// does not reproduce the recurrence.
//
//   k_chunk_table  chunk -> (sequence, first row, length)
//   k_prep         one workgroup per (chunk, head): the chunk's q, k, v rows
//                  loaded once into registers, g, Gram matrices, T in LDS,
//                  then the operands of the sequential passes, staged through
//                  LDS in 64-wide slices of dk and dv.  Forward: W~, Kbar^T, U~,
//                  P, diag(e^g) Q.  Backward (recompute): W~, Kbar^T, U~, and
//                  for the reverse pass K, P^T, T^T, -W~^T, (e^g Q)^T, plus
//                  strictLower(Gamma K K^T)^T for the gradient kernel.
//                  Forward with save: both sets.
#include "gdn_device.h"
#include "gdn_kernels.h"
#include "gdn_prologue.h"

namespace gdn {

// One workgroup of 256 threads.  Sequences are taken 256 at a time: thread
// i reads the bounds of sequence base + i, an exclusive scan of the chunk
// counts in LDS (plus the running total of the earlier groups) gives its
// first chunk, and the thread writes that sequence's chunk entries.
__global__ void k_chunk_table(const int32_t* cu, int N, int T, int4* info, int* seq_chunk0) {
  __shared__ int scan[2][256];
  const int tid = threadIdx.x;
  int carry = 0;  // chunks of the sequences before this group
  for (int base = 0; base < N; base += 256) {
    const int n = base + tid;
    const int s = n < N ? (cu ? cu[n] : n * T) : 0;
    const int L = n < N ? (cu ? cu[n + 1] - s : T) : 0;
    const int c = (L + CH - 1) / CH;
    // inclusive Hillis-Steele scan of c over the 256 threads
    int p = 0;
    scan[p][tid] = c;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {
      scan[p ^ 1][tid] = scan[p][tid] + (tid >= d ? scan[p][tid - d] : 0);
      p ^= 1;
      __syncthreads();
    }
    const int c0 = carry + scan[p][tid] - c;
    if (n < N) {
      seq_chunk0[n] = c0;
      for (int j = 0; j < c; ++j) info[c0 + j] = make_int4(n, s + j * CH, min(CH, L - j * CH), 0);
    }
    carry += scan[p][255];
    __syncthreads();  // the scan buffers are reused by the next group
  }
  if (tid == 0) seq_chunk0[N] = carry;
}

// ------------------------------------------------------------------ prep

// A buffers (permuted order) of a 64 x 64 LDS matrix src[r * ld + k]: the raw
// values into dst_raw (skipped when null) and the values times scale[k] into
// dst_scaled, from one LDS read per element.
template <class E, int NTH>
__device__ inline void export_afrag_perm_pair(E* dst_raw, E* dst_scaled, const E* src, int ld,
                                              const float* scale) {
  using M = Mfma<E>;
  constexpr int NKT = CH / M::K, UNITS = CH * CH / M::KPL;
  for (int u = threadIdx.x; u < UNITS; u += NTH) {
    const int tile = u >> 6, l = u & 63;
    const int mt = tile / NKT, kt = tile - mt * NKT;
    const int r = mt * 16 + (l & 15), g = l >> 4;
    union {
      typename M::frag f;
      E e[M::KPL];
    } xr, xs;
#pragma unroll
    for (int j = 0; j < M::KPL; ++j) {
      const int k = kperm<E>(kt, g, j);
      const E x = src[r * ld + k];
      xr.e[j] = x;
      xs.e[j] = to_e<E>(to_f(x) * scale[k]);
    }
    if (dst_raw) store_stream_small(dst_raw + (size_t)u * M::KPL, xr.f);
    store_stream_small(dst_scaled + (size_t)u * M::KPL, xs.f);
  }
}
// Grid (NC, H), 256 threads (4 waves).  LDS stays below 80 KB for bf16 so
// that two workgroups share a CU: one streams while the other solves.

// BLK: the block prologue (Sec. 3.4: short causal convolution, SiLU, and L2
// normalisation of q and k) runs in place of the row loads: the rule's q, k
// and v are formed in registers from the projections a.xq, a.xk, a.xv (and
// written to a.yq, a.yk, a.yv where those are set).
template <class E, int DK, int DV, int MODE, bool BLK = false>
__global__ __launch_bounds__(256, 2) void k_prep(Args a) {
  using M = Mfma<E>;
  // operands of the forward pass (diag(e^g) Q, P), of the reverse pass and
  // gradient kernel (K, P^T, T^T, -W~^T, (e^g Q)^T, Ak^T), or both
  constexpr bool FOUT = MODE != PREP_BWD, BOUT = MODE != PREP_FWD;
  constexpr int PADE = 16 / sizeof(E);
  constexpr int LD = CH + PADE;  // rows of 64 elements
  constexpr int LDA = CH + 1;
  constexpr int NKC = CH / M::K;
  __shared__ __align__(16) E sX[CH * LD];  // K slice (Gram), then K_s^T or (b V_s)^T
  __shared__ __align__(16) E sY[CH * LD];  // Q slice (Gram), then Q_s^T (backward)
  __shared__ __align__(16) E sT[CH * LD];  // T, row-major
  __shared__ __align__(16) E sP[CH * LD];  // P, row-major
  __shared__ float sA[CH * LDA];           // diag(b) A
  __shared__ float sTf[CH * LDA];          // T in fp32
  __shared__ float sYb[32 * 33];         // products of the block recursion
  __shared__ float sg[CH], sb[CH], seg[CH], sdec[CH], sbeg[CH];

  const int c = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(wave_id());
  const int H = a.H;
  const int4 ci = chunk_info(a, c);
  const int start = ci.y, len = ci.z;
  const size_t ch = (size_t)c * H + h;
  const size_t row0 = (size_t)start * H + h;
  const E* K = (const E*)a.k + row0 * DK;
  const E* Q = (const E*)a.q + row0 * DK;
  const E* V = (const E*)a.v + row0 * DV;

  // The chunk's raw k, q and v rows, loaded once at the start and kept in
  // registers for both the row-major and the transposed staging: lane = row
  // t, 16-byte vectors cv = w + 4 i of each 64-wide column slice.
  constexpr int EPV = 16 / sizeof(E), NI = 64 / EPV / 4;
  constexpr int KS = DK / 64, VS = DV / 64;
  uint4 rk[KS][NI], rq[KS][NI], rv[VS][NI];
  if constexpr (!BLK) {
    const int t = lane_id();
    const bool tv = t < len;
    const size_t ko = (size_t)(tv ? t : 0) * H * DK, vo = (size_t)(tv ? t : 0) * H * DV;
#pragma unroll
    for (int sl = 0; sl < KS; ++sl)
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int c = 64 * sl + (w + 4 * i) * EPV;
        rk[sl][i] = tv ? *reinterpret_cast<const uint4*>(K + ko + c) : uint4{0u, 0u, 0u, 0u};
        rq[sl][i] = tv ? *reinterpret_cast<const uint4*>(Q + ko + c) : uint4{0u, 0u, 0u, 0u};
      }
#pragma unroll
    for (int sl = 0; sl < VS; ++sl)
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int c = 64 * sl + (w + 4 * i) * EPV;
        rv[sl][i] = tv ? *reinterpret_cast<const uint4*>(V + vo + c) : uint4{0u, 0u, 0u, 0u};
      }
  }
  if constexpr (BLK) {
    // ---- block prologue, instead of the row loads: each 64-wide slice of
    // x (the chunk's rows and the three before them) is staged in LDS; lane
    // t forms row t from its four taps there and keeps the fp32 z of the
    // tensor in progress until its row norm is known, then packs y into the
    // registers the prep works on (rq, rk, rv)
    using S = ProStage<E, 64, 256>;
    static_assert(sizeof(E) == 2, "the fused block prologue is built for bf16");
    static_assert((S::BYTES + 15) / 16 * 16 + 4 * CH * sizeof(float) <= CH * LDA * sizeof(float),
                  "staging and row sums must fit in A");
    E* sXs = reinterpret_cast<E*>(sA);                    // staged slice (A is not formed yet)
    float* sNrm = sA + (S::BYTES + 15) / 16 * 4;          // [4 waves][CH] row sums
    // weights by lag of the q | k | v channels, in the fp32 T buffer, which
    // the inverse does not use yet
    float4* sWl = reinterpret_cast<float4*>(sTf);
    static_assert((2 * DK + DV) * sizeof(float4) <= CH * LDA * sizeof(float),
                  "weights must fit in T");
    pro_weights(sWl, a.cwq + (size_t)h * DK * a.cw, a.cw, DK, tid, 256);
    pro_weights(sWl + DK, a.cwk + (size_t)h * DK * a.cw, a.cw, DK, tid, 256);
    pro_weights(sWl + 2 * DK, a.cwv + (size_t)h * DV * a.cw, a.cw, DV, tid, 256);
    const int nprev = start > pro_seq_start(a, ci) ? 3 : 0;  // chunks start 64-aligned in a sequence
    // the chunk's rows of all three projections into L2 first, where the
    // workgroups an XCD runs at once (two per CU, 32 CUs) keep theirs within
    // its 4 MB L2: 64 x 67 rows x (2 dk + dv) x 2 bytes is 3.3 MB at 128/128
    // (prep 1.29 -> 1.20 ms at 65,536 tokens x 16 heads) but 8.8 MB at
    // 256/512, where the warmed lines are gone before they are read (0.54 ->
    // 0.57 ms).  Their offsets from the first staged row fit 32 bits.
    __shared__ float sWarm[64];
    constexpr bool WARM = 64 * (CH + 3) * (2 * DK + DV) * (int)sizeof(E) <= (4 << 20);
    if (WARM && (size_t)(CH + 3) * H * DV * sizeof(E) < (1u << 31)) {
      pro_warm((const E*)a.xq, DK, H, h, start, len, nprev, sWarm, tid, 256);
      pro_warm((const E*)a.xk, DK, H, h, start, len, nprev, sWarm, tid, 256);
      pro_warm((const E*)a.xv, DV, H, h, start, len, nprev, sWarm, tid, 256);
    }
    const int t = lane_id();
    S st;
    auto pack = [&](const float (&y)[EPV]) {
      union {
        uint4 u;
        E e[EPV];
      } x;
#pragma unroll
      for (int q = 0; q < EPV; ++q) x.e[q] = to_e<E>(t < len ? y[q] : 0.f);
      return x.u;
    };
    // one slice's z for this lane's groups of channels (wt: the weights by
    // lag of the tensor's channels); the slice is staged first
    auto slice_z = [&](const E* X, int D, const float4* wt, int sl, int nsl, float (&z)[NI][EPV]) {
      lds_barrier();  // the previous slice's taps (and the row sums) are read
      st.store(sXs, tid);
      if (sl + 1 < nsl) st.fetch(X, D, H, h, start, len, nprev, 64 * (sl + 1), tid);
      lds_barrier();
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int cg = (w + 4 * i) * EPV;
        S::u_of(sXs, wt + 64 * sl + cg, t, cg, z[i]);
#pragma unroll
        for (int q = 0; q < EPV; ++q) z[i][q] *= sigmoidf(z[i][q]);
      }
    };
    // one tensor with a row norm (q or k): out[sl][i] = y
    auto prologue_l2 = [&](const E* X, const float4* wt, uint4 (&out)[KS][NI], void* yout) {
      float z[KS][NI][EPV], ss = 0.f;
      st.fetch(X, DK, H, h, start, len, nprev, 0, tid);
#pragma unroll
      for (int sl = 0; sl < KS; ++sl) {
        slice_z(X, DK, wt, sl, KS, z[sl]);
#pragma unroll
        for (int i = 0; i < NI; ++i)
#pragma unroll
          for (int q = 0; q < EPV; ++q) ss += z[sl][i][q] * z[sl][i][q];
      }
      sNrm[w * CH + t] = ss;
      lds_barrier();
      const float sc = rsqrtf(sNrm[t] + sNrm[CH + t] + sNrm[2 * CH + t] + sNrm[3 * CH + t] + a.ceps);
#pragma unroll
      for (int sl = 0; sl < KS; ++sl)
#pragma unroll
        for (int i = 0; i < NI; ++i) {
#pragma unroll
          for (int q = 0; q < EPV; ++q) z[sl][i][q] *= sc;
          out[sl][i] = pack(z[sl][i]);
          if (yout && t < len)
            *reinterpret_cast<uint4*>((E*)yout + (row0 + (size_t)t * H) * DK + 64 * sl +
                                      (w + 4 * i) * EPV) = out[sl][i];
        }
    };
    prologue_l2((const E*)a.xq, sWl, rq, a.yq);
    prologue_l2((const E*)a.xk, sWl + DK, rk, a.yk);
    {  // v: no norm
      const E* X = (const E*)a.xv;
      const float4* wt = sWl + 2 * DK;
      st.fetch(X, DV, H, h, start, len, nprev, 0, tid);
#pragma unroll
      for (int sl = 0; sl < VS; ++sl) {
        float z[NI][EPV];
        slice_z(X, DV, wt, sl, VS, z);
#pragma unroll
        for (int i = 0; i < NI; ++i) {
          rv[sl][i] = pack(z[i]);
          if (a.yv && t < len)
            *reinterpret_cast<uint4*>((E*)a.yv + (row0 + (size_t)t * H) * DV + 64 * sl +
                                      (w + 4 * i) * EPV) = rv[sl][i];
        }
      }
    }
    if constexpr (WARM) wait_vmcnt<0>();  // the warm-up's loads into sWarm have landed
    lds_barrier();    // A and T are formed below
  }

  // a slice of raw rows into LDS, row-major (dst[t][c]) or transposed
  // (dst[c][t], element scaled by scale)
  auto put_rows = [&](E* dst, const uint4 (&r)[NI]) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
      *reinterpret_cast<uint4*>(dst + lane_id() * LD + (w + 4 * i) * EPV) = r[i];
  };
  auto put_T = [&](E* dstT, const uint4 (&r)[NI], float scale) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      union {
        uint4 u;
        E e[EPV];
      } x;
      x.u = r[i];
#pragma unroll
      for (int j = 0; j < EPV; ++j)
        dstT[((w + 4 * i) * EPV + j) * LD + lane_id()] = to_e<E>(to_f(x.e[j]) * scale);
    }
  };

  const bool gated = a.gated;
  if (tid < CH) {
    const float b = tid < len ? a.beta[row0 + (size_t)tid * H] : 0.f;
    sb[tid] = b;
    if (gated) {
      const float la = tid < len ? a.log_alpha[row0 + (size_t)tid * H] : 0.f;
      const float g = wave_incl_scan(la);  // pads repeat g at the last token
      const float gn = __shfl(g, CH - 1, 64);
      sg[tid] = g;
      seg[tid] = __expf(g);
      sdec[tid] = __expf(gn - g);
      sbeg[tid] = b * __expf(g);
      a.g[ch * CH + tid] = g;
    } else {  // alpha == 1 (DeltaNet): no decay anywhere
      sg[tid] = 0.f;
      seg[tid] = 1.f;
      sdec[tid] = 1.f;
      sbeg[tid] = b;
      a.g[ch * CH + tid] = 0.f;  // read by a backward from a saved buffer
    }
  }

  // ---- Gram blocks K K^T and Q K^T over 64-wide slices of dk; wave w owns
  // rows 16w..16w+15.
  f32x4 kk[1][4], qk[1][4];
  zero_acc(kk);
  zero_acc(qk);
  static_for<0, KS>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    put_rows(sX, rk[s]);
    put_rows(sY, rq[s]);
    lds_barrier();
    wave_mma_nt<E, 1, 4, 64>(kk, sX + w * 16 * LD, LD, sX, LD);
    wave_mma_nt<E, 1, 4, 64>(qk, sY + w * 16 * LD, LD, sX, LD);
    if (FOUT) {
      // diag(e^g) Q as A operands (rows t, k = d) for the output of the forward pass
      export_afrag_perm_kslice<E, CH, DK, 64, 256>(
          (E*)a.Qf + ch * CH * DK, 64 * s, [&](int t, int d) { return seg[t] * to_f(sY[t * LD + d]); });
    }
    if (BOUT) {
      // raw K as A operands (rows t, k = d) for K dS in the reverse pass
      export_afrag_perm_kslice<E, CH, DK, 64, 256>(
          (E*)a.Kf + ch * CH * DK, 64 * s, [&](int t, int d) { return to_f(sX[t * LD + d]); });
    }
    lds_barrier();
  });
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int r = w * 16 + acc_row(e), i = j * 16 + acc_col();
      // select, never multiply by an overflowed exp above the diagonal
      const float gam = (i <= r) ? (gated ? __expf(sg[r] - sg[i]) : 1.f) : 0.f;
      const float ak = (i < r) ? gam * kk[0][j][e] : 0.f;
      const float p = (i <= r) ? gam * qk[0][j][e] : 0.f;
      sA[r * LDA + i] = sb[r] * ak;
      sP[r * LD + i] = to_e<E>(p);
      kk[0][j][e] = ak;
      qk[0][j][e] = p;
    }
  if (BOUT) {
    // strictLower(Gamma K K^T) as the A buffer of its transpose, like P^T
#pragma unroll
    for (int j = 0; j < 4; ++j) afrag_put_T<E>((E*)a.Ak + ch * CH * CH, CH, j, w, kk[0][j]);
  }
  lds_barrier();

  // ---- T = (I + A)^-1, A strictly lower, by block recursion.  The 16x16
  // diagonal blocks by forward substitution (one column per thread); then,
  // with fp32 MFMA, the off-diagonal block of each 32x32 diagonal block and
  // finally the lower-left 32x32 block, each as
  //   T_21 = -T_22 (A_21 T_11)
  // for a block lower-triangular [[T_11, 0], [T_21, T_22]].
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
    for (int i = 0; i < 16; ++i) sTf[(o + i) * LDA + o + j] = x[i];
  }
  lds_barrier();
  {
    using MF = Mfma<float>;
    const int lr = lane_id() & 15, lg = lane_id() >> 4;
    // 16 x 16 x 16 product tile: acc += X[xr.., xc..] Y[yr.., yc..] (fp32 LDS, leading dims)
    auto mm16 = [&](f32x4& acc, const float* X, int ldx, int xr, int xc, const float* Y, int ldy,
                    int yr, int yc) {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
        acc = MF::mma(X[(xr + lr) * ldx + xc + 4 * ks + lg], Y[(yr + 4 * ks + lg) * ldy + yc + lr], acc);
    };
    // 32x32 diagonal blocks (waves 0 and 1): T[o+16.., o..] = -T[o+16.., o+16..] (A[o+16.., o..] T[o.., o..])
    if (w < 2) {
      const int o = 32 * w;
      float* yb = sYb + w * 16 * 17;
      f32x4 y = {0.f, 0.f, 0.f, 0.f}, z = {0.f, 0.f, 0.f, 0.f};
      mm16(y, sA, LDA, o + 16, o, sTf, LDA, o, o);
#pragma unroll
      for (int e = 0; e < 4; ++e) yb[(4 * lg + e) * 17 + lr] = y[e];  // read back by this wave only
      mm16(z, sTf, LDA, o + 16, o + 16, yb, 17, 0, 0);
#pragma unroll
      for (int e = 0; e < 4; ++e) sTf[(o + 16 + 4 * lg + e) * LDA + o + lr] = -z[e];
    }
    lds_barrier();
    // lower-left 32x32 block, one 16x16 tile (I, J) per wave:
    //   Y = A[32.., 0..32] T[0..32, 0..32]  (T lower: k-blocks K >= J)
    //   T[32 + 16 I.., 16 J..] = -sum_{K <= I} T[32 + 16 I.., 32 + 16 K..] Y[16 K.., 16 J..]
    const int I = w >> 1, J = w & 1;
    f32x4 y = {0.f, 0.f, 0.f, 0.f}, z = {0.f, 0.f, 0.f, 0.f};
    for (int K = J; K < 2; ++K) mm16(y, sA, LDA, 32 + 16 * I, 16 * K, sTf, LDA, 16 * K, 16 * J);
#pragma unroll
    for (int e = 0; e < 4; ++e) sYb[(16 * I + 4 * lg + e) * 33 + 16 * J + lr] = y[e];
    lds_barrier();
    for (int K = 0; K <= I; ++K) mm16(z, sTf, LDA, 32 + 16 * I, 32 + 16 * K, sYb, 33, 16 * K, 16 * J);
#pragma unroll
    for (int e = 0; e < 4; ++e) sTf[(32 + 16 * I + 4 * lg + e) * LDA + 16 * J + lr] = -z[e];
  }
  lds_barrier();
  for (int idx = tid; idx < CH * CH; idx += 256) {
    const int r = idx >> 6, i = idx & 63;
    sT[r * LD + i] = to_e<E>(((i >> 4) > (r >> 4)) ? 0.f : sTf[r * LDA + i]);
  }
  lds_barrier();

  // ---- 64 x 64 operands
  if (FOUT) {
    export_afrag_perm<E, CH, CH, 256>((E*)a.Pf + ch * CH * CH,
                                      [&](int t, int i) { return to_f(sP[t * LD + i]); });
  }
  if (BOUT) {
    export_afrag_perm<E, CH, CH, 256>((E*)a.PTf + ch * CH * CH,
                                      [&](int i, int t) { return to_f(sP[t * LD + i]); });
    export_afrag_perm<E, CH, CH, 256>((E*)a.TTf + ch * CH * CH,
                                      [&](int i, int t) { return to_f(sT[t * LD + i]); });
  }

  // ---- dk slices: W~ (and -W~^T), Kbar^T, (e^g Q)^T
  static_for<0, KS>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    put_T(sX, rk[s], 1.f);  // sX[d][t]
    if (BOUT) put_T(sY, rq[s], 1.f);
    lds_barrier();
    // W~^T (rows d of this wave, columns t'):  sum_t (b e^g K)^T[d][t] T[t'][t]
    f32x4 Wt[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) Wt[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    const E* xrow = sX + (w * 16 + (lane_id() & 15)) * LD;
#pragma unroll
    for (int kt = 0; kt < NKC; ++kt) {
      const typename M::frag af = load_frag_scaled<E>(xrow, kt, sbeg);
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        const typename M::frag bf =
            M::load(sT + (n * 16 + (lane_id() & 15)) * LD + kt * M::K + (lane_id() >> 4) * M::KPL);
        Wt[n] = M::mma(af, bf, Wt[n]);
      }
    }
    // W~ as A operands (rows t', k = d) for the state passes
#pragma unroll
    for (int n = 0; n < 4; ++n) afrag_put_T<E>((E*)a.Wf + ch * CH * DK, DK, n, 4 * s + w, Wt[n]);
    // Kbar^T as A operands (rows d, k = t)
    export_afrag_perm_pair<E, 256>(nullptr, (E*)a.KbT + ch * DK * CH + (size_t)64 * s * CH, sX, LD,
                                   sdec);
    if (BOUT) {
      // W~ (rows t' of this wave, columns d):  sum_t T[t'][t] (b e^g K)[t][d]
      f32x4 W[4];
#pragma unroll
      for (int n = 0; n < 4; ++n) W[n] = f32x4{0.f, 0.f, 0.f, 0.f};
      const E* trow = sT + (w * 16 + (lane_id() & 15)) * LD;
#pragma unroll
      for (int kt = 0; kt < NKC; ++kt) {
        const typename M::frag af =
            M::load(trow + kt * M::K + (lane_id() >> 4) * M::KPL);
#pragma unroll
        for (int n = 0; n < 4; ++n) {
          const typename M::frag bf =
              load_frag_scaled<E>(sX + (n * 16 + (lane_id() & 15)) * LD, kt, sbeg);
          W[n] = M::mma(af, bf, W[n]);
        }
      }
      // -W~^T as A operands (rows d, k = t')
#pragma unroll
      for (int n = 0; n < 4; ++n) afrag_put_T<E>((E*)a.nWT + ch * DK * CH, CH, 4 * s + n, w, -W[n]);
      // (e^g Q)^T as A operands (rows d, k = t)
      export_afrag_perm_pair<E, 256>(nullptr, (E*)a.QgT + ch * DK * CH + (size_t)64 * s * CH, sY,
                                     LD, seg);
    }
    lds_barrier();
  });

  // ---- dv slices: U~ = T (b V), accumulator layout
  const float bt = sb[lane_id()];
  static_for<0, VS>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    put_T(sX, rv[s], bt);  // sX[v][t] = b_t V
    lds_barrier();
    f32x4 U[1][4];
    zero_acc(U);
    wave_mma_nt<E, 1, 4, CH>(U, sT + w * 16 * LD, LD, sX, LD);
    E* gU = (E*)a.Uc + ch * CH * DV;
#pragma unroll
    for (int n = 0; n < 4; ++n) store4<E>(gU + cfrag_index(w, 4 * s + n, DV), U[0][n]);
    lds_barrier();
  });
}

// ------------------------------------------------------------------ launchers

hipError_t launch_chunk_table(const Args& a, hipStream_t s) {
  hipLaunchKernelGGL(k_chunk_table, dim3(1), dim3(256), 0, s, a.cu, a.N, a.T, a.info,
                     a.seq_chunk0);
  return hipGetLastError();
}

hipError_t launch_prep(Dt dt, int dk, int dv, int mode, const Args& a, hipStream_t s,
                       bool block) {
  if (block && (!a.xq || !a.xk || !a.xv || !a.cwq || !a.cwk || !a.cwv || a.cw < 1 || a.cw > 4))
    return hipErrorInvalidValue;
  if (block && mode == PREP_SAVE && (!a.yq || !a.yk || !a.yv))
    return hipErrorInvalidValue;  // the backward reads the rule's q, k, v
  auto f = [&]<class E, int DK, int DV>() {
    if (block) {  // fused block prologue (bf16): forward and saving forward only
      if constexpr (sizeof(E) != 2) return hipErrorInvalidValue;
      else if (mode == PREP_SAVE)
        hipLaunchKernelGGL((k_prep<E, DK, DV, PREP_SAVE, true>), dim3(a.NC, a.H), dim3(256), 0, s,
                           a);
      else if (mode == PREP_FWD)
        hipLaunchKernelGGL((k_prep<E, DK, DV, PREP_FWD, true>), dim3(a.NC, a.H), dim3(256), 0, s,
                           a);
      else
        return hipErrorInvalidValue;
      return hipGetLastError();
    }
    if (mode == PREP_BWD)
      hipLaunchKernelGGL((k_prep<E, DK, DV, PREP_BWD>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    else if (mode == PREP_SAVE)
      hipLaunchKernelGGL((k_prep<E, DK, DV, PREP_SAVE>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL((k_prep<E, DK, DV, PREP_FWD>), dim3(a.NC, a.H), dim3(256), 0, s, a);
    return hipGetLastError();
  };
  GDN_DISPATCH(dt, dk, dv, f);
}

}  // namespace gdn

// Device helpers for the gfx950 gated-delta-rule kernels: MFMA fragments,
// wave-level tile products from LDS, tile staging between HBM and LDS.
//
// MFMA conventions (16x16 output tiles, wave64):
//   A operand   : lane l holds row (l & 15), KPL consecutive k starting at
//                 (l >> 4) * KPL of the current k-step;
//   B operand   : lane l holds column (l & 15), the same k range; we always
//                 keep B transposed in memory ("Bt[n][k]"), so both operands
//                 are read with the contraction index contiguous;
//   accumulator : lane l holds rows 4*(l >> 4) + {0,1,2,3}, column (l & 15).
// bf16 uses v_mfma_f32_16x16x32_bf16 (K = 32, 8 k per lane, fp32 accumulate);
// fp32 uses v_mfma_f32_16x16x4_f32 (K = 4, 1 k per lane, full fp32).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

namespace gdn {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int CH = 64;  // chunk length in tokens

// Chunk c's {sequence, first token row, length}, and the first chunk of
// sequence n.  Dense input (no cu_seqlens): B sequences of T tokens, each cut
// into ceil(T / CH) consecutive chunks, so both are arithmetic; packed input
// reads the chunk table.  (A is the kernels' argument struct.)
template <class A>
__device__ inline int4 chunk_info(const A& a, int c) {
  if (a.cu) return a.info[c];
  const int nch = (a.T + CH - 1) / CH, n = c / nch, j = c - n * nch;
  return make_int4(n, n * a.T + j * CH, min(CH, a.T - j * CH), 0);
}
template <class A>
__device__ inline int seq_first_chunk(const A& a, int n) {
  return a.cu ? a.seq_chunk0[n] : n * ((a.T + CH - 1) / CH);
}

template <class E> struct Mfma;

template <> struct Mfma<bf16> {
  static constexpr int K = 32;
  static constexpr int KPL = 8;
  using frag = bf16x8;
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const bf16* p) {
    return *reinterpret_cast<const frag*>(p);
  }
};

template <> struct Mfma<float> {
  static constexpr int K = 4;
  static constexpr int KPL = 1;
  using frag = float;
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const float* p) { return *p; }
};

// Four raw elements of an accumulator-layout tile (converted at use).
template <class E> struct Raw4;
template <> struct Raw4<bf16> {
  typedef bf16 type __attribute__((ext_vector_type(4)));
};
template <> struct Raw4<float> {
  typedef f32x4 type;
};

template <class E> __device__ inline E to_e(float x);
template <> __device__ inline float to_e<float>(float x) { return x; }
template <> __device__ inline bf16 to_e<bf16>(float x) { return (bf16)x; }  // RNE

__device__ inline float to_f(float x) { return x; }
__device__ inline float to_f(bf16 x) { return (float)x; }

// Workgroup barrier that orders LDS traffic only: each wave waits for its
// own outstanding LDS operations and then meets the others.  Unlike
// __syncthreads(), whose workgroup-scope fence also waits for every
// outstanding global load, this leaves prefetched global loads in flight
// across the barrier.  It must not be used to publish global-memory writes
// to other threads of the workgroup.
__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ inline int lane_id() { return threadIdx.x & 63; }
__device__ inline int wave_id() { return threadIdx.x >> 6; }

template <int MT, int NT>
__device__ inline void zero_acc(f32x4 (&acc)[MT][NT]) {
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// acc[i][j] (+)= sum_k A[i*16 + m][k] * Bt[j*16 + n][k], k in [0, KDIM).
// A and Bt point at the wave's first row; lda/ldb in elements.
template <class E, int MT, int NT, int KDIM>
__device__ inline void wave_mma_nt(f32x4 (&acc)[MT][NT], const E* A, int lda,
                                   const E* Bt, int ldb) {
  using M = Mfma<E>;
  const int l = lane_id();
  const int r = l & 15, kq = (l >> 4) * M::KPL;
#pragma unroll
  for (int k0 = 0; k0 < KDIM; k0 += M::K) {
    typename M::frag a[MT], b[NT];
#pragma unroll
    for (int i = 0; i < MT; ++i) a[i] = M::load(A + (i * 16 + r) * lda + k0 + kq);
#pragma unroll
    for (int j = 0; j < NT; ++j) b[j] = M::load(Bt + (j * 16 + r) * ldb + k0 + kq);
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) acc[i][j] = M::mma(a[i], b[j], acc[i][j]);
  }
}

// Row (within a 16x16 tile) of accumulator element e for this lane.
__device__ inline int acc_row(int e) { return ((lane_id() >> 4) << 2) + e; }
__device__ inline int acc_col() { return lane_id() & 15; }

// ---- operand layouts in HBM
// A-fragment layout of an R x KD matrix M (logical row-major): the MFMA A
// tile (mt, kt) covers rows 16mt.. and k = K*kt..; lane l's KPL elements
// M[16mt + (l & 15)][K*kt + KPL*(l >> 4) + j] are stored contiguously at
// ((mt * (KD / K) + kt) * 64 + l) * KPL, so a wave reads one tile with one
// fully coalesced load (1 KiB for bf16).

// C-fragment (accumulator) layout of an R x N matrix: tile (mt, nt), lane l
// holds rows 16mt + 4(l >> 4) + e, column 16nt + (l & 15), stored at
// ((mt * (N / 16) + nt) * 64 + l) * 4 + e.
__device__ inline size_t cfrag_index(int mt, int nt, int N) {
  return ((size_t)(mt * (N / 16) + nt) * 64 + lane_id()) * 4;
}

template <class E>
__device__ inline f32x4 load4(const E* p);
template <>
__device__ inline f32x4 load4<float>(const float* p) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  return f32x4{x.x, x.y, x.z, x.w};
}
template <>
__device__ inline f32x4 load4<bf16>(const bf16* p) {
  typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 x = *reinterpret_cast<const bf16x4*>(p);
  return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
}
template <class E>
__device__ inline void store4(E* p, f32x4 v) {
  p[0] = to_e<E>(v[0]);
  p[1] = to_e<E>(v[1]);
  p[2] = to_e<E>(v[2]);
  p[3] = to_e<E>(v[3]);
}

// 16-byte store of data that this kernel does not read back (a streamed
// output or an intermediate for a later kernel): non-temporal, so it does
// not displace operands that other workgroups are about to read.
__device__ inline void store_stream(void* p, const uint4& v) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(&v), reinterpret_cast<u32x4*>(p));
}
// The same for one MFMA fragment (16 bytes for bf16, 4 for fp32) or 8 bytes.
template <class T>
__device__ inline void store_stream_small(void* p, const T& v) {
  static_assert(sizeof(T) == 16 || sizeof(T) == 8 || sizeof(T) == 4, "unsupported size");
  if constexpr (sizeof(T) == 16) {
    store_stream(p, *reinterpret_cast<const uint4*>(&v));
  } else if constexpr (sizeof(T) == 8) {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    __builtin_nontemporal_store(*reinterpret_cast<const u32x2*>(&v), reinterpret_cast<u32x2*>(p));
  } else {
    __builtin_nontemporal_store(*reinterpret_cast<const unsigned*>(&v), reinterpret_cast<unsigned*>(p));
  }
}


// ---- permuted contraction order
// An MFMA sums over its K index in any order, provided both operands agree.
// The kernels use an order in which the accumulator tiles of a matrix are
// directly the B operand of a product that contracts over that matrix's
// rows (and the A operand of one that contracts over the rows of its
// transpose):
//   bf16, k-step kt covers k in [32 kt, 32 kt + 32); lane group g = l >> 4,
//         slot j holds k = 32 kt + 4 g + j (j < 4) or 32 kt + 12 + 4 g + j
//         (j >= 4), i.e. rows 4g..4g+3 of the two 16-row accumulator tiles
//         2 kt and 2 kt + 1;
//   fp32, k-step kt holds k = 16 (kt >> 2) + 4 g + (kt & 3), i.e. element
//         (kt & 3) of accumulator tile kt >> 2.
// Every operand that meets such an accumulator-derived operand in a product
// is stored (or loaded) in the same order.
template <class E> __device__ inline int kperm(int kt, int g, int j);
template <> __device__ inline int kperm<bf16>(int kt, int g, int j) {
  return 32 * kt + (j < 4 ? 4 * g + j : 12 + 4 * g + j);
}
template <> __device__ inline int kperm<float>(int kt, int g, int) {
  return 16 * (kt >> 2) + 4 * g + (kt & 3);
}

// Element position, in a 64-column A buffer (permuted order), of element
// (r, k) of the matrix: fragment (r / 16, kt), lane r % 16 + 16 g, slot j,
// where kperm(kt, g, j) = k.
template <class E> __device__ inline int afrag_pos64(int r, int k);
template <> __device__ inline int afrag_pos64<bf16>(int r, int k) {
  const int kk = k & 31;
  return ((((r >> 4) << 1) + (k >> 5)) * 64 + (r & 15) + 16 * ((kk & 15) >> 2)) * 8 +
         4 * (kk >> 4) + (kk & 3);
}
template <> __device__ inline int afrag_pos64<float>(int r, int k) {
  return ((r >> 4) * 16 + 4 * (k >> 4) + (k & 3)) * 64 + (r & 15) + 16 * ((k & 15) >> 2);
}

// Fragment buffers.  A "B buffer" holds the B operands of a K x N matrix
// (N = 16 NT): fragment (kt, nt) of lane l at ((kt NT + nt) 64 + l) KPL.
// An "A buffer" holds the A operands of an R x KD matrix: fragment (mt, kt)
// of lane l at ((mt (KD / K) + kt) 64 + l) KPL.  Both are written from an
// accumulator tile whose rows run along K (for an A buffer: the tile of the
// transposed matrix), one 8-byte (bf16) or four 4-byte (fp32) stores per
// lane, each wave store fully coalesced.
__device__ inline size_t frag_slot_bf16(size_t frag, int i16) {
  return (frag * 64 + lane_id()) * 8 + (i16 & 1) * 4;
}
template <class E> __device__ inline void bfrag_put(E* buf, int NT, int i16, int n, f32x4 v);
template <> __device__ inline void bfrag_put<bf16>(bf16* buf, int NT, int i16, int n, f32x4 v) {
  typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 x = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
  *reinterpret_cast<bf16x4*>(buf + frag_slot_bf16((size_t)(i16 >> 1) * NT + n, i16)) = x;
}
template <> __device__ inline void bfrag_put<float>(float* buf, int NT, int i16, int n, f32x4 v) {
#pragma unroll
  for (int e = 0; e < 4; ++e) buf[((size_t)(4 * i16 + e) * NT + n) * 64 + lane_id()] = v[e];
}
template <class E>
__device__ inline typename Mfma<E>::frag bfrag_get(const E* buf, int NT, int kt, int n) {
  return Mfma<E>::load(buf + ((size_t)(kt * NT + n) * 64 + lane_id()) * Mfma<E>::KPL);
}
// A buffer of an R x KD matrix M from the accumulator tile of M^T that
// covers k rows 16 i16.. and M rows 16 mt..
template <class E> __device__ inline void afrag_put_T(E* dst, int KD, int mt, int i16, f32x4 v);
template <> __device__ inline void afrag_put_T<bf16>(bf16* dst, int KD, int mt, int i16, f32x4 v) {
  typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 x = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
  store_stream_small(dst + frag_slot_bf16((size_t)mt * (KD / 32) + (i16 >> 1), i16), x);
}
template <> __device__ inline void afrag_put_T<float>(float* dst, int KD, int mt, int i16, f32x4 v) {
#pragma unroll
  for (int e = 0; e < 4; ++e) dst[((size_t)mt * (KD / 4) + 4 * i16 + e) * 64 + lane_id()] = v[e];
}

// The inverse read: the accumulator tile (rows 16 i16 + 4 g + e, column
// 16 mt + l % 16, as f32) of a 64 x 64 matrix M^T held as the A buffer of M,
// one 8-byte load per lane for bf16.
template <class E> __device__ inline f32x4 afrag_get_T(const E* src, int mt, int i16);
template <> __device__ inline f32x4 afrag_get_T<bf16>(const bf16* src, int mt, int i16) {
  typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 x = *reinterpret_cast<const bf16x4*>(src + frag_slot_bf16((size_t)mt * 2 + (i16 >> 1), i16));
  return f32x4{(float)x[0], (float)x[1], (float)x[2], (float)x[3]};
}
template <> __device__ inline f32x4 afrag_get_T<float>(const float* src, int mt, int i16) {
  f32x4 v;
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = src[((size_t)mt * 16 + 4 * i16 + e) * 64 + lane_id()];
  return v;
}

// Write the A buffer (permuted order) of an R x KD matrix whose elements are
// val(r, k).
template <class E, int R, int KD, int NTH, class F>
__device__ inline void export_afrag_perm(E* dst, F&& val) {
  using M = Mfma<E>;
  constexpr int UNITS = R * KD / M::KPL;
  for (int u = threadIdx.x; u < UNITS; u += NTH) {
    const int tile = u >> 6, l = u & 63;
    const int mt = tile / (KD / M::K), kt = tile - mt * (KD / M::K);
    const int r = mt * 16 + (l & 15), g = l >> 4;
    union {
      typename M::frag f;
      E e[M::KPL];
    } x;
#pragma unroll
    for (int j = 0; j < M::KPL; ++j) x.e[j] = to_e<E>(val(r, kperm<E>(kt, g, j)));
    store_stream_small(dst + (size_t)u * M::KPL, x.f);
  }
}

// Write the A-buffer fragments (permuted order) that cover k in [k0, k0 + KS)
// of an R x KD matrix whose elements are val(r, k) (k relative to k0).
template <class E, int R, int KD, int KS, int NTH, class F>
__device__ inline void export_afrag_perm_kslice(E* dst, int k0, F&& val) {
  using M = Mfma<E>;
  constexpr int NKS = KS / M::K;
  constexpr int UNITS = R * KS / M::KPL;
  for (int u = threadIdx.x; u < UNITS; u += NTH) {
    const int tile = u >> 6, l = u & 63;
    const int mt = tile / NKS, ktl = tile - mt * NKS;
    const int r = mt * 16 + (l & 15), g = l >> 4;
    union {
      typename M::frag f;
      E e[M::KPL];
    } x;
#pragma unroll
    for (int j = 0; j < M::KPL; ++j) x.e[j] = to_e<E>(val(r, kperm<E>(ktl, g, j)));
    const size_t frag = (size_t)mt * (KD / M::K) + k0 / M::K + ktl;
    store_stream_small(dst + (frag * 64 + l) * M::KPL, x.f);
  }
}

// A or B operand (standard order) of row `row` of an LDS matrix, k-step kt,
// element k multiplied by sc[k].
template <class E>
__device__ inline typename Mfma<E>::frag load_frag_scaled(const E* row, int kt, const float* sc) {
  using M = Mfma<E>;
  const int k0 = kt * M::K + (lane_id() >> 4) * M::KPL;
  union {
    typename M::frag f;
    E e[M::KPL];
  } x;
  x.f = M::load(row + k0);
#pragma unroll
  for (int j = 0; j < M::KPL; ++j) x.e[j] = to_e<E>(to_f(x.e[j]) * sc[k0 + j]);
  return x.f;
}

// Copy one MFMA fragment (KPL elements per lane, lane-contiguous) from global
// memory straight into LDS with global_load_lds: lane l's elements land at
// lds_frag + l * KPL.  `lds_frag` must be the same for the whole wave.  It is
// issued from inline assembly so that the compiler does not wait on it: the
// caller owns the vmcnt bookkeeping (s_waitcnt before reading the LDS, and
// vmcnt(0) before the LDS is reused for anything else).  Copies are taken
// to complete in issue order among themselves, but an ordinary load issued
// after a copy may return before it: a partial vmcnt wait is sound only
// while no ordinary load issued after the awaited copies is in flight.
// The statement sets m0 (the LDS base of the copy).  The compiler treats m0
// as reserved and does not honour it as an asm clobber; these kernels rely
// on the compiler never holding a value in m0 itself, which
// tests/test_m0_use.py checks on the built code object: every write of m0 is
// one of these statements, directly followed by its copy.
template <class E> __device__ inline void dma_frag(const E* src_lane, E* lds_frag);
template <> __device__ inline void dma_frag<bf16>(const bf16* src_lane, bf16* lds_frag) {
  const unsigned lds = (unsigned)(uintptr_t)lds_frag;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src_lane)
               : "memory");
}
template <> __device__ inline void dma_frag<float>(const float* src_lane, float* lds_frag) {
  const unsigned lds = (unsigned)(uintptr_t)lds_frag;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(lds), "v"(src_lane)
               : "memory");
}
// Wait until at most N vector-memory operations of this wave are in flight.
template <int N> __device__ inline void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Copy a [ROWS][BV] tile from LDS (leading dim LD; columns v0..v0+BV of an
// R x N matrix) to global memory in MFMA fragment order over the columns:
// fragment (row tile rt, k-step kt) of lane l (row rt*16 + (l & 15), columns
// kt*K + KPL*(l >> 4) ..) at ((rt * NKT + kt) * 64 + l) * KPL, NKT = N / K.
// A reader then loads one fragment as one contiguous 1 KiB (bf16) block.
// Unrolled: all of a thread's LDS reads are issued before its stores, so no
// store waits on its own read.  ROLLED: one piece per loop trip, which keeps
// registers low.
template <class E, int ROWS, int BV, int LD, int NTH, bool ROLLED = false>
__device__ inline void copy_out_frags(E* g, int NKT, int v0, const E* lds) {
  using M = Mfma<E>;
  constexpr int EPV = 16 / sizeof(E);
  constexpr int VPR = BV / EPV;
  constexpr int PER = ROWS * VPR / NTH;  // 16-byte pieces per thread
  static_assert(ROWS * VPR % NTH == 0, "tile does not divide over the threads");
  auto put = [&](int idx, const uint4& val) {
    const int r = idx / VPR, cv = idx - r * VPR;
    const int v = v0 + cv * EPV;
    if (sizeof(E) == 2) {
      const int kt = v / M::K, lane = (r & 15) + 16 * ((v % M::K) / M::KPL);
      store_stream(g + ((size_t)((r >> 4) * NKT + kt) * 64 + lane) * M::KPL, val);
    } else {
      const E* x = reinterpret_cast<const E*>(&val);
#pragma unroll
      for (int q = 0; q < EPV; ++q) {
        const int vv = v + q, kt = vv / M::K, lane = (r & 15) + 16 * (vv % M::K);
        g[(size_t)((r >> 4) * NKT + kt) * 64 + lane] = x[q];
      }
    }
  };
  auto get = [&](int idx) {
    const int r = idx / VPR, cv = idx - r * VPR;
    return *reinterpret_cast<const uint4*>(lds + r * LD + cv * EPV);
  };
  if constexpr (ROLLED) {
    for (int idx = threadIdx.x; idx < ROWS * VPR; idx += NTH) put(idx, get(idx));
  } else {
    uint4 val[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) val[i] = get(threadIdx.x + i * NTH);
#pragma unroll
    for (int i = 0; i < PER; ++i) put(threadIdx.x + i * NTH, val[i]);
  }
}

// One wave writes its 16 rows of a 64 x BV tile staged in LDS (row-major, row
// stride LD, rows 16 w ..) to global rows of stride rs, 16 bytes per lane and
// store; rows at or past nvalid are skipped.
template <class E, int BV, int LD>
__device__ inline void wave_rows_out(E* g, size_t rs, const E* lds, int w, int nvalid) {
  constexpr int EPV = 16 / sizeof(E);
  constexpr int VPR = BV / EPV;          // 16-byte pieces per row
  constexpr int PER = 16 * VPR / 64;     // pieces per lane
  static_assert(16 * VPR % 64 == 0, "rows do not divide over the lanes");
  const int l = threadIdx.x & 63;
  uint4 val[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int idx = l + 64 * i, r = 16 * w + idx / VPR, cv = idx % VPR;
    val[i] = *reinterpret_cast<const uint4*>(lds + r * LD + cv * EPV);
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int idx = l + 64 * i, r = 16 * w + idx / VPR, cv = idx % VPR;
    if (r < nvalid) store_stream(g + (size_t)r * rs + cv * EPV, val[i]);
  }
}

// 1 / (1 + e^-x) with the hardware reciprocal (1 ulp) instead of a full
// IEEE division sequence (the block prologue's and epilogue's SiLU)
__device__ inline float sigmoidf(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

// Inclusive prefix sum across the 64 lanes of a wave.
__device__ inline float wave_incl_scan(float x) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float y = __shfl_up(x, off, 64);
    if (l >= off) x += y;
  }
  return x;
}

// f(std::integral_constant<int, i>) for i = I .. N-1, unrolled at compile
// time (for code whose constants depend on the iteration, such as wait counts).
template <int I, int N, class F>
__device__ inline void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// x of another lane of the same 16-lane row, by a DPP lane pattern.
template <int CTRL>
__device__ inline float dpp_row(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), CTRL,
                                                            0xF, 0xF, true));
}

// Sum over the 16 lanes that share (l >> 4) (the columns of an accumulator
// tile): pairs (lane ^ 1), then (lane ^ 2), then the two quads of each half
// row (mirror within 8 lanes), then the two halves (mirror within 16).  Four
// VALU adds with DPP operands, no LDS traffic; every lane ends with the same
// sum, formed in the same order as an xor butterfly.  All 64 lanes must be
// active.
__device__ inline float reduce16(float x) {
  x += dpp_row<0xB1>(x);   // quad_perm [1, 0, 3, 2]
  x += dpp_row<0x4E>(x);   // quad_perm [2, 3, 0, 1]
  x += dpp_row<0x141>(x);  // row_half_mirror
  x += dpp_row<0x140>(x);  // row_mirror
  return x;
}

}  // namespace gdn

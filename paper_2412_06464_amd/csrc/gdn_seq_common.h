// Helpers of the sequential state passes (gdn_seq.hip).
#pragma once
#include "gdn_device.h"

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

// L2 warm-up of a later chunk: the state passes read each chunk's dk-side
// operands when they reach it, and their latency from HBM is most of a
// chunk's time.  The dv slices of a unit share those operands through L2;
// here wave 0 of slice `slice` (of `nslices`) loads one dword of each of its
// 128-byte lines (lines slice, slice + nslices, ...) of each buffer, so that
// the slices' own loads, a few chunks later, find them in L2.  The loads
// land in LDS (global_load_lds_dword into `sink`, 256 bytes that nothing
// reads), so no register stays live for them.  The compiler does not see
// these loads, so its own vmcnt waits only get stricter, never looser; the
// caller waits for them (vmcnt(0)) before the workgroup ends.  Like
// dma_frag (gdn_device.h), the statement sets m0, which the compiler never
// uses in these kernels (checked on the built code object).
template <int NB>
__device__ inline void warm_l2(const unsigned char* const (&base)[NB], const int (&bytes)[NB],
                               int slice, int nslices, float* sink) {
  constexpr int WL = 128;  // L2 line
  const unsigned lds = (unsigned)(uintptr_t)sink;
  const int idx = slice + nslices * lane_id();
  const unsigned off = (unsigned)idx * WL;  // lane offset (the bases are uniform, in SGPRs)
#pragma unroll
  for (int b = 0; b < NB; ++b)
    if (idx < bytes[b] / WL)
      asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2" ::"s"(lds), "v"(off),
                   "s"(base[b])
                   : "memory");
}

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

}  // namespace gdn

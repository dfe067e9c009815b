// Launch sequences of the forward and backward calls, with optional event
// recording around every launch.
#include "gdn_kernels.h"

namespace gdn {

namespace {

// Run one launch, bracketed by the caller's timing events if any.
template <class F>
hipError_t timed(Timing* t, const char* name, hipStream_t s, F&& launch) {
  const int i = t ? t->launched : 0;
  const bool rec = t && 2 * i + 1 < t->capacity;
  if (rec && hipEventRecord(t->events[2 * i], s) != hipSuccess) return hipErrorInvalidValue;
  const hipError_t e = launch();
  if (e != hipSuccess) return e;
  if (rec && hipEventRecord(t->events[2 * i + 1], s) != hipSuccess) return hipErrorInvalidValue;
  if (t) {
    if (i < 8) t->names[i] = name;
    t->launched = i + 1;
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t,
                      bool block) {
  hipError_t e;
  // the chunk table serves packed input only; dense chunks are arithmetic
  if (a.cu && (e = timed(t, "k_chunk_table", s, [&] { return launch_chunk_table(a, s); })) !=
                  hipSuccess)
    return e;
  if ((e = timed(t, block ? "k_prep_block" : "k_prep", s,
                 [&] { return launch_prep(dt, dk, dv, PREP_FWD, a, s, block); })) != hipSuccess)
    return e;
  return timed(t, "k_fwd_seq", s, [&] { return launch_fwd_seq(dt, dk, dv, SEQ_FWD, a, s); });
}

hipError_t launch_bwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t) {
  hipError_t e;
  // the chunk table serves packed input only; dense chunks are arithmetic
  if (a.cu && (e = timed(t, "k_chunk_table", s, [&] { return launch_chunk_table(a, s); })) !=
                  hipSuccess)
    return e;
  if ((e = timed(t, "k_prep", s, [&] { return launch_prep(dt, dk, dv, PREP_BWD, a, s); })) !=
      hipSuccess)
    return e;
  if ((e = timed(t, "k_fwd_seq_store", s,
                 [&] { return launch_fwd_seq(dt, dk, dv, SEQ_STORE, a, s); })) != hipSuccess)
    return e;
  if ((e = timed(t, "k_bwd_seq", s, [&] { return launch_bwd_seq(dt, dk, dv, a, s); })) !=
      hipSuccess)
    return e;
  return timed(t, "k_grad", s, [&] { return launch_grad(dt, dk, dv, a, s); });
}

// Forward that keeps what the backward needs: the prep writes both operand
// sets and the state pass stores chunk states and V' beside O.
hipError_t launch_fwd_save(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t,
                           bool block) {
  hipError_t e;
  // the chunk table serves packed input only; dense chunks are arithmetic
  if (a.cu && (e = timed(t, "k_chunk_table", s, [&] { return launch_chunk_table(a, s); })) !=
                  hipSuccess)
    return e;
  if ((e = timed(t, block ? "k_prep_save_block" : "k_prep_save", s,
                 [&] { return launch_prep(dt, dk, dv, PREP_SAVE, a, s, block); })) != hipSuccess)
    return e;
  return timed(t, "k_fwd_seq_save", s,
               [&] { return launch_fwd_seq(dt, dk, dv, SEQ_SAVE, a, s); });
}

// Backward from a saving forward's buffer: no prep, no recompute.
hipError_t launch_bwd_saved(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t) {
  hipError_t e;
  // the chunk table serves packed input only; dense chunks are arithmetic
  if (a.cu && (e = timed(t, "k_chunk_table", s, [&] { return launch_chunk_table(a, s); })) !=
                  hipSuccess)
    return e;
  if ((e = timed(t, "k_bwd_seq", s, [&] { return launch_bwd_seq(dt, dk, dv, a, s); })) !=
      hipSuccess)
    return e;
  return timed(t, "k_grad", s, [&] { return launch_grad(dt, dk, dv, a, s); });
}

// Backward of the fused block from a saving fused forward's buffer.  The
// chunk table is built for dense input too: the v prologue's backward reads
// it.  The reverse pass writes the rule's dv (a.dv, a temporary here), the
// gradient kernel folds in the q and k prologue, the fix-up finishes dx
// across chunk boundaries and sums dw, and the v prologue's backward runs
// on the rule's dv.
hipError_t launch_block_bwd_saved(int dk, int dv, const Args& a, const ConvArgs& cv,
                                  hipStream_t s, Timing* t) {
  hipError_t e;
  if ((e = timed(t, "k_chunk_table", s, [&] { return launch_chunk_table(a, s); })) != hipSuccess)
    return e;
  if ((e = timed(t, "k_bwd_seq", s, [&] { return launch_bwd_seq(Dt::BF16, dk, dv, a, s); })) !=
      hipSuccess)
    return e;
  if ((e = timed(t, "k_grad_block", s,
                 [&] { return launch_grad(Dt::BF16, dk, dv, a, s, true); })) != hipSuccess)
    return e;
  if ((e = timed(t, "k_block_fixup", s, [&] { return launch_block_fixup(dk, a, s); })) !=
      hipSuccess)
    return e;
  return timed(t, "k_conv_bwd", s, [&] { return launch_conv_bwd(Dt::BF16, dv, cv, s); });
}

// Token-by-token form: one launch, no workspace.
hipError_t launch_recurrent_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t) {
  return timed(t, "k_recurrent", s, [&] { return launch_recurrent(dt, dk, dv, a, s); });
}

}  // namespace gdn

// Launch sequences of the forward and backward calls, with optional event
// recording around every launch.
#include <string.h>

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

// Pointer fields of Args, in audit order.
#define GDN_AUDIT_FIELDS(X)                                                                    \
  X(q) X(k) X(v) X(beta) X(log_alpha) X(h0) X(dO) X(dht) X(o) X(ht) X(dq) X(dk) X(dv) X(dbeta) \
  X(dlog_alpha) X(dh0) X(cu) X(info) X(seq_chunk0) X(g) X(Wf) X(KbT) X(Uc) X(Pf) X(Qf) X(Kf)  \
  X(PTf) X(TTf) X(nWT) X(QgT) X(Ak) X(Sc) X(Vp) X(dSc) X(dXb) X(gpart) X(xq) X(xk) X(xv)      \
  X(cwq) X(cwk) X(cwv) X(yq) X(yk) X(yv) X(bhead) X(btail) X(bpart) X(btmp) X(dwq) X(dwk)

enum Field : int {
#define GDN_ENUM(f) F_##f,
  GDN_AUDIT_FIELDS(GDN_ENUM)
#undef GDN_ENUM
  F_COUNT
};
static_assert(F_COUNT == AUDIT_FIELDS, "audit field count");

constexpr uint64_t bit(Field f) { return 1ull << f; }
template <class... F>
constexpr uint64_t bits(F... f) {
  return (bit(f) | ...);
}

// What each sequence reads or writes unconditionally.
constexpr uint64_t FWD_OPS = bits(F_g, F_Wf, F_KbT, F_Uc, F_Pf, F_Qf);
constexpr uint64_t SAVED = bits(F_g, F_Kf, F_PTf, F_TTf, F_nWT, F_QgT, F_Ak, F_Sc, F_Vp);
constexpr uint64_t BWD_WS = bits(F_dSc, F_dXb, F_gpart);
constexpr uint64_t BWD_IO = bits(F_beta, F_dO, F_dq, F_dk, F_dv, F_dbeta);
constexpr uint64_t RULE_IN = bits(F_q, F_k, F_v, F_beta);
constexpr uint64_t PRO_IN = bits(F_xq, F_xk, F_xv, F_cwq, F_cwk, F_cwv, F_beta);

uint64_t required(Seq s) {
  switch (s) {
    case Seq::Fwd: return RULE_IN | bit(F_o) | FWD_OPS;
    case Seq::Bwd: return RULE_IN | BWD_IO | bits(F_Wf, F_KbT, F_Uc) | SAVED | BWD_WS;
    case Seq::FwdSave: return RULE_IN | bit(F_o) | FWD_OPS | SAVED;
    case Seq::BwdSaved: return RULE_IN | BWD_IO | SAVED | BWD_WS;
    case Seq::Recurrent: return RULE_IN | bit(F_o);
    case Seq::BlockFwd: return PRO_IN | bit(F_o) | FWD_OPS;
    case Seq::BlockFwdSave: return PRO_IN | bit(F_o) | FWD_OPS | SAVED | bits(F_yq, F_yk, F_yv);
    case Seq::BlockBwdSaved:
      return RULE_IN | BWD_IO | SAVED | BWD_WS | bits(F_xq, F_xk, F_cwq, F_cwk, F_info,
                                                        F_seq_chunk0, F_bhead, F_btail, F_bpart,
                                                        F_btmp, F_dwq, F_dwk);
  }
  return 0;
}

const void* field(const Args& a, int i) {
  switch (i) {
#define GDN_CASE(f) \
  case F_##f:       \
    return (const void*)a.f;
    GDN_AUDIT_FIELDS(GDN_CASE)
#undef GDN_CASE
  }
  return nullptr;
}

}  // namespace

const char* const audit_field_names[AUDIT_FIELDS] = {
#define GDN_NAME(f) #f,
    GDN_AUDIT_FIELDS(GDN_NAME)
#undef GDN_NAME
};

int audit(Seq s, const Args& a) {
  uint64_t need = required(s);
  // the gates are read unless alpha == 1 (the saved backward reads them from
  // the saved buffer); packed input reads the chunk table
  if (a.gated && s != Seq::BwdSaved && s != Seq::BlockBwdSaved) need |= bit(F_log_alpha);
  if (a.cu && s != Seq::Recurrent) need |= bits(F_info, F_seq_chunk0);
  for (int i = 0; i < F_COUNT; ++i)
    if ((need >> i & 1) && !field(a, i)) return i;
  return -1;
}

Args audit_probe(uint64_t present) {
  Args a;
  memset(&a, 0, sizeof a);
  char* dummy = reinterpret_cast<char*>(0x1000);
#define GDN_SET(f) \
  if (present >> F_##f & 1) a.f = reinterpret_cast<decltype(a.f)>(dummy);
  GDN_AUDIT_FIELDS(GDN_SET)
#undef GDN_SET
  a.gated = a.log_alpha != nullptr;
  return a;
}

hipError_t launch_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t,
                      bool block) {
  if (audit(block ? Seq::BlockFwd : Seq::Fwd, a) >= 0) return hipErrorInvalidValue;
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
  if (audit(Seq::Bwd, a) >= 0) return hipErrorInvalidValue;
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
  if (audit(block ? Seq::BlockFwdSave : Seq::FwdSave, a) >= 0) return hipErrorInvalidValue;
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
  if (audit(Seq::BwdSaved, a) >= 0) return hipErrorInvalidValue;
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
                                  const ConvArgs* cq, const ConvArgs* ck, hipStream_t s,
                                  Timing* t) {
  if (audit(Seq::BlockBwdSaved, a) >= 0) return hipErrorInvalidValue;
  hipError_t e;
  if ((e = timed(t, "k_chunk_table", s, [&] { return launch_chunk_table(a, s); })) != hipSuccess)
    return e;
  if ((e = timed(t, "k_bwd_seq", s, [&] { return launch_bwd_seq(Dt::BF16, dk, dv, a, s); })) !=
      hipSuccess)
    return e;
  if (cq && ck) {  // composed: the rule's dq, dk, then the prologue's backward of q and k
    if (!a.dq || !a.dk || !cq->dy || !ck->dy || !cq->part || !ck->part || !cq->tmp)
      return hipErrorInvalidValue;
    if ((e = timed(t, "k_grad", s, [&] { return launch_grad(Dt::BF16, dk, dv, a, s, false); })) !=
        hipSuccess)
      return e;
    if ((e = timed(t, "k_conv_bwd_qk", s, [&] {
           hipError_t r = launch_conv_bwd(Dt::BF16, dk, *cq, s);
           return r == hipSuccess ? launch_conv_bwd(Dt::BF16, dk, *ck, s) : r;
         })) != hipSuccess)
      return e;
  } else {
    if ((e = timed(t, "k_grad_block", s,
                   [&] { return launch_grad(Dt::BF16, dk, dv, a, s, true); })) != hipSuccess)
      return e;
    if ((e = timed(t, "k_block_fixup", s, [&] { return launch_block_fixup(dk, a, s); })) !=
        hipSuccess)
      return e;
  }
  return timed(t, "k_conv_bwd", s, [&] { return launch_conv_bwd(Dt::BF16, dv, cv, s); });
}

// Token-by-token form: one launch, no workspace.
hipError_t launch_recurrent_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t) {
  if (audit(Seq::Recurrent, a) >= 0) return hipErrorInvalidValue;
  return timed(t, "k_recurrent", s, [&] { return launch_recurrent(dt, dk, dv, a, s); });
}

}  // namespace gdn

// Kernel argument block and launcher declarations shared by the HIP
// translation units of libgdn.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

// One packed description of a call.  Device pointers unless noted.
// Per-chunk buffers are indexed by ch = chunk * H + head.
struct Args {
  int H;       // heads
  int N;       // sequences (dense: B)
  int NC;      // total chunks over all sequences
  int T;       // dense sequence length (used when cu == nullptr)
  int gated;   // 0: alpha == 1 (no log_alpha input): g = 0, no gate math
  const int32_t* cu;  // packed boundaries [N+1] or nullptr (dense)
  // inputs
  const void *q, *k, *v, *dO;
  const float *beta, *log_alpha, *h0, *dht;
  // outputs
  void *o, *dq, *dk, *dv;
  float *ht, *dbeta, *dlog_alpha, *dh0;
  // workspace: chunk table and per-chunk gates
  int4* info;       // [NC] {sequence, first token row, length, 0}
  int* seq_chunk0;  // [N+1] first chunk of every sequence
  float* g;         // [ch][64]     cumulative log gate inside the chunk
  // workspace: per-chunk operands of the sequential passes (dtype E), as MFMA
  // A operands in fragment order with the permuted contraction order
  void* Wf;   // W~ = T diag(b e^g) K      rows t, k = d     64 x dk
  void* KbT;  // Kbar^T                    rows d, k = t     dk x 64
  void* Uc;   // U~ = T diag(b) V          accumulator layout 64 x dv
  void* Pf;   // P                         rows t, k = t'    64 x 64  (forward)
  void* Qf;   // diag(e^g) Q               rows t, k = d     64 x dk  (forward)
  void* Kf;   // K                         rows t, k = d     64 x dk  (backward)
  void* PTf;  // P^T                       rows t', k = t    64 x 64  (backward)
  void* TTf;  // T^T                       rows t', k = t    64 x 64  (backward)
  void* nWT;  // -W~^T                     rows d, k = t     dk x 64  (backward)
  void* QgT;  // (diag(e^g) Q)^T           rows d, k = t     dk x 64  (backward)
  // workspace: backward intermediate for the gradient kernel (which also
  // reads P^T)
  void* Ak;   // Ak^T, Ak = strictLower(Gamma K K^T)
              //                           rows t', k = t    64 x 64  (backward)
  // per-chunk matrices over dv, B operands of the gradient kernel in
  // fragment order over dv (fragment (16-row tile, k-step) of 64 lanes)
  void* Sc;   // [ch] chunk entry states          dk x dv
  void* Vp;   // [ch] V' = U~ - W~ S              64 x dv
  void* dSc;  // [ch] gradient of each chunk's exit state  dk x dv
  void* dXb;  // [ch] dX = T^T dV'                64 x dv
  // workspace: the gradient kernel's partial row sums for the gate gradients
  float* gpart;  // [ch][GRAD_PART_FLOATS]
  // fused block prologue: causal depthwise convolution of width cw, SiLU,
  // and L2 (eps ceps) for q and k, of the projections xq, xk, xv
  const void *xq, *xk, *xv;      // [*, T, H, d]
  const float *cwq, *cwk, *cwv;  // weights [H * d][cw]
  int cw;
  float ceps;
  void *yq, *yk, *yv;            // the forward's outputs: the rule's q, k, v
  // its backward in the gradient kernel (which reads the rule's q, k, v
  // through q, k, v; dq, dk are then dxq, dxk), for q and then k:
  // [2][NC * H][3][dk] du of each chunk's first three rows and partial dx of
  // its last three, [2][NC * H][dk][cw] per-chunk partial weight gradients,
  // their slice sums, and the weight gradients [H * dk][cw]
  float *bhead, *btail, *bpart, *btmp;
  float *dwq, *dwk;
};

// Floats per chunk-head of Args::gpart (twelve blocks of one chunk, 64).
constexpr int GRAD_PART_FLOATS = 12 * 64;

enum class Dt { F32, BF16 };

// Block prologue: short causal convolution + SiLU (+ L2) over [*, T, H, D].
struct ConvArgs {
  int H, N, NC, T;           // heads, sequences, chunks, dense length
  int W, l2;                 // convolution width (1..4), L2 normalisation on/off
  float eps;
  const int32_t* cu;         // packed boundaries or nullptr
  const int4* info;          // chunk table (sequence, first token, length)
  const void* x;             // input  [*, T, H, D]
  const float* w;            // weights [H * D][W]
  const void* dy;            // gradient of the output
  void* y;                   // output
  void* dx;                  // gradient of the input
  float* part;               // [NC][H][D][W] per-chunk partial weight gradients
  float* tmp;                // [ceil(NC / 256)][H][D][W] slice sums of part
  float* dw;                 // weight gradient [H * D][W]
};

// Block epilogue: RMS normalisation x weight x SiLU gate over the dv channels.
struct NormArgs {
  long rows;                 // (token, head) rows
  int nblk;                  // workgroups (64 rows each)
  float eps;
  const void *o, *g, *dy;    // [rows][dv]
  const float* w;            // [dv]
  void *y, *dout, *dg;       // [rows][dv]
  float* part;               // [nblk][dv] partial weight gradients
  float* tmp;                // [ceil(nblk / 256)][dv] slice sums of part
  float* dw;                 // [dv]
};

// What a prep launch writes: the forward pass's operands, the stateless
// backward's (including those its forward recompute needs), or both (a
// forward that saves what the backward needs).
enum { PREP_FWD = 0, PREP_BWD = 1, PREP_SAVE = 2 };
// What a forward state pass does: the forward (O, final state), the
// backward's recompute (chunk states and V'), or both.
enum { SEQ_FWD = 0, SEQ_STORE = 1, SEQ_SAVE = 2 };

// Optional event recording around every launch (caller-owned events).
struct Timing {
  hipEvent_t* events;
  int capacity;
  int launched;
  const char** names;  // at least 8 entries
};

// The launch sequences, for the pointer audit.
enum class Seq { Fwd, Bwd, FwdSave, BwdSaved, Recurrent, BlockFwd, BlockFwdSave, BlockBwdSaved };
constexpr int SEQ_COUNT = 8;
// The Args pointers the audit knows, by index (names for diagnostics).
constexpr int AUDIT_FIELDS = 51;
extern const char* const audit_field_names[AUDIT_FIELDS];
// Index of the first pointer that sequence s dereferences and a lacks, or
// -1.  (Whether log_alpha and the chunk table are needed follows a.gated and
// a.cu.)  Every launch sequence below checks it before its first launch.
int audit(Seq s, const Args& a);
// An Args whose pointer fields are a dummy non-null address where bit i of
// present is set (for tests of the audit only; never launched).
Args audit_probe(uint64_t present);

// Individual launches (each returns the launch status).
hipError_t launch_chunk_table(const Args& a, hipStream_t s);
hipError_t launch_prep(Dt dt, int dk, int dv, int mode, const Args& a, hipStream_t s,
                       bool block = false);
hipError_t launch_fwd_seq(Dt dt, int dk, int dv, int mode, const Args& a, hipStream_t s);
hipError_t launch_bwd_seq(Dt dt, int dk, int dv, const Args& a, hipStream_t s);
hipError_t launch_grad(Dt dt, int dk, int dv, const Args& a, hipStream_t s, bool block = false);
hipError_t launch_block_fixup(int dk, const Args& a, hipStream_t s);
hipError_t launch_sum_rows(const float* part, int N, int M, float* tmp, float* out, hipStream_t s);
hipError_t launch_recurrent(Dt dt, int dk, int dv, const Args& a, hipStream_t s);
hipError_t launch_conv_fwd(Dt dt, int d, const ConvArgs& a, hipStream_t s);
hipError_t launch_conv_bwd(Dt dt, int d, const ConvArgs& a, hipStream_t s);
hipError_t launch_norm_gate_fwd(Dt dt, int dv, const NormArgs& a, hipStream_t s);
hipError_t launch_norm_gate_bwd(Dt dt, int dv, const NormArgs& a, hipStream_t s);

// The forward / backward sequences, with optional timing.
hipError_t launch_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t,
                      bool block = false);
hipError_t launch_bwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t);
hipError_t launch_fwd_save(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t,
                           bool block = false);
hipError_t launch_bwd_saved(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t);
// Backward of prologue + rule from a saving fused forward: the rule's
// backward with the q and k prologue folded into the gradient kernel, then
// the v prologue's backward (cv, on the rule's dv).
hipError_t launch_block_bwd_saved(int dk, int dv, const Args& a, const ConvArgs& cv,
                                  const ConvArgs* cq, const ConvArgs* ck, hipStream_t s,
                                  Timing* t);
hipError_t launch_recurrent_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s, Timing* t);

// Call a lambda templated on (element type, dk, dv) for the supported
// shapes; returns hipErrorInvalidValue for anything else.
#define GDN_DISPATCH(dt, dk, dv, f)                                                         \
  do {                                                                                      \
    if ((dt) == Dt::F32 && (dk) == 64 && (dv) == 64)                                        \
      return (f).template operator()<float, 64, 64>();                                      \
    if ((dt) == Dt::F32 && (dk) == 128 && (dv) == 128)                                      \
      return (f).template operator()<float, 128, 128>();                                    \
    if ((dt) == Dt::F32 && (dk) == 256 && (dv) == 512)                                      \
      return (f).template operator()<float, 256, 512>();                                    \
    if ((dt) == Dt::BF16 && (dk) == 64 && (dv) == 64)                                       \
      return (f).template operator()<__bf16, 64, 64>();                                     \
    if ((dt) == Dt::BF16 && (dk) == 128 && (dv) == 128)                                     \
      return (f).template operator()<__bf16, 128, 128>();                                   \
    if ((dt) == Dt::BF16 && (dk) == 256 && (dv) == 512)                                     \
      return (f).template operator()<__bf16, 256, 512>();                                   \
    return hipErrorInvalidValue;                                                            \
  } while (0)

}  // namespace gdn

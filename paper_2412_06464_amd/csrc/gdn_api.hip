// C ABI of libgdn: argument validation, workspace carve-up and launch
// sequencing.  Every check runs before the first launch; nothing here
// allocates, frees or synchronises.
#include <atomic>
#include <stdint.h>
#include <string.h>

#include <math.h>

#include <mutex>
#include <new>

#include "../../include/gdn.h"
#include "gdn_kernels.h"

namespace {

using gdn::Args;
using gdn::Dt;

constexpr int CH = 64;
constexpr size_t ALIGN = 256;

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

struct Shape {
  int N = 0;      // sequences
  long NC = 0;    // chunks
  long Ttot = 0;  // tokens
  size_t esz = 0; // element bytes of q/k/v
};

gdn_status check_problem(const gdn_problem* p, Shape* out) {
  if (!p) return GDN_ERR_NULL;
  if (p->dtype != GDN_F32 && p->dtype != GDN_BF16) return GDN_ERR_UNSUPPORTED;
  if (p->B < 1 || p->T < 1 || p->H < 1) return GDN_ERR_SHAPE;
  const bool ok_dims = (p->dk == 64 && p->dv == 64) || (p->dk == 128 && p->dv == 128) ||
                       (p->dk == 256 && p->dv == 512);
  if (!ok_dims) return GDN_ERR_UNSUPPORTED;
  const long Ttot = (long)p->B * p->T;
  if (Ttot * (long)p->H * (p->dk > p->dv ? p->dk : p->dv) >= (1L << 40)) return GDN_ERR_SHAPE;
  if (Ttot >= (1L << 31)) return GDN_ERR_SHAPE;
  Shape s;
  s.Ttot = Ttot;
  s.esz = p->dtype == GDN_F32 ? 4 : 2;
  if (p->cu_seqlens) {
    if (p->B != 1) return GDN_ERR_SHAPE;
    if (!p->cu_seqlens_host || p->num_seqs < 1) return GDN_ERR_CU_SEQLENS;
    const int32_t* cu = p->cu_seqlens_host;
    if (cu[0] != 0 || cu[p->num_seqs] != p->T) return GDN_ERR_CU_SEQLENS;
    long nc = 0;
    for (int n = 0; n < p->num_seqs; ++n) {
      if (cu[n + 1] < cu[n]) return GDN_ERR_CU_SEQLENS;
      nc += (cu[n + 1] - cu[n] + CH - 1) / CH;
    }
    s.N = p->num_seqs;
    s.NC = nc;
  } else {
    if (p->cu_seqlens_host) return GDN_ERR_CU_SEQLENS;
    s.N = p->B;
    s.NC = (long)p->B * ((p->T + CH - 1) / CH);
  }
  if (s.NC >= (1L << 31) / CH) return GDN_ERR_SHAPE;
  *out = s;
  return GDN_OK;
}

// Buffer layouts; `base` may be null to only compute the size.
enum class Use { Fwd, Bwd, FwdSave, BwdSaved };

struct Carver {
  unsigned char* base;
  size_t off = 0;
  unsigned char* take(size_t bytes) {
    unsigned char* ptr = base ? base + off : nullptr;
    off += up(bytes);
    return ptr;
  }
};

struct Sizes {
  size_t kside, vside, cc, st;
  Sizes(const gdn_problem* p, const Shape& s) {
    const size_t NC = (size_t)s.NC, H = (size_t)p->H;
    kside = NC * H * CH * (size_t)p->dk * s.esz;        // 64 x dk per chunk
    vside = NC * H * CH * (size_t)p->dv * s.esz;        // 64 x dv per chunk
    cc = NC * H * CH * CH * s.esz;                      // 64 x 64 per chunk
    st = NC * H * (size_t)p->dk * p->dv * s.esz;        // dk x dv per chunk
  }
};

// What the backward reads from the forward: the gates' cumulative sums, the
// reverse pass's and gradient kernel's per-chunk operands, each chunk's entry
// state and V'.  A saving forward writes it; the stateless backward keeps it
// in its workspace.
void carve_saved(const gdn_problem* p, const Shape& s, Carver& c, Args* a) {
  const Sizes z(p, s);
  unsigned char* g = c.take((size_t)s.NC * p->H * CH * sizeof(float));
  unsigned char* Kf = c.take(z.kside);
  unsigned char* PTf = c.take(z.cc);
  unsigned char* TTf = c.take(z.cc);
  unsigned char* nWT = c.take(z.kside);
  unsigned char* QgT = c.take(z.kside);
  unsigned char* Ak = c.take(z.cc);
  unsigned char* Sc = c.take(z.st);
  unsigned char* Vp = c.take(z.vside);
  if (a) {
    a->g = (float*)g;
    a->Kf = Kf;
    a->PTf = PTf;
    a->TTf = TTf;
    a->nWT = nWT;
    a->QgT = QgT;
    a->Ak = Ak;
    a->Sc = Sc;
    a->Vp = Vp;
  }
}

size_t saved_bytes(const gdn_problem* p, const Shape& s) {
  Carver c{nullptr};
  carve_saved(p, s, c, nullptr);
  return c.off;
}

// Workspace of one entry point: the chunk table, then what its kernels pass
// between each other and the caller does not keep.
size_t carve(const gdn_problem* p, const Shape& s, Use u, unsigned char* base, Args* a) {
  const Sizes z(p, s);
  Carver c{base};
  unsigned char* info = c.take((size_t)s.NC * sizeof(int4) + 16);
  unsigned char* sc0 = c.take(((size_t)s.N + 1) * sizeof(int));
  if (a) {
    a->info = (int4*)info;
    a->seq_chunk0 = (int*)sc0;
  }
  if (u != Use::BwdSaved) {  // the forward pass's operands (the recompute's too)
    unsigned char* Wf = c.take(z.kside);
    unsigned char* KbT = c.take(z.kside);
    unsigned char* Uc = c.take(z.vside);
    if (a) {
      a->Wf = Wf;
      a->KbT = KbT;
      a->Uc = Uc;
    }
  }
  if (u == Use::Fwd || u == Use::FwdSave) {  // those only the output needs
    unsigned char* Pf = c.take(z.cc);
    unsigned char* Qf = c.take(z.kside);
    if (a) {
      a->Pf = Pf;
      a->Qf = Qf;
    }
  }
  if (u == Use::Fwd) {
    unsigned char* g = c.take((size_t)s.NC * p->H * CH * sizeof(float));
    if (a) a->g = (float*)g;
  }
  if (u == Use::Bwd) carve_saved(p, s, c, a);
  if (u == Use::Bwd || u == Use::BwdSaved) {  // the reverse pass's chunk states and dX,
    // and the gradient kernel's partial sums
    unsigned char* dSc = c.take(z.st);
    unsigned char* dXb = c.take(z.vside);
    unsigned char* gp = c.take((size_t)s.NC * p->H * gdn::GRAD_PART_FLOATS * sizeof(float));
    if (a) {
      a->dSc = dSc;
      a->dXb = dXb;
      a->gpart = (float*)gp;
    }
  }
  return c.off;
}

// Bridges the C timing struct to the launchers' view of it.
class TimingGuard {
 public:
  explicit TimingGuard(gdn_timing* t) : t_(t) {
    if (t_) {
      t_->launched = 0;
      for (auto& n : t_->names) n = nullptr;
      impl_.events = (hipEvent_t*)t_->events;
      impl_.capacity = t_->events ? t_->capacity : 0;
      impl_.launched = 0;
      impl_.names = t_->names;
    }
  }
  ~TimingGuard() {
    if (t_) t_->launched = impl_.launched;
  }
  gdn::Timing* get() { return t_ ? &impl_ : nullptr; }

 private:
  gdn_timing* t_;
  gdn::Timing impl_{};
};

// Block prologue: argument checks and workspace (chunk table, then the
// per-chunk partial weight gradients of the backward).
gdn_status check_conv(const gdn_problem* p, int dim, int width, float eps, Shape* s) {
  const gdn_status st = check_problem(p, s);
  if (st != GDN_OK) return st;
  if (dim != p->dk && dim != p->dv) return GDN_ERR_UNSUPPORTED;
  if (width < 1 || width > 4 || !(eps >= 0.f) || !isfinite(eps)) return GDN_ERR_VALUE;
  return GDN_OK;
}

size_t carve_conv(const gdn_problem* p, const Shape& s, int dim, int width, unsigned char* base,
                  Args* t, gdn::ConvArgs* a) {
  Carver c{base};
  unsigned char* info = c.take((size_t)s.NC * sizeof(int4) + 16);
  unsigned char* sc0 = c.take(((size_t)s.N + 1) * sizeof(int));
  const size_t row = (size_t)p->H * dim * width * sizeof(float);
  unsigned char* part = c.take((size_t)s.NC * row);
  unsigned char* tmp = c.take((size_t)((s.NC + 255) / 256) * row);
  if (t) {
    t->info = (int4*)info;
    t->seq_chunk0 = (int*)sc0;
  }
  if (a) {
    a->info = (const int4*)info;
    a->part = (float*)part;
    a->tmp = (float*)tmp;
  }
  return c.off;
}

// Fused block (prologue + rule): checks of the prologue description.
gdn_status check_block(const gdn_problem* p, const gdn_block_prologue* b, Shape* s) {
  const gdn_status st = check_problem(p, s);
  if (st != GDN_OK) return st;
  if (!b) return GDN_ERR_NULL;
  if (p->dtype != GDN_BF16) return GDN_ERR_UNSUPPORTED;
  if (b->width < 1 || b->width > 4 || !(b->eps >= 0.f) || !isfinite(b->eps)) return GDN_ERR_VALUE;
  const void* ptrs[] = {b->xq, b->xk, b->xv, b->wq, b->wk, b->wv};
  for (const void* x : ptrs)
    if (!x) return GDN_ERR_NULL;
  for (const void* x : ptrs)
    if (!aligned16(x)) return GDN_ERR_ALIGN;
  return GDN_OK;
}

void fill_prologue(const gdn_block_prologue* b, Args* a) {
  a->xq = b->xq;
  a->xk = b->xk;
  a->xv = b->xv;
  a->cwq = b->wq;
  a->cwk = b->wk;
  a->cwv = b->wv;
  a->cw = b->width;
  a->ceps = b->eps;
}

// Workspace of the fused block's backward: the rule's backward workspace,
// then the rule's dv (the v prologue's input gradient), the q and k
// prologue's side buffers and per-chunk weight gradients, and the v
// prologue's per-chunk weight gradients.
// Backward of the fused block at dk >= 128: the gradient kernel with the
// prologue's backward inside holds one workgroup per CU there, and the plain
// gradient kernel followed by the standalone convolution backward of q and k
// measured faster; at dk = 64 the fused kernel is the faster.  A test can
// force either form (gdn_debug_block_bwd).
std::atomic<int> block_bwd_mode{0};  // 0: by dk, 1: fused, 2: composed

bool block_bwd_composed(const gdn_problem* p) {
  const int m = block_bwd_mode.load();
  return m == 2 || (m == 0 && p->dk >= 128);
}

// dyqk (when given) receives the two buffers of the composed form's rule
// gradients dq, dk.
size_t carve_block_bwd(const gdn_problem* p, const Shape& s, int width, unsigned char* base,
                       Args* a, gdn::ConvArgs* cv, unsigned char** dyqk = nullptr) {
  Carver c{base, carve(p, s, Use::BwdSaved, base, a)};
  const size_t NCH = (size_t)s.NC * p->H, NS = (size_t)((s.NC + 255) / 256);
  unsigned char* dyq = c.take((size_t)s.Ttot * p->H * p->dk * s.esz);
  unsigned char* dyk = c.take((size_t)s.Ttot * p->H * p->dk * s.esz);
  if (dyqk) {
    dyqk[0] = dyq;
    dyqk[1] = dyk;
  }
  unsigned char* dyv = c.take((size_t)s.Ttot * p->H * p->dv * s.esz);
  unsigned char* head = c.take(2 * NCH * 3 * p->dk * sizeof(float));
  unsigned char* tail = c.take(2 * NCH * 3 * p->dk * sizeof(float));
  unsigned char* part = c.take(2 * NCH * p->dk * width * sizeof(float));
  unsigned char* tmp = c.take(NS * p->H * p->dk * width * sizeof(float));
  unsigned char* vpart = c.take(NCH * p->dv * width * sizeof(float));
  unsigned char* vtmp = c.take(NS * p->H * p->dv * width * sizeof(float));
  if (a) {
    a->dv = dyv;
    a->bhead = (float*)head;
    a->btail = (float*)tail;
    a->bpart = (float*)part;
    a->btmp = (float*)tmp;
  }
  if (cv) {
    cv->dy = dyv;
    cv->part = (float*)vpart;
    cv->tmp = (float*)vtmp;
  }
  return c.off;
}

void fill_common(const gdn_problem* p, const Shape& s, Args* a) {
  a->gated = 1;
  a->H = p->H;
  a->N = s.N;
  a->NC = (int)s.NC;
  a->T = p->cu_seqlens ? 0 : p->T;
  a->cu = p->cu_seqlens;
}

constexpr size_t NOALLOC_BYTES = GDN_NOALLOC_SCRATCH_BYTES;
constexpr int MAX_DEVICES = 64;
static_assert(NOALLOC_BYTES % ALIGN == 0, "scratch size must keep the carve-up aligned");

}  // namespace

// Workspace of gdn_chunk_fwd_noalloc: a file-scope device array, one copy on
// every GPU the library runs on, held until the process ends.  In host code
// `scratch` is only the registration handle of that array, not a device
// address: the device address of each GPU's copy is looked up once per
// device (hipGetSymbolAddress with that device current) and kept below.
static __device__ __align__(256) unsigned char scratch[GDN_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex scratch_mu;
void* scratch_ptr[MAX_DEVICES];  // device address of `scratch` per device, once looked up

// The current device's copy of the scratch array, or nullptr on failure.
void* scratch_for_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lk(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    scratch_ptr[dev] = ptr;
  }
  return scratch_ptr[dev];
}

}  // namespace

extern "C" {

size_t gdn_chunk_fwd_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  return carve(p, s, Use::Fwd, nullptr, nullptr);
}

size_t gdn_chunk_bwd_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  return carve(p, s, Use::Bwd, nullptr, nullptr);
}

gdn_status gdn_chunk_fwd_timed(const gdn_problem* p, const void* q, const void* k,
                               const void* v, const float* beta, const float* log_alpha,
                               const float* h0, void* o, float* ht, void* workspace,
                               size_t workspace_bytes, void* stream, gdn_timing* timing) {
  Shape s;
  gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !o) return GDN_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, log_alpha, h0, o, ht, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  const size_t need = carve(p, s, Use::Fwd, nullptr, nullptr);
  if (!workspace || workspace_bytes < need) return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  carve(p, s, Use::Fwd, (unsigned char*)workspace, &a);
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.gated = log_alpha != nullptr;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  TimingGuard tg(timing);
  const hipError_t e = gdn::launch_fwd(p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16, p->dk, p->dv, a,
                                       (hipStream_t)stream, tg.get());
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_chunk_fwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                         const float* beta, const float* log_alpha, const float* h0, void* o,
                         float* ht, void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_chunk_fwd_timed(p, q, k, v, beta, log_alpha, h0, o, ht, workspace, workspace_bytes,
                             stream, nullptr);
}

gdn_status gdn_chunk_fwd_noalloc(const gdn_problem* p, const void* q, const void* k,
                                 const void* v, const float* beta, const float* log_alpha,
                                 const float* h0, void* o, float* ht, void* stream) {
  Shape s;
  const gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !o) return GDN_ERR_NULL;
  // the size check runs before any HIP call
  if (carve(p, s, Use::Fwd, nullptr, nullptr) > NOALLOC_BYTES) return GDN_ERR_WORKSPACE;
  void* ws = scratch_for_current_device();
  if (!ws) return GDN_ERR_HIP;
  // every byte of the forward's workspace that a kernel reads is written by
  // an earlier kernel of the same call: nothing needs clearing
  return gdn_chunk_fwd_timed(p, q, k, v, beta, log_alpha, h0, o, ht, ws, NOALLOC_BYTES, stream,
                             nullptr);
}

gdn_status gdn_chunk_bwd_timed(const gdn_problem* p, const void* q, const void* k,
                               const void* v, const float* beta, const float* log_alpha,
                               const float* h0, const void* dO, const float* dht, void* dq,
                               void* dk, void* dv, float* dbeta, float* dlog_alpha, float* dh0,
                               void* workspace, size_t workspace_bytes, void* stream,
                               gdn_timing* timing) {
  Shape s;
  gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !dO || !dq || !dk || !dv || !dbeta) return GDN_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, log_alpha, h0, dO, dht, dq, dk, dv, dbeta, dlog_alpha,
                        dh0, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  const size_t need = carve(p, s, Use::Bwd, nullptr, nullptr);
  if (!workspace || workspace_bytes < need) return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  carve(p, s, Use::Bwd, (unsigned char*)workspace, &a);
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.gated = log_alpha != nullptr;
  a.h0 = h0;
  a.dO = dO;
  a.dht = dht;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.dbeta = dbeta;
  a.dlog_alpha = dlog_alpha;
  a.dh0 = dh0;
  TimingGuard tg(timing);
  const hipError_t e = gdn::launch_bwd(p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16, p->dk, p->dv, a,
                                       (hipStream_t)stream, tg.get());
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_chunk_bwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                         const float* beta, const float* log_alpha, const float* h0,
                         const void* dO, const float* dht, void* dq, void* dk, void* dv,
                         float* dbeta, float* dlog_alpha, float* dh0, void* workspace,
                         size_t workspace_bytes, void* stream) {
  return gdn_chunk_bwd_timed(p, q, k, v, beta, log_alpha, h0, dO, dht, dq, dk, dv, dbeta,
                             dlog_alpha, dh0, workspace, workspace_bytes, stream, nullptr);
}

size_t gdn_chunk_saved_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  return saved_bytes(p, s);
}

size_t gdn_chunk_fwd_save_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  return carve(p, s, Use::FwdSave, nullptr, nullptr);
}

size_t gdn_chunk_bwd_saved_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  return carve(p, s, Use::BwdSaved, nullptr, nullptr);
}

gdn_status gdn_chunk_fwd_save_timed(const gdn_problem* p, const void* q, const void* k,
                                    const void* v, const float* beta, const float* log_alpha,
                                    const float* h0, void* o, float* ht, void* saved,
                                    size_t saved_bytes_, void* workspace, size_t workspace_bytes,
                                    void* stream, gdn_timing* timing) {
  Shape s;
  gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !o) return GDN_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, log_alpha, h0, o, ht, saved, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  if (!saved || saved_bytes_ < saved_bytes(p, s)) return GDN_ERR_SAVED;
  if (!workspace || workspace_bytes < carve(p, s, Use::FwdSave, nullptr, nullptr))
    return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  carve(p, s, Use::FwdSave, (unsigned char*)workspace, &a);
  Carver c{(unsigned char*)saved};
  carve_saved(p, s, c, &a);
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.gated = log_alpha != nullptr;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  TimingGuard tg(timing);
  const hipError_t e = gdn::launch_fwd_save(p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16, p->dk,
                                            p->dv, a, (hipStream_t)stream, tg.get());
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_chunk_fwd_save(const gdn_problem* p, const void* q, const void* k, const void* v,
                              const float* beta, const float* log_alpha, const float* h0,
                              void* o, float* ht, void* saved, size_t saved_bytes_,
                              void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_chunk_fwd_save_timed(p, q, k, v, beta, log_alpha, h0, o, ht, saved, saved_bytes_,
                                  workspace, workspace_bytes, stream, nullptr);
}

gdn_status gdn_chunk_bwd_saved_timed(const gdn_problem* p, const void* q, const void* k,
                                     const void* v, const float* beta,
                                     const void* dO, const float* dht, const void* saved,
                                     size_t saved_bytes_, void* dq, void* dk, void* dv,
                                     float* dbeta, float* dlog_alpha, float* dh0,
                                     void* workspace, size_t workspace_bytes, void* stream,
                                     gdn_timing* timing) {
  Shape s;
  gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !dO || !dq || !dk || !dv || !dbeta) return GDN_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, dO, dht, saved, dq, dk, dv, dbeta, dlog_alpha, dh0, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  if (!saved || saved_bytes_ < saved_bytes(p, s)) return GDN_ERR_SAVED;
  if (!workspace || workspace_bytes < carve(p, s, Use::BwdSaved, nullptr, nullptr))
    return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  carve(p, s, Use::BwdSaved, (unsigned char*)workspace, &a);
  Carver c{(unsigned char*)const_cast<void*>(saved)};
  carve_saved(p, s, c, &a);
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.dO = dO;
  a.dht = dht;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.dbeta = dbeta;
  a.dlog_alpha = dlog_alpha;
  a.dh0 = dh0;
  TimingGuard tg(timing);
  const hipError_t e = gdn::launch_bwd_saved(p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16, p->dk,
                                             p->dv, a, (hipStream_t)stream, tg.get());
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_chunk_bwd_saved(const gdn_problem* p, const void* q, const void* k, const void* v,
                               const float* beta, const void* dO, const float* dht,
                               const void* saved, size_t saved_bytes_, void* dq, void* dk,
                               void* dv, float* dbeta, float* dlog_alpha, float* dh0,
                               void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_chunk_bwd_saved_timed(p, q, k, v, beta, dO, dht, saved, saved_bytes_, dq, dk, dv, dbeta,
                                   dlog_alpha, dh0, workspace, workspace_bytes, stream, nullptr);
}

gdn_status gdn_recurrent_fwd_timed(const gdn_problem* p, const void* q, const void* k,
                                   const void* v, const float* beta, const float* log_alpha,
                                   const float* h0, void* o, float* ht, void* stream,
                                   gdn_timing* timing) {
  Shape s;
  gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !o) return GDN_ERR_NULL;
  const void* ptrs[] = {q, k, v, beta, log_alpha, h0, o, ht};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  a.q = q;
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.gated = log_alpha != nullptr;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  TimingGuard tg(timing);
  const hipError_t e = gdn::launch_recurrent_fwd(p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16, p->dk,
                                                 p->dv, a, (hipStream_t)stream, tg.get());
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_recurrent_fwd(const gdn_problem* p, const void* q, const void* k, const void* v,
                             const float* beta, const float* log_alpha, const float* h0, void* o,
                             float* ht, void* stream) {
  return gdn_recurrent_fwd_timed(p, q, k, v, beta, log_alpha, h0, o, ht, stream, nullptr);
}

gdn_status gdn_block_fwd_timed(const gdn_problem* p, const gdn_block_prologue* pro,
                               const float* beta, const float* log_alpha, const float* h0,
                               void* o, float* ht, void* q, void* k, void* v, void* workspace,
                               size_t workspace_bytes, void* stream, gdn_timing* timing) {
  Shape s;
  gdn_status st = check_block(p, pro, &s);
  if (st != GDN_OK) return st;
  if (!beta || !o) return GDN_ERR_NULL;
  const void* ptrs[] = {beta, log_alpha, h0, o, ht, q, k, v, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  if (!workspace || workspace_bytes < carve(p, s, Use::Fwd, nullptr, nullptr))
    return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  carve(p, s, Use::Fwd, (unsigned char*)workspace, &a);
  fill_prologue(pro, &a);
  a.yq = q;
  a.yk = k;
  a.yv = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.gated = log_alpha != nullptr;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  TimingGuard tg(timing);
  const hipError_t e =
      gdn::launch_fwd(Dt::BF16, p->dk, p->dv, a, (hipStream_t)stream, tg.get(), true);
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_block_fwd(const gdn_problem* p, const gdn_block_prologue* pro, const float* beta,
                         const float* log_alpha, const float* h0, void* o, float* ht, void* q,
                         void* k, void* v, void* workspace, size_t workspace_bytes,
                         void* stream) {
  return gdn_block_fwd_timed(p, pro, beta, log_alpha, h0, o, ht, q, k, v, workspace,
                             workspace_bytes, stream, nullptr);
}

gdn_status gdn_block_fwd_save_timed(const gdn_problem* p, const gdn_block_prologue* pro,
                                    const float* beta, const float* log_alpha, const float* h0,
                                    void* o, float* ht, void* q, void* k, void* v, void* saved,
                                    size_t saved_bytes_, void* workspace,
                                    size_t workspace_bytes, void* stream, gdn_timing* timing) {
  Shape s;
  gdn_status st = check_block(p, pro, &s);
  if (st != GDN_OK) return st;
  if (!beta || !o || !q || !k || !v) return GDN_ERR_NULL;
  const void* ptrs[] = {beta, log_alpha, h0, o, ht, q, k, v, saved, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  if (!saved || saved_bytes_ < saved_bytes(p, s)) return GDN_ERR_SAVED;
  if (!workspace || workspace_bytes < carve(p, s, Use::FwdSave, nullptr, nullptr))
    return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  fill_common(p, s, &a);
  carve(p, s, Use::FwdSave, (unsigned char*)workspace, &a);
  Carver c{(unsigned char*)saved};
  carve_saved(p, s, c, &a);
  fill_prologue(pro, &a);
  a.yq = q;
  a.yk = k;
  a.yv = v;
  a.beta = beta;
  a.log_alpha = log_alpha;
  a.gated = log_alpha != nullptr;
  a.h0 = h0;
  a.o = o;
  a.ht = ht;
  TimingGuard tg(timing);
  const hipError_t e =
      gdn::launch_fwd_save(Dt::BF16, p->dk, p->dv, a, (hipStream_t)stream, tg.get(), true);
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_block_fwd_save(const gdn_problem* p, const gdn_block_prologue* pro,
                              const float* beta, const float* log_alpha, const float* h0,
                              void* o, float* ht, void* q, void* k, void* v, void* saved,
                              size_t saved_bytes_, void* workspace, size_t workspace_bytes,
                              void* stream) {
  return gdn_block_fwd_save_timed(p, pro, beta, log_alpha, h0, o, ht, q, k, v, saved,
                                  saved_bytes_, workspace, workspace_bytes, stream, nullptr);
}

size_t gdn_block_bwd_saved_workspace_size(const gdn_problem* p, int width) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK || width < 1 || width > 4) return 0;
  return carve_block_bwd(p, s, width, nullptr, nullptr, nullptr);
}

gdn_status gdn_block_bwd_saved_timed(const gdn_problem* p, const gdn_block_prologue* pro,
                                     const void* q, const void* k, const void* v,
                                     const float* beta, const void* dO,
                                     const float* dht, const void* saved, size_t saved_bytes_,
                                     void* dxq, void* dxk, void* dxv, float* dwq, float* dwk,
                                     float* dwv, float* dbeta, float* dlog_alpha, float* dh0,
                                     void* workspace, size_t workspace_bytes, void* stream,
                                     gdn_timing* timing) {
  Shape s;
  gdn_status st = check_block(p, pro, &s);
  if (st != GDN_OK) return st;
  if (!q || !k || !v || !beta || !dO || !dxq || !dxk || !dxv || !dwq || !dwk || !dwv || !dbeta)
    return GDN_ERR_NULL;
  const void* ptrs[] = {q,   k,   v,     beta,  dO,         dht, saved,    dxq,
                        dxk, dxv, dwq,   dwk,   dwv,        dbeta, dlog_alpha, dh0, workspace};
  for (const void* x : ptrs)
    if (x && !aligned16(x)) return GDN_ERR_ALIGN;
  if (!saved || saved_bytes_ < saved_bytes(p, s)) return GDN_ERR_SAVED;
  if (!workspace ||
      workspace_bytes < carve_block_bwd(p, s, pro->width, nullptr, nullptr, nullptr))
    return GDN_ERR_WORKSPACE;
  Args a;
  memset(&a, 0, sizeof a);
  gdn::ConvArgs cv;
  memset(&cv, 0, sizeof cv);
  fill_common(p, s, &a);
  unsigned char* dyqk[2];
  carve_block_bwd(p, s, pro->width, (unsigned char*)workspace, &a, &cv, dyqk);
  const bool composed = block_bwd_composed(p);
  Carver c{(unsigned char*)const_cast<void*>(saved)};
  carve_saved(p, s, c, &a);
  fill_prologue(pro, &a);
  a.q = q;  // the rule's q, k, v (the saving forward's outputs)
  a.k = k;
  a.v = v;
  a.beta = beta;
  a.dO = dO;
  a.dht = dht;
  a.dq = dxq;
  a.dk = dxk;
  a.dwq = dwq;
  a.dwk = dwk;
  a.dbeta = dbeta;
  a.dlog_alpha = dlog_alpha;
  a.dh0 = dh0;
  cv.H = p->H;
  cv.N = s.N;
  cv.NC = (int)s.NC;
  cv.T = a.T;
  cv.W = pro->width;
  cv.l2 = 0;
  cv.eps = pro->eps;
  cv.cu = p->cu_seqlens;
  cv.info = a.info;
  cv.x = pro->xv;
  cv.w = pro->wv;
  cv.dx = dxv;
  cv.dw = dwv;
  // the composed form: the rule's dq, dk into the workspace, then the
  // convolution backward of q and k (with L2) on them; the per-chunk weight
  // partials of q and k reuse the fused form's buffers
  gdn::ConvArgs cq = cv, ck = cv;
  if (composed) {
    a.dq = dyqk[0];
    a.dk = dyqk[1];
    const size_t per = (size_t)s.NC * p->H * p->dk * pro->width;
    cq.l2 = ck.l2 = 1;
    cq.x = pro->xq;
    cq.w = pro->wq;
    cq.dy = dyqk[0];
    cq.dx = dxq;
    cq.dw = dwq;
    cq.part = a.bpart;
    cq.tmp = a.btmp;
    ck.x = pro->xk;
    ck.w = pro->wk;
    ck.dy = dyqk[1];
    ck.dx = dxk;
    ck.dw = dwk;
    ck.part = a.bpart + per;
    ck.tmp = a.btmp;
  }
  TimingGuard tg(timing);
  const hipError_t e = gdn::launch_block_bwd_saved(p->dk, p->dv, a, cv,
                                                   composed ? &cq : nullptr,
                                                   composed ? &ck : nullptr,
                                                   (hipStream_t)stream, tg.get());
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_block_bwd_saved(const gdn_problem* p, const gdn_block_prologue* pro,
                               const void* q, const void* k, const void* v, const float* beta,
                               const void* dO, const float* dht, const void* saved,
                               size_t saved_bytes_, void* dxq, void* dxk, void* dxv, float* dwq,
                               float* dwk, float* dwv, float* dbeta, float* dlog_alpha,
                               float* dh0, void* workspace, size_t workspace_bytes,
                               void* stream) {
  return gdn_block_bwd_saved_timed(p, pro, q, k, v, beta, dO, dht, saved, saved_bytes_, dxq, dxk, dxv,
                                   dwq, dwk, dwv, dbeta, dlog_alpha, dh0, workspace,
                                   workspace_bytes, stream, nullptr);
}

size_t gdn_conv_silu_workspace_size(const gdn_problem* p, int dim, int width) {
  Shape s;
  if (check_conv(p, dim, width, 0.f, &s) != GDN_OK) return 0;
  return carve_conv(p, s, dim, width, nullptr, nullptr, nullptr);
}

static gdn_status conv_call(const gdn_problem* p, int dim, int width, int l2norm, float eps,
                            const void* x, const float* w, const void* dy, void* y, void* dx,
                            float* dw, void* workspace, size_t workspace_bytes, void* stream,
                            bool bwd) {
  Shape s;
  gdn_status st = check_conv(p, dim, width, eps, &s);
  if (st != GDN_OK) return st;
  if (!x || !w || (bwd ? (!dy || !dx || !dw) : !y)) return GDN_ERR_NULL;
  const void* ptrs[] = {x, w, dy, y, dx, dw, workspace};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GDN_ERR_ALIGN;
  if (!workspace || workspace_bytes < carve_conv(p, s, dim, width, nullptr, nullptr, nullptr))
    return GDN_ERR_WORKSPACE;
  Args t;
  memset(&t, 0, sizeof t);
  fill_common(p, s, &t);
  gdn::ConvArgs a;
  memset(&a, 0, sizeof a);
  carve_conv(p, s, dim, width, (unsigned char*)workspace, &t, &a);
  a.H = p->H;
  a.N = s.N;
  a.NC = (int)s.NC;
  a.T = t.T;
  a.W = width;
  a.l2 = l2norm ? 1 : 0;
  a.eps = eps;
  a.cu = p->cu_seqlens;
  a.x = x;
  a.w = w;
  a.dy = dy;
  a.y = y;
  a.dx = dx;
  a.dw = dw;
  const Dt dt = p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16;
  hipError_t e = gdn::launch_chunk_table(t, (hipStream_t)stream);
  if (e == hipSuccess)
    e = bwd ? gdn::launch_conv_bwd(dt, dim, a, (hipStream_t)stream)
            : gdn::launch_conv_fwd(dt, dim, a, (hipStream_t)stream);
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_conv_silu_fwd(const gdn_problem* p, int dim, int width, int l2norm, float eps,
                             const void* x, const float* w, void* y, void* workspace,
                             size_t workspace_bytes, void* stream) {
  return conv_call(p, dim, width, l2norm, eps, x, w, nullptr, y, nullptr, nullptr, workspace,
                   workspace_bytes, stream, false);
}

gdn_status gdn_conv_silu_bwd(const gdn_problem* p, int dim, int width, int l2norm, float eps,
                             const void* x, const float* w, const void* dy, void* dx, float* dw,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return conv_call(p, dim, width, l2norm, eps, x, w, dy, nullptr, dx, dw, workspace,
                   workspace_bytes, stream, true);
}

static long norm_rows(const gdn_problem* p, const Shape& s) { return s.Ttot * p->H; }
static int norm_blocks(long rows) { return (int)((rows + 63) / 64); }
// partial dw rows, then their slice sums (256 rows a slice)
static size_t norm_ws(const gdn_problem* p, int nblk) {
  return up((size_t)nblk * p->dv * sizeof(float)) +
         up((size_t)((nblk + 255) / 256) * p->dv * sizeof(float));
}

size_t gdn_norm_gate_workspace_size(const gdn_problem* p) {
  Shape s;
  if (check_problem(p, &s) != GDN_OK) return 0;
  return norm_ws(p, norm_blocks(norm_rows(p, s)));
}

static gdn_status norm_call(const gdn_problem* p, float eps, const void* o, const void* g,
                            const float* w, const void* dy, void* y, void* dout, void* dg,
                            float* dw, void* workspace, size_t workspace_bytes, void* stream,
                            bool bwd) {
  Shape s;
  gdn_status st = check_problem(p, &s);
  if (st != GDN_OK) return st;
  if (!(eps >= 0.f) || !isfinite(eps)) return GDN_ERR_VALUE;
  if (!o || !g || !w || (bwd ? (!dy || !dout || !dg || !dw) : !y)) return GDN_ERR_NULL;
  const void* ptrs[] = {o, g, w, dy, y, dout, dg, dw, workspace};
  for (const void* q : ptrs)
    if (q && !aligned16(q)) return GDN_ERR_ALIGN;
  gdn::NormArgs a;
  memset(&a, 0, sizeof a);
  a.rows = norm_rows(p, s);
  a.nblk = norm_blocks(a.rows);
  if (bwd && (!workspace || workspace_bytes < norm_ws(p, a.nblk))) return GDN_ERR_WORKSPACE;
  a.eps = eps;
  a.o = o;
  a.g = g;
  a.dy = dy;
  a.w = w;
  a.y = y;
  a.dout = dout;
  a.dg = dg;
  a.part = (float*)workspace;
  a.tmp = workspace ? (float*)((unsigned char*)workspace +
                               up((size_t)a.nblk * p->dv * sizeof(float)))
                    : nullptr;
  a.dw = dw;
  const Dt dt = p->dtype == GDN_F32 ? Dt::F32 : Dt::BF16;
  const hipError_t e = bwd ? gdn::launch_norm_gate_bwd(dt, p->dv, a, (hipStream_t)stream)
                           : gdn::launch_norm_gate_fwd(dt, p->dv, a, (hipStream_t)stream);
  return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

gdn_status gdn_norm_gate_fwd(const gdn_problem* p, float eps, const void* o, const void* g,
                             const float* w, void* y, void* stream) {
  return norm_call(p, eps, o, g, w, nullptr, y, nullptr, nullptr, nullptr, nullptr, 0, stream,
                   false);
}

gdn_status gdn_norm_gate_bwd(const gdn_problem* p, float eps, const void* o, const void* g,
                             const float* w, const void* dy, void* dout, void* dg, float* dw,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return norm_call(p, eps, o, g, w, dy, nullptr, dout, dg, dw, workspace, workspace_bytes, stream,
                   true);
}

const char* gdn_status_string(gdn_status s) {
  switch (s) {
    case GDN_OK: return "GDN_OK";
    case GDN_ERR_NULL: return "GDN_ERR_NULL: a required pointer is NULL";
    case GDN_ERR_SHAPE: return "GDN_ERR_SHAPE: invalid B, T or H";
    case GDN_ERR_UNSUPPORTED: return "GDN_ERR_UNSUPPORTED: (dtype, dk, dv) not supported";
    case GDN_ERR_CU_SEQLENS: return "GDN_ERR_CU_SEQLENS: malformed cu_seqlens";
    case GDN_ERR_WORKSPACE: return "GDN_ERR_WORKSPACE: workspace missing or too small";
    case GDN_ERR_HIP: return "GDN_ERR_HIP: a kernel launch failed";
    case GDN_ERR_ALIGN: return "GDN_ERR_ALIGN: pointer not 16-byte aligned";
    case GDN_ERR_SAVED: return "GDN_ERR_SAVED: saved buffer missing or too small";
    case GDN_ERR_VALUE: return "GDN_ERR_VALUE: a scalar argument is out of range";
  }
  return "GDN: unknown status";
}

int gdn_debug_block_bwd(int mode) {
  if (mode < 0 || mode > 2) return -1;
  return block_bwd_mode.exchange(mode);
}

int gdn_debug_audit(int sequence, uint64_t present) {
  if (sequence < 0 || sequence >= gdn::SEQ_COUNT) return -2;
  return gdn::audit((gdn::Seq)sequence, gdn::audit_probe(present));
}

const char* gdn_debug_audit_field(int index) {
  return index >= 0 && index < gdn::AUDIT_FIELDS ? gdn::audit_field_names[index] : nullptr;
}

}  // extern "C"

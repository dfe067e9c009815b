// Kernel argument block and launcher declarations shared by the HIP
// translation units of libgdn.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

// One packed description of a call.  Device pointers unless noted.
struct Args {
  int H;       // heads
  int N;       // sequences (dense: B)
  int NC;      // total chunks over all sequences
  int T;       // dense sequence length (used when cu == nullptr)
  const int32_t* cu;  // packed boundaries [N+1] or nullptr (dense)
  // inputs
  const void *q, *k, *v, *dO;
  const float *beta, *log_alpha, *h0, *dht;
  // outputs
  void *o, *dq, *dk, *dv;
  float *ht, *dbeta, *dlog_alpha, *dh0;
  // workspace
  int4* info;       // [NC] {sequence, first token row, length, 0}
  int* seq_chunk0;  // [N+1] first chunk of every sequence
  float* g;         // [NC][H][64]     cumulative log gate inside the chunk
  float* Tm;        // [NC][H][64][64] (I + A)^-1
  float* Pm;        // [NC][H][64][64] Gamma * Q K^T (lower, with diagonal)
  float* Ak;        // [NC][H][64][64] strictLower(Gamma * K K^T)
  void* Sc;         // [NC][H][dk][dv] chunk entry states          (backward)
  void* Vp;         // [NC][H][64][dv] V' = T X                    (backward)
  void* dSc;        // [NC][H][dk][dv] gradient of each exit state (backward)
  void* dXb;        // [NC][H][64][dv] dX = T^T dV'                (backward)
};

enum class Dt { F32, BF16 };

// Launch the forward / backward kernel sequence for one (dtype, dk, dv).
// Return the first launch error (hipSuccess if none).
hipError_t launch_fwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s);
hipError_t launch_bwd(Dt dt, int dk, int dv, const Args& a, hipStream_t s);

}  // namespace gdn

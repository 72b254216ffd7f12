// Internal interface between the C-ABI front end (qm_attn.cpp) and the gfx950
// kernels (attn_fwd_gfx950.hip).  Not installed; callers use include/qm_attn.h.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace qm {

// How the kernel conditions Q when it loads it into registers.  Both changes
// are exact in 16-bit arithmetic, so the kernel can always use a positive
// exponent-domain scale:
//   kQNormal  - use Q as stored (scale > 0);
//   kQNegate  - flip every sign bit (scale < 0: scale*q.k = |scale|*(-q).k);
//   kQZero    - replace Q by zeros (scale == 0 or too small to change any
//               score: every visible score is then exactly 0).
enum QMode : int { kQNormal = 0, kQNegate = 1, kQZero = 2 };

struct AttnArgs {
  const void* q;       // 16-bit or FP8 (one byte) elements
  const void* k;
  const void* v;
  uint16_t* o;
  float* lse;
  int B, H, N, d;  // d: head dimension of q and k (d_qk)
  int dv;         // head dimension of v and o: d, or 128 when d = 192
  int Hkv;      // key/value heads; H % Hkv == 0, query head h reads h / (H / Hkv)
  int causal;   // 0 or 1
  int dtype;    // 0 = fp16, 1 = bf16, 2 = FP8 E4M3 inputs with a bf16 output
  float c;      // |scale| * log2(e) (FP8: |scale * q_scale * k_scale| * log2(e)), normal, > 0
  float vscale; // factor applied to O: 1, or the FP8 value scale
  int qmode;    // QMode
  int layout;   // 0: [B][heads][N][width], 1: [B][N][heads][width] (q, k, v, o)
  int tile_rows;  // query rows per workgroup: 0 = chosen from the shape, 128 or 256
};

// Enqueues the kernel instance for (d, dv, dtype, causal, workgroup size).
// Arguments have been
// validated by the caller.  Returns the HIP launch status.
hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t stream);

}  // namespace qm

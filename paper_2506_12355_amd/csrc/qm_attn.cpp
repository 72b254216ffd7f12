// C-ABI front end of the attention library: argument validation, the choice of
// the Q conditioning mode for the scale, and dispatch to the gfx950 kernels.
// The operation and every argument are documented in include/qm_attn.h.

#include "qm_attn.h"

#include <atomic>
#include <float.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "attn_fwd_launch.h"

namespace {

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
  return a0 < b0 + nb && b0 < a0 + na;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// finite iff the exponent field is not all ones (independent of fast-math flags)
bool finite_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof(u));
  return (u & 0x7F800000u) != 0x7F800000u;
}

constexpr int kFp8 = 2;   // internal dtype code: FP8 E4M3 inputs, bf16 output

// query rows per workgroup: 0 = chosen per call from the shape (qm_attn_set_tile_rows)
std::atomic<int> g_tile_rows{0};

// Validation and dispatch shared by the entry points: H query heads read Hkv
// key/value heads (Hkv == H for plain multi-head attention); q and k have head
// dimension d, v and o head dimension dv.  dtype kFp8: q, k, v hold one-byte
// E4M3 codes scaled by qs, ks, vs, and o is bf16.
int attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H,
             int Hkv, int N, int d, int dv, float scale, int causal, hipStream_t stream,
             int dtype, float qs = 1.0f, float ks = 1.0f, float vs = 1.0f, int layout = QM_BHND) {
  if (!q || !k || !v || !o || !lse) return QM_ERR_NULL;
  if (B < 1 || H < 1 || N < 1 || Hkv < 1 || Hkv > H || H % Hkv != 0) return QM_ERR_SHAPE;
  if (!((d == 64 && dv == 64) || (d == 128 && dv == 128) || (d == 192 && dv == 128)))
    return QM_ERR_HEADDIM;
  if (dtype == kFp8 && !(d == 128 && dv == 128)) return QM_ERR_HEADDIM;
  // element counts: the whole tensor in 62 bits, one head's [N][d] slab and the
  // workgroup count in 31 bits (the kernels index within a head in 32 bits)
  const uint64_t bh = (uint64_t)B * (uint64_t)H;
  const uint64_t bhkv = (uint64_t)B * (uint64_t)Hkv;
  const uint64_t nd = (uint64_t)N * (uint64_t)d;     // d >= dv
  const uint64_t ndv = (uint64_t)N * (uint64_t)dv;
  // a head's byte offsets, including the padded last 256-row query block, fit
  // in 32 bits; the workgroup count fits an int
  if (((uint64_t)N + 256) * (uint64_t)d >= (1ull << 31) || bh >= (1ull << 62) / nd)
    return QM_ERR_SHAPE;
  if ((((uint64_t)N + 127) / 128) * bh > (uint64_t)INT_MAX) return QM_ERR_SHAPE;   // 128-row tiles
  if (dtype != QM_F16 && dtype != QM_BF16 && dtype != kFp8) return QM_ERR_DTYPE;
  if (!finite_bits(scale) || !finite_bits(qs) || !finite_bits(ks) || !finite_bits(vs))
    return QM_ERR_SCALE;
  if (causal != 0 && causal != 1) return QM_ERR_CAUSAL;
  // QM_BNHD: head dimensions 64 and 128 (the kernels for 192-wide keys read
  // contiguous heads only)
  if (layout != QM_BHND && !(layout == QM_BNHD && d == dv)) return QM_ERR_LAYOUT;
  if (layout == QM_BNHD) {
    // rows of one head are max(H, Hkv) rows apart: the kernels' 32-bit byte
    // offsets, including the padded last query block, must still fit
    const uint64_t heads = (uint64_t)(H > Hkv ? H : Hkv);
    const uint64_t row = heads * (uint64_t)d * (dtype == kFp8 ? 1u : 2u);
    if (((uint64_t)N + 256) * row >= (1ull << 32)) return QM_ERR_SHAPE;
  }

  const size_t es = dtype == kFp8 ? 1 : 2;   // bytes per q, k, v element
  const size_t q_bytes = (size_t)(bh * nd) * es;
  const size_t k_bytes = (size_t)(bhkv * nd) * es;
  const size_t v_bytes = (size_t)(bhkv * ndv) * es;
  const size_t o_bytes = (size_t)(bh * ndv) * 2;
  const size_t lse_bytes = (size_t)(bh * (uint64_t)N) * sizeof(float);
  if (overlaps(o, o_bytes, q, q_bytes) || overlaps(o, o_bytes, k, k_bytes) ||
      overlaps(o, o_bytes, v, v_bytes) || overlaps(lse, lse_bytes, q, q_bytes) ||
      overlaps(lse, lse_bytes, k, k_bytes) || overlaps(lse, lse_bytes, v, v_bytes) ||
      overlaps(lse, lse_bytes, o, o_bytes))
    return QM_ERR_ALIAS;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse))
    return QM_ERR_UNSUPPORTED;

  qm::AttnArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.B = B;
  a.H = H;
  a.Hkv = Hkv;
  a.N = N;
  a.d = d;
  a.dv = dv;
  a.causal = causal;
  a.dtype = dtype;
  a.vscale = vs;
  // exp2-domain scale of the stored codes' dot product (FP8: times the q and k
  // scales); the sign goes into Q (exact), a zero or negligible scale becomes
  // all-zero scores (exact: every visible score is 0)
  const double qk = (double)scale * (double)qs * (double)ks;
  const double c = fabs(qk) * 1.4426950408889634074;
  a.c = (float)c;
  if (!(a.c >= FLT_MIN) || !(c < (double)FLT_MAX)) {
    if (!(a.c >= FLT_MIN)) {
      a.c = 1.0f;
      a.qmode = qm::kQZero;
    } else {
      return QM_ERR_SCALE;   // the combined scale overflows fp32
    }
  } else {
    a.qmode = qk < 0.0 ? qm::kQNegate : qm::kQNormal;
  }
  a.layout = layout;
  a.tile_rows = g_tile_rows.load(std::memory_order_relaxed);
  return qm::launch_attn_fwd(a, stream) == hipSuccess ? QM_OK : QM_ERR_LAUNCH;
}

}  // namespace

extern "C" int qm_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                           int B, int H, int N, int d, float scale, int causal,
                           hipStream_t stream, int dtype) {
  return attn_fwd(q, k, v, o, lse, B, H, H, N, d, d, scale, causal, stream,
                  dtype == kFp8 ? -1 : dtype);   // FP8 has its own entry point
}

extern "C" int qm_attn_fwd_gqa(const void* q, const void* k, const void* v, void* o,
                               float* lse, int B, int H, int Hkv, int N, int d, float scale,
                               int causal, hipStream_t stream, int dtype) {
  return attn_fwd(q, k, v, o, lse, B, H, Hkv, N, d, d, scale, causal, stream,
                  dtype == kFp8 ? -1 : dtype);   // FP8 has its own entry point
}

extern "C" int qm_attn_fwd_fp8(const void* q, const void* k, const void* v, void* o,
                               float* lse, int B, int H, int N, int d, float q_scale,
                               float k_scale, float v_scale, float scale, int causal,
                               hipStream_t stream) {
  return attn_fwd(q, k, v, o, lse, B, H, H, N, d, d, scale, causal, stream, kFp8, q_scale,
                  k_scale, v_scale);
}

extern "C" int qm_attn_fwd_mla(const void* q, const void* k, const void* v, void* o,
                               float* lse, int B, int H, int N, int d_qk, int d_v, float scale,
                               int causal, hipStream_t stream, int dtype) {
  return attn_fwd(q, k, v, o, lse, B, H, H, N, d_qk, d_v, scale, causal, stream,
                  dtype == kFp8 ? -1 : dtype);   // FP8 has its own entry point
}

extern "C" int qm_attn_fwd_layout(const void* q, const void* k, const void* v, void* o,
                                  float* lse, int B, int H, int Hkv, int N, int d_qk, int d_v,
                                  float scale, int causal, hipStream_t stream, int dtype,
                                  int layout) {
  return attn_fwd(q, k, v, o, lse, B, H, Hkv, N, d_qk, d_v, scale, causal, stream,
                  dtype == kFp8 ? -1 : dtype, 1.0f, 1.0f, 1.0f, layout);
}

extern "C" int qm_attn_fwd_fp8_layout(const void* q, const void* k, const void* v, void* o,
                                      float* lse, int B, int H, int Hkv, int N, int d,
                                      float q_scale, float k_scale, float v_scale, float scale,
                                      int causal, hipStream_t stream, int layout) {
  return attn_fwd(q, k, v, o, lse, B, H, Hkv, N, d, d, scale, causal, stream, kFp8, q_scale,
                  k_scale, v_scale, layout);
}

extern "C" int qm_attn_set_tile_rows(int rows) {
  if (rows != 0 && rows != 128 && rows != 256) return QM_ERR_TILE;
  g_tile_rows.store(rows, std::memory_order_relaxed);
  return QM_OK;
}

extern "C" const char* qm_attn_strerror(int status) {
  switch (status) {
    case QM_OK: return "success";
    case QM_ERR_NULL: return "a tensor pointer is NULL";
    case QM_ERR_SHAPE:
      return "B, H or N is below 1, Hkv does not divide H, or the tensors are too large";
    case QM_ERR_HEADDIM:
      return "head dimensions must be 64 or 128 (or d_qk = 192 with d_v = 128; FP8: 128)";
    case QM_ERR_DTYPE: return "dtype must be QM_F16 (0) or QM_BF16 (1)";
    case QM_ERR_SCALE: return "scale (and the FP8 tensor scales) must be finite";
    case QM_ERR_ALIAS: return "o or lse overlaps an input or each other";
    case QM_ERR_CAUSAL: return "causal must be 0 or 1";
    case QM_ERR_LAUNCH: return "the HIP runtime rejected the kernel launch";
    case QM_ERR_UNSUPPORTED: return "tensor pointers must be 16-byte aligned";
    case QM_ERR_LAYOUT:
      return "layout must be QM_BHND (0), or QM_BNHD (1) with head dimension 64 or 128";
    case QM_ERR_TILE: return "tile rows must be 0 (chosen per call), 128 or 256";
  }
  return "unknown status";
}

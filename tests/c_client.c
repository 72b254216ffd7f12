/*
 * A plain C consumer of the attention library (include/qm_attn.h), used by the
 * GPU tests to show that the C ABI works without Python or torch: device
 * memory comes from hipMalloc, the stream from hipStreamCreate, and inputs and
 * outputs cross with hipMemcpy.  Built by tests/build_c_client.py into
 * libqm_c_client.so and loaded with ctypes.
 *
 * qmc_run copies q, k and v (host buffers of the given byte sizes) to fresh
 * device buffers, fills o and lse with 0xFF bytes (NaN in every output type),
 * calls one entry point on its own stream, synchronises, and copies o and lse
 * back.  `entry` selects the call: 0 qm_attn_fwd, 1 qm_attn_fwd_gqa,
 * 2 qm_attn_fwd_mla, 3 qm_attn_fwd_fp8, 4 qm_attn_fwd_layout,
 * 5 qm_attn_fwd_fp8_layout.  Returns the entry point's status, or
 * QMC_ERR_HIP (with the HIP error text in `msg`) when a HIP call fails.
 */
#include <stdio.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "qm_attn.h"

#define QMC_ERR_HIP (-100)

static int hip_failed(hipError_t e, const char* what, char* msg, int msglen) {
  if (e == hipSuccess) return 0;
  if (msg && msglen > 0) snprintf(msg, (size_t)msglen, "%s: %s", what, hipGetErrorString(e));
  return 1;
}

int qmc_run(int entry, const void* q, size_t q_bytes, const void* k, size_t k_bytes,
            const void* v, size_t v_bytes, void* o, size_t o_bytes, float* lse,
            size_t lse_bytes, int B, int H, int Hkv, int N, int d_qk, int d_v, float scale,
            int causal, int dtype, int layout, float q_scale, float k_scale, float v_scale,
            char* msg, int msglen) {
  void *dq = NULL, *dk = NULL, *dv = NULL, *dout = NULL, *dlse = NULL;
  hipStream_t stream = NULL;
  int status = QMC_ERR_HIP;
  if (msg && msglen > 0) msg[0] = '\0';

  /* every buffer must hold what the shape says the call reads or writes */
  if (B > 0 && H > 0 && Hkv > 0 && N > 0 && d_qk > 0 && d_v > 0) {
    const int fp8 = entry == 3 || entry == 5;
    const unsigned long long es = fp8 ? 1 : 2;
    const unsigned long long kvh = (entry == 1 || entry == 4 || entry == 5) ? Hkv : H;
    const unsigned long long dvv = (entry == 2 || entry == 4) ? d_v : d_qk;
    const unsigned long long bn = (unsigned long long)B * (unsigned long long)N;
    if (q_bytes < bn * H * d_qk * es || k_bytes < bn * kvh * d_qk * es ||
        v_bytes < bn * kvh * dvv * es || o_bytes < bn * H * dvv * 2 ||
        lse_bytes < bn * H * sizeof(float)) {
      if (msg && msglen > 0) snprintf(msg, (size_t)msglen, "a buffer is smaller than its shape");
      return QMC_ERR_HIP;
    }
  }

  if (hip_failed(hipMalloc(&dq, q_bytes), "hipMalloc q", msg, msglen) ||
      hip_failed(hipMalloc(&dk, k_bytes), "hipMalloc k", msg, msglen) ||
      hip_failed(hipMalloc(&dv, v_bytes), "hipMalloc v", msg, msglen) ||
      hip_failed(hipMalloc(&dout, o_bytes), "hipMalloc o", msg, msglen) ||
      hip_failed(hipMalloc(&dlse, lse_bytes), "hipMalloc lse", msg, msglen) ||
      hip_failed(hipStreamCreate(&stream), "hipStreamCreate", msg, msglen) ||
      hip_failed(hipMemcpy(dq, q, q_bytes, hipMemcpyHostToDevice), "copy q", msg, msglen) ||
      hip_failed(hipMemcpy(dk, k, k_bytes, hipMemcpyHostToDevice), "copy k", msg, msglen) ||
      hip_failed(hipMemcpy(dv, v, v_bytes, hipMemcpyHostToDevice), "copy v", msg, msglen) ||
      hip_failed(hipMemset(dout, 0xFF, o_bytes), "poison o", msg, msglen) ||
      hip_failed(hipMemset(dlse, 0xFF, lse_bytes), "poison lse", msg, msglen))
    goto done;

  switch (entry) {
    case 0:
      status = qm_attn_fwd(dq, dk, dv, dout, (float*)dlse, B, H, N, d_qk, scale, causal, stream,
                           dtype);
      break;
    case 1:
      status = qm_attn_fwd_gqa(dq, dk, dv, dout, (float*)dlse, B, H, Hkv, N, d_qk, scale,
                               causal, stream, dtype);
      break;
    case 2:
      status = qm_attn_fwd_mla(dq, dk, dv, dout, (float*)dlse, B, H, N, d_qk, d_v, scale,
                               causal, stream, dtype);
      break;
    case 3:
      status = qm_attn_fwd_fp8(dq, dk, dv, dout, (float*)dlse, B, H, N, d_qk, q_scale,
                               k_scale, v_scale, scale, causal, stream);
      break;
    case 4:
      status = qm_attn_fwd_layout(dq, dk, dv, dout, (float*)dlse, B, H, Hkv, N, d_qk, d_v,
                                  scale, causal, stream, dtype, layout);
      break;
    case 5:
      status = qm_attn_fwd_fp8_layout(dq, dk, dv, dout, (float*)dlse, B, H, Hkv, N, d_qk,
                                      q_scale, k_scale, v_scale, scale, causal, stream, layout);
      break;
    default:
      if (msg && msglen > 0) snprintf(msg, (size_t)msglen, "unknown entry %d", entry);
      status = QMC_ERR_HIP;
      goto done;
  }
  if (status != QM_OK) {
    if (msg && msglen > 0) snprintf(msg, (size_t)msglen, "%s", qm_attn_strerror(status));
    goto done;
  }
  if (hip_failed(hipStreamSynchronize(stream), "hipStreamSynchronize", msg, msglen) ||
      hip_failed(hipMemcpy(o, dout, o_bytes, hipMemcpyDeviceToHost), "copy o", msg, msglen) ||
      hip_failed(hipMemcpy(lse, dlse, lse_bytes, hipMemcpyDeviceToHost), "copy lse", msg,
                 msglen))
    status = QMC_ERR_HIP;

done:
  if (stream) hipStreamDestroy(stream);
  hipFree(dq);
  hipFree(dk);
  hipFree(dv);
  hipFree(dout);
  hipFree(dlse);
  return status;
}

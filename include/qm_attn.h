/*
 * qm_attn.h - fused scaled-dot-product attention forward for AMD MI355X (gfx950).
 *
 * The operation is the paper's statement of the attention problem (Background,
 * subsection "Attention Operators and acceleration"): for queries Q, keys K and
 * values V holding N tokens of head dimension d,
 *
 *     O = softmax(Mask(scale * Q K^T)) V,     lse_i = ln sum_{j visible} exp(scale * q_i . k_j)
 *
 * evaluated independently for every (batch, head), the way the paper's kernels
 * give each thread block a fixed batch and head of Q (Method, "Parameter
 * Analysis and Reasoning").  The N x N score matrix is never stored: scores are
 * formed block by block on chip with an online softmax that keeps a running row
 * maximum and row sum (the paper's Appendix B listings: "Softmax S with Smax and
 * Ssum" between the two fused GEMMs).
 *
 * Conventions shared by every entry point:
 *   - All tensor pointers are DEVICE pointers owned by the caller.  The library
 *     never allocates, frees, retains or synchronises them.
 *   - q and o are contiguous row-major [B][H][N][d] arrays, k and v
 *     [B][Hkv][N][d] (Hkv = H except in qm_attn_fwd_gqa and the _layout
 *     calls; in qm_attn_fwd_mla v and o have their own head dimension; the
 *     _layout calls also take [B][N][heads][d]), of the 16-bit type named by
 *     `dtype` (FP8 calls: one-byte E4M3 codes, bf16 o); otherwise o has the
 *     input type.  lse is a contiguous [B][H][N] float32 array.  Base
 *     pointers must be 16-byte aligned.
 *   - The call validates its arguments on the host, then enqueues one kernel on
 *     `stream` (NULL = the null stream) and returns; results are valid once the
 *     caller has synchronised that stream.  On any error nothing is enqueued and
 *     no output is written.
 *   - Calls are thread-safe; calls on different streams may run concurrently,
 *     and calls may be captured into a HIP graph (nothing but the one kernel
 *     launch is enqueued).
 *   - Input elements are expected to be finite.  An infinite or NaN element
 *     gives unspecified values in the outputs that read it: its own query row
 *     (an element of q), or every row of the query heads that use its
 *     key/value head (an element of k or v).  All other outputs are unaffected,
 *     and the addresses the kernel touches, its barriers and its loop trip
 *     counts never depend on element values.
 *   - Range: the kernel forms each dot product q_i . k_j in fp32 and works in
 *     base 2, multiplying it by |scale| * log2(e) in fp32; lse is fp32 too.
 *     Every q_i . k_j (of the stored codes, for the FP8 calls) and every
 *     |scale * q_i . k_j| * log2(e) (FP8: with scale * q_scale * k_scale)
 *     must therefore be finite in fp32, i.e. below 3.4e38.  A row with a
 *     larger one gets unspecified O and lse (in practice NaN or infinity);
 *     the other rows are unaffected.  The front end rejects a combined scale
 *     whose fp32 value overflows (QM_ERR_SCALE); it cannot see the inputs.
 */
#ifndef QM_ATTN_H
#define QM_ATTN_H

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* 16-bit storage types of q, k, v and o. */
typedef enum {
  QM_F16 = 0,  /* IEEE binary16 */
  QM_BF16 = 1  /* bfloat16 (top half of an IEEE binary32) */
} qm_dtype_t;

/* Memory layouts of q, k, v and o (the _layout entry points; lse is always [B][H][N]). */
typedef enum {
  QM_BHND = 0,  /* [B][heads][N][width]: each head a contiguous N x width slab */
  QM_BNHD = 1   /* [B][N][heads][width]: each token's heads side by side */
} qm_layout_t;

/* Status codes returned by every qm_attn_fwd* entry point. */
enum {
  QM_OK = 0,
  QM_ERR_NULL = -1,        /* q, k, v, o or lse is NULL */
  QM_ERR_SHAPE = -2,       /* B, H or N < 1, Hkv not a divisor of H, B*H*N*d
                              does not fit in 62 bits, or (N + 256) * d (QM_BNHD:
                              times the heads, in bytes) does not fit in 31 (32) bits */
  QM_ERR_HEADDIM = -3,     /* d is not 64 or 128 (qm_attn_fwd_mla: (d_qk, d_v) is not
                              (64, 64), (128, 128) or (192, 128)) */
  QM_ERR_DTYPE = -4,       /* dtype is not QM_F16 or QM_BF16 */
  QM_ERR_SCALE = -5,       /* scale (or an FP8 tensor scale) is infinite or NaN, or the
                              combined scale times log2(e) overflows fp32 */
  QM_ERR_ALIAS = -6,       /* o or lse overlaps q, k, v or each other */
  QM_ERR_CAUSAL = -7,      /* causal is neither 0 nor 1 */
  QM_ERR_LAUNCH = -8,      /* the HIP runtime rejected the kernel launch */
  QM_ERR_UNSUPPORTED = -9, /* a pointer is not 16-byte aligned */
  QM_ERR_LAYOUT = -10,     /* layout is not QM_BHND or QM_BNHD, or QM_BNHD with
                              d_qk = 192 */
  QM_ERR_TILE = -11        /* qm_attn_set_tile_rows: rows is not 0, 128 or 256 */
};

/*
 * qm_attn_fwd - attention forward for B batches x H heads of N tokens.
 *
 *   q, k, v  [in]  device, [B][H][N][d] of `dtype`.  May alias one another.
 *   o        [out] device, [B][H][N][d] of `dtype`: the attention output,
 *                  rounded to the storage type (round-to-nearest-even).
 *   lse      [out] device, [B][H][N] float32: natural-log log-sum-exp of the
 *                  visible scaled scores of each query row.
 *   B, H, N        batch, heads, tokens (any N >= 1; tails are masked on chip).
 *   d              head dimension: 64 or 128 (the paper's head dimensions,
 *                  Evaluation section, "Benchmark setting").
 *   scale          any finite float multiplying q_i . k_j (usually 1/sqrt(d)).
 *                  It is applied to the fp32 dot product, never to 16-bit Q.
 *   causal         0: every key is visible; 1: key j is visible to query i
 *                  iff j <= i (the paper's causal mask; fully masked key blocks
 *                  are skipped, not computed).
 *   stream         HIP stream to enqueue on (NULL = null stream).
 *   dtype          a qm_dtype_t.
 *
 * Arithmetic: 16-bit products with fp32 accumulation on the matrix cores; the
 * softmax in fp32; probabilities rounded to `dtype` before the second product.
 * Results are deterministic: the same inputs give byte-identical outputs.
 *
 * Returns QM_OK or one of the QM_ERR_* codes above; every check except
 * QM_ERR_LAUNCH happens before anything is enqueued.
 */
int qm_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
                int B, int H, int N, int d, float scale, int causal,
                hipStream_t stream, int dtype);

/*
 * qm_attn_fwd_gqa - attention forward where H query heads share Hkv key/value
 * heads: multi-query (Hkv = 1) and grouped-query attention, the variants the
 * paper names beside multi-head attention in its Background and evaluates in
 * its Evaluation section ("Attention variants"; the appendix table of LLM
 * configurations: 64 query / 8 key-value heads, 128 / 8).  Query head h of a
 * batch attends with key/value head h / (H / Hkv) of that batch: consecutive
 * query heads form a group.  Every query head is otherwise exactly the
 * qm_attn_fwd operation.
 *
 *   q, o     [B][H][N][d] of `dtype` (o [out]).
 *   k, v     [in] device, [B][Hkv][N][d] of `dtype`.
 *   lse      [out] device, [B][H][N] float32.
 *   Hkv      key/value heads: 1 <= Hkv <= H and H % Hkv == 0, else
 *            QM_ERR_SHAPE.  Hkv = H is exactly qm_attn_fwd.
 *   all other arguments, the arithmetic, determinism and the status codes are
 *   those of qm_attn_fwd.
 */
int qm_attn_fwd_gqa(const void* q, const void* k, const void* v, void* o, float* lse,
                    int B, int H, int Hkv, int N, int d, float scale, int causal,
                    hipStream_t stream, int dtype);

/*
 * qm_attn_fwd_mla - attention forward with a wider query/key head than value
 * head: the multi-head latent attention shape the paper evaluates (its MLA
 * table: DeepSeek-V3's configuration, head dimension 128 plus a 64-wide RoPE
 * part, so d_qk = 192 and d_v = 128, with the causal mask), taken in its
 * explicit form where every head has its own keys and values.
 *
 *   q, k     [in]  device, [B][H][N][d_qk] of `dtype`.
 *   v        [in]  device, [B][H][N][d_v] of `dtype`.
 *   o        [out] device, [B][H][N][d_v] of `dtype`.
 *   lse      [out] device, [B][H][N] float32.
 *   d_qk, d_v      (192, 128); (64, 64) and (128, 128) are qm_attn_fwd.
 *                  Any other pair: QM_ERR_HEADDIM.
 *   scale          multiplies q_i . k_j over all d_qk columns (usually
 *                  1/sqrt(d_qk)).
 *   all other arguments, the arithmetic, determinism and the status codes are
 *   those of qm_attn_fwd.
 */
int qm_attn_fwd_mla(const void* q, const void* k, const void* v, void* o, float* lse,
                    int B, int H, int N, int d_qk, int d_v, float scale, int causal,
                    hipStream_t stream, int dtype);

/*
 * qm_attn_fwd_fp8 - attention forward on FP8 inputs, the variant the paper's
 * case study generates (its FP8 table: MHA with the causal mask at head
 * dimension 128).  q, k and v hold OCP E4M3 codes (1 sign, 4 exponent bits
 * with bias 7, 3 mantissa bits; the largest value 448), each with one scale
 * factor for the whole tensor: the operation is qm_attn_fwd's on the real
 * tensors q_scale*Q, k_scale*K and v_scale*V.  The products run on the FP8
 * matrix cores with fp32 accumulation; the probabilities are rounded to E4M3
 * (to nearest even) before the second product; per output row i that bounds
 * the error by 2^-4 sum_j P_ij |v_j| + 2^-10 exp(m_i - lse_i) sum_j |v_j| (P the
 * exact probabilities, m_i the row's largest score, v the real values), and the
 * row sums and lse stay in fp32.  The matrix cores sum each group of 8
 * products after truncating them to multiples of 2^-13 of the group's
 * largest, which adds at most 7 * 2^-13 of sum_j P_ij |v_j| to O and of
 * |scale| sum_c |q_ic k_jc| to each score.
 *
 *   q, k, v  [in]  device, [B][H][N][d] uint8 E4M3 codes.
 *   o        [out] device, [B][H][N][d] bfloat16 (round to nearest even).
 *   lse      [out] device, [B][H][N] float32, of the scaled scores.
 *   d              128; any other value: QM_ERR_HEADDIM.
 *   q_scale, k_scale, v_scale   finite per-tensor factors (QM_ERR_SCALE otherwise).
 *   scale          finite, multiplies the dot product of the real tensors.
 *   B, H, N, causal, stream: as for qm_attn_fwd; there is no dtype argument.
 */
int qm_attn_fwd_fp8(const void* q, const void* k, const void* v, void* o, float* lse,
                    int B, int H, int N, int d, float q_scale, float k_scale, float v_scale,
                    float scale, int causal, hipStream_t stream);

/*
 * qm_attn_fwd_layout - the 16-bit entry points in one call, with the memory
 * layout as an argument.  Computes exactly what qm_attn_fwd_gqa (Hkv < H) and
 * qm_attn_fwd_mla (d_qk = 192, d_v = 128) compute, on tensors stored as
 * `layout`:
 *
 *   QM_BHND  q [B][H][N][d_qk], k [B][Hkv][N][d_qk], v [B][Hkv][N][d_v],
 *            o [B][H][N][d_v] (the other entry points' layout);
 *   QM_BNHD  q [B][N][H][d_qk], k [B][N][Hkv][d_qk], v [B][N][Hkv][d_v],
 *            o [B][N][H][d_v]: the layout a projection writes before any
 *            transpose.
 *
 *   lse      [out] device, [B][H][N] float32 in either layout.
 *   (d_qk, d_v)    (64, 64), (128, 128) or (192, 128); QM_ERR_HEADDIM otherwise.
 *   layout         a qm_layout_t; QM_BNHD takes (d_qk, d_v) = (64, 64) or
 *                  (128, 128).  QM_ERR_LAYOUT otherwise.
 *   all other arguments, the arithmetic, determinism and the status codes are
 *   those of qm_attn_fwd.  Both layouts give byte-identical results.
 */
int qm_attn_fwd_layout(const void* q, const void* k, const void* v, void* o, float* lse,
                       int B, int H, int Hkv, int N, int d_qk, int d_v, float scale,
                       int causal, hipStream_t stream, int dtype, int layout);

/*
 * qm_attn_fwd_fp8_layout - qm_attn_fwd_fp8 with grouped-query key/value heads
 * and the memory layout as arguments: k and v hold Hkv heads (H % Hkv == 0;
 * query head h reads key/value head h / (H / Hkv), as in qm_attn_fwd_gqa),
 * and q, k, v and o are stored as `layout` (QM_BHND or QM_BNHD, as in
 * qm_attn_fwd_layout).  The arithmetic, its error bound and the status codes
 * are those of qm_attn_fwd_fp8, plus QM_ERR_SHAPE for an Hkv that is below 1,
 * above H or not a divisor of H, and QM_ERR_LAYOUT for any other layout.
 * Hkv = H with QM_BHND is exactly qm_attn_fwd_fp8; both layouts give
 * byte-identical results.
 */
int qm_attn_fwd_fp8_layout(const void* q, const void* k, const void* v, void* o, float* lse,
                           int B, int H, int Hkv, int N, int d, float q_scale, float k_scale,
                           float v_scale, float scale, int causal, hipStream_t stream,
                           int layout);

/*
 * qm_attn_set_tile_rows - a tuning control: the query rows one workgroup
 * owns, for every later call in the process.
 *
 *   rows = 0 (the default): chosen per call from the shape.  256-row
 *            workgroups (eight wavefronts, one per CU) keep each K/V block in
 *            LDS for the most rows; 128-row workgroups (four wavefronts, two
 *            per CU) overlap one workgroup's start and end with the other's
 *            work, and run when N <= 2048 (FP8: N <= 4096, where its
 *            four-wavefront workgroups keep four-block K/V rings) or when
 *            the 256-row workgroups,
 *            dealt out in rounds over the device's CUs, would keep them less
 *            than 80% busy (fewer workgroups than CUs, or 1.5 rounds' worth).
 *   rows = 128 or 256: that size wherever it exists ([B][H][N][d] tensors with
 *            head dimension 64 or 128; everything else runs 256).
 *
 * Results do not depend on it: every query row takes the same arithmetic in
 * the same order, so outputs are byte-identical either way; only speed
 * changes.  Returns QM_OK, or QM_ERR_TILE for any other value (the setting is
 * then unchanged).  Thread-safe; a call racing with attention calls on other
 * threads may or may not apply to them.
 */
int qm_attn_set_tile_rows(int rows);

/* qm_attn_strerror - a static, human-readable string for a status code. */
const char* qm_attn_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* QM_ATTN_H */

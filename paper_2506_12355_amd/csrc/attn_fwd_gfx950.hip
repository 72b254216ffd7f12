// Fused attention forward for gfx950 (MI355X): S = scale * Q K^T, online
// softmax with a running row maximum and row sum, O = P V; the N x N score
// matrix never leaves the chip.
//
// Work decomposition (the paper's Method section gives each thread block a
// fixed batch and head of Q, a (BM, HeadDim) tile at coordinate L = block
// index): one workgroup owns BM = 128 query rows of one (batch, head); its four
// wavefronts own 32 rows each and walk the key/value sequence in blocks of
// BN = 64 keys (the loop of the paper's Appendix B listings).
//
// The two products are arranged for the 32x32x16 MFMA of CDNA4:
//
//   GEMM-I   S^T[key][query] = K[key][:] . Q[query][:]
//            A operand = K rows read from LDS (K keeps its stored layout, the
//            point of the paper's "GEMM error" case), B operand = Q, loaded
//            once from HBM and resident in VGPRs.  The accumulator gives each
//            lane one query column, so the row max / row sum of a query are an
//            in-register reduction plus one exchange between the two lane
//            halves that share the column.
//
//   GEMM-II  O^T[d][query] += V^T[d][key] . P^T[key][query]
//            B operand = P^T, taken straight from the GEMM-I accumulator
//            registers after an fp32 -> 16-bit pack.  This is the paper's
//            "Reshape S from MMA_C to MMA_A" step, done without moving data:
//            the accumulator holds, per lane half, keys {0-3, 8-11, ...} or
//            {4-7, 12-15, ...}; V^T is stored in LDS with bits 2 and 3 of the
//            key index swapped, so one 128-bit LDS read returns exactly the
//            keys whose probabilities the lane holds.  The contraction order
//            over keys is free, so nothing else changes.
//
// K/V staging: the next key block is fetched from HBM into registers with
// 128-bit loads while the current block is consumed from LDS, then written to
// the other LDS buffer (two buffers, one barrier per block).  V is transposed
// on the way in (4 keys x 8 dims per thread, 64-bit LDS writes).
//
// Online softmax (exp2 domain, c = |scale| * log2 e):
//   m_blk = c * max_j s_j;   p_j = 2^(c*s_j - m);   l += sum_j p_j
//   The running maximum m is only raised when a block's maximum exceeds it by
//   more than TAU = 8 (then O and l are rescaled by 2^(m_old - m_new)).  The
//   result is exact for any m not below the true maximum minus TAU: every p_j
//   stays <= 2^8, and O = sum p v / sum p, lse = (m + log2 l) * ln 2 use the
//   same m.  Rescaling becomes rare after the first blocks.
//
// Causal masking: key blocks entirely above the diagonal of the workgroup are
// never loaded; a wavefront skips the blocks entirely above its own rows;
// elementwise masking runs only on blocks that straddle the diagonal or the
// sequence tail.  Heavy (late) query blocks are dispatched first.
//
// Dispatch order: workgroup i runs on XCD i % 8.  The linear id is remapped so
// that consecutive query blocks of the same head land on the same XCD and
// share its L2 for the K/V stream.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "attn_fwd_launch.h"

namespace qm {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kBM = 128;      // query rows per workgroup
constexpr int kBN = 64;       // keys per block
constexpr int kWaves = 4;     // 32 query rows per wavefront
constexpr int kThreads = 64 * kWaves;
constexpr float kTau = 8.0f;  // lazy-rescale threshold (log2 units)
constexpr int kXcds = 8;

struct KParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  int N;
  int nq;      // query blocks per head
  int total;   // nq * B * H workgroups
  float c;     // |scale| * log2 e
  int qmode;
};

// 16-bit type traits: the MFMA and the fp32 -> 16-bit pack (round to nearest even).
template <int DT>
struct Half;

template <>
struct Half<0> {  // fp16
  static __device__ __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack(float x, float y) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x, y}, f16x2));
  }
};

template <>
struct Half<1> {  // bf16
  static __device__ __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
  static __device__ __forceinline__ uint32_t pack(float x, float y) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x, y}, bf16x2));
  }
};

// Position of key k inside a V^T row of LDS: bits 2 and 3 swapped (an involution).
__device__ __forceinline__ int vt_pos(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

template <int D, int DT, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(KParams p) {
  constexpr int KSTR = D + 8;         // LDS row stride of K (halfs): 4 banks of skew per row
  constexpr int VSTR = kBN + 8;       // LDS row stride of V^T (halfs)
  constexpr int KTILE = kBN * KSTR;
  constexpr int VTILE = D * VSTR;
  constexpr int BUF = KTILE + VTILE;
  constexpr int DCH = D / 8;                      // 16-byte chunks per row
  constexpr int KCH = kBN * DCH / kThreads;       // K chunks per thread per block
  constexpr int VTASKS = (kBN / 4) * DCH;         // (4 keys x 8 dims) V tasks per block
  constexpr int NKS = D / 16;                     // GEMM-I k-steps
  constexpr int NMT = D / 32;                     // GEMM-II M tiles
  static_assert(KCH * kThreads == kBN * DCH, "K staging must tile the block");
  static_assert(VTASKS <= kThreads, "one V task per thread at most");

  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int l32 = lane & 31;
  const int hi = lane >> 5;
  const int N = p.N;

  // ---- which (batch*head, query block) this workgroup owns ----
  int id = blockIdx.x;
  const int per_xcd = p.total / kXcds;
  if (id < per_xcd * kXcds) id = (id % kXcds) * per_xcd + id / kXcds;
  const int bh = id / p.nq;
  int qb = id - bh * p.nq;
  if (CAUSAL) qb = p.nq - 1 - qb;  // longest rows first

  const size_t head = (size_t)bh * (size_t)N * D;
  const uint16_t* __restrict__ Qh = p.q + head;
  const uint16_t* __restrict__ Kh = p.k + head;
  const uint16_t* __restrict__ Vh = p.v + head;

  const int q0 = qb * kBM;
  const int qw = q0 + wave * 32;   // first query row of this wavefront
  const int qrow = qw + l32;       // the query row whose column this lane holds

  // ---- Q: B operand of GEMM-I, resident for the whole key loop ----
  u32x4 qf[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) {
    qf[ks] = (qrow < N) ? ld16(Qh + (size_t)qrow * D + 16 * ks + 8 * hi) : u32x4{0, 0, 0, 0};
    if (p.qmode == kQNegate) qf[ks] ^= 0x80008000u;
    if (p.qmode == kQZero) qf[ks] = u32x4{0, 0, 0, 0};
  }

  const int kv_end = CAUSAL ? min(N, q0 + kBM) : N;
  const int nkv = (kv_end + kBN - 1) / kBN;

  f32x16 oacc[NMT];
#pragma unroll
  for (int mt = 0; mt < NMT; ++mt) oacc[mt] = f32x16{};
  float m_run = -INFINITY;   // running maximum, exp2 domain
  float l_run = 0.f;         // this lane's share of the running row sum

  // ---- HBM -> register staging of one key block ----
  u32x4 kst[KCH];
  u32x4 vst[4];
  const int vkg = tid / DCH;   // V task: keys 4*vkg .. 4*vkg+3
  const int vdc = tid % DCH;   //         dims 8*vdc .. 8*vdc+7
  const bool vtask = (VTASKS == kThreads) || (tid < VTASKS);

  auto gload = [&](int j0) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + kThreads * i;
      const int row = j0 + c / DCH;
      kst[i] = (row < N) ? ld16(Kh + (size_t)row * D + 8 * (c % DCH)) : u32x4{0, 0, 0, 0};
    }
    if (vtask) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = j0 + 4 * vkg + i;
        vst[i] = (row < N) ? ld16(Vh + (size_t)row * D + 8 * vdc) : u32x4{0, 0, 0, 0};
      }
    }
  };

  auto swrite = [&](int buf) {
    uint16_t* Ks = smem + buf * BUF;
    uint16_t* Vs = Ks + KTILE;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + kThreads * i;
      *reinterpret_cast<u32x4*>(Ks + (c / DCH) * KSTR + 8 * (c % DCH)) = kst[i];
    }
    if (vtask) {
      const int pos = vt_pos(4 * vkg);
#pragma unroll
      for (int w = 0; w < 4; ++w) {   // dims 8*vdc + 2w (low halves) and + 2w + 1 (high halves)
        const uint32_t a0 = vst[0][w], a1 = vst[1][w], a2 = vst[2][w], a3 = vst[3][w];
        const u32x2 ev = {(a0 & 0xFFFFu) | (a1 << 16), (a2 & 0xFFFFu) | (a3 << 16)};
        const u32x2 od = {(a0 >> 16) | (a1 & 0xFFFF0000u), (a2 >> 16) | (a3 & 0xFFFF0000u)};
        *reinterpret_cast<u32x2*>(Vs + (8 * vdc + 2 * w) * VSTR + pos) = ev;
        *reinterpret_cast<u32x2*>(Vs + (8 * vdc + 2 * w + 1) * VSTR + pos) = od;
      }
    }
  };

  gload(0);
  swrite(0);
  __syncthreads();

  for (int j = 0; j < nkv; ++j) {
    const int j0 = j * kBN;
    if (j + 1 < nkv) gload(j0 + kBN);

    const uint16_t* Ks = smem + (j & 1) * BUF;
    const uint16_t* Vs = Ks + KTILE;
    const bool active = (qw < N) && (!CAUSAL || j0 <= qw + 31);
    if (active) {
      // GEMM-I: two 32-key tiles of S^T
      f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(Ks + (32 * kt + l32) * KSTR + 16 * ks + 8 * hi);
          s[kt] = Half<DT>::mfma(a, qf[ks], s[kt]);
        }
      }

      // mask: keys past the end of the sequence, keys after the query (causal)
      const bool need_mask = (j0 + kBN > N) || (CAUSAL && j0 + kBN - 1 > qw);
      if (need_mask) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = j0 + 32 * kt + 8 * (r / 4) + 4 * hi + (r % 4);
            if (key >= N || (CAUSAL && key > qrow)) s[kt][r] = -INFINITY;
          }
        }
      }

      // block row maximum: 32 values in-lane, then the other lane half
      float mx = s[0][0];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_blk = mx * p.c;

      const bool need = m_blk > m_run + kTau;
      if (__any(need)) {
        const float m_new = need ? m_blk : m_run;
        const float alpha = need ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) oacc[mt] *= alpha;
        l_run *= alpha;
        m_run = m_new;
      }
      const float mu = (m_run == -INFINITY) ? 0.f : m_run;

      // probabilities, row-sum share, and the 16-bit P^T operands
      float lsum = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          s[kt][r] = __builtin_amdgcn_exp2f(fmaf(s[kt][r], p.c, -mu));
          lsum += s[kt][r];
        }
      }
      l_run += lsum;

      u32x4 pb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          pb[u][w] = Half<DT>::pack(s[u / 2][8 * (u % 2) + 2 * w], s[u / 2][8 * (u % 2) + 2 * w + 1]);
        }
      }

      // GEMM-II: O^T += V^T P^T
#pragma unroll
      for (int mt = 0; mt < NMT; ++mt) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(Vs + (32 * mt + l32) * VSTR + 16 * u + 8 * hi);
          oacc[mt] = Half<DT>::mfma(a, pb[u], oacc[mt]);
        }
      }
    }

    if (j + 1 < nkv) swrite((j + 1) & 1);
    __syncthreads();
  }

  // ---- epilogue: O = O / l in the storage type, lse in natural log ----
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (qrow < N) {
    const float inv = 1.0f / l_tot;
    uint16_t* Orow = p.o + head + (size_t)qrow * D;
#pragma unroll
    for (int mt = 0; mt < NMT; ++mt) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2 w = {Half<DT>::pack(oacc[mt][4 * g] * inv, oacc[mt][4 * g + 1] * inv),
                         Half<DT>::pack(oacc[mt][4 * g + 2] * inv, oacc[mt][4 * g + 3] * inv)};
        *reinterpret_cast<u32x2*>(Orow + 32 * mt + 8 * g + 4 * hi) = w;
      }
    }
    if (hi == 0) p.lse[(size_t)bh * N + qrow] = (m_run + log2f(l_tot)) * 0.69314718055994531f;
  }
}

template <int D>
constexpr size_t lds_bytes() {
  return 2 * (size_t)(kBN * (D + 8) + D * (kBN + 8)) * sizeof(uint16_t);
}

template <int D, int DT, bool CAUSAL>
hipError_t launch_instance(const KParams& kp, hipStream_t stream) {
  auto kern = attn_fwd_kernel<D, DT, CAUSAL>;
  constexpr size_t lds = lds_bytes<D>();
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kern, dim3(kp.total), dim3(kThreads), lds, stream, kp);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t stream) {
  KParams kp;
  kp.q = a.q;
  kp.k = a.k;
  kp.v = a.v;
  kp.o = a.o;
  kp.lse = a.lse;
  kp.N = a.N;
  kp.nq = (a.N + kBM - 1) / kBM;
  kp.total = kp.nq * a.B * a.H;
  kp.c = a.c;
  kp.qmode = a.qmode;
  const int key = (a.d == 128 ? 4 : 0) | (a.dtype << 1) | a.causal;
  switch (key) {
    case 0: return launch_instance<64, 0, false>(kp, stream);
    case 1: return launch_instance<64, 0, true>(kp, stream);
    case 2: return launch_instance<64, 1, false>(kp, stream);
    case 3: return launch_instance<64, 1, true>(kp, stream);
    case 4: return launch_instance<128, 0, false>(kp, stream);
    case 5: return launch_instance<128, 0, true>(kp, stream);
    case 6: return launch_instance<128, 1, false>(kp, stream);
    case 7: return launch_instance<128, 1, true>(kp, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace qm

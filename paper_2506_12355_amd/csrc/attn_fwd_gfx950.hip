// Fused attention forward for gfx950 (MI355X): S = scale * Q K^T, online
// softmax with a running row maximum and row sum, O = P V; the N x N score
// matrix never leaves the chip.
//
// Work decomposition (the paper's Method section gives each thread block a
// fixed batch and head of Q, a (BM, HeadDim) tile at coordinate L = block
// index): a tile is BM = 256 query rows of one (batch, head); the eight
// wavefronts of the workgroup that owns it (two per SIMD) own 32 rows each and
// walk the key/value
// sequence in blocks of BN = 64 keys (the loop of the paper's Appendix B
// listings).  A K/V block staged in LDS serves all 256 rows.  For short
// sequences the same kernel runs with four wavefronts (BM = 128) and several
// workgroups per CU (see ring_depth, wgs_per_cu and launch_attn_fwd).
//
// The two products use the 32x32x16 MFMA of CDNA4 (FP8 inputs: the 32x32x64
// one, with ds_read_b64_tr_b8 for V^T and E4M3 packs for P^T; see Fp8 below):
//
//   GEMM-I   S^T[key][query] = K[key][:] . Q[query][:]
//            A operand = K rows read from LDS (K keeps its stored layout, the
//            point of the paper's "GEMM error" case), B operand = Q, loaded
//            once and resident in VGPRs.  The accumulator gives each lane one
//            query column, so a query's row statistics are in-register
//            reductions plus one swap between the two lane halves sharing the
//            column (v_permlane32_swap).
//
//   GEMM-II  O^T[d][query] += V^T[d][key] . P^T[key][query]
//            B operand = P^T, taken straight from the GEMM-I accumulator after
//            an fp32 -> 16-bit pack.  This is the paper's "Reshape S from
//            MMA_C to MMA_A" step, done without moving data: per lane half the
//            accumulator holds keys {0-3, 8-11, ...} or {4-7, 12-15, ...}, and
//            the A operand V^T is gathered from row-major V in LDS with the
//            transposing read ds_read_b64_tr_b16 (within each 16-lane group,
//            output lane i, slot r takes element i%4 of source lane 4r + i/4),
//            pointing its four lane quads at exactly those four key rows.  The
//            contraction order over keys is free, so nothing else changes.
//
// Pipeline: K and V blocks go HBM -> LDS with direct buffer loads
// (buffer_load_dwordx4 ... lds; rows past the end of the sequence read as
// zeros) into four-block rings (two-block rings for 192-wide keys), K further
// ahead than V, each wave's loads spread over its MFMA slots.  While the
// exponentials of block j are formed, the MFMAs of GEMM-I for block j+1 run
// beside them (16 interleaved slots, the exponentials software-pipelined three
// deep, the wave at raised issue priority); then GEMM-II of block j, or, for
// FP8 and d = 64, GEMM-II of block j-1 in the same interleaved region (see
// DEFER below).  One barrier per two blocks (per block with two-block rings).
//
// Online softmax (exp2 domain, c = |scale| * log2 e): probabilities
// p = 2^(c s - m) are formed against the running maximum m without first
// reducing the block's own maximum.  A lane whose 32 probabilities sum to at
// most 2^8 has every p <= 2^8; only when some lane exceeds that (the running
// maximum must rise; always on the first block), or, for 16-bit inputs, when
// the block outweighs four times the row's sum so far (its new keys dominate
// the row, and their largest weight must be exactly 1 before it is rounded to
// 16 bits), is the block's exact maximum taken, O and l rescaled by
// 2^(m_old - m_new) and the probabilities redone.
// O = sum p v / sum p and lse = (m + log2 l) ln 2 use the same m, so the
// result is exact in either case.
//
// Causal masking: key blocks entirely above the diagonal of the workgroup are
// never loaded; a wavefront skips the blocks entirely above its own rows;
// elementwise masking runs only on blocks that straddle the diagonal or the
// sequence tail.  A workgroup runs a long and a short query block, the long
// one first, so that all workgroups cost the same.
//
// Dispatch order: workgroup i runs on XCD i % 8.  The linear tile id is
// remapped so that consecutive query blocks of the same head (and the heads
// sharing one key/value head) land on the same XCD and share its L2 for the
// K/V stream.  With 16-bit inputs the workgroups are persistent: as many as
// the CUs hold at once (a multiple of 8), workgroup w taking tiles w,
// w + grid, ..., which keeps tile t on XCD t % 8 and the same tiles side by
// side as one workgroup per tile would.
//
// Shapes: head dimension 64 or 128 (q, k, v alike), or 192-wide queries and
// keys with 128-wide values (the MLA shape); H query heads may share Hkv
// key/value heads (grouped-query and multi-query attention).

#include <hip/hip_runtime.h>
#include <float.h>
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <type_traits>

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
typedef int32_t i32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i32x2 lds_i32x2;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

constexpr int kBN = 64;       // keys per block
// A workgroup has WAVES wavefronts (a template parameter, 8 or 4) of 32 query
// rows each: BM = 32 WAVES query rows.
// Largest probability allowed against a stale running maximum, 2^8: sums of
// 64K such values stay far from fp32 overflow, and P fits fp16 and E4M3 (448).
constexpr float kPmax = 256.0f;
// 16-bit inputs also take the exact path when a block's probabilities outweigh
// kDominant times everything the row has summed before (its new keys carry
// more than 80% of the row's weight): the new maximum is then taken exactly,
// so the row's dominant weight is 2^0 = 1 exactly instead of a value up to 2^8
// that rounding to bf16 for the second product can move by 2^-8 of itself
// (an error O carries in full when that key dominates).  Rare for diffuse
// rows; on near-one-hot rows it keeps O within 1e-2 plus half a bf16 ulp.
constexpr float kDominant = 4.0f;
constexpr int kXcds = 8;
constexpr int kRsrcWord3 = 0x00020000;  // raw buffer, 32-bit data
// s_waitcnt immediate for vmcnt(0) and lgkmcnt(0): the direct LDS loads of
// this wave have landed
constexpr int kWaitLoads = 0x0070;
// Checking build (compiled with -DQM_DEBUG_SYNC): every key block ends with a
// barrier (after this wave's loads and LDS reads have completed), on top of the
// ring protocol's own barriers.  Extra barriers only remove overlap, so this
// build must give the same bytes as the release build; a difference would
// expose a read of a ring slot that its loads had not yet filled, or a load
// into a slot that another wave was still reading.
#ifdef QM_DEBUG_SYNC
constexpr bool kDebugSync = true;
#else
constexpr bool kDebugSync = false;
#endif

struct KParams {
  const uint8_t* q;   // 16-bit or FP8 elements, addressed in bytes
  const uint8_t* k;
  const uint8_t* v;
  uint16_t* o;
  float* lse;
  int N;
  int H;            // query heads
  int Hkv;          // key/value heads
  int group;        // H / Hkv: query heads per key/value head
  int nq;           // query blocks per head
  int wg_per_head;  // workgroups per head: nq, or ceil(nq / 2) pairs when causal
  int total;        // wg_per_head * B * H workgroups
  float c;     // |scale| * log2 e (FP8: |scale * q_scale * k_scale| * log2 e)
  float vscale;  // factor of O: 1, or the FP8 value scale
  int qmode;
  int layout;    // 0: q, k, v, o as [B][heads][N][width]; 1: as [B][N][heads][width]
};

// 16-bit type traits: the MFMA and the fp32 -> 16-bit pack (round to nearest
// even).
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

// FP8 (OCP E4M3) operands: the 32x32x64 MFMA, 32 one-byte values per lane
// (lane l: row or column l % 32, k = 32 (l / 32) + byte), and the fp32 -> E4M3
// pack of two values into one half of a word (round to nearest even; the
// values packed here are at most 2^8, below the 448 limit).  Zero scale
// operands select the unscaled form of the instruction, which issues faster
// than the block-scaled one.
struct Fp8 {
  static __device__ __forceinline__ f32x16 mfma(i32x8 a, i32x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
  }
  template <bool HIGH>   // into bits 16..31 (else 0..15) of old
  static __device__ __forceinline__ int32_t pack(float x, float y, int32_t old) {
    return __builtin_amdgcn_cvt_pk_fp8_f32(x, y, old, HIGH);
  }
};

// Operand traits: DT 0 = fp16, 1 = bf16 (16-bit operands, 32x32x16 MFMA),
// 2 = FP8 E4M3 (32x32x64 MFMA, bf16 output).
template <int DT>
struct Ops {
  static constexpr bool kFp8 = DT == 2;
  static constexpr int ES = kFp8 ? 1 : 2;        // bytes per input element
  static constexpr int KSTEP = kFp8 ? 64 : 16;   // MFMA contraction length
  static constexpr int KGB = KSTEP / 2 * ES;     // bytes of one lane's k-group
  using Frag = typename std::conditional<kFp8, i32x8, u32x4>::type;
  static __device__ __forceinline__ f32x16 mfma(Frag a, Frag b, f32x16 c) {
    if constexpr (kFp8) return Fp8::mfma(a, b, c);
    else return Half<DT>::mfma(a, b, c);
  }
};

// LDS layout of one K or V tile (kBN rows of ROWB bytes).  One direct load
// writes 1 KB = RPL whole rows; load group g holds rows g, g + NG, g + 2 NG,
// ... (NG groups), and groups are padded: K by 16 bytes, V by VPAD bytes (64
// for the 16-bit transposing reads, 16 for the byte ones).  Then a 128-bit K
// read of 16 consecutive rows in one column, and a transposing V read (16-bit:
// 4 consecutive rows x 4 consecutive 16-byte units; bytes: 4 rows of two
// groups x two 8-byte units), each touch distinct banks, and every operand
// address is a per-lane base plus a compile-time offset.
template <int ROWB, int VPAD = 64>
struct Layout {
  static constexpr int U = ROWB / 16;             // 16-byte units per row
  static constexpr int ROW = 16 * U;              // bytes per row
  static constexpr int RPL = 64 / U;              // rows per 1 KB load
  static constexpr int NG = kBN / RPL;            // load groups per tile
  static constexpr int KGS = 1024 + 16;           // K group stride (bytes)
  static constexpr int VGS = 1024 + VPAD;         // V group stride (bytes)
  static constexpr int KBYTES = NG * KGS;
  static constexpr int VBYTES = NG * VGS;
  static constexpr int BUF = KBYTES + VBYTES;     // one K tile + one V tile
  static_assert(NG >= 8, "a transposing read's 8 key rows must fall in distinct groups");
  static_assert(BUF % 16 == 0, "buffers stay 16-byte aligned");
};

// LDS layout of one K tile of DK columns of ES-byte elements: the first
// min(DK, 128) columns as a Layout part, and (DK = 192) the remaining 64
// columns as a second part right after it.  Each part keeps whole rows per
// direct load; the WAVES wavefronts share a tile's loads evenly.
template <int DK, int ES, int KSTEP, int WAVES>
struct KTile {
  static constexpr int W0 = DK < 128 ? DK : 128;  // columns of part 0
  static constexpr int W1 = DK - W0;              // columns of part 1 (0 or 64)
  using L0 = Layout<W0 * ES>;
  using L1 = Layout<W1 ? W1 * ES : 128>;          // unused when W1 == 0
  static constexpr int NKS0 = W0 / KSTEP;         // GEMM-I k-steps in part 0
  static constexpr int OFF1 = L0::NG * L0::KGS;   // byte offset of part 1
  static constexpr int BYTES = OFF1 + (W1 ? L1::NG * L1::KGS : 0);
  static constexpr int GPW0 = L0::NG / WAVES;     // direct loads per wave, part 0
  static constexpr int GPW1 = W1 ? L1::NG / WAVES : 0;
  static constexpr int GPW = GPW0 + GPW1;         // direct loads per wave per K block
  static_assert(W1 == 0 || W1 == 64, "K head dimensions 64, 128 and 192");
  static_assert(L0::NG % WAVES == 0 && L1::NG % WAVES == 0,
                "each wave issues whole load groups");
};

// Depth of the K and V rings.  Eight-wave workgroups (one per CU): four
// 64-key blocks (one barrier per two blocks) when four K and four V tiles fit
// the 160 KB of LDS, else two (one barrier per block).  Four-wave workgroups
// share a CU two or three at a time, so that one's prologue and epilogue
// overlap another's key loop: two blocks, except for FP8, whose one-byte
// tiles fit four-block rings (and the deferred GEMM-II) twice over.
template <int DK, int DV, int DT, int WAVES>
using KTileOf = KTile<DK, Ops<DT>::ES, Ops<DT>::KSTEP, WAVES>;
template <int DV, int DT>
using VTileOf = Layout<DV * Ops<DT>::ES, Ops<DT>::kFp8 ? 16 : 64>;

template <int DK, int DV, int DT, int WAVES>
constexpr int ring_depth() {
  return (WAVES == 8 || Ops<DT>::kFp8) &&
                 4 * (KTileOf<DK, DV, DT, WAVES>::BYTES + VTileOf<DV, DT>::VBYTES) <= 160 * 1024
             ? 4
             : 2;
}

template <int DK, int DV, int DT, int WAVES>
constexpr size_t lds_bytes() {
  return (size_t)ring_depth<DK, DV, DT, WAVES>() *
         (KTileOf<DK, DV, DT, WAVES>::BYTES + VTileOf<DV, DT>::VBYTES);
}

// Slot of exponential chunk c (of 16) in region 1 of NSLOT slots, and the
// chunk placed in slot s (-1: none).
__host__ __device__ constexpr int chunk_slot(int c, int nslot) { return c * nslot / 16; }
__host__ __device__ constexpr int slot_chunk(int s, int nslot) {
  for (int c = 0; c < 16; ++c)
    if (chunk_slot(c, nslot) == s) return c;
  return -1;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRsrcWord3);
}

// Exchange between the two lane halves that share a query column:
// v_permlane32_swap(a, b) swaps a's upper 32 lanes with b's lower 32 lanes, so
// with a = b = x, lane i < 32 ends with (x_i, x_{i+32}) and lane i >= 32 with
// (x_{i-32}, x_i): own and partner value in every lane.  The two results are
// copied to scalars before any bit cast (a bit cast applied to an element of
// the returned vector reads element 0).
__device__ __forceinline__ float max_across_halves(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const uint32_t a = r[0], b = r[1];
  return fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}

__device__ __forceinline__ float sum_across_halves(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const uint32_t a = r[0], b = r[1];
  return __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b);
}

// Buffer descriptor for the direct loads, as the four SGPRs the instruction
// takes: base, base high bits (stride 0), size in bytes, raw 32-bit format.
__device__ __forceinline__ i32x4 make_dma_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return i32x4{(int32_t)__builtin_amdgcn_readfirstlane((uint32_t)b),
               (int32_t)(__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32)) & 0xffff),
               (int32_t)bytes, kRsrcWord3};
}

// The same buffer seen from byte off on (base + off, size reduced by off), or,
// when live is false, a zero-size descriptor (a load through it touches no
// memory and writes zeros).  A load at per-lane offset v through it reads what
// a load at v + off through rs reads, under the same range check.  off must
// not exceed rs's size when live.
__device__ __forceinline__ i32x4 dma_rsrc_at(i32x4 rs, uint32_t off, bool live) {
  const uint64_t base = ((uint64_t)(uint32_t)rs[1] << 32 | (uint32_t)rs[0]) + off;
  return i32x4{(int32_t)(uint32_t)base, (int32_t)(uint32_t)(base >> 32),
               live ? (int32_t)((uint32_t)rs[2] - off) : 0, rs[3]};
}

// One 16-byte-per-lane direct load HBM -> LDS: lane l's 16 bytes at byte
// offset voff of the buffer land at LDS address lds + 16 l (M0 holds lds).
// The whole offset is in the VGPR operand: the range check covers only that
// operand (not the SGPR offset), and it is what turns rows past the end of
// the sequence into zeros.
//
// Written as inline assembly rather than the compiler builtin: the compiler
// cannot tell which LDS bytes a transposing read touches, so after a builtin
// direct load it waits for every load in flight before the first V read,
// which stalls the wave mid-block.  Here the only waits are the explicit
// ones before each barrier.  The compiler does not resolve hazards on an
// inline instruction's operands.  WAIT wait states precede the load: one
// (what the M0 write needs) for the loads of the key loop, where the compiled
// kernels have no VALU write of an SGPR the load reads within five wait
// states on any path into it (the build's assembly is checked for that);
// five for a run's first loads, where the compiler reloads spilled
// descriptor words with v_readlane (a VALU write of an SGPR needs five
// before a vector memory instruction reads it).  Five on every load instead
// cost 1-2.5% of the kernel's throughput.
template <int WAIT>
__device__ __forceinline__ void lds_load16(i32x4 rs, uint32_t lds, uint32_t voff) {
  static_assert(WAIT == 1 || WAIT == 5, "one or five wait states");
  if constexpr (WAIT == 1) {
    asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %2, 0 offen lds"
                 :: "v"(voff), "{m0}"(lds), "s"(rs) : "memory");
  } else {
    asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %0, %2, 0 offen lds"
                 :: "v"(voff), "{m0}"(lds), "s"(rs) : "memory");
  }
}

// The lane's index in its wavefront, as volatile inline assembly so that the
// compiler recomputes it where it is asked for instead of keeping one value
// live (or spilled) across long stretches of code.
__device__ __forceinline__ int lane_id() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Workgroups per CU the register budget is sized for: one of eight waves; two
// of four waves, or three at d = 64 (168 VGPRs, 33 KB of LDS each), where the
// third workgroup's waves fill the latency of the exponential-bound loop.
template <int DK, int WAVES>
constexpr int wgs_per_cu() {
  return WAVES == 8 ? 1 : (DK == 64 ? 3 : 2);
}

template <int DK, int DV, int DT, bool CAUSAL, int WAVES>
__global__ __launch_bounds__(64 * WAVES, (wgs_per_cu<DK, WAVES>())) void attn_fwd_kernel(KParams p) {
  using OP = Ops<DT>;
  using Frag = typename OP::Frag;        // one MFMA A or B operand
  constexpr bool FP8 = OP::kFp8;
  constexpr int ES = OP::ES;             // bytes per input element
  using KT = KTileOf<DK, DV, DT, WAVES>; // K tile (DK columns)
  using LV = VTileOf<DV, DT>;            // V tile (DV columns)
  constexpr int NKS = DK / OP::KSTEP;    // GEMM-I k-steps
  constexpr int NMT = DV / 32;           // GEMM-II M tiles
  constexpr int BM = 32 * WAVES;         // query rows per workgroup
  static_assert(LV::NG % WAVES == 0, "each wave issues whole load groups");
  constexpr int GPWV = LV::NG / WAVES;   // V direct loads per wave per block
  constexpr int RING = ring_depth<DK, DV, DT, WAVES>();
  // Deferred GEMM-II: with four-block rings, GEMM-II of block j can run in
  // block j+1's region, interleaved with that block's exponentials and GEMM-I,
  // so that no MFMA-only stretch remains in a block.  Used where the
  // exponentials outweigh the MFMAs (FP8, d = 64), where it gains 2-6%; at
  // d = 128 with 16-bit inputs it gains nothing at long sequences and costs
  // 1-3% at short ones, so GEMM-II stays at the end of its own block there.
  constexpr bool DEFER = RING == 4 && (FP8 || DK == 64);
  constexpr int NPB = FP8 ? 1 : 4;       // P^T operand fragments per block

  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  char* const lds = reinterpret_cast<char*>(smem);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int N = p.N;

  // ---- which tiles this workgroup owns ----
  // A tile is one (batch*head, query block), or, causal, the pair (nq-1-i, i)
  // of query blocks (query block qb costs qb + 1 units of key blocks, so every
  // pair costs the same and the grid has no long tail; the longer runs first).
  // 16-bit inputs: the grid holds as many workgroups as the CUs run at once
  // (a multiple of 8), and workgroup w walks tiles w, w + grid, ..., so the
  // launch gap and set-up of a new workgroup are paid once per CU, not per
  // tile.  FP8 launches one workgroup per tile (its loop measured slower).
  const int per_xcd = p.total / kXcds;
  auto do_tile = [&](int tile) __attribute__((always_inline)) {
  int id = tile;
  if (id < per_xcd * kXcds) id = (id % kXcds) * per_xcd + id / kXcds;
  const int bh = id / p.wg_per_head;
  const int slot_in_head = id - bh * p.wg_per_head;
  int qbs[2] = {slot_in_head, -1};
  if (CAUSAL) {
    qbs[0] = p.nq - 1 - slot_in_head;
    qbs[1] = (slot_in_head != p.nq - 1 - slot_in_head) ? slot_in_head : -1;
  }

  // query head h of batch b reads key/value head h / group (grouped-query
  // attention; group = 1 is multi-head attention).  Consecutive query heads
  // share a key/value head, so with the id order above a whole group's
  // workgroups run on one XCD and share its L2 for the K/V stream.
  const int b = bh / p.H;
  const int bhkv = b * p.Hkv + (bh - b * p.H) / p.group;
  // One head's rows: w bytes each, rs bytes apart ([B][heads][N][w]: rs = w,
  // heads contiguous; [B][N][heads][w]: rs = heads * w, heads interleaved).
  // Every access goes through a buffer resource spanning exactly the head's
  // rows, (N - 1) rs + w bytes, so rows past the end read as zeros and
  // stores to them are dropped.
  // (The two-block-ring instances, 192-wide keys, take [B][heads][N][w] only:
  // runtime strides there spill registers.)
  const bool bnhd = RING == 4 && p.layout != 0;
  constexpr uint32_t WQ = DK * ES, WV = DV * ES, WO = DV * 2;
  const uint32_t rs_q = bnhd ? p.H * WQ : WQ;
  const uint32_t rs_k = bnhd ? p.Hkv * WQ : WQ;
  const uint32_t rs_v = bnhd ? p.Hkv * WV : WV;
  const uint32_t rs_o = bnhd ? p.H * WO : WO;
  auto head_off = [&](int bb, int h, int heads, uint32_t w) -> size_t {
    return bnhd ? ((size_t)bb * N * heads + h) * w : ((size_t)bb * heads + h) * N * w;
  };
  auto span = [&](uint32_t rs, uint32_t w) { return (uint32_t)(N - 1) * rs + w; };
  const int h_q = bh - b * p.H, h_kv = bhkv - b * p.Hkv;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(p.q + head_off(b, h_q, p.H, WQ), span(rs_q, WQ));
  const i32x4 rk = make_dma_rsrc(p.k + head_off(b, h_kv, p.Hkv, WQ), span(rs_k, WQ));
  const i32x4 rv = make_dma_rsrc(p.v + head_off(b, h_kv, p.Hkv, WV), span(rs_v, WV));

  auto run = [&](int qb) __attribute__((always_inline)) {
    // this lane's index, formed afresh in each run: no lane value stays live
    // from one query block to the next (kept live, it spills)
    const int lane = lane_id();
    const int l32 = lane & 31;
    const int hi = lane >> 5;
    const int q0 = qb * BM;
    const int qw = q0 + wave * 32;   // first query row of this wavefront
    const int qrow = qw + l32;       // the query row whose column this lane holds

    // ---- Q: B operand of GEMM-I, resident for the whole key loop ----
    // lane: query row qrow, k-group hi (OP::KGB bytes of each k-step)
    Frag qf[NKS];
  #pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const uint32_t off = (uint32_t)qrow * rs_q + (uint32_t)(ks * OP::KSTEP * ES + hi * OP::KGB);
      if constexpr (FP8) {
        const u32x4 lo = __builtin_amdgcn_raw_buffer_load_b128(rq, off, 0, 0);
        const u32x4 up = __builtin_amdgcn_raw_buffer_load_b128(rq, off + 16, 0, 0);
        qf[ks] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                       (int)up[0], (int)up[1], (int)up[2], (int)up[3]};
        if (p.qmode == kQNegate) qf[ks] ^= (int)0x80808080u;
      } else {
        qf[ks] = __builtin_amdgcn_raw_buffer_load_b128(rq, off, 0, 0);
        if (p.qmode == kQNegate) qf[ks] ^= 0x80008000u;
      }
      if (p.qmode == kQZero) qf[ks] = Frag{};
    }

    const int kv_end = CAUSAL ? min(N, q0 + BM) : N;
    const int nkv = (kv_end + kBN - 1) / kBN;

    f32x16 oacc[NMT];
  #pragma unroll
    for (int mt = 0; mt < NMT; ++mt) oacc[mt] = f32x16{};
    // running maximum, exp2 domain; -FLT_MAX (not -inf) while a lane has seen
    // no visible key, so that it serves as the exponentials' offset directly:
    // every visible key then overflows to +inf and forces the exact path
    float m_run = -FLT_MAX;
    float l_run = 0.f;         // this lane's share of the running row sum

    // ---- HBM -> LDS: this wave's load groups of one K or V block ----
    // LDS: RING K slots, then RING V slots, of one 64-key block each
    constexpr int VOFF = RING * KT::BYTES;
    // lane parts of the global offsets (row slot, 16-byte unit, column of the
    // K part); the row of the load group is added per load
    const uint32_t koff0 = (uint32_t)(KT::L0::NG * (lane / KT::L0::U)) * rs_k +
                           (uint32_t)((lane % KT::L0::U) * 16);
    const uint32_t koff1 = (uint32_t)(KT::L1::NG * (lane / KT::L1::U)) * rs_k +
                           (uint32_t)(KT::W0 * ES + (lane % KT::L1::U) * 16);
    const uint32_t voff = (uint32_t)(LV::NG * (lane / LV::U)) * rs_v + (uint32_t)((lane % LV::U) * 16);
    auto lds_addr = [&](int byte_off) { return (uint32_t)(uintptr_t)(lds_void*)(lds + byte_off); };
    // wait states before a direct load: a run's first loads, or the key loop's
    using Wait5 = std::integral_constant<int, 5>;
    using Wait1 = std::integral_constant<int, 1>;
    // The block's first row goes into the descriptor (scalar work, once per
    // block and tensor); the group's row and the lane's part stay in a
    // per-lane offset that does not change from block to block.  live: the
    // block is one this query block uses; its first row is then inside the
    // sequence, so the shifted size does not wrap.
    // load i (of KT::GPW) of this wave for K block blk into K slot kb
    auto k_load = [&](auto wait, int i, int blk, int kb, bool live) __attribute__((always_inline)) {
      constexpr int W = decltype(wait)::value;
      const i32x4 rs = dma_rsrc_at(rk, (uint32_t)(blk * kBN) * rs_k, live);
      if (i < KT::GPW0) {
        const int g = wave * KT::GPW0 + i;
        lds_load16<W>(rs, lds_addr(kb * KT::BYTES + g * KT::L0::KGS), koff0 + (uint32_t)g * rs_k);
      } else {
        const int g = wave * KT::GPW1 + (i - KT::GPW0);
        lds_load16<W>(rs, lds_addr(kb * KT::BYTES + KT::OFF1 + g * KT::L1::KGS),
                   koff1 + (uint32_t)g * rs_k);
      }
    };
    // load i (of GPWV) of this wave for V block blk into V slot vb
    auto v_load = [&](auto wait, int i, int blk, int vb, bool live) __attribute__((always_inline)) {
      constexpr int W = decltype(wait)::value;
      const i32x4 rs = dma_rsrc_at(rv, (uint32_t)(blk * kBN) * rs_v, live);
      const int g = wave * GPWV + i;
      lds_load16<W>(rs, lds_addr(VOFF + vb * LV::VBYTES + g * LV::VGS), voff + (uint32_t)g * rs_v);
    };
    auto load_k = [&](int blk, int kb) {
  #pragma unroll
      for (int i = 0; i < KT::GPW; ++i) k_load(Wait5{}, i, blk, kb, true);
    };
    auto load_v = [&](int blk, int vb) {
  #pragma unroll
      for (int i = 0; i < GPWV; ++i) v_load(Wait5{}, i, blk, vb, true);
    };

    // Direct loads issued during block j, Q = j % 4 (loads of blocks past the
    // last go through the zero-size descriptor, into slots no one reads again).
    //   RING = 4: an even block loads K(j+3) and K(j+4) into K slots (Q+3) % 4
    //             and Q, an odd block V(j+1) and V(j+2) into V slots (Q+1) % 4
    //             and (Q+2) % 4, or, when GEMM-II of block j runs during block
    //             j+1, V(j) and V(j+1) into V slots Q and (Q+1) % 4;
    //   RING = 2: every block loads K(j+2) into K slot Q % 2 and V(j+1) into V
    //             slot (Q+1) % 2.
    auto n_dma = [](auto ph) {
      constexpr int Q = decltype(ph)::value;
      return RING == 4 ? (Q % 2 == 0 ? 2 * KT::GPW : 2 * GPWV) : KT::GPW + GPWV;
    };
    auto dma = [&](auto ph, int n, int j) __attribute__((always_inline)) {
      constexpr int Q = decltype(ph)::value;
      if (RING == 4 && Q % 2 == 0) {
        const int second = n >= KT::GPW ? 1 : 0;
        const int blk = j + 3 + second;
        k_load(Wait1{}, n - second * KT::GPW, blk, (Q + 3 + second) % 4, blk < nkv);
      } else if (RING == 4) {
        const int second = n >= GPWV ? 1 : 0;
        const int lead = DEFER ? 0 : 1;   // deferred GEMM-II reads V(j) a block later
        const int blk = j + lead + second;
        v_load(Wait1{}, n - second * GPWV, blk, (Q + lead + second) % 4, blk < nkv);
      } else if (n < KT::GPW) {
        k_load(Wait1{}, n, j + 2, Q % 2, j + 2 < nkv);
      } else {
        v_load(Wait1{}, n - KT::GPW, j + 1, (Q + 1) % 2, j + 1 < nkv);
      }
    };

    // per-lane LDS byte bases of the operand reads; every read adds a constant
    //   K (A of GEMM-I): row r = 32 kt + l32 -> group r % NG, slot r / NG of
    //   its part; unit 2 ks + hi
    const int k_base0 = (l32 % KT::L0::NG) * KT::L0::KGS + (l32 / KT::L0::NG) * KT::L0::ROW +
                        OP::KGB * hi;
    const int k_base1 = KT::OFF1 + (l32 % KT::L1::NG) * KT::L1::KGS +
                        (l32 / KT::L1::NG) * KT::L1::ROW + OP::KGB * hi;
    //   V (A of GEMM-II, transposing read): key = 16 u + 8 h2 + kq, dims d0 .. d0+3
    const int grp = lane >> 4;
    const int sl = lane & 15;
    const int kq = 4 * (grp >> 1) + (sl >> 2);
    const int v_base = VOFF + kq * LV::VGS + 2 * (16 * (grp & 1) + 4 * (sl & 3));
    //   V, FP8 (byte-transposing read; within each 16-lane group G, output lane
    //   i, byte r is byte i % 8 of source lane 2 r + i / 8): source lane
    //   2 r + e of group G reads 8 bytes of key 32 (t/2) + 16 (t%2) + 8 (r/4) +
    //   4 (G/2) + r%4 (read t of 4), columns 32 mt + 16 (G%2) + 8 e onward, so
    //   that output lane l gets column 32 mt + l%32 of exactly the keys its P
    //   bytes hold (byte j: key 32 (j/16) + 8 ((j/4)%4) + 4 (l/32) + j%4)
    const int v8_base = VOFF + (4 * (grp >> 1) + ((sl >> 1) & 3)) * LV::VGS +
                        (sl >> 3) * LV::ROW + 16 * (grp & 1) + 8 * (sl & 1);

    auto k_read = [&](int kb, int kt, int ks) {
      constexpr int KSB = OP::KSTEP * ES;   // bytes per k-step of a row
      const char* a = (ks < KT::NKS0)
          ? lds + kb * KT::BYTES + k_base0 + kt * (32 / KT::L0::NG) * KT::L0::ROW + KSB * ks
          : lds + kb * KT::BYTES + k_base1 + kt * (32 / KT::L1::NG) * KT::L1::ROW +
                KSB * (ks - KT::NKS0);
      if constexpr (FP8) {
        const u32x4 lo = *reinterpret_cast<const u32x4*>(a);
        const u32x4 up = *reinterpret_cast<const u32x4*>(a + 16);
        return i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                     (int)up[0], (int)up[1], (int)up[2], (int)up[3]};
      } else {
        return *reinterpret_cast<const u32x4*>(a);
      }
    };
    auto v_read = [&](int vb, int mt, int u, int h2) {
      // group of key 16 u + 8 h2 + kq is (16 u + 8 h2) % NG + kq, slot (16 u + 8 h2) / NG
      const int g_off = (16 * u + 8 * h2) % LV::NG;
      const int slot = (16 * u + 8 * h2) / LV::NG;
      return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (lds_i16x4*)(lds + vb * LV::VBYTES + v_base + g_off * LV::VGS + slot * LV::ROW + 64 * mt));
    };

    // GEMM-II operand from V slot vb: V^T fragment t (M tile t % NMT, key step
    // t / NMT), so consecutive MFMAs accumulate into different O tiles
    auto v_frag = [&](int vb, int t) __attribute__((always_inline)) {
      if constexpr (FP8) {
        // M tile t, all 64 keys: four byte-transposing reads of 8 bytes
        i32x8 f;
  #pragma unroll
        for (int c = 0; c < 4; ++c) {
          const i32x2 x = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
              (lds_i32x2*)(lds + vb * LV::VBYTES + v8_base + 2 * c * LV::ROW + 32 * t));
          f[2 * c] = x[0];
          f[2 * c + 1] = x[1];
        }
        return f;
      } else {
        const int mt = t % NMT, u = t / NMT;
        const u32x2 a0 = __builtin_bit_cast(u32x2, v_read(vb, mt, u, 0));
        const u32x2 a1 = __builtin_bit_cast(u32x2, v_read(vb, mt, u, 1));
        return u32x4{a0[0], a0[1], a1[0], a1[1]};
      }
    };
    // GEMM-II of one block on its own: O^T += V^T P^T from V slot vb (a wave's
    // last block, when GEMM-II is deferred)
    auto gemm2 = [&](int vb, const Frag (&pin)[NPB]) __attribute__((always_inline)) {
      constexpr int NV = FP8 ? NMT : 4 * NMT;
      // one fragment in flight at a time: this runs once per wave, and reading
      // every fragment up front would raise the register peak of the kernel
  #pragma unroll
      for (int t = 0; t < NV; ++t) {
        oacc[t % NMT] = OP::mfma(v_frag(vb, t), pin[FP8 ? 0 : t / NMT], oacc[t % NMT]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // GEMM-I: two 32-key tiles of S^T for the block in K buffer kb
    auto gemm1 = [&](int kb, f32x16 (&s)[2]) {
      s[0] = f32x16{};
      s[1] = f32x16{};
  #pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
  #pragma unroll
        for (int kt = 0; kt < 2; ++kt) s[kt] = OP::mfma(k_read(kb, kt, ks), qf[ks], s[kt]);
      }
    };

    // Block j: mask, row max and (rare) rescale; then, in one straight-line
    // region, the exponentials of block j interleaved with the MFMAs of GEMM-I
    // for block j+1 (and, deferred, of GEMM-II for block j-1); then GEMM-II of
    // block j unless deferred.  GEMM-I always runs: on a wave's
    // last block it reads a stale (in-bounds) K buffer and its result is dropped,
    // which keeps a single code path and the register allocation compact.
    // row maximum of a block's (masked) scores, both lane halves, raw units
    auto row_max = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) {
      float mx = fmaxf(sc[0][0], sc[1][0]);
  #pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(sc[0][r], sc[1][r]));
      return max_across_halves(mx);
    };

    // Block j.  Probabilities are formed against the running maximum m_run
    // without looking at the block's own maximum; since every p >= 0, a lane
    // whose 32 probabilities sum to at most 2^8 (kPmax) has every p <= 2^8, which
    // keeps all sums in range.  Only when some lane exceeds that (the running
    // maximum must rise, and always on a wave's first block, where m_run is
    // -FLT_MAX), or, for 16-bit inputs, when some lane's block sum exceeds
    // kDominant times its running sum, is the block's exact maximum taken, O
    // and l rescaled and the probabilities recomputed.  Results are exact
    // either way: O and lse use the same m_run.
    // vb: the V slot GEMM-II reads (block j's, or block j-1's when deferred);
    // pin: P^T of block j-1 (deferred GEMM-II); pout: P^T of block j; first:
    // block 0, which has no deferred GEMM-II to run
    auto block = [&](auto ph, auto first, int j, int kb_next, int vb, f32x16 (&s)[2],
                     f32x16 (&s_next)[2], const Frag (&pin)[NPB], Frag (&pout)[NPB])
        __attribute__((always_inline)) {
      constexpr bool DEF = DEFER && !decltype(first)::value;   // GEMM-II of block j-1 here
      const int j0 = j * kBN;
      constexpr int AHEAD = FP8 ? 2 : 4;              // operand reads ahead of their MFMA
      constexpr int NG1 = 2 * NKS;                    // GEMM-I MFMAs per block
      constexpr int NV = FP8 ? NMT : 4 * NMT;         // GEMM-II MFMAs per block
      constexpr int NM = DEF ? NV + NG1 : NG1;        // MFMAs of region 1
      constexpr int NSLOT = NM > 16 ? NM : 16;        // slots of region 1
      constexpr int NDMA = n_dma(decltype(ph){});     // direct loads in this block
      constexpr int DSTRIDE = (NSLOT / 2) / NDMA > 0 ? (NSLOT / 2) / NDMA : 1;
      // first operand fragments of region 1 (deferred: V of GEMM-II, else K of
      // GEMM-I for block j+1): their LDS latency runs under the mask work below
      Frag kring[AHEAD];
      Frag vring[AHEAD];
  #pragma unroll
      for (int m = 0; m < AHEAD; ++m) {
        if constexpr (DEF) vring[m] = v_frag(vb, m);
        else kring[m] = k_read(kb_next, m % 2, m / 2);
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
      float mu = m_run;

      // P^T operands of GEMM-II: 16-bit, four fragments of 8 values (key step
      // u = 16 keys); FP8, one fragment of all 32 of the lane's values, byte
      // j = the score of key tile j / 16, register j % 16
      Frag (&pb)[NPB] = pout;
      // the pair of probabilities of chunk i (keys r0 and r0 + 1 of key tile
      // kt = i / 8, r0 = 8 ((i / 4) % 2) + 2 (i % 4)) into the operand
      auto put = [&](int i, float e0, float e1) __attribute__((always_inline)) {
        const int u = i / 4, w = i % 4;
        if constexpr (FP8) {
          const int word = 2 * u + w / 2;
          // the low half first; the stale high half it keeps is overwritten next
          int32_t pk = (w % 2) ? Fp8::pack<true>(e0, e1, pb[0][word])
                               : Fp8::pack<false>(e0, e1, pb[0][word]);
          asm volatile("" : "+v"(pk));
          pb[0][word] = pk;
        } else {
          uint32_t pk = Half<DT>::pack(e0, e1);
          asm volatile("" : "+v"(pk));
          pb[u][w] = pk;
        }
      };
      float lsum = 0.f;
      // one 16-bit pair of P^T (chunk i of 16): two FMAs, two exponentials, the
      // row-sum adds, one pack.  The row sum stays in fp32 (a sum of the
      // rounded values would carry their rounding into lse whenever a few keys
      // dominate the row).
      auto exp_chunk = [&](int i) __attribute__((always_inline)) {
        const int u = i / 4, w = i % 4;
        const int r0 = 8 * (u % 2) + 2 * w;
        const float e0 = __builtin_amdgcn_exp2f(fmaf(s[u / 2][r0], p.c, -mu));
        const float e1 = __builtin_amdgcn_exp2f(fmaf(s[u / 2][r0 + 1], p.c, -mu));
        put(i, e0, e1);
        lsum += e0 + e1;
      };

      // Straight-line region 1, written as NSLOT = max(NM, 16) slots for its NM
      // MFMAs: GEMM-I for block j+1 (16 at DK = 128, 24 at DK = 192, 8 at 64,
      // 4 for FP8), preceded, when GEMM-II is deferred, by GEMM-II of block j-1
      // (8 at d = 64, 4 for FP8).  The MFMAs are spread evenly over the slots,
      // and the slots advance the 16 exponential chunks of block j through a
      // three-stage software pipeline: the FMAs of pair i+2, the exponentials
      // of pair i+1, and the pack and row-sum adds of pair i, so that no
      // instruction waits on a result produced in its own slot.  Operand reads
      // run AHEAD MFMAs early from small register rings (the last slots start
      // on the next MFMA kind's fragments); a scheduling fence after each slot
      // keeps the order and the live ranges.
      s_next[0] = f32x16{};
      s_next[1] = f32x16{};
      float xa[18], xb[18], ea[17], eb[17];
      float lsum_even = 0.f, lsum_odd = 0.f;
      auto arg = [&](int i, int k) __attribute__((always_inline)) {
        const int u = i / 4, w = i % 4;
        return fmaf(s[u / 2][8 * (u % 2) + 2 * w + k], p.c, -mu);
      };
      // Raised issue priority while this wave has both MFMAs and VALU work: the
      // other wave of the SIMD, in its MFMA-only GEMM-II, fills the gaps.
      __builtin_amdgcn_s_setprio(1);
      xa[0] = arg(0, 0);
      xb[0] = arg(0, 1);
      xa[1] = arg(1, 0);
      xb[1] = arg(1, 1);
      ea[0] = __builtin_amdgcn_exp2f(xa[0]);
      eb[0] = __builtin_amdgcn_exp2f(xb[0]);
  #pragma unroll
      for (int sidx = 0; sidx < NSLOT; ++sidx) {
        if ((sidx * NM) % NSLOT == 0) {
          // deferred: MFMAs 0 .. NV-1 are GEMM-II of block j-1 (fragment t = m),
          // then GEMM-I; else all are GEMM-I
          const int m = sidx * NM / NSLOT;
          if (DEF && m < NV) {
            const Frag a = vring[m % AHEAD];
            if (m + AHEAD < NV) {
              vring[m % AHEAD] = v_frag(vb, m + AHEAD);
            } else {
              const int g = m + AHEAD - NV;   // first K fragments of GEMM-I
              kring[g % AHEAD] = k_read(kb_next, g % 2, g / 2);
            }
            oacc[m % NMT] = OP::mfma(a, pin[FP8 ? 0 : m / NMT], oacc[m % NMT]);
          } else {
            const int g = DEF ? m - NV : m;   // GEMM-I MFMA g: k-step g / 2, key tile g % 2
            const Frag a = kring[g % AHEAD];
            if (g + AHEAD < NG1) kring[g % AHEAD] = k_read(kb_next, (g + AHEAD) % 2, (g + AHEAD) / 2);
            s_next[g % 2] = OP::mfma(a, qf[g / 2], s_next[g % 2]);
          }
        }
        if (!DEFER && sidx >= NSLOT - AHEAD) vring[sidx - (NSLOT - AHEAD)] = v_frag(vb, sidx - (NSLOT - AHEAD));
        // this block's direct loads, spread over the first half of the region
        if (sidx % DSTRIDE == 0 && sidx / DSTRIDE < NDMA) dma(ph, sidx / DSTRIDE, j);
        const int i = slot_chunk(sidx, NSLOT);
        if (i < 0) {
          __builtin_amdgcn_sched_barrier(0);
          continue;
        }
        if (i + 1 < 16) {
          ea[i + 1] = __builtin_amdgcn_exp2f(xa[i + 1]);
          eb[i + 1] = __builtin_amdgcn_exp2f(xb[i + 1]);
        }
        if (i + 2 < 16) {
          xa[i + 2] = arg(i + 2, 0);
          xb[i + 2] = arg(i + 2, 1);
        }
        // 16-bit P^T operands; the row sum stays in fp32 (a sum of the rounded
        // values would carry their rounding into lse whenever a few keys
        // dominate the row)
        // (the empty asm statement in put keeps the pack in this slot: left
        // alone, the compiler sinks all 16 packs past the exact-path branch
        // below, where no MFMA runs beside them)
        put(i, ea[i], eb[i]);
        if (i % 2 == 0) lsum_even += ea[i] + eb[i];
        else lsum_odd += ea[i] + eb[i];
        __builtin_amdgcn_sched_barrier(0);
      }
      __builtin_amdgcn_s_setprio(0);
      lsum = lsum_even + lsum_odd;

      // exact path (rare): the running maximum rises.  One compare against
      // min(kPmax, kDominant * l_run), whose operands are ready before the
      // region ends (two compares joined before the vote cost a select and a
      // second compare on the critical path)
      const float l_thr = FP8 ? kPmax : fminf(kPmax, kDominant * l_run);
      if (__any(lsum > l_thr)) {
        // a use of GEMM-I's results on this path too keeps the compiler from
        // sinking GEMM-I's MFMAs out of region 1 to past this branch
        asm volatile("" :: "v"(s_next[0]), "v"(s_next[1]));
        const float m_blk = row_max(s) * p.c;
        const float m_new = fmaxf(m_run, m_blk);
        // 0 on a lane's first visible keys (m_run = -FLT_MAX); O and l are
        // then 0 anyway
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
  #pragma unroll
        for (int mt = 0; mt < NMT; ++mt) oacc[mt] *= alpha;
        l_run *= alpha;
        m_run = m_new;
        mu = m_run;
        lsum = 0.f;
  #pragma unroll
        for (int i = 0; i < 16; ++i) exp_chunk(i);
      }
      l_run += lsum;

      // Straight-line region 2 (not deferred): GEMM-II, O^T += V^T P^T
      if constexpr (!DEFER) {
  #pragma unroll
        for (int t = 0; t < NV; ++t) {
          const Frag a = vring[t % AHEAD];
          if (t + AHEAD < NV) vring[t % AHEAD] = v_frag(vb, t + AHEAD);
          oacc[t % NMT] = OP::mfma(a, pb[FP8 ? 0 : t / NMT], oacc[t % NMT]);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    };

    // Pipeline.  Block j (Q = j % 4) finds K(j+1) in K slot (Q+1) % RING and
    // V(j) in V slot Q % RING (deferred: V(j-1) in V slot (Q+3) % 4), and
    // issues direct loads (see dma above).  Deferred schedule: a pair of blocks
    // (j, j+1), j even, reads V slots (j+3) % 4 and j % 4 and loads V(j+1) and
    // V(j+2) into slots (j+1) % 4 and (j+2) % 4, so loads and reads of one pair
    // never share a slot; V(i) is loaded by the odd block i or i-1 and read by
    // block i+1, after the barrier that ends that odd block.
    // RING = 4: one barrier per pair of blocks, after each odd block: it
    // publishes the pair's loads (each wave first waits for its own) and
    // retires the pair's reads of the slots the next pair refills, so the
    // rings hold two blocks being read and two being loaded.  RING = 2: one
    // barrier per block, one block read and one loaded.  Blocks a wave skips
    // (causal) come only after all the blocks it computes; it still issues
    // their loads.
    f32x16 sa[2], sb[2];
    // P^T of the even and the odd blocks (read by the next block when deferred)
    Frag p_even[NPB] = {}, p_odd[NPB] = {};
    auto sync = [&]() __attribute__((always_inline)) {
      __builtin_amdgcn_s_waitcnt(kWaitLoads);
      __syncthreads();
    };
    // Blocks this wave computes: 0 .. j_act-1 (causal: the blocks up to its
    // last row; none for a wave past the sequence end).  It still issues the
    // loads of the blocks after those, and takes every barrier.
    const int j_act = (qw >= N) ? 0 : (CAUSAL ? min(nkv, (qw + 31) / kBN + 1) : nkv);
    // The computed blocks run in one loop and the skipped ones in a second,
    // so that no block tests whether it computes; only the four-wave causal
    // d = 64 instance, at its register ceiling, keeps that test inside one
    // loop over all blocks (the split loops spill there).
    constexpr bool kSplitLoops = DEFER || !(DK == 64 && WAVES == 4 && CAUSAL);
    auto iteration = [&](auto ph, auto first, int j, f32x16 (&s_cur)[2], f32x16 (&s_next)[2],
                         Frag (&pin)[NPB], Frag (&pout)[NPB]) __attribute__((always_inline)) {
      constexpr int Q = decltype(ph)::value;
      constexpr int VB = DEFER ? (Q + 3) % 4 : Q % RING;   // the V slot GEMM-II reads
      if (kSplitLoops || j < j_act) {
        block(ph, first, j, (Q + 1) % RING, VB, s_cur, s_next, pin, pout);
      } else {
  #pragma unroll
        for (int n = 0; n < n_dma(ph); ++n) dma(ph, n, j);
      }
      if (RING == 2 || Q % 2 == 1 || kDebugSync) sync();
    };
    // a block this wave skips: its loads and its barrier only
    auto skipped = [&](auto ph, int j) __attribute__((always_inline)) {
      constexpr int Q = decltype(ph)::value;
  #pragma unroll
      for (int n = 0; n < n_dma(ph); ++n) dma(ph, n, j);
      if (RING == 2 || Q % 2 == 1 || kDebugSync) sync();
    };

    load_k(0, 0);
    load_v(0, 0);
    if (nkv > 1) load_k(1, 1);
    if (RING == 4 && nkv > 2) load_k(2, 2);
    if (RING == 4 && !DEFER && nkv > 1) load_v(1, 1);
    __builtin_amdgcn_s_waitcnt(kWaitLoads);
    __syncthreads();
    if (j_act > 0) gemm1(0, sa);
    __syncthreads();   // K slot 0 is refilled by block 0

    using C0 = std::integral_constant<int, 0>;
    using C1 = std::integral_constant<int, 1>;
    using C2 = std::integral_constant<int, 2>;
    using C3 = std::integral_constant<int, 3>;
    using Later = std::false_type;
    using First = std::true_type;
    // Deferred: block 0 (no GEMM-II of its own to run), then the other
    // computed blocks, the skipped ones after the last GEMM-II below.
    // Otherwise one loop over the computed blocks (over all blocks where
    // kSplitLoops is off), the skipped ones after it.
    const int j_loop = kSplitLoops ? j_act : nkv;
    if constexpr (DEFER) {
      if (j_act > 0) {
        iteration(C0{}, First{}, 0, sa, sb, p_odd, p_even);
        for (int j = 1; j < j_act; j += 4) {
          iteration(C1{}, Later{}, j, sb, sa, p_even, p_odd);
          if (j + 1 >= j_act) break;
          iteration(C2{}, Later{}, j + 1, sa, sb, p_odd, p_even);
          if (j + 2 >= j_act) break;
          iteration(C3{}, Later{}, j + 2, sb, sa, p_even, p_odd);
          if (j + 3 >= j_act) break;
          iteration(C0{}, Later{}, j + 3, sa, sb, p_odd, p_even);
        }
      }
    } else {
      for (int j = 0; j < j_loop; j += 4) {
        iteration(C0{}, Later{}, j, sa, sb, p_odd, p_even);
        if (j + 1 >= j_loop) break;
        iteration(C1{}, Later{}, j + 1, sb, sa, p_even, p_odd);
        if (j + 2 >= j_loop) break;
        iteration(C2{}, Later{}, j + 2, sa, sb, p_odd, p_even);
        if (j + 3 >= j_loop) break;
        iteration(C3{}, Later{}, j + 3, sb, sa, p_even, p_odd);
      }
    }
    // the deferred GEMM-II of the wave's last computed block, at the point
    // where the next block would have run it (its V slot is refilled only
    // after the next barrier)
    if constexpr (DEFER) {
      if (j_act > 0) {
        if ((j_act - 1) % 2 == 0) gemm2((j_act - 1) % 4, p_even);
        else gemm2((j_act - 1) % 4, p_odd);
      }
    }
    for (int j = j_loop; j < nkv; ++j) {
      switch (j % 4) {
        case 0: skipped(C0{}, j); break;
        case 1: skipped(C1{}, j); break;
        case 2: skipped(C2{}, j); break;
        default: skipped(C3{}, j); break;
      }
    }
    // a lone last block still ends with a barrier (kept out of the loops: a
    // barrier on a loop exit path makes the register allocator spill)
    if (RING == 4 && nkv % 2 == 1) sync();

    // ---- epilogue: O = O / l in the storage type, lse in natural log ----
    const float l_tot = sum_across_halves(l_run);
    const float inv = p.vscale / l_tot;
    // the output is 16-bit for every input type (FP8 inputs give bf16)
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(p.o + head_off(b, h_q, p.H, WO) / 2, span(rs_o, WO));
  #pragma unroll
    for (int mt = 0; mt < NMT; ++mt) {
  #pragma unroll
      for (int g = 0; g < 4; ++g) {
        using OutT = Half<FP8 ? 1 : DT>;   // FP8 inputs give a bf16 output
        const u32x2 w = {OutT::pack(oacc[mt][4 * g] * inv, oacc[mt][4 * g + 1] * inv),
                         OutT::pack(oacc[mt][4 * g + 2] * inv, oacc[mt][4 * g + 3] * inv)};
        __builtin_amdgcn_raw_buffer_store_b64(
            w, ro, (uint32_t)qrow * rs_o + (uint32_t)(32 * mt + 8 * g + 4 * hi) * 2, 0, 0);
      }
    }
    if (hi == 0) {
      const __amdgpu_buffer_rsrc_t rl = make_rsrc(p.lse + (size_t)bh * N, (uint32_t)N * 4);
      const float lse = (m_run + log2f(l_tot)) * 0.69314718055994531f;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, lse), rl, (uint32_t)qrow * 4, 0, 0);
    }
  };
  run(qbs[0]);
  if (CAUSAL && qbs[1] >= 0) {
    // the last deferred GEMM-II reads a V slot after the final barrier, which
    // the next block's first loads may refill
    if (DEFER) __syncthreads();
    run(qbs[1]);
  }
  };
  if constexpr (FP8) {
    do_tile(blockIdx.x);
  } else {
    for (int tile = blockIdx.x; tile < p.total; tile += gridDim.x) {
      do_tile(tile);
      // the next tile's first loads refill ring slots that the last blocks
      // (and a deferred GEMM-II) read
      __syncthreads();
    }
  }
}

template <int DK, int DV, int DT, bool CAUSAL, int WAVES>
hipError_t launch_instance(const KParams& kp, hipStream_t stream) {
  auto kern = attn_fwd_kernel<DK, DV, DT, CAUSAL, WAVES>;
  constexpr size_t lds = lds_bytes<DK, DV, DT, WAVES>();
  static_assert(lds * wgs_per_cu<DK, WAVES>() <= 160 * 1024, "the workgroups of a CU fit its LDS");
  // The dynamic LDS limit is a per-device attribute of the kernel: raise it
  // once on each device this instance runs on (bit d of `ready`: device d;
  // devices past 63 set it on every call).  Concurrent first calls may both
  // set it, which is harmless.
  static std::atomic<uint64_t> ready{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? 1ull << dev : 0;
  if (!bit || !(ready.load(std::memory_order_acquire) & bit)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    ready.fetch_or(bit, std::memory_order_release);
  }
  // 16-bit inputs: persistent workgroups, as many as the CUs hold at once,
  // rounded down to a multiple of the XCD count so that tile t still runs on
  // XCD t % 8 (the dispatcher deals workgroup w to XCD w % 8)
  int grid = kp.total;
  if (!Ops<DT>::kFp8) {
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const int resident = cus * wgs_per_cu<DK, WAVES>() / kXcds * kXcds;
    if (resident >= kXcds && resident < grid) grid = resident;
  }
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * WAVES), lds, stream, kp);
  return hipGetLastError();
}

template <int DK, int DV, int DT, int WAVES>
hipError_t launch_masks(const KParams& kp, bool causal, hipStream_t stream) {
  return causal ? launch_instance<DK, DV, DT, true, WAVES>(kp, stream)
                : launch_instance<DK, DV, DT, false, WAVES>(kp, stream);
}

template <int DK, int DV, int DT>
hipError_t launch_waves(const KParams& kp, bool causal, int waves, hipStream_t stream) {
  return waves == 4 ? launch_masks<DK, DV, DT, 4>(kp, causal, stream)
                    : launch_masks<DK, DV, DT, 8>(kp, causal, stream);
}

}  // namespace

hipError_t launch_attn_fwd(const AttnArgs& a, hipStream_t stream) {
  // Workgroup size.  Eight waves (256 query rows, one workgroup per CU) keep
  // K/V tiles in LDS for the most rows; four waves (128 rows, two or three
  // workgroups per CU) let one workgroup's prologue and epilogue run beside
  // another's key loop.  That wins where workgroups are short (N <= 2048;
  // FP8, whose four-wave workgroups keep four-block rings: N <= 4096), and
  // where the 256-row workgroups, dealt out in rounds over the CUs, would
  // keep them under 80% busy (a lone four-wave workgroup in the last round
  // uses its CU better than an idle CU does).  Both give the same bytes: a
  // query row's arithmetic does not depend on its tile.  The [B][N][H][d]
  // layout and 192-wide keys run eight waves only.
  int waves = 8;
  if (a.layout == 0 && a.d != 192) {
    if (a.tile_rows == 128) {
      waves = 4;
    } else if (a.tile_rows == 0) {
      const long long nq8 = (a.N + 255) / 256;
      const long long wg8 = (a.causal ? (nq8 + 1) / 2 : nq8) * a.B * a.H;
      int dev = 0, cus = 0;
      const bool have_cus =
          hipGetDevice(&dev) == hipSuccess &&
          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
          cus > 0;
      // the 256-row grid's work as a share of its rounds over the CUs
      const bool ragged =
          have_cus && 5 * wg8 < 4 * ((wg8 + cus - 1) / cus) * (long long)cus;
      // FP8 four-wave workgroups keep four-block rings and stay ahead longer
      if (a.N <= (a.dtype == 2 ? 4096 : 2048) || ragged) waves = 4;
    }
  }
  const int bm = 32 * waves;

  KParams kp;
  kp.q = static_cast<const uint8_t*>(a.q);
  kp.k = static_cast<const uint8_t*>(a.k);
  kp.v = static_cast<const uint8_t*>(a.v);
  kp.o = a.o;
  kp.lse = a.lse;
  kp.N = a.N;
  kp.H = a.H;
  kp.Hkv = a.Hkv;
  kp.group = a.H / a.Hkv;
  kp.nq = (a.N + bm - 1) / bm;
  kp.wg_per_head = a.causal ? (kp.nq + 1) / 2 : kp.nq;
  kp.total = kp.wg_per_head * a.B * a.H;
  kp.c = a.c;
  kp.vscale = a.vscale;
  kp.qmode = a.qmode;
  kp.layout = a.layout;
  // head dimensions (d_qk, d_v): 64/64, 128/128, 192/128; FP8: 128/128
  const bool causal = a.causal != 0;
  if (a.dtype == 2) return launch_waves<128, 128, 2>(kp, causal, waves, stream);
  if (a.d == 64) {
    return a.dtype == 0 ? launch_waves<64, 64, 0>(kp, causal, waves, stream)
                        : launch_waves<64, 64, 1>(kp, causal, waves, stream);
  }
  if (a.d == 128) {
    return a.dtype == 0 ? launch_waves<128, 128, 0>(kp, causal, waves, stream)
                        : launch_waves<128, 128, 1>(kp, causal, waves, stream);
  }
  if (a.d == 192) {
    return a.dtype == 0 ? launch_masks<192, 128, 0, 8>(kp, causal, stream)
                        : launch_masks<192, 128, 1, 8>(kp, causal, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace qm

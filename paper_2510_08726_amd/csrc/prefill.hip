// Fused attention prefill for gfx950: the loop nest that rolling update
// (Section "Rolling Update", Algorithm 1, Eq. fixed-recurrent) produces from
// the plain attention definition, with the tile structure of the appendix
// "Privatization" (a local max per key tile, then the running max).
//
// Work split.  One workgroup = 4 wave64s, one per SIMD, each owning 32 query
// rows of one query head for the whole key loop: 128 rows of one (batch,
// query head), or, when several query heads share a KV head (GQA), the same
// 128 / hg rows of hg such heads, so that every wave sees the same keys (no
// wave idles while the others finish their causal diagonal) and all of them
// read the same K and V tiles.  Two such workgroups share each compute unit
// (two waves per SIMD): they run independently, so one's barrier waits,
// per-item setup and output overlap the other's key loop.  Key tiles are
// BN = 32 keys.  Every wave runs the whole loop body for its rows,
// software-pipelined over three tiles: iteration j
//
//   S^T(j+1) = K_{j+1} . Q^T          8 (D = 128) 32x32x16 MFMAs, K from LDS,
//                                      Q in AGPRs
//   P(j) = exp2(S(j) - m)              VALU, against the row's reference max
//                                      m, rounded to the input type (the
//                                      compute definition casts exp to the
//                                      input dtype before the second matmul)
//   O^T = a O^T + V_{j-1}^T . P(j-1)^T 8 MFMAs, V from LDS, O^T in AGPRs,
//   l = a l + rowsum P(j-1)            row sums by 4x4x4 MFMAs
//
// with the two kinds of MFMA alternating slot by slot and the softmax steps
// of tile j spread over the same slots from the third on, so that the VALU work of a wave
// issues while its own MFMAs run (within one wave the matrix unit and the
// VALU overlap almost completely; across the two waves of a SIMD the same
// mix overlaps far less).  The factor a = exp2(m - m') is applied only when
// a row's tile max exceeds m by more than the lazy threshold.
//
// Computing S transposed puts one query row per lane pair (rows are the
// MFMA N index): row reductions stay in registers, the rescale of O^T is a
// per-lane scale, and the fp32 S^T accumulator converts in place into the
// layout of the B operand of the P.V product.  V stays row-major in LDS; its
// operand is gathered with the gfx950 transposing LDS read, in the key order
// in which the S^T accumulator holds keys.
//
// The K and V tiles of the workgroup pass through LDS rings of kRing slots,
// filled by buffer loads with the LDS bit (HBM -> LDS without VGPRs) that all
// waves issue in the P.V slots, kRing - 1 tiles ahead of their use, through
// one buffer resource per head and work item; one barrier per iteration
// publishes them.  Between work items each wave borrows one ring slot that
// the next item's first copies leave free: its O rows go out and its next
// Q rows come in through it, as whole 1 KB blocks.
//
// The MFMAs are written as inline assembly to fix their register files: the
// S^T accumulators in VGPRs (the softmax reads them), Q, O^T and l in fixed
// AGPRs.  The compiler does not model the latency of those instructions;
// explicit s_nop padding covers it, and a test checks the generated code.
//
// Lazy rescale.  The reference max used in the exponent is only moved when a
// row's tile max exceeds it by more than 8 (log2 units); until then every
// P <= 2^8 (well inside the fp16 / bf16 range) and the O^T rescale is
// skipped.  The state is the same as with an always moving max, written
// relative to another reference point; the final division by l cancels it.
//
// Scores are in log2 units: t = s * scale * log2(e) (+ ALiBi bias * log2(e)),
// so each exponential is one v_exp_f32.  With ALiBi at D = 64 the key part of
// the bias starts the S^T accumulator, so that preparing a score is one FMA.

#include <algorithm>
#include <atomic>
#include <type_traits>
#include <utility>

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kWgPerCu = 2;                 // resident workgroups per compute unit
constexpr int BMW = 32;                     // query rows per wave
constexpr int BM = BMW * kWaves;            // query rows per workgroup of one head
constexpr int BN = 32;                      // keys per tile
constexpr int kRing = 4;                    // LDS slots per operand; copies run kRing - 1 tiles ahead
static_assert(kRing >= 4, "the first V tiles are staged before the item, the rest copied kRing - 2 ahead");
// The key loop is unrolled so that ring slots and the parity of the score
// buffers are compile-time choices.
constexpr int kUnroll = kRing % 2 == 0 ? kRing : 2 * kRing;
// A row's reference maximum moves only when a tile's maximum exceeds it by
// more than this (log2 units), so that P <= 2^kLazyThreshold.
constexpr float kLazyThreshold = 8.f;
// Reference max (times c) before the first visible key: finite, so the first
// visible tile takes the slow path like any other move.
constexpr float kMcInit = -1e30f;
// Accelerator dies (XCDs), each with its own L2; consecutive workgroups of a
// launch are dealt to them in turn.
constexpr int kXcds = 8;

__device__ __forceinline__ float as_f(unsigned u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ unsigned as_u(float f) { return __builtin_bit_cast(unsigned, f); }

// A row's values are split over lanes l and l ^ 32: combine them.
// permlane32_swap(x, x) returns the upper half's value in the lower half and
// the other way round.
__device__ __forceinline__ float max_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(as_u(x), as_u(x), false, false);
  return fmaxf(as_f((unsigned)r[0]), as_f((unsigned)r[1]));
}

__device__ __forceinline__ float sum_halves(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(as_u(x), as_u(x), false, false);
  return as_f((unsigned)r[0]) + as_f((unsigned)r[1]);
}

// Empty volatile asm that uses and redefines x: keeps the computation of x in
// the MFMA slot where it is written (the compiler would otherwise sink the
// softmax arithmetic towards its first use in a later slot or iteration).
template <typename V>
__device__ __forceinline__ void pin(V& x) {
  asm volatile("" : "+v"(x));
}

// Marks x as used here (no instruction).
__device__ __forceinline__ void keep_live(const f32x16& x) {
  asm volatile("" : : "v"(x));
}

__device__ __forceinline__ void hazard_pad() {
  // 32 wait states: more than any gfx950 MFMA result latency.
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// This file is compiled once per (head dim, element type) shard, selected by
// ATTN_PREFILL_SHARD (0, 1: D = 128; 2, 3: D = 64), so the instantiations
// build in parallel and each shard gets the register split of its head dim.
#ifndef ATTN_PREFILL_SHARD
#define ATTN_PREFILL_SHARD 0
#endif
constexpr int kShardD = ATTN_PREFILL_SHARD >= 2 ? 64 : 128;

// Register files.  The S^T accumulators, P and the LDS operands are ordinary
// values in VGPRs, allocated by the compiler.  The operands that live through
// the whole key loop are in fixed AGPRs that only the inline assembly below
// names: O^T block db in a[16 db .. + 15] (D / 2 registers), Q fragment kx in
// a[kQAgpr + 4 kx .. + 3] (D / 4), l in a[kLAgpr .. + 3], the ones in
// a[kOnesAgpr .. + 1]: 102 AGPRs for D = 128, 54 for D = 64.  The build sets
// each kernel's AGPR allocation to that count rounded up to 4 (104 or 56),
// which leaves 152 or 200 of a wave's 256 registers (two waves per SIMD) to
// the VGPRs.  Every statement that touches the fixed AGPRs lists all of them
// as clobbered, so the compiler keeps none of its own values there, and
// counts them as used.
#define ATTN_A10(p) "a" #p "0", "a" #p "1", "a" #p "2", "a" #p "3", "a" #p "4", \
                    "a" #p "5", "a" #p "6", "a" #p "7", "a" #p "8", "a" #p "9"
#if ATTN_PREFILL_SHARD >= 2
#define ATTN_AGPRS "a0", "a1", "a2", "a3", "a4", "a5", "a6", "a7", "a8", "a9", \
    ATTN_A10(1), ATTN_A10(2), ATTN_A10(3), ATTN_A10(4), "a50", "a51", "a52", "a53"
#else
#define ATTN_AGPRS "a0", "a1", "a2", "a3", "a4", "a5", "a6", "a7", "a8", "a9", \
    ATTN_A10(1), ATTN_A10(2), ATTN_A10(3), ATTN_A10(4), ATTN_A10(5), ATTN_A10(6), ATTN_A10(7), ATTN_A10(8), ATTN_A10(9), \
    "a100", "a101"
#endif
constexpr int kOAgpr = 0;
constexpr int kQAgpr = kOAgpr + kShardD / 2;
constexpr int kLAgpr = kQAgpr + kShardD / 4;    // exp-sum accumulator
constexpr int kOnesAgpr = kLAgpr + 4;           // two registers holding (1.0, 1.0)
constexpr int kAgprAlloc = (kOnesAgpr + 2 + 3) / 4 * 4;
constexpr int kVgprBudget = 256 - kAgprAlloc;
static_assert(kOnesAgpr + 2 == (kShardD == 64 ? 54 : 102), "the clobber list names every fixed AGPR");

// 32x32x16 MFMAs.  qk0/qk: S^T accumulator in VGPRs (qk0 starts from zero,
// qk0c from the accumulator c), K
// operand in VGPRs, Q operand from AGPRs a[QA .. QA + 3]; with PAD, two wait
// states first, for an operand that the compiler reloads (VALU) just before.  pv: O^T accumulator
// a[OA .. OA + 15], both operands in VGPRs.  rowsum: a 4x4x4 MFMA with the
// all-ones operand, which adds the four 16-bit values each lane holds in b to
// every register of its accumulator a[LA .. LA + 3]: the exp-sum l is
// accumulated from the same rounded weights that multiply V, on the matrix
// unit.  Its b was packed an iteration earlier; the wait-state check of the
// generated code confirms that no VALU write of b comes within two states.
template <typename T> struct Mma;
template <> struct Mma<_Float16> {
  typedef f16x8 v8;
  template <int QA, bool PAD> static __device__ __forceinline__ void qk0(f32x16& d, v8 a) {
    if constexpr (PAD)
      asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], 0" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
    else
      asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], 0" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int QA, bool PAD> static __device__ __forceinline__ void qk(f32x16& d, v8 a) {
    if constexpr (PAD)
      asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], %0" : "+v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
    else
      asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], %0" : "+v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int QA, bool PAD> static __device__ __forceinline__ void qk0c(f32x16& d, v8 a, const f32x16& c) {
    if constexpr (PAD)
      asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], %4" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3), "v"(c) : ATTN_AGPRS);
    else
      asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], %4" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3), "v"(c) : ATTN_AGPRS);
  }
  template <int OA> static __device__ __forceinline__ void pv(v8 a, v8 b) {
    asm volatile("v_mfma_f32_32x32x16_f16 a[%2:%3], %0, %1, a[%2:%3]" : : "v"(a), "v"(b), "n"(OA), "n"(OA + 15) : ATTN_AGPRS);
  }
  static constexpr uint32_t kOnes = 0x3c003c00u;   // (1.0, 1.0)
  template <int LA> static __device__ __forceinline__ void rowsum(uint2 b) {
    asm volatile("v_mfma_f32_4x4x4_16b_f16 a[%1:%2], a[%3:%4], %0, a[%1:%2]"
                 : : "v"(b), "n"(LA), "n"(LA + 3), "n"(kOnesAgpr), "n"(kOnesAgpr + 1) : ATTN_AGPRS);
  }
  // Clear 16 (zero16) or 4 (zero4) AGPRs: an MFMA with zero operands and C = 0
  // (two wait states first: the zero operand is written just before).
  template <int A> static __device__ __forceinline__ void zero16(v8 z) {
    asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_f16 a[%1:%2], %0, %0, 0" : : "v"(z), "n"(A), "n"(A + 15) : ATTN_AGPRS);
  }
  template <int A> static __device__ __forceinline__ void zero4(uint2 z) {
    asm volatile("s_nop 1\n\tv_mfma_f32_4x4x4_16b_f16 a[%1:%2], %0, %0, 0" : : "v"(z), "n"(A), "n"(A + 3) : ATTN_AGPRS);
  }
};
template <> struct Mma<__bf16> {
  typedef bf16x8 v8;
  template <int QA, bool PAD> static __device__ __forceinline__ void qk0(f32x16& d, v8 a) {
    if constexpr (PAD)
      asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], 0" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
    else
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], 0" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int QA, bool PAD> static __device__ __forceinline__ void qk(f32x16& d, v8 a) {
    if constexpr (PAD)
      asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], %0" : "+v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
    else
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], %0" : "+v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int QA, bool PAD> static __device__ __forceinline__ void qk0c(f32x16& d, v8 a, const f32x16& c) {
    if constexpr (PAD)
      asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], %4" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3), "v"(c) : ATTN_AGPRS);
    else
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], %4" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3), "v"(c) : ATTN_AGPRS);
  }
  template <int OA> static __device__ __forceinline__ void pv(v8 a, v8 b) {
    asm volatile("v_mfma_f32_32x32x16_bf16 a[%2:%3], %0, %1, a[%2:%3]" : : "v"(a), "v"(b), "n"(OA), "n"(OA + 15) : ATTN_AGPRS);
  }
  static constexpr uint32_t kOnes = 0x3f803f80u;   // (1.0, 1.0)
  template <int LA> static __device__ __forceinline__ void rowsum(uint2 b) {
    asm volatile("v_mfma_f32_4x4x4_16b_bf16 a[%1:%2], a[%3:%4], %0, a[%1:%2]"
                 : : "v"(b), "n"(LA), "n"(LA + 3), "n"(kOnesAgpr), "n"(kOnesAgpr + 1) : ATTN_AGPRS);
  }
  // Clear 16 (zero16) or 4 (zero4) AGPRs: an MFMA with zero operands and C = 0
  // (two wait states first: the zero operand is written just before).
  template <int A> static __device__ __forceinline__ void zero16(v8 z) {
    asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 a[%1:%2], %0, %0, 0" : : "v"(z), "n"(A), "n"(A + 15) : ATTN_AGPRS);
  }
  template <int A> static __device__ __forceinline__ void zero4(uint2 z) {
    asm volatile("s_nop 1\n\tv_mfma_f32_4x4x4_16b_bf16 a[%1:%2], %0, %0, 0" : : "v"(z), "n"(A), "n"(A + 3) : ATTN_AGPRS);
  }
};

template <int I>
__device__ __forceinline__ void agpr_write(uint32_t v) {
  asm volatile("v_accvgpr_write_b32 a[%1], %0" : : "v"(v), "n"(I) : ATTN_AGPRS);
}
template <int I>
__device__ __forceinline__ void agpr_zero() {
  asm volatile("v_accvgpr_write_b32 a[%0], 0" : : "n"(I) : ATTN_AGPRS);
}
template <int I>
__device__ __forceinline__ float agpr_read() {
  float x;
  asm volatile("v_accvgpr_read_b32 %0, a[%1]" : "=v"(x) : "n"(I));
  return x;
}
template <int I>
__device__ __forceinline__ void agpr_scale(float s) {
  float t;
  asm volatile("v_accvgpr_read_b32 %0, a[%1]\n\tv_mul_f32 %0, %0, %2\n\tv_accvgpr_write_b32 a[%1], %0"
               : "=&v"(t) : "n"(I), "v"(s) : ATTN_AGPRS);
}

template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  [&]<int... Is>(std::integer_sequence<int, Is...>) { (f(std::integral_constant<int, Is>{}), ...); }(
      std::make_integer_sequence<int, N>{});
}

// The softmax of one tile (16 scores per lane) as a list of steps (weights
// are their VALU cost in issue cycles, used to spread the steps over the MFMA
// slots of an iteration):
//   prep   4 steps (ALiBi or masked tiles): bias and mask of 4 keys
//   exp    8 steps: 2 exponentials and their packing
//   max    4 steps: 4 scores folded into this lane's partial max
// (the exp-sum is accumulated by rowsum MFMAs beside P.V).
template <bool PREP, bool MASKED, bool ALIBI, bool CAP, bool ACCB = false>
struct SoftPlan {
  // Steps [0, MAX0) prepare the scores, four registers a step; then come 8
  // exponential steps (two registers each) and 4 steps of the lane's running
  // maximum (four registers each), as exp, exp, max.
  static constexpr int MAX0 = PREP ? 4 : 0;
  static constexpr int NSTEP = MAX0 + 12;
  static constexpr bool is_exp(int k) { return k >= MAX0 && (k - MAX0) % 3 != 2; }
  static constexpr int exp_index(int k) { return 2 * ((k - MAX0) / 3) + (k - MAX0) % 3; }
  static constexpr int max_index(int k) { return (k - MAX0) / 3; }
  static constexpr int weight(int k) {
    if (k < MAX0) return (ALIBI ? (ACCB ? 4 : 8) : 0) + (MASKED ? 8 : 0) + (CAP ? 52 : 0);
    return is_exp(k) ? 26 : 10;
  }
  // First step of slot s when the steps are spread over ns slots.
  static constexpr int begin(int s, int ns) {
    if (s <= 0) return 0;
    if (s >= ns) return NSTEP;
    int total = 0;
    for (int k = 0; k < NSTEP; ++k) total += weight(k);
    const int target = total * s / ns;
    int cum = 0, k = 0;
    while (k < NSTEP && cum < target) cum += weight(k++);
    return k;
  }
};

template <int D, typename T, bool CAUSAL, bool ALIBI, bool CAP, bool WIN>
struct Prefill {
  // Scores are prepared in log2 units (the scale folded in) whenever a bias
  // or the cap has to act on the scaled value.
  static constexpr bool LOG2 = ALIBI || CAP;
  // ALiBi at D = 64: the key-dependent part of the bias starts the S^T
  // accumulator (kb, per work item), so preparing a score takes one FMA with
  // the tile's per-row base instead of computing the bias first.  (At
  // D = 128 the 16 registers of kb do not fit.)
  static constexpr bool ACCB = ALIBI && D == 64;
  typedef Elem<T> E;
  typedef Mma<T> M;
  typedef typename E::vec8 vec8;
  static constexpr int KX = D / 16;                        // MFMA K-steps of Q.K^T
  static constexpr int DB = D / 32;                        // 32-dim blocks of O^T
  static constexpr int TE = BN * D;                        // elements of one K or V tile
  static constexpr int NB = TE * (int)sizeof(T) / 1024;    // 1 KB copy blocks per tile
  static constexpr int CPW = 2 * NB / kWaves;              // copies per wave per iteration (K and V)
  static constexpr int CPR = D / 8;                        // 16-byte chunks per row
  static constexpr int NG = KX;                            // K (or V) operand fragments per tile
  static constexpr int NS = 2 * NG;                        // MFMA slots per iteration
  static_assert(NG == 2 * DB, "as many V fragments as K fragments");
  static_assert(CPW >= 1 && 2 * NB == CPW * kWaves, "the copies of a tile divide evenly over the waves");
  // K and V operand fragments read ahead of their MFMA (one K fragment is two
  // MFMA slots).  At D = 128 the VGPR budget allows one K fragment ahead and,
  // with ALiBi or SoftCap (more live state), one V fragment; deeper rings
  // push the per-item code into scratch.  At D = 64 the smaller AGPR share
  // leaves room for three of each.
  static constexpr int PFD_K = D == 64 && !ACCB ? 3 : 1;
  static constexpr int PFD_V = (LOG2 || WIN) ? 1 : 3;
  template <bool IS_K> static constexpr int pfd() { return IS_K ? PFD_K : PFD_V; }
  static_assert(NG % (PFD_K + 1) == 0 && NG % (PFD_V + 1) == 0, "fragment ring positions must repeat every iteration");
  static_assert(kOAgpr + 16 * DB <= kQAgpr && kQAgpr + 4 * KX <= kLAgpr, "AGPR map");

  // S^T accumulator of one tile: register r of lane (n, hh) is key
  // 8 (r / 4) + 4 hh + r % 4 of row n.
  typedef f32x16 Scores;
  // P^T as the B operand of P.V: w[c][..] = keys of 16-key slice c.
  struct Probs {
    uint32_t w[2][4];
  };
  struct State {
    float mc;     // reference max of the row, times ce (log2 units)
    float alpha;  // rescale factor of O^T and l set by the slow path
  };
  static constexpr int oagpr(int db) { return kOAgpr + 16 * db; }
  static constexpr int qagpr(int kx) { return kQAgpr + 4 * kx; }
  // Per-lane LDS byte offsets inside a tile: K fragment kx, V fragment
  // (c16, db); c16 only adds an immediate.
  struct Addr {
    int k[KX];
    int v[DB][2];
  };
  struct TileArgs {
    float c;      // scale * log2(e) (with ALiBi or SoftCap) or max(|scale| * log2(e), tiny)
    float k2, cl; // SoftCap: 2 c / cap (c folded in) and cap * log2(e)
    float sl2;    // ALiBi slope * log2(e)
    float abase;  // ALiBi bias of key j0 + 4 hh relative to the wave's first row
    float mb;     // (ALiBi bias base, or SoftCap cl) minus the row's reference max
    f32x16 kb;    // ACCB: slope * log2(e) * kconst(r) / c, the start of each S^T accumulator
    int lim;      // last visible key offset (key - j0 - 4 hh) of this lane's row
    int llo;      // first visible key offset of this lane's row (sliding window)
    float t;      // this lane's maximum score of the tile
  };

  // HBM -> LDS copy of 1 KB block `blk` of tile t (rows t BN .. t BN + BN -
  // 1) of one head (base) into the LDS slot at byte address `slot`; dof is
  // the lane's byte offset within the tile.  The buffer range ends at row
  // `rows` or at the tile's end, whichever comes first, so rows past it read
  // as zero, and a tile past it (or a negative one) has an empty range and
  // writes zeros.  The tile offset lives in the (scalar) buffer base.  Used
  // for the Q rows of a work item; K and V go through copy_tile.  Issued as
  // inline assembly: the compiler then adds no waits of its own for the LDS
  // writes; the kernel waits for them explicitly before its barriers.
  static __device__ __forceinline__ void copy_block(const T* base, int rows, uint32_t slot, int t, int blk, int dof) {
    const int left = t >= 0 ? max(rows - t * BN, 0) : 0;
    const uint64_t a = reinterpret_cast<uint64_t>(base + (left > 0 ? (size_t)t * TE : 0));
    // The words are uniform; readfirstlane keeps them in SGPRs even where the
    // compiler computes the 64-bit address with vector instructions.
    const u32x4 rsrc = {(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                        (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
                        (uint32_t)__builtin_amdgcn_readfirstlane(min(left, BN) * D * (int)sizeof(T)), 0x00020000u};
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 : : "s"(slot + (uint32_t)(blk * 1024)), "v"(dof), "s"(rsrc) : "memory", "m0");
  }
  // The buffer resource of one head's K or V for a work item: base = the
  // head's first row, range = the item's staged rows (`rows`, in bytes).
  static __device__ __forceinline__ u32x4 head_rsrc(const T* base, int rows) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    return u32x4{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
                 (uint32_t)__builtin_amdgcn_readfirstlane(rows * D * (int)sizeof(T)), 0x00020000u};
  }
  // The same copy as copy_block through a head's resource: the tile offset
  // goes into the lane offset, which the buffer range check covers, so rows
  // past the range, tiles past it and negative tiles (whose offsets wrap to
  // above 2^31) read as zero.  Per copy, one VALU add and the m0 write; the
  // host keeps Lk * D * sizeof(T) below 2^31.
  static __device__ __forceinline__ void copy_tile(const u32x4& rs, uint32_t slot, int t, int blk, int dof) {
    // The tile's byte offset passes through an opaque scalar copy, so that
    // the add happens here rather than being hoisted out of the unrolled
    // loop into a register per copy.
    int tb = __builtin_amdgcn_readfirstlane(t * (TE * (int)sizeof(T)));
    asm volatile("" : "+s"(tb));
    const int off = dof + tb;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 : : "s"(slot + (uint32_t)(blk * 1024)), "v"(off), "s"(rs) : "memory", "m0");
  }
  // Copy u of a wave moves a block of the K tile (else of the V tile).
  static __device__ __forceinline__ bool copies_k(int u, int wave) {
    return NB >= kWaves ? u * kWaves < NB : wave < NB;
  }
  // MFMA slot of an iteration at which copy u is issued: spread over the
  // iteration, so that the copies' issue overlaps the matrix unit, in odd
  // (P.V) slots, beside an MFMA whose operands are already in registers
  // (measured: ALiBi at D = 64 2.6 % faster than in the even slots).
  static constexpr int copy_slot(int u) { return 3 + u * (NS / CPW); }

  static __device__ __forceinline__ void make_addr(Addr& ad, int lane) {
    {
      const int n = lane & 31, hh = lane >> 5;
#pragma unroll
      for (int kx = 0; kx < KX; ++kx) ad.k[kx] = 2 * (n * D + 8 * ((2 * kx + hh) ^ swz<D>(n)));
    }
    const int G = lane >> 4, i = lane & 15;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int lh = 0; lh < 2; ++lh) {
        const int d = 32 * db + 16 * (G & 1) + 4 * (i & 3);   // this source lane's 4 head dims
        const int k = 4 * (G >> 1) + (i >> 2) + 8 * lh;        // this source lane's key in the slice
        ad.v[db][lh] = 2 * (k * D + 8 * ((d >> 3) ^ swz<D>(k)) + (d & 7));
      }
  }

  // K operand kx: lane (n, hh) reads key n, head dims 16 kx + 8 hh .. + 7.
  static __device__ __forceinline__ vec8 kfrag(const T* tile, const Addr& ad, int kx) {
    return __builtin_bit_cast(vec8, *reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(tile) + ad.k[kx]));
  }

  // V^T operand g (head dims 32 db + m, 16-key slice c16, g = c16 DB + db):
  // lane (m, half hh) receives keys 16 c16 + 4 hh + 0..3 and 16 c16 + 8 + 4 hh
  // + 0..3, the order in which the S^T accumulator holds keys in the B operand.
  static __device__ __forceinline__ vec8 vfrag(const T* tile, const Addr& ad, int g) {
    const char* base = reinterpret_cast<const char*>(tile) + (g / DB) * 32 * D;
    const uint2 lo = lds_read_tr(base + ad.v[g % DB][0]);
    const uint2 hi = lds_read_tr(base + ad.v[g % DB][1]);
    return __builtin_bit_cast(vec8, make_uint4(lo.x, lo.y, hi.x, hi.y));
  }

  static __device__ __forceinline__ vec8 probs_b(const Probs& pr, int c16) {
    return __builtin_bit_cast(vec8, make_uint4(pr.w[c16][0], pr.w[c16][1], pr.w[c16][2], pr.w[c16][3]));
  }

  static constexpr int kconst(int r) { return 8 * (r / 4) + (r % 4); }

  // Softmax step K of a tile (see SoftPlan).  Without ALiBi the exponent is
  // s * c - m * c.  With ALiBi the score is first made s * c + bias in log2
  // units; the bias is written relative to the wave's first row,
  // -slope (i - j) = slope (j - iw - off) - slope (i - iw), and the last term
  // is dropped: it shifts a whole row by a constant, which the row's softmax
  // does not see.  Masked tiles set keys past Lk and (causal) keys after the
  // row to -inf before the max.
  //
  // REL (whole tiles of ALiBi or SoftCap kernels after a wave's first tile,
  // when every row has a finite reference): the reference max is folded into
  // the additive term of the bias or cap, so the prepared value is already
  // the exponent, s c + bias - m (or the capped score - m), and the maximum
  // and the lazy check work relative to m.
  template <int K, bool PREP, bool MASKED, bool REL>
  static __device__ __forceinline__ void soft_step(State& st, Scores& sc, Probs& pr, TileArgs& ta) {
    typedef SoftPlan<PREP, MASKED, ALIBI, CAP, ACCB> P;
    const float ce = LOG2 ? 1.f : ta.c;
    static_assert(!REL || (LOG2 && !MASKED), "the relative form is for whole tiles with a bias or cap");
    if constexpr (K < P::MAX0) {
      constexpr int r0 = 4 * K;
      // Registers r0 .. r0 + 3 hold keys kconst(r0) + 0..3: their biases are
      // the bias of the first plus 0..3 slopes.
      [[maybe_unused]] float b[4] = {0.f, 0.f, 0.f, 0.f};
      if constexpr (ALIBI && ACCB) {
        // sc already holds s + kb = s + slope log2(e) kconst(r) / c.
        const float base = REL ? ta.mb : ta.abase;
        b[0] = b[1] = b[2] = b[3] = base;
      } else if constexpr (ALIBI) {
        const float base = REL ? ta.mb : ta.abase;
        b[0] = r0 == 0 ? base : __builtin_fmaf(ta.sl2, (float)kconst(r0), base);
        b[1] = b[0] + ta.sl2;
        b[2] = __builtin_fmaf(ta.sl2, 2.f, b[0]);
        b[3] = __builtin_fmaf(ta.sl2, 2.f, b[1]);
      }
#pragma unroll
      for (int r = r0; r < r0 + 4; ++r) {
        if constexpr (CAP) {
          const float x = soft_cap(sc[r], ta.k2, ta.cl, REL && !ALIBI ? ta.mb : ta.cl);
          sc[r] = ALIBI ? x + b[r - r0] : x;
        } else if constexpr (ALIBI) {
          sc[r] = __builtin_fmaf(sc[r], ta.c, b[r - r0]);
        }
        if constexpr (MASKED) {
          if (kconst(r) > ta.lim || (WIN && kconst(r) < ta.llo)) sc[r] = kNegInf;
        }
        float x = sc[r];
        pin(x);
        sc[r] = x;
      }
    } else if constexpr (P::is_exp(K)) {
      constexpr int r = 2 * P::exp_index(K);
      const float p0 = fast_exp2(REL ? sc[r] : __builtin_fmaf(sc[r], ce, -st.mc));
      const float p1 = fast_exp2(REL ? sc[r + 1] : __builtin_fmaf(sc[r + 1], ce, -st.mc));
      uint32_t w = E::pack2(p0, p1);
      pin(w);
      pr.w[r / 8][(r % 8) / 2] = w;
    } else {
      constexpr int q = P::max_index(K);
      // A running chain: two v_max3 a step (the tree of four and a fold
      // took one more).
      if constexpr (q == 0) ta.t = fmaxf(fmaxf(fmaxf(sc[0], sc[1]), sc[2]), sc[3]);
      else ta.t = fmaxf(fmaxf(fmaxf(fmaxf(ta.t, sc[4 * q]), sc[4 * q + 1]), sc[4 * q + 2]), sc[4 * q + 3]);
      pin(ta.t);
    }
  }

  // After the steps of a tile: does some score of this lane exceed the
  // reference maximum by more than the lazy threshold?  (Then the tile's P,
  // computed against the old reference, must be recomputed: see resolve.)
  template <bool REL>
  static __device__ __forceinline__ bool exceeds(const State& st, const TileArgs& ta) {
    const float ce = LOG2 ? 1.f : ta.c;
    return (REL ? ta.t : __builtin_fmaf(ta.t, ce, -st.mc)) > kLazyThreshold;
  }

  // Slow path of a tile whose maximum moved past the threshold in some row
  // of the wave (always the case for a row's first visible tile, whose
  // reference is still kMcInit): the row maximum is combined over the lane
  // pair holding the row, rows that moved take it as their new reference
  // and the factor 2^-(move) by which O^T and l are rescaled before this
  // tile's products are added (the products so far used the old reference),
  // and the tile's P is recomputed.  Rows that did not move keep their
  // reference and factor 1.
  template <bool REL>
  static __device__ __forceinline__ void resolve(State& st, Scores& sc, Probs& pr, TileArgs& ta) {
    typedef SoftPlan<false, false, ALIBI, CAP, ACCB> P;
    const float ce = LOG2 ? 1.f : ta.c;
    const float tm = max_halves(ta.t);
    const float d = REL ? tm : __builtin_fmaf(tm, ce, -st.mc);
    const bool move = d > kLazyThreshold;
    st.alpha = move ? fast_exp2(-d) : 1.f;
    if constexpr (REL) {
      // The prepared values are relative to the old reference: shift them to
      // the new one, then recompute the tile's weights.
      const float dd = move ? d : 0.f;
      st.mc += dd;
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[r] -= dd;
    } else {
      st.mc = move ? tm * ce : st.mc;
    }
    static_for<P::NSTEP>([&](auto kc) {
      constexpr int K = decltype(kc)::value;
      if constexpr (P::is_exp(K)) soft_step<K, false, false, REL>(st, sc, pr, ta);
    });
  }

  template <int B0, int B1, bool PREP, bool MASKED, bool REL>
  static __device__ __forceinline__ void soft_range(State& st, Scores& sc, Probs& pr, TileArgs& ta) {
    if constexpr (B1 > B0) {
      [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
        (soft_step<B0 + Ks, PREP, MASKED, REL>(st, sc, pr, ta), ...);
      }(std::make_integer_sequence<int, B1 - B0>{});
    }
  }

  // Operand fragment rings: fragment i of an iteration (K fragment kx = i for
  // S^T, V fragment g = i = c16 DB + db for P.V) lives in ring entry
  // i mod (pfd + 1) and is read pfd fragments ahead of its MFMA; the first
  // pfd fragments of an iteration are read at the end of the iteration before.
  template <bool IS_K> using Ring = vec8[pfd<IS_K>() + 1];
  // LDS instructions that read the first fragments of an iteration (one per
  // K fragment, two per V fragment): they stay in flight across the barrier.
  static constexpr int kPrime = PFD_K + 2 * PFD_V;

  template <bool IS_K, int I>
  static __device__ __forceinline__ void read_frag(Ring<IS_K>& fr, const T* tile, const Addr& ad) {
    if constexpr (IS_K) fr[I % (PFD_K + 1)] = kfrag(tile, ad, I);
    else fr[I % (PFD_V + 1)] = vfrag(tile, ad, I);
  }
  template <bool IS_K>
  static __device__ __forceinline__ void prime(Ring<IS_K>& fr, const T* tile, const Addr& ad) {
    static_for<pfd<IS_K>()>([&](auto ic) { read_frag<IS_K, decltype(ic)::value>(fr, tile, ad); });
  }

  // First softmax step of MFMA slot s (plan P): none in the first kSoftLag
  // slots, then the plan spread over the other NS - kSoftLag.
  static constexpr int kSoftLag = 2;
  static_assert(NS > kSoftLag, "slots left for the softmax steps");
  template <typename P>
  static constexpr int step_begin(int s) { return P::begin(s > kSoftLag ? s - kSoftLag : 0, NS - kSoftLag); }

  // Whole tiles after a wave's first one (SM 1 with P.V) take the relative
  // form in kernels with a bias or cap: every row of the wave has seen a key
  // by then (its own causal diagonal, or the whole first tile), so its
  // reference is finite.
  static constexpr bool rel(int SM, bool PV) { return LOG2 && SM == 1 && PV; }

  // The 2 NG MFMA slots of one iteration.  Slot 2 i: S^T MFMA with K fragment
  // i of tile j+1 (kl; QK), slot 2 i + 1: P.V MFMA with V fragment i of tile
  // j-1 (vl; PV) and P(j-1) (pp), plus the row-sum MFMAs of the same
  // weights; the softmax steps of tile j (SM: 0 none, 1 whole, 2 masked) on
  // sc / pc spread over the slots.  The fragments past the end of the
  // iteration come from the next iteration's tiles kln (K_{j+2}) and vln (V_j).
  template <bool QK, int SM, bool PV, typename CP>
  static __device__ __forceinline__ void slots(State& st, Scores& s_cur, Scores& s_next, Probs& p_cur,
                                               const Probs& p_prev, Ring<true>& fk, Ring<false>& fv, const T* kl,
                                               const T* kln, const T* vl, const T* vln, const Addr& ad,
                                               TileArgs& ta, CP&& copy) {
    constexpr bool MASKED = SM == 2;
    constexpr bool PREP = LOG2 || MASKED;
    constexpr bool REL = rel(SM, PV);
    typedef SoftPlan<PREP, MASKED, ALIBI, CAP, ACCB> P;
    // The softmax steps start kSoftLag slots into the iteration (the first
    // slots issue only MFMAs, copies and operand reads; measured 1-2 % faster
    // than starting at slot 0) and are spread over the remaining slots.
    // Every step of the tile runs inside these NS slots, before the
    // lazy-rescale check reads the lane maximum and before the next
    // iteration's P.V reads the packed weights: a step left past the last
    // slot would leave P words unwritten (uninitialised registers on the
    // first tiles of an item) and the lane maximum incomplete.
    static_assert(step_begin<P>(0) == 0 && step_begin<P>(NS) == P::NSTEP, "the steps cover the tile within the slots");
    [&]<int... Ss>(std::integer_sequence<int, Ss...>) {
      (
          [&] {
            constexpr int S = Ss;
            constexpr int i = S / 2;
            static_for<CPW>([&](auto uc) {
              if constexpr (copy_slot(decltype(uc)::value) == S) copy(uc);
            });
            if constexpr (S % 2 == 0) {
              if constexpr (QK) {
                constexpr int f = i + PFD_K;
                if constexpr (f < NG) read_frag<true, f>(fk, kl, ad);
                else read_frag<true, f - NG>(fk, kln, ad);
                // Without the causal mask the kernel has the register
                // pressure at which the compiler parks K operands in spare
                // AGPRs and reloads them right before their MFMA.
                if constexpr (i == 0 && ACCB) M::template qk0c<qagpr(i), !CAUSAL>(s_next, fk[i % (PFD_K + 1)], ta.kb);
                else if constexpr (i == 0) M::template qk0<qagpr(i), !CAUSAL>(s_next, fk[i % (PFD_K + 1)]);
                else M::template qk<qagpr(i), !CAUSAL>(s_next, fk[i % (PFD_K + 1)]);
              }
            } else {
              if constexpr (PV) {
                constexpr int f = i + PFD_V;
                if constexpr (f < NG) read_frag<false, f>(fv, vl, ad);
                else read_frag<false, f - NG>(fv, vln, ad);
                constexpr int c16 = i / DB, db = i % DB;
                M::template pv<oagpr(db)>(fv[i % (PFD_V + 1)], probs_b(p_prev, c16));
                // Exp-sum of the same weights: words 2 db, 2 db + 1 of the
                // slice, at fragments db = 0 and 1 (a large MFMA always
                // separates two rowsum MFMAs on one accumulator).
                if constexpr (db < 2)
                  M::template rowsum<kLAgpr>(make_uint2(p_prev.w[c16][2 * db], p_prev.w[c16][2 * db + 1]));
              }
            }
            if constexpr (SM != 0) soft_range<step_begin<P>(S), step_begin<P>(S + 1), PREP, MASKED, REL>(st, s_cur, p_cur, ta);
            __builtin_amdgcn_sched_barrier(0);
          }(),
          ...);
    }(std::make_integer_sequence<int, NS>{});
    // A variant without one kind of MFMA still leaves the next iteration's
    // first fragments of that kind in its ring.
    if constexpr (!QK) prime<true>(fk, kln, ad);
    if constexpr (!PV) prime<false>(fv, vln, ad);
  }

  // O^T *= alpha and l *= alpha, in place in the AGPRs.
  static __device__ __forceinline__ void repair(float alpha) {
    hazard_pad();
    static_for<DB * 16>([&](auto ic) { agpr_scale<kOAgpr + decltype(ic)::value>(alpha); });
    static_for<4>([&](auto ic) { agpr_scale<kLAgpr + decltype(ic)::value>(alpha); });
    hazard_pad();
  }
};

// Two waves per SIMD (two workgroups per compute unit) leave each wave 256
// registers: the fixed AGPRs named by the inline assembly and at most
// kVgprBudget VGPRs.  (By itself the compiler would halve the file once AGPRs
// are used; the build sets the kernels' AGPR allocation to kAgprAlloc in the
// device IR.)
template <int D, typename T, bool CAUSAL, bool ALIBI, bool CAP, bool WIN>
__global__ __launch_bounds__(kThreads, kWgPerCu) __attribute__((amdgpu_num_vgpr(kVgprBudget))) void prefill_kernel(PrefillParams p) {
  static_assert(D == kShardD, "one head dim per shard");
  typedef Prefill<D, T, CAUSAL, ALIBI, CAP, WIN> PF;
  constexpr bool REV = ALIBI;
  typedef typename PF::State State;
  typedef typename PF::Scores Scores;
  typedef typename PF::Probs Probs;
  typedef typename PF::Addr Addr;
  typedef typename PF::TileArgs TileArgs;
  constexpr int KX = PF::KX;
  constexpr int DB = PF::DB;
  constexpr int TE = PF::TE;
  constexpr int NB = PF::NB;
  constexpr int CPW = PF::CPW;
  constexpr int CPR = PF::CPR;
  // LDS: a ring of kRing K tiles and a ring of kRing V tiles (64 KB for
  // D = 128, so that two workgroups fit a compute unit).
  __shared__ __attribute__((aligned(1024))) T lds[2 * kRing * TE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31;
  const int hh = lane >> 5;

  // LDS byte addresses of the K and V slots.
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void*)lds;
  auto kslot = [&](int s) __attribute__((always_inline)) { return lds0 + (uint32_t)(s * TE * (int)sizeof(T)); };
  auto vslot = [&](int s) __attribute__((always_inline)) {
    return lds0 + (uint32_t)((kRing + s) * TE * (int)sizeof(T));
  };

  // This wave's share of every tile copy: copy u (u < CPW) moves 1 KB block
  // b = u kWaves + wave of the pair (K tile, V tile), K for b < NB.  In a
  // block the lane writes bytes 16 lane .. 16 lane + 15, i.e. chunk position
  // lane % CPR of row (block * 1024 / (2 D) + lane / CPR), and reads the
  // global chunk that the swizzle puts there.
  int dof[CPW];
#pragma unroll
  for (int u = 0; u < CPW; ++u) {
    const int blk = (u * kWaves + wave) % NB;
    const int r = blk * (1024 / (2 * D)) + lane / CPR;
    const int pos = lane % CPR;
    dof[u] = (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T);
  }

  // Persistent workgroups.  The work items (query block, group of hg query
  // heads) are numbered KV head first, then query block by decreasing key
  // count, then head group within the KV head's group, so that neighbouring
  // items read the same K and V.  Wave w takes head w mod hg of the group and
  // row block w / hg of the query block.  Workgroup g runs on XCD g mod kXcds (the order in
  // which the dispatcher hands out the first workgroups), and each XCD takes
  // one contiguous share of the items, so the concurrent readers of a K/V
  // tile share that XCD's L2.  Within an XCD, round r gives item r * Pl + c
  // to the c-th of its Pl workgroups on even rounds and r * Pl + Pl - 1 - c on
  // odd ones: heavy and light query blocks pair up, and with causal masking
  // (key counts falling linearly with the block index) every workgroup gets
  // the same number of key tiles.
  const int P = gridDim.x;
  const int wg = blockIdx.x;
  const int X = p.nxcd;
  const int xcd = wg % X, c = wg / X, Pl = P / X;
  const int s0 = (int)((long long)p.nitems * xcd / X);
  const int s1 = (int)((long long)p.nitems * (xcd + 1) / X);
  const int hg = p.hg;
  const int ngrp = p.group / hg;              // head groups per KV head
  const int bm = BMW * (kWaves / hg);         // query rows per work item
  const int per_kv = p.nqb * ngrp;
  const int Lq = p.Lq, Lk = p.Lk;
  const int off = Lk - Lq;

  // One work item: its query block and head, the key tiles [t0, t1) that the
  // workgroup stages (iteration j handles tile(j), j = 0 .. t1 - t0 - 1),
  // the iterations [f0, f1] in which this wave sees keys and [w0, w1) in
  // which no row of the wave masks any key of the tile.  rows: the staged
  // key rows end there (rows past it read as zero).
  struct Item {
    int qb, head, kvh, hq, iw, t0, t1, f0, f1, w0, w1, rows;
  };
  const int W = WIN ? p.window : 0;   // sliding window (keys per row)
  auto item_at = [&](int round, Item& it) __attribute__((always_inline)) {
    const int sl = round * Pl + ((round & 1) ? Pl - 1 - c : c);
    if (sl >= s1 - s0) return false;
    const int s = s0 + sl;
    it.kvh = s / per_kv;
    const int rem = s - it.kvh * per_kv;
    it.qb = p.nqb - 1 - rem / ngrp;
    it.head = it.kvh * p.group + (rem % ngrp) * hg + wave % hg;
    it.hq = it.head % p.Hq;
    const int i0 = it.qb * bm;
    it.iw = i0 + BMW * (wave / hg);
    // Row i sees keys [lo(i), hi(i)): hi(i) = i + off + 1 with the causal
    // mask, lo(i) = i + off + 1 - W with the window (clamped to [0, Lk]).
    auto hi = [&](int i) { return CAUSAL ? min(Lk, max(0, i + off + 1)) : Lk; };
    auto lo = [&](int i) { return WIN ? min(Lk, max(0, i + off + 1 - W)) : 0; };
    const int ilast = min(i0 + bm, Lq) - 1;               // the item's last row
    const int klo = lo(i0), khi = hi(ilast);
    it.t0 = klo / BN;
    it.t1 = khi > klo ? (khi + BN - 1) / BN : it.t0;
    it.rows = min(Lk, it.t1 * BN);
    // This wave's rows [iw, wlast]: visible tiles [a, b), whole tiles
    // [wl, wh) (every row sees every key of the tile).
    const int wlast = min(it.iw + BMW, Lq) - 1;
    int a = 0, b = 0, wl = 0, wh = 0;
    if (it.iw < Lq && hi(wlast) > lo(it.iw)) {
      a = lo(it.iw) / BN;
      b = (hi(wlast) + BN - 1) / BN;
      wl = (lo(wlast) + BN - 1) / BN;
      wh = hi(it.iw) / BN;
    }
    if (REV) {
      it.f0 = it.t1 - b;  it.f1 = it.t1 - 1 - a;
      it.w0 = it.t1 - wh; it.w1 = it.t1 - wl;
    } else {
      it.f0 = a - it.t0;  it.f1 = b - 1 - it.t0;
      it.w0 = wl - it.t0; it.w1 = wh - it.t0;
    }
    return true;
  };
  // Iteration j handles key tile tile(j).  With ALiBi the tiles are visited
  // from the last to the first: the bias grows with the key index, so the
  // first tile holds the largest bias of each row and the running maximum
  // rarely grows afterwards (each growth beyond the lazy threshold costs a
  // rescale of O^T).  Otherwise the keys run forward.
  auto tile_of = [&](const Item& it, int j) __attribute__((always_inline)) { return REV ? it.t1 - 1 - j : it.t0 + j; };

  Addr ad;
  PF::make_addr(ad, lane);

  // This wave's staging tile: Q rows in at the start of a work item, O rows
  // out at its end.  It is a ring slot that the first copies of a work item
  // (K slots 0 .. kRing-2, V slots 0 .. kRing-4, issued by stage_kv) leave
  // free: K slot kRing-1 for wave 0, V slot kRing-4+w for wave w >= 1.  The
  // ring takes it back in the item's first iterations, after the barrier
  // that follows the Q reads.
  static_assert(kWaves == 4, "three free V slots and one free K slot between work items");
  const int xs = wave == 0 ? kRing - 1 : kRing + kRing - 4 + wave;
  const T* xl = lds + xs * TE;
  const uint32_t xslot = lds0 + (uint32_t)(xs * TE * (int)sizeof(T));
  // The first tiles of a work item: K tiles 0 .. kRing-2 and V tiles
  // 0 .. kRing-4, each wave its blocks.  Issued once the previous item's last barrier has
  // passed (every ring slot is free then), before that item's output.
  auto stage_kv = [&](const Item& it) __attribute__((always_inline)) {
    const u32x4 rk = PF::head_rsrc(reinterpret_cast<const T*>(p.k) + (size_t)it.kvh * Lk * D, it.rows);
    const u32x4 rv = PF::head_rsrc(reinterpret_cast<const T*>(p.v) + (size_t)it.kvh * Lk * D, it.rows);
#pragma unroll
    for (int u = 0; u < CPW; ++u) {
      const int b = (u * kWaves + wave) % NB;
      if (PF::copies_k(u, wave)) {
#pragma unroll
        for (int t = 0; t < kRing - 1; ++t) PF::copy_tile(rk, kslot(t), tile_of(it, t), b, dof[u]);
      } else {
#pragma unroll
        for (int t = 0; t < kRing - 3; ++t) PF::copy_tile(rv, vslot(t), tile_of(it, t), b, dof[u]);
      }
    }
  };
  // The wave's 32 Q rows of a work item (rows past Lq read as zero) into its
  // staging tile, as whole 1 KB blocks; issued after the wave has read its
  // previous output out of that tile.  The lane index passes through an
  // opaque copy so that the block offsets are computed here.
  auto stage_q = [&](const Item& it) __attribute__((always_inline)) {
    int ln = lane;
    pin(ln);
    const T* qp = reinterpret_cast<const T*>(p.q) + ((size_t)it.head * Lq + it.iw) * D;
    const int qrows = max(min(Lq - it.iw, BMW), 0);
    static_for<NB>([&](auto bc) {
      constexpr int b = decltype(bc)::value;
      const int r = b * (1024 / (2 * D)) + ln / CPR;
      const int pos = ln % CPR;
      PF::copy_block(qp, qrows, xslot, 0, b, (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T));
    });
  };

  Item cur;
  if (!item_at(0, cur)) return;
  agpr_write<kOnesAgpr>(PF::M::kOnes);
  agpr_write<kOnesAgpr + 1>(PF::M::kOnes);
  stage_kv(cur);
  stage_q(cur);

  for (int round = 0;; ++round) {
    const int nt = cur.t1 - cur.t0;   // iterations with a tile
    const int iw = cur.iw;
    const int row = iw + n;           // this lane's query row
    const u32x4 rk = PF::head_rsrc(reinterpret_cast<const T*>(p.k) + (size_t)cur.kvh * Lk * D, cur.rows);
    const u32x4 rv = PF::head_rsrc(reinterpret_cast<const T*>(p.v) + (size_t)cur.kvh * Lk * D, cur.rows);
    auto tile = [&](int j) __attribute__((always_inline)) { return tile_of(cur, j); };
    // Copy u of this wave in iteration j: its block of K tile(j + kRing) into
    // K slot j mod kRing (whose tile j was last read in iteration j - 1), or
    // of V tile(j + kRing - 2) into V slot (j - 2) mod kRing (whose tile j - 2
    // was last read in iteration j - 1), anywhere in the iteration.
    auto copy = [&](int j, auto slotc, auto uc) __attribute__((always_inline)) {
      constexpr int k = decltype(slotc)::value % kRing;
      constexpr int u = decltype(uc)::value;
      const int b = (u * kWaves + wave) % NB;
      if (PF::copies_k(u, wave)) PF::copy_tile(rk, kslot(k), tile(j + kRing), b, dof[u]);
      else PF::copy_tile(rv, vslot((k + kRing - 2) % kRing), tile(j + kRing - 2), b, dof[u]);
    };
    // Iterations j in [j0, j1), j0 >= -1, of one variant; the loop body is
    // unrolled by kUnroll so that slots and parities are compile-time choices.
    // Every iteration ends in one barrier, so the waves of the workgroup stay
    // in step whatever their phase boundaries.
    auto phase = [&](auto& iteration, int j0, int j1, auto var) __attribute__((always_inline)) {
      for (int jb = j0 - ((j0 % kUnroll) + kUnroll) % kUnroll; jb < j1; jb += kUnroll) {
        static_for<kUnroll>([&](auto kc) __attribute__((always_inline)) {
          const int j = jb + decltype(kc)::value;
          if (j >= j0 && j < j1) iteration(j, var, kc);
        });
      }
    };

    // Q of this work item: from the wave's staging tile (copied in by
    // stage_q) into its AGPRs, read like a K fragment (B operand of S^T: lane
    // (n, hh) holds Q[row][16 kx + 8 hh + 0..7]), negated for a negative
    // scale; O^T and l zeroed.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    // (An opaque zero offset keeps the staging tile's per-fragment addresses
    // from being hoisted out of the item loop.)
    int zero = 0;
    pin(zero);
    if (p.qsign == 0) {
      // Straight from LDS into the AGPRs (the barrier below waits for them).
      static_for<KX>([&](auto ic) {
        constexpr int kx = decltype(ic)::value;
        const uint32_t a = xslot + (uint32_t)(zero + ad.k[kx]);
        asm volatile("ds_read_b128 a[%1:%2], %0" : : "v"(a), "n"(PF::qagpr(kx)), "n"(PF::qagpr(kx) + 3)
                     : "memory", ATTN_AGPRS);
      });
    } else {
      static_for<KX>([&](auto ic) {
        constexpr int kx = decltype(ic)::value;
        const u32x4 w = __builtin_bit_cast(u32x4, PF::kfrag(xl + zero, ad, kx));
        agpr_write<PF::qagpr(kx) + 0>(w[0] ^ p.qsign);
        agpr_write<PF::qagpr(kx) + 1>(w[1] ^ p.qsign);
        agpr_write<PF::qagpr(kx) + 2>(w[2] ^ p.qsign);
        agpr_write<PF::qagpr(kx) + 3>(w[3] ^ p.qsign);
      });
    }
    // O^T and l start at zero: one MFMA with zero operands and C = 0 clears
    // 16 AGPRs (68 AGPR writes otherwise).
    {
      typename PF::M::v8 z8 = {};
      pin(z8);
      static_for<DB>([&](auto dc) { PF::M::template zero16<PF::oagpr(decltype(dc)::value)>(z8); });
      uint2 z2 = make_uint2(0u, 0u);
      pin(z2);
      PF::M::template zero4<kLAgpr>(z2);
    }
    State st;
    st.mc = kMcInit;
    st.alpha = 1.f;
    TileArgs ta;
    ta.c = p.c;
    ta.sl2 = ALIBI ? p.slopes[cur.hq] * kLog2e : 0.f;
    if constexpr (PF::ACCB) {
      // c (s + kb) + base = c s + slope log2(e) kconst(r) + base.  A zero
      // scale takes a tiny c instead, whose product with s vanishes.
      if (ta.c == 0.f) ta.c = 1e-30f;
      const float ik = 1.f / ta.c;
      static_for<16>([&](auto rc) {
        constexpr int r = decltype(rc)::value;
        ta.kb[r] = ta.sl2 * (float)PF::kconst(r) * ik;
      });
    }
    ta.k2 = p.cap_k2 * ta.c;   // the scale folded into the cap's exponent
    ta.cl = p.cap_cl;
    ta.t = kNegInf;
    // Per-tile softmax parameters of tile(j).
    auto set_tile = [&](int j) __attribute__((always_inline)) {
      const int j0 = tile(j) * BN;
      ta.abase = ALIBI ? ta.sl2 * (float)(j0 + 4 * hh - iw - off) : 0.f;
      int l = Lk - 1 - j0 - 4 * hh;
      if (CAUSAL) l = min(l, row + off - j0 - 4 * hh);
      ta.lim = l;
      if (WIN) ta.llo = row + off + 1 - W - j0 - 4 * hh;
      if (ALIBI) ta.mb = ta.abase - st.mc;
      else if (CAP) ta.mb = ta.cl - st.mc;
    };
    // The first iteration with a softmax: O^T and l are still zero there, so
    // its rescale is skipped.
    const int jfirst = cur.f0;
    Scores sc[2];
    Probs pr[2];
    typename PF::template Ring<true> fk;
    typename PF::template Ring<false> fv;
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    // The first fragments of iteration -1: K tile 0 and V tile -2 (read but
    // not used: iteration -1 has no P.V).
    PF::template prime<true>(fk, lds, ad);
    PF::template prime<false>(fv, lds + (kRing + kRing - 2) * TE, ad);

    // Iteration j (from -1): copies, S^T of tile j+1 from K slot (j+1) mod
    // kRing (QK), softmax of tile j (SM), P.V of tile j-1 from V slot
    // (j-1) mod kRing (PV), the slow path when the tile's maximum moved past
    // the threshold in some row of the wave.  A tile's first fragments are
    // read at the end of the iteration before its use, so its copy, issued
    // kRing - 1 iterations before its use, must be complete at the barrier
    // that ends the iteration two before its use: vmcnt lets the copies of
    // the last kRing - 3 iterations stay in flight (every iteration issues
    // the same number of copies), and lgkmcnt lets the reads of the next iteration's
    // first fragments, which touch neither slot copied into next, cross the
    // barrier.
    auto iteration = [&](int j, auto var, auto slotc) __attribute__((always_inline)) {
      constexpr int VAR = decltype(var)::value;     // QK + 2 SM + 8 PV
      constexpr bool QK = (VAR & 1) != 0;
      constexpr int SM = (VAR >> 1) & 3;
      constexpr bool PV = (VAR & 8) != 0;
      constexpr int par = decltype(slotc)::value & 1;   // j mod 2
      constexpr int k = decltype(slotc)::value % kRing;   // j mod kRing
      const T* kl_use = lds + ((k + 1) % kRing) * TE;                   // K_{j+1}
      const T* kl_nxt = lds + ((k + 2) % kRing) * TE;                   // K_{j+2}
      const T* vl_use = lds + (kRing + (k + kRing - 1) % kRing) * TE;   // V_{j-1}
      const T* vl_nxt = lds + (kRing + k) * TE;                         // V_j
      if constexpr (SM != 0) set_tile(j);
      PF::template slots<QK, SM, PV>(st, sc[par], sc[par ^ 1], pr[par], pr[par ^ 1], fk, fv, kl_use, kl_nxt,
                                     vl_use, vl_nxt, ad, ta, [&](auto uc) { copy(j, slotc, uc); });
      if constexpr (SM != 0) {
        constexpr bool REL = PF::rel(SM, PV);
        if (__builtin_amdgcn_ballot_w64(PF::template exceeds<REL>(st, ta)) != 0) {
          PF::template resolve<REL>(st, sc[par], pr[par], ta);
          if (j != jfirst && __builtin_amdgcn_ballot_w64(st.alpha != 1.f) != 0) PF::repair(st.alpha);
        }
      }
      // 16 wait states between this iteration's last MFMAs and the next
      // iteration's first reads of their results; this iteration's copies
      // may stay in flight; then the barrier.
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_waitcnt vmcnt(%0) lgkmcnt(%1)\n\ts_barrier"
                   : : "n"((kRing - 3) * CPW), "n"(PF::kPrime) : "memory");
    };
    constexpr int PRO = 1, EPI = 8;
    constexpr int FIRST_WHOLE = 1 + 2, FIRST_MASKED = 1 + 4;
    constexpr int WHOLE = 1 + 2 + 8, MASKED = 1 + 4 + 8, IDLE = 0;
    const std::integral_constant<int, IDLE> idle;
    const int f0 = cur.f0, f1 = cur.f1;
    if (f1 < f0) {
      phase(iteration, -1, nt + 1, idle);
    } else if constexpr (!WIN && !REV) {
      // Keys run forward from tile 0, which every wave sees (f0 = 0, w0 <= 0):
      // the whole tiles come first, the masked ones (the causal diagonal, the
      // ragged end) last.
      iteration(-1, std::integral_constant<int, PRO>{}, std::integral_constant<int, kUnroll - 1>{});
      if (cur.w1 > 0) iteration(0, std::integral_constant<int, FIRST_WHOLE>{}, std::integral_constant<int, 0>{});
      else iteration(0, std::integral_constant<int, FIRST_MASKED>{}, std::integral_constant<int, 0>{});
      phase(iteration, 1, cur.w1, std::integral_constant<int, WHOLE>{});
      phase(iteration, max(cur.w1, 1), f1 + 1, std::integral_constant<int, MASKED>{});
      phase(iteration, f1 + 1, f1 + 2, std::integral_constant<int, EPI>{});
      phase(iteration, f1 + 2, nt + 1, idle);
    } else if constexpr (!WIN) {
      // Keys run from the last tile to tile 0, which every wave sees last
      // (f1 = nt - 1, w1 = nt): the masked tiles come first.
      phase(iteration, -1, f0 - 1, idle);
      phase(iteration, f0 - 1, f0, std::integral_constant<int, PRO>{});
      if (f0 >= cur.w0) phase(iteration, f0, f0 + 1, std::integral_constant<int, FIRST_WHOLE>{});
      else phase(iteration, f0, f0 + 1, std::integral_constant<int, FIRST_MASKED>{});
      phase(iteration, f0 + 1, cur.w0, std::integral_constant<int, MASKED>{});
      phase(iteration, max(cur.w0, f0 + 1), nt, std::integral_constant<int, WHOLE>{});
      phase(iteration, nt, nt + 1, std::integral_constant<int, EPI>{});
    } else {
      // Visible iterations f0 .. f1: the first one (no P.V yet), then the
      // masked ones before the whole ones (the window's lower edge, or with
      // ALiBi the causal diagonal), the whole ones, the masked ones after
      // them (the causal diagonal, or with ALiBi the window's edge).
      const int ws = min(max(cur.w0, f0 + 1), f1 + 1);
      const int we = min(max(cur.w1, ws), f1 + 1);
      phase(iteration, -1, f0 - 1, idle);
      phase(iteration, f0 - 1, f0, std::integral_constant<int, PRO>{});
      if (cur.w0 <= f0 && f0 < cur.w1) phase(iteration, f0, f0 + 1, std::integral_constant<int, FIRST_WHOLE>{});
      else phase(iteration, f0, f0 + 1, std::integral_constant<int, FIRST_MASKED>{});
      phase(iteration, f0 + 1, ws, std::integral_constant<int, MASKED>{});
      phase(iteration, ws, we, std::integral_constant<int, WHOLE>{});
      phase(iteration, we, f1 + 1, std::integral_constant<int, MASKED>{});
      phase(iteration, f1 + 1, f1 + 2, std::integral_constant<int, EPI>{});
      phase(iteration, f1 + 2, nt + 1, idle);
    }
    // The scores of the last iterations are dead, but are kept live past
    // the padding so that their registers are not reused while the MFMAs
    // writing them are in flight.
    hazard_pad();
    keep_live(sc[0]);
    keep_live(sc[1]);
    // The last iterations' copies (of tiles past the item, which write
    // zeros) may still be in flight into the slots that stage the output:
    // every wave waits for its own, then the barrier.
    asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");

    Item nxt;
    const bool more = item_at(round + 1, nxt);
    if (more) stage_kv(nxt);

    // Finalize: O = O^T / l, rounded to the input type.  Lane (n, hh) holds
    // head dims 32 db + 8 g + 4 hh + 0..3 of its row: it writes them to the
    // wave's staging tile (chunk 4 db + g of the row, half hh; no other wave
    // touches that tile), then the wave stores the tile row-major, 16 bytes a
    // lane, whole rows per instruction.
    {
      const float lt = sum_halves(agpr_read<kLAgpr>());
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      char* xo = reinterpret_cast<char*>(const_cast<T*>(xl));
      // The lane index passes through an opaque copy, so that the addresses
      // below are computed here, once per work item, rather than hoisted out
      // of the item loop into registers held through the key loop.
      int ln = lane;
      pin(ln);
      const int n2 = ln & 31, h2 = ln >> 5;
      const int sw = swz<D>(n2);
      static_for<DB * 4>([&](auto ic) {
        constexpr int f = decltype(ic)::value;
        constexpr int db = f / 4, g = f % 4;
        constexpr int a0 = PF::oagpr(db) + 4 * g;
        uint2 w;
        w.x = PF::E::pack2(agpr_read<a0>() * inv, agpr_read<a0 + 1>() * inv);
        w.y = PF::E::pack2(agpr_read<a0 + 2>() * inv, agpr_read<a0 + 3>() * inv);
        *reinterpret_cast<uint2*>(xo + 2 * (n2 * D + 8 * ((4 * db + g) ^ sw) + 4 * h2)) = w;
      });
      constexpr int RPI = 64 / CPR;   // rows per store instruction
      const int pos = ln % CPR;
      T* op = reinterpret_cast<T*>(p.o) + ((size_t)cur.head * Lq + iw) * D;
      static_for<BMW / RPI>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const int r = i * RPI + ln / CPR;
        const uint4 w = *reinterpret_cast<const uint4*>(xo + 2 * (r * D + 8 * (pos ^ swz<D>(r))));
        if (iw + r < Lq) *reinterpret_cast<uint4*>(op + (size_t)r * D + 8 * pos) = w;
      });
    }

    if (!more) break;
    stage_q(nxt);
    cur = nxt;
  }
}

// Compute units of the current device: kWgPerCu persistent workgroups each.
int compute_units() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  int n = cached[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <int D, typename T, bool CAUSAL, bool ALIBI, bool CAP, bool WIN = false>
hipError_t launch_t(const PrefillParams& p, hipStream_t stream) {
  PrefillParams q = p;
  // Query heads per workgroup: the largest power of two (up to the wave
  // count) that divides the GQA group.
  q.hg = 1;
  while (q.hg < kWaves && p.group % (2 * q.hg) == 0) q.hg *= 2;
  const int bm = BMW * (kWaves / q.hg);
  q.nqb = (p.Lq + bm - 1) / bm;
  q.nheads = p.B * p.Hq;
  q.nitems = q.nqb * (q.nheads / q.hg);
  if (q.nitems == 0) return hipSuccess;
  const int grid = std::min(q.nitems, kWgPerCu * compute_units());
  q.nxcd = grid % kXcds == 0 ? kXcds : 1;
  hipLaunchKernelGGL((prefill_kernel<D, T, CAUSAL, ALIBI, CAP, WIN>), dim3(grid), dim3(kThreads), 0, stream, q);
  return hipGetLastError();
}

template <int D, typename T>
hipError_t launch_d(const PrefillParams& p, hipStream_t s) {
  const PrefillFlags f = prefill_flags(p.causal != 0, p.slopes != nullptr, p.cap_cl != 0.f, p.window > 0);
  if (f.win) {
    if (f.cap) return launch_t<D, T, true, false, true, true>(p, s);
    return f.alibi ? launch_t<D, T, true, true, false, true>(p, s) : launch_t<D, T, true, false, false, true>(p, s);
  }
  if (f.cap) return launch_t<D, T, true, false, true>(p, s);
  if (f.causal) return f.alibi ? launch_t<D, T, true, true, false>(p, s) : launch_t<D, T, true, false, false>(p, s);
  return f.alibi ? launch_t<D, T, false, true, false>(p, s) : launch_t<D, T, false, false, false>(p, s);
}

}  // namespace

// Shard 0 also holds the dispatcher.
#if ATTN_PREFILL_SHARD == 0
hipError_t launch_prefill_d128_f16(const PrefillParams& p, hipStream_t s) { return launch_d<128, _Float16>(p, s); }
#elif ATTN_PREFILL_SHARD == 1
hipError_t launch_prefill_d128_bf16(const PrefillParams& p, hipStream_t s) { return launch_d<128, __bf16>(p, s); }
#elif ATTN_PREFILL_SHARD == 2
hipError_t launch_prefill_d64_f16(const PrefillParams& p, hipStream_t s) { return launch_d<64, _Float16>(p, s); }
#elif ATTN_PREFILL_SHARD == 3
hipError_t launch_prefill_d64_bf16(const PrefillParams& p, hipStream_t s) { return launch_d<64, __bf16>(p, s); }
#endif

#if ATTN_PREFILL_SHARD == 0
int prefill_block_rows() { return BM; }

hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
  if (p.D == 64) return p.bf16 ? launch_prefill_d64_bf16(p, stream) : launch_prefill_d64_f16(p, stream);
  return p.bf16 ? launch_prefill_d128_bf16(p, stream) : launch_prefill_d128_f16(p, stream);
}
#endif

}  // namespace attn

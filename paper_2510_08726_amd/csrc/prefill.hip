// Fused attention prefill for gfx950: the loop nest that rolling update
// (Section "Rolling Update", Algorithm 1, Eq. fixed-recurrent) produces from
// the plain attention definition, with the tile structure of the appendix
// "Privatization" (a local max per key tile, then the running max).
//
// Work split.  One workgroup = 4 wave64s = 256 query rows of one (batch,
// query head); each wave owns 64 rows (two 32-row blocks) for the whole key
// loop and runs alone on its SIMD with the full register file.  Key tiles
// are BN = 32 keys.  Per tile j and wave:
//
//   S^T = K_j . Q^T            32x32x16 MFMAs, K from LDS, Q resident in AGPRs
//   m'  = max(m, rowmax S)     in-lane max + permlane32 swaps
//   a   = exp2(m - m')         the repair factor h(t, r, r') = t exp(r - r')
//   P   = exp2(S - m')         rounded to the input type (the compute
//                              definition casts exp to the input dtype
//                              before the second matmul)
//   l   = a l + rowsum P       fp32 sum of the weights before rounding
//   O^T = a O^T + V_j^T . P^T  32x32x16 MFMAs, V from LDS, P taken straight
//                              from the S^T accumulator registers
//
// Computing S transposed puts one query row per lane (rows are the MFMA N
// index): row reductions stay in registers, the per-row repair of O^T is a
// per-lane scale, and the fp32 S^T accumulator converts in place into the B
// operand of the P.V product.  V stays row-major in LDS; its operand is
// gathered with the gfx950 transposing LDS read, in the key order in which
// the S^T accumulator holds keys.  Each K or V operand fragment read from
// LDS feeds the MFMAs of both 32-row blocks, which halves the LDS traffic
// per flop compared with 32 rows per wave.
//
// Schedule.  On gfx950 a wave's VALU instructions issued behind its own
// MFMA overlap with it, while VALU work of another wave on the same SIMD
// barely does.  So every wave software-pipelines its own loop: iteration j
// issues the MFMAs of S^T for tile j+1 and of P.V for tile j-1, and spreads
// the softmax of tile j (pure VALU, independent of both) over the gaps
// between them: the iteration is a fixed sequence of MFMA slots, each
// followed by its share of the softmax and by the LDS reads of the operands
// a few fragments ahead, fenced so the compiler keeps that order.  K and V
// tiles are copied HBM -> LDS by the buffer unit (loads with the LDS bit, no
// registers involved) into double buffers, one tile ahead of their first
// use; one barrier per iteration publishes them.
//
// The MFMAs are written as inline assembly to fix their register files: the
// S^T accumulators in VGPRs (the softmax reads them), O^T and Q in AGPRs.
// The compiler does not model the latency of those instructions, so every
// VALU reader of an MFMA result is at least two MFMAs and a barrier away
// from it, or behind explicit s_nop padding.
//
// Lazy repair.  The running max used in the exponent is only moved when a
// row's tile max exceeds it by more than 2^8 (in log2 units); until then the
// stale max keeps every P <= 2^8 (well inside the fp16 / bf16 range) and the
// O^T repair is skipped.  The repaired state is the same as with an always
// moving max, written relative to another reference point; the final
// division by l cancels it.
//
// Scores are in log2 units: t = s * scale * log2(e) (+ ALiBi bias * log2(e)),
// so each exponential is one v_exp_f32.

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
constexpr int RB = 2;                       // 32-row blocks per wave
constexpr int BMW = 32 * RB;                // query rows per wave
static_assert(RB == 2, "the row-max exchange and the finalisation handle two row blocks");
constexpr int BM = BMW * kWaves;            // query rows per workgroup
constexpr int BN = 32;                      // keys per tile
constexpr int PFD = 3;                      // operand fragments read ahead
constexpr int kRing = 4;                    // LDS slots per operand; copies run kRing - 1 tiles ahead
// A row's reference maximum moves only when a tile's maximum exceeds it by
// more than this (log2 units), so that P <= 2^kLazyThreshold.
constexpr float kLazyThreshold = 8.f;
// Reference max (times c) before the first visible key: finite, so the first
// visible tile takes the slow path like any other move and its rescale factor
// underflows to 0 (O^T and l are still 0 then).
constexpr float kMcInit = -1e30f;
// Accelerator dies (XCDs), each with its own L2; consecutive workgroups of a
// launch are dealt to them in turn.
constexpr int kXcds = 8;

// K and V tiles live in LDS row-major, [BN][D], with the 16-byte chunks of
// each row XOR-swizzled: chunk c of row r sits at chunk position c ^ swz(r).
// That keeps the K operand reads (16 consecutive rows at one chunk) and the
// transposing V reads (4 consecutive rows x 4 consecutive chunks per
// half-wave) free of bank conflicts; the copy engine writes whole 1 KB
// blocks, so the swizzle is applied on the global side of the copy.
// swz depends on r % 16 only.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if (D == 128) return 4 * (r & 3) + ((r >> 2) & 3);
  return 4 * ((r >> 1) & 1) + ((r >> 2) & 3);
}

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) void lds_void;

// Transposing LDS read: within each 16-lane group, output lane i element j is
// element (i % 4) of the 8 bytes addressed by lane (i / 4 + 4 j).
__device__ __forceinline__ uint2 lds_read_tr(const void* p) {
  v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p));
  return __builtin_bit_cast(uint2, r);
}

__device__ __forceinline__ float as_f(unsigned u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ unsigned as_u(float f) { return __builtin_bit_cast(unsigned, f); }

// Row maxima of two 32-row blocks whose rows are split over lanes l and l^32:
// returns max(a[l], a[l^32]) in `a` and max(b[l], b[l^32]) in `b`, in every
// lane.  permlane32_swap(x, y) exchanges the upper half of x with the lower
// half of y.
__device__ __forceinline__ void max_halves2(float& a, float& b) {
  auto r = __builtin_amdgcn_permlane32_swap(as_u(a), as_u(b), false, false);
  const float u = fmaxf(as_f((unsigned)r[0]), as_f((unsigned)r[1]));  // lanes < 32: block a, else block b
  auto t = __builtin_amdgcn_permlane32_swap(as_u(u), as_u(u), false, false);
  a = as_f((unsigned)t[0]);
  b = as_f((unsigned)t[1]);
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

// Register files.  The S^T accumulators, P and the LDS operands are ordinary
// values in VGPRs, allocated by the compiler.  O^T, Q, the exp-sums and a
// constant (1, 1) operand live in fixed AGPRs that only the inline assembly
// below names: O^T block (rb, db) in a[16 (rb DB + db) .. + 15], Q fragment
// (rb, kx) in a[128 + 4 (rb KX + kx) .. + 3], l of row block rb in
// a[192 + 4 rb .. + 3], the ones in a[200 .. 201].
// Every statement that touches them lists all AGPRs as clobbered, so the
// compiler keeps none of its own values there, and counts them as used.
#define ATTN_A10(p) "a" #p "0", "a" #p "1", "a" #p "2", "a" #p "3", "a" #p "4", \
                    "a" #p "5", "a" #p "6", "a" #p "7", "a" #p "8", "a" #p "9"
#define ATTN_AGPRS "a0", "a1", "a2", "a3", "a4", "a5", "a6", "a7", "a8", "a9", \
    ATTN_A10(1), ATTN_A10(2), ATTN_A10(3), ATTN_A10(4), ATTN_A10(5), ATTN_A10(6), ATTN_A10(7), ATTN_A10(8), ATTN_A10(9), ATTN_A10(10), ATTN_A10(11), ATTN_A10(12), ATTN_A10(13), ATTN_A10(14), ATTN_A10(15), ATTN_A10(16), ATTN_A10(17), ATTN_A10(18), ATTN_A10(19), ATTN_A10(20)
constexpr int kQAgpr = 128;
constexpr int kLAgpr = 192;     // exp-sum accumulators, 4 per row block
constexpr int kOnesAgpr = 200;  // two registers holding (1.0, 1.0)

// 32x32x16 MFMAs.  qk0/qk: S^T accumulator in VGPRs (qk0 starts from zero), K
// operand in VGPRs, Q operand from AGPRs a[QA .. QA + 3].  pv: O^T accumulator
// a[OA .. OA + 15], both operands in VGPRs.  rowsum: a 4x4x4 MFMA with the
// all-ones operand, which adds the four 16-bit values each lane holds in b to
// every register of its accumulator a[LA .. LA + 3]: the exp-sum l is
// accumulated from the same rounded weights that multiply V, on the matrix
// unit.  (Its s_nop 1 covers a VALU write of b just before it.)
template <typename T> struct Mma;
template <> struct Mma<_Float16> {
  typedef f16x8 v8;
  template <int QA> static __device__ __forceinline__ void qk0(f32x16& d, v8 a) {
    asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], 0" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int QA> static __device__ __forceinline__ void qk(f32x16& d, v8 a) {
    asm volatile("v_mfma_f32_32x32x16_f16 %0, %1, a[%2:%3], %0" : "+v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int OA> static __device__ __forceinline__ void pv(v8 a, v8 b) {
    asm volatile("v_mfma_f32_32x32x16_f16 a[%2:%3], %0, %1, a[%2:%3]" : : "v"(a), "v"(b), "n"(OA), "n"(OA + 15) : ATTN_AGPRS);
  }
  static constexpr uint32_t kOnes = 0x3c003c00u;   // (1.0, 1.0)
  template <int LA> static __device__ __forceinline__ void rowsum(uint2 b) {
    asm volatile("s_nop 1\n\tv_mfma_f32_4x4x4_16b_f16 a[%1:%2], a[%3:%4], %0, a[%1:%2]"
                 : : "v"(b), "n"(LA), "n"(LA + 3), "n"(kOnesAgpr), "n"(kOnesAgpr + 1) : ATTN_AGPRS);
  }
};
template <> struct Mma<__bf16> {
  typedef bf16x8 v8;
  template <int QA> static __device__ __forceinline__ void qk0(f32x16& d, v8 a) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], 0" : "=&v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int QA> static __device__ __forceinline__ void qk(f32x16& d, v8 a) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, a[%2:%3], %0" : "+v"(d) : "v"(a), "n"(QA), "n"(QA + 3) : ATTN_AGPRS);
  }
  template <int OA> static __device__ __forceinline__ void pv(v8 a, v8 b) {
    asm volatile("v_mfma_f32_32x32x16_bf16 a[%2:%3], %0, %1, a[%2:%3]" : : "v"(a), "v"(b), "n"(OA), "n"(OA + 15) : ATTN_AGPRS);
  }
  static constexpr uint32_t kOnes = 0x3f803f80u;   // (1.0, 1.0)
  template <int LA> static __device__ __forceinline__ void rowsum(uint2 b) {
    asm volatile("s_nop 1\n\tv_mfma_f32_4x4x4_16b_bf16 a[%1:%2], a[%3:%4], %0, a[%1:%2]"
                 : : "v"(b), "n"(LA), "n"(LA + 3), "n"(kOnesAgpr), "n"(kOnesAgpr + 1) : ATTN_AGPRS);
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

// The softmax of one tile as a list of steps, spread over the MFMA slots of
// an iteration in proportion to their VALU cost (in issue cycles):
//   prep   4 steps (ALiBi or masked tiles): bias and mask of 4 keys x 2 rows
//   max    8 steps: 4 scores folded into the partial max of a row block
//   fin    1 step : row maxima, lazy decisions, repair factors
//   exp   16 steps: 2 exponentials and their packing
// (the exp-sum is accumulated by rowsum MFMAs beside P.V).
template <bool PREP, bool MASKED, bool ALIBI>
struct SoftPlan {
  // Steps [0, MAX0) prepare the scores (ALiBi bias, mask), four registers a
  // step; then come 16 exponential steps (two registers each) and 8 steps of
  // the lane's running maximum (four registers each), as exp, exp, max.
  static constexpr int MAX0 = PREP ? 4 : 0;
  static constexpr int NSTEP = MAX0 + 24;
  static constexpr bool is_exp(int k) { return k >= MAX0 && (k - MAX0) % 3 != 2; }
  static constexpr int exp_index(int k) { return 2 * ((k - MAX0) / 3) + (k - MAX0) % 3; }
  static constexpr int max_index(int k) { return (k - MAX0) / 3; }
  static constexpr int weight(int k) {
    if (k < MAX0) return (ALIBI ? 12 : 0) * 4 + (MASKED ? 16 : 0) * 4;
    return is_exp(k) ? 30 : 8;
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

template <int D, typename T, bool CAUSAL, bool ALIBI>
struct Prefill {
  typedef Elem<T> E;
  typedef Mma<T> M;
  typedef typename E::vec8 vec8;
  static constexpr int KX = D / 16;                        // MFMA K-steps of Q.K^T
  static constexpr int DB = D / 32;                        // 32-dim blocks of O^T
  static constexpr int TE = BN * D;                        // elements of one K or V tile
  static constexpr int NI = TE * (int)sizeof(T) / 1024 / kWaves;  // 1 KB copies per wave per tile
  static constexpr int CPR = D / 8;                        // 16-byte chunks per row
  static constexpr int NG = KX;                            // K (or V) operand fragments per tile
  static_assert(NG == 2 * DB, "as many V fragments as K fragments");
  static_assert(NI >= 1, "a tile is at least one 1 KB copy per wave");

  // S^T accumulators of one tile: s[rb] holds keys 0..31 of row block rb.
  // Register r of lane (n, hh) is key 8 (r / 4) + 4 hh + r % 4 of row 32 rb + n.
  struct Scores {
    f32x16 s[RB];
  };
  // P^T as the B operand of P.V: w[rb][c][..] = keys of 16-key slice c.
  struct Probs {
    uint32_t w[RB][2][4];
  };
  struct State {
    float mc[RB];     // reference max of the row, times ce (log2 units)
    float alpha[RB];  // rescale factor of O^T and l set by the slow path
  };
  static constexpr int oagpr(int rb, int db) { return 16 * (rb * DB + db); }
  static constexpr int qagpr(int rb, int kx) { return kQAgpr + 4 * (rb * KX + kx); }
  // Per-lane LDS byte offsets inside a tile: K fragment kx, V fragment
  // (c16, db); c16 only adds an immediate.
  struct Addr {
    int k[KX];
    int v[DB][2];
  };
  // Softmax scratch of one tile.
  struct Tmp {
    float t[RB];      // this lane's maximum score of the tile, per row block
  };
  struct TileArgs {
    float c;      // scale * log2(e) (with ALiBi) or max(|scale| * log2(e), tiny)
    float sl2;    // ALiBi slope * log2(e)
    float abase;  // ALiBi bias of key j0 + 4 hh relative to the wave's first row
    int lim[RB];  // last visible key offset (key - j0 - 4 hh) of each row block
  };

  // HBM -> LDS copy of key/value tile t (rows t BN .. t BN + BN - 1) of one
  // head into the LDS slot at byte address `slot`: copy u of wave w fills the
  // 1 KB block u kWaves + w; dof holds the lane's global byte offsets.  The
  // buffer range ends at row `rows` (the workgroup's last staged row), so rows
  // past it read as zero, and a tile past it moves no data at all.  Issued as
  // inline assembly: the compiler then adds no waits of its own for the LDS
  // writes; the kernel waits for them explicitly before its barriers.
  static __device__ __forceinline__ void copy_tile(const T* base, uint32_t slot, int t, int rows, int wave,
                                                   const int (&dof)[NI]) {
    const int left = t >= 0 ? max(rows - t * BN, 0) : 0;
    const uint64_t a = reinterpret_cast<uint64_t>(base + (left > 0 ? (size_t)t * TE : 0));
    // The words are uniform; readfirstlane keeps them in SGPRs even where the
    // compiler computes the 64-bit address with vector instructions.
    const u32x4 rsrc = {(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                        (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
                        (uint32_t)__builtin_amdgcn_readfirstlane(left * D * (int)sizeof(T)), 0x00020000u};
#pragma unroll
    for (int u = 0; u < NI; ++u)
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   : : "s"(slot + (uint32_t)((u * kWaves + wave) * 1024)), "v"(dof[u]), "s"(rsrc) : "memory", "m0");
  }

  // This wave's copy of the RB * 32 rows at `base` into its LDS region at
  // byte address `dst`, in the layout of a K tile (row r at r * D elements,
  // chunk c at chunk position c ^ swz(r)); rows at or past `left` read as
  // zero.  Only the copying wave reads the region.
  static __device__ __forceinline__ void copy_rows(const T* base, uint32_t dst, int left, int lane) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    const int nb = max(min(left, RB * 32), 0) * D * (int)sizeof(T);
    const u32x4 rsrc = {(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                        (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
                        (uint32_t)__builtin_amdgcn_readfirstlane(nb), 0x00020000u};
#pragma unroll
    for (int blk = 0; blk < RB * TE * (int)sizeof(T) / 1024; ++blk) {
      const int r = blk * (1024 / (2 * D)) + lane / CPR;
      const int pos = lane % CPR;
      const int goff = (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T);
      asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                   : : "s"(dst + (uint32_t)(blk * 1024)), "v"(goff), "s"(rsrc) : "memory", "m0");
    }
  }

  static __device__ __forceinline__ void make_addr(Addr& ad, int lane) {
    const int n = lane & 31, hh = lane >> 5;
#pragma unroll
    for (int kx = 0; kx < KX; ++kx) ad.k[kx] = 2 * (n * D + 8 * ((2 * kx + hh) ^ swz<D>(n)));
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

  static __device__ __forceinline__ vec8 probs_b(const Probs& pr, int rb, int c16) {
    return __builtin_bit_cast(vec8, make_uint4(pr.w[rb][c16][0], pr.w[rb][c16][1], pr.w[rb][c16][2], pr.w[rb][c16][3]));
  }

  static constexpr int kconst(int r) { return 8 * (r / 4) + (r % 4); }

  // Softmax step K of a tile (see SoftPlan).  Without ALiBi the exponent is
  // s * c - m * c.  With ALiBi the score is first made s * c + bias in log2
  // units; the bias is written relative to the wave's first row,
  // -slope (i - j) = slope (j - iw - off) - slope (i - iw), and the last term
  // is dropped: it shifts a whole row by a constant, which the row's softmax
  // does not see.  Masked tiles set keys past Lk and (causal) keys after the
  // row to -inf before the max.
  template <int K, bool PREP, bool MASKED>
  static __device__ __forceinline__ void soft_step(State& st, Scores& sc, Probs& pr, Tmp& tp, const TileArgs& ta) {
    typedef SoftPlan<PREP, MASKED, ALIBI> P;
    const float ce = ALIBI ? 1.f : ta.c;
    if constexpr (K < P::MAX0) {
      constexpr int r0 = 4 * K;
#pragma unroll
      for (int r = r0; r < r0 + 4; ++r) {
        if constexpr (ALIBI) {
          const float bias = __builtin_fmaf(ta.sl2, (float)kconst(r), ta.abase);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) sc.s[rb][r] = __builtin_fmaf(sc.s[rb][r], ta.c, bias);
        }
        if constexpr (MASKED) {
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            if (kconst(r) > ta.lim[rb]) sc.s[rb][r] = kNegInf;
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          float x = sc.s[rb][r];
          pin(x);
          sc.s[rb][r] = x;
        }
      }
    } else if constexpr (P::is_exp(K)) {
      constexpr int k = P::exp_index(K);
      constexpr int rb = k % 2, r = 2 * (k / 2);
      const float p0 = fast_exp2(__builtin_fmaf(sc.s[rb][r], ce, -st.mc[rb]));
      const float p1 = fast_exp2(__builtin_fmaf(sc.s[rb][r + 1], ce, -st.mc[rb]));
      uint32_t w = E::pack2(p0, p1);
      pin(w);
      pr.w[rb][r / 8][(r % 8) / 2] = w;
    } else {
      constexpr int k = P::max_index(K);
      constexpr int q = k / 2, rb = k % 2;
      const f32x16& s = sc.s[rb];
      const float m4 = fmaxf(fmaxf(s[4 * q], s[4 * q + 1]), fmaxf(s[4 * q + 2], s[4 * q + 3]));
      if constexpr (q == 0) tp.t[rb] = m4;
      else tp.t[rb] = fmaxf(tp.t[rb], m4);
      pin(tp.t[rb]);
    }
  }

  // After the steps of a tile: does some score of this lane exceed the
  // reference maximum by more than the lazy threshold?  (Then the tile's P,
  // computed against the old reference, must be recomputed: see resolve.)
  static __device__ __forceinline__ bool exceeds(const State& st, const Tmp& tp, const TileArgs& ta) {
    const float ce = ALIBI ? 1.f : ta.c;
    bool x = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) x |= __builtin_fmaf(tp.t[rb], ce, -st.mc[rb]) > kLazyThreshold;
    return x;
  }

  // Slow path of a tile whose maximum moved past the threshold in some row
  // of the wave (always the case for a row's first visible tile, whose
  // reference is still kMcInit): the row maximum is combined over the lane
  // pair holding the row, rows that moved take it as their new reference,
  // O^T and l are rescaled by 2^-(move) (the P.V products so far used the
  // old reference), and the tile's P is recomputed.  Rows that did not move
  // keep their reference and factor 1.
  static __device__ __forceinline__ void resolve(State& st, Scores& sc, Probs& pr, Tmp& tp, const TileArgs& ta) {
    typedef SoftPlan<false, false, ALIBI> P;
    const float ce = ALIBI ? 1.f : ta.c;
    float t0 = tp.t[0], t1 = tp.t[1];
    max_halves2(t0, t1);
    const float tm[RB] = {t0, t1};
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float d = __builtin_fmaf(tm[rb], ce, -st.mc[rb]);
      const bool move = d > kLazyThreshold;
      st.alpha[rb] = move ? fast_exp2(-d) : 1.f;
      st.mc[rb] = move ? tm[rb] * ce : st.mc[rb];
    }
    repair(st);
    static_for<P::NSTEP>([&](auto kc) {
      constexpr int K = decltype(kc)::value;
      if constexpr (P::is_exp(K)) soft_step<K, false, false>(st, sc, pr, tp, ta);
    });
  }

  template <int B0, int B1, bool PREP, bool MASKED>
  static __device__ __forceinline__ void soft_range(State& st, Scores& sc, Probs& pr, Tmp& tp, const TileArgs& ta) {
    if constexpr (B1 > B0) {
      [&]<int... Ks>(std::integer_sequence<int, Ks...>) {
        (soft_step<B0 + Ks, PREP, MASKED>(st, sc, pr, tp, ta), ...);
      }(std::make_integer_sequence<int, B1 - B0>{});
    }
  }

  // Fragment i of an iteration: group i / 2, the K fragment of the group
  // first, then its V fragment.  Fragment i lives in ring entry i mod
  // (PFD + 1) and is read PFD fragments ahead of its MFMAs; the first PFD
  // fragments of an iteration are read at the end of the iteration before.
  static constexpr int NF = 2 * NG;   // fragments per iteration
  static_assert(NF % (PFD + 1) == 0, "fragment ring positions must repeat every iteration");
  // LDS instructions that read the first PFD fragments (a K fragment takes
  // one, a V fragment two).
  static constexpr int kPrimeReads = (PFD + 1) / 2 + 2 * (PFD / 2);
  typedef vec8 Ring[PFD + 1];

  template <int I>
  static __device__ __forceinline__ void read_frag(Ring& fr, const T* kl, const T* vl, const Addr& ad) {
    if constexpr (I % 2 == 0) fr[I % (PFD + 1)] = kfrag(kl, ad, I / 2);
    else fr[I % (PFD + 1)] = vfrag(vl, ad, I / 2);
  }
  // The first PFD fragments of the iteration whose tiles are kl and vl.
  static __device__ __forceinline__ void prime(Ring& fr, const T* kl, const T* vl, const Addr& ad) {
    static_for<PFD>([&](auto ic) { read_frag<decltype(ic)::value>(fr, kl, vl, ad); });
  }

  // One iteration of the software pipeline: S^T of tile j+1 (QK), softmax of
  // tile j (SM: 1 unmasked, 2 masked), P.V of tile j-1 (PV).  Group g holds
  // the slots [QK rb 0, QK rb 1, PV rb 0, PV rb 1] of K fragment g and V
  // fragment g.  kl, vl are this iteration's K and V tiles, kln, vln the next
  // iteration's (its first fragments are read in the last slots).

  template <bool QK, int SM, bool PV>
  static __device__ __forceinline__ bool iterate(State& st, Scores& s_cur, Scores& s_next, Probs& p_cur,
                                                 const Probs& p_prev, Ring& fr, const T* kl, const T* vl,
                                                 const T* kln, const T* vln, const Addr& ad, const TileArgs& ta,
                                                 Tmp& tp) {
    static_assert(QK && PV, "every iteration issues both products");
    constexpr bool MASKED = SM == 2;
    constexpr bool PREP = ALIBI || MASKED;
    typedef SoftPlan<PREP, MASKED, ALIBI> P;
    constexpr int FPG = 2;        // fragments per group
    constexpr int NS = 2 * NF;    // MFMA slots
    // Fragments NF .. NF + PFD - 1 are the first ones of the next iteration.
    auto read = [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i < NF) read_frag<i>(fr, kl, vl, ad);
      else read_frag<i - NF>(fr, kln, vln, ad);
    };
    {
      [&]<int... Ss>(std::integer_sequence<int, Ss...>) {
        (
            [&] {
              constexpr int S = Ss;
              constexpr int i = S / 2, rb = S % 2;
              constexpr int g = i / FPG;
              constexpr bool is_k = QK && (i % FPG == 0);
              if constexpr (rb == 0) read(std::integral_constant<int, i + PFD>{});
              if constexpr (is_k) {
                if constexpr (g == 0) M::template qk0<qagpr(rb, g)>(s_next.s[rb], fr[i % (PFD + 1)]);
                else M::template qk<qagpr(rb, g)>(s_next.s[rb], fr[i % (PFD + 1)]);
              } else {
                constexpr int c16 = g / DB, db = g % DB;
                M::template pv<oagpr(rb, db)>(fr[i % (PFD + 1)], probs_b(p_prev, rb, c16));
                // Exp-sum of the same weights: words 2 db, 2 db + 1 of the
                // slice, at fragments db = 0 and 1 (a large MFMA always
                // separates two rowsum MFMAs on one accumulator).
                if constexpr (db < 2)
                  M::template rowsum<kLAgpr + 4 * rb>(
                      make_uint2(p_prev.w[rb][c16][2 * db], p_prev.w[rb][c16][2 * db + 1]));
              }
              if constexpr (SM != 0)
                soft_range<P::begin(S, NS), P::begin(S + 1, NS), PREP, MASKED>(st, s_cur, p_cur, tp, ta);
              __builtin_amdgcn_sched_barrier(0);
            }(),
            ...);
      }(std::make_integer_sequence<int, NS>{});
    }
    return exceeds(st, tp, ta);
  }

  // O^T *= alpha and l *= alpha, in place in the AGPRs.
  static __device__ __forceinline__ void repair(const State& st) {
    hazard_pad();
    static_for<RB * DB * 16>([&](auto ic) {
      constexpr int e = decltype(ic)::value;
      agpr_scale<e>(st.alpha[e / (16 * DB)]);
    });
    static_for<RB * 4>([&](auto ic) {
      constexpr int e = decltype(ic)::value;
      agpr_scale<kLAgpr + e>(st.alpha[e / 4]);
    });
    hazard_pad();
  }
};

template <int D, typename T, bool CAUSAL, bool ALIBI>
__global__ __launch_bounds__(kThreads, 1) void prefill_kernel(PrefillParams p) {
  typedef Prefill<D, T, CAUSAL, ALIBI> PF;
  constexpr bool REV = ALIBI;
  typedef typename PF::vec8 vec8;
  typedef typename PF::State State;
  typedef typename PF::Scores Scores;
  typedef typename PF::Probs Probs;
  typedef typename PF::Addr Addr;
  typedef typename PF::TileArgs TileArgs;
  constexpr int KX = PF::KX;
  constexpr int TE = PF::TE;
  constexpr int NI = PF::NI;
  constexpr int CPR = PF::CPR;
  // LDS: a ring of kRing K tiles, a ring of kRing V tiles, then one region
  // of RB * 32 rows per wave that stages its Q block in and its O block out.
  __shared__ __attribute__((aligned(1024))) T lds[2 * kRing * TE + kWaves * RB * TE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31;
  const int hh = lane >> 5;

  Addr ad;
  PF::make_addr(ad, lane);
  // Global offsets of this lane's HBM -> LDS copies: in copy u the lane writes
  // bytes 16 lane .. 16 lane + 15 of 1 KB block u * kWaves + wave, i.e. chunk
  // position lane % CPR of row (block * 1024 / (2 D) + lane / CPR), and reads
  // the global chunk that the swizzle puts there.
  int dof[NI];
#pragma unroll
  for (int u = 0; u < NI; ++u) {
    const int blk = u * kWaves + wave;
    const int r = blk * (1024 / (2 * D)) + lane / CPR;
    const int pos = lane % CPR;
    dof[u] = (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T);
  }
  // LDS byte addresses of the K and V slots.
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void*)lds;
  auto kslot = [&](int s) __attribute__((always_inline)) { return lds0 + (uint32_t)(s * TE * (int)sizeof(T)); };
  auto vslot = [&](int s) __attribute__((always_inline)) {
    return lds0 + (uint32_t)((kRing + s) * TE * (int)sizeof(T));
  };

  // Persistent workgroups.  The work items (query block, query head) are
  // numbered KV head first, then query block by decreasing key count, then
  // query head within the KV head's group, so that neighbouring items read
  // the same K and V.  Workgroup g runs on XCD g mod kXcds (the order in
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
  const int per_kv = p.nqb * p.group;
  const int Lq = p.Lq, Lk = p.Lk;
  const int off = Lk - Lq;

  // One work item: its query block and head, and the key tiles [0, nt) that
  // the workgroup stages, [0, n_w) that this wave computes and [0, fm_w) that
  // no row of this wave masks.
  struct Item {
    int qb, head, kvh, hq, iw, nt, n_w, fm_w, rows;
  };
  auto item_at = [&](int round, Item& it) __attribute__((always_inline)) {
    const int sl = round * Pl + ((round & 1) ? Pl - 1 - c : c);
    if (sl >= s1 - s0) return false;
    const int s = s0 + sl;
    it.kvh = s / per_kv;
    const int rem = s - it.kvh * per_kv;
    it.qb = p.nqb - 1 - rem / p.group;
    it.head = it.kvh * p.group + rem % p.group;
    it.hq = it.head % p.Hq;
    const int i0 = it.qb * BM;
    it.iw = i0 + BMW * wave;
    int kend = Lk, kend_w = Lk;
    if (CAUSAL) {
      kend = min(Lk, min(i0 + BM, Lq) + off);
      kend_w = min(Lk, min(it.iw + BMW, Lq) + off);
    }
    if (it.iw >= Lq) kend_w = 0;
    it.nt = kend > 0 ? (kend + BN - 1) / BN : 0;
    it.n_w = kend_w > 0 ? (kend_w + BN - 1) / BN : 0;
    int fm = Lk / BN;
    if (CAUSAL) fm = min(fm, max(0, (it.iw + off + 1) / BN));
    it.fm_w = min(fm, it.n_w);
    it.rows = min(Lk, it.nt * BN);
    return true;
  };
  auto kbase = [&](const Item& it) __attribute__((always_inline)) {
    return reinterpret_cast<const T*>(p.k) + (size_t)it.kvh * Lk * D;
  };
  auto vbase = [&](const Item& it) __attribute__((always_inline)) {
    return reinterpret_cast<const T*>(p.v) + (size_t)it.kvh * Lk * D;
  };
  // Iteration j handles key tile tile(j).  With ALiBi the tiles are visited
  // from the last to the first: the bias grows with the key index, so the
  // first tile holds the largest bias of each row and the running maximum
  // rarely grows afterwards (each growth beyond the lazy threshold costs a
  // rescale of O^T).  Otherwise the keys run forward.
  auto tile_of = [&](const Item& it, int j) __attribute__((always_inline)) { return REV ? it.nt - 1 - j : j; };

  // Start of an item: the V slots of iterations -1 and -2 zeroed (the first
  // two iterations multiply them by P = 0) and the copies of the K tiles of
  // iterations 0 .. kRing-2 and of the V tile of iteration 0 issued.  It runs
  // after the barrier that ends the previous item's last LDS reads, while the
  // previous item's output is still being written; the caller waits for it.
  auto start_item = [&](const Item& it) __attribute__((always_inline)) {
    {
      constexpr int NV16 = TE * (int)sizeof(T) / 16;
      uint4* vz = reinterpret_cast<uint4*>(lds + (kRing + kRing - 2) * TE);   // slots kRing-2, kRing-1
#pragma unroll
      for (int i = tid; i < 2 * NV16; i += kThreads) vz[i] = make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kRing - 1; ++j) PF::copy_tile(kbase(it), kslot(j), tile_of(it, j), it.rows, wave, dof);
    PF::copy_tile(vbase(it), vslot(0), tile_of(it, 0), it.rows, wave, dof);
  };
  // This wave's staging region (Q rows in, O rows out) and the copy of an
  // item's Q rows into it; the region's previous contents must have been read.
  T* const qo = lds + 2 * kRing * TE + wave * RB * TE;
  const uint32_t qo_addr = (uint32_t)(uintptr_t)(lds_void*)qo;
  auto copy_q = [&](const Item& it) __attribute__((always_inline)) {
    PF::copy_rows(reinterpret_cast<const T*>(p.q) + ((size_t)it.head * Lq + it.iw) * D, qo_addr, Lq - it.iw, lane);
  };

  Item cur;
  if (!item_at(0, cur)) return;
  start_item(cur);
  copy_q(cur);
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
  agpr_write<kOnesAgpr>(PF::M::kOnes);
  agpr_write<kOnesAgpr + 1>(PF::M::kOnes);

  for (int round = 0;; ++round) {
    const int nt = cur.nt, n_w = cur.n_w, fm_w = cur.fm_w;
    const int iw = cur.iw;
    const int row0 = iw + n;          // this lane's row in row block 0
    const T* kp = kbase(cur);
    const T* vp = vbase(cur);

    // Q fragments (B operand of S^T: lane (n, hh) holds Q[row][16 kx + 8 hh
    // + 0..7], read like K fragments) into their AGPRs, negated for a
    // negative scale; O^T and l start at zero.
    static_for<RB * KX>([&](auto ic) {
      constexpr int f = decltype(ic)::value;
      constexpr int rb = f / KX, kx = f % KX;
      const u32x4 w = __builtin_bit_cast(u32x4, PF::kfrag(qo + rb * TE, ad, kx));
      agpr_write<PF::qagpr(rb, kx) + 0>(w[0] ^ p.qsign);
      agpr_write<PF::qagpr(rb, kx) + 1>(w[1] ^ p.qsign);
      agpr_write<PF::qagpr(rb, kx) + 2>(w[2] ^ p.qsign);
      agpr_write<PF::qagpr(rb, kx) + 3>(w[3] ^ p.qsign);
    });
    static_for<RB * PF::DB * 16>([&](auto ic) { agpr_zero<decltype(ic)::value>(); });
    static_for<RB * 4>([&](auto ic) { agpr_zero<kLAgpr + decltype(ic)::value>(); });
    State st;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      st.mc[rb] = kMcInit;
      st.alpha[rb] = 1.f;
    }
    auto tile = [&](int j) __attribute__((always_inline)) { return tile_of(cur, j); };
    auto copy_tile = [&](const T* base, uint32_t slot, int j) __attribute__((always_inline)) {
      PF::copy_tile(base, slot, tile(j), cur.rows, wave, dof);
    };

    TileArgs ta;
    ta.c = p.c;
    ta.sl2 = ALIBI ? p.slopes[cur.hq] * kLog2e : 0.f;
    // Per-tile softmax parameters.  Tiles outside [0, n_w) are fully masked
    // (lim = -1): their softmax leaves the state unchanged and gives P = 0.
    auto set_tile = [&](int j) __attribute__((always_inline)) {
      const int t = tile(j);
      const int j0 = t * BN;
      ta.abase = ALIBI ? ta.sl2 * (float)(j0 + 4 * hh - iw - off) : 0.f;
      const bool live = t >= 0 && t < n_w;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        int l = Lk - 1 - j0 - 4 * hh;
        if (CAUSAL) l = min(l, row0 + 32 * rb + off - j0 - 4 * hh);
        ta.lim[rb] = live ? l : -1;
      }
    };

    Scores sc[2];
    Probs pr[2];
    typename PF::Ring fr;
    // P of iteration -2 is zero (iteration -1 writes a zero P as well, and
    // idle iterations leave both in place).  Pinned, so that the zeros are
    // materialised in VGPRs here and not just before the first P.V MFMA that
    // reads them.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int cc = 0; cc < 2; ++cc)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          uint32_t z = 0u;
          pin(z);
          pr[0].w[rb][cc][w] = z;
        }

    // Iteration j (from -1; "tile j" below is tile(j)): copies of K_{j+kRing}
    // and V_{j+kRing-2}; S^T of tile j+1, softmax of tile j, P.V of tile j-1,
    // then, if tile j's maximum moved past the threshold in some row of the
    // wave, the slow path (rescale of O^T and l, P recomputed).  The K or V tile of iteration j lives in
    // slot j mod kRing.  A tile's first fragments are read at the end of the
    // iteration before its use, so its copy, issued kRing - 1 iterations
    // before its use into the slot read by the iteration before, must be
    // complete at the barrier that ends the iteration two before its use:
    // vmcnt lets only the current iteration's copies stay in flight (every
    // iteration issues the same number of copies), and lgkmcnt lets the reads
    // of the next iteration's first fragments, which touch neither slot
    // copied into next, cross the barrier.  The scores and probabilities of
    // iteration j live in the register buffers of the parity of j.  VAR is 1
    // for tiles every row of the wave sees whole, 2 for masked tiles
    // (including the tiles outside [0, n_w), whose softmax is a no-op: P = 0,
    // K unused), 0 for iterations in which the wave has no S^T, softmax or
    // P.V to do (copies, the next iteration's first fragments and the
    // barrier only).
    auto iteration = [&](int j, auto var, auto slotc) __attribute__((always_inline)) {
      constexpr int VAR = decltype(var)::value;
      constexpr int k = decltype(slotc)::value;   // j mod kRing
      constexpr int par = k & 1;
      copy_tile(kp, kslot(k), j + kRing);
      copy_tile(vp, vslot((k + kRing - 2) % kRing), j + kRing - 2);
      const T* kl_nxt = lds + ((k + 2) % kRing) * TE;   // K_{j+2}
      const T* vl_nxt = lds + (kRing + k) * TE;         // V_j
      if constexpr (VAR != 0) {
        set_tile(j);
        const T* kl_use = lds + ((k + 1) % kRing) * TE;                  // K_{j+1}
        const T* vl_use = lds + (kRing + (k + kRing - 1) % kRing) * TE;  // V_{j-1}
        typename PF::Tmp tp;
        const bool moved = PF::template iterate<true, VAR, true>(st, sc[par], sc[par ^ 1], pr[par], pr[par ^ 1], fr,
                                                                 kl_use, vl_use, kl_nxt, vl_nxt, ad, ta, tp);
        if (__builtin_amdgcn_ballot_w64(moved) != 0) PF::resolve(st, sc[par], pr[par], tp, ta);
      } else {
        PF::prime(fr, kl_nxt, vl_nxt, ad);
      }
      // 16 wait states between this iteration's last MFMAs and the next
      // iteration's first reads of their results, the waits described above,
      // then the barrier that publishes the completed copies.
      asm volatile("s_nop 7\n\ts_nop 7\n\ts_waitcnt vmcnt(%0) lgkmcnt(%1)\n\ts_barrier"
                   : : "n"(2 * NI), "n"(PF::kPrimeReads) : "memory");
    };
    // Iterations j in [j0, j1), j0 >= 0, of one variant; the loop body is
    // unrolled by kRing so that slots and parities are compile-time choices.
    // Every iteration of every wave ends in one barrier, so the waves of the
    // workgroup stay in step whatever their phase boundaries.
    auto phase = [&](int j0, int j1, auto var) __attribute__((always_inline)) {
      for (int jb = j0 & ~(kRing - 1); jb < j1; jb += kRing) {
        static_for<kRing>([&](auto kc) __attribute__((always_inline)) {
          const int j = jb + decltype(kc)::value;
          if (j >= j0 && j < j1) iteration(j, var, kc);
        });
      }
    };

    const std::integral_constant<int, 0> idle;
    const std::integral_constant<int, 1> whole;
    const std::integral_constant<int, 2> masked;
    // The first fragments of iteration -1: K_0 and the zeroed V slot.
    PF::prime(fr, lds, lds + (kRing + kRing - 2) * TE, ad);
    iteration(-1, masked, std::integral_constant<int, kRing - 1>{});
    if constexpr (REV) {
      // Tiles [n_w + 1, nt) first (nothing to do), then n_w (its S^T of
      // tile n_w - 1 is the first needed), the masked tiles [fm_w, n_w), the
      // whole tiles, and the P.V of tile 0.
      const int a = max(0, nt - n_w - 1);
      phase(0, a, idle);
      phase(a, nt - fm_w, masked);
      phase(nt - fm_w, nt, whole);
      phase(nt, nt + 1, masked);
    } else {
      phase(0, fm_w, whole);
      phase(max(fm_w, 0), n_w + 1, masked);
      phase(n_w + 1, nt + 1, idle);
    }

    // The next item's K/V copies go out before this item's output is
    // written, so that their latencies overlap.
    Item nxt;
    const bool more = item_at(round + 1, nxt);
    if (more) start_item(nxt);

    // Finalize: O = O^T / l, rounded to the input type.  Lane (n, hh) holds
    // head dims 32 db + 8 g + 4 hh + 0..3 of its row; they go to the wave's
    // staging region in the K-tile layout, come back as whole 16-byte chunks
    // (1 KB of consecutive rows per instruction) and are stored from there,
    // rows past Lq falling outside the store's range.  The scores of the last
    // iteration are dead, but are kept live past the padding so that their
    // registers are not reused while the MFMAs writing them are in flight.
    hazard_pad();
#pragma unroll
    for (int pb = 0; pb < 2; ++pb)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) keep_live(sc[pb].s[rb]);
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float lt = sum_halves(rb == 0 ? agpr_read<kLAgpr>() : agpr_read<kLAgpr + 4>());
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      st.alpha[rb] = inv;
    }
    static_for<RB * PF::DB * 4>([&](auto ic) {
      constexpr int f = decltype(ic)::value;
      constexpr int rb = f / (PF::DB * 4), db = (f / 4) % PF::DB, g = f % 4;
      constexpr int a0 = PF::oagpr(rb, db) + 4 * g;
      const float inv = st.alpha[rb];
      uint2 w;
      w.x = PF::E::pack2(agpr_read<a0>() * inv, agpr_read<a0 + 1>() * inv);
      w.y = PF::E::pack2(agpr_read<a0 + 2>() * inv, agpr_read<a0 + 3>() * inv);
      const int r = 32 * rb + n;
      *reinterpret_cast<uint2*>(qo + r * D + 8 * ((4 * db + g) ^ swz<D>(r)) + 4 * hh) = w;
    });
    {
      constexpr int NB = RB * TE * (int)sizeof(T) / 1024;
      const int left = max(min(Lq - iw, RB * 32), 0) * D * (int)sizeof(T);
      const __amdgpu_buffer_rsrc_t orsrc = __builtin_amdgcn_make_buffer_rsrc(
          reinterpret_cast<T*>(p.o) + ((size_t)cur.head * Lq + iw) * D, 0, left, 0x00020000);
      const char* qob = reinterpret_cast<const char*>(qo);
#pragma unroll
      for (int blk = 0; blk < NB; ++blk) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(qob + blk * 1024 + lane * 16);
        const int r = blk * (1024 / (2 * D)) + lane / CPR;
        const int pos = lane % CPR;
        __builtin_amdgcn_raw_buffer_store_b128(w, orsrc, (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T), 0, 0);
      }
    }
    // The region is free once its reads have returned: the next item's Q.
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (more) copy_q(nxt);
    if (!more) break;
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    cur = nxt;
  }
}

// Compute units of the current device: one persistent workgroup each.
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

template <int D, typename T, bool CAUSAL, bool ALIBI>
hipError_t launch_t(const PrefillParams& p, hipStream_t stream) {
  PrefillParams q = p;
  q.nheads = p.B * p.Hq;
  q.nitems = p.nqb * q.nheads;
  if (q.nitems == 0) return hipSuccess;
  const int grid = std::min(q.nitems, compute_units());
  q.nxcd = grid % kXcds == 0 ? kXcds : 1;
  hipLaunchKernelGGL((prefill_kernel<D, T, CAUSAL, ALIBI>), dim3(grid), dim3(kThreads), 0, stream, q);
  return hipGetLastError();
}

template <int D, typename T>
hipError_t launch_d(const PrefillParams& p, hipStream_t s) {
  if (p.causal) {
    return p.slopes ? launch_t<D, T, true, true>(p, s) : launch_t<D, T, true, false>(p, s);
  }
  return p.slopes ? launch_t<D, T, false, true>(p, s) : launch_t<D, T, false, false>(p, s);
}

}  // namespace

// This file is compiled once per (head dim, element type) shard, selected by
// ATTN_PREFILL_SHARD, so the instantiations build in parallel; shard 0 also
// holds the dispatcher.
#ifndef ATTN_PREFILL_SHARD
#define ATTN_PREFILL_SHARD 0
#endif
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

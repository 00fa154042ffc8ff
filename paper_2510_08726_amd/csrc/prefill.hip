// Fused attention prefill for gfx950: the loop nest that rolling update
// (Section "Rolling Update", Algorithm 1, Eq. fixed-recurrent) produces from
// the plain attention definition, with the tile structure of the appendix
// "Privatization" (a local max per key tile, then the running max).
//
// Work split.  One workgroup = 8 wave64s = 256 query rows of one (batch,
// query head), two waves per SIMD.  The two waves of a SIMD share 64 rows
// (two 32-row blocks) for the whole key loop and split the work on them.
// Key tiles are BN = 32 keys.  Per tile j:
//
//   softmax wave  S^T = K_j . Q^T       32x32x16 MFMAs, K from LDS, Q in AGPRs
//                 P = exp2(S - m)       against the row's reference max m,
//                                       rounded to the input type (the compute
//                                       definition casts exp to the input dtype
//                                       before the second matmul)
//                 a = exp2(m - m')      only when the tile's max exceeds m by
//                                       more than the lazy threshold (then m'
//                                       replaces m and P is recomputed)
//   P.V wave      O^T = a O^T + V_j^T . P^T,  l = a l + rowsum P
//                                       32x32x16 MFMAs, V from LDS, O^T and l
//                                       in AGPRs
//
// P and the factors a pass from the softmax wave to its P.V wave through a
// lane-private LDS exchange buffer.  Computing S transposed puts one query
// row per lane (rows are the MFMA N index): row reductions stay in
// registers, the per-row rescale of O^T is a per-lane scale, and the fp32
// S^T accumulator converts in place into the layout of the B operand of the
// P.V product.  V stays row-major in LDS; its operand is gathered with the
// gfx950 transposing LDS read, in the key order in which the S^T accumulator
// holds keys.  Each K or V operand fragment read from LDS feeds the MFMAs of
// both 32-row blocks.
//
// Schedule.  Iteration j: the softmax wave issues the MFMAs of S^T for tile
// j+1 back to back, then the softmax of tile j (pure VALU); the P.V wave
// issues P.V for tile j-1 and the HBM -> LDS copies of K and V (buffer loads
// with the LDS bit, into rings of kRing tiles).  The P.V MFMAs run on the
// matrix unit while the softmax wave's VALU work runs beside them; one
// barrier per iteration publishes the copies and the exchange buffers.
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
// so each exponential is one v_exp_f32.

#include <algorithm>
#include <atomic>
#include <type_traits>
#include <utility>

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

// Two waves per SIMD: wave p (p < kPairs) computes S^T and the softmax of
// its 64 rows, wave p + kPairs (same SIMD) the P.V products and row sums of
// the same rows.
constexpr int kPairs = 4;
constexpr int kWaves = 2 * kPairs;
constexpr int kThreads = 64 * kWaves;
constexpr int kCopyWaves = kPairs;          // the P.V waves also issue the HBM -> LDS copies
constexpr int RB = 2;                       // 32-row blocks per wave
constexpr int BMW = 32 * RB;                // query rows per wave
static_assert(RB == 2, "the row-max exchange and the finalisation handle two row blocks");
constexpr int BM = BMW * kPairs;            // query rows per workgroup
constexpr int BN = 32;                      // keys per tile
constexpr int PFD_K = 1;                    // K fragments read ahead (softmax wave)
constexpr int PFD_V = 3;                    // V fragments read ahead (P.V wave)
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
// values in VGPRs, allocated by the compiler.  The operands that live through
// the whole key loop are in fixed AGPRs that only the inline assembly below
// names, per role: in the softmax wave Q fragment (rb, kx) in
// a[4 (rb KX + kx) .. + 3]; in the P.V wave O^T block (rb, db) in
// a[16 (rb DB + db) .. + 15], l of row block rb in a[128 + 4 rb .. + 3], the
// ones in a[136 .. 137].  So at most 138 AGPRs, which leaves 118 VGPRs of a
// wave's 256 at two waves per SIMD.
// Every statement that touches them lists all AGPRs as clobbered, so the
// compiler keeps none of its own values there, and counts them as used.
#define ATTN_A10(p) "a" #p "0", "a" #p "1", "a" #p "2", "a" #p "3", "a" #p "4", \
                    "a" #p "5", "a" #p "6", "a" #p "7", "a" #p "8", "a" #p "9"
#define ATTN_AGPRS "a0", "a1", "a2", "a3", "a4", "a5", "a6", "a7", "a8", "a9", \
    ATTN_A10(1), ATTN_A10(2), ATTN_A10(3), ATTN_A10(4), ATTN_A10(5), ATTN_A10(6), ATTN_A10(7), ATTN_A10(8), ATTN_A10(9), ATTN_A10(10), ATTN_A10(11), ATTN_A10(12), \
    "a130", "a131", "a132", "a133", "a134", "a135", "a136", "a137"
constexpr int kQAgpr = 0;
constexpr int kLAgpr = 128;     // exp-sum accumulators, 4 per row block
constexpr int kOnesAgpr = 136;  // two registers holding (1.0, 1.0)

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

// The softmax of one tile as a list of steps (weights are their VALU cost in
// issue cycles, used to spread steps over MFMA slots where that is wanted):
//   prep   4 steps (ALiBi or masked tiles): bias and mask of 4 keys x 2 rows
//   exp   16 steps: 2 exponentials and their packing
//   max    8 steps: 4 scores folded into this lane's partial max of a row block
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
  static constexpr int NI = TE * (int)sizeof(T) / 1024 / kCopyWaves;  // 1 KB copies per copying wave per tile
  static constexpr int CPR = D / 8;                        // 16-byte chunks per row
  static constexpr int NG = KX;                            // K (or V) operand fragments per tile
  static_assert(NG == 2 * DB, "as many V fragments as K fragments");
  static_assert(NI >= 1, "a tile is at least one 1 KB copy per copying wave");

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
  static_assert(16 * RB * DB <= kLAgpr && kQAgpr + 4 * RB * KX <= kLAgpr, "AGPR map");
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
    u32x4* xp;    // this lane's exchange units for the tile's P (unit rb * 2 + c16, stride 64)
  };

  // HBM -> LDS copy of key/value tile t (rows t BN .. t BN + BN - 1) of one
  // head into the LDS slot at byte address `slot`: copy u of copying wave cw
  // fills the 1 KB block u kCopyWaves + cw; dof holds the lane's global byte
  // offsets.  The
  // buffer range ends at row `rows` (the workgroup's last staged row), so rows
  // past it read as zero, and a tile past it moves no data at all.  Issued as
  // inline assembly: the compiler then adds no waits of its own for the LDS
  // writes; the kernel waits for them explicitly before its barriers.
  static __device__ __forceinline__ void copy_tile(const T* base, uint32_t slot, int t, int rows, int cw,
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
                   : : "s"(slot + (uint32_t)((u * kCopyWaves + cw) * 1024)), "v"(dof[u]), "s"(rsrc) : "memory", "m0");
  }

  static __device__ __forceinline__ void make_addr_k(Addr& ad, int lane) {
    const int n = lane & 31, hh = lane >> 5;
#pragma unroll
    for (int kx = 0; kx < KX; ++kx) ad.k[kx] = 2 * (n * D + 8 * ((2 * kx + hh) ^ swz<D>(n)));
  }
  static __device__ __forceinline__ void make_addr_v(Addr& ad, int lane) {
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
      // A complete 16-key slice of P goes to the exchange buffer at once.
      if constexpr (r % 8 == 6) {
        const u32x4 u = {pr.w[rb][r / 8][0], pr.w[rb][r / 8][1], pr.w[rb][r / 8][2], pr.w[rb][r / 8][3]};
        ta.xp[64 * (rb * 2 + r / 8)] = u;
      }
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
  // pair holding the row, rows that moved take it as their new reference
  // and the factor 2^-(move) by which the P.V wave rescales O^T and l before
  // it adds this tile (the products so far used the old reference), and the
  // tile's P is recomputed.  Rows that did not move keep their reference and
  // factor 1.
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

  // Operand fragments: an iteration of either wave uses NG fragments, K
  // fragments (kx = 0..NG-1) for S^T, V fragments (g = c16 DB + db) for P.V.
  // Fragment i lives in ring entry i mod (PFD + 1) and is read PFD fragments
  // ahead of its MFMAs; the first PFD fragments of an iteration are read at
  // the end of the iteration before.
  template <bool IS_K> static constexpr int pfd() { return IS_K ? PFD_K : PFD_V; }
  static_assert(NG % (PFD_K + 1) == 0 && NG % (PFD_V + 1) == 0, "fragment ring positions must repeat every iteration");
  template <bool IS_K> using Ring = vec8[pfd<IS_K>() + 1];
  // LDS instructions that read the first fragments of an iteration.
  static constexpr int kPrimeK = PFD_K;
  static constexpr int kPrimeV = 2 * PFD_V;

  template <bool IS_K, int I>
  static __device__ __forceinline__ void read_frag(Ring<IS_K>& fr, const T* tile, const Addr& ad) {
    if constexpr (IS_K) fr[I % (PFD_K + 1)] = kfrag(tile, ad, I);
    else fr[I % (PFD_V + 1)] = vfrag(tile, ad, I);
  }
  template <bool IS_K>
  static __device__ __forceinline__ void prime(Ring<IS_K>& fr, const T* tile, const Addr& ad) {
    static_for<pfd<IS_K>()>([&](auto ic) { read_frag<IS_K, decltype(ic)::value>(fr, tile, ad); });
  }

  // One iteration of the softmax wave: the 2 NG MFMAs of S^T of tile j+1 (kl:
  // its K tile; order [kx, rb]) back to back, then the softmax of tile j (SM:
  // 1 unmasked, 2 masked); kln is the next iteration's K tile, whose first
  // fragments are read during the last MFMAs.  Returns whether some score of
  // this lane exceeds its row's reference by more than the threshold.  (The
  // partner P.V wave's MFMAs fill the matrix unit while this wave runs its
  // VALU work; interleaving both kinds in this wave stalled it whenever the
  // partner's MFMAs held the matrix unit.)
  template <int SM>
  static __device__ __forceinline__ bool iterate_s(State& st, Scores& s_cur, Scores& s_next, Probs& p_cur,
                                                   Ring<true>& fr, const T* kl, const T* kln,
                                                   const Addr& ad, const TileArgs& ta, Tmp& tp) {
    constexpr bool MASKED = SM == 2;
    constexpr bool PREP = ALIBI || MASKED;
    typedef SoftPlan<PREP, MASKED, ALIBI> P;
    constexpr int NS = 2 * NG;
    auto read = [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i < NG) read_frag<true, i>(fr, kl, ad);
      else read_frag<true, i - NG>(fr, kln, ad);
    };
    [&]<int... Ss>(std::integer_sequence<int, Ss...>) {
      (
          [&] {
            constexpr int S = Ss;
            constexpr int kx = S / 2, rb = S % 2;
            if constexpr (rb == 0) read(std::integral_constant<int, kx + PFD_K>{});
            if constexpr (kx == 0) M::template qk0<qagpr(rb, kx)>(s_next.s[rb], fr[kx % (PFD_K + 1)]);
            else M::template qk<qagpr(rb, kx)>(s_next.s[rb], fr[kx % (PFD_K + 1)]);
          }(),
          ...);
    }(std::make_integer_sequence<int, NS>{});
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (SM != 0) soft_range<0, P::NSTEP, PREP, MASKED>(st, s_cur, p_cur, tp, ta);
    if constexpr (SM != 0) return exceeds(st, tp, ta);
    return false;
  }

  // One iteration of the P.V wave: O^T += V^T P^T of tile j-1 (vl: its V
  // tile; the 2 NG slots are [g, rb], g = c16 DB + db) with the row sums of
  // the same weights; vln is the next iteration's V tile.
  static __device__ __forceinline__ void iterate_o(const Probs& pr, Ring<false>& fr, const T* vl, const T* vln,
                                                   const Addr& ad) {
    constexpr int NS = 2 * NG;
    auto read = [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i < NG) read_frag<false, i>(fr, vl, ad);
      else read_frag<false, i - NG>(fr, vln, ad);
    };
    [&]<int... Ss>(std::integer_sequence<int, Ss...>) {
      (
          [&] {
            constexpr int S = Ss;
            constexpr int g = S / 2, rb = S % 2;
            constexpr int c16 = g / DB, db = g % DB;
            if constexpr (rb == 0) read(std::integral_constant<int, g + PFD_V>{});
            M::template pv<oagpr(rb, db)>(fr[g % (PFD_V + 1)], probs_b(pr, rb, c16));
            // Exp-sum of the same weights: words 2 db, 2 db + 1 of the slice,
            // at fragments db = 0 and 1 (a large MFMA always separates two
            // rowsum MFMAs on one accumulator).
            if constexpr (db < 2)
              M::template rowsum<kLAgpr + 4 * rb>(make_uint2(pr.w[rb][c16][2 * db], pr.w[rb][c16][2 * db + 1]));
            __builtin_amdgcn_sched_barrier(0);
          }(),
          ...);
    }(std::make_integer_sequence<int, NS>{});
  }

  // O^T *= alpha and l *= alpha, in place in the P.V wave's AGPRs.
  static __device__ __forceinline__ void repair(const float (&alpha)[RB]) {
    hazard_pad();
    static_for<RB * DB * 16>([&](auto ic) {
      constexpr int e = decltype(ic)::value;
      agpr_scale<e>(alpha[e / (16 * DB)]);
    });
    static_for<RB * 4>([&](auto ic) {
      constexpr int e = decltype(ic)::value;
      agpr_scale<kLAgpr + e>(alpha[e / 4]);
    });
    hazard_pad();
  }
};

// Two waves per SIMD leave each wave 256 registers: the 138 AGPRs named by
// the inline assembly and at most 116 VGPRs (the compiler does not subtract
// the inline assembly's AGPRs from its budget by itself).
template <int D, typename T, bool CAUSAL, bool ALIBI>
__global__ __launch_bounds__(kThreads, 1) __attribute__((amdgpu_num_vgpr(116))) void prefill_kernel(PrefillParams p) {
  typedef Prefill<D, T, CAUSAL, ALIBI> PF;
  constexpr bool REV = ALIBI;
  typedef typename PF::vec8 vec8;
  typedef typename PF::State State;
  typedef typename PF::Scores Scores;
  typedef typename PF::Probs Probs;
  typedef typename PF::Addr Addr;
  typedef typename PF::TileArgs TileArgs;
  constexpr int KX = PF::KX;
  constexpr int DB = PF::DB;
  constexpr int TE = PF::TE;
  constexpr int NI = PF::NI;
  constexpr int CPR = PF::CPR;
  // LDS: a ring of kRing K tiles, a ring of kRing V tiles, then per pair of
  // waves two exchange buffers (tile parity) in which the softmax wave leaves
  // P (units rb * 2 + c16: the four words of slice c16 of row block rb) and
  // the rescale factors (unit 2 RB) for its P.V wave, 16 bytes per lane and
  // unit, lane-private.
  constexpr int XU = 2 * RB + 1;
  __shared__ __attribute__((aligned(1024))) T lds[2 * kRing * TE];
  __shared__ __attribute__((aligned(16))) u32x4 xch[kPairs][2][XU][64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int pair = wave & (kPairs - 1);
  const bool soft_wave = wave < kPairs;
  const int n = lane & 31;
  const int hh = lane >> 5;

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
  // the workgroup stages, [0, n_w) that this pair of waves computes and
  // [0, fm_w) that no row of the pair masks.
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
    it.iw = i0 + BMW * pair;
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
  // Iteration j handles key tile tile(j).  With ALiBi the tiles are visited
  // from the last to the first: the bias grows with the key index, so the
  // first tile holds the largest bias of each row and the running maximum
  // rarely grows afterwards (each growth beyond the lazy threshold costs a
  // rescale of O^T).  Otherwise the keys run forward.
  auto tile_of = [&](const Item& it, int j) __attribute__((always_inline)) { return REV ? it.nt - 1 - j : j; };

  const std::integral_constant<int, 0> idle;
  const std::integral_constant<int, 1> whole;
  const std::integral_constant<int, 2> masked;

  Item cur;
  if (!item_at(0, cur)) return;

  for (int round = 0;; ++round) {
    const int nt = cur.nt, n_w = cur.n_w, fm_w = cur.fm_w;
    const int iw = cur.iw;
    const int row0 = iw + n;          // this lane's row in row block 0
    const T* kp = reinterpret_cast<const T*>(p.k) + (size_t)cur.kvh * Lk * D;
    const T* vp = reinterpret_cast<const T*>(p.v) + (size_t)cur.kvh * Lk * D;
    auto tile = [&](int j) __attribute__((always_inline)) { return tile_of(cur, j); };
    // Iterations j in [j0, j1), j0 >= 0, of one variant; the loop body is
    // unrolled by kRing so that slots and parities are compile-time choices.
    // Every iteration of every wave ends in one barrier, so the waves of the
    // workgroup stay in step whatever their phase boundaries.
    auto phase = [&](auto& iteration, int j0, int j1, auto var) __attribute__((always_inline)) {
      for (int jb = j0 & ~(kRing - 1); jb < j1; jb += kRing) {
        static_for<kRing>([&](auto kc) __attribute__((always_inline)) {
          const int j = jb + decltype(kc)::value;
          if (j >= j0 && j < j1) iteration(j, var, kc);
        });
      }
    };

    if (soft_wave) {
      // ---- softmax wave: S^T of tile j+1 and the softmax of tile j ----
      Addr ad;
      PF::make_addr_k(ad, lane);
      // Q fragments (B operand of S^T: lane (n, hh) holds Q[row][16 kx + 8 hh
      // + 0..7]) into their AGPRs, negated for a negative scale.
      {
        const T* qp = reinterpret_cast<const T*>(p.q) + (size_t)cur.head * Lq * D;
        static_for<RB * KX>([&](auto ic) {
          constexpr int f = decltype(ic)::value;
          constexpr int rb = f / KX, kx = f % KX;
          const int row = row0 + 32 * rb;
          u32x4 w = {0u, 0u, 0u, 0u};
          if (row < Lq) w = *reinterpret_cast<const u32x4*>(qp + (size_t)row * D + 16 * kx + 8 * hh);
          agpr_write<PF::qagpr(rb, kx) + 0>(w[0] ^ p.qsign);
          agpr_write<PF::qagpr(rb, kx) + 1>(w[1] ^ p.qsign);
          agpr_write<PF::qagpr(rb, kx) + 2>(w[2] ^ p.qsign);
          agpr_write<PF::qagpr(rb, kx) + 3>(w[3] ^ p.qsign);
        });
      }
      State st;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        st.mc[rb] = kMcInit;
        st.alpha[rb] = 1.f;
      }
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
      Probs pr;
      typename PF::template Ring<true> fr;
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      // The first fragments of iteration -1: K_0.
      PF::template prime<true>(fr, lds, ad);
      // Iteration j (from -1; "tile j" below is tile(j)): S^T of tile j+1 from
      // the K slot (j+1) mod kRing, softmax of tile j (VAR 1 whole, 2 masked,
      // 0 none), then, if the tile's maximum moved past the threshold in some
      // row of the wave, the slow path; P and the rescale factors go to the
      // exchange buffer of parity j.  The barrier that ends the iteration
      // publishes them to the P.V wave, whose iteration j+1 uses them.
      auto iteration = [&](int j, auto var, auto slotc) __attribute__((always_inline)) {
        constexpr int VAR = decltype(var)::value;
        constexpr int k = decltype(slotc)::value;   // j mod kRing
        constexpr int par = k & 1;
        const T* kl_use = lds + ((k + 1) % kRing) * TE;   // K_{j+1}
        const T* kl_nxt = lds + ((k + 2) % kRing) * TE;   // K_{j+2}
        if constexpr (VAR != 0) {
          set_tile(j);
          ta.xp = &xch[pair][par][0][lane];
          typename PF::Tmp tp;
          const bool moved = PF::template iterate_s<VAR>(st, sc[par], sc[par ^ 1], pr, fr, kl_use, kl_nxt,
                                                          ad, ta, tp);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) st.alpha[rb] = 1.f;
          if (__builtin_amdgcn_ballot_w64(moved) != 0) PF::resolve(st, sc[par], pr, tp, ta);
          const u32x4 a = {as_u(st.alpha[0]), as_u(st.alpha[1]), 0u, 0u};
          xch[pair][par][2 * RB][lane] = a;
        } else {
          PF::template prime<true>(fr, kl_nxt, ad);
        }
        // 16 wait states between this iteration's last MFMAs and the next
        // iteration's first reads of their results; this wave's LDS traffic
        // complete; then the barrier.
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
      };
      iteration(-1, masked, std::integral_constant<int, kRing - 1>{});
      if constexpr (REV) {
        // Tiles [n_w + 1, nt) first (nothing to do), then n_w (its S^T of
        // tile n_w - 1 is the first needed), the masked tiles [fm_w, n_w), the
        // whole tiles, and the iteration after tile 0.
        const int a = max(0, nt - n_w - 1);
        phase(iteration, 0, a, idle);
        phase(iteration, a, nt - fm_w, masked);
        phase(iteration, nt - fm_w, nt, whole);
        phase(iteration, nt, nt + 1, masked);
      } else {
        phase(iteration, 0, fm_w, whole);
        phase(iteration, max(fm_w, 0), n_w + 1, masked);
        phase(iteration, n_w + 1, nt + 1, idle);
      }
      // The scores of the last iterations are dead, but are kept live past
      // the padding so that their registers are not reused while the MFMAs
      // writing them are in flight.
      hazard_pad();
#pragma unroll
      for (int pb = 0; pb < 2; ++pb)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) keep_live(sc[pb].s[rb]);
    } else {
      // ---- P.V wave: O^T += V^T P^T of tile j-1, and the HBM -> LDS copies ----
      Addr ad;
      PF::make_addr_v(ad, lane);
      // Global offsets of this lane's HBM -> LDS copies (copying wave cw =
      // pair): in copy u the lane writes bytes 16 lane .. 16 lane + 15 of 1 KB
      // block u * kCopyWaves + cw, i.e. chunk position lane % CPR of row
      // (block * 1024 / (2 D) + lane / CPR), and reads the global chunk that
      // the swizzle puts there.
      const int cw = pair;
      int dof[NI];
#pragma unroll
      for (int u = 0; u < NI; ++u) {
        const int blk = u * kCopyWaves + cw;
        const int r = blk * (1024 / (2 * D)) + lane / CPR;
        const int pos = lane % CPR;
        dof[u] = (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T);
      }
      auto copy_tile = [&](const T* base, uint32_t slot, int j) __attribute__((always_inline)) {
        PF::copy_tile(base, slot, tile(j), cur.rows, cw, dof);
      };
      // The V slots of iterations -1 and -2 zeroed (nothing multiplies them:
      // the first P.V iterations are idle, but a zero tile keeps the ring
      // free of stale non-finite values), the copies of the K tiles of
      // iterations 0 .. kRing-2 and of the V tile of iteration 0 issued.
      {
        constexpr int NV16 = TE * (int)sizeof(T) / 16;
        uint4* vz = reinterpret_cast<uint4*>(lds + (kRing + kRing - 2) * TE);   // slots kRing-2, kRing-1
#pragma unroll
        for (int i = tid - kPairs * 64; i < 2 * NV16; i += kPairs * 64) vz[i] = make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < kRing - 1; ++j) copy_tile(kp, kslot(j), j);
      copy_tile(vp, vslot(0), 0);
      static_for<RB * DB * 16>([&](auto ic) { agpr_zero<PF::oagpr(0, 0) + decltype(ic)::value>(); });
      static_for<RB * 4>([&](auto ic) { agpr_zero<kLAgpr + decltype(ic)::value>(); });
      agpr_write<kOnesAgpr>(PF::M::kOnes);
      agpr_write<kOnesAgpr + 1>(PF::M::kOnes);
      typename PF::template Ring<false> fr;
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      // The first fragments of iteration -1: the zeroed V slot of tile -2.
      PF::template prime<false>(fr, lds + (kRing + kRing - 2) * TE, ad);
      // Iteration j: copies of K_{j+kRing} and V_{j+kRing-2}; with VAR 1, P and
      // the rescale factors of tile j-1 from the exchange buffer of parity
      // j-1, the rescale of O^T and l when some factor differs from 1, then
      // P.V of tile j-1 from the V slot (j-1) mod kRing.  A tile's first
      // fragments are read at the end of the iteration before its use, so
      // its copy, issued kRing - 1 iterations before its use into the slot
      // read by the iteration before, must be complete at the barrier that
      // ends the iteration two before its use: vmcnt lets only the current
      // iteration's copies stay in flight (every iteration issues the same
      // number of copies), and lgkmcnt lets the reads of the next
      // iteration's first fragments, which touch neither slot copied into
      // next, cross the barrier.
      auto iteration = [&](int j, auto var, auto slotc) __attribute__((always_inline)) {
        constexpr int VAR = decltype(var)::value;
        constexpr int k = decltype(slotc)::value;   // j mod kRing
        constexpr int par = (k + 1) & 1;            // parity of j - 1
        copy_tile(kp, kslot(k), j + kRing);
        copy_tile(vp, vslot((k + kRing - 2) % kRing), j + kRing - 2);
        const T* vl_use = lds + (kRing + (k + kRing - 1) % kRing) * TE;  // V_{j-1}
        const T* vl_nxt = lds + (kRing + k) * TE;                        // V_j
        if constexpr (VAR != 0) {
          Probs pr;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
              const u32x4 w = xch[pair][par][rb * 2 + cc][lane];
#pragma unroll
              for (int e = 0; e < 4; ++e) pr.w[rb][cc][e] = w[e];
            }
          const u32x4 a = xch[pair][par][2 * RB][lane];
          const float alpha[RB] = {as_f(a[0]), as_f(a[1])};
          if (__builtin_amdgcn_ballot_w64(alpha[0] != 1.f || alpha[1] != 1.f) != 0) PF::repair(alpha);
          PF::iterate_o(pr, fr, vl_use, vl_nxt, ad);
        } else {
          PF::template prime<false>(fr, vl_nxt, ad);
        }
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_waitcnt vmcnt(%0) lgkmcnt(%1)\n\ts_barrier"
                     : : "n"(2 * NI), "n"(PF::kPrimeV) : "memory");
      };
      iteration(-1, idle, std::integral_constant<int, kRing - 1>{});
      if constexpr (REV) {
        // P.V of tile(j-1) = nt - j is needed for nt - n_w < j <= nt.
        phase(iteration, 0, nt - n_w + 1, idle);
        phase(iteration, nt - n_w + 1, nt + 1, whole);
      } else {
        // P.V of tile j-1 is needed for 1 <= j <= n_w.
        phase(iteration, 0, 1, idle);
        phase(iteration, 1, n_w + 1, whole);
        phase(iteration, n_w + 1, nt + 1, idle);
      }

      // Finalize: O = O^T / l, rounded to the input type.  Lane (n, hh) holds
      // head dims 32 db + 8 g + 4 hh + 0..3 of its row.
      hazard_pad();
      float inv[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const float lt = sum_halves(rb == 0 ? agpr_read<kLAgpr>() : agpr_read<kLAgpr + 4>());
        inv[rb] = lt > 0.f ? 1.f / lt : 0.f;
      }
      static_for<RB * DB * 4>([&](auto ic) {
        constexpr int f = decltype(ic)::value;
        constexpr int rb = f / (DB * 4), db = (f / 4) % DB, g = f % 4;
        constexpr int a0 = PF::oagpr(rb, db) + 4 * g;
        uint2 w;
        w.x = PF::E::pack2(agpr_read<a0>() * inv[rb], agpr_read<a0 + 1>() * inv[rb]);
        w.y = PF::E::pack2(agpr_read<a0 + 2>() * inv[rb], agpr_read<a0 + 3>() * inv[rb]);
        const int row = row0 + 32 * rb;
        if (row < Lq) {
          T* op = reinterpret_cast<T*>(p.o) + ((size_t)cur.head * Lq + row) * D;
          *reinterpret_cast<uint2*>(op + 32 * db + 8 * g + 4 * hh) = w;
        }
      });
    }

    Item nxt;
    if (!item_at(round + 1, nxt)) break;
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

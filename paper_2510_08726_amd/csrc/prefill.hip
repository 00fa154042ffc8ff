// Fused attention prefill for gfx950: the loop nest that rolling update
// (Section "Rolling Update", Algorithm 1, Eq. fixed-recurrent) produces from
// the plain attention definition, with the tile structure of the appendix
// "Privatization" (a local max per key tile, then the running max).
//
// Work split.  One workgroup = 8 wave64s = 256 query rows of one (batch,
// query head).  Each wave owns 32 rows for the whole key loop.  Key tiles
// are BN = 64 keys.  Per tile j and wave:
//
//   S^T = K_j . Q^T            32x32x16 MFMAs, K from LDS, Q resident in VGPRs
//   m'  = max(m, rowmax S)     in-lane max + one exchange with lane ^ 32
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
// the S^T accumulator holds keys.
//
// Schedule.  The 8 waves run the tile loop independently between one
// barrier per tile; the two waves sharing a SIMD (rows 32 s and 32 s + 128)
// interleave their MFMA and softmax work.  All 512 threads stage K and V of
// tile j+1 into the other LDS buffer pair while tile j is computed, from
// registers loaded one tile earlier, so the global loads stay in flight
// across a whole tile.

// Lazy repair.  The running max used in the exponent is only moved when a
// row's tile max exceeds it by more than 2^8 (in log2 units); until then the
// stale max keeps every P <= 2^8 (well inside the fp16 / bf16 range) and the
// O^T repair is skipped.  The repaired state is the same as with an always
// moving max, written relative to another reference point; the final
// division by l cancels it.
//
// Scores are in log2 units: t = s * scale * log2(e) (+ ALiBi bias * log2(e)),
// so each exponential is one v_exp_f32.

#include <type_traits>

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 32 * kWaves;             // query rows per workgroup
constexpr int BN = 64;                      // keys per tile
constexpr float kLazyThreshold = 8.f;       // log2 units

// K and V tiles live in LDS row-major, [BN][D], with the 16-byte chunks of
// each row XOR-swizzled: chunk c of row r sits at chunk position c ^ swz(r).
// That keeps the three access patterns conflict free: the staging stores
// (one row per 16 lanes), the K operand reads (16 consecutive rows at one
// chunk) and the transposing V reads (4 consecutive rows x 4 consecutive
// chunks per half-wave).
template <int D>
__device__ __forceinline__ int swz(int r) {
  if (D == 128) return 4 * (r & 3) + ((r >> 2) & 3);
  return 4 * ((r >> 1) & 1) + ((r >> 2) & 3);
}

template <int D>
__device__ __forceinline__ int lds_off(int r, int c) {  // element offset of chunk c of row r
  return r * D + 8 * (c ^ swz<D>(r));
}

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

// Transposing LDS read: within each 16-lane group, output lane i element j is
// element (i % 4) of the 8 bytes addressed by lane (i / 4 + 4 j).
__device__ __forceinline__ uint2 lds_read_tr(const void* p) {
  v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p));
  return __builtin_bit_cast(uint2, r);
}

__device__ __forceinline__ float row_max_across_halves(float x) {
  return fmaxf(x, __shfl_xor(x, 32, 64));
}

__device__ __forceinline__ float row_sum_across_halves(float x) {
  return x + __shfl_xor(x, 32, 64);
}

template <int D, typename T, bool CAUSAL, bool ALIBI>
struct Prefill {
  typedef Elem<T> E;
  typedef typename E::vec8 vec8;
  static constexpr int KX = D / 16;                        // MFMA K-steps of Q.K^T
  static constexpr int DB = D / 32;                        // 32-dim blocks of O^T
  static constexpr int TE = BN * D;                        // elements of one K or V tile

  struct State {
    float m;          // reference max (log2 units of the exponent)
    float l;          // this lane half's share of the exp-sum
    f32x16 o[DB];     // O^T accumulators
  };

  // S^T = K tile . Q^T: s[kb] covers keys 32 kb .. 32 kb + 31.  A operand:
  // lane (n, hh) reads row 32 kb + n, head dims 16 kx + 8 hh .. + 7.
  static __device__ __forceinline__ void qk(f32x16 (&s)[2], const T* ks, const vec8 (&qf)[KX], int n, int hh) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
    for (int kx = 0; kx < KX; ++kx)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {   // the two accumulator chains alternate
        const uint4 a = *reinterpret_cast<const uint4*>(ks + lds_off<D>(32 * kb + n, 2 * kx + hh));
        s[kb] = E::mfma(__builtin_bit_cast(vec8, a), qf[kx], s[kb]);
      }
    // Keep kPre K fragments in flight ahead of the MFMA that consumes them.
    constexpr int kPre = 6;
    __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
    for (int g = 0; g < 2 * KX - kPre; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kPre, 0);
  }

  // O^T += V^T P^T.  The A operand (head dims 32 db + m, 16-key slice c16) is
  // gathered from the row-major V tile with two transposing reads: lane
  // (m, half hh) receives keys 16 c16 + 4 hh + 0..3 and 16 c16 + 8 + 4 hh + 0..3,
  // the order in which the S^T accumulator holds keys in the B operand.
  static __device__ __forceinline__ void pv(State& st, const uint32_t (&pw)[BN / 16][4], const T* vs, int lane) {
    const int G = lane >> 4, i = lane & 15;
    const int hh = G >> 1;
#pragma unroll
    for (int c16 = 0; c16 < BN / 16; ++c16) {
      const vec8 bop = __builtin_bit_cast(vec8, make_uint4(pw[c16][0], pw[c16][1], pw[c16][2], pw[c16][3]));
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int d = 32 * db + 16 * (G & 1) + 4 * (i & 3);   // this source lane's 4 head dims
        const int k = 16 * c16 + 4 * hh + (i >> 2);            // this source lane's key
        const uint2 lo = lds_read_tr(vs + lds_off<D>(k, d >> 3) + (d & 7));
        const uint2 hi = lds_read_tr(vs + lds_off<D>(k + 8, d >> 3) + (d & 7));
        const vec8 a = __builtin_bit_cast(vec8, make_uint4(lo.x, lo.y, hi.x, hi.y));
        st.o[db] = E::mfma(a, bop, st.o[db]);
      }
    }
    // Keep four operands (eight transposing reads) in flight ahead of the MFMAs.
    constexpr int kPre = 4;
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * kPre, 0);
#pragma unroll
    for (int g = 0; g < DB * (BN / 16) - kPre; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, kPre, 0);
  }

  // Softmax of one tile: rolling update of the reference max and l, P packed
  // for the P.V MFMA.  Returns whether the reference max moved (then `alpha`
  // is the repair factor of O^T).  Register r of block kb holds key
  // j0 + 32 kb + 8 (r / 4) + 4 hh + r % 4 of row `row`.
  template <bool MASKED>
  static __device__ __forceinline__ bool softmax(State& st, f32x16 (&s)[2], uint32_t (&pw)[BN / 16][4],
                                                 float& alpha, const float c, const float sl2, int j0, int row,
                                                 int off, int Lk, int hh) {
    const float ce = ALIBI ? 1.f : c;
    float base = 0.f;
    if (ALIBI) base = sl2 * (float)(j0 + 4 * hh - (row + off));
    float tmax = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = s[kb][r];
        if (ALIBI) x = __builtin_fmaf(x, c, __builtin_fmaf(sl2, (float)(32 * kb + 8 * (r / 4) + (r % 4)), base));
        if (MASKED) {
          const int j = j0 + 32 * kb + 8 * (r / 4) + 4 * hh + (r % 4);
          if (j >= Lk || (CAUSAL && j > row + off)) x = kNegInf;
        }
        s[kb][r] = x;
        tmax = fmaxf(tmax, x);
      }
    tmax = row_max_across_halves(tmax);
    const float m = st.m;
    const bool move = (m == kNegInf) ? (tmax != kNegInf) : ((tmax - m) * ce > kLazyThreshold);
    float a = 1.f, mref = m;
    if (move) {
      a = (m == kNegInf) ? 0.f : fast_exp2((m - tmax) * ce);
      mref = tmax;
    }
    st.m = mref;
    alpha = a;
    const float mc = (mref == kNegInf) ? 0.f : mref * ce;
    // The row sum adds the fp32 weights (two partial sums); the packed dot
    // product would sum the rounded weights exactly, but it blocks the MFMA
    // pipe for far longer than plain adds on gfx950.
    float lsum0 = 0.f, lsum1 = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        float p0 = fast_exp2(__builtin_fmaf(s[kb][r], ce, -mc));
        float p1 = fast_exp2(__builtin_fmaf(s[kb][r + 1], ce, -mc));
        if (MASKED) {
          p0 = s[kb][r] == kNegInf ? 0.f : p0;
          p1 = s[kb][r + 1] == kNegInf ? 0.f : p1;
        }
        lsum0 += p0;
        lsum1 += p1;
        pw[2 * kb + r / 8][(r % 8) / 2] = E::pack2(p0, p1);
      }
    const float lsum = lsum0 + lsum1;
    st.l = __builtin_fmaf(st.l, a, lsum);
    return move;
  }
};

template <int D, typename T, bool CAUSAL, bool ALIBI>
__global__ __launch_bounds__(kThreads, 1) void prefill_kernel(PrefillParams p) {
  typedef Prefill<D, T, CAUSAL, ALIBI> PF;
  typedef typename PF::vec8 vec8;
  typedef typename PF::State State;
  constexpr int KX = PF::KX;
  constexpr int TE = PF::TE;
  constexpr int CH = BN * D / 8 / kThreads;   // 16-byte chunks of one tile per thread
  // [K buf 0][K buf 1][V buf 0][V buf 1]
  __shared__ __attribute__((aligned(16))) T smem[4 * TE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31;
  const int hh = lane >> 5;

  // Workgroup -> (query block, head); consecutive logical blocks share an XCD,
  // and within a head the query blocks with the most keys run first.
  int bid = blockIdx.x;
  if (p.xcd_remap) bid = (bid & 7) * (gridDim.x >> 3) + (bid >> 3);
  const int head = bid / p.nqb;
  const int qb = p.nqb - 1 - (bid - head * p.nqb);
  const int b = head / p.Hq;
  const int hq = head - b * p.Hq;
  const int hk = hq / p.group;
  const int Lq = p.Lq, Lk = p.Lk;
  const int off = Lk - Lq;
  const int i0 = qb * BM;
  const int iw = i0 + 32 * wave;   // first row of this wave
  const int row = iw + n;          // this lane's row

  // Tiles: the workgroup stages [0, n_wg); this wave computes [0, n_w); tiles
  // [0, fm_w) need no mask for any of its rows.
  int kend = Lk, kend_w = Lk;
  if (CAUSAL) {
    kend = min(Lk, min(i0 + BM, Lq) + off);
    kend_w = min(Lk, min(iw + 32, Lq) + off);
  }
  if (iw >= Lq) kend_w = 0;
  const int n_wg = kend > 0 ? (kend + BN - 1) / BN : 0;
  const int n_w = kend_w > 0 ? (kend_w + BN - 1) / BN : 0;
  int fm_w = Lk / BN;
  if (CAUSAL) fm_w = min(fm_w, max(0, (iw + off + 1) / BN));
  fm_w = min(fm_w, n_w);

  const T* qp = reinterpret_cast<const T*>(p.q) + (size_t)head * Lq * D;
  const T* kp = reinterpret_cast<const T*>(p.k) + (size_t)(b * p.Hkv + hk) * Lk * D;
  const T* vp = reinterpret_cast<const T*>(p.v) + (size_t)(b * p.Hkv + hk) * Lk * D;

  // Q fragments (B operand of S^T): lane (n, hh) holds Q[row][16 kx + 8 hh + 0..7].
  vec8 qf[KX];
#pragma unroll
  for (int kx = 0; kx < KX; ++kx) {
    uint4 w = make_uint4(0, 0, 0, 0);
    if (row < Lq) w = *reinterpret_cast<const uint4*>(qp + (size_t)row * D + 16 * kx + 8 * hh);
    w.x ^= p.qsign; w.y ^= p.qsign; w.z ^= p.qsign; w.w ^= p.qsign;
    qf[kx] = __builtin_bit_cast(vec8, w);
  }

  T* const kbuf = smem;
  T* const vbuf = smem + 2 * TE;

  // Staging of K and V tiles through registers, one tile ahead: thread t owns
  // chunks idx = c * 512 + t (row idx / (D/8), chunk idx % (D/8)), so 16
  // lanes read one 256-byte row.  Loads go through buffer resources bounded
  // at the head's Lk rows: rows past Lk read as zero (such keys are always
  // masked), and the per-lane offsets are loop invariant.
  const __amdgpu_buffer_rsrc_t krs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(kp), (short)0, Lk * D * (int)sizeof(T), 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(vp), (short)0, Lk * D * (int)sizeof(T), 0x00020000);
  int goff[CH], loff[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    const int idx = c * kThreads + tid;
    const int r = idx / (D / 8), ch = idx % (D / 8);
    goff[c] = (r * D + ch * 8) * (int)sizeof(T);
    loff[c] = lds_off<D>(r, ch);
  }
  u32x4 kst[CH], vst[CH];
  // The tile offset is folded into the per-lane (VGPR) offset, which the
  // buffer range check covers, so rows at or past Lk read as zero.
  auto sload = [&](int t) {
    const unsigned tk = (unsigned)t * (unsigned)(BN * D * sizeof(T));
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      kst[c] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(krs, (int)(tk + goff[c]), 0, 0));
      vst[c] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vrs, (int)(tk + goff[c]), 0, 0));
    }
  };
  auto sstore = [&](int par) {
    T* kd = kbuf + par * TE;
    T* vd = vbuf + par * TE;
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      *reinterpret_cast<u32x4*>(kd + loff[c]) = kst[c];
      *reinterpret_cast<u32x4*>(vd + loff[c]) = vst[c];
    }
  };

  State st;
  st.m = kNegInf;
  st.l = 0.f;
#pragma unroll
  for (int db = 0; db < PF::DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) st.o[db][r] = 0.f;

  const float c = p.c;
  float sl2 = 0.f;
  if (ALIBI) sl2 = p.slopes[hq] * kLog2e;

  f32x16 s[2];
  uint32_t pw[BN / 16][4];

  if (n_wg > 0) {
    sload(0);
    sstore(0);
    sload(1);
  }
  __syncthreads();

  // Tile j lives in LDS buffer pair j & 1; the loop is unrolled by two so the
  // buffer offsets are compile-time constants.
  auto step = [&](int j, auto parity) {
    constexpr int par = decltype(parity)::value;
    const T* kc = kbuf + par * TE;
    const T* vc = vbuf + par * TE;
    if (j < n_w) {
      PF::qk(s, kc, qf, n, hh);
      float alpha = 1.f;
      bool moved;
      if (j < fm_w)
        moved = PF::template softmax<false>(st, s, pw, alpha, c, sl2, j * BN, row, off, Lk, hh);
      else
        moved = PF::template softmax<true>(st, s, pw, alpha, c, sl2, j * BN, row, off, Lk, hh);
      if (moved) {
#pragma unroll
        for (int db = 0; db < PF::DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) st.o[db][r] *= alpha;
      }
      PF::pv(st, pw, vc, lane);
    }
    // Tile j+1 goes into the other buffer pair (last read in step j-1); then
    // the loads of tile j+2 are issued and stay in flight across the barrier.
    if (j + 1 < n_wg) sstore(par ^ 1);
    sload(j + 2);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
  int j = 0;
  for (; j + 1 < n_wg; j += 2) {
    step(j, std::integral_constant<int, 0>{});
    step(j + 1, std::integral_constant<int, 1>{});
  }
  if (j < n_wg) step(j, std::integral_constant<int, 0>{});

  // Finalize: O = O^T / l, rounded to the input type.  Lane (n, hh) holds
  // head dims 32 db + 8 g + 4 hh + 0..3 of its row.
  const float lt = row_sum_across_halves(st.l);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (row < Lq) {
    T* op = reinterpret_cast<T*>(p.o) + ((size_t)head * Lq + row) * D;
#pragma unroll
    for (int db = 0; db < PF::DB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 w;
        w.x = PF::E::pack2(st.o[db][4 * g] * inv, st.o[db][4 * g + 1] * inv);
        w.y = PF::E::pack2(st.o[db][4 * g + 2] * inv, st.o[db][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(op + 32 * db + 8 * g + 4 * hh) = w;
      }
  }
}

template <int D, typename T, bool CAUSAL, bool ALIBI>
hipError_t launch_t(const PrefillParams& p, hipStream_t stream) {
  const int nblocks = p.nqb * p.B * p.Hq;
  PrefillParams q = p;
  q.xcd_remap = (nblocks % 8 == 0) ? 1 : 0;
  hipLaunchKernelGGL((prefill_kernel<D, T, CAUSAL, ALIBI>), dim3(nblocks), dim3(kThreads), 0, stream, q);
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

int prefill_block_rows() { return BM; }

hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
  if (p.D == 64) return p.bf16 ? launch_d<64, __bf16>(p, stream) : launch_d<64, _Float16>(p, stream);
  return p.bf16 ? launch_d<128, __bf16>(p, stream) : launch_d<128, _Float16>(p, stream);
}

}  // namespace attn

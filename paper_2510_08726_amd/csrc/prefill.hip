// Fused attention prefill for gfx950: the loop nest that rolling update
// (Section "Rolling Update", Algorithm 1, Eq. fixed-recurrent) produces from
// the plain attention definition, with the tile structure of the appendix
// "Privatization" (a local max per key tile, then the running max).
//
// Work split.  One workgroup = 8 wave64s = 256 query rows of one (batch,
// query head).  Each wave owns 32 rows for the whole key loop; the two waves
// that share a SIMD (waves s and s + 4) own adjacent 32-row blocks.  Key tiles
// are BN = 64 keys.  Per tile j and wave:
//
//   S^T = K_j . Q^T            32x32x16 MFMAs, K from LDS, Q resident in VGPRs
//   m'  = max(m, rowmax S)     in-lane max + one exchange with lane ^ 32
//   a   = exp2(m - m')         the repair factor h(t, r, r') = t exp(r - r')
//   P   = exp2(S - m')         rounded to the input type (the compute
//                              definition casts exp to the input dtype
//                              before the second matmul)
//   l   = a l + rowsum P       summed from the rounded P with v_dot2, so the
//                              weights applied to V sum exactly to l
//   O^T = a O^T + V_j^T . P^T  32x32x16 MFMAs, V^T from LDS, P taken straight
//                              from the S^T accumulator registers
//
// Computing S transposed puts one query row per lane (rows are the MFMA N
// index): row reductions stay in registers, the per-row repair of O^T is a
// per-lane scale, and the fp32 S^T accumulator converts in place into the B
// operand of the P.V product.  V tiles are stored transposed in LDS (keys
// contiguous, permuted inside 16-key slices to the order in which the S^T
// accumulator holds keys), so every MFMA operand is one 16-byte LDS read.
//
// Ping-pong.  The two waves on a SIMD alternate between an MFMA phase and a
// VALU phase, one phase apart, separated by workgroup barriers:
//   MFMA phase of tile j:  S^T of tile j, and the P.V product of tile j-1
//                          (deferred by one tile), plus staging of the next
//                          K or V tile (global -> registers -> LDS)
//   VALU phase of tile j:  softmax of tile j, repair of O^T and l
// While one wave keeps the matrix core busy the other runs the exponentials,
// so MFMA and softmax work overlap on every SIMD.  The repair of O^T by tile
// j's factor always follows the P.V of tile j-1, keeping O^T consistent with
// the running max.
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

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kGroupThreads = 256;          // one ping-pong group = 4 waves, one per SIMD
constexpr int BM = 32 * kWaves;             // query rows per workgroup
constexpr int BN = 64;                      // keys per tile
constexpr int KPAD = 8;                     // elements of padding per K row in LDS
constexpr int VPAD = 8;                     // elements of padding per V^T row in LDS
constexpr float kLazyThreshold = 8.f;       // log2 units

__device__ __forceinline__ float row_max_across_halves(float x) {
  return fmaxf(x, __shfl_xor(x, 32, 64));
}

__device__ __forceinline__ float row_sum_across_halves(float x) {
  return x + __shfl_xor(x, 32, 64);
}

// Column, inside a V^T row, at which the 4-key group q4 (keys 4 q4 .. 4 q4 + 3)
// is stored: within each 16-key slice, key offset 8a + 4h + i goes to
// 8h + 4a + i, so that lane half h finds its 8 keys in one 16-byte chunk.
__device__ __forceinline__ int vt_col(int q4) {
  return 4 * ((q4 & ~3) | ((q4 & 1) << 1) | ((q4 >> 1) & 1));
}

template <int D, typename T, bool CAUSAL, bool ALIBI>
struct Prefill {
  typedef Elem<T> E;
  typedef typename E::vec8 vec8;
  static constexpr int KX = D / 16;                        // MFMA K-steps of Q.K^T
  static constexpr int DB = D / 32;                        // 32-dim blocks of O^T
  static constexpr int KS = BN * (D + KPAD);               // K tile: [BN][D + KPAD]
  static constexpr int VS = D * (BN + VPAD);               // V^T tile: [D][BN + VPAD]
  static constexpr int KCH = BN * D / 8 / kGroupThreads;   // 16-byte K chunks per group thread
  static constexpr int VBL = (BN / 4) * (D / 4) / kGroupThreads;  // 4x4 V blocks per group thread

  struct State {
    float m;          // reference max (log2 units of the exponent)
    float l;          // this lane half's share of the exp-sum
    f32x16 o[DB];     // O^T accumulators
  };

  // S^T = K tile . Q^T: s[kb] covers keys 32 kb .. 32 kb + 31.
  static __device__ __forceinline__ void qk(f32x16 (&s)[2], const T* ks, const vec8 (&qf)[KX], int n, int hh) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
      for (int kx = 0; kx < KX; ++kx) {
        const uint4 a = *reinterpret_cast<const uint4*>(ks + (32 * kb + n) * (D + KPAD) + 16 * kx + 8 * hh);
        s[kb] = E::mfma(__builtin_bit_cast(vec8, a), qf[kx], s[kb]);
      }
    }
  }

  // O^T += V^T P^T; A operand: lane (n, hh) reads V^T[32 db + n][16 c16 + 8 hh .. + 7].
  static __device__ __forceinline__ void pv(State& st, const uint32_t (&pw)[BN / 16][4], const T* vs, int n,
                                            int hh) {
#pragma unroll
    for (int c16 = 0; c16 < BN / 16; ++c16) {
      const vec8 bop = __builtin_bit_cast(vec8, make_uint4(pw[c16][0], pw[c16][1], pw[c16][2], pw[c16][3]));
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const uint4 a = *reinterpret_cast<const uint4*>(vs + (32 * db + n) * (BN + VPAD) + 16 * c16 + 8 * hh);
        st.o[db] = E::mfma(__builtin_bit_cast(vec8, a), bop, st.o[db]);
      }
    }
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
    const uint32_t ones = E::pack2(1.f, 1.f);
    float lsum = 0.f;
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
        const uint32_t w = E::pack2(p0, p1);
        lsum = E::dot2(w, ones, lsum);
        pw[2 * kb + r / 8][(r % 8) / 2] = w;
      }
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
  constexpr int KS = PF::KS, VS = PF::VS;
  constexpr int KCH = PF::KCH, VBL = PF::VBL;
  // [K buf 0][K buf 1][V^T buf 0][V^T buf 1]
  __shared__ __attribute__((aligned(16))) T smem[2 * KS + 2 * VS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = wave >> 2;        // 0: first MFMA phase at phase 0; 1: one phase later
  const int simd = wave & 3;
  const int gt = tid & (kGroupThreads - 1);
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
  const int iw = i0 + 64 * simd + 32 * grp;   // first row of this wave
  const int row = iw + n;                      // this lane's row

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
  T* const vbuf = smem + 2 * KS;

  // Staging.  Group 0 stages K tiles, group 1 stages V tiles (transposed),
  // each through registers loaded one tile ahead.
  uint4 kreg[KCH];
  uint2 vreg[VBL][4];
  auto kload = [&](int t) {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      const int idx = c * kGroupThreads + gt;
      const int key = idx / (D / 8), ch = idx % (D / 8);
      const int g = t * BN + key;
      kreg[c] = (t < n_wg && g < Lk) ? *reinterpret_cast<const uint4*>(kp + (size_t)g * D + ch * 8)
                                     : make_uint4(0, 0, 0, 0);
    }
  };
  auto kstore = [&](int t) {
    T* ks = kbuf + (t & 1) * KS;
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      const int idx = c * kGroupThreads + gt;
      const int key = idx / (D / 8), ch = idx % (D / 8);
      *reinterpret_cast<uint4*>(ks + key * (D + KPAD) + ch * 8) = kreg[c];
    }
  };
  // V block idx -> (kq, dq): 16 consecutive lanes take 16 key groups of one
  // dim group; the two half-waves take dim groups two apart, so the 8-byte
  // stores of a half-wave cover all 64 LDS banks once.
  auto vblock = [&](int bl, int& kq, int& dq) {
    const int idx = bl * kGroupThreads + gt;
    kq = idx & 15;
    const int dl = idx >> 4;
    dq = (dl & ~3) | ((dl & 1) << 1) | ((dl >> 1) & 1);
  };
  auto vload = [&](int t) {
#pragma unroll
    for (int bl = 0; bl < VBL; ++bl) {
      int kq, dq;
      vblock(bl, kq, dq);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int g = t * BN + 4 * kq + kk;
        vreg[bl][kk] = (t < n_wg && g < Lk) ? *reinterpret_cast<const uint2*>(vp + (size_t)g * D + 4 * dq)
                                            : make_uint2(0, 0);
      }
    }
  };
  auto vstore = [&](int t) {
    T* vs = vbuf + (t & 1) * VS;
#pragma unroll
    for (int bl = 0; bl < VBL; ++bl) {
      int kq, dq;
      vblock(bl, kq, dq);
      const uint2* r = vreg[bl];
      // 4 keys x 4 dims of 16-bit values, transposed to 4 dims x 4 keys.
      uint2 t0, t1, t2, t3;
      t0.x = (r[0].x & 0xffffu) | (r[1].x << 16);        t0.y = (r[2].x & 0xffffu) | (r[3].x << 16);
      t1.x = (r[0].x >> 16) | (r[1].x & 0xffff0000u);    t1.y = (r[2].x >> 16) | (r[3].x & 0xffff0000u);
      t2.x = (r[0].y & 0xffffu) | (r[1].y << 16);        t2.y = (r[2].y & 0xffffu) | (r[3].y << 16);
      t3.x = (r[0].y >> 16) | (r[1].y & 0xffff0000u);    t3.y = (r[2].y >> 16) | (r[3].y & 0xffff0000u);
      T* dst = vs + (4 * dq) * (BN + VPAD) + vt_col(kq);
      *reinterpret_cast<uint2*>(dst) = t0;
      *reinterpret_cast<uint2*>(dst + (BN + VPAD)) = t1;
      *reinterpret_cast<uint2*>(dst + 2 * (BN + VPAD)) = t2;
      *reinterpret_cast<uint2*>(dst + 3 * (BN + VPAD)) = t3;
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

  // Prologue: K_0 into LDS (all threads share the chunks), then group 0 holds
  // K_1 in registers and group 1 holds V_0.
  if (grp == 0) {
    kload(0);
    kstore(0);
    kload(1);
  } else {
    vload(0);
  }
  __syncthreads();

  f32x16 s[2];
  uint32_t pw[BN / 16][4];

  // Phase ph: group g runs the MFMA phase of tile (ph - g) / 2 when ph - g is
  // even and the VALU phase of tile (ph - g - 1) / 2 when it is odd.
  const int nphases = 2 * n_wg + 2;
  for (int ph = 0; ph < nphases; ++ph) {
    const int u = ph - grp;
    if (u >= 0 && (u & 1) == 0) {
      const int j = u >> 1;
      // MFMA phase of tile j: P.V of tile j-1 (its P is ready), S^T of tile j.
      if (j >= 1 && j <= n_w) PF::pv(st, pw, vbuf + ((j - 1) & 1) * VS, n, hh);
      if (j < n_w) PF::qk(s, kbuf + (j & 1) * KS, qf, n, hh);
      // staging: group 0 writes K_{j+1} and loads K_{j+2}; group 1 writes V_j and loads V_{j+1}
      if (grp == 0) {
        if (j + 1 < n_wg) kstore(j + 1);
        kload(j + 2);
      } else {
        if (j < n_wg) vstore(j);
        vload(j + 1);
      }
    } else if (u >= 1) {
      const int j = (u - 1) >> 1;
      // VALU phase of tile j.
      if (j < n_w) {
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
      }
    }
    __syncthreads();
  }

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

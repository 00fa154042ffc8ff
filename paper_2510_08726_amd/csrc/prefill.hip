// Fused attention prefill for gfx950: the loop nest that rolling update
// (Section "Rolling Update", Algorithm 1, Eq. fixed-recurrent) produces from
// the plain attention definition, with the tile structure of the appendix
// "Privatization" (local max per key tile, then the running max).
//
// One workgroup = 4 wave64s = 128 query rows of one (batch, query head); each
// wave owns 32 rows for the whole key loop.  Per key tile of BN = 64 keys:
//
//   S^T = K_j . Q^T           32x32x16 MFMA, K from LDS, Q resident in VGPRs
//   m'  = max(m, rowmax S)    in-lane max + one swap with lane ^ 32
//   a   = exp2(m - m')        the repair factor h(t, r, r') = t exp(r - r')
//   P   = exp2(S - m')        rounded to the input type (the compute
//                             definition casts exp to the input dtype before
//                             the second matmul)
//   l   = a l + rowsum P      (sum of the rounded P, so the weights applied to
//                             V sum exactly to the divisor)
//   O^T = a O^T + V_j^T . P^T 32x32x16 MFMA, V^T from LDS, P straight from the
//                             S^T accumulator registers
//
// Computing S transposed puts one query row in each lane (rows are the MFMA
// N index), so the row reductions and the per-row repair of O need no LDS
// round trip, and the fp32 accumulator of S^T converts in place into the B
// operand of the P.V product.  The price is that V must be presented with
// keys contiguous: tiles of V are transposed through registers on their way
// into LDS, with the key order inside each 16-key slice permuted to match the
// order in which the S^T accumulator holds keys.
//
// Scores are kept in log2 units: t = s * scale * log2(e) (+ ALiBi bias *
// log2(e)), so every exponential is a single v_exp_f32.

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int BM = 32 * kWaves;  // query rows per workgroup
constexpr int BN = 64;           // keys per tile
constexpr int KPAD = 8;          // elements of padding per K row in LDS
constexpr int VPAD = 8;          // elements of padding per V^T row in LDS

template <int D>
struct Tile {
  static constexpr int KS = BN * (D + KPAD);   // K tile, [BN][D + KPAD]
  static constexpr int VS = D * (BN + VPAD);   // V^T tile, [D][BN + VPAD]
  static constexpr int STAGE = KS + VS;
  static constexpr int KCHUNKS = BN * D / 8 / kThreads;        // 16-byte K loads per thread
  static constexpr int VBLOCKS = (BN / 4) * (D / 4) / kThreads; // 4x4 V blocks per thread
};

// Position, inside a tile, at which key offset k (0..BN-1) is stored in V^T.
// Within each 16-key slice the key offset 8a + 4h + i is stored at 8h + 4a + i:
// that is the order in which lane half h holds keys in the S^T accumulator.
__device__ __forceinline__ int vt_pos_of_group(int q4) {
  return 4 * ((q4 & ~3) | ((q4 & 1) << 1) | ((q4 >> 1) & 1));
}

template <int D, typename T, bool CAUSAL, bool ALIBI>
__global__ __launch_bounds__(kThreads, 2) void prefill_kernel(PrefillParams p) {
  typedef Elem<T> E;
  typedef typename E::vec8 vec8;
  typedef Tile<D> TL;
  __shared__ __attribute__((aligned(16))) T smem[2 * TL::STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int n = lane & 31;   // MFMA column: this lane's query row within the wave
  const int hh = lane >> 5;  // lane half

  // Workgroup -> (query block, head).  Consecutive logical blocks land on one
  // XCD (dispatch is round-robin over the 8 XCDs), and within a head the
  // query blocks run from the last (most keys under a causal mask) down.
  int bid = blockIdx.x;
  if (p.xcd_remap) bid = (bid & 7) * (gridDim.x >> 3) + (bid >> 3);
  const int head = bid / p.nqb;               // b * Hq + hq
  const int qb = p.nqb - 1 - (bid - head * p.nqb);
  const int b = head / p.Hq;
  const int hq = head - b * p.Hq;
  const int hk = hq / p.group;
  const int Lq = p.Lq, Lk = p.Lk;
  const int off = Lk - Lq;                    // bottom-right causal alignment
  const int i0 = qb * BM;
  const int iw = i0 + wave * 32;
  const int row = iw + n;

  int kend = Lk;      // keys [0, kend) are visible to some row of the workgroup
  int kend_w = Lk;    // ... to some row of this wave
  if (CAUSAL) {
    kend = min(Lk, min(i0 + BM, Lq) + off);
    kend_w = min(Lk, min(iw + 32, Lq) + off);
  }
  if (iw >= Lq) kend_w = 0;
  const int ntiles = kend > 0 ? (kend + BN - 1) / BN : 0;

  const T* qp = reinterpret_cast<const T*>(p.q) + (size_t)head * Lq * D;
  const T* kp = reinterpret_cast<const T*>(p.k) + (size_t)(b * p.Hkv + hk) * Lk * D;
  const T* vp = reinterpret_cast<const T*>(p.v) + (size_t)(b * p.Hkv + hk) * Lk * D;

  // Q fragments, resident for the whole key loop: B operand of S^T = K Q^T,
  // lane (n, hh) holds Q[row][16 ks + 8 hh + 0..7].
  vec8 qf[D / 16];
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    uint4 w = make_uint4(0, 0, 0, 0);
    if (row < Lq) w = *reinterpret_cast<const uint4*>(qp + (size_t)row * D + 16 * ks + 8 * hh);
    w.x ^= p.qsign; w.y ^= p.qsign; w.z ^= p.qsign; w.w ^= p.qsign;
    qf[ks] = __builtin_bit_cast(vec8, w);
  }

  // Register staging of the next K / V tile (global -> VGPR -> LDS).
  uint4 kreg[TL::KCHUNKS];
  uint2 vreg[TL::VBLOCKS][4];
  auto gload = [&](int j0) {
#pragma unroll
    for (int c = 0; c < TL::KCHUNKS; ++c) {
      const int idx = c * kThreads + tid;
      const int key = idx / (D / 8), ch = idx % (D / 8);
      const int g = j0 + key;
      kreg[c] = g < Lk ? *reinterpret_cast<const uint4*>(kp + (size_t)g * D + ch * 8)
                       : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int bl = 0; bl < TL::VBLOCKS; ++bl) {
      const int idx = bl * kThreads + tid;
      const int dq = idx % (D / 4), kq = idx / (D / 4);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int g = j0 + 4 * kq + kk;
        vreg[bl][kk] = g < Lk ? *reinterpret_cast<const uint2*>(vp + (size_t)g * D + 4 * dq)
                              : make_uint2(0, 0);
      }
    }
  };
  auto swrite = [&](int buf) {
    T* ks = smem + buf * TL::STAGE;
    T* vs = ks + TL::KS;
#pragma unroll
    for (int c = 0; c < TL::KCHUNKS; ++c) {
      const int idx = c * kThreads + tid;
      const int key = idx / (D / 8), ch = idx % (D / 8);
      *reinterpret_cast<uint4*>(ks + key * (D + KPAD) + ch * 8) = kreg[c];
    }
#pragma unroll
    for (int bl = 0; bl < TL::VBLOCKS; ++bl) {
      const int idx = bl * kThreads + tid;
      const int dq = idx % (D / 4), kq = idx / (D / 4);
      const int pos = vt_pos_of_group(kq);
      const uint2* r = vreg[bl];
      // 4 keys x 4 dims of 16-bit values, transposed to 4 dims x 4 keys.
      uint2 t0, t1, t2, t3;
      t0.x = (r[0].x & 0xffffu) | (r[1].x << 16);  t0.y = (r[2].x & 0xffffu) | (r[3].x << 16);
      t1.x = (r[0].x >> 16) | (r[1].x & 0xffff0000u);  t1.y = (r[2].x >> 16) | (r[3].x & 0xffff0000u);
      t2.x = (r[0].y & 0xffffu) | (r[1].y << 16);  t2.y = (r[2].y & 0xffffu) | (r[3].y << 16);
      t3.x = (r[0].y >> 16) | (r[1].y & 0xffff0000u);  t3.y = (r[2].y >> 16) | (r[3].y & 0xffff0000u);
      T* dst = vs + (4 * dq) * (BN + VPAD) + pos;
      *reinterpret_cast<uint2*>(dst) = t0;
      *reinterpret_cast<uint2*>(dst + (BN + VPAD)) = t1;
      *reinterpret_cast<uint2*>(dst + 2 * (BN + VPAD)) = t2;
      *reinterpret_cast<uint2*>(dst + 3 * (BN + VPAD)) = t3;
    }
  };

  // Running state of this lane's row: max m (log2 units), this lane half's
  // share of the exp-sum l, and O^T (lane = row, registers = head dims).
  float m = kNegInf, l = 0.f;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;

  // Score scaling.  Without ALiBi, t = s and the scale is applied inside the
  // exponent (exp2(s c - m c)), which needs c >= 0: a negative scale is
  // folded into the sign of Q by the host (qsign).  With ALiBi, t = s c + bias
  // is formed explicitly and the exponent scale is 1.
  const float c = p.c;
  const float ce = ALIBI ? 1.f : c;
  float sl2 = 0.f;
  if (ALIBI) sl2 = p.slopes[hq] * kLog2e;

  if (ntiles > 0) {
    gload(0);
    swrite(0);
  }
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int j0 = t * BN;
    const int buf = t & 1;
    if (t + 1 < ntiles) gload(j0 + BN);

    if (j0 < kend_w) {
      const T* ks = smem + buf * TL::STAGE;
      const T* vs = ks + TL::KS;

      // S^T tile: lane (n, hh), register r of block kb holds the score of
      // query row `row` and key j0 + 32 kb + 8 (r / 4) + 4 hh + r % 4.
      f32x16 s[BN / 32];
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
        for (int kx = 0; kx < D / 16; ++kx) {
          const uint4 a = *reinterpret_cast<const uint4*>(ks + (32 * kb + n) * (D + KPAD) + 16 * kx + 8 * hh);
          s[kb] = E::mfma(__builtin_bit_cast(vec8, a), qf[kx], s[kb]);
        }
      }

      // Score epilogue: scale / ALiBi bias, mask, local (tile) max.
      const bool masked_tile = (j0 + BN > Lk) || (CAUSAL && j0 + BN - 1 > iw + off);
      float base = 0.f;
      if (ALIBI) base = sl2 * (float)(j0 + 4 * hh - (row + off));
      float tmax = kNegInf;
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = s[kb][r];
          if (ALIBI) x = __builtin_fmaf(x, c, __builtin_fmaf(sl2, (float)(32 * kb + 8 * (r / 4) + (r % 4)), base));
          if (masked_tile) {
            const int j = j0 + 32 * kb + 8 * (r / 4) + 4 * hh + (r % 4);
            if (j >= Lk || (CAUSAL && j > row + off)) x = kNegInf;
          }
          s[kb][r] = x;
          tmax = fmaxf(tmax, x);
        }
      tmax = fmaxf(tmax, swap_halves(tmax));

      // Rolling update of the running max and the repair factor.
      const float mnew = fmaxf(m, tmax);
      float alpha, mc;
      if (mnew == kNegInf) {          // nothing visible yet in this row
        alpha = 1.f;
        mc = 0.f;
      } else {
        alpha = (m == kNegInf) ? 0.f : fast_exp2((m - mnew) * ce);
        mc = mnew * ce;
      }
      m = mnew;

      // P = exp2(t - m'), packed to the input type as the B operand of O^T.
      // Register r of block kb is element (r % 8) of the operand for the
      // 16-key slice 2 kb + r / 8.
      uint32_t pw[BN / 16][4];
      float lsum = 0.f;
      const uint32_t ones = E::pack2(1.f, 1.f);
#pragma unroll
      for (int kb = 0; kb < BN / 32; ++kb)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          float p0 = fast_exp2(__builtin_fmaf(s[kb][r], ce, -mc));
          float p1 = fast_exp2(__builtin_fmaf(s[kb][r + 1], ce, -mc));
          if (masked_tile) {
            p0 = s[kb][r] == kNegInf ? 0.f : p0;
            p1 = s[kb][r + 1] == kNegInf ? 0.f : p1;
          }
          const uint32_t w = E::pack2(p0, p1);
          lsum = E::dot2(w, ones, lsum);   // exp-sum of the rounded P
          pw[2 * kb + r / 8][(r % 8) / 2] = w;
        }
      l = __builtin_fmaf(l, alpha, lsum);

#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;

      // O^T += V^T P^T.  A operand: lane (n, hh) reads V^T[32 db + n][16 c + 8 hh ..+7].
#pragma unroll
      for (int c16 = 0; c16 < BN / 16; ++c16) {
        const vec8 bop = __builtin_bit_cast(vec8, make_uint4(pw[c16][0], pw[c16][1], pw[c16][2], pw[c16][3]));
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const uint4 a = *reinterpret_cast<const uint4*>(vs + (32 * db + n) * (BN + VPAD) + 16 * c16 + 8 * hh);
          oacc[db] = E::mfma(__builtin_bit_cast(vec8, a), bop, oacc[db]);
        }
      }
    }

    if (t + 1 < ntiles) swrite(buf ^ 1);
    __syncthreads();
  }

  // Finalize: O = O^T / l, rounded to the input type.  Lane (n, hh) holds
  // head dims 32 db + 8 g + 4 hh + 0..3 of its row.
  const float lt = l + swap_halves(l);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  if (row < Lq) {
    T* op = reinterpret_cast<T*>(p.o) + ((size_t)head * Lq + row) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        uint2 w;
        w.x = E::pack2(oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv);
        w.y = E::pack2(oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv);
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

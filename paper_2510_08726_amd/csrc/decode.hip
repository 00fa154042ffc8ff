// Single-token decode for gfx950: the two loop nests that split-k update
// (Section "Split-K Update", Algorithm 2, Fig. su-result) produces from the
// attention definition when the key reduction is privatised into chunks.
//
//  split kernel    one workgroup per (chunk s, key/value head, batch, query
//                  head group).  It streams its chunk of K and V exactly once
//                  from HBM and runs the LOCAL nests for every query head
//                  that shares the key/value head (grouped-query attention):
//                  chunk max, exp-sum and unnormalised P.V.  These partials
//                  are not repaired; they are written to the workspace.
//  combine kernel  the GLOBAL nests: max over chunks, then every partial is
//                  rescaled by exp(max_l - max_g) (the repair function on the
//                  right of the reducer, Eq. su:rewrite) and summed.
//
// Decode moves ~1 flop per byte, so the split kernel is an HBM stream: each
// key row (D * 2 bytes) is read by D / 8 lanes with 16-byte loads, the dot
// products use v_dot2 on packed pairs, and the per-key partial dot is
// reduced across those lanes with DPP.  Inside a workgroup every lane group
// keeps its own online-softmax state over its keys; the groups are merged
// once at the end.
//
// K and V are read once per call, so both kernels load them nontemporally
// (the nt cache policy: streamed past the caches instead of displacing what
// they hold), which measured 10-15 % faster than ordinary loads.

#include <mutex>

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

// Decode workspace of attn_decode_noalloc, for callers that cannot allocate:
// one array per device, loaded with this code object and held until the
// process ends.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in); it uses the device address that
// hipGetSymbolAddress returns for the current device, kept per device.
static __device__ __align__(256) char scratch[kDecodeScratchBytes];
constexpr int kMaxDevices = 64;

constexpr int kThreads = 256;
constexpr int kUnroll = 4;  // keys per lane group per step (loads in flight)

// Sum over aligned groups of LPK lanes (LPK = 8 or 16); every lane of the
// group receives the sum.  quad_perm swaps lanes ^1 and ^2, row_half_mirror
// pairs the two quads of an 8-lane half row, row_mirror the two halves of a
// 16-lane row.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}

template <int LPK>
__device__ __forceinline__ float group_sum(float x) {
  x += dpp_move<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp_move<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp_move<0x141>(x);  // row_half_mirror
  if (LPK == 16) x += dpp_move<0x140>(x);  // row_mirror
  return x;
}

template <int D, typename T, int GH, bool ALIBI, bool CAP>
__global__ __launch_bounds__(kThreads) void decode_split_kernel(DecodeParams p) {
  typedef Elem<T> E;
  constexpr int LPK = D / 8;               // lanes per key row
  constexpr int GPW = 64 / LPK;            // lane groups per wave
  constexpr int NG = GPW * (kThreads / 64);  // lane groups per workgroup

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int lig = lane % LPK;              // lane within its group: dims 8 lig .. 8 lig + 7
  const int grp = wave * GPW + lane / LPK;  // group index in the workgroup

  const int S = p.splits;
  const int ngrp = p.group / GH;
  int bid = blockIdx.x;
  const int s = bid % S;  bid /= S;
  const int hg = bid % ngrp;  bid /= ngrp;
  const int hk = bid % p.Hkv;
  const int b = bid / p.Hkv;
  const int hq0 = hk * p.group + hg * GH;   // first query head of this workgroup
  const int Lk = p.Lk;
  const int ks = min(s * p.chunk, Lk);
  const int ke = min(ks + p.chunk, Lk);

  const T* kp = reinterpret_cast<const T*>(p.k) + (size_t)(b * p.Hkv + hk) * Lk * D + 8 * lig;
  const T* vp = reinterpret_cast<const T*>(p.v) + (size_t)(b * p.Hkv + hk) * Lk * D + 8 * lig;

  // Query rows of the GH heads (packed pairs), the scale is applied after the dot.
  uint4 qv[GH];
  float sl2[GH];
#pragma unroll
  for (int g = 0; g < GH; ++g) {
    const T* qp = reinterpret_cast<const T*>(p.q) + ((size_t)b * p.Hq + hq0 + g) * D + 8 * lig;
    qv[g] = *reinterpret_cast<const uint4*>(qp);
    sl2[g] = ALIBI ? p.slopes[hq0 + g] * kLog2e : 0.f;
  }

  float m[GH], l[GH], o[GH][8];
#pragma unroll
  for (int g = 0; g < GH; ++g) {
    m[g] = kNegInf;
    l[g] = 0.f;
#pragma unroll
    for (int d = 0; d < 8; ++d) o[g][d] = 0.f;
  }

  const float c = p.c;
  for (int base = ks; base < ke; base += NG * kUnroll) {
    uint4 kr[kUnroll], vr[kUnroll];
    int key[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      key[u] = base + u * NG + grp;
      const bool ok = key[u] < ke;
      if (ok) {
        const u32x4 k4 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + (size_t)key[u] * D));
        const u32x4 v4 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vp + (size_t)key[u] * D));
        kr[u] = make_uint4(k4[0], k4[1], k4[2], k4[3]);
        vr[u] = make_uint4(v4[0], v4[1], v4[2], v4[3]);
      } else {
        kr[u] = make_uint4(0, 0, 0, 0);
        vr[u] = make_uint4(0, 0, 0, 0);
      }
    }
    float vf[kUnroll][8];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      vf[u][0] = E::lo(vr[u].x); vf[u][1] = E::hi(vr[u].x);
      vf[u][2] = E::lo(vr[u].y); vf[u][3] = E::hi(vr[u].y);
      vf[u][4] = E::lo(vr[u].z); vf[u][5] = E::hi(vr[u].z);
      vf[u][6] = E::lo(vr[u].w); vf[u][7] = E::hi(vr[u].w);
    }
#pragma unroll
    for (int g = 0; g < GH; ++g) {
      float sc[kUnroll];
      float mt = kNegInf;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float part = E::dot2(qv[g].x, kr[u].x, 0.f);
        part = E::dot2(qv[g].y, kr[u].y, part);
        part = E::dot2(qv[g].z, kr[u].z, part);
        part = E::dot2(qv[g].w, kr[u].w, part);
        float x = group_sum<LPK>(part) * c;
        if (CAP) x = soft_cap(x, p.cap_k2, p.cap_cl);
        if (ALIBI) x = __builtin_fmaf(sl2[g], (float)(key[u] - (Lk - 1)), x);
        sc[u] = key[u] < ke ? x : kNegInf;
        mt = fmaxf(mt, sc[u]);
      }
      const float mnew = fmaxf(m[g], mt);
      if (mnew != kNegInf) {
        const float alpha = m[g] == kNegInf ? 0.f : fast_exp2(m[g] - mnew);
        float ps = 0.f;
        float pu[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          pu[u] = sc[u] == kNegInf ? 0.f : fast_exp2(sc[u] - mnew);
          ps += pu[u];
        }
        l[g] = __builtin_fmaf(l[g], alpha, ps);
#pragma unroll
        for (int d = 0; d < 8; ++d) {
          float acc = o[g][d] * alpha;
#pragma unroll
          for (int u = 0; u < kUnroll; ++u) acc = __builtin_fmaf(pu[u], vf[u][d], acc);
          o[g][d] = acc;
        }
        m[g] = mnew;
      }
    }
  }

  // Merge the lane groups of each wave (lanes LPK apart), then the 4 waves
  // through LDS.  All in log2 units.
  __shared__ float sh_m[4][GH];
  __shared__ float sh_l[4][GH];
  __shared__ float sh_o[4][GH][D];
#pragma unroll
  for (int g = 0; g < GH; ++g) {
    float M = m[g];
#pragma unroll
    for (int x = LPK; x < 64; x <<= 1) M = fmaxf(M, __shfl_xor(M, x, 64));
    const float w = (m[g] == kNegInf) ? 0.f : fast_exp2(m[g] - M);
    float L = l[g] * w;
#pragma unroll
    for (int x = LPK; x < 64; x <<= 1) L += __shfl_xor(L, x, 64);
    float ov[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      float v = o[g][d] * w;
#pragma unroll
      for (int x = LPK; x < 64; x <<= 1) v += __shfl_xor(v, x, 64);
      ov[d] = v;
    }
    if (lane < LPK) {
#pragma unroll
      for (int d = 0; d < 8; ++d) sh_o[wave][g][8 * lig + d] = ov[d];
      if (lig == 0) {
        sh_m[wave][g] = M;
        sh_l[wave][g] = L;
      }
    }
  }
  __syncthreads();

  const size_t rowbase = (size_t)b * p.Hq + hq0;
  for (int idx = tid; idx < GH * D; idx += kThreads) {
    const int g = idx / D, d = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, sh_m[w][g]);
    float L = 0.f, acc = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float mw = sh_m[w][g];
        const float f = mw == kNegInf ? 0.f : fast_exp2(mw - M);
        L = __builtin_fmaf(sh_l[w][g], f, L);
        acc = __builtin_fmaf(sh_o[w][g][d], f, acc);
      }
    }
    const size_t slot = (rowbase + g) * S + s;
    p.ws_o[slot * D + d] = acc;
    if (d == 0) {
      p.ws_m[slot] = M == kNegInf ? kNegInf : M * kLn2;   // natural-log units
      p.ws_l[slot] = L;
    }
    // One chunk: this partial is the whole row, and the output is what the
    // combine kernel would compute from it (weight exp(0) = 1), which then
    // does not run.
    if (S == 1) reinterpret_cast<T*>(p.o)[(rowbase + g) * D + d] = (T)(L > 0.f ? acc / L : 0.f);
  }
}

// Grouped-query decode on the matrix unit.  One workgroup per (chunk s, key/
// value head, batch) serves all G = Hq / Hkv query heads of the key/value
// head (G <= 32).  The heads are the N columns of 32x32x16 MFMAs:
//   S^T = K . Q^T     (32 keys x G heads per tile; columns >= G hold zero Q)
//   O^T += V^T . P^T  (head dims x G heads)
// so the per-key work left on the VALU is the softmax of 16 keys per lane.
// The chunk is split into four contiguous key ranges, one per wave; each wave
// streams its keys in 32-key tiles into a wave-private, double-buffered LDS
// region with buffer loads that write LDS directly (K and V tiles in the
// swizzled row-major layout, K read back as operand fragments, V through the
// transposing LDS read), and keeps an online-softmax state per head column.
// The four waves' states are merged at the end into the same partials as the
// vector kernel writes.  P is rounded to the input type as the MFMA operand
// (the compute definition casts exp to the input type before the second
// matmul), while the chunk's exp-sum l is accumulated from the fp32 values,
// as that definition sums them.
template <int D, typename T, bool ALIBI, bool CAP>
__global__ __launch_bounds__(kThreads) void decode_mfma_kernel(DecodeParams p) {
  typedef Elem<T> E;
  typedef typename E::vec8 vec8;
  constexpr int KX = D / 16;                 // MFMA K-steps of K.Q^T
  constexpr int DB = D / 32;                 // 32-dim blocks of O^T
  constexpr int TN = 32;                     // keys per tile
  constexpr int TB = TN * D * (int)sizeof(T);  // bytes of a K or V tile
  constexpr int NBLK = TB / 1024;            // 1 KB copies per tile
  constexpr int CPR = D / 8;                 // 16-byte chunks per row
  // LDS: per wave, two buffers of (K tile, V tile).  After the key loop the
  // same memory holds the merge: o [4][32][D] floats, then m and l [4][32].
  constexpr int kLdsBytes = 4 * 2 * 2 * TB;
  static_assert(4 * 32 * D * 4 + 2 * 4 * 32 * 4 <= kLdsBytes, "merge fits the tile buffers");
  __shared__ __attribute__((aligned(1024))) char lds[kLdsBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, hh = lane >> 5;

  const int S = p.splits;
  const int G = p.group;
  int bid = blockIdx.x;
  const int s = bid % S;  bid /= S;
  const int hk = bid % p.Hkv;
  const int b = bid / p.Hkv;
  const int hq0 = hk * G;
  const int Lk = p.Lk;
  const int ks = min(s * p.chunk, Lk);
  const int ke = min(ks + p.chunk, Lk);
  const int per = (ke - ks + 4 * TN - 1) / (4 * TN) * TN;   // keys per wave, whole tiles
  const int kw0 = min(ks + wave * per, ke);
  const int kw1 = min(kw0 + per, ke);
  const int ntile = (kw1 - kw0 + TN - 1) / TN;

  const T* kbase = reinterpret_cast<const T*>(p.k) + (size_t)(b * p.Hkv + hk) * Lk * D;
  const T* vbase = reinterpret_cast<const T*>(p.v) + (size_t)(b * p.Hkv + hk) * Lk * D;
  char* const wl = lds + wave * 2 * 2 * TB;                 // this wave's buffers
  const uint32_t wl_addr = (uint32_t)(uintptr_t)(lds_void*)wl;

  // Copy of tile t (keys kw0 + 32 t ..) into buffer bf: block blk of a tile
  // holds rows blk * 1024 / (2 D) + lane / CPR, chunk position lane % CPR,
  // filled from the global chunk the swizzle puts there; keys at or past kw1
  // read as zero.
  int goff[NBLK];
#pragma unroll
  for (int blk = 0; blk < NBLK; ++blk) {
    const int r = blk * (1024 / (2 * D)) + lane / CPR;
    const int pos = lane % CPR;
    goff[blk] = (r * D + 8 * (pos ^ swz<D>(r))) * (int)sizeof(T);
  }
  auto copy_tile = [&](int t, int bf) __attribute__((always_inline)) {
    const int k0 = kw0 + TN * t;
    const int left = min(max(kw1 - k0, 0), TN) * D * (int)sizeof(T);
#pragma unroll
    for (int kv = 0; kv < 2; ++kv) {
      const uint64_t a = reinterpret_cast<uint64_t>((kv == 0 ? kbase : vbase) + (size_t)k0 * D);
      const u32x4 rsrc = {(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                          (uint32_t)__builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
                          (uint32_t)__builtin_amdgcn_readfirstlane(left), 0x00020000u};
      const uint32_t dst = wl_addr + (uint32_t)((bf * 2 + kv) * TB);
#pragma unroll
      for (int blk = 0; blk < NBLK; ++blk)
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
                     : : "s"(dst + (uint32_t)(blk * 1024)), "v"(goff[blk]), "s"(rsrc) : "memory", "m0");
    }
  };

  // Per-lane LDS offsets: K fragment kx (lane (n, hh): key n, dims 16 kx +
  // 8 hh .. + 7) and V^T fragment (c16, db) (see the prefill kernel).
  int ak[KX], av[DB][2];
#pragma unroll
  for (int kx = 0; kx < KX; ++kx) ak[kx] = 2 * (n * D + 8 * ((2 * kx + hh) ^ swz<D>(n)));
  {
    const int Gq = lane >> 4, i = lane & 15;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int lh = 0; lh < 2; ++lh) {
        const int d = 32 * db + 16 * (Gq & 1) + 4 * (i & 3);
        const int k = 4 * (Gq >> 1) + (i >> 2) + 8 * lh;
        av[db][lh] = 2 * (k * D + 8 * ((d >> 3) ^ swz<D>(k)) + (d & 7));
      }
  }

  // Q^T as the B operand: lane (n, hh) holds Q[head hq0 + n][16 kx + 8 hh ..]
  // for n < G, zero otherwise.
  vec8 qf[KX];
  {
    const T* qp = reinterpret_cast<const T*>(p.q) + ((size_t)b * p.Hq + hq0 + n) * D;
#pragma unroll
    for (int kx = 0; kx < KX; ++kx) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (n < G) w = *reinterpret_cast<const u32x4*>(qp + 16 * kx + 8 * hh);
      qf[kx] = __builtin_bit_cast(vec8, w);
    }
  }
  const float c = p.c;
  const float sl2 = (ALIBI && n < G) ? p.slopes[hq0 + n] * kLog2e : 0.f;

  float m = kNegInf, l = 0.f;      // log2 units; l: this lane's half of the keys
  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16{};

  if (ntile > 0) copy_tile(0, 0);
  if (ntile > 1) copy_tile(1, 1);
  for (int t = 0; t < ntile; ++t) {
    const int bf = t & 1;
    if (t + 1 < ntile) asm volatile("s_waitcnt vmcnt(%0)" : : "n"(2 * NBLK) : "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const char* kt = wl + (bf * 2) * TB;
    const char* vt = wl + (bf * 2 + 1) * TB;

    f32x16 sacc = f32x16{};
#pragma unroll
    for (int kx = 0; kx < KX; ++kx) {
      const vec8 kf = __builtin_bit_cast(vec8, *reinterpret_cast<const u32x4*>(kt + ak[kx]));
      sacc = E::mfma(kf, qf[kx], sacc);
    }
    // Register r of lane (n, hh) is key 8 (r / 4) + 4 hh + r % 4 of the tile,
    // head column n.
    const int k0 = kw0 + TN * t;
    float x[16];
    float tmax = kNegInf;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = k0 + 8 * (r / 4) + 4 * hh + (r % 4);
      float v = sacc[r] * c;
      if (CAP) v = soft_cap(v, p.cap_k2, p.cap_cl);
      if (ALIBI) v = __builtin_fmaf(sl2, (float)(key - (Lk - 1)), v);
      x[r] = key < kw1 ? v : kNegInf;
      tmax = fmaxf(tmax, x[r]);
    }
    tmax = fmaxf(tmax, swap_halves(tmax));
    const float mnew = fmaxf(m, tmax);
    const float alpha = (m == kNegInf) ? 0.f : fast_exp2(m - mnew);
    uint32_t w[2][4];
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 16; r += 2) {
      const float p0 = x[r] == kNegInf ? 0.f : fast_exp2(x[r] - mnew);
      const float p1 = x[r + 1] == kNegInf ? 0.f : fast_exp2(x[r + 1] - mnew);
      w[r / 8][(r % 8) / 2] = E::pack2(p0, p1);
      ps += p0 + p1;
    }
    if (mnew != kNegInf) {
      m = mnew;
      l = __builtin_fmaf(l, alpha, ps);
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= alpha;
    }
#pragma unroll
    for (int c16 = 0; c16 < 2; ++c16) {
      const vec8 pb = __builtin_bit_cast(vec8, make_uint4(w[c16][0], w[c16][1], w[c16][2], w[c16][3]));
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const char* base = vt + c16 * 32 * D;
        const uint2 lo = lds_read_tr(base + av[db][0]);
        const uint2 hi = lds_read_tr(base + av[db][1]);
        const vec8 vf = __builtin_bit_cast(vec8, make_uint4(lo.x, lo.y, hi.x, hi.y));
        o[db] = E::mfma(vf, pb, o[db]);
      }
    }
    // Buffer bf is free once this tile's reads have returned.
    if (t + 2 < ntile) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      copy_tile(t + 2, bf);
    }
  }

  // Merge the four waves through LDS (the tile buffers are free after the
  // barrier).  Lane (n, hh) holds O^T[32 db + 8 i + 4 hh + j][head n] in
  // register 4 i + j of block db.
  __syncthreads();
  float* sh_o = reinterpret_cast<float*>(lds);               // [4][32][D]
  float* sh_m = sh_o + 4 * 32 * D;                           // [4][32]
  float* sh_l = sh_m + 4 * 32;                               // [4][32]
  const float lt = l + swap_halves(l);
  if (n < G) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sh_o[(wave * 32 + n) * D + 32 * db + 8 * (r / 4) + 4 * hh + (r % 4)] = o[db][r];
    if (hh == 0) {
      sh_m[wave * 32 + n] = m;
      sh_l[wave * 32 + n] = lt;
    }
  }
  __syncthreads();
  const size_t rowbase = (size_t)b * p.Hq + hq0;
  for (int idx = tid; idx < G * D; idx += kThreads) {
    const int g = idx / D, d = idx % D;
    float M = kNegInf;
#pragma unroll
    for (int wv = 0; wv < 4; ++wv) M = fmaxf(M, sh_m[wv * 32 + g]);
    float L = 0.f, acc = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int wv = 0; wv < 4; ++wv) {
        const float mw = sh_m[wv * 32 + g];
        const float f = mw == kNegInf ? 0.f : fast_exp2(mw - M);
        L = __builtin_fmaf(sh_l[wv * 32 + g], f, L);
        acc = __builtin_fmaf(sh_o[(wv * 32 + g) * D + d], f, acc);
      }
    }
    const size_t slot = (rowbase + g) * S + s;
    p.ws_o[slot * D + d] = acc;
    if (d == 0) {
      p.ws_m[slot] = M == kNegInf ? kNegInf : M * kLn2;   // natural-log units
      p.ws_l[slot] = L;
    }
    // One chunk: this partial is the whole row, and the output is what the
    // combine kernel would compute from it (weight exp(0) = 1), which then
    // does not run.
    if (S == 1) reinterpret_cast<T*>(p.o)[(rowbase + g) * D + d] = (T)(L > 0.f ? acc / L : 0.f);
  }
}

// Global nests: one workgroup per (batch, query head), one thread per head
// dim.  Pass 1 takes max_g over all chunk maxima (a block reduction); pass 2
// computes each chunk's weight exp(max_l - max_g) once into LDS, in batches,
// and sums the weighted partial outputs and sums with all loads in flight.
// The workspace is only read.
template <int D, typename T>
__global__ __launch_bounds__(D) void decode_combine_kernel(DecodeParams p) {
  constexpr int kBatch = 512;
  __shared__ float sh_w[kBatch];
  __shared__ float sh_l[kBatch];
  __shared__ float sh_red[D / 64];
  const int row = blockIdx.x;   // b * Hq + hq
  const int d = threadIdx.x;
  const int S = p.splits;
  const float* mp = p.ws_m + (size_t)row * S;
  const float* lp = p.ws_l + (size_t)row * S;
  const float* op = p.ws_o + (size_t)row * S * D + d;

  float mloc = kNegInf;
  for (int s = d; s < S; s += D) mloc = fmaxf(mloc, mp[s]);
#pragma unroll
  for (int x = 32; x >= 1; x >>= 1) mloc = fmaxf(mloc, __shfl_xor(mloc, x, 64));
  if ((d & 63) == 0) sh_red[d >> 6] = mloc;
  __syncthreads();
  float M = kNegInf;
#pragma unroll
  for (int w = 0; w < D / 64; ++w) M = fmaxf(M, sh_red[w]);

  float acc = 0.f, L = 0.f;
  if (M != kNegInf) {
    for (int s0 = 0; s0 < S; s0 += kBatch) {
      const int ns = min(kBatch, S - s0);
      for (int s = d; s < ns; s += D) {
        const float m = mp[s0 + s];
        sh_w[s] = (m == kNegInf) ? 0.f : fast_exp2((m - M) * kLog2e);
        sh_l[s] = lp[s0 + s];
      }
      __syncthreads();
      int s = 0;
      for (; s + 8 <= ns; s += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = op[(size_t)(s0 + s + u) * D];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          acc = __builtin_fmaf(sh_w[s + u], v[u], acc);
          L = __builtin_fmaf(sh_w[s + u], sh_l[s + u], L);
        }
      }
      for (; s < ns; ++s) {
        acc = __builtin_fmaf(sh_w[s], op[(size_t)(s0 + s) * D], acc);
        L = __builtin_fmaf(sh_w[s], sh_l[s], L);
      }
      __syncthreads();
    }
  }
  const float out = L > 0.f ? acc / L : 0.f;
  reinterpret_cast<T*>(p.o)[(size_t)row * D + d] = (T)out;
}

template <int D, typename T, int GH>
hipError_t launch_split(const DecodeParams& p, hipStream_t stream) {
  const int nblocks = p.splits * (p.group / GH) * p.Hkv * p.B;
  const dim3 grid(nblocks), block(kThreads);
  if (p.slopes && p.cap_cl != 0.f)
    hipLaunchKernelGGL((decode_split_kernel<D, T, GH, true, true>), grid, block, 0, stream, p);
  else if (p.slopes)
    hipLaunchKernelGGL((decode_split_kernel<D, T, GH, true, false>), grid, block, 0, stream, p);
  else if (p.cap_cl != 0.f)
    hipLaunchKernelGGL((decode_split_kernel<D, T, GH, false, true>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((decode_split_kernel<D, T, GH, false, false>), grid, block, 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;   // one chunk: the split kernel wrote O
  hipLaunchKernelGGL((decode_combine_kernel<D, T>), dim3(p.B * p.Hq), dim3(D), 0, stream, p);
  return hipGetLastError();
}

template <int D, typename T>
hipError_t launch_mfma(const DecodeParams& p, hipStream_t stream) {
  const int nblocks = p.splits * p.Hkv * p.B;
  const dim3 grid(nblocks), block(kThreads);
  if (p.slopes && p.cap_cl != 0.f)
    hipLaunchKernelGGL((decode_mfma_kernel<D, T, true, true>), grid, block, 0, stream, p);
  else if (p.slopes)
    hipLaunchKernelGGL((decode_mfma_kernel<D, T, true, false>), grid, block, 0, stream, p);
  else if (p.cap_cl != 0.f)
    hipLaunchKernelGGL((decode_mfma_kernel<D, T, false, true>), grid, block, 0, stream, p);
  else
    hipLaunchKernelGGL((decode_mfma_kernel<D, T, false, false>), grid, block, 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;   // one chunk: the split kernel wrote O
  hipLaunchKernelGGL((decode_combine_kernel<D, T>), dim3(p.B * p.Hq), dim3(D), 0, stream, p);
  return hipGetLastError();
}

// Grouped heads (2 <= G <= 32) go to the matrix-unit kernel; single heads to
// the vector kernel, whose lane groups stream key rows with nothing wasted.
template <int D, typename T>
hipError_t launch_g(const DecodeParams& p, hipStream_t stream) {
  switch (decode_split_heads(p.group)) {
    case 0: return launch_mfma<D, T>(p, stream);
    case 8: return launch_split<D, T, 8>(p, stream);
    case 4: return launch_split<D, T, 4>(p, stream);
    case 2: return launch_split<D, T, 2>(p, stream);
    default: return launch_split<D, T, 1>(p, stream);
  }
}

}  // namespace

hipError_t decode_scratch(void** ptr) {
  static std::once_flag once[kMaxDevices];
  static void* addr[kMaxDevices];
  static hipError_t err[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(once[dev], [dev] { err[dev] = hipGetSymbolAddress(&addr[dev], HIP_SYMBOL(scratch)); });
  if (err[dev] != hipSuccess) return err[dev];
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_decode(const DecodeParams& p, hipStream_t stream) {
  if (p.D == 64) return p.bf16 ? launch_g<64, __bf16>(p, stream) : launch_g<64, _Float16>(p, stream);
  return p.bf16 ? launch_g<128, __bf16>(p, stream) : launch_g<128, _Float16>(p, stream);
}

}  // namespace attn

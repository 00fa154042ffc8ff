// Row reductions fused by rolling update and split by split-k update: the
// stable L2 norm and RMSNorm with the row max of its output (the paper's
// second workload; see include/norms.h).  Both are HBM streams: every lane
// reads 16-byte vectors of its row chunk, folds each vector into its state
// with one repaired update (the vector's own max and sum first, the
// privatised local reduction), the lanes' states are combined with the same
// repair, and the chunk partials of a row are combined by a second kernel.
// With one chunk per row the combine is the workgroup's own: the L2 norm
// writes the norm from the first kernel, and RMSNorm, when the row fits in
// the workgroup's registers, writes y from them without reading X again.
//
// Cache policy: X is read once by the L2 norm and by the one-pass RMSNorm,
// and last by RMSNorm's second kernel, so those loads are nontemporal, and
// so are the second kernel's stores of y; RMSNorm's first pass reads X with
// ordinary loads so that the second pass finds what the caches (L2 and the
// memory-side cache) still hold of it.  (The one-pass kernel's stores of y
// are ordinary: 1.5 % faster there.)

#include <type_traits>

#include "kernel_common.h"
#include "launch.h"

namespace attn {

namespace {

constexpr int kNormThreads = 256;
constexpr int kL2RowThreads = 256;   // the L2 norm with one chunk per row
constexpr int kL2RowUnroll = 16;     // its 16-byte loads in flight per lane
constexpr int kRowThreads = 1024;    // the one-pass RMSNorm: one row per workgroup
constexpr int kRowVecs = (int)(kNormRowBytes / (kRowThreads * 16));   // 16-byte vectors per lane
constexpr int kRowBatch = 2;         // of which loaded (and folded) at a time
static_assert(kRowVecs % kRowBatch == 0, "whole batches");
constexpr int kNormUnroll = 8;    // 16-byte loads in flight per lane, first pass
constexpr int kApplyUnroll = 4;   // the same in RMSNorm's second pass

template <bool NT>
static __device__ __forceinline__ u32x4 load16(const u32x4* a) {
  if constexpr (NT) return __builtin_nontemporal_load(a);
  else return *a;
}

template <typename T> struct Vec;
template <> struct Vec<_Float16> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void load(const u32x4& w, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t u = w[i];   // (a bit_cast of the element itself reads element 0 on this compiler)
      const f16x2 h = __builtin_bit_cast(f16x2, u);
      f[2 * i] = (float)h[0];
      f[2 * i + 1] = (float)h[1];
    }
  }
  static __device__ __forceinline__ u32x4 store(const float* f) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = Elem<_Float16>::pack2(f[2 * i], f[2 * i + 1]);
    return w;
  }
};
template <> struct Vec<__bf16> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void load(const u32x4& w, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = Elem<__bf16>::lo(w[i]);
      f[2 * i + 1] = Elem<__bf16>::hi(w[i]);
    }
  }
  static __device__ __forceinline__ u32x4 store(const float* f) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = Elem<__bf16>::pack2(f[2 * i], f[2 * i + 1]);
    return w;
  }
};
template <> struct Vec<float> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void load(const u32x4& w, float* f) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t u = w[i];   // as above
      f[i] = __builtin_bit_cast(float, u);
    }
  }
  static __device__ __forceinline__ u32x4 store(const float* f) {
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float x = f[i];
      w[i] = __builtin_bit_cast(uint32_t, x);
    }
    return w;
  }
};

// The rolling state of one lane and its two updates: fold one vector of VN
// values (privatised: the vector's own reduction, then one repaired global
// update), and merge another state (the split-k combine of two partials).
//
// L2: r = max |x| so far, t = sum of (x / r)^2 so far.
struct L2State {
  float r = 0.f, t = 0.f;
  template <int VN>
  __device__ __forceinline__ void fold(const float* c, float, float) {
    float vm = 0.f;
#pragma unroll
    for (int k = 0; k < VN; ++k) vm = fmaxf(vm, fabsf(c[k]));
    const float rn = fmaxf(r, vm);
    if (rn > 0.f) {                                    // uniform over real data; zeros change nothing
      const float inv = 1.f / rn;
      const float a = r * inv;                         // h: t (r / r')^2
      float tn = t * a * a;
#pragma unroll
      for (int k = 0; k < VN; ++k) {
        const float q = c[k] * inv;                    // g(r', c) = (c / r')^2
        tn = __builtin_fmaf(q, q, tn);
      }
      t = tn;
      r = rn;
    }
  }
  __device__ __forceinline__ void merge(float r2, float t2, float) {
    const float rn = fmaxf(r, r2);
    if (rn > 0.f) {
      const float a = r / rn, b = r2 / rn;
      t = t * a * a + t2 * b * b;
      r = rn;
    }
  }
};

// RMSNorm statistics: r = sum of x^2 / M so far (the running mean), t = max
// of x / sqrt(r + eps) so far.
struct RmsState {
  float r = 0.f, t = kNegInf;
  template <int VN>
  __device__ __forceinline__ void fold(const float* c, float invM, float eps) {
    float s = 0.f, vm = kNegInf;
#pragma unroll
    for (int k = 0; k < VN; ++k) {
      s = __builtin_fmaf(c[k], c[k], s);
      vm = fmaxf(vm, c[k]);
    }
    const float rn = __builtin_fmaf(s, invM, r);
    const float q = __builtin_amdgcn_rsqf(rn + eps);   // 1 / sqrt(r' + eps)
    // h(t, r, r') = t sqrt(r + eps) / sqrt(r' + eps); g(r', c) = c / sqrt(r' + eps).
    // Before the first value t is -inf and stays so under h (also when
    // r + eps = 0, where the factor would be 0).
    t = fmaxf(repair(t, r, q, eps), vm * q);
    r = rn;
  }
  __device__ __forceinline__ void merge(float r2, float t2, float eps) {
    const float rn = r + r2;
    const float q = __builtin_amdgcn_rsqf(rn + eps);
    t = fmaxf(repair(t, r, q, eps), repair(t2, r2, q, eps));
    r = rn;
  }
  // h(t, r, r') with q = 1 / sqrt(r' + eps).
  static __device__ __forceinline__ float repair(float t, float r, float q, float eps) {
    return t == kNegInf ? kNegInf : t * (__builtin_sqrtf(r + eps) * q);
  }
};

template <typename T, bool NT, int NTH, int UNR, typename S>
__device__ __forceinline__ void fold_chunk(const NormParams& p, int n, int c, S& st) {
  constexpr int VN = Vec<T>::N;
  // This chunk's vectors.
  const int v0 = (int)(min((long long)c * p.chunk, (long long)p.M) / VN);
  const int v1 = (int)(min((long long)(c + 1) * p.chunk, (long long)p.M) / VN);
  const u32x4* row = reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(p.x) + (size_t)n * p.M);
  int v = v0 + threadIdx.x;
  for (; v + (UNR - 1) * NTH < v1; v += UNR * NTH) {
    u32x4 w[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) w[u] = load16<NT>(row + v + u * NTH);
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      float f[VN];
      Vec<T>::load(w[u], f);
      st.template fold<VN>(f, p.invM, p.eps);
    }
  }
  for (; v < v1; v += NTH) {
    float f[VN];
    Vec<T>::load(load16<NT>(row + v), f);
    st.template fold<VN>(f, p.invM, p.eps);
  }
}

// Combine the states of the workgroup's NTH lanes (the same repaired merge),
// leaving the result in lane 0 of wave 0.
template <int NTH, typename S>
__device__ __forceinline__ void block_merge(S& st, float eps) {
  __shared__ float sr[NTH / 64], stt[NTH / 64];
#pragma unroll
  for (int x = 32; x >= 1; x >>= 1) {
    const float r2 = __shfl_xor(st.r, x, 64), t2 = __shfl_xor(st.t, x, 64);
    st.merge(r2, t2, eps);
  }
  if ((threadIdx.x & 63) == 0) {
    sr[threadIdx.x >> 6] = st.r;
    stt[threadIdx.x >> 6] = st.t;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int w = 1; w < NTH / 64; ++w) st.merge(sr[w], stt[w], eps);
  }
}

// Local nests: one workgroup per (chunk c, row n) writes its partial (r, t).
template <typename T, bool RMS>
__global__ __launch_bounds__(kNormThreads) void norm_split_kernel(NormParams p) {
  const int c = blockIdx.x % p.chunks, n = blockIdx.x / p.chunks;
  typename std::conditional<RMS, RmsState, L2State>::type st;
  fold_chunk<T, !RMS, kNormThreads, kNormUnroll>(p, n, c, st);
  block_merge<kNormThreads>(st, p.eps);
  if (threadIdx.x == 0) {
    p.ws_r[blockIdx.x] = st.r;
    p.ws_t[blockIdx.x] = st.t;
  }
}

// The L2 norm with one chunk per row: one workgroup of 256 lanes per row, 16
// loads in flight a lane (measured at steady clock on 256 x 2^17 fp32 rows:
// 5.66 TB/s, against 5.36 with 512 lanes and 8 loads, 5.26 with 1024 and 4,
// and less with more or fewer bytes in flight), writes the row's partial and
// its norm.
template <typename T>
__global__ __launch_bounds__(kL2RowThreads) void l2_row_kernel(NormParams p) {
  const int n = blockIdx.x;
  L2State st;
  fold_chunk<T, true, kL2RowThreads, kL2RowUnroll>(p, n, 0, st);
  block_merge<kL2RowThreads>(st, 0.f);
  if (threadIdx.x == 0) {
    p.ws_r[n] = st.r;
    p.ws_t[n] = st.t;
    p.out[n] = st.r * __builtin_sqrtf(st.t);
  }
}

// Global nest of the L2 norm: one thread per row combines its chunks.
__global__ __launch_bounds__(kNormThreads) void l2_combine_kernel(NormParams p) {
  const int n = blockIdx.x * kNormThreads + threadIdx.x;
  if (n >= p.N) return;
  L2State st;
  for (int c = 0; c < p.chunks; ++c) st.merge(p.ws_r[n * p.chunks + c], p.ws_t[n * p.chunks + c], 0.f);
  p.out[n] = st.r * __builtin_sqrtf(st.t);
}

// RMSNorm output: every workgroup (chunk c, row n) combines its row's
// partials (s = the row mean of x^2, m = the row max of y), writes m if it
// holds chunk 0, and writes its chunk of y = x / sqrt(s + eps).
template <typename T>
__global__ __launch_bounds__(kNormThreads) void rms_apply_kernel(NormParams p) {
  constexpr int VN = Vec<T>::N;
  const int c = blockIdx.x % p.chunks, n = blockIdx.x / p.chunks;
  __shared__ float s_q;
  if (threadIdx.x < 64) {
    RmsState st;
    for (int k = threadIdx.x; k < p.chunks; k += 64) st.merge(p.ws_r[n * p.chunks + k], p.ws_t[n * p.chunks + k], p.eps);
#pragma unroll
    for (int x = 32; x >= 1; x >>= 1) {
      const float r2 = __shfl_xor(st.r, x, 64), t2 = __shfl_xor(st.t, x, 64);
      st.merge(r2, t2, p.eps);
    }
    if (threadIdx.x == 0) {
      s_q = 1.f / __builtin_sqrtf(st.r + p.eps);
      if (c == 0) p.out[n] = st.t;
    }
  }
  __syncthreads();
  const float q = s_q;
  const int v0 = (int)(min((long long)c * p.chunk, (long long)p.M) / VN);
  const int v1 = (int)(min((long long)(c + 1) * p.chunk, (long long)p.M) / VN);
  const u32x4* row = reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(p.x) + (size_t)n * p.M);
  u32x4* yrow = reinterpret_cast<u32x4*>(reinterpret_cast<T*>(p.y) + (size_t)n * p.M);
  auto scale = [&](u32x4 w) {
    float f[VN];
    Vec<T>::load(w, f);
#pragma unroll
    for (int k = 0; k < VN; ++k) f[k] *= q;
    return Vec<T>::store(f);
  };
  int v = v0 + threadIdx.x;
  for (; v + (kApplyUnroll - 1) * kNormThreads < v1; v += kApplyUnroll * kNormThreads) {
    u32x4 w[kApplyUnroll];
#pragma unroll
    for (int u = 0; u < kApplyUnroll; ++u) w[u] = load16<true>(row + v + u * kNormThreads);
#pragma unroll
    for (int u = 0; u < kApplyUnroll; ++u) __builtin_nontemporal_store(scale(w[u]), yrow + v + u * kNormThreads);
  }
  for (; v < v1; v += kNormThreads) __builtin_nontemporal_store(scale(load16<true>(row + v)), yrow + v);
}

// One-pass RMSNorm, one workgroup per row of at most kRowThreads x kRowVecs
// vectors: every lane loads its vectors of the row (all loads in flight at
// once) and keeps them in registers, folds them into its state, the lanes'
// states are merged (the row's statistics, written as its one partial and
// its row max), and y is written from the registers.
template <typename T>
__global__ __launch_bounds__(kRowThreads) void rms_row_kernel(NormParams p) {
  constexpr int VN = Vec<T>::N;
  const int n = blockIdx.x;
  const int nv = p.M / VN;
  const u32x4* row = reinterpret_cast<const u32x4*>(reinterpret_cast<const T*>(p.x) + (size_t)n * p.M);
  u32x4* yrow = reinterpret_cast<u32x4*>(reinterpret_cast<T*>(p.y) + (size_t)n * p.M);
  // Rows of exactly kRowThreads x kRowVecs vectors take no per-vector
  // branches (measured 0.8 % faster).
  const bool full = nv == kRowThreads * kRowVecs;
  // The row is read in batches of kRowBatch vectors a lane, each folded
  // before the next is issued (the empty asm with a memory clobber keeps the
  // next batch's loads after the fold): 2 vectors a lane, 32 KiB of loads in
  // flight per workgroup, measured 5.33 TB/s on 256 x 2^17 bf16 rows against
  // 4.78 with the whole row's 16 vectors in flight at once (4 a batch: 5.13;
  // 1: 5.03).
  u32x4 w[kRowVecs];
  RmsState st;
#pragma unroll
  for (int b0 = 0; b0 < kRowVecs; b0 += kRowBatch) {
#pragma unroll
    for (int u = b0; u < b0 + kRowBatch; ++u) {
      const int v = threadIdx.x + u * kRowThreads;
      w[u] = (full || v < nv) ? load16<true>(row + v) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = b0; u < b0 + kRowBatch; ++u) {
      if (full || threadIdx.x + u * kRowThreads < nv) {
        float f[VN];
        Vec<T>::load(w[u], f);
        st.template fold<VN>(f, p.invM, p.eps);
      }
      // Keep the loaded words, not their conversions, live until the stores
      // (half the registers for fp16 and bf16).
      asm volatile("" : "+v"(w[u]));
    }
    asm volatile("" ::: "memory");
  }
  block_merge<kRowThreads>(st, p.eps);
  __shared__ float s_q;
  if (threadIdx.x == 0) {
    p.ws_r[n] = st.r;
    p.ws_t[n] = st.t;
    p.out[n] = st.t;
    s_q = 1.f / __builtin_sqrtf(st.r + p.eps);
  }
  __syncthreads();
  const float q = s_q;
#pragma unroll
  for (int u = 0; u < kRowVecs; ++u) {
    const int v = threadIdx.x + u * kRowThreads;
    if (v < nv) {
      float f[VN];
      Vec<T>::load(w[u], f);
#pragma unroll
      for (int k = 0; k < VN; ++k) f[k] *= q;
      yrow[v] = Vec<T>::store(f);
    }
  }
}

template <typename T>
hipError_t launch_norm_t(const NormParams& p, hipStream_t stream) {
  const dim3 grid(p.N * p.chunks), block(kNormThreads);
  if (norm_one_kernel(p.rms != 0, p.M, (int)sizeof(T), p.chunks)) {
    if (p.rms)
      hipLaunchKernelGGL((rms_row_kernel<T>), grid, dim3(kRowThreads), 0, stream, p);
    else
      hipLaunchKernelGGL((l2_row_kernel<T>), grid, dim3(kL2RowThreads), 0, stream, p);
    return hipGetLastError();
  }
  if (p.rms) {
    hipLaunchKernelGGL((norm_split_kernel<T, true>), grid, block, 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((rms_apply_kernel<T>), grid, block, 0, stream, p);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((norm_split_kernel<T, false>), grid, block, 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(l2_combine_kernel, dim3((p.N + kNormThreads - 1) / kNormThreads), block, 0, stream, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_norm(const NormParams& p, hipStream_t stream) {
  if (p.dtype == 2) return launch_norm_t<float>(p, stream);
  return p.dtype == 1 ? launch_norm_t<__bf16>(p, stream) : launch_norm_t<_Float16>(p, stream);
}

}  // namespace attn

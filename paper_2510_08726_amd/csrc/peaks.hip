// Achievable-peak probes for the attention rooflines (see include/peaks.h):
// a streaming HBM read and an MFMA loop on changing random operands.

#include "../../include/peaks.h"
#include "kernel_common.h"

namespace attn {

namespace {

constexpr int kReadThreads = 256;
constexpr int kReadBlocks = 1024;
constexpr int kReadUnroll = 16;   // 16-byte loads in flight per lane

// Streaming read, one contiguous chunk per workgroup (ceil(words / grid)
// 16-byte words): lane t of the workgroup reads words t, t + 256, ... of its
// chunk, kReadUnroll words at a time.  (A grid-stride order, where the whole
// grid sweeps the buffer together with 4 loads in flight a lane, measured
// 6.16 TB/s against 7.1 for this one.)
__global__ __launch_bounds__(kReadThreads) void hbm_read_kernel(const u32x4* __restrict__ buf, size_t words,
                                                                  float* sink) {
  const size_t per = (words + gridDim.x - 1) / gridDim.x;
  const size_t end = min((size_t)(blockIdx.x + 1) * per, words);
  const size_t n = kReadThreads;
  size_t i = min((size_t)blockIdx.x * per, words) + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kReadUnroll - 1) * n < end; i += kReadUnroll * n) {
    u32x4 w[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) w[u] = __builtin_nontemporal_load(buf + i + u * n);
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= w[u][0] ^ w[u][1] ^ w[u][2] ^ w[u][3];
  }
  for (; i < end; i += n) {
    const u32x4 w = __builtin_nontemporal_load(buf + i);
    acc ^= w[0] ^ w[1] ^ w[2] ^ w[3];
  }
  // One value per workgroup: the XOR of its lanes' words (as a float bit pattern).
  __shared__ uint32_t red[kReadThreads / 64];
  for (int x = 32; x >= 1; x >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, x, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
    for (int w = 0; w < kReadThreads / 64; ++w) r ^= red[w];
    sink[blockIdx.x] = __builtin_bit_cast(float, r & 0x3fffffffu);
  }
}

constexpr int kMfmaThreads = 256;   // 4 waves, one per SIMD
constexpr int kMfmaWgPerCu = 2;     // two waves per SIMD, as the prefill kernel
constexpr int kFrags = 16;          // operand fragments per lane
constexpr int kChains = 4;          // independent accumulators per wave

template <typename T>
__global__ __launch_bounds__(kMfmaThreads, kMfmaWgPerCu) void mfma_loop_kernel(const u32x4* __restrict__ operands,
                                                                               int iters, float* sink,
                                                                               unsigned long long* clocks) {
  typedef Elem<T> E;
  typedef typename E::vec8 vec8;
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kMfmaThreads / 64) + (threadIdx.x >> 6);
  vec8 f[kFrags];
#pragma unroll
  for (int i = 0; i < kFrags; ++i) {
    const u32x4 w = operands[(i * 64 + lane + 7 * wave) % (kFrags * 64 * 4)];
    f[i] = __builtin_bit_cast(vec8, w);
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c) acc[c] = f32x16{};
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
#pragma unroll 1
  for (int it = 0; it < iters; ++it) {
    // 16 MFMAs, each on a different (A, B) pair, accumulators in rotation.
#pragma unroll
    for (int m = 0; m < 16; ++m) acc[m % kChains] = E::mfma(f[m], f[(5 * m + 3) % kFrags], acc[m % kChains]);
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  for (int x = 32; x >= 1; x >>= 1) s += __shfl_xor(s, x, 64);
  if (lane == 0) sink[wave] = s;
  if (wave == 0 && lane == 0) {
    clocks[0] = t1 - t0;
    clocks[1] = r1 - r0;
  }
}

int compute_units_now() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0)
    n = 256;
  return n;
}

}  // namespace

hipError_t launch_hbm_read(const void* buf, size_t bytes, float* sink, hipStream_t stream) {
  hipLaunchKernelGGL(hbm_read_kernel, dim3(kReadBlocks), dim3(kReadThreads), 0, stream,
                     reinterpret_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError();
}

int hbm_read_sink_floats() { return kReadBlocks; }

int mfma_loop_waves() { return compute_units_now() * kMfmaWgPerCu * (kMfmaThreads / 64); }

size_t mfma_loop_operand_bytes() { return (size_t)kFrags * 64 * 4 * 16; }

hipError_t launch_mfma_loop(int bf16, int iters, const void* operands, float* sink, unsigned long long* clocks,
                            hipStream_t stream) {
  const dim3 grid(compute_units_now() * kMfmaWgPerCu), block(kMfmaThreads);
  const u32x4* ops = reinterpret_cast<const u32x4*>(operands);
  if (bf16)
    hipLaunchKernelGGL(mfma_loop_kernel<__bf16>, grid, block, 0, stream, ops, iters, sink, clocks);
  else
    hipLaunchKernelGGL(mfma_loop_kernel<_Float16>, grid, block, 0, stream, ops, iters, sink, clocks);
  return hipGetLastError();
}

}  // namespace attn

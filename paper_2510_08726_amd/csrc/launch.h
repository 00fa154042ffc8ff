// Host-side launch interface between the C ABI (attn_api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>

namespace attn {

struct PrefillParams {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  const float* slopes;  // device, [Hq], or nullptr
  int B, Hq, Hkv, Lq, Lk, D;
  int group;            // Hq / Hkv
  int causal;
  int bf16;
  float c;              // |scale| * log2(e) without ALiBi or SoftCap, scale * log2(e) with either
  unsigned qsign;       // 0x80008000 to negate Q (negative scale, no ALiBi or SoftCap), else 0
  float cap_k2;         // SoftCap: 2 / cap
  float cap_cl;         // SoftCap: cap * log2(e), or 0 for no cap
  int window;           // sliding window (keys per row, causal only), 0 for none
  int nqb;              // query blocks per head
  int nheads;           // B * Hq, set by the launcher
  int nitems;           // nqb * nheads, set by the launcher
  int nxcd;             // XCDs the workgroups are spread over, set by the launcher
  int hg;               // query heads per workgroup (sharing one KV head), set by the launcher
};

struct DecodeParams {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  const float* slopes;  // device, [Hq], or nullptr
  float* ws_o;          // [B*Hq*S, D]
  float* ws_m;          // [B*Hq*S]
  float* ws_l;          // [B*Hq*S]
  int B, Hq, Hkv, Lk, D;
  int group;            // Hq / Hkv
  int splits;           // S
  int chunk;            // ceil(Lk / S)
  int bf16;
  float c;              // scale * log2(e)
  float cap_k2;         // SoftCap: 2 / cap
  float cap_cl;         // SoftCap: cap * log2(e), or 0 for no cap
};

// Template flags of the prefill kernel that a call launches.  SoftCap and the
// sliding window are built for the causal mask (the entry point rejects the
// other combinations), SoftCap without ALiBi.
struct PrefillFlags {
  bool causal, alibi, cap, win;
};
inline PrefillFlags prefill_flags(bool causal, bool alibi, bool cap, bool win) {
  return {causal || cap || win, alibi && !cap, cap, win};
}

// Decode kernel for a GQA group of `group` query heads per KV head: 0 for the
// grouped matrix-unit kernel (2..32 heads), else the heads per workgroup of
// the vector split kernel (the largest of 8, 4, 2, 1 dividing the group).
inline int decode_split_heads(int group) {
  if (group >= 2 && group <= 32) return 0;
  if (group % 8 == 0) return 8;
  if (group % 4 == 0) return 4;
  if (group % 2 == 0) return 2;
  return 1;
}

int prefill_block_rows();
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream);
// One per (head dim, element type); launch_prefill dispatches to them.
hipError_t launch_prefill_d128_f16(const PrefillParams& p, hipStream_t stream);
hipError_t launch_prefill_d128_bf16(const PrefillParams& p, hipStream_t stream);
hipError_t launch_prefill_d64_f16(const PrefillParams& p, hipStream_t stream);
hipError_t launch_prefill_d64_bf16(const PrefillParams& p, hipStream_t stream);
hipError_t launch_decode(const DecodeParams& p, hipStream_t stream);

// Bytes of the static decode workspace of attn_decode_noalloc.
constexpr size_t kDecodeScratchBytes = size_t(16) << 20;
// Device address of that workspace on the current device (resolved once per
// device, then cached).
hipError_t decode_scratch(void** ptr);

// Row reductions (norms.hip): the stable L2 norm, or RMSNorm with its row max.
struct NormParams {
  const void* x;
  void* y;              // RMSNorm output [N, M], or nullptr
  float* out;           // [N]: the norms, or the row maxima of y
  float* ws_r;          // [N * chunks] partials r
  float* ws_t;          // [N * chunks] partials t
  int N, M;
  int chunks;           // chunks per row
  int chunk;            // elements per chunk (whole 16-byte vectors)
  int dtype;            // 0 fp16, 1 bf16, 2 fp32
  int rms;              // 1: RMSNorm with row max, 0: L2 norm
  float eps;
  float invM;           // 1 / M
};
hipError_t launch_norm(const NormParams& p, hipStream_t stream);
// Longest row (bytes) that RMSNorm with one chunk per row holds in the
// registers of one workgroup (1024 lanes x 16 vectors of 16 bytes), reading X once.
constexpr long long kNormRowBytes = 1024LL * 16 * 16;
// True when a row reduction with `chunks` chunks per row runs one kernel
// (one workgroup per row: the L2 norm always, RMSNorm when the row fits)
// rather than the chunk partials and a second kernel.
inline bool norm_one_kernel(bool rms, long long M, int elem, int chunks) {
  return chunks == 1 && (!rms || M * elem <= kNormRowBytes);
}

// Achievable-peak probes (peaks.hip).
hipError_t launch_hbm_read(const void* buf, size_t bytes, float* sink, hipStream_t stream);
int hbm_read_sink_floats();
hipError_t launch_mfma_loop(int bf16, int iters, const void* operands, float* sink, unsigned long long* clocks,
                            hipStream_t stream);
int mfma_loop_waves();
size_t mfma_loop_operand_bytes();

}  // namespace attn

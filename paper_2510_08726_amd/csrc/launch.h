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
  float c;              // |scale| * log2(e) without ALiBi, scale * log2(e) with it
  unsigned qsign;       // 0x80008000 to negate Q (negative scale without ALiBi), else 0
  int nqb;              // query blocks per head
  int xcd_remap;        // set by the launcher
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
};

int prefill_block_rows();
hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream);
hipError_t launch_decode(const DecodeParams& p, hipStream_t stream);

}  // namespace attn

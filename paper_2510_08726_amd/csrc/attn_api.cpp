// C ABI of the fused-attention library: argument validation on the host,
// dispatch to the gfx950 kernels, error reporting.  Every check runs before
// any HIP call, so a rejected call enqueues nothing.

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include "../../include/attn.h"
#include "../../include/peaks.h"
#include "../../include/norms.h"
#include "launch.h"

namespace {

thread_local int g_last_hip_error = 0;

constexpr float kLog2e = 1.4426950408889634f;
constexpr int64_t kMaxGrid = std::numeric_limits<int32_t>::max();
constexpr int kMinChunk = 256;    // keys per decode chunk chosen by the heuristic (one head per KV head)
constexpr int kBlocksPerCu = 1;   // per-head decode workgroups per compute unit chosen by the heuristic
constexpr int kMinChunkGrouped = 128;   // grouped heads: at least one 32-key tile per wave

bool shape_ok(int B, int Hq, int Hkv, int Lq, int Lk) {
  return B >= 1 && Hq >= 1 && Hkv >= 1 && Lq >= 1 && Lk >= 1 && Hq % Hkv == 0;
}

bool dims_supported(int D, attn_dtype dtype) {
  return (D == 64 || D == 128) && (dtype == ATTN_F16 || dtype == ATTN_BF16);
}

// Element counts must stay addressable and the grids within 2^31 - 1 blocks.
bool sizes_fit(int B, int Hq, int Hkv, int Lq, int Lk, int D) {
  const int64_t q = (int64_t)B * Hq * Lq * D;
  const int64_t k = (int64_t)B * Hkv * Lk * D;
  return q < (int64_t(1) << 40) && k < (int64_t(1) << 40);
}

int hip_fail(hipError_t e) {
  g_last_hip_error = (int)e;
  return ATTN_ERR_HIP;
}

// Compute units of the current device (the grouped decode kernel wants one
// workgroup per compute unit: each holds 128 KB of LDS, so more would run one
// after another, each paying its start-up and merge again).
int compute_units() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n <= 0)
    n = 256;
  return n;
}

// Query heads that one decode workgroup serves (the grid divides the group by it).
int decode_heads_per_block(int group) {
  const int gh = attn::decode_split_heads(group);
  return gh == 0 ? group : gh;
}

const char* dtype_name(attn_dtype dtype) { return dtype == ATTN_BF16 ? "bf16" : "f16"; }

int put(char* buf, size_t len, const char* s) {
  const size_t n = std::strlen(s);
  if (!buf || n + 1 > len) return ATTN_ERR_SHAPE;
  std::memcpy(buf, s, n + 1);
  return ATTN_OK;
}

}  // namespace

extern "C" {

const char* attn_status_string(int status) {
  switch (status) {
    case ATTN_OK: return "ATTN_OK: success";
    case ATTN_ERR_NULL: return "ATTN_ERR_NULL: a required pointer is NULL";
    case ATTN_ERR_SHAPE: return "ATTN_ERR_SHAPE: invalid sizes (need B,Hq,Hkv,Lq,Lk >= 1, Hq % Hkv == 0, num_splits >= 0, window >= 0, finite scale, finite softcap >= 0)";
    case ATTN_ERR_UNSUPPORTED: return "ATTN_ERR_UNSUPPORTED: head dim must be 64 or 128 and dtype ATTN_F16 or ATTN_BF16; softcap and window need the causal mask, softcap excludes ALiBi";
    case ATTN_ERR_WORKSPACE: return "ATTN_ERR_WORKSPACE: decode workspace too small (attn_decode_noalloc: the split count needs more than its 16 MiB static workspace)";
    case ATTN_ERR_HIP: return "ATTN_ERR_HIP: a HIP launch failed (see attn_last_hip_error)";
    default: return "unknown attn_status";
  }
}

int attn_last_hip_error(void) { return g_last_hip_error; }

int attn_fwd_mod(const void* Q, const void* K, const void* V, void* O,
                 int B, int Hq, int Hkv, int Lq, int Lk, int D,
                 int causal, float scale, const float* alibi_slopes, float softcap, int window,
                 attn_dtype dtype, hipStream_t stream) {
  if (!Q || !K || !V || !O) return ATTN_ERR_NULL;
  if (!shape_ok(B, Hq, Hkv, Lq, Lk) || !std::isfinite(scale)) return ATTN_ERR_SHAPE;
  if (!std::isfinite(softcap) || softcap < 0.f || window < 0) return ATTN_ERR_SHAPE;
  if (!dims_supported(D, dtype)) return ATTN_ERR_UNSUPPORTED;
  if (softcap > 0.f && (!causal || alibi_slopes)) return ATTN_ERR_UNSUPPORTED;
  if (window > 0 && !causal) return ATTN_ERR_UNSUPPORTED;
  if (!sizes_fit(B, Hq, Hkv, Lq, Lk, D)) return ATTN_ERR_SHAPE;
  // The prefill kernel addresses one head's K and V with 32-bit byte offsets.
  if ((int64_t)Lk * D * 2 >= (int64_t(1) << 31)) return ATTN_ERR_SHAPE;
  const int bm = attn::prefill_block_rows();
  const int64_t nqb = ((int64_t)Lq + bm - 1) / bm;
  if (nqb * B * Hq > kMaxGrid) return ATTN_ERR_SHAPE;

  attn::PrefillParams p{};
  p.q = Q; p.k = K; p.v = V; p.o = O;
  p.slopes = alibi_slopes;
  p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.Lq = Lq; p.Lk = Lk; p.D = D;
  p.group = Hq / Hkv;
  p.causal = causal ? 1 : 0;
  p.bf16 = dtype == ATTN_BF16;
  p.cap_k2 = softcap > 0.f ? 2.f / softcap : 0.f;
  p.cap_cl = softcap > 0.f ? softcap * kLog2e : 0.f;
  p.window = window;
  if (alibi_slopes || softcap > 0.f) {
    p.c = scale * kLog2e;
    p.qsign = 0;
  } else {
    // Kept above zero so that masked (-inf) scores times c stay -inf when
    // scale is 0; exp2(s * 1e-30) rounds to exactly 1 for any finite score,
    // the same weights as c = 0.
    p.c = std::fmax(std::fabs(scale) * kLog2e, 1e-30f);
    p.qsign = std::signbit(scale) ? 0x80008000u : 0u;
  }
  p.nqb = (int)nqb;
  hipError_t e = attn::launch_prefill(p, stream);
  return e == hipSuccess ? ATTN_OK : hip_fail(e);
}

int attn_fwd(const void* Q, const void* K, const void* V, void* O,
             int B, int Hq, int Hkv, int Lq, int Lk, int D,
             int causal, float scale, const float* alibi_slopes,
             attn_dtype dtype, hipStream_t stream) {
  return attn_fwd_mod(Q, K, V, O, B, Hq, Hkv, Lq, Lk, D, causal, scale, alibi_slopes, 0.f, 0, dtype, stream);
}

int attn_decode_num_splits(int B, int Hq, int Hkv, int Lk, int D) {
  if (!shape_ok(B, Hq, Hkv, 1, Lk) || (D != 64 && D != 128)) return 0;
  const int group = Hq / Hkv;
  if (group >= 2 && group <= 32) {
    // The grouped kernel: one workgroup per (chunk, KV head, batch).
    const int64_t units = (int64_t)B * Hkv;
    int64_t s = (compute_units() + units - 1) / units;
    const int64_t smax = ((int64_t)Lk + kMinChunkGrouped - 1) / kMinChunkGrouped;
    if (s > smax) s = smax;
    if (s < 1) s = 1;
    return (int)s;
  }
  // The per-head kernel: about one workgroup per compute unit (measured at
  // steady clock with nontemporal K/V loads on five shapes, batch 1-32,
  // 2048-32768 keys, D 64 and 128: 2-4 % ahead of two per compute unit on
  // four of them, 1 % behind on the ALiBi one).
  const int64_t groups = Hq / Hkv / decode_heads_per_block(Hq / Hkv);
  const int64_t units = (int64_t)B * Hkv * groups;
  const int64_t target = (int64_t)kBlocksPerCu * compute_units();
  int64_t s = (target + units - 1) / units;
  const int64_t smax = ((int64_t)Lk + kMinChunk - 1) / kMinChunk;
  if (s > smax) s = smax;
  if (s < 1) s = 1;
  return (int)s;
}

size_t attn_decode_workspace_bytes(int B, int Hq, int D, int num_splits) {
  if (B < 1 || Hq < 1 || num_splits < 1 || (D != 64 && D != 128)) return 0;
  const size_t n = (size_t)B * Hq * num_splits;
  const size_t bytes = n * (size_t)(D + 2) * sizeof(float);
  return (bytes + 255) & ~(size_t)255;
}

}  // extern "C"

namespace {

// Argument checks of the decode entry points (everything but the workspace);
// on success *S is the resolved chunk count.
int decode_check(const void* Q, const void* K, const void* V, void* O, int B, int Hq, int Hkv, int Lk, int D,
                 float scale, float softcap, int num_splits, attn_dtype dtype, int* S) {
  if (!Q || !K || !V || !O) return ATTN_ERR_NULL;
  if (!shape_ok(B, Hq, Hkv, 1, Lk) || num_splits < 0 || !std::isfinite(scale)) return ATTN_ERR_SHAPE;
  if (!std::isfinite(softcap) || softcap < 0.f) return ATTN_ERR_SHAPE;
  if (!dims_supported(D, dtype)) return ATTN_ERR_UNSUPPORTED;
  if (!sizes_fit(B, Hq, Hkv, 1, Lk, D)) return ATTN_ERR_SHAPE;
  *S = num_splits ? num_splits : attn_decode_num_splits(B, Hq, Hkv, Lk, D);
  const int group = Hq / Hkv;
  const int64_t nblocks = (int64_t)*S * (group / decode_heads_per_block(group)) * Hkv * B;
  if (nblocks > kMaxGrid || (int64_t)B * Hq > kMaxGrid) return ATTN_ERR_SHAPE;
  return ATTN_OK;
}

// Launch the split and combine kernels with a checked workspace.
int decode_launch(const void* Q, const void* K, const void* V, void* O, int B, int Hq, int Hkv, int Lk, int D,
                  float scale, const float* alibi_slopes, float softcap, int S, void* workspace, attn_dtype dtype,
                  hipStream_t stream) {
  attn::DecodeParams p{};
  p.q = Q; p.k = K; p.v = V; p.o = O;
  p.slopes = alibi_slopes;
  const size_t n = (size_t)B * Hq * S;
  p.ws_o = static_cast<float*>(workspace);
  p.ws_m = p.ws_o + n * D;
  p.ws_l = p.ws_m + n;
  p.B = B; p.Hq = Hq; p.Hkv = Hkv; p.Lk = Lk; p.D = D;
  p.group = Hq / Hkv;
  p.splits = S;
  p.chunk = (Lk + S - 1) / S;
  p.bf16 = dtype == ATTN_BF16;
  p.c = scale * kLog2e;
  p.cap_k2 = softcap > 0.f ? 2.f / softcap : 0.f;
  p.cap_cl = softcap > 0.f ? softcap * kLog2e : 0.f;
  hipError_t e = attn::launch_decode(p, stream);
  return e == hipSuccess ? ATTN_OK : hip_fail(e);
}

}  // namespace

extern "C" {

int attn_decode_mod(const void* Q, const void* K, const void* V, void* O,
                    int B, int Hq, int Hkv, int Lk, int D,
                    float scale, const float* alibi_slopes, float softcap, int num_splits,
                    void* workspace, size_t workspace_bytes,
                    attn_dtype dtype, hipStream_t stream) {
  int S = 0;
  const int rc = decode_check(Q, K, V, O, B, Hq, Hkv, Lk, D, scale, softcap, num_splits, dtype, &S);
  if (rc != ATTN_OK) return rc;
  if (!workspace) return ATTN_ERR_NULL;
  const size_t need = attn_decode_workspace_bytes(B, Hq, D, S);
  if (workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 15)) return ATTN_ERR_WORKSPACE;
  return decode_launch(Q, K, V, O, B, Hq, Hkv, Lk, D, scale, alibi_slopes, softcap, S, workspace, dtype, stream);
}

int attn_decode_noalloc(const void* Q, const void* K, const void* V, void* O,
                        int B, int Hq, int Hkv, int Lk, int D,
                        float scale, const float* alibi_slopes, float softcap, int num_splits,
                        attn_dtype dtype, hipStream_t stream) {
  int S = 0;
  const int rc = decode_check(Q, K, V, O, B, Hq, Hkv, Lk, D, scale, softcap, num_splits, dtype, &S);
  if (rc != ATTN_OK) return rc;
  if (attn_decode_workspace_bytes(B, Hq, D, S) > attn::kDecodeScratchBytes) return ATTN_ERR_WORKSPACE;
  void* ws = nullptr;
  const hipError_t e = attn::decode_scratch(&ws);
  if (e != hipSuccess) return hip_fail(e);
  return decode_launch(Q, K, V, O, B, Hq, Hkv, Lk, D, scale, alibi_slopes, softcap, S, ws, dtype, stream);
}

int attn_decode(const void* Q, const void* K, const void* V, void* O,
                int B, int Hq, int Hkv, int Lk, int D,
                float scale, const float* alibi_slopes, int num_splits,
                void* workspace, size_t workspace_bytes,
                attn_dtype dtype, hipStream_t stream) {
  return attn_decode_mod(Q, K, V, O, B, Hq, Hkv, Lk, D, scale, alibi_slopes, 0.f, num_splits, workspace,
                         workspace_bytes, dtype, stream);
}

int attn_fwd_kernels(int D, attn_dtype dtype, int causal, int alibi, float softcap, int window,
                     char* buf, size_t len) {
  if (!std::isfinite(softcap) || softcap < 0.f || window < 0) return ATTN_ERR_SHAPE;
  if (!dims_supported(D, dtype)) return ATTN_ERR_UNSUPPORTED;
  if ((softcap > 0.f && (!causal || alibi)) || (window > 0 && !causal)) return ATTN_ERR_UNSUPPORTED;
  const attn::PrefillFlags f = attn::prefill_flags(causal != 0, alibi != 0, softcap > 0.f, window > 0);
  char s[96];
  std::snprintf(s, sizeof s, "prefill_kernel<%d,%s,%d,%d,%d,%d>", D, dtype_name(dtype), (int)f.causal, (int)f.alibi,
                (int)f.cap, (int)f.win);
  return put(buf, len, s);
}

int attn_decode_kernels(int Hq, int Hkv, int D, attn_dtype dtype, int alibi, float softcap, char* buf, size_t len) {
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || !std::isfinite(softcap) || softcap < 0.f) return ATTN_ERR_SHAPE;
  if (!dims_supported(D, dtype)) return ATTN_ERR_UNSUPPORTED;
  const int gh = attn::decode_split_heads(Hq / Hkv);
  const int a = alibi ? 1 : 0, c = softcap > 0.f ? 1 : 0;
  char s[160];
  if (gh == 0)
    std::snprintf(s, sizeof s, "decode_mfma_kernel<%d,%s,%d,%d>;decode_combine_kernel<%d,%s>", D, dtype_name(dtype), a,
                  c, D, dtype_name(dtype));
  else
    std::snprintf(s, sizeof s, "decode_split_kernel<%d,%s,%d,%d,%d>;decode_combine_kernel<%d,%s>", D,
                  dtype_name(dtype), gh, a, c, D, dtype_name(dtype));
  return put(buf, len, s);
}

int peaks_hbm_read(const void* buf, size_t bytes, float* sink, hipStream_t stream) {
  if (!buf || !sink || bytes < 16 || bytes % 16 || (reinterpret_cast<uintptr_t>(buf) & 15)) return ATTN_ERR_SHAPE;
  const hipError_t e = attn::launch_hbm_read(buf, bytes, sink, stream);
  return e == hipSuccess ? ATTN_OK : hip_fail(e);
}

int peaks_hbm_read_sink_floats(void) { return attn::hbm_read_sink_floats(); }

int peaks_mfma(int dtype, int iters, const void* operands, float* sink, unsigned long long* clocks,
               hipStream_t stream) {
  if (!operands || !sink || !clocks || iters < 1 || (dtype != 0 && dtype != 1)) return ATTN_ERR_SHAPE;
  const hipError_t e = attn::launch_mfma_loop(dtype, iters, operands, sink, clocks, stream);
  return e == hipSuccess ? ATTN_OK : hip_fail(e);
}

int peaks_mfma_waves(void) { return attn::mfma_loop_waves(); }

size_t peaks_mfma_operand_bytes(void) { return attn::mfma_loop_operand_bytes(); }

int norm_chunks(int rms, int N, int M, norm_dtype dtype) {
  if (N < 1 || M < 1 || (dtype != NORM_F16 && dtype != NORM_BF16 && dtype != NORM_F32)) return 0;
  // One chunk per row (one kernel, a workgroup per row) when the rows fill at
  // least 85 % of the compute units' rounds and, for RMSNorm, a row fits the
  // workgroup's registers (X is then read once; that workgroup takes a whole
  // compute unit).  On the 256 x 2^17 workloads, from HBM: the one-pass
  // RMSNorm ran 1.19x the two kernels with 2 chunks, the L2 norm's one-chunk
  // kernel 1.03x its two chunks.
  const int64_t elem = dtype == NORM_F32 ? 4 : 2, cu = compute_units();
  const int64_t rounds = (N + cu - 1) / cu;
  if (attn::norm_one_kernel(rms != 0, M, (int)elem, 1) && N >= cu && (int64_t)N * 100 >= rounds * cu * 85) return 1;
  // Otherwise about two workgroups per compute unit (measured on the 256 x
  // 2^17 row reductions: 2 chunks per row beat 4, 8 and 16), chunks of at
  // least 4096 elements.
  constexpr int kTargetBlocks = 512, kMinChunk = 4096;
  int64_t c = (kTargetBlocks + N - 1) / N;
  const int64_t cmax = ((int64_t)M + kMinChunk - 1) / kMinChunk;
  if (c > cmax) c = cmax;
  return c < 1 ? 1 : (int)c;
}

int norm_kernels(int rms, int M, norm_dtype dtype, int chunks, char* buf, size_t len) {
  if (dtype != NORM_F16 && dtype != NORM_BF16 && dtype != NORM_F32) return ATTN_ERR_UNSUPPORTED;
  const int elem = dtype == NORM_F32 ? 4 : 2;
  if (M < 1 || M % (16 / elem) || chunks < 1) return ATTN_ERR_SHAPE;
  const char* t = dtype == NORM_F32 ? "f32" : dtype == NORM_BF16 ? "bf16" : "f16";
  char s[96];
  if (attn::norm_one_kernel(rms != 0, M, elem, chunks))
    std::snprintf(s, sizeof s, "%s_row_kernel<%s>", rms ? "rms" : "l2", t);
  else if (rms)
    std::snprintf(s, sizeof s, "norm_split_kernel<%s,1>;rms_apply_kernel<%s>", t, t);
  else
    std::snprintf(s, sizeof s, "norm_split_kernel<%s,0>;l2_combine_kernel", t);
  return put(buf, len, s);
}

size_t norm_workspace_bytes(int N, int chunks) {
  if (N < 1 || chunks < 1) return 0;
  const size_t bytes = (size_t)N * chunks * 2 * sizeof(float);
  return (bytes + 255) & ~(size_t)255;
}

}  // extern "C"

namespace {

int norm_run(const void* X, void* Y, float* out, int N, int M, float eps, norm_dtype dtype, int chunks,
             void* workspace, size_t workspace_bytes, bool rms, hipStream_t stream) {
  if (!X || !out || !workspace || (rms && !Y)) return ATTN_ERR_NULL;
  if (dtype != NORM_F16 && dtype != NORM_BF16 && dtype != NORM_F32) return ATTN_ERR_UNSUPPORTED;
  const int vec = dtype == NORM_F32 ? 4 : 8;
  if (N < 1 || M < 1 || M % vec || chunks < 0 || !std::isfinite(eps) || eps < 0.f) return ATTN_ERR_SHAPE;
  if ((int64_t)N * M >= (int64_t(1) << 40)) return ATTN_ERR_SHAPE;
  const int C = chunks ? chunks : norm_chunks(rms ? 1 : 0, N, M, dtype);
  if ((int64_t)N * C > kMaxGrid) return ATTN_ERR_SHAPE;
  if (workspace_bytes < norm_workspace_bytes(N, C) || (reinterpret_cast<uintptr_t>(workspace) & 15))
    return ATTN_ERR_WORKSPACE;
  attn::NormParams p{};
  p.x = X; p.y = Y; p.out = out;
  p.ws_r = static_cast<float*>(workspace);
  p.ws_t = p.ws_r + (size_t)N * C;
  p.N = N; p.M = M; p.chunks = C;
  const int64_t per = ((int64_t)M + C - 1) / C;
  p.chunk = (int)((per + vec - 1) / vec * vec);
  p.dtype = (int)dtype;
  p.rms = rms ? 1 : 0;
  p.eps = eps;
  p.invM = 1.f / (float)M;
  const hipError_t e = attn::launch_norm(p, stream);
  return e == hipSuccess ? ATTN_OK : hip_fail(e);
}

}  // namespace

extern "C" {

int norm_l2(const void* X, float* out, int N, int M, norm_dtype dtype, int chunks,
            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return norm_run(X, nullptr, out, N, M, 0.f, dtype, chunks, workspace, workspace_bytes, false, stream);
}

int rmsnorm_rowmax(const void* X, void* Y, float* rowmax, int N, int M, float eps, norm_dtype dtype,
                   int chunks, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return norm_run(X, Y, rowmax, N, M, eps, dtype, chunks, workspace, workspace_bytes, true, stream);
}

}  // extern "C"

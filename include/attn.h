/*
 * attn.h — fused scaled-dot-product attention for AMD Instinct MI355X (gfx950).
 *
 * The operation is plain attention as the paper defines it (Eq. attention in
 * the appendix "Additional Example Operators", with the compute definition of
 * Fig. appendix-attention for the product order and the rounding of exp):
 *
 *     S = Q K^T * scale + bias          (masked entries are -inf)
 *     O = softmax_rows(S) V             (exp rounded to the input dtype before P.V)
 *
 * computed without ever materialising S:
 *   - attn_fwd    is the kernel that "rolling update" (Section "Rolling Update",
 *                 Algorithm 1, Eq. fixed-recurrent) produces from that
 *                 definition: one pass over key tiles, the running max / sum /
 *                 P.V state repaired by h(t, r, r') = t * exp(r - r') whenever
 *                 the running max moves;
 *   - attn_decode is what "split-k update" (Section "Split-K Update",
 *                 Algorithm 2, Eq. su:rewrite) produces for one query token:
 *                 independent local nests over key chunks write partial
 *                 (O, max, sum) triples, and a global nest combines them with
 *                 the same repair factor.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensor pointers are DEVICE pointers to contiguous row-major tensors laid
 *    out [B, H, L, D] (D fastest).  Q, K, V and O share one element type
 *    (attn_dtype).  Q and O have Hq heads, K and V have Hkv heads.
 *  - Grouped-query attention: Hq must be a multiple of Hkv; query head hq reads
 *    key/value head hq / (Hq / Hkv) (contiguous groups).  Hkv == Hq is
 *    multi-head attention.
 *  - scale multiplies Q K^T only (callers normally pass 1/sqrt(D)); the ALiBi
 *    bias is added after scaling: bias[i][j] = -alibi_slopes[hq] * (i + Lk - Lq - j).
 *    alibi_slopes is a DEVICE array of Hq floats, or NULL for no bias.
 *  - causal masking is aligned bottom-right: query row i sees key j iff
 *    j <= i + (Lk - Lq).  With Lq == Lk that is j <= i.  A row that sees no
 *    key (only possible when Lq > Lk) produces zeros.
 *  - Accumulation and the softmax state are fp32; the output is rounded to
 *    the input type (round to nearest even).
 *  - Ownership: the caller allocates and frees every buffer (including the
 *    decode workspace).  The library holds no device memory and no global
 *    mutable state apart from a thread-local copy of the last HIP error.
 *  - Asynchrony: work is enqueued on `stream` and the call returns without
 *    synchronising.  Argument errors are detected on the host before
 *    anything is enqueued; in that case nothing runs and no HIP call is made.
 *  - O must not alias Q, K or V.  Each call is deterministic: the same inputs
 *    and arguments give bitwise identical outputs (no atomics).
 *  - Return value: ATTN_OK or a negative attn_status.
 */
#ifndef ATTN_H
#define ATTN_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ATTN_F16 = 0,  /* IEEE binary16 */
  ATTN_BF16 = 1  /* bfloat16 */
} attn_dtype;

typedef enum {
  ATTN_OK = 0,
  ATTN_ERR_NULL = -1,        /* a required pointer is NULL */
  ATTN_ERR_SHAPE = -2,       /* a size is < 1, Hq % Hkv != 0, num_splits < 0, a size overflows,
                                scale is not finite, softcap is negative or not finite, or
                                window is negative */
  ATTN_ERR_UNSUPPORTED = -3, /* head dim not 64 or 128, unknown dtype, or (attn_fwd_mod)
                                softcap or window without the causal mask, or softcap
                                together with ALiBi */
  ATTN_ERR_WORKSPACE = -4,   /* decode workspace smaller than attn_decode_workspace_bytes(), or
                                (attn_decode_noalloc) larger than ATTN_DECODE_NOALLOC_BYTES */
  ATTN_ERR_HIP = -5          /* a HIP launch failed; see attn_last_hip_error() */
} attn_status;

/*
 * Prefill / general attention (rolling update).
 *
 *   Q [B, Hq, Lq, D], K and V [B, Hkv, Lk, D], O [B, Hq, Lq, D]   (device)
 *   B, Hq, Hkv, Lq, Lk >= 1; Hq % Hkv == 0; D in {64, 128}
 *   Lk * D * 2 < 2^31 (one head's K or V in bytes; Lk < 8388608 at D = 128),
 *   and B * Hq * Lq * D, B * Hkv * Lk * D < 2^40
 *   causal  0 or 1 (non-zero means 1)
 *   scale   finite float
 *   alibi_slopes  device float[Hq] or NULL
 *
 * Errors: ATTN_ERR_NULL if Q, K, V or O is NULL; ATTN_ERR_SHAPE for bad sizes;
 * ATTN_ERR_UNSUPPORTED for D or dtype; ATTN_ERR_HIP if the launch fails.
 */
int attn_fwd(const void* Q, const void* K, const void* V, void* O,
             int B, int Hq, int Hkv, int Lq, int Lk, int D,
             int causal, float scale, const float* alibi_slopes,
             attn_dtype dtype, hipStream_t stream);

/*
 * attn_fwd with the score modifiers of the paper's operator table (Table
 * tab:operators) that go beyond causal masking and ALiBi.  softcap = 0 and
 * window = 0 make it exactly attn_fwd.
 *
 *   softcap 0 for none, or cap > 0 (causal only, without ALiBi): the SoftCap
 *           operator (attention with a SoftCap score modifier, GQA heads and
 *           the causal mask, from Gemma 2; the formula is not printed): each
 *           scaled score becomes cap * tanh(score * scale / cap) before the
 *           mask.
 *   window  0 for none, or W >= 1 (causal only): the Window operator
 *           (attention with a windowed mask, from Gemma 2), read as Gemma 2's
 *           causal sliding window: query row i sees key j iff
 *           i + (Lk - Lq) - W < j <= i + (Lk - Lq), i.e. its last W keys.
 *           W >= Lk is plain causal attention; W = 1 selects V[i + Lk - Lq].
 *           It combines with ALiBi and with softcap.
 *
 * Errors: as attn_fwd, plus ATTN_ERR_SHAPE for a negative or non-finite
 * softcap or a negative window, and ATTN_ERR_UNSUPPORTED for softcap or
 * window without the causal mask, or softcap together with ALiBi.
 */
int attn_fwd_mod(const void* Q, const void* K, const void* V, void* O,
                 int B, int Hq, int Hkv, int Lq, int Lk, int D,
                 int causal, float scale, const float* alibi_slopes, float softcap, int window,
                 attn_dtype dtype, hipStream_t stream);

/*
 * Bytes of decode workspace needed for (B, Hq, D, num_splits), num_splits >= 1
 * (resolve 0 with attn_decode_num_splits first).  Returns 0 for invalid sizes.
 *
 * Workspace layout (fp32, offsets in floats, n = B*Hq*num_splits): the local
 * nests' results of the split-k update (Fig. su-result), in natural-log units,
 * for head row r = b*Hq + hq and chunk s:
 *   o_l   at [0, n*D)        o_l[(r*num_splits + s)*D + d]   unnormalised sum of
 *                                                            exp(score - max_l) * V
 *   max_l at [n*D, n*D + n)  max_l[r*num_splits + s]         chunk max of the scores
 *   sum_l at [n*D + n, n*D + 2n) sum_l[r*num_splits + s]     sum of exp(score - max_l)
 * A chunk with no key has max_l = -inf, sum_l = 0, o_l = 0.
 */
size_t attn_decode_workspace_bytes(int B, int Hq, int D, int num_splits);

/*
 * The number of key chunks attn_decode uses when num_splits == 0 (the library
 * heuristic): about one workgroup per compute unit of the current device (256
 * if it cannot be queried).  With one query head per KV head (or more than
 * 32), one workgroup per (chunk, KV head, batch, query-head group) and
 * chunks of at least 256 keys; with 2..32 query heads per KV head, served
 * together by one workgroup per (chunk, KV head, batch), chunks of at least
 * 128 keys.
 * Returns a value >= 1, or 0 for invalid sizes.
 */
int attn_decode_num_splits(int B, int Hq, int Hkv, int Lk, int D);

/*
 * Single-token decode (split-k update).
 *
 *   Q [B, Hq, 1, D], K and V [B, Hkv, Lk, D], O [B, Hq, 1, D]   (device)
 *   The query is the token at position Lk - 1, so every key is visible (the
 *   causal mask is a no-op).  alibi_slopes as for attn_fwd, with i = Lk - 1.
 *   num_splits  >= 1 chunks of ceil(Lk / num_splits) keys (the last chunk may
 *               be short, chunks past Lk are empty), or 0 for the heuristic.
 *   workspace   device buffer of at least attn_decode_workspace_bytes(B, Hq,
 *               D, resolved num_splits) bytes, 16-byte aligned; its contents
 *               after the call are the local partials described above.
 *
 * Two kernels run on `stream`: the local split kernel, then the combine.
 * With one chunk (num_splits resolving to 1) the split kernel also writes O,
 * exactly what the combine would compute from its single partial, and the
 * combine does not run.
 * Errors: ATTN_ERR_NULL (Q, K, V, O or workspace NULL), ATTN_ERR_SHAPE,
 * ATTN_ERR_UNSUPPORTED, ATTN_ERR_WORKSPACE, ATTN_ERR_HIP.
 */
int attn_decode(const void* Q, const void* K, const void* V, void* O,
                int B, int Hq, int Hkv, int Lk, int D,
                float scale, const float* alibi_slopes, int num_splits,
                void* workspace, size_t workspace_bytes,
                attn_dtype dtype, hipStream_t stream);

/*
 * attn_decode with the SoftCap score modifier (softcap = 0 makes it exactly
 * attn_decode):
 *   softcap     0 for none, or cap > 0: the SoftCap operator of the paper's
 *               operator table (Table tab:operators); each scaled score
 *               becomes cap * tanh(score * scale / cap) before the ALiBi bias
 *               is added.
 * Errors: as attn_decode, plus ATTN_ERR_SHAPE for a negative or non-finite
 * softcap.
 */
int attn_decode_mod(const void* Q, const void* K, const void* V, void* O,
                    int B, int Hq, int Hkv, int Lk, int D,
                    float scale, const float* alibi_slopes, float softcap, int num_splits,
                    void* workspace, size_t workspace_bytes,
                    attn_dtype dtype, hipStream_t stream);

/* Bytes of the static workspace that attn_decode_noalloc uses. */
#define ATTN_DECODE_NOALLOC_BYTES ((size_t)16 << 20)

/*
 * attn_decode_mod for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * kernels and results, with the workspace taken from a static device array of
 * ATTN_DECODE_NOALLOC_BYTES that the library holds on each GPU it runs on
 * until the process ends.  The caller passes inputs and outputs only.  It
 * calls no hipMalloc, hipFree or allocating routine; the first call on a
 * device looks the array's address up (hipGetSymbolAddress) and keeps it.
 *   Limit: attn_decode_workspace_bytes(B, Hq, D, resolved num_splits) must
 *   not exceed ATTN_DECODE_NOALLOC_BYTES (ATTN_ERR_WORKSPACE otherwise).
 *   Every call on a GPU shares that GPU's array, which keeps the last call's
 *   partials: calls that overlap on one GPU (other streams, other threads)
 *   race and must be serialised by the caller.  Every partial is written
 *   before it is read, so nothing has to start at zero.
 * Errors: as attn_decode_mod (no workspace arguments), ATTN_ERR_WORKSPACE for
 * the size limit, ATTN_ERR_HIP if the address lookup or a launch fails.
 */
int attn_decode_noalloc(const void* Q, const void* K, const void* V, void* O,
                        int B, int Hq, int Hkv, int Lk, int D,
                        float scale, const float* alibi_slopes, float softcap, int num_splits,
                        attn_dtype dtype, hipStream_t stream);

/*
 * The kernels that attn_fwd_mod (attn_fwd: softcap = 0, window = 0) launches
 * for these arguments, written to buf as a NUL-terminated string such as
 * "prefill_kernel<128,f16,1,0,0,0>" (head dim, element type, then the
 * causal, ALiBi, SoftCap and window template flags).  Host only: no HIP call.
 * For coverage checks and profiles of the rolling-update kernel (Section
 * "Rolling Update").  alibi: non-zero if slopes would be passed.
 * Errors: the argument errors of attn_fwd_mod; ATTN_ERR_SHAPE if buf is NULL
 * or shorter than the name.
 */
int attn_fwd_kernels(int D, attn_dtype dtype, int causal, int alibi, float softcap, int window,
                     char* buf, size_t len);

/*
 * The kernels that attn_decode_mod (attn_decode: softcap = 0) launches, as
 * "split;combine" with the template arguments, e.g.
 * "decode_mfma_kernel<128,f16,0,0>;decode_combine_kernel<128,f16>" (local
 * and global nests of Fig. su-result; with one chunk only the split kernel
 * runs).  Host only.  Errors as attn_fwd_kernels.
 */
int attn_decode_kernels(int Hq, int Hkv, int D, attn_dtype dtype, int alibi, float softcap, char* buf, size_t len);

/* Static, human-readable name of an attn_status value. */
const char* attn_status_string(int status);

/* The hipError_t of the last ATTN_ERR_HIP returned on this thread (0 if none). */
int attn_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_H */

"""Fused attention for AMD Instinct MI355X (gfx950) — Python binding of libattn.so.

A thin ctypes layer over the C ABI declared in ``include/attn.h``: the
functions below have the same names as the C entry points and only marshal
arguments (device pointers, sizes, the current HIP stream).  Every step of the
computation runs in the HIP kernels of ``libattn.so``; PyTorch only provides
device memory and streams.  There is no fallback: if the library is missing
or a call fails, an exception is raised.
"""

import ctypes
import math
import os

import torch

__all__ = [
    "attn_fwd", "attn_fwd_mod", "attn_decode", "attn_decode_mod", "attn_decode_workspace_bytes",
    "attn_decode_num_splits", "attn_decode_noalloc", "peaks_hbm_read", "peaks_mfma", "peaks_mfma_waves",
    "peaks_mfma_operand_bytes", "norm_chunks", "norm_kernels", "norm_workspace_bytes", "norm_l2", "rmsnorm_rowmax", "attn_fwd_kernels", "attn_decode_kernels",
    "attn_status_string", "attn_last_hip_error", "library_path", "load_library", "AttnError",
    "ATTN_OK", "ATTN_ERR_NULL", "ATTN_ERR_SHAPE", "ATTN_ERR_UNSUPPORTED", "ATTN_ERR_WORKSPACE",
    "ATTN_ERR_HIP",
]

ATTN_OK = 0
ATTN_ERR_NULL = -1
ATTN_ERR_SHAPE = -2
ATTN_ERR_UNSUPPORTED = -3
ATTN_ERR_WORKSPACE = -4
ATTN_ERR_HIP = -5

ATTN_F16 = 0
ATTN_BF16 = 1
_DTYPE_CODE = {torch.float16: ATTN_F16, torch.bfloat16: ATTN_BF16}

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


class AttnError(RuntimeError):
    """A call into libattn.so returned an error status."""

    def __init__(self, status, msg):
        super().__init__(msg)
        self.status = status


def library_path():
    return os.path.join(_HERE, "libattn.so")


def load_library():
    """Load (once) and return the ctypes handle of libattn.so; raises if absent."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is not built; run `python -c 'import __graft_entry__ as g; g.build()'` "
            "or `python paper_2510_08726_amd/build.py` first")
    lib = ctypes.CDLL(path)
    vp, ci, cf, cs = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.attn_fwd.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, ci, cf, vp, ci, vp]
    lib.attn_fwd.restype = ci
    lib.attn_fwd_mod.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, ci, cf, vp, cf, ci, ci, vp]
    lib.attn_fwd_mod.restype = ci
    lib.attn_decode.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, cf, vp, ci, vp, cs, ci, vp]
    lib.attn_decode.restype = ci
    lib.attn_decode_mod.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, cf, vp, cf, ci, vp, cs, ci, vp]
    lib.attn_decode_mod.restype = ci
    lib.attn_decode_workspace_bytes.argtypes = [ci, ci, ci, ci]
    lib.attn_decode_workspace_bytes.restype = cs
    lib.attn_decode_num_splits.argtypes = [ci, ci, ci, ci, ci]
    lib.attn_decode_num_splits.restype = ci
    lib.attn_decode_noalloc.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, cf, vp, cf, ci, ci, vp]
    lib.attn_decode_noalloc.restype = ci
    lib.attn_fwd_kernels.argtypes = [ci, ci, ci, ci, cf, ci, ctypes.c_char_p, cs]
    lib.attn_fwd_kernels.restype = ci
    lib.attn_decode_kernels.argtypes = [ci, ci, ci, ci, ci, cf, ctypes.c_char_p, cs]
    lib.attn_decode_kernels.restype = ci
    lib.norm_kernels.argtypes = [ci, ci, ci, ci, ctypes.c_char_p, cs]
    lib.norm_kernels.restype = ci
    lib.peaks_hbm_read.argtypes = [vp, cs, vp, vp]
    lib.peaks_hbm_read.restype = ci
    lib.peaks_hbm_read_sink_floats.argtypes = []
    lib.peaks_hbm_read_sink_floats.restype = ci
    lib.peaks_mfma.argtypes = [ci, ci, vp, vp, vp, vp]
    lib.peaks_mfma.restype = ci
    lib.peaks_mfma_waves.argtypes = []
    lib.peaks_mfma_waves.restype = ci
    lib.peaks_mfma_operand_bytes.argtypes = []
    lib.peaks_mfma_operand_bytes.restype = cs
    lib.norm_chunks.argtypes = [ci, ci, ci, ci]
    lib.norm_chunks.restype = ci
    lib.norm_workspace_bytes.argtypes = [ci, ci]
    lib.norm_workspace_bytes.restype = cs
    lib.norm_l2.argtypes = [vp, vp, ci, ci, ci, ci, vp, cs, vp]
    lib.norm_l2.restype = ci
    lib.rmsnorm_rowmax.argtypes = [vp, vp, vp, ci, ci, cf, ci, ci, vp, cs, vp]
    lib.rmsnorm_rowmax.restype = ci
    lib.attn_status_string.argtypes = [ci]
    lib.attn_status_string.restype = ctypes.c_char_p
    lib.attn_last_hip_error.argtypes = []
    lib.attn_last_hip_error.restype = ci
    _LIB = lib
    return lib


def attn_status_string(status):
    return load_library().attn_status_string(int(status)).decode()


def attn_last_hip_error():
    return load_library().attn_last_hip_error()


def _check(rc):
    if rc != ATTN_OK:
        msg = attn_status_string(rc)
        if rc == ATTN_ERR_HIP:
            msg += f" (hipError_t {attn_last_hip_error()})"
        raise AttnError(rc, msg)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _require(cond, msg):
    if not cond:
        raise ValueError(msg)


def _check_tensors(q, k, v, slopes):
    for name, t in (("q", q), ("k", k), ("v", v)):
        _require(t.is_cuda, f"{name} must be a GPU tensor")
        _require(t.is_contiguous(), f"{name} must be contiguous [B, H, L, D]")
        _require(t.dim() == 4, f"{name} must be 4-D [B, H, L, D]")
    _require(q.dtype == k.dtype == v.dtype, "q, k, v must share one dtype")
    _require(q.dtype in _DTYPE_CODE, "dtype must be float16 or bfloat16")
    _require(k.shape == v.shape, "k and v must have the same shape")
    if slopes is not None:
        _require(slopes.is_cuda and slopes.dtype == torch.float32 and slopes.is_contiguous(),
                 "alibi_slopes must be a contiguous float32 GPU tensor")
        _require(slopes.numel() == q.shape[1], "alibi_slopes needs one value per query head")


def _fwd_args(q, k, v, o, alibi_slopes):
    _check_tensors(q, k, v, alibi_slopes)
    B, Hq, Lq, D = q.shape
    _require(k.shape[0] == B and k.shape[3] == D, "k/v batch and head dim must match q")
    if o is None:
        o = torch.empty_like(q)
    _require(o.shape == q.shape and o.dtype == q.dtype and o.is_contiguous() and o.is_cuda,
             "o must be a contiguous GPU tensor shaped like q")
    return o


def attn_fwd(q, k, v, o=None, *, causal=False, scale=None, alibi_slopes=None, softcap=None,
             window=None, stream=None):
    """O = softmax(Q K^T * scale + bias) V by the fused prefill kernel.

    q [B, Hq, Lq, D], k and v [B, Hkv, Lk, D] (float16 or bfloat16, contiguous,
    on the GPU); ``o`` is written if given, else allocated.  ``scale``
    defaults to 1/sqrt(D).  ``softcap`` (cap > 0) and ``window`` (W >= 1)
    select the score modifiers of ``attn_fwd_mod``; without them the call
    goes to the C entry point ``attn_fwd``.  Returns ``o``.
    """
    if softcap or window:
        return attn_fwd_mod(q, k, v, o, causal=causal, scale=scale, alibi_slopes=alibi_slopes,
                            softcap=softcap, window=window, stream=stream)
    o = _fwd_args(q, k, v, o, alibi_slopes)
    B, Hq, Lq, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    _check(load_library().attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, Hq, Hkv, Lq, Lk, D,
                                   int(bool(causal)), sc, _ptr(alibi_slopes), _DTYPE_CODE[q.dtype],
                                   _stream(stream)))
    return o


def attn_fwd_mod(q, k, v, o=None, *, causal=False, scale=None, alibi_slopes=None, softcap=None,
                 window=None, stream=None):
    """attn_fwd with the SoftCap modifier (``softcap``: None or cap > 0) and the
    causal sliding window (``window``: None or W >= 1 keys per row)."""
    o = _fwd_args(q, k, v, o, alibi_slopes)
    B, Hq, Lq, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    _check(load_library().attn_fwd_mod(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, Hq, Hkv, Lq, Lk, D,
                                       int(bool(causal)), sc, _ptr(alibi_slopes), float(softcap or 0.0),
                                       int(window or 0), _DTYPE_CODE[q.dtype], _stream(stream)))
    return o


def attn_decode_workspace_bytes(B, Hq, D, num_splits):
    return load_library().attn_decode_workspace_bytes(B, Hq, D, num_splits)


def attn_decode_num_splits(B, Hq, Hkv, Lk, D):
    return load_library().attn_decode_num_splits(B, Hq, Hkv, Lk, D)


def _decode_args(q, k, v, o, alibi_slopes, num_splits, workspace):
    _check_tensors(q, k, v, alibi_slopes)
    B, Hq, Lq, D = q.shape
    _require(Lq == 1, "decode takes one query token (q.shape[2] == 1)")
    Hkv, Lk = k.shape[1], k.shape[2]
    _require(k.shape[0] == B and k.shape[3] == D, "k/v batch and head dim must match q")
    if o is None:
        o = torch.empty_like(q)
    _require(o.shape == q.shape and o.dtype == q.dtype and o.is_contiguous() and o.is_cuda,
             "o must be a contiguous GPU tensor shaped like q")
    lib = load_library()
    S = num_splits if num_splits else lib.attn_decode_num_splits(B, Hq, Hkv, Lk, D)
    need = lib.attn_decode_workspace_bytes(B, Hq, D, max(S, 1))
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    return o, workspace


def attn_decode(q, k, v, o=None, *, scale=None, alibi_slopes=None, softcap=None, num_splits=0,
                workspace=None, stream=None):
    """Single-token decode by split-k: q [B, Hq, 1, D] against k, v [B, Hkv, Lk, D].

    ``softcap``: None, or the cap > 0 of the SoftCap score modifier
    (cap * tanh(scale q.k / cap)); with it the call goes to ``attn_decode_mod``.
    ``num_splits`` = 0 lets the library choose.  ``workspace`` (uint8 GPU
    tensor) is allocated when not given.  Returns ``o`` [B, Hq, 1, D].
    """
    if softcap:
        return attn_decode_mod(q, k, v, o, scale=scale, alibi_slopes=alibi_slopes, softcap=softcap,
                               num_splits=num_splits, workspace=workspace, stream=stream)
    o, workspace = _decode_args(q, k, v, o, alibi_slopes, num_splits, workspace)
    B, Hq, _, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    _check(load_library().attn_decode(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, Hq, Hkv, Lk, D, sc,
                                      _ptr(alibi_slopes), int(num_splits), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _DTYPE_CODE[q.dtype],
                                      _stream(stream)))
    return o


def attn_decode_mod(q, k, v, o=None, *, scale=None, alibi_slopes=None, softcap=None, num_splits=0,
                    workspace=None, stream=None):
    """attn_decode with the SoftCap score modifier (``softcap``: None or cap > 0)."""
    o, workspace = _decode_args(q, k, v, o, alibi_slopes, num_splits, workspace)
    B, Hq, _, D = q.shape
    Hkv, Lk = k.shape[1], k.shape[2]
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    _check(load_library().attn_decode_mod(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, Hq, Hkv, Lk, D, sc,
                                          _ptr(alibi_slopes), float(softcap or 0.0), int(num_splits),
                                          _ptr(workspace), workspace.numel() * workspace.element_size(),
                                          _DTYPE_CODE[q.dtype], _stream(stream)))
    return o


ATTN_DECODE_NOALLOC_BYTES = 16 << 20


def attn_decode_noalloc(q, k, v, o=None, *, scale=None, alibi_slopes=None, softcap=None, num_splits=0,
                        stream=None):
    """attn_decode_mod with the workspace in the library's static device array
    (no allocation inside the library; ``o`` is allocated here if not given).
    Calls that overlap on one GPU race on that array."""
    _check_tensors(q, k, v, alibi_slopes)
    B, Hq, Lq, D = q.shape
    _require(Lq == 1, "decode takes one query token (q.shape[2] == 1)")
    Hkv, Lk = k.shape[1], k.shape[2]
    _require(k.shape[0] == B and k.shape[3] == D, "k/v batch and head dim must match q")
    if o is None:
        o = torch.empty_like(q)
    _require(o.shape == q.shape and o.dtype == q.dtype and o.is_contiguous() and o.is_cuda,
             "o must be a contiguous GPU tensor shaped like q")
    sc = 1.0 / math.sqrt(D) if scale is None else float(scale)
    _check(load_library().attn_decode_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), B, Hq, Hkv, Lk, D, sc,
                                              _ptr(alibi_slopes), float(softcap or 0.0), int(num_splits),
                                              _DTYPE_CODE[q.dtype], _stream(stream)))
    return o


def attn_fwd_kernels(D, dtype, causal, alibi, softcap=0.0, window=0):
    """Names of the kernels attn_fwd_mod launches for these arguments (host only)."""
    buf = ctypes.create_string_buffer(256)
    _check(load_library().attn_fwd_kernels(D, _DTYPE_CODE.get(dtype, dtype), int(bool(causal)), int(bool(alibi)),
                                           float(softcap or 0.0), int(window or 0), buf, 256))
    return buf.value.decode().split(";")


def attn_decode_kernels(Hq, Hkv, D, dtype, alibi, softcap=0.0):
    """Names of the kernels attn_decode_mod launches for these arguments (host only)."""
    buf = ctypes.create_string_buffer(256)
    _check(load_library().attn_decode_kernels(Hq, Hkv, D, _DTYPE_CODE.get(dtype, dtype), int(bool(alibi)),
                                              float(softcap or 0.0), buf, 256))
    return buf.value.decode().split(";")


def peaks_hbm_read(buf, sink=None, stream=None):
    """Stream-read every byte of the GPU tensor ``buf`` once (peaks.h).  Returns ``sink``."""
    lib = load_library()
    if sink is None:
        sink = torch.empty(lib.peaks_hbm_read_sink_floats(), dtype=torch.float32, device=buf.device)
    _check(lib.peaks_hbm_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream)))
    return sink


def peaks_mfma(dtype, iters, operands, sink=None, clocks=None, stream=None):
    """Run the MFMA loop of peaks.h; returns (sink, clocks) tensors."""
    lib = load_library()
    if sink is None:
        sink = torch.empty(lib.peaks_mfma_waves(), dtype=torch.float32, device=operands.device)
    if clocks is None:
        clocks = torch.zeros(2, dtype=torch.int64, device=operands.device)
    _check(lib.peaks_mfma(_DTYPE_CODE.get(dtype, dtype), int(iters), _ptr(operands), _ptr(sink), _ptr(clocks),
                          _stream(stream)))
    return sink, clocks


def peaks_mfma_waves():
    return load_library().peaks_mfma_waves()


def peaks_mfma_operand_bytes():
    return load_library().peaks_mfma_operand_bytes()


NORM_F16, NORM_BF16, NORM_F32 = 0, 1, 2
_NORM_CODE = {torch.float16: NORM_F16, torch.bfloat16: NORM_BF16, torch.float32: NORM_F32}


def norm_chunks(op, N, M, dtype):
    """Chunks per row that norm_l2 (op "l2") or rmsnorm_rowmax (op "rms") uses for chunks=0."""
    return load_library().norm_chunks(int(op == "rms"), N, M, _NORM_CODE[dtype])


def norm_kernels(op, M, dtype, chunks):
    """Names of the kernels norm_l2 (op "l2") or rmsnorm_rowmax (op "rms")
    launches for rows of M elements and `chunks` >= 1 chunks per row (host only)."""
    buf = ctypes.create_string_buffer(128)
    _check(load_library().norm_kernels(int(op == "rms"), int(M), _NORM_CODE.get(dtype, dtype), int(chunks), buf, 128))
    return buf.value.decode().split(";")


def norm_workspace_bytes(N, chunks):
    return load_library().norm_workspace_bytes(N, chunks)


def _norm_args(op, x, chunks, workspace):
    _require(x.is_cuda and x.is_contiguous() and x.dim() == 2, "x must be a contiguous 2-D GPU tensor [N, M]")
    _require(x.dtype in _NORM_CODE, "x must be float16, bfloat16 or float32")
    N, M = x.shape
    lib = load_library()
    C = chunks or lib.norm_chunks(int(op == "rms"), N, M, _NORM_CODE[x.dtype])
    if workspace is None:
        workspace = torch.empty(max(lib.norm_workspace_bytes(N, max(C, 1)), 16), dtype=torch.uint8,
                                device=x.device)
    return N, M, workspace


def norm_l2(x, out=None, *, chunks=0, workspace=None, stream=None):
    """Row L2 norms of x [N, M] (single pass, split over the row): out [N] float32."""
    N, M, workspace = _norm_args("l2", x, chunks, workspace)
    if out is None:
        out = torch.empty(N, dtype=torch.float32, device=x.device)
    _require(out.is_cuda and out.dtype == torch.float32 and out.numel() == N, "out must be float32 [N]")
    _check(load_library().norm_l2(_ptr(x), _ptr(out), N, M, _NORM_CODE[x.dtype], int(chunks), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def rmsnorm_rowmax(x, y=None, rowmax=None, *, eps=1e-6, chunks=0, workspace=None, stream=None):
    """y = x / sqrt(mean(x^2) + eps) (x's dtype) and rowmax [N] = max of each row of y (float32)."""
    N, M, workspace = _norm_args("rms", x, chunks, workspace)
    if y is None:
        y = torch.empty_like(x)
    if rowmax is None:
        rowmax = torch.empty(N, dtype=torch.float32, device=x.device)
    _require(y.shape == x.shape and y.dtype == x.dtype and y.is_contiguous() and y.is_cuda, "y must match x")
    _require(rowmax.is_cuda and rowmax.dtype == torch.float32 and rowmax.numel() == N, "rowmax must be float32 [N]")
    _check(load_library().rmsnorm_rowmax(_ptr(x), _ptr(y), _ptr(rowmax), N, M, float(eps), _NORM_CODE[x.dtype],
                                         int(chunks), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                         _stream(stream)))
    return y, rowmax


def norm_partials(workspace, N, chunks):
    """View a norm workspace as (r [N, chunks], t [N, chunks]) float32."""
    f = workspace.view(torch.float32)
    n = N * chunks
    return f[:n].view(N, chunks), f[n:2 * n].view(N, chunks)


def decode_partials(workspace, B, Hq, D, num_splits):
    """View the decode workspace as (o_l [B,Hq,S,D], max_l [B,Hq,S], sum_l [B,Hq,S]) fp32."""
    n = B * Hq * num_splits
    f = workspace.view(torch.float32)
    return (f[:n * D].view(B, Hq, num_splits, D), f[n * D:n * D + n].view(B, Hq, num_splits),
            f[n * D + n:n * D + 2 * n].view(B, Hq, num_splits))

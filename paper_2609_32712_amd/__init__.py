"""Python binding of libmala.so, the MI355X (gfx950) MALA causal-attention library.

Argument marshalling only: every step of forward, backward and decode runs in the
HIP kernels behind the C ABI of include/mala.h.  PyTorch provides device memory
and the current stream.  There is no fallback: if libmala.so is missing or no
GPU is present, the calls raise.

Low-level functions carry the C names and arguments (mala_fwd, mala_bwd,
mala_fwd_varlen, mala_bwd_varlen, mala_decode, mala_decode_noalloc, mala_geometry,
mala_bwd_workspace_size, mala_bwd_varlen_workspace_size, mala_decode_workspace_size);
fwd / bwd / fwd_varlen /
bwd_varlen / decode allocate their outputs and return them in a dict.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmala.so")

MALA_OK, MALA_ERR_INVALID_ARG, MALA_ERR_UNSUPPORTED = 0, -1, -2
MALA_ERR_WORKSPACE, MALA_ERR_HIP = -3, -4
PASS_FWD, PASS_BWD, PASS_DECODE = 0, 1, 2
OUT_F32, OUT_BF16 = 0, 1
CNT_LEGAL, CNT_RETAINED, CNT_V_TILES, CNT_SLOTS = 0, 1, 2, 3
CNT_RETAINED_KV, CNT_V_NEEDED, CNT_SET_HASH, CNT_SET_HASH_KV = 4, 5, 6, 7
NUM_COUNTERS = 8

EXPORTS = ("mala_geometry", "mala_strerror", "mala_last_error", "mala_fwd",
           "mala_bwd_workspace_size", "mala_bwd", "mala_fwd_varlen", "mala_bwd_varlen",
           "mala_decode_workspace_size", "mala_decode", "mala_decode_noalloc",
           "mala_bwd_varlen_workspace_size")
DECODE_SCRATCH_BYTES = 16 << 20   # MALA_DECODE_SCRATCH_BYTES


class MalaError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__("libmala status %d: %s" % (status, detail))
        self.status = status


class _Geometry(ctypes.Structure):
    _fields_ = [("block_q", ctypes.c_int32), ("block_k", ctypes.c_int32)]


_lib = None


def load_library():
    """Load libmala.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libmala.so not found at %s; build it with "
                           "`python paper_2609_32712_amd/build.py`" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.mala_geometry.argtypes = [i, i]
    lib.mala_geometry.restype = _Geometry
    lib.mala_strerror.argtypes = [i]
    lib.mala_strerror.restype = ctypes.c_char_p
    lib.mala_last_error.argtypes = []
    lib.mala_last_error.restype = ctypes.c_char_p
    lib.mala_fwd.argtypes = [vp] * 7 + [i] * 7 + [f, f, i, vp]
    lib.mala_fwd.restype = i
    lib.mala_bwd_workspace_size.argtypes = [i] * 6
    lib.mala_bwd_workspace_size.restype = sz
    lib.mala_bwd_varlen_workspace_size.argtypes = [i] * 6
    lib.mala_bwd_varlen_workspace_size.restype = sz
    lib.mala_bwd.argtypes = [vp] * 12 + [sz] + [i] * 7 + [f, f, i, i, vp]
    lib.mala_bwd.restype = i
    lib.mala_fwd_varlen.argtypes = [vp] * 9 + [i] * 8 + [f, f, i, vp]
    lib.mala_fwd_varlen.restype = i
    lib.mala_bwd_varlen.argtypes = [vp] * 14 + [sz] + [i] * 8 + [f, f, i, i, vp]
    lib.mala_bwd_varlen.restype = i
    lib.mala_decode_workspace_size.argtypes = [i] * 4
    lib.mala_decode_workspace_size.restype = sz
    lib.mala_decode.argtypes = [vp] * 8 + [i, vp, sz] + [i] * 5 + [f, f, i, vp]
    lib.mala_decode.restype = i
    lib.mala_decode_noalloc.argtypes = [vp] * 8 + [i] * 6 + [f, f, i, vp]
    lib.mala_decode_noalloc.restype = i
    _lib = lib
    return lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(status):
    if status != MALA_OK:
        lib = load_library()
        detail = lib.mala_last_error().decode() or lib.mala_strerror(status).decode()
        raise MalaError(status, detail)


_OUT = (torch.float32, torch.bfloat16)


def _spec(t, name, dtype, shape, optional=False):
    """Check a tensor argument's type, dtype, exact shape and contiguity (raises
    TypeError / ValueError); the device is checked by _on_device afterwards."""
    if t is None:
        if optional:
            return None
        raise TypeError("%s is required" % name)
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
    if not ok:
        raise TypeError("%s must have dtype %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def _dims(t, name, ndim):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    if t.dim() != ndim:
        raise ValueError("%s must be %d-d, got shape %s" % (name, ndim, tuple(t.shape)))
    return tuple(t.shape)


def _on_device(named):
    """Every given tensor (None skipped) is a CUDA (HIP) tensor on one device."""
    dev = None
    for name, t in named:
        if t is None:
            continue
        if not t.is_cuda:
            raise TypeError("%s must be a CUDA (HIP) tensor" % name)
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise TypeError("%s is on %s, the other tensors on %s" % (name, t.device, dev))


def _workspace(ws):
    if not isinstance(ws, torch.Tensor) or not ws.is_contiguous():
        raise TypeError("workspace must be a contiguous tensor")
    return ws


def _out_code(*ts):
    """MALA_OUT_* of output tensors that must share one type (fp32 or bf16)."""
    if len({t.dtype for t in ts}) != 1:
        raise TypeError("these outputs must share one dtype")
    return OUT_BF16 if ts[0].dtype == torch.bfloat16 else OUT_F32


# ---------------------------------------------------------------- C names
def mala_geometry(head_dim, pass_):
    g = load_library().mala_geometry(head_dim, pass_)
    return int(g.block_q), int(g.block_k)


def mala_bwd_workspace_size(B, Hq, Hkv, Nq, Nk, D):
    return int(load_library().mala_bwd_workspace_size(B, Hq, Hkv, Nq, Nk, D))


def mala_bwd_varlen_workspace_size(num_seqs, max_seqlen_k, total_q, Hq, Hkv, D):
    return int(load_library().mala_bwd_varlen_workspace_size(num_seqs, max_seqlen_k, total_q, Hq,
                                                             Hkv, D))


def mala_decode_workspace_size(B, Hq, D, num_splits):
    return int(load_library().mala_decode_workspace_size(B, Hq, D, num_splits))


def _stats_specs(row_tiles, counters, rows_shape):
    _spec(row_tiles, "row_tiles", torch.int32, rows_shape, optional=True)
    _spec(counters, "counters", torch.int64, (NUM_COUNTERS,), optional=True)


def _fwd_specs(q, k, v, o, lse, row_tiles, counters):
    B, Hq, Nq, D = _dims(q, "q", 4)
    _spec(q, "q", torch.bfloat16, (B, Hq, Nq, D))
    _, Hkv, Nk, _ = _dims(k, "k", 4)
    _spec(k, "k", torch.bfloat16, (B, Hkv, Nk, D))
    _spec(v, "v", torch.bfloat16, (B, Hkv, Nk, D))
    _spec(o, "o", _OUT, (B, Hq, Nq, D))
    _spec(lse, "lse", torch.float32, (B, Hq, Nq))
    _stats_specs(row_tiles, counters, (B, Hq, Nq))
    return B, Hq, Hkv, Nq, Nk, D


def mala_fwd(q, k, v, o, lse, row_tiles, counters, scale, tau, causal=1, stream=None):
    B, Hq, Hkv, Nq, Nk, D = _fwd_specs(q, k, v, o, lse, row_tiles, counters)
    _on_device((("q", q), ("k", k), ("v", v), ("o", o), ("lse", lse), ("row_tiles", row_tiles),
                ("counters", counters)))
    _check(load_library().mala_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(row_tiles),
                                   _ptr(counters), B, Hq, Hkv, Nq, Nk, D, causal, scale, tau,
                                   _out_code(o), _stream(stream)))


def _bwd_specs(q, k, v, o, lse, dout, dq, dk, dv, row_tiles, counters, workspace):
    B, Hq, Hkv, Nq, Nk, D = _fwd_specs(q, k, v, o, lse, row_tiles, counters)
    _spec(dout, "dout", torch.bfloat16, (B, Hq, Nq, D))
    _spec(dq, "dq", _OUT, (B, Hq, Nq, D))
    _spec(dk, "dk", _OUT, (B, Hkv, Nk, D))
    _spec(dv, "dv", _OUT, (B, Hkv, Nk, D))
    _out_code(dq, dk, dv)
    _workspace(workspace)
    return B, Hq, Hkv, Nq, Nk, D


def mala_bwd(q, k, v, o, lse, dout, dq, dk, dv, row_tiles, counters, workspace, scale, tau,
             causal=1, stream=None):
    B, Hq, Hkv, Nq, Nk, D = _bwd_specs(q, k, v, o, lse, dout, dq, dk, dv, row_tiles, counters,
                                       workspace)
    _on_device((("q", q), ("k", k), ("v", v), ("o", o), ("lse", lse), ("dout", dout),
                ("dq", dq), ("dk", dk), ("dv", dv), ("row_tiles", row_tiles),
                ("counters", counters), ("workspace", workspace)))
    _check(load_library().mala_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(dout),
                                   _ptr(dq), _ptr(dk), _ptr(dv), _ptr(row_tiles), _ptr(counters),
                                   _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   B, Hq, Hkv, Nq, Nk, D, causal, scale, tau, _out_code(o),
                                   _out_code(dq, dk, dv), _stream(stream)))


def _decode_specs(q, k_cache, v_cache, o, lse, head_tiles, counters, workspace, cache_lens):
    B, Hq, D = _dims(q, "q", 3)
    _spec(q, "q", torch.bfloat16, (B, Hq, D))
    _, Hkv, Nk, _ = _dims(k_cache, "k_cache", 4)
    _spec(k_cache, "k_cache", torch.bfloat16, (B, Hkv, Nk, D))
    _spec(v_cache, "v_cache", torch.bfloat16, (B, Hkv, Nk, D))
    _spec(o, "o", _OUT, (B, Hq, D))
    _spec(lse, "lse", torch.float32, (B, Hq))
    _spec(head_tiles, "head_tiles", torch.int32, (B, Hq), optional=True)
    _spec(counters, "counters", torch.int64, (NUM_COUNTERS,), optional=True)
    _spec(cache_lens, "cache_lens", torch.int32, (B,), optional=True)
    if workspace is not None:
        _workspace(workspace)
    return B, Hq, Hkv, Nk, D


def mala_decode(q, k_cache, v_cache, o, lse, head_tiles, counters, num_splits, workspace, scale,
                tau, stream=None, cache_lens=None):
    B, Hq, Hkv, Nk, D = _decode_specs(q, k_cache, v_cache, o, lse, head_tiles, counters,
                                      workspace, cache_lens)
    if workspace is None:
        raise TypeError("workspace is required")
    _on_device((("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("o", o), ("lse", lse),
                ("head_tiles", head_tiles), ("counters", counters), ("workspace", workspace),
                ("cache_lens", cache_lens)))
    _check(load_library().mala_decode(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(cache_lens),
                                      _ptr(o), _ptr(lse), _ptr(head_tiles), _ptr(counters),
                                      num_splits, _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), B, Hq, Hkv,
                                      Nk, D, scale, tau, _out_code(o), _stream(stream)))


def mala_decode_noalloc(q, k_cache, v_cache, o, lse, head_tiles, counters, num_splits, scale,
                        tau, stream=None, cache_lens=None):
    """mala_decode without a workspace: the split partials use the library's own
    buffer of DECODE_SCRATCH_BYTES on the GPU (for callers that cannot allocate).
    Neither this function nor the library allocates device memory; calls that may
    overlap on one GPU race on that buffer."""
    B, Hq, Hkv, Nk, D = _decode_specs(q, k_cache, v_cache, o, lse, head_tiles, counters, None,
                                      cache_lens)
    _on_device((("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("o", o), ("lse", lse),
                ("head_tiles", head_tiles), ("counters", counters), ("cache_lens", cache_lens)))
    _check(load_library().mala_decode_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache),
                                              _ptr(cache_lens), _ptr(o), _ptr(lse),
                                              _ptr(head_tiles), _ptr(counters), num_splits, B, Hq,
                                              Hkv, Nk, D, scale, tau, _out_code(o),
                                              _stream(stream)))


def _varlen_specs(q, k, v, cu_seqlens, max_seqlen, cu_seqlens_k, max_seqlen_k, o, lse,
                  row_tiles, counters):
    """Sizes of a packed batch: q [Hq, total_q, D], k, v [Hkv, total_k, D], the int32
    [num_seqs + 1] arrays of query and (optionally) key starts, and the longest runs.
    Returns (num_seqs, Hq, Hkv, total_q, total_k, D, max_q, max_k)."""
    Hq, tq, D = _dims(q, "q", 3)
    _spec(q, "q", torch.bfloat16, (Hq, tq, D))
    Hkv, tk, _ = _dims(k, "k", 3)
    _spec(k, "k", torch.bfloat16, (Hkv, tk, D))
    _spec(v, "v", torch.bfloat16, (Hkv, tk, D))
    (n1,) = _dims(cu_seqlens, "cu_seqlens", 1)
    _spec(cu_seqlens, "cu_seqlens", torch.int32, (n1,))
    if n1 < 2:
        raise ValueError("cu_seqlens needs at least one sequence (two entries)")
    if cu_seqlens_k is None:
        max_seqlen_k = max_seqlen
    else:
        _spec(cu_seqlens_k, "cu_seqlens_k", torch.int32, (n1,))
        if max_seqlen_k is None:
            raise ValueError("cu_seqlens_k needs max_seqlen_k")
    _spec(o, "o", _OUT, (Hq, tq, D))
    _spec(lse, "lse", torch.float32, (Hq, tq))
    _stats_specs(row_tiles, counters, (Hq, tq))
    return n1 - 1, Hq, Hkv, tq, tk, D, int(max_seqlen), int(max_seqlen_k)


def mala_fwd_varlen(q, k, v, cu_seqlens, max_seqlen, o, lse, row_tiles, counters, scale, tau,
                    stream=None, cu_seqlens_k=None, max_seqlen_k=None):
    S, Hq, Hkv, tq, tk, D, mq, mk = _varlen_specs(q, k, v, cu_seqlens, max_seqlen, cu_seqlens_k,
                                                  max_seqlen_k, o, lse, row_tiles, counters)
    _on_device((("q", q), ("k", k), ("v", v), ("cu_seqlens", cu_seqlens),
                ("cu_seqlens_k", cu_seqlens_k), ("o", o), ("lse", lse),
                ("row_tiles", row_tiles), ("counters", counters)))
    _check(load_library().mala_fwd_varlen(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens),
                                          _ptr(cu_seqlens_k), _ptr(o), _ptr(lse),
                                          _ptr(row_tiles), _ptr(counters), S, mq, mk, tq, tk,
                                          Hq, Hkv, D, scale, tau, _out_code(o), _stream(stream)))


def mala_bwd_varlen(q, k, v, cu_seqlens, max_seqlen, o, lse, dout, dq, dk, dv, row_tiles,
                    counters, workspace, scale, tau, stream=None, cu_seqlens_k=None,
                    max_seqlen_k=None):
    S, Hq, Hkv, tq, tk, D, mq, mk = _varlen_specs(q, k, v, cu_seqlens, max_seqlen, cu_seqlens_k,
                                                  max_seqlen_k, o, lse, row_tiles, counters)
    _spec(dout, "dout", torch.bfloat16, (Hq, tq, D))
    _spec(dq, "dq", _OUT, (Hq, tq, D))
    _spec(dk, "dk", _OUT, (Hkv, tk, D))
    _spec(dv, "dv", _OUT, (Hkv, tk, D))
    _out_code(dq, dk, dv)
    _workspace(workspace)
    _on_device((("q", q), ("k", k), ("v", v), ("cu_seqlens", cu_seqlens),
                ("cu_seqlens_k", cu_seqlens_k), ("o", o), ("lse", lse), ("dout", dout),
                ("dq", dq), ("dk", dk), ("dv", dv), ("row_tiles", row_tiles),
                ("counters", counters), ("workspace", workspace)))
    _check(load_library().mala_bwd_varlen(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens),
                                          _ptr(cu_seqlens_k), _ptr(o), _ptr(lse), _ptr(dout),
                                          _ptr(dq), _ptr(dk), _ptr(dv), _ptr(row_tiles),
                                          _ptr(counters), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(), S, mq,
                                          mk, tq, tk, Hq, Hkv, D, scale, tau, _out_code(o),
                                          _out_code(dq, dk, dv), _stream(stream)))


# ---------------------------------------------------------------- allocating wrappers
def fwd(q, k, v, scale, tau, stats=True, stream=None, out_dtype=torch.float32):
    """out_dtype: torch.float32 or torch.bfloat16 for O (LSE is always fp32)."""
    B, Hq, Nq, D = q.shape
    o = torch.empty((B, Hq, Nq, D), dtype=out_dtype, device=q.device)
    lse = torch.empty((B, Hq, Nq), dtype=torch.float32, device=q.device)
    rt = torch.empty((B, Hq, Nq), dtype=torch.int32, device=q.device) if stats else None
    cnt = torch.empty(NUM_COUNTERS, dtype=torch.int64, device=q.device) if stats else None
    mala_fwd(q, k, v, o, lse, rt, cnt, scale, tau, stream=stream)
    return dict(o=o, lse=lse, row_tiles=rt, counters=cnt)


def bwd(q, k, v, o, lse, dout, scale, tau, stats=True, workspace=None, stream=None,
        grad_dtype=torch.float32):
    """o as fwd returned it (fp32 or bf16); grad_dtype: fp32 or bf16 dQ, dK, dV."""
    B, Hq, Nq, D = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    dq = torch.empty((B, Hq, Nq, D), dtype=grad_dtype, device=q.device)
    dk = torch.empty((B, Hkv, Nk, D), dtype=grad_dtype, device=q.device)
    dv = torch.empty((B, Hkv, Nk, D), dtype=grad_dtype, device=q.device)
    rt = torch.empty((B, Hq, Nq), dtype=torch.int32, device=q.device) if stats else None
    cnt = torch.empty(NUM_COUNTERS, dtype=torch.int64, device=q.device) if stats else None
    if workspace is None:
        n = mala_bwd_workspace_size(B, Hq, Hkv, Nq, Nk, D)
        workspace = torch.empty(max(n, 16), dtype=torch.uint8, device=q.device)
    mala_bwd(q, k, v, o, lse, dout, dq, dk, dv, rt, cnt, workspace, scale, tau, stream=stream)
    return dict(dq=dq, dk=dk, dv=dv, row_tiles=rt, counters=cnt)


def decode(q, k_cache, v_cache, scale, tau, num_splits, stats=True, workspace=None, stream=None,
           cache_lens=None, out_dtype=torch.float32):
    """cache_lens: optional int32 [B] device tensor of valid cache tokens per sequence
    (keys [0, n_b) of k_cache[b] / v_cache[b]); None means every sequence holds Nk."""
    B, Hq, D = q.shape
    o = torch.empty((B, Hq, D), dtype=out_dtype, device=q.device)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    ht = torch.empty((B, Hq), dtype=torch.int32, device=q.device) if stats else None
    cnt = torch.empty(NUM_COUNTERS, dtype=torch.int64, device=q.device) if stats else None
    if workspace is None:
        n = mala_decode_workspace_size(B, Hq, D, num_splits)
        workspace = torch.empty(max(n, 16), dtype=torch.uint8, device=q.device)
    mala_decode(q, k_cache, v_cache, o, lse, ht, cnt, num_splits, workspace, scale, tau,
                stream=stream, cache_lens=cache_lens)
    return dict(o=o, lse=lse, head_tiles=ht, counters=cnt)


def fwd_varlen(q, k, v, cu_seqlens, max_seqlen, scale, tau, stats=True, stream=None,
               out_dtype=torch.float32, cu_seqlens_k=None, max_seqlen_k=None):
    """Packed batch: q [Hq, total_q, D], k, v [Hkv, total_k, D], cu_seqlens (and, for
    prefill against cached keys, cu_seqlens_k) int32 [S + 1].  Rows that no sequence
    covers come back as zeros."""
    Hq, total, D = q.shape
    o = torch.zeros((Hq, total, D), dtype=out_dtype, device=q.device)
    lse = torch.zeros((Hq, total), dtype=torch.float32, device=q.device)
    rt = torch.zeros((Hq, total), dtype=torch.int32, device=q.device) if stats else None
    cnt = torch.empty(NUM_COUNTERS, dtype=torch.int64, device=q.device) if stats else None
    mala_fwd_varlen(q, k, v, cu_seqlens, max_seqlen, o, lse, rt, cnt, scale, tau, stream=stream,
                    cu_seqlens_k=cu_seqlens_k, max_seqlen_k=max_seqlen_k)
    return dict(o=o, lse=lse, row_tiles=rt, counters=cnt)


def bwd_varlen(q, k, v, cu_seqlens, max_seqlen, o, lse, dout, scale, tau, stats=True,
               workspace=None, stream=None, grad_dtype=torch.float32, cu_seqlens_k=None,
               max_seqlen_k=None):
    Hq, total, D = q.shape
    Hkv, total_k = k.shape[0], k.shape[1]
    dq = torch.zeros((Hq, total, D), dtype=grad_dtype, device=q.device)
    dk = torch.zeros((Hkv, total_k, D), dtype=grad_dtype, device=q.device)
    dv = torch.zeros((Hkv, total_k, D), dtype=grad_dtype, device=q.device)
    rt = torch.zeros((Hq, total), dtype=torch.int32, device=q.device) if stats else None
    cnt = torch.empty(NUM_COUNTERS, dtype=torch.int64, device=q.device) if stats else None
    if workspace is None:
        mk = max_seqlen if cu_seqlens_k is None else max_seqlen_k
        n = mala_bwd_varlen_workspace_size(cu_seqlens.shape[0] - 1, int(mk), total, Hq, Hkv, D)
        workspace = torch.empty(max(n, 16), dtype=torch.uint8, device=q.device)
    mala_bwd_varlen(q, k, v, cu_seqlens, max_seqlen, o, lse, dout, dq, dk, dv, rt, cnt,
                    workspace, scale, tau, stream=stream, cu_seqlens_k=cu_seqlens_k,
                    max_seqlen_k=max_seqlen_k)
    return dict(dq=dq, dk=dk, dv=dv, row_tiles=rt, counters=cnt)


def default_num_splits(B, Hkv, Nk, num_cus=256, waves_per_simd=2):
    """Splits that give about num_cus * 4 * waves_per_simd decode wavefronts (one
    wavefront per batch x KV head x split), capped so that each split keeps at
    least 16 tiles of 32 keys."""
    tiles = -(-Nk // 32)
    want = max(1, (num_cus * 4 * waves_per_simd) // max(1, B * Hkv))
    return int(max(1, min(want, tiles // 16 if tiles >= 16 else 1)))

"""fp64 CPU oracle for MALA causal attention (forward, backward, split-KV decode).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no code
with the HIP library: the arithmetic lives in ``mala_oracle.c`` (plain C, fp64),
this file only marshals numpy arrays and loops over batch and heads.

Conventions (the paper's problem statement, Methodology section):
  * tensors are [B, H, N, D] float64 arrays holding the exact bf16 input values;
  * GQA maps query head h to key/value head h // (Hq // Hkv);
  * causal visibility is bottom-right aligned, L_q = q + 1 + Nk - Nq;
  * lse is the natural-log normalizer z_q = log Z_{R,q}.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mala_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int32)
_bp = ctypes.POINTER(ctypes.c_int8)


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no fast-math, OpenMP over blocks)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
                               "-fPIC", "-shared", "-std=c11", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        i, d = ctypes.c_int, ctypes.c_double
        lib.oracle_dense_fwd.argtypes = [_dp, _dp, _dp, i, i, i, d, i, i, _dp, _dp]
        lib.oracle_dense_bwd.argtypes = [_dp, _dp, _dp, _dp, i, i, i, d, _dp, _dp, _dp]
        lib.oracle_mala_fwd.argtypes = [_dp, _dp, _dp, i, i, i, d, d, i, i, i, i,
                                        _dp, _dp, _ip, _dp, _dp, _bp]
        lib.oracle_mala_bwd.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp, i, i, i, d, d, i, i,
                                        i, i, i, i, _dp, _dp, _dp, _ip, _dp, _dp, _bp]
        lib.oracle_mala_decode.argtypes = [_dp, _dp, _dp, i, i, d, d, i, i, _dp, _dp, _ip,
                                           _dp, _dp, _bp]
        for f in ("oracle_dense_fwd", "oracle_dense_bwd", "oracle_mala_fwd", "oracle_mala_bwd",
                  "oracle_mala_decode"):
            getattr(lib, f).restype = None
        _lib = lib
    return _lib


def _p(a, t=_dp):
    return None if a is None else a.ctypes.data_as(t)


def _c64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _group(Hq, Hkv):
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    return Hq // Hkv


def dense_fwd(q, k, v, scale):
    """Dense causal attention by its definition. Returns (o, lse)."""
    lib = _load()
    q, k, v = _c64(q), _c64(k), _c64(v)
    B, Hq, Nq, D = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    g = _group(Hq, Hkv)
    o = np.zeros_like(q)
    lse = np.zeros((B, Hq, Nq))
    for b in range(B):
        for h in range(Hq):
            oh, lh = np.zeros((Nq, D)), np.zeros(Nq)
            lib.oracle_dense_fwd(_p(q[b, h]), _p(k[b, h // g]), _p(v[b, h // g]), Nq, Nk, D,
                                 scale, 0, Nq, _p(oh), _p(lh))
            o[b, h], lse[b, h] = oh, lh
    return o, lse


def dense_bwd(q, k, v, do, scale):
    """Gradient of <O, dO> of dense causal attention. Returns (dq, dk, dv)."""
    lib = _load()
    q, k, v, do = _c64(q), _c64(k), _c64(v), _c64(do)
    B, Hq, Nq, D = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    g = _group(Hq, Hkv)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(Hq):
            dqh = np.zeros((Nq, D))
            dkh = np.ascontiguousarray(dk[b, h // g])
            dvh = np.ascontiguousarray(dv[b, h // g])
            lib.oracle_dense_bwd(_p(q[b, h]), _p(k[b, h // g]), _p(v[b, h // g]), _p(do[b, h]),
                                 Nq, Nk, D, scale, _p(dqh), _p(dkh), _p(dvh))
            dq[b, h], dk[b, h // g], dv[b, h // g] = dqh, dkh, dvh
    return dq, dk, dv


def mala_fwd(q, k, v, scale, tau, bq, bk, blocks=None, heads=None, want_tiles=False):
    """Algorithm 1 (MALA forward) in fp64.

    blocks: optional (i0, i1) range of query blocks; heads: optional list of
    (b, h) pairs.  Rows outside the processed blocks/heads are left as NaN (o,
    lse, ties) and -1 (row_tiles).
    Returns dict with o, lse, row_tiles, tie_abs, tie_rel and (want_tiles)
    tile_keep[B, Hq, Tr, Tc].
    """
    lib = _load()
    q, k, v = _c64(q), _c64(k), _c64(v)
    B, Hq, Nq, D = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    g = _group(Hq, Hkv)
    Tr, Tc = -(-Nq // bq), -(-Nk // bk)
    i0, i1 = blocks if blocks is not None else (0, Tr)
    o = np.full(q.shape, np.nan)
    lse = np.full((B, Hq, Nq), np.nan)
    rt = np.full((B, Hq, Nq), -1, dtype=np.int32)
    ta = np.full((B, Hq, Nq), np.nan)
    tr = np.full((B, Hq, Nq), np.nan)
    keep = np.full((B, Hq, Tr, Tc), -1, dtype=np.int8) if want_tiles else None
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hq)]
    for b, h in pairs:
        oh, lh = np.full((Nq, D), np.nan), np.full(Nq, np.nan)
        rth = np.full(Nq, -1, dtype=np.int32)
        tah, trh = np.full(Nq, np.nan), np.full(Nq, np.nan)
        kh = np.full((Tr, Tc), -1, dtype=np.int8) if want_tiles else None
        lib.oracle_mala_fwd(_p(q[b, h]), _p(k[b, h // g]), _p(v[b, h // g]), Nq, Nk, D, scale,
                            tau, bq, bk, i0, i1, _p(oh), _p(lh), _p(rth, _ip), _p(tah), _p(trh),
                            _p(kh, _bp))
        o[b, h], lse[b, h], rt[b, h], ta[b, h], tr[b, h] = oh, lh, rth, tah, trh
        if want_tiles:
            keep[b, h] = kh
    out = dict(o=o, lse=lse, row_tiles=rt, tie_abs=ta, tie_rel=tr)
    if want_tiles:
        out["tile_keep"] = keep
    return out


def mala_bwd(q, k, v, o, lse, do, scale, tau, bq, bk, qblocks=None, kblocks=None,
             want_tiles=False):
    """Algorithm 2 (MALA backward) in fp64, given the forward's o and lse.

    qblocks: (i0, i1) query blocks whose dq rows are computed (default all);
    kblocks: (j0, j1) key blocks whose dk/dv rows are computed (default all).
    dk, dv of a key/value head sum over the query heads of its GQA group.
    Returns dict with dq, dk, dv, row_tiles, tie_abs, tie_rel (+ tile_keep).
    """
    lib = _load()
    q, k, v, o, lse, do = _c64(q), _c64(k), _c64(v), _c64(o), _c64(lse), _c64(do)
    B, Hq, Nq, D = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    g = _group(Hq, Hkv)
    Tr, Tc = -(-Nq // bq), -(-Nk // bk)
    qi0, qi1 = qblocks if qblocks is not None else (0, Tr)
    kj0, kj1 = kblocks if kblocks is not None else (0, Tc)
    dq = np.full(q.shape, np.nan)
    dk = np.zeros(k.shape)
    dv = np.zeros(v.shape)
    rt = np.full((B, Hq, Nq), -1, dtype=np.int32)
    ta = np.full((B, Hq, Nq), np.nan)
    tr = np.full((B, Hq, Nq), np.nan)
    keep = np.full((B, Hq, Tr, Tc), -1, dtype=np.int8) if want_tiles else None
    for b in range(B):
        for h in range(Hq):
            dqh = np.full((Nq, D), np.nan)
            dkh = np.ascontiguousarray(dk[b, h // g])
            dvh = np.ascontiguousarray(dv[b, h // g])
            rth = np.full(Nq, -1, dtype=np.int32)
            tah, trh = np.full(Nq, np.nan), np.full(Nq, np.nan)
            kh = np.full((Tr, Tc), -1, dtype=np.int8) if want_tiles else None
            lib.oracle_mala_bwd(_p(q[b, h]), _p(k[b, h // g]), _p(v[b, h // g]), _p(o[b, h]),
                                _p(lse[b, h]), _p(do[b, h]), Nq, Nk, D, scale, tau, bq, bk,
                                qi0, qi1, kj0, kj1, _p(dqh), _p(dkh), _p(dvh), _p(rth, _ip),
                                _p(tah), _p(trh), _p(kh, _bp))
            dq[b, h], dk[b, h // g], dv[b, h // g] = dqh, dkh, dvh
            rt[b, h], ta[b, h], tr[b, h] = rth, tah, trh
            if want_tiles:
                keep[b, h] = kh
    out = dict(dq=dq, dk=dk, dv=dv, row_tiles=rt, tie_abs=ta, tie_rel=tr)
    if want_tiles:
        out["tile_keep"] = keep
    return out


def mala_decode(q, kc, vc, scale, tau, bk, num_splits, heads=None, want_tiles=False):
    """Split-KV MALA decode of one query token per (b, h) over a KV cache.

    q: [B, Hq, D]; kc, vc: [B, Hkv, Nk, D].  heads: optional list of (b, h).
    Returns dict with o[B, Hq, D], lse[B, Hq], tiles[B, Hq] (retained tiles summed
    over splits), tie_abs, tie_rel (+ keep[B, Hq, T] per-tile decisions).
    """
    lib = _load()
    q, kc, vc = _c64(q), _c64(kc), _c64(vc)
    B, Hq, D = q.shape
    Hkv, Nk = kc.shape[1], kc.shape[2]
    g = _group(Hq, Hkv)
    T = -(-Nk // bk)
    o = np.full((B, Hq, D), np.nan)
    lse = np.full((B, Hq), np.nan)
    tiles = np.full((B, Hq), -1, dtype=np.int32)
    ta = np.full((B, Hq), np.nan)
    tr = np.full((B, Hq), np.nan)
    keep = np.full((B, Hq, T), -1, dtype=np.int8) if want_tiles else None
    pairs = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hq)]
    for b, h in pairs:
        oh = np.zeros(D)
        l_, t_, a_, r_ = (np.zeros(1), np.zeros(1, dtype=np.int32), np.zeros(1), np.zeros(1))
        kh = np.full(T, -1, dtype=np.int8) if want_tiles else None
        lib.oracle_mala_decode(_p(q[b, h]), _p(kc[b, h // g]), _p(vc[b, h // g]), Nk, D, scale,
                               tau, bk, num_splits, _p(oh), _p(l_), _p(t_, _ip), _p(a_), _p(r_),
                               _p(kh, _bp))
        o[b, h], lse[b, h], tiles[b, h], ta[b, h], tr[b, h] = oh, l_[0], t_[0], a_[0], r_[0]
        if want_tiles:
            keep[b, h] = kh
    out = dict(o=o, lse=lse, tiles=tiles, tie_abs=ta, tie_rel=tr)
    if want_tiles:
        out["keep"] = keep
    return out

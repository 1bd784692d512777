"""Seeded synthetic inputs for MALA attention, shared by the HIP path's tests and
benchmark and by the oracle's tests.  This module holds none of the method's
arithmetic: it only draws random numbers and rounds them to bf16.

The paper measures operator latency on unspecified inputs and operator fidelity
on hidden states of a 14B checkpoint that is not available; these generators
stand in for both.  Recipe (identical for every workload):

  * one independent PCG64 stream per (tensor, batch, head), seeded with
    ``numpy.random.default_rng([seed, stream_id, tensor_id, b, h])`` (stream_id
    fixed per named workload, 0 for specs given as dicts), so any single head can
    be regenerated without drawing the others;
  * standard normals drawn as float32 (PCG64 + ziggurat), combined in float64,
    and rounded to bf16 with round-to-nearest-even;
  * K and V ~ N(0, 1); dO ~ N(0, 1);
  * planted-needle queries: Q_i = g_i + beta * K_{r(i)} with g ~ N(0, 1) and
    r(i) uniform on {0..i}, built from the ROUNDED K of the head's KV head and
    rounded again; optional local term Q_i += alpha * K_{i-1};
  * language-model-like structure (options of the same generator): needles shared
    by blocks of rows (rows of block c draw one r(c), uniform on {0 .. first row of
    the block}), an attention sink (Q_i += sink * K_0), and a Rademacher dO probe
    (entries +-1 with equal probability);
  * decode queries: q = g + beta * sum of K at 4 distinct random positions.

Arrays are returned as uint16 bf16 bit patterns in [B, H, N, D] layout.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

# tensor ids of the per-slice streams
_T_K, _T_V, _T_Q, _T_DO, _T_BETA, _T_POS = 1, 2, 3, 4, 5, 6

# The named workloads.  "kind": "train" (fwd + bwd) or "decode".
WORKLOADS = {
    "needle_1k_d64": dict(kind="train", B=1, Hq=1, Hkv=1, N=1024, D=64, beta=2.0, local=0.0,
            taus=(0.0, 1e-4, 1e-3), desc="causal fwd+bwd, 1x1x1024x64, needle beta=2"),
    "mha16_8k": dict(kind="train", B=1, Hq=16, Hkv=16, N=8192, D=128, beta=2.0, local=1.0,
            taus=(0.0, 1e-4, 1e-3),
            desc="causal fwd+bwd, MHA 16 heads, 8192x128, needle beta=2 + local 1.0"),
    "gqa32x8_32k": dict(kind="train", B=1, Hq=32, Hkv=8, N=32768, D=128, beta=(0.5, 3.0), local=0.0,
            taus=(0.0, 1e-4), desc="causal fwd+bwd, GQA 32/8, 32768x128, per-head beta~U[0.5,3]"),
    "gqa8x2_128k": dict(kind="train", B=1, Hq=8, Hkv=2, N=131072, D=128, beta=2.0, local=0.0,
            taus=(0.0, 1e-4),
            desc="causal fwd+bwd, GQA 8/2 (one TP=8 share), 131072x128, beta=2"),
    "decode_gqa32x8_128k": dict(kind="decode", B=16, Hq=32, Hkv=8, N=131072, D=128, beta=3.0, needles=4,
            taus=(0.0, 1e-4),
            desc="decode, 16 x GQA 32/8 over 131072-token caches, 4 needles beta=3"),
    # supplementary: a workload on which the forward rule can skip (a dominant local
    # key found in the diagonal tile, needles shared by 32-row blocks, a sink), with
    # a Rademacher dO for the fidelity measurements
    "lm_like_gqa8x2_32k": dict(kind="train", B=1, Hq=8, Hkv=2, N=32768, D=128, beta=2.0, local=2.0,
            needle_block=32, sink=1.5, do="rademacher", taus=(0.0, 1e-4, 1.0),
            desc="causal fwd+bwd, GQA 8/2, 32768x128, LM-like: local 2, block needles beta=2, "
                 "sink 1.5"),
}
# the random-stream id of each named workload (part of every generator seed)
STREAM = {"needle_1k_d64": 1, "mha16_8k": 2, "gqa32x8_32k": 3, "gqa8x2_128k": 4,
          "decode_gqa32x8_128k": 5, "lm_like_gqa8x2_32k": 6}


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (round-to-nearest-even); return uint16 bits.

    Rounds the float64 bit pattern directly at bf16's last mantissa bit (no
    intermediate float32 rounding, hence no double rounding): add 2^44 - 1 plus the
    bit that will become the last kept one, then clear the 45 dropped bits.  The
    bit arithmetic runs in torch (CPU, multi-threaded).  Magnitudes outside the
    normal bf16 range take an exact slower path."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    xt = torch.from_numpy(x)
    u = xt.view(torch.int64)
    r = ((u + (((u >> 45) & 1) + ((1 << 44) - 1))) >> 45) << 45
    bits = (r.view(torch.float64).to(torch.float32).view(torch.int32) >> 16) & 0xFFFF
    out = bits.to(torch.int16).numpy().view(np.uint16)
    ax = xt.abs()
    odd_t = (ax < 2.0 ** -126) | (ax >= 2.0 ** 127) | ~torch.isfinite(xt)
    if bool(odd_t.any()):
        odd = odd_t.numpy()
        xs = x[odd]
        m, e = np.frexp(xs)
        rs = np.ldexp(np.round(np.ldexp(m, 8)), e - 8)
        with np.errstate(over="ignore", invalid="ignore"):
            out[odd] = (rs.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float64 (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def _rng(seed, stream, tensor, b, h):
    return np.random.default_rng([int(seed), int(stream), tensor, int(b), int(h)])


def _normal(seed, stream, tensor, b, h, shape):
    return _rng(seed, stream, tensor, b, h).standard_normal(shape, dtype=np.float32)


def _normal_bits(seed, stream, tensor, b, h, shape):
    return bf16_round(_normal(seed, stream, tensor, b, h, shape))


class Workload:
    """Lazily generated inputs of one workload (any subset of heads): a name of
    WORKLOADS or a spec dict."""

    def __init__(self, workload, seed: int = 0, **overrides):
        if isinstance(workload, str):
            self.stream = STREAM[workload]
            spec = dict(WORKLOADS[workload])
        else:
            spec = dict(workload)
            self.stream = int(spec.pop("id", 0))
        spec.update(overrides)
        self.spec = spec
        self.seed = seed
        self.kind = spec["kind"]
        self.B, self.Hq, self.Hkv = spec["B"], spec["Hq"], spec["Hkv"]
        self.N, self.D = spec["N"], spec["D"]
        self.g = self.Hq // self.Hkv
        self.scale = 1.0 / math.sqrt(self.D)
        self._k = {}

    # ---- per-slice generators -------------------------------------------
    def k_head(self, b, hkv):
        key = (b, hkv)
        if key not in self._k:
            self._k[key] = _normal_bits(self.seed, self.stream, _T_K, b, hkv, (self.N, self.D))
        return self._k[key]

    def v_head(self, b, hkv):
        return _normal_bits(self.seed, self.stream, _T_V, b, hkv, (self.N, self.D))

    def do_head(self, b, h):
        if self.spec.get("do") == "rademacher":
            rng = _rng(self.seed, self.stream, _T_DO, b, h)
            return bf16_round(rng.integers(0, 2, size=(self.N, self.D)) * 2.0 - 1.0)
        return _normal_bits(self.seed, self.stream, _T_DO, b, h, (self.N, self.D))

    def beta(self, h):
        beta = self.spec["beta"]
        if isinstance(beta, tuple):
            lo, hi = beta
            return float(_rng(self.seed, self.stream, _T_BETA, 0, h).uniform(lo, hi))
        return float(beta)

    def q_head(self, b, h):
        """Planted-needle query rows for a training workload (or the decode query)."""
        kf = bf16_to_f64(self.k_head(b, h // self.g))
        rng = _rng(self.seed, self.stream, _T_Q, b, h)
        beta = self.beta(h)
        if self.kind == "decode":
            g = rng.standard_normal(self.D, dtype=np.float32).astype(np.float64)
            n = self.spec.get("needles", 4)
            pos = rng.choice(self.N, size=n, replace=False)
            return bf16_round(g + beta * kf[pos].sum(axis=0))
        N = self.N
        g = rng.standard_normal((N, self.D), dtype=np.float32).astype(np.float64)
        nb = int(self.spec.get("needle_block", 1))
        if nb > 1:   # one needle per block of nb rows, visible to all of them
            starts = np.arange(0, N, nb)
            r = np.repeat(rng.integers(0, starts + 1), nb)[:N]
        else:
            r = rng.integers(0, np.arange(1, N + 1))    # r(i) uniform on {0..i}
        q = g + beta * kf[r]
        alpha = float(self.spec.get("local", 0.0))
        if alpha:
            q[1:] += alpha * kf[:-1]
        sink = float(self.spec.get("sink", 0.0))
        if sink:
            q += sink * kf[0]
        return bf16_round(q)

    def needle_rows(self, b, h):
        """Training only: the key r(i) planted in each query row of head (b, h)."""
        rng = _rng(self.seed, self.stream, _T_Q, b, h)
        N = self.N
        rng.standard_normal((N, self.D), dtype=np.float32)
        nb = int(self.spec.get("needle_block", 1))
        if nb > 1:
            starts = np.arange(0, N, nb)
            return np.repeat(rng.integers(0, starts + 1), nb)[:N]
        return rng.integers(0, np.arange(1, N + 1))

    def needle_positions(self, b, h):
        """Decode only: the planted positions of query head (b, h)."""
        rng = _rng(self.seed, self.stream, _T_Q, b, h)
        rng.standard_normal(self.D, dtype=np.float32)
        return np.sort(rng.choice(self.N, size=self.spec.get("needles", 4), replace=False))

    # ---- whole tensors ---------------------------------------------------
    def _stack(self, fn, H, threads):
        idx = [(b, h) for b in range(self.B) for h in range(H)]
        with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
            parts = list(ex.map(lambda bh: fn(*bh), idx))
        shape = parts[0].shape
        out = np.empty((self.B, H) + shape, dtype=np.uint16)
        for (b, h), p in zip(idx, parts):
            out[b, h] = p
        return out

    def tensors(self, threads: int = 8, with_do: bool = True):
        """All inputs as uint16 bf16 bits: q [B,Hq,N,D] (decode: [B,Hq,D]), k, v [B,Hkv,N,D], do."""
        k = self._stack(self.k_head, self.Hkv, threads)
        v = self._stack(self.v_head, self.Hkv, threads)
        q = self._stack(self.q_head, self.Hq, threads)
        out = dict(q=q, k=k, v=v)
        if with_do and self.kind == "train":
            out["do"] = self._stack(self.do_head, self.Hq, threads)
        self._k.clear()
        return out

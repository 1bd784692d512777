"""Helpers shared by the GPU parity tests: device upload of bf16 bit patterns,
the tolerance bar and the decision-count comparison with the tie band.

The bar (for bf16 inputs, fp32 accumulation, against the fp64 oracle):
  * O, dQ, dK, dV: max-abs <= 1e-2 and mean-abs <= 1e-3;
  * per-row retained-tile counts equal the oracle's, except on rows whose query
    block (forward) or whose tiles (backward) saw a test value T with
    |T - tau| <= 1e-5 in the oracle's own trajectory (tau > 0 only): there two
    correct finite-precision implementations may decide differently.
"""
import numpy as np
import torch

TOL_MAX = 1e-2
TOL_MEAN = 1e-3
TIE_BAND = 1e-5
LSE_DIAG = 1e-3


def dev(bits):
    """uint16 bf16 bit patterns (numpy) -> bf16 tensor on cuda:0."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to("cuda").view(torch.bfloat16)


def host(t):
    return t.detach().to("cpu").numpy().astype(np.float64)


def assert_close(name, got, ref, where=None):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if where is not None:
        got, ref = got[where], ref[where]
    assert np.isfinite(got).all(), "%s: non-finite values" % name
    err = np.abs(got - ref)
    mx, mean = float(err.max()), float(err.mean())
    print("[parity] %-12s max-abs %.3e mean-abs %.3e" % (name, mx, mean), flush=True)
    assert mx <= TOL_MAX and mean <= TOL_MEAN, "%s: max-abs %.3e mean-abs %.3e" % (name, mx, mean)
    return mx, mean


def exempt_rows(tau, *ties):
    """Rows exempt from count parity: any given tie array within the band (tau > 0)."""
    ex = np.zeros(np.shape(ties[0]), dtype=bool)
    if tau > 0:
        for t in ties:
            ex |= np.nan_to_num(np.asarray(t), nan=np.inf) <= TIE_BAND
    return ex


def assert_counts(name, got, ref, exempt):
    got = np.asarray(got)
    ref = np.asarray(ref)
    bad = (got != ref) & ~exempt
    assert not bad.any(), "%s: %d rows differ outside the tie band (first %s: gpu %s oracle %s)" % (
        name, int(bad.sum()), np.argwhere(bad)[:3].tolist(), got[bad][:3], ref[bad][:3])
    return float(exempt.mean())

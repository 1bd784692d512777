"""Helpers shared by the GPU parity tests: device upload of bf16 bit patterns,
the tolerance bar and the decision-count comparison with the tie band.

The bar (for bf16 inputs, fp32 accumulation, against the fp64 oracle):
  * O, dQ, dK, dV: max-abs <= 1e-2 and mean-abs <= 1e-3;
  * per-row retained-tile counts equal the oracle's, except on rows whose query
    block (forward) or whose tiles (backward) saw a decisive test value T with
    |T - tau| <= 1e-5 in the oracle's own trajectory (tau > 0 only): there two
    correct finite-precision implementations may decide differently.
Beyond that rule, every comparison of counts reports the fraction of rows the
absolute band exempts, the fraction inside the relative band |T / tau - 1| <= 1e-5
(a diagnostic: at tau = 1e-4 the absolute band is +-10% of tau), and the rows
that actually differ; at most 1% of the rows (and at least one) may differ.  The
figures are collected and printed at the end of the pytest run.
"""
import math
import os

import numpy as np
import torch

TOL_MAX = 1e-2
TOL_MEAN = 1e-3
TIE_BAND = 1e-5
LSE_DIAG = 1e-3
MAX_DIFFER_FRAC = 0.01

# one entry per count comparison: (test, name, rows, exempt, relative band, differing)
COUNT_LOG = []


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


def ties(out, sl=()):
    """The (tie_abs, tie_rel) pair of an oracle result dict, optionally sliced."""
    return np.asarray(out["tie_abs"])[sl], np.asarray(out["tie_rel"])[sl]


def tie_masks(tau, *pairs):
    """Rows exempt from count parity (|T - tau| <= TIE_BAND for a tile of the row in
    any given oracle trajectory, tau > 0) and rows inside the relative band
    |T / tau - 1| <= TIE_BAND.  pairs: (tie_abs, tie_rel) arrays of one shape."""
    ex = np.zeros(np.shape(pairs[0][0]), dtype=bool)
    rel = np.zeros_like(ex)
    if tau > 0:
        for a, r in pairs:
            ex |= np.nan_to_num(np.asarray(a, dtype=np.float64), nan=np.inf) <= TIE_BAND
            rel |= np.nan_to_num(np.asarray(r, dtype=np.float64), nan=np.inf) <= TIE_BAND
    return ex, rel


def assert_counts(name, got, ref, tau, *pairs):
    """Per-row retained-tile counts: equal outside the tie band, and at most
    MAX_DIFFER_FRAC of the rows (at least one) differing inside it.  Returns the
    exempt mask."""
    got = np.asarray(got)
    ref = np.asarray(ref)
    ex, rel = tie_masks(tau, *pairs)
    differ = got != ref
    bad = differ & ~ex
    assert not bad.any(), "%s: %d rows differ outside the tie band (first %s: gpu %s oracle %s)" % (
        name, int(bad.sum()), np.argwhere(bad)[:3].tolist(), got[bad][:3], ref[bad][:3])
    n = int(got.size)
    nd = int(differ.sum())
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    COUNT_LOG.append((test, name, n, float(ex.mean()), float(rel.mean()), nd))
    print("[counts] %-22s rows %8d | exempt %.4f | relative band %.4f | differing %d"
          % (name, n, ex.mean(), rel.mean(), nd), flush=True)
    assert nd <= max(1, math.ceil(MAX_DIFFER_FRAC * n)), \
        "%s: %d of %d rows differ inside the tie band" % (name, nd, n)
    return ex


def count_summary():
    """Lines summarising COUNT_LOG for the end of the test run."""
    if not COUNT_LOG:
        return []
    rows = sum(e[2] for e in COUNT_LOG)
    differ = sum(e[5] for e in COUNT_LOG)
    w_ex = sum(e[2] * e[3] for e in COUNT_LOG) / rows
    w_rel = sum(e[2] * e[4] for e in COUNT_LOG) / rows
    lines = ["retained-tile count parity: %d comparisons, %d rows; exempt by |T - tau| <= 1e-5: "
             "%.4f of rows (largest in one comparison %.4f); inside |T / tau - 1| <= 1e-5: %.4f "
             "(largest %.4f); rows that differ: %d"
             % (len(COUNT_LOG), rows, w_ex, max(e[3] for e in COUNT_LOG), w_rel,
                max(e[4] for e in COUNT_LOG), differ)]
    top = sorted(COUNT_LOG, key=lambda e: -e[3])[:5]
    for t, name, n, ex, rel, nd in top:
        if ex > 0:
            lines.append("  exempt %.4f rel %.4f differ %d rows %d  %s %s"
                         % (ex, rel, nd, n, t.split("::")[-1], name))
    return lines


def _splitmix64(z):
    # the output function of Steele, Lea and Flood's SplitMix64 generator (uint64)
    with np.errstate(over="ignore"):
        z = z + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def set_fingerprint(keep, b0=0):
    """The retained-set fingerprint the library reports (MALA_CNT_SET_HASH) of an
    oracle decision array: keep [B, H, Tr, Tc] (forward / backward tile_keep) or
    [B, H, T] (decode keep, query tile 0), 1 = retained; b0 offsets the sequence
    index.  Sum modulo 2^64 of splitmix64(b << 52 | h << 40 | i << 20 | j), returned
    as a signed 64-bit value like the int64 counters."""
    keep = np.asarray(keep)
    if keep.ndim == 3:
        keep = keep[:, :, None, :]
    b, h, i, j = (x.astype(np.uint64) for x in np.nonzero(keep == 1))
    z = ((b + np.uint64(b0)) << np.uint64(52)) | (h << np.uint64(40)) | (i << np.uint64(20)) | j
    total = int(_splitmix64(z).sum(dtype=np.uint64)) if z.size else 0
    return total - (1 << 64) if total >= (1 << 63) else total


def fwd_v_loads(keep, rows_per_group=256, bq=32):
    """(workgroup, key tile) pairs of the forward in which some query tile of the
    workgroup retains the key tile (the V tiles a retained tile uses), for an oracle
    tile_keep [B, H, Tr, Tc]: a workgroup owns rows_per_group consecutive query rows
    of one head."""
    keep = np.asarray(keep) == 1
    B, H, Tr, Tc = keep.shape
    g = rows_per_group // bq
    pad = (-Tr) % g
    k = np.concatenate([keep, np.zeros((B, H, pad, Tc), bool)], axis=2) if pad else keep
    return int(k.reshape(B, H, -1, g, Tc).any(axis=3).sum())


def bwd_do_loads(keep, keys_per_group=128, bk=32):
    """dO tiles the key-major backward pass loads for an oracle tile_keep [B, Hq, Tr,
    Tc]: a workgroup owns keys_per_group consecutive keys of one KV head and loads a
    query tile of a query head iff that tile retains one of its key tiles."""
    keep = np.asarray(keep) == 1
    B, H, Tr, Tc = keep.shape
    g = keys_per_group // bk
    pad = (-Tc) % g
    k = np.concatenate([keep, np.zeros((B, H, Tr, pad), bool)], axis=3) if pad else keep
    return int(k.reshape(B, H, Tr, -1, g).any(axis=4).sum())


def dkdv_splits(B, Hq, Hkv, Nq, Nk=None, groups=1024, part_min=512, keys=128, bq=32):
    """Whether a fixed-length backward call of this causal shape splits its dK/dV
    sweeps (the rule of the library's launch: fewer than `groups` key-block
    workgroups, and a first sweep longer than the part size)."""
    Nk = Nq if Nk is None else Nk
    nkblk = -(-Nk // keys)
    if nkblk * B * Hkv >= groups:
        return False
    grp, nqt = Hq // Hkv, -(-Nq // bq)
    first = lambda j: max(0, j * keys - (Nk - Nq)) // bq
    total = B * Hkv * sum(grp * (nqt - first(j)) for j in range(nkblk))
    ps = part_min
    while ps * 2 * groups <= total:
        ps *= 2
    return ps < grp * nqt

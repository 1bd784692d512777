"""The operator-fidelity measurements of the benchmark (relative L2 errors per head
and the omitted mass recovered from two normalizers), checked on the CPU against
values fixed by construction and against the dense mass of the tiles the oracle
skipped, computed by brute force from the softmax definition."""
import math

import numpy as np
import pytest
import torch

import bench
import oracle


def test_head_fidelity_known_values():
    B, Hq, Hkv, N, D = 2, 3, 1, 5, 4
    rng = np.random.default_rng(0)
    ref = {k: torch.from_numpy(rng.standard_normal((B, h, N, D)))
           for k, h in (("o", Hq), ("dq", Hq), ("dk", Hkv), ("dv", Hkv))}
    ref["lse"] = torch.from_numpy(rng.standard_normal((B, Hq, N)))
    c = torch.tensor([0.5, -0.25, 0.0, 1e-3, 2.0, -1.0], dtype=torch.float64).reshape(B, Hq, 1, 1)
    out = {k: ref[k].clone() for k in ref}
    out["o"] = ref["o"] * (1 + c)             # rel L2 of head (b, h) = |c_bh|
    out["dq"] = ref["dq"] + 3 * ref["dq"]      # 3 for every head
    out["dv"] = -ref["dv"]                     # 2
    eps = torch.from_numpy(rng.uniform(0, 0.9, (B, Hq, N)))
    out["lse"] = ref["lse"] + torch.log1p(-eps)  # Z_R / Z = 1 - eps
    f = bench.head_fidelity(ref, out)
    np.testing.assert_allclose(f["o"], c.abs().flatten().numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(f["dq"], 3.0, rtol=1e-12)
    np.testing.assert_allclose(f["dk"], 0.0, atol=0)
    np.testing.assert_allclose(f["dv"], 2.0, rtol=1e-12)
    np.testing.assert_allclose(f["omitted_mass"], eps.mean(dim=2).flatten().numpy(), rtol=1e-12)
    assert f["omitted_mass_row_max"] == pytest.approx(float(eps.max()), rel=1e-12)
    assert f["o"].shape == (B * Hq,) and f["dk"].shape == (B * Hkv,)


def test_mean_p95():
    x = np.arange(1, 101, dtype=np.float64)
    m, p = bench.mean_p95(x)
    assert m == 50.5 and p == pytest.approx(95.05)
    assert bench.mean_p95([7.0]) == (7.0, 7.0)


@pytest.mark.parametrize("tau,bq,bk", [(1.0, 8, 8), (0.3, 4, 16), (1.0, 16, 4)])
def test_omitted_mass_equals_dense_mass_of_skipped_tiles(tau, bq, bk):
    # The normalizers of a screened and an unscreened forward give the dense softmax
    # mass of the keys in the skipped tiles (Appendix, omitted-mass proposition):
    # check against the softmax written out, summed over the oracle's skipped tiles.
    rng = np.random.default_rng(5)
    N, D, Hq, Hkv = 96, 16, 2, 1
    k = rng.standard_normal((1, Hkv, N, D))
    v = rng.standard_normal((1, Hkv, N, D))
    q = rng.standard_normal((1, Hq, N, D))
    for h in range(Hq):
        q[0, h, 1:] += 3.0 * k[0, 0, :-1]       # a dominant local key makes tiles skippable
    scale = 1 / math.sqrt(D)
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk, want_tiles=True)
    d = oracle.mala_fwd(q, k, v, scale, 0.0, bq, bk)
    keep = f["tile_keep"]
    assert (keep == 0).sum() > 0
    eps = bench.omitted_mass_rows(torch.from_numpy(d["lse"]), torch.from_numpy(f["lse"])).numpy()
    for h in range(Hq):
        s = q[0, h] @ k[0, 0].T * scale
        s[np.triu_indices(N, 1)] = -np.inf
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        for r in range(N):
            i = r // bq
            skipped = [j for j in range(keep.shape[3]) if keep[0, h, i, j] == 0]
            mass = sum(p[r, j * bk:(j + 1) * bk].sum() for j in skipped)
            assert abs(eps[0, h, r] - mass) <= 1e-12, (h, r, eps[0, h, r], mass)
    full = {"o": f["o"], "lse": f["lse"], "dq": f["o"], "dk": v, "dv": v}
    ref = {"o": d["o"], "lse": d["lse"], "dq": d["o"], "dk": v, "dv": v}
    fid = bench.head_fidelity({x: torch.from_numpy(y) for x, y in ref.items()},
                              {x: torch.from_numpy(y) for x, y in full.items()})
    assert (fid["omitted_mass"] <= tau / (1 + tau)).all()
    np.testing.assert_allclose(fid["omitted_mass"], eps[0].mean(axis=1), rtol=0, atol=1e-15)

"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with a retyped copy of itself:
  * dense attention against a brute-force numpy softmax (the definition);
  * dense gradients against central finite differences;
  * MALA at tau = 0 against dense (the tau -> 0 limit of the Attention Cost section);
  * MALA decisions against an independent direct-sum implementation of the rule
    (Eqs. running normalizer / contribution ratio, no m/l recurrence);
  * Proposition 1 (omitted mass <= tau/(1+tau)) and its L1/output corollaries;
  * support nesting (Offline Sparse Probability paragraph);
  * the first legal tile is always retained (empty-state convention);
  * closed-form cases: the two-token boundary and uniform scores (tests/golden);
  * the per-row tie distances (how close some tile's decisive test value T came to
    tau; they decide which rows the GPU tests exempt from count parity) against T
    from the direct sums and against the closed forms of the golden cases;
  * GQA equals MHA on repeated K/V; decode with one split equals the forward's
    last row; the split merge equals softmax restricted to the retained set;
  * MALA gradients at tau > 0 against finite differences of the softmax restricted
    to the frozen retained set, when the backward keeps the forward's support.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from workloads import Workload, bf16_round, bf16_to_f64

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# independent reference implementations (numpy / pure Python)
# --------------------------------------------------------------------------
def scores(q, k, scale):
    """[Nq, Nk] scores with -inf above the bottom-right aligned causal diagonal."""
    Nq, Nk = q.shape[0], k.shape[0]
    S = scale * (q @ k.T)
    off = Nk - Nq
    mask = np.arange(Nk)[None, :] > (np.arange(Nq)[:, None] + off)
    S[mask] = -np.inf
    return S


def softmax_rows(S, keep=None):
    """Row softmax of S (optionally restricted to keep); returns (P, lse)."""
    S = S.copy()
    if keep is not None:
        S[~keep] = -np.inf
    mx = S.max(axis=1, keepdims=True)
    E = np.exp(S - mx)
    Z = E.sum(axis=1, keepdims=True)
    return E / Z, (mx + np.log(Z))[:, 0]


def direct_sum_forward(S, tau, bq, bk):
    """The forward rule with direct sums: Z^(t) = sum of exp(s) over retained keys,
    ratio r = exp(tile row max) / Z^(t), skip iff r < tau / L for every row with a
    legal key in the tile; blocks visited from the diagonal downwards.  Also returns
    each tile's decisive value T = max over those rows of L * r (+inf while one of
    them has Z = 0), NaN for tiles that are not visited."""
    Nq, Nk = S.shape
    Tr, Tc = -(-Nq // bq), -(-Nk // bk)
    keep = np.full((Tr, Tc), -1, dtype=np.int8)
    Tval = np.full((Tr, Tc), np.nan)
    R = np.zeros((Nq, Nk), dtype=bool)
    L = np.arange(Nq) + 1 + (Nk - Nq)
    for i in range(Tr):
        rows = range(i * bq, min(Nq, (i + 1) * bq))
        Z = {r: 0.0 for r in rows}
        top = (max(rows) + Nk - Nq) // bk
        for j in range(top, -1, -1):
            cols = range(j * bk, min(Nk, (j + 1) * bk))
            demand = False
            T = -math.inf
            for r in rows:
                legal = [c for c in cols if np.isfinite(S[r, c])]
                if not legal:
                    continue
                if Z[r] == 0.0:
                    demand = True
                    T = math.inf
                    continue
                ratio = math.exp(max(S[r, c] for c in legal)) / Z[r]
                if ratio >= tau / L[r]:
                    demand = True
                T = max(T, L[r] * ratio)
            keep[i, j] = int(demand)
            Tval[i, j] = T
            if demand:
                for r in rows:
                    for c in cols:
                        if np.isfinite(S[r, c]):
                            Z[r] += math.exp(S[r, c])
                            R[r, c] = True
    return keep, R, Tval


def direct_sum_backward(S, lse, tau, bq, bk):
    """The offline rule with probabilities: tile (j, i) retained iff some valid entry
    has exp(s - lse) >= tau / L.  Also returns each tile's decisive value
    T = max over its valid entries of L * exp(s - lse) (NaN without a valid entry)."""
    Nq, Nk = S.shape
    Tr, Tc = -(-Nq // bq), -(-Nk // bk)
    keep = np.full((Tr, Tc), -1, dtype=np.int8)
    Tval = np.full((Tr, Tc), np.nan)
    L = np.arange(Nq) + 1 + (Nk - Nq)
    for i in range(Tr):
        for j in range(Tc):
            rs = slice(i * bq, min(Nq, (i + 1) * bq))
            cs = slice(j * bk, min(Nk, (j + 1) * bk))
            blk = S[rs, cs]
            if not np.isfinite(blk).any():
                continue
            P = np.exp(blk - lse[rs, None])
            keep[i, j] = int((P >= tau / L[rs, None]).any())
            Tval[i, j] = float((L[rs, None] * P).max())
    return keep, Tval


def row_tie_distances(Tval, Nq, bq, tau):
    """Per query row: the smallest |T - tau| and |T / tau - 1| over the finite decisive
    values of the tiles of its query block (+inf if there is none)."""
    ta = np.full(Nq, np.inf)
    tr = np.full(Nq, np.inf)
    for i in range(Tval.shape[0]):
        t = Tval[i][np.isfinite(Tval[i])]
        if t.size:
            rows = slice(i * bq, min(Nq, (i + 1) * bq))
            ta[rows] = np.abs(t - tau).min()
            tr[rows] = np.abs(t / tau - 1).min()
    return ta, tr


def rand_inputs(rng, B, Hq, Hkv, Nq, Nk, D, spread=1.0):
    q = rng.standard_normal((B, Hq, Nq, D)) * spread
    k = rng.standard_normal((B, Hkv, Nk, D)) * spread
    v = rng.standard_normal((B, Hkv, Nk, D))
    do = rng.standard_normal((B, Hq, Nq, D))
    return q, k, v, do


def needle_inputs(rng, N, D, beta, local=0.0, Hq=1, Hkv=1):
    k = rng.standard_normal((1, Hkv, N, D))
    v = rng.standard_normal((1, Hkv, N, D))
    q = rng.standard_normal((1, Hq, N, D))
    g = Hq // Hkv
    for h in range(Hq):
        r = rng.integers(0, np.arange(1, N + 1))
        q[0, h] += beta * k[0, h // g][r]
        if local:
            q[0, h, 1:] += local * k[0, h // g][:-1]
    do = rng.standard_normal((1, Hq, N, D))
    return q, k, v, do


# --------------------------------------------------------------------------
# dense attention: the definition
# --------------------------------------------------------------------------
@pytest.mark.parametrize("Nq,Nk,D", [(1, 1, 4), (7, 7, 4), (33, 33, 8), (64, 64, 64), (5, 19, 8)])
def test_dense_forward_equals_bruteforce_softmax(Nq, Nk, D):
    rng = np.random.default_rng(Nq * 100 + D)
    q, k, v, _ = rand_inputs(rng, 1, 2, 1, Nq, Nk, D, spread=1.5)
    scale = 1 / math.sqrt(D)
    o, lse = oracle.dense_fwd(q, k, v, scale)
    for h in range(2):
        P, l = softmax_rows(scores(q[0, h], k[0, 0], scale))
        np.testing.assert_allclose(o[0, h], P @ v[0, 0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[0, h], l, rtol=0, atol=1e-12)


def _f_dense(q, k, v, do, scale):
    o, _ = oracle.dense_fwd(q, k, v, scale)
    return float((o * do).sum())


@pytest.mark.parametrize("Nq,Nk", [(5, 5), (3, 6)])
def test_dense_gradients_equal_finite_differences(Nq, Nk):
    rng = np.random.default_rng(7 + Nq)
    q, k, v, do = rand_inputs(rng, 1, 2, 1, Nq, Nk, 3)
    scale = 0.7
    dq, dk, dv = oracle.dense_bwd(q, k, v, do, scale)
    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        it = np.nditer(x, flags=["multi_index"])
        for _ in it:
            idx = it.multi_index
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args = {"q": q, "k": k, "v": v}
            fp = _f_dense(*(xp if n == name else args[n] for n in "qkv"), do, scale)
            fm = _f_dense(*(xm if n == name else args[n] for n in "qkv"), do, scale)
            num[idx] = (fp - fm) / (2 * h)
        np.testing.assert_allclose(g, num, rtol=1e-6, atol=1e-7, err_msg=name)


# --------------------------------------------------------------------------
# MALA forward / backward
# --------------------------------------------------------------------------
@pytest.mark.parametrize("N,bq,bk", [(100, 32, 32), (77, 16, 32), (64, 8, 8), (45, 4, 12)])
def test_tau_zero_reproduces_dense(N, bq, bk):
    rng = np.random.default_rng(N)
    q, k, v, do = needle_inputs(rng, N, 16, 2.0, Hq=2, Hkv=1)
    scale = 0.25
    o, lse = oracle.dense_fwd(q, k, v, scale)
    f = oracle.mala_fwd(q, k, v, scale, 0.0, bq, bk, want_tiles=True)
    np.testing.assert_allclose(f["o"], o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(f["lse"], lse, rtol=0, atol=1e-12)
    assert (f["tile_keep"] != 0).all()
    dq, dk, dv = oracle.dense_bwd(q, k, v, do, scale)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, 0.0, bq, bk)
    for x, y in ((b["dq"], dq), (b["dk"], dk), (b["dv"], dv)):
        np.testing.assert_allclose(x, y, rtol=0, atol=1e-10)


def _decision_inputs(bq, bk, tau):
    rng = np.random.default_rng(int(bq * 31 + bk * 7 + tau * 1000))
    return needle_inputs(rng, 23, 4, 3.0, local=2.5)


@pytest.mark.parametrize("bq,bk", [(1, 1), (2, 4), (4, 2), (3, 5), (4, 8)])
@pytest.mark.parametrize("tau", [1e-3, 0.05, 1.0, 4.0])
def test_forward_and_backward_decisions_match_direct_sums(bq, bk, tau):
    q, k, v, do = _decision_inputs(bq, bk, tau)
    N, scale = q.shape[2], 1.0
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk, want_tiles=True)
    S = scores(q[0, 0], k[0, 0], scale)
    keep, R, _ = direct_sum_forward(S, tau, bq, bk)
    np.testing.assert_array_equal(f["tile_keep"][0, 0], keep)
    P, lse = softmax_rows(S, R)
    np.testing.assert_allclose(f["o"][0, 0], P @ v[0, 0], rtol=0, atol=1e-11)
    np.testing.assert_allclose(f["lse"][0, 0], lse, rtol=0, atol=1e-11)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, tau, bq, bk, want_tiles=True)
    np.testing.assert_array_equal(b["tile_keep"][0, 0], direct_sum_backward(S, lse, tau, bq, bk)[0])


def _assert_ties(got_abs, got_rel, exp_abs, exp_rel, what):
    # both sides are fp64; their T values differ by the order of the sums only
    for got, exp, name in ((got_abs, exp_abs, "tie_abs"), (got_rel, exp_rel, "tie_rel")):
        got, exp = np.asarray(got, dtype=np.float64), np.asarray(exp, dtype=np.float64)
        assert (np.isinf(got) == np.isinf(exp)).all(), (what, name, got, exp)
        fin = np.isfinite(exp)
        np.testing.assert_allclose(got[fin], exp[fin], rtol=1e-9, atol=1e-13,
                                   err_msg="%s %s" % (what, name))


@pytest.mark.parametrize("bq,bk", [(1, 1), (2, 4), (4, 2), (3, 5), (4, 8)])
@pytest.mark.parametrize("tau", [1e-3, 0.05, 1.0, 4.0])
def test_tie_distances_match_direct_sums(bq, bk, tau):
    # the oracle's per-row tie distance (min |T - tau| and |T/tau - 1| over the tiles
    # of the row's query block) decides which rows the GPU parity tests exempt from
    # count parity; here T comes from the direct sums instead of the m / l recurrence
    q, k, v, do = _decision_inputs(bq, bk, tau)
    scale = 1.0
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk)
    S = scores(q[0, 0], k[0, 0], scale)
    N = S.shape[0]
    _, R, Tf = direct_sum_forward(S, tau, bq, bk)
    _assert_ties(f["tie_abs"][0, 0], f["tie_rel"][0, 0], *row_tie_distances(Tf, N, bq, tau),
                 "forward")
    _, lse = softmax_rows(S, R)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, tau, bq, bk)
    _, Tb = direct_sum_backward(S, lse, tau, bq, bk)
    _assert_ties(b["tie_abs"][0, 0], b["tie_rel"][0, 0], *row_tie_distances(Tb, N, bq, tau),
                 "backward")


def test_tie_distances_on_gqa_prefill_and_ragged_blocks():
    # several heads of a group, fewer query rows than keys and a partial last block:
    # the tie distances still follow the direct sums row by row
    rng = np.random.default_rng(17)
    q, k, v, do = needle_inputs(rng, 41, 6, 3.0, local=2.0, Hq=4, Hkv=2)
    q, do = q[:, :, -29:].copy(), do[:, :, -29:].copy()
    tau, scale, bq, bk = 0.02, 0.8, 4, 6
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, tau, bq, bk)
    for h in range(4):
        S = scores(q[0, h], k[0, h // 2], scale)
        _, R, Tf = direct_sum_forward(S, tau, bq, bk)
        _assert_ties(f["tie_abs"][0, h], f["tie_rel"][0, h], *row_tie_distances(Tf, 29, bq, tau),
                     "forward head %d" % h)
        _, lse = softmax_rows(S, R)
        _, Tb = direct_sum_backward(S, lse, tau, bq, bk)
        _assert_ties(b["tie_abs"][0, h], b["tie_rel"][0, h], *row_tie_distances(Tb, 29, bq, tau),
                     "backward head %d" % h)


def test_some_decision_cases_actually_skip():
    # guards the direct-sum comparison above against being vacuous
    for tau in (0.05, 1.0, 4.0):
        skipped = 0
        for bq, bk in ((1, 1), (2, 4), (4, 2), (3, 5), (4, 8)):
            q, k, v, do = _decision_inputs(bq, bk, tau)
            f = oracle.mala_fwd(q, k, v, 1.0, tau, bq, bk, want_tiles=True)
            skipped += int((f["tile_keep"] == 0).sum())
        assert skipped >= 5, tau


@pytest.mark.parametrize("tau", [1e-4, 1e-3, 1e-2, 0.1, 1.0, 3.0])
@pytest.mark.parametrize("bq,bk", [(1, 1), (8, 8), (16, 32)])
def test_proposition1_omitted_mass_and_output_bound(tau, bq, bk):
    rng = np.random.default_rng(11)
    N, D = 200, 16
    q, k, v, _ = needle_inputs(rng, N, D, 3.0, local=2.0, Hq=2, Hkv=1)
    scale = 0.5
    o, lse = oracle.dense_fwd(q, k, v, scale)
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk)
    eps = -np.expm1(f["lse"] - lse)           # omitted dense mass per row
    assert (eps >= -1e-13).all()
    assert (eps <= tau / (1 + tau) + 1e-12).all()
    vmax = np.linalg.norm(v[0, 0], axis=1).max()
    err = np.linalg.norm(f["o"] - o, axis=-1)
    assert (err <= 2 * tau / (1 + tau) * vmax + 1e-10).all()
    if tau >= 1e-2:
        assert eps.max() > 0                   # the rule did omit something


@pytest.mark.parametrize("tau", [1e-3, 0.1, 1.0])
def test_backward_support_nested_in_forward_support(tau):
    rng = np.random.default_rng(5)
    q, k, v, do = needle_inputs(rng, 150, 16, 3.0, local=2.0, Hq=2, Hkv=1)
    f = oracle.mala_fwd(q, k, v, 0.5, tau, 8, 8, want_tiles=True)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, 0.5, tau, 8, 8, want_tiles=True)
    fk, bk_ = f["tile_keep"], b["tile_keep"]
    assert ((fk == -1) == (bk_ == -1)).all()          # same legal tiles
    assert not ((fk == 0) & (bk_ == 1)).any()          # skipped forward => skipped backward
    if tau >= 0.1:
        assert ((fk == 1) & (bk_ == 0)).any()          # backward can be more selective


def test_first_legal_tile_retained_and_rows_nonempty():
    rng = np.random.default_rng(9)
    N = 130
    q, k, v, _ = needle_inputs(rng, N, 8, 4.0, local=3.0)
    for bq, bk in ((8, 8), (8, 16), (5, 7)):
        f = oracle.mala_fwd(q, k, v, 1.0, 5.0, bq, bk, want_tiles=True)
        keep = f["tile_keep"][0, 0]
        for i in range(keep.shape[0]):
            top = (min(N, (i + 1) * bq) - 1) // bk
            assert keep[i, top] == 1
            assert (keep[i, top + 1:] == -1).all()
        assert (f["row_tiles"] >= 1).all()


def test_gqa_equals_mha_on_repeated_kv():
    rng = np.random.default_rng(3)
    q, k, v, do = needle_inputs(rng, 70, 8, 2.0, Hq=4, Hkv=2)
    kr, vr = np.repeat(k, 2, axis=1), np.repeat(v, 2, axis=1)
    for tau in (0.0, 0.02):
        fg = oracle.mala_fwd(q, k, v, 0.5, tau, 8, 16)
        fm = oracle.mala_fwd(q, kr, vr, 0.5, tau, 8, 16)
        np.testing.assert_array_equal(fg["o"], fm["o"])
        np.testing.assert_array_equal(fg["row_tiles"], fm["row_tiles"])
        bg = oracle.mala_bwd(q, k, v, fg["o"], fg["lse"], do, 0.5, tau, 8, 16)
        bm = oracle.mala_bwd(q, kr, vr, fm["o"], fm["lse"], do, 0.5, tau, 8, 16)
        np.testing.assert_array_equal(bg["dq"], bm["dq"])
        np.testing.assert_allclose(bg["dk"], bm["dk"].reshape(1, 2, 2, 70, 8).sum(2), atol=1e-12)
        np.testing.assert_allclose(bg["dv"], bm["dv"].reshape(1, 2, 2, 70, 8).sum(2), atol=1e-12)


def _f_restricted(q, k, v, do, scale, R):
    S = scores(q, k, scale)
    P, _ = softmax_rows(S, R)
    return float(((P @ v) * do).sum())


def test_tau_positive_gradients_equal_finite_differences_on_frozen_support():
    """When the backward keeps exactly the forward's tiles, Algorithm 2 is the exact
    gradient of softmax attention restricted to the (frozen) retained set."""
    found = False
    for seed in range(200):
        rng = np.random.default_rng(1000 + seed)
        N, D = 9, 3
        k = rng.standard_normal((1, 1, N, D))
        v = rng.standard_normal((1, 1, N, D))
        q = 2.5 * k + 0.3 * rng.standard_normal((1, 1, N, D))   # strong self-attention
        do = rng.standard_normal((1, 1, N, D))
        tau, scale = 0.05, 1.0
        f = oracle.mala_fwd(q, k, v, scale, tau, 1, 1, want_tiles=True)
        b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, tau, 1, 1, want_tiles=True)
        fk, bk_ = f["tile_keep"][0, 0], b["tile_keep"][0, 0]
        if (fk == 0).sum() >= 3 and ((fk == 1) == (bk_ == 1)).all():
            found = True
            break
    assert found, "no input with a skipping forward and an identical backward support"
    R = fk == 1
    h = 1e-6
    for name, x, g in (("q", q, b["dq"]), ("k", k, b["dk"]), ("v", v, b["dv"])):
        num = np.zeros(x.shape[2:])
        for idx in np.ndindex(*x.shape[2:]):
            xs = {"q": q[0, 0], "k": k[0, 0], "v": v[0, 0]}
            xp, xm = xs[name].copy(), xs[name].copy()
            xp[idx] += h
            xm[idx] -= h
            fp = _f_restricted(**{**xs, name: xp}, do=do[0, 0], scale=scale, R=R)
            fm = _f_restricted(**{**xs, name: xm}, do=do[0, 0], scale=scale, R=R)
            num[idx] = (fp - fm) / (2 * h)
        np.testing.assert_allclose(g[0, 0], num, rtol=1e-6, atol=1e-7, err_msg=name)


# --------------------------------------------------------------------------
# closed-form cases (tests/golden/closed_form_cases.json)
# --------------------------------------------------------------------------
def _golden():
    with open(os.path.join(GOLDEN, "closed_form_cases.json")) as fh:
        return json.load(fh)


@pytest.mark.parametrize("case", _golden()["two_token"], ids=lambda c: c["name"])
def test_two_token_closed_form(case):
    # one-dimensional head, scale 1: s_{1,1} = a, s_{1,0} = a - delta, B_q = B_k = 1
    a, delta, tau = case["a"], case["delta"], case["tau"]
    q = np.array([[[[1.0], [1.0]]]])
    k = np.array([[[[a - delta], [a]]]])
    v = np.array([[[[3.0], [-2.0]]]])
    do = np.array([[[[0.5], [1.5]]]])
    f = oracle.mala_fwd(q, k, v, 1.0, tau, 1, 1, want_tiles=True)
    keep = f["tile_keep"][0, 0]
    assert keep[1, 1] == 1 and keep[0, 0] == 1
    assert keep[1, 0] == case["row1_keeps_key0"]
    # decisive values (golden "tie_rules"): forward T(1,0) = 2 exp(-delta); row 0 only
    # has its diagonal tile, tested in the empty state
    e = math.exp(-delta)
    _assert_ties(f["tie_abs"][0, 0], f["tie_rel"][0, 0], [math.inf, abs(2 * e - tau)],
                 [math.inf, abs(2 * e / tau - 1)], "forward")
    kept = case["row1_keeps_key0"]
    t10, t11 = (2 * e / (1 + e), 2 / (1 + e)) if kept else (2 * e, 2.0)
    bt = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, 1.0, tau, 1, 1)
    _assert_ties(bt["tie_abs"][0, 0], bt["tie_rel"][0, 0],
                 [abs(1 - tau), min(abs(t10 - tau), abs(t11 - tau))],
                 [abs(1 / tau - 1), min(abs(t10 / tau - 1), abs(t11 / tau - 1))], "backward")
    if not case["row1_keeps_key0"]:
        assert f["o"][0, 0, 1, 0] == -2.0 and abs(f["lse"][0, 0, 1] - a) < 1e-15
        o, lse = oracle.dense_fwd(q, k, v, 1.0)
        eps = -math.expm1(f["lse"][0, 0, 1] - lse[0, 0, 1])
        assert abs(eps - math.exp(-delta) / (1 + math.exp(-delta))) < 1e-15
        assert eps <= tau / (1 + tau)
        b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, 1.0, tau, 1, 1, want_tiles=True)
        assert b["tile_keep"][0, 0, 1, 0] == 0
        # each row now attends to exactly one key: dV = dO, dS = 0, dQ = dK = 0
        np.testing.assert_array_equal(b["dv"][0, 0, :, 0], [0.5, 1.5])
        np.testing.assert_array_equal(b["dq"], 0.0)
        np.testing.assert_array_equal(b["dk"], 0.0)


@pytest.mark.parametrize("case", _golden()["uniform"], ids=lambda c: c["name"])
def test_uniform_scores_closed_form(case):
    # q = 0 makes every score exactly 0; with one-key tiles the forward retains the
    # first n keys while n <= L / tau, i.e. min(L, floor(L / tau) + 1) keys, and the
    # backward keeps a key iff 1/n_R >= tau / L
    N, tau = case["N"], case["tau"]
    rng = np.random.default_rng(0)
    q = np.zeros((1, 1, N, 2))
    k = rng.standard_normal((1, 1, N, 2))
    v = rng.standard_normal((1, 1, N, 2))
    do = rng.standard_normal((1, 1, N, 2))
    f = oracle.mala_fwd(q, k, v, 1.0, tau, 1, 1, want_tiles=True)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, 1.0, tau, 1, 1, want_tiles=True)
    for r in range(N):
        L = r + 1
        n = min(L, math.floor(L / tau) + 1)
        assert f["row_tiles"][0, 0, r] == n == case["forward_kept"][r]
        np.testing.assert_array_equal(f["tile_keep"][0, 0, r, : r + 1],
                                      [0] * (L - n) + [1] * n)
        assert abs(f["lse"][0, 0, r] - math.log(n)) < 1e-14
        np.testing.assert_allclose(f["o"][0, 0, r], v[0, 0, L - n: L].mean(axis=0), atol=1e-14)
        assert b["row_tiles"][0, 0, r] == case["backward_kept"][r]
        # decisive values (golden "tie_rules"): forward T in {L / n : n = 1 ..
        # min(n_f, L - 1)}, backward T = L / n_f on every tile of the row
        Ts = [L / m for m in range(1, min(n, L - 1) + 1)]
        fa = min((abs(t - tau) for t in Ts), default=math.inf)
        fr = min((abs(t / tau - 1) for t in Ts), default=math.inf)
        _assert_ties([f["tie_abs"][0, 0, r]], [f["tie_rel"][0, 0, r]], [fa], [fr], "fwd row %d" % r)
        _assert_ties([b["tie_abs"][0, 0, r]], [b["tie_rel"][0, 0, r]], [abs(L / n - tau)],
                     [abs(L / n / tau - 1)], "bwd row %d" % r)
    if tau == 1.0:
        # every backward T equals tau: each row lies in the tie band
        assert (b["tie_abs"] <= 1e-12).all()


# --------------------------------------------------------------------------
# decode
# --------------------------------------------------------------------------
def test_decode_single_split_equals_forward_last_row():
    rng = np.random.default_rng(21)
    Nk, D = 300, 16
    q, k, v, _ = needle_inputs(rng, Nk, D, 3.0, Hq=2, Hkv=1)
    for tau in (0.0, 1e-3, 0.1, 1.0):
        f = oracle.mala_fwd(q, k, v, 0.5, tau, 1, 32)
        d = oracle.mala_decode(q[:, :, -1], k, v, 0.5, tau, 32, 1)
        np.testing.assert_allclose(d["o"], f["o"][:, :, -1], rtol=0, atol=1e-13)
        np.testing.assert_allclose(d["lse"], f["lse"][:, :, -1], rtol=0, atol=1e-13)
        np.testing.assert_array_equal(d["tiles"], f["row_tiles"][:, :, -1])


@pytest.mark.parametrize("splits", [1, 3, 7, 16])
@pytest.mark.parametrize("tau", [0.0, 1e-3, 0.3, 2.0])
def test_decode_split_rule_and_merge(splits, tau):
    rng = np.random.default_rng(splits * 10 + int(tau * 100))
    Nk, D, bk = 203, 8, 16
    k = rng.standard_normal((1, 1, Nk, D))
    v = rng.standard_normal((1, 1, Nk, D))
    q = rng.standard_normal((1, 1, D)) + 2.0 * k[0, :, rng.choice(Nk, 4, replace=False)].sum(0)
    d = oracle.mala_decode(q, k, v, 0.7, tau, bk, splits, want_tiles=True)
    s = 0.7 * (k[0, 0] @ q[0, 0])
    T = -(-Nk // bk)
    tps = -(-T // splits)
    keep = np.zeros(T, dtype=np.int8)
    Tvals = []                                        # decisive values of non-empty tests
    for sp in range(splits):                          # direct sums, per split
        Z = 0.0
        for t in range(min(T, (sp + 1) * tps) - 1, sp * tps - 1, -1):
            blk = s[t * bk: (t + 1) * bk]
            if Z > 0.0:
                Tvals.append(Nk * math.exp(blk.max()) / Z)
            if Z == 0.0 or math.exp(blk.max()) / Z >= tau / Nk:
                keep[t] = 1
                Z += np.exp(blk).sum()
    np.testing.assert_array_equal(d["keep"][0, 0], keep)
    if tau > 0:
        _assert_ties(d["tie_abs"][0], d["tie_rel"][0],
                     [min((abs(t - tau) for t in Tvals), default=math.inf)],
                     [min((abs(t / tau - 1) for t in Tvals), default=math.inf)], "decode")
    Rk = np.repeat(keep.astype(bool), bk)[:Nk]
    p = np.exp(s[Rk] - s[Rk].max())
    np.testing.assert_allclose(d["o"][0, 0], (p / p.sum()) @ v[0, 0][Rk], rtol=0, atol=1e-12)
    lse_full = s.max() + math.log(np.exp(s - s.max()).sum())
    eps = -math.expm1(d["lse"][0, 0] - lse_full)
    assert eps <= tau / (1 + tau) + 1e-12


# --------------------------------------------------------------------------
# the input generators
# --------------------------------------------------------------------------
def test_bf16_rounding_is_round_to_nearest_even():
    import torch
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.float32([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -1e-30])])
    ours = bf16_round(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(bf16_to_f64(ours), torch.from_numpy(ref.view(np.int16)).view(
        torch.bfloat16).to(torch.float64).numpy())


def test_workload_generator_shapes_and_needles():
    w = Workload("needle_1k_d64")
    t = w.tensors()
    assert t["q"].shape == (1, 1, 1024, 64) and t["do"].shape == (1, 1, 1024, 64)
    np.testing.assert_array_equal(Workload("needle_1k_d64").tensors()["q"], t["q"])   # seeded
    w5 = Workload("decode_gqa32x8_128k", N=512, B=2)
    q = bf16_to_f64(w5.q_head(1, 5))
    k = bf16_to_f64(w5.k_head(1, 5 // 4))
    pos = w5.needle_positions(1, 5)
    s = k @ q
    assert set(np.argsort(s)[-4:]) == set(pos)       # the planted needles dominate

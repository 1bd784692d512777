"""Property tests of the fp64 oracle over random shapes, tile sizes, tolerances and
needle strengths (hypothesis), for the invariants the paper states or the
mathematics fixes:
  * tau = 0 reproduces dense attention, forward and backward (the tau -> 0 limit);
  * the omitted dense mass of every row is at most tau / (1 + tau) (Appendix,
    omitted-mass proposition), and the output moves by at most 2 tau / (1 + tau)
    times the largest value norm;
  * the backward's retained tiles are a subset of the forward's (nested support);
  * every row's first legal tile is retained and no row is empty;
  * Nq < Nk (prefill) equals the last Nq rows of the full causal problem.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle

SETTINGS = dict(max_examples=120, deadline=None, derandomize=True,
                suppress_health_check=[HealthCheck.too_slow])


@st.composite
def problems(draw):
    N = draw(st.integers(1, 72))
    D = draw(st.sampled_from([4, 8, 16]))
    g = draw(st.sampled_from([1, 2]))
    bq = draw(st.integers(1, 12))
    bk = draw(st.integers(1, 12))
    beta = draw(st.floats(0.0, 4.0))
    local = draw(st.floats(0.0, 4.0))
    tau = draw(st.sampled_from([1e-4, 1e-2, 0.3, 1.0, 3.0]))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((1, 1, N, D))
    v = rng.standard_normal((1, 1, N, D))
    q = rng.standard_normal((1, g, N, D))
    for h in range(g):
        r = rng.integers(0, np.arange(1, N + 1))
        q[0, h] += beta * k[0, 0][r]
        if local and N > 1:
            q[0, h, 1:] += local * k[0, 0][:-1]
    do = rng.standard_normal((1, g, N, D))
    return q, k, v, do, 1.0 / np.sqrt(D), tau, bq, bk


@settings(**SETTINGS)
@given(problems())
def test_tau_zero_is_dense(prob):
    q, k, v, do, scale, _, bq, bk = prob
    o, lse = oracle.dense_fwd(q, k, v, scale)
    f = oracle.mala_fwd(q, k, v, scale, 0.0, bq, bk)
    np.testing.assert_allclose(f["o"], o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(f["lse"], lse, rtol=0, atol=1e-12)
    dq, dk, dv = oracle.dense_bwd(q, k, v, do, scale)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, 0.0, bq, bk)
    for got, ref in ((b["dq"], dq), (b["dk"], dk), (b["dv"], dv)):
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10)


@settings(**SETTINGS)
@given(problems())
def test_omitted_mass_and_output_bounds(prob):
    q, k, v, _, scale, tau, bq, bk = prob
    o, lse = oracle.dense_fwd(q, k, v, scale)
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk)
    eps = -np.expm1(f["lse"] - lse)
    assert (eps >= -1e-12).all()
    assert (eps <= tau / (1 + tau) + 1e-12).all()
    vmax = np.linalg.norm(v[0, 0], axis=1).max()
    assert (np.linalg.norm(f["o"] - o, axis=-1) <= 2 * tau / (1 + tau) * vmax + 1e-10).all()


@settings(**SETTINGS)
@given(problems())
def test_nested_support_and_nonempty_rows(prob):
    q, k, v, do, scale, tau, bq, bk = prob
    f = oracle.mala_fwd(q, k, v, scale, tau, bq, bk, want_tiles=True)
    b = oracle.mala_bwd(q, k, v, f["o"], f["lse"], do, scale, tau, bq, bk, want_tiles=True)
    fk, bkp = f["tile_keep"], b["tile_keep"]
    assert ((fk == -1) == (bkp == -1)).all()
    assert not ((fk == 0) & (bkp == 1)).any()
    assert (f["row_tiles"] >= 1).all()
    N = q.shape[2]
    for h in range(q.shape[1]):
        for i in range(fk.shape[2]):
            top = (min(N, (i + 1) * bq) - 1) // bk
            assert fk[0, h, i, top] == 1


@settings(**SETTINGS)
@given(problems(), st.integers(1, 72))
def test_prefill_is_the_tail_of_the_full_problem_at_tau_zero(prob, nq):
    q, k, v, _, scale, _, bq, bk = prob
    N = q.shape[2]
    nq = min(nq, N)
    full = oracle.dense_fwd(q, k, v, scale)
    f = oracle.mala_fwd(np.ascontiguousarray(q[:, :, N - nq:]), k, v, scale, 0.0, bq, bk)
    np.testing.assert_allclose(f["o"], full[0][:, :, N - nq:], rtol=0, atol=1e-12)
    np.testing.assert_allclose(f["lse"], full[1][:, :, N - nq:], rtol=0, atol=1e-12)

"""The seeded input generators (host logic, CPU): the options that give the
language-model-like supplementary workload its structure."""
import numpy as np

from workloads import WORKLOADS, Workload, bf16_round, bf16_to_f64


def _small(**over):
    spec = dict(WORKLOADS["lm_like_gqa8x2_32k"])
    spec.update(dict(N=300, Hq=2, Hkv=1, D=64), **over)
    return Workload(spec, seed=3)


def test_block_needles_are_shared_and_visible():
    w = _small()
    r = w.needle_rows(0, 1)
    nb = w.spec["needle_block"]
    for c0 in range(0, w.N, nb):
        blk = r[c0:c0 + nb]
        assert (blk == blk[0]).all()          # one needle per block of rows
        assert 0 <= blk[0] <= c0              # visible to the block's first row


def test_unblocked_needles_lie_in_each_rows_causal_range():
    w = _small(needle_block=1)
    r = w.needle_rows(0, 0)
    assert (r >= 0).all() and (r <= np.arange(w.N)).all()
    assert len(np.unique(r)) > w.N // 4       # drawn per row


def test_sink_adds_the_first_key_to_every_query():
    with_sink, without = _small(), _small(sink=0.0)
    q1 = bf16_to_f64(with_sink.q_head(0, 0))
    q0 = bf16_to_f64(without.q_head(0, 0))
    k0 = bf16_to_f64(with_sink.k_head(0, 0))[0]
    diff = q1 - q0 - with_sink.spec["sink"] * k0
    # both sides were rounded to bf16 once: at most one half-ulp each
    bound = 2.0 ** -8 * (np.abs(q1) + np.abs(q0)) + 1e-12
    assert (np.abs(diff) <= bound).all()


def test_rademacher_probe():
    d = bf16_to_f64(_small().do_head(0, 1))
    assert set(np.unique(d)) == {-1.0, 1.0}
    assert abs(d.mean()) < 0.05


def test_existing_configurations_unchanged_by_the_new_options():
    # the default paths draw exactly as before: no block needles, no sink, normal dO
    w = Workload(dict(WORKLOADS["mha16_8k"], N=64, Hq=1, Hkv=1))
    g = w.do_head(0, 0)
    assert bf16_to_f64(g).std() > 0.5 and len(np.unique(g)) > 100
    r = w.needle_rows(0, 0)
    assert len(np.unique(r)) > 16

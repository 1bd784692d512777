"""The load-count helpers of the GPU parity tests against direct loops on small
random decision arrays (no GPU)."""
import numpy as np
import pytest

from parity_util import bwd_do_loads, fwd_v_loads


def _fwd_direct(keep, rows, bq):
    B, H, Tr, Tc = keep.shape
    g = rows // bq
    n = 0
    for b in range(B):
        for h in range(H):
            for w0 in range(0, Tr, g):
                for j in range(Tc):
                    n += any(keep[b, h, i, j] == 1 for i in range(w0, min(w0 + g, Tr)))
    return n


def _bwd_direct(keep, keys, bk):
    B, H, Tr, Tc = keep.shape
    g = keys // bk
    n = 0
    for b in range(B):
        for h in range(H):
            for i in range(Tr):
                for k0 in range(0, Tc, g):
                    n += any(keep[b, h, i, j] == 1 for j in range(k0, min(k0 + g, Tc)))
    return n


@pytest.mark.parametrize("seed", range(4))
def test_load_counts_match_direct_loops(seed):
    rng = np.random.default_rng(seed)
    B, H, Tr, Tc = 2, 3, int(rng.integers(1, 20)), int(rng.integers(1, 20))
    # 1 retained, 0 skipped, -1 not legal (the oracle's encoding)
    keep = rng.choice([-1, 0, 1], size=(B, H, Tr, Tc), p=[0.3, 0.5, 0.2])
    assert fwd_v_loads(keep) == _fwd_direct(keep, 256, 32)
    assert fwd_v_loads(keep, 64, 32) == _fwd_direct(keep, 64, 32)
    assert bwd_do_loads(keep) == _bwd_direct(keep, 128, 32)
    assert bwd_do_loads(keep, 64, 32) == _bwd_direct(keep, 64, 32)


def test_load_counts_extremes():
    keep = np.ones((1, 1, 9, 7), int)
    assert fwd_v_loads(keep) == 2 * 7          # two workgroups of 8 query tiles
    assert bwd_do_loads(keep) == 9 * 2         # two key blocks of 4 tiles
    assert fwd_v_loads(np.zeros_like(keep)) == 0 == bwd_do_loads(-np.ones_like(keep))

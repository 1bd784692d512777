"""The test side's retained-set fingerprint (the statistic the library reports as
MALA_CNT_SET_HASH / MALA_CNT_SET_HASH_KV), pinned on the CPU: its mixing function
is SplitMix64's output function (Steele, Lea and Flood, 2014), checked against the
generator's published outputs, and the sum over a set does not depend on order."""
import numpy as np

from parity_util import _splitmix64, set_fingerprint

GAMMA = 0x9E3779B97F4A7C15


def test_splitmix64_published_outputs():
    # SplitMix64 from seed s returns mix(s + k * gamma) for k = 1, 2, ...; mix here
    # takes the state before its increment
    seq = lambda s, n: [int(_splitmix64(np.array([(s + k * GAMMA) % (1 << 64)],
                                                 dtype=np.uint64))[0]) for k in range(n)]
    assert seq(0, 1) == [0xE220A8397B1DCDAF]
    assert seq(1234567, 5) == [6457827717110365317, 3203168211198807973, 9817491932198370423,
                               4593380528125082431, 16408922859458223821]


def test_fingerprint_is_a_set_function():
    rng = np.random.default_rng(0)
    keep = (rng.random((2, 3, 5, 7)) < 0.4).astype(np.int8)
    keep[0, 0, 0, 0] = -1                          # not legal: not part of the set
    f = set_fingerprint(keep)
    # the packed key of one tile, by hand: b = 1, h = 2, i = 3, j = 4
    one = np.zeros_like(keep)
    one[1, 2, 3, 4] = 1
    key = (1 << 52) | (2 << 40) | (3 << 20) | 4
    v = int(_splitmix64(np.array([key], dtype=np.uint64))[0])
    assert set_fingerprint(one) == (v - (1 << 64) if v >= 1 << 63 else v)
    # flipping one tile changes it; the sum is over the set only
    flipped = keep.copy()
    flipped[1, 2, 3, 4] = 1 - max(0, flipped[1, 2, 3, 4])
    assert set_fingerprint(flipped) != f
    assert set_fingerprint(np.zeros_like(keep)) == 0
    # a decode array [B, H, T] is the tile row i = 0; b0 offsets the sequence index
    d = (rng.random((1, 4, 9)) < 0.5).astype(np.int8)
    assert set_fingerprint(d) == set_fingerprint(d[:, :, None, :])
    both = np.concatenate([np.zeros_like(d), d])
    assert set_fingerprint(d, b0=1) == set_fingerprint(both)

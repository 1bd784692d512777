"""mala_decode_noalloc (the decode entry point that allocates nothing, for callers
that cannot allocate device memory) against mala_decode with a caller workspace:
the same kernels, so the outputs and statistics must be equal bit for bit, on two
calls in a row that share the library's buffer, the second smaller than the first."""
import numpy as np
import pytest
import torch

import paper_2609_32712_amd as mala
from parity_util import dev
from workloads import Workload

pytestmark = pytest.mark.gpu


def _inputs(spec):
    w = Workload(spec)
    t = w.tensors()
    return w, dev(t["q"]), dev(t["k"]), dev(t["v"])


def _outputs(w):
    f = dict(device="cuda")
    return (torch.full((w.B, w.Hq, w.D), -7.0, **f), torch.full((w.B, w.Hq), -7.0, **f),
            torch.full((w.B, w.Hq), -7, dtype=torch.int32, **f),
            torch.full((mala.NUM_COUNTERS,), -7, dtype=torch.int64, **f))


CALLS = [
    # a large call first (split partials ~4.3 MB of the 16 MiB buffer), then a smaller one
    # with ragged cache lengths that reuses the buffer's leading bytes
    (dict(kind="decode", B=16, Hq=32, Hkv=8, N=8192, D=128, beta=3.0, needles=4), 16, 1e-4, None),
    (dict(kind="decode", B=3, Hq=8, Hkv=2, N=3001, D=64, beta=3.0, needles=4), 5, 1e-2,
     [3001, 17, 1500]),
]


def test_noalloc_decode_equals_workspace_decode_on_consecutive_calls():
    for spec, splits, tau, lens in CALLS:
        w, q, k, v = _inputs(spec)
        cl = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
        scale = float(np.float32(w.scale))
        ref = _outputs(w)
        ws = torch.empty(mala.mala_decode_workspace_size(w.B, w.Hq, w.D, splits),
                         dtype=torch.uint8, device="cuda")
        mala.mala_decode(q, k, v, *ref[:2], ref[2], ref[3], splits, ws, scale, tau,
                         cache_lens=cl)
        got = _outputs(w)
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        mala.mala_decode_noalloc(q, k, v, got[0], got[1], got[2], got[3], splits, scale, tau,
                                 cache_lens=cl)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        for name, a, b in zip(("o", "lse", "head_tiles", "counters"), got, ref):
            assert torch.equal(a, b), (spec, name)
        assert torch.isfinite(got[0]).all()


def test_noalloc_decode_rejects_a_call_beyond_its_buffer():
    w, q, k, v = _inputs(dict(kind="decode", B=16, Hq=32, Hkv=8, N=4096, D=128, beta=3.0,
                              needles=4))
    o, lse, ht, cnt = _outputs(w)
    with pytest.raises(mala.MalaError) as e:
        mala.mala_decode_noalloc(q, k, v, o, lse, ht, cnt, 64, 0.088, 1e-4)
    assert e.value.status == mala.MALA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (o == -7.0).all()          # nothing was launched

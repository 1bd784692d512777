"""The C ABI without a GPU: the library loads, exports every function that
include/mala.h declares, reports its geometry and workspace sizes, and rejects
invalid arguments synchronously (before any HIP call)."""
import ctypes
import os
import re

import pytest

import paper_2609_32712_amd as mala
from parity_util import dkdv_splits

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mala.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    decl = r"^\s*(?:const\s+)?[\w]+\*?\s+\**(mala_\w+)\s*\("
    return sorted(set(re.findall(decl, src, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mala.LIB_PATH):
        pytest.fail("libmala.so is not built (run __graft_entry__.build())")
    return mala.load_library()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("mala_fwd", "mala_bwd", "mala_decode", "mala_geometry", "mala_strerror",
              "mala_last_error", "mala_bwd_workspace_size", "mala_decode_workspace_size"):
        assert n in names
    assert set(names) == set(mala.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_geometry(lib):
    for d in (64, 128):
        assert mala.mala_geometry(d, mala.PASS_FWD) == mala.mala_geometry(d, mala.PASS_BWD)
        bq, bk = mala.mala_geometry(d, mala.PASS_FWD)
        assert bq > 0 and bk > 0 and bk % bq == 0
        assert mala.mala_geometry(d, mala.PASS_DECODE)[0] == 1
    assert mala.mala_geometry(96, mala.PASS_FWD) == (0, 0)
    assert mala.mala_geometry(128, 7) == (0, 0)


def test_workspace_sizes(lib):
    # D_q (B Hq Nq floats) and one decision byte per query tile, head and 128-key block
    assert mala.mala_bwd_workspace_size(1, 8, 2, 1000, 1000, 128) >= 4 * 8 * 1000 + 8 * 32 * 8
    assert mala.mala_bwd_workspace_size(1, 8, 2, 131072, 131072, 128) >= 8 * 4096 * 1024
    assert mala.mala_bwd_workspace_size(0, 8, 2, 1000, 1000, 128) == 0
    assert mala.mala_bwd_workspace_size(1, 8, 3, 1000, 1000, 128) == 0
    assert mala.mala_bwd_workspace_size(1, 8, 2, 1000, 1000, 96) == 0
    # few key-block workgroups (2 KV heads x 256 blocks): the sweeps run in 4 parts
    # whose fp32 partial dV / dK the workspace holds; 2048 workgroups: no parts
    assert mala.mala_bwd_workspace_size(1, 8, 2, 32768, 32768, 128) >= 4 * 2 * 2 * 32768 * 128 * 4
    assert mala.mala_bwd_workspace_size(1, 8, 2, 131072, 131072, 128) < (
        8 * 131072 * 4 + 8 * 4096 * 1024 + 2 ** 20)


def test_split_rule_of_the_tests_matches_the_library(lib):
    # the GPU tests' mirror of the launch rule (parity_util.dkdv_splits) against the
    # library: the backward workspace holds partial sums exactly when sweeps split
    ru = lambda x: (x + 255) // 256 * 256
    shapes = [(1, 16, 1, 12000, 12000), (2, 8, 1, 6000, 6000), (1, 16, 1, 5000, 12000),
              (1, 8, 2, 32768, 32768), (1, 8, 2, 16384, 16384), (1, 8, 2, 8192, 8192),
              (1, 8, 2, 4096, 4096), (1, 8, 2, 131072, 131072), (1, 32, 8, 32768, 32768),
              (1, 1, 1, 1024, 1024), (4, 8, 2, 8192, 8192), (1, 4, 1, 3000, 9000)]
    for B, Hq, Hkv, Nq, Nk in shapes:
        base = ru(B * Hq * Nq * 4) + ru(Hq * -(-Nk // 128) * B * -(-Nq // 32))
        split = mala.mala_bwd_workspace_size(B, Hq, Hkv, Nq, Nk, 128) > base
        assert split == dkdv_splits(B, Hq, Hkv, Nq, Nk), (B, Hq, Hkv, Nq, Nk)
    assert mala.mala_decode_workspace_size(16, 32, 128, 8) >= 16 * 32 * 8 * 130 * 4
    assert mala.mala_decode_workspace_size(16, 32, 96, 8) == 0


def _fwd(lib, **kw):
    a = dict(q=16, k=16, v=16, o=16, lse=16, B=1, Hq=2, Hkv=1, Nq=64, Nk=64, D=128, causal=1,
             scale=0.1, tau=1e-3, out=mala.OUT_F32)
    a.update(kw)
    P = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.mala_fwd(P(a["q"]), P(a["k"]), P(a["v"]), P(a["o"]), P(a["lse"]), None, None,
                        a["B"], a["Hq"], a["Hkv"], a["Nq"], a["Nk"], a["D"], a["causal"],
                        a["scale"], a["tau"], a["out"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), mala.MALA_ERR_INVALID_ARG),
    (dict(lse=None), mala.MALA_ERR_INVALID_ARG),
    (dict(B=0), mala.MALA_ERR_INVALID_ARG),
    (dict(Hq=3, Hkv=2), mala.MALA_ERR_INVALID_ARG),
    (dict(Nq=65), mala.MALA_ERR_INVALID_ARG),
    (dict(tau=-1e-3), mala.MALA_ERR_INVALID_ARG),
    (dict(tau=float("nan")), mala.MALA_ERR_INVALID_ARG),
    (dict(tau=float("inf")), mala.MALA_ERR_INVALID_ARG),
    (dict(scale=0.0), mala.MALA_ERR_INVALID_ARG),
    (dict(scale=float("inf")), mala.MALA_ERR_INVALID_ARG),
    (dict(D=96), mala.MALA_ERR_UNSUPPORTED),
    (dict(causal=0), mala.MALA_ERR_UNSUPPORTED),
    (dict(Nq=64, Nk=1 << 24), mala.MALA_ERR_UNSUPPORTED),   # Nk x D x 2 bytes reach 2^32
    (dict(out=2), mala.MALA_ERR_INVALID_ARG),                # no such output type
    (dict(out=-1), mala.MALA_ERR_INVALID_ARG),
])
def test_fwd_rejects_invalid_arguments(lib, kw, status):
    assert _fwd(lib, **kw) == status
    assert lib.mala_last_error().decode() != ""
    assert lib.mala_strerror(status).decode() not in ("", "unknown status")


def test_bwd_and_decode_reject_missing_workspace(lib):
    P = ctypes.c_void_p
    f32, b16 = mala.OUT_F32, mala.OUT_BF16
    st = lib.mala_bwd(*([P(16)] * 9), None, None, None, 0, 1, 2, 1, 64, 64, 128, 1, 0.1, 0.0,
                      f32, f32, None)
    assert st == mala.MALA_ERR_WORKSPACE
    st = lib.mala_bwd(*([P(16)] * 9), None, None, P(16), 8, 1, 2, 1, 64, 64, 128, 1, 0.1, 0.0,
                      b16, b16, None)
    assert st == mala.MALA_ERR_WORKSPACE
    st = lib.mala_bwd(*([P(16)] * 9), None, None, P(16), 1 << 20, 1, 2, 1, 64, 64, 128, 1, 0.1,
                      0.0, f32, 3, None)
    assert st == mala.MALA_ERR_INVALID_ARG
    qkv, ol = [P(16)] * 3, [P(16)] * 2     # q, k_cache, v_cache / o, lse (cache_lens NULL)
    st = lib.mala_decode(*qkv, None, *ol, None, None, 4, None, 0, 1, 2, 1, 64, 128, 0.1, 0.0,
                         f32, None)
    assert st == mala.MALA_ERR_WORKSPACE
    st = lib.mala_decode(*qkv, None, *ol, None, None, 0, P(16), 1 << 20, 1, 2, 1, 64, 128, 0.1,
                         0.0, f32, None)
    assert st == mala.MALA_ERR_INVALID_ARG
    st = lib.mala_decode(*qkv, None, *ol, None, None, 4, P(16), 1 << 20, 1, 2, 1, 64, 128, 0.1,
                         0.0, 7, None)
    assert st == mala.MALA_ERR_INVALID_ARG
    st = lib.mala_decode(*qkv, None, *ol, None, None, 2, P(16), 1 << 20, 1, 32, 1, 64, 96, 0.1,
                         0.0, f32, None)
    assert st == mala.MALA_ERR_UNSUPPORTED       # head_dim 96


def test_varlen_argument_validation(lib):
    P = ctypes.c_void_p
    qkv = [P(16)] * 3

    def fwd(cu, num_seqs, max_len, total, Hq=2, Hkv=1, D=64, tau=0.0, cu_k=None, max_k=None,
            total_k=None):
        max_k = max_len if max_k is None else max_k
        total_k = total if total_k is None else total_k
        return lib.mala_fwd_varlen(*qkv, cu, cu_k, P(16), P(16), None, None, num_seqs, max_len,
                                   max_k, total, total_k, Hq, Hkv, D, 0.125, tau, mala.OUT_BF16,
                                   None)

    assert fwd(None, 2, 8, 16) == mala.MALA_ERR_INVALID_ARG          # no cu_seqlens
    assert fwd(P(16), 0, 8, 16) == mala.MALA_ERR_INVALID_ARG         # no sequence
    assert fwd(P(16), 2, 17, 16) == mala.MALA_ERR_INVALID_ARG        # max_seqlen > total
    assert fwd(P(16), 2, 8, 16, Hq=3, Hkv=2) == mala.MALA_ERR_INVALID_ARG
    assert fwd(P(16), 2, 8, 16, D=96) == mala.MALA_ERR_UNSUPPORTED
    assert fwd(P(16), 2, 8, 1 << 24, D=128) == mala.MALA_ERR_UNSUPPORTED   # slice range
    assert fwd(P(16), 2, 8, 16, tau=-1.0) == mala.MALA_ERR_INVALID_ARG
    assert fwd(P(16), 2, 8, 16, max_k=9) == mala.MALA_ERR_INVALID_ARG     # key sizes without cu_k
    assert fwd(P(16), 2, 8, 16, cu_k=P(16), max_k=40, total_k=32) == mala.MALA_ERR_INVALID_ARG
    assert fwd(P(16), 2, 8, 16, cu_k=P(16), total_k=8) == mala.MALA_ERR_INVALID_ARG  # Nq > Nk
    st = lib.mala_bwd_varlen(*qkv, P(16), None, *([P(16)] * 6), None, None, P(16), 8, 2, 8, 8,
                             16, 16, 2, 1, 64, 0.125, 0.0, mala.OUT_F32, mala.OUT_F32, None)
    assert st == mala.MALA_ERR_WORKSPACE
    assert lib.mala_bwd_workspace_size(1, 2, 1, 16, 16, 64) > 8
    # the varlen workspace: D_q for every row and the decision bytes of each sequence's
    # query tiles (up to total / 32 + num_seqs tile rows) per head and 128-key block
    dq_bytes = 4 * 2 * 1000
    assert lib.mala_bwd_varlen_workspace_size(3, 600, 1000, 2, 1, 64) >= dq_bytes + 2 * 5 * (31 + 3)
    assert lib.mala_bwd_varlen_workspace_size(0, 600, 1000, 2, 1, 64) == 0


def test_python_binding_requires_device_tensors():
    import torch
    x = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(TypeError):
        mala.fwd(x, x, x, 0.125, 0.0)


# ---------------------------------------------------------------------------
# the Python binding checks every tensor argument (dtype, exact shape, contiguity,
# then device) before it calls the library; on the CPU the shape and dtype checks
# raise first, and tensors with the right shapes fail the device check
# ---------------------------------------------------------------------------
def _tensors(spec, over):
    import torch
    out = {}
    for name, (shape, dtype) in spec.items():
        x = over.get(name, shape)
        if isinstance(x, tuple):
            out[name] = torch.zeros(x, dtype=over.get(name + "_dtype", dtype))
        else:
            out[name] = x
    return out


def _fwd_spec():
    import torch
    bf, f32, i32, i64 = torch.bfloat16, torch.float32, torch.int32, torch.int64
    return {"q": ((1, 4, 64, 128), bf), "k": ((1, 2, 64, 128), bf), "v": ((1, 2, 64, 128), bf),
            "o": ((1, 4, 64, 128), f32), "lse": ((1, 4, 64), f32),
            "row_tiles": ((1, 4, 64), i32), "counters": ((mala.NUM_COUNTERS,), i64)}


def _bwd_spec():
    import torch
    sp = _fwd_spec()
    sp.update({"dout": ((1, 4, 64, 128), torch.bfloat16), "dq": ((1, 4, 64, 128), torch.float32),
               "dk": ((1, 2, 64, 128), torch.float32), "dv": ((1, 2, 64, 128), torch.float32),
               "workspace": ((4096,), torch.uint8)})
    return sp


def _dec_spec():
    import torch
    bf, f32, i32, i64 = torch.bfloat16, torch.float32, torch.int32, torch.int64
    return {"q": ((2, 8, 128), bf), "k_cache": ((2, 2, 300, 128), bf),
            "v_cache": ((2, 2, 300, 128), bf), "o": ((2, 8, 128), f32), "lse": ((2, 8), f32),
            "head_tiles": ((2, 8), i32), "counters": ((mala.NUM_COUNTERS,), i64),
            "workspace": ((1 << 16,), torch.uint8), "cache_lens": ((2,), i32)}


def _call_fwd(over):
    t = _tensors(_fwd_spec(), over)
    mala.mala_fwd(t["q"], t["k"], t["v"], t["o"], t["lse"], t["row_tiles"], t["counters"],
                  0.088, 1e-3)


def _call_bwd(over):
    t = _tensors(_bwd_spec(), over)
    mala.mala_bwd(t["q"], t["k"], t["v"], t["o"], t["lse"], t["dout"], t["dq"], t["dk"], t["dv"],
                  t["row_tiles"], t["counters"], t["workspace"], 0.088, 1e-3)


def _call_dec(over):
    t = _tensors(_dec_spec(), over)
    mala.mala_decode(t["q"], t["k_cache"], t["v_cache"], t["o"], t["lse"], t["head_tiles"],
                     t["counters"], 2, t["workspace"], 0.088, 1e-3, cache_lens=t["cache_lens"])


@pytest.mark.parametrize("over", [
    dict(k=(2, 2, 64, 128)), dict(k=(1, 2, 64, 64)), dict(v=(1, 2, 65, 128)),
    dict(v=(1, 1, 64, 128)), dict(o=(1, 4, 64, 64)), dict(o=(1, 4, 63, 128)),
    dict(lse=(1, 4, 63)), dict(lse=(4, 64)), dict(row_tiles=(1, 4, 65)), dict(counters=(4,)),
    dict(q=(4, 64, 128)),
])
def test_binding_fwd_rejects_shape_mismatch(over):
    with pytest.raises(ValueError):
        _call_fwd(over)


@pytest.mark.parametrize("over", [
    dict(dout=(1, 4, 64, 64)), dict(dq=(1, 4, 32, 128)), dict(dk=(1, 4, 64, 128)),
    dict(dv=(2, 2, 64, 128)), dict(lse=(1, 2, 64)), dict(k=(1, 2, 64, 64)),
])
def test_binding_bwd_rejects_shape_mismatch(over):
    with pytest.raises(ValueError):
        _call_bwd(over)


@pytest.mark.parametrize("over", [
    dict(k_cache=(1, 2, 300, 128)), dict(k_cache=(2, 2, 300, 64)), dict(v_cache=(2, 2, 299, 128)),
    dict(o=(2, 8, 64)), dict(o=(8, 128)), dict(lse=(2, 4)), dict(head_tiles=(2, 7)),
    dict(cache_lens=(3,)), dict(counters=(4,)),
])
def test_binding_decode_rejects_shape_mismatch(over):
    with pytest.raises(ValueError):
        _call_dec(over)


def test_binding_rejects_dtype_mismatch():
    import torch
    for call, over in ((_call_fwd, dict(q_dtype=torch.float32)),
                       (_call_fwd, dict(lse_dtype=torch.bfloat16)),
                       (_call_fwd, dict(counters_dtype=torch.int32)),
                       (_call_fwd, dict(row_tiles_dtype=torch.int64)),
                       (_call_bwd, dict(dout_dtype=torch.float32)),
                       (_call_bwd, dict(dk_dtype=torch.bfloat16)),      # dq fp32, dk bf16
                       (_call_dec, dict(k_cache_dtype=torch.float16)),
                       (_call_dec, dict(cache_lens_dtype=torch.int64))):
        with pytest.raises(TypeError):
            call(over)


def test_binding_rejects_non_contiguous_and_host_tensors():
    import torch
    o = torch.zeros(1, 4, 128, 64, dtype=torch.float32).transpose(2, 3)
    with pytest.raises(ValueError):
        _call_fwd(dict(o=o))
    # every shape right: the tensors live on the host, which the device check rejects
    for call in (_call_fwd, _call_bwd, _call_dec):
        with pytest.raises(TypeError, match="CUDA"):
            call({})


def test_binding_varlen_checks():
    import torch
    bf = torch.bfloat16
    q, k = torch.zeros(4, 100, 64, dtype=bf), torch.zeros(2, 100, 64, dtype=bf)
    o, lse = torch.zeros(4, 100, 64), torch.zeros(4, 100)
    cu = torch.tensor([0, 40, 100], dtype=torch.int32)
    args = lambda **kw: dict(dict(q=q, k=k, v=k, cu_seqlens=cu, max_seqlen=60, o=o, lse=lse,
                                  row_tiles=None, counters=None, scale=0.125, tau=0.0), **kw)
    with pytest.raises(TypeError):
        mala.mala_fwd_varlen(**args(cu_seqlens=cu.long()))
    with pytest.raises(ValueError):
        mala.mala_fwd_varlen(**args(cu_seqlens_k=torch.tensor([0, 100], dtype=torch.int32),
                                    max_seqlen_k=100))
    with pytest.raises(ValueError):
        mala.mala_fwd_varlen(**args(v=torch.zeros(2, 100, 128, dtype=bf)))
    with pytest.raises(ValueError):
        mala.mala_fwd_varlen(**args(lse=torch.zeros(4, 99)))
    with pytest.raises(TypeError, match="CUDA"):
        mala.mala_fwd_varlen(**args())


def test_decode_noalloc_rejects_sizes_beyond_its_buffer(lib):
    # 16 sequences x 32 heads x 64 splits of (128 + 4) floats exceed the 16 MiB buffer:
    # rejected before any HIP call (so also without a GPU); 32 splits fit
    P = ctypes.c_void_p
    qkv, ol = [P(16)] * 3, [P(16)] * 2
    need64 = mala.mala_decode_workspace_size(16, 32, 128, 64)
    assert need64 > mala.DECODE_SCRATCH_BYTES >= mala.mala_decode_workspace_size(16, 32, 128, 32)
    st = lib.mala_decode_noalloc(*qkv, None, *ol, None, None, 64, 16, 32, 8, 131072, 128, 0.088,
                                 1e-4, mala.OUT_F32, None)
    assert st == mala.MALA_ERR_WORKSPACE
    assert "buffer" in lib.mala_last_error().decode()
    st = lib.mala_decode_noalloc(*qkv, None, *ol, None, None, 0, 16, 32, 8, 131072, 128, 0.088,
                                 1e-4, mala.OUT_F32, None)
    assert st == mala.MALA_ERR_INVALID_ARG       # num_splits < 1, before the size check

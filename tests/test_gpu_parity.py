"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on the same
seeded inputs.  Small cases compare every element; the full-size workloads compare
sampled query blocks, the last key blocks and sampled decode heads (those the
oracle can compute one by one), in the launch configuration the benchmark uses.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_32712_amd as mala
from parity_util import (LSE_DIAG, TOL_MAX, assert_close, assert_counts, bwd_do_loads, dev,
                         dkdv_splits, fwd_v_loads, host,
                         set_fingerprint, tie_masks, ties)
from workloads import WORKLOADS, Workload, bf16_to_f64

pytestmark = pytest.mark.gpu


def f32(x):
    return float(np.float32(x))


def legal_tiles(B, Hq, Nq, Nk, bq, bk):
    off = Nk - Nq
    n = 0
    for i in range(-(-Nq // bq)):
        n += (min(i * bq + bq - 1, Nq - 1) + off) // bk + 1
    return n * B * Hq


# --------------------------------------------------------------------------
# small cases: every element
# --------------------------------------------------------------------------
TRAIN_CASES = {
    "needle_1k_d64": dict(spec="needle_1k_d64", over={}),
    "local_d64_ragged": dict(spec=dict(kind="train", B=1, Hq=2, Hkv=1, N=1000, D=64, beta=3.0,
                                       local=4.0), over={}),
    "gqa_d128_ragged": dict(spec=dict(kind="train", B=2, Hq=4, Hkv=2, N=700, D=128, beta=2.5,
                                      local=2.0), over={}),
    # 16 query heads per KV head: the key-major sweep of the early key blocks holds 375
    # query tiles x 16 heads = 6000 iterations, more than one compaction chunk (4096)
    "gqa16_chunks": dict(spec=dict(kind="train", B=1, Hq=16, Hkv=1, N=12000, D=128, beta=2.0,
                                   local=2.0), over={}),
    "tiny_d128": dict(spec=dict(kind="train", B=1, Hq=2, Hkv=2, N=37, D=128, beta=2.0, local=1.0),
                      over={}),
    "single_row_d64": dict(spec=dict(kind="train", B=1, Hq=1, Hkv=1, N=1, D=64, beta=1.0), over={}),
    # the language-model-like supplementary workload at a small size
    "lm_d128_ragged": dict(spec="lm_like_gqa8x2_32k", over=dict(N=1000, Hq=4, Hkv=2)),
    # two sequences, d = 64, 47 key blocks of one KV head each: the key-block sweeps run
    # in parts (1504 iterations in the first, parts of 512) summed by the reduction
    "split_d64_b2": dict(spec=dict(kind="train", B=2, Hq=8, Hkv=1, N=6000, D=64, beta=2.0,
                                   local=2.0), over={}),
}
TRAIN_TAUS = {
    "needle_1k_d64": (0.0, 1e-4, 1e-3),
    "local_d64_ragged": (0.0, 1e-2, 0.3, 1.0),
    # 1e-40 is an fp32 denormal (log2 tau = -132.9: nothing is skipped); 1e30 keeps
    # only each row's first tile in the forward and no tile in the backward
    "gqa_d128_ragged": (0.0, 1e-40, 1e-3, 0.1, 1.0, 1e30),
    "tiny_d128": (0.0, 0.5),
    # tau = 1 would put the only tile exactly on the threshold (P = 1 = tau / L):
    # 0.5 retains and 1.5 skips it in the backward, both unambiguously
    "single_row_d64": (0.0, 0.5, 1.5),
    # 1e30: every backward tile is skipped (empty compaction chunks, zero gradients)
    "gqa16_chunks": (1e-3, 1.0, 1e30),
    "lm_d128_ragged": (0.0, 1e-4, 1.0),
    "split_d64_b2": (0.0, 1e-3, 1.0),
}


def _train_case(name, tau, Nq=None, seed=0):
    c = TRAIN_CASES[name]
    w = Workload(c["spec"], seed=seed, **c["over"])
    t = w.tensors()
    q, k, v, do = t["q"], t["k"], t["v"], t["do"]
    if Nq is not None:   # prefill of the last Nq tokens against the whole cache
        q, do = np.ascontiguousarray(q[:, :, -Nq:]), np.ascontiguousarray(do[:, :, -Nq:])
    return w, q, k, v, do


def counters(t):
    """An int64 counters tensor as Python ints (the fingerprints use all 64 bits)."""
    return [int(x) for x in t.cpu().numpy()]


def _check_backward_passes_agree(cb):
    # the key-major dK/dV pass and the query-major dQ pass take the same decisions:
    # equal retained counts and equal fingerprints of the retained tile sets
    assert cb[mala.CNT_RETAINED_KV] == cb[mala.CNT_RETAINED], cb
    assert cb[mala.CNT_SET_HASH_KV] == cb[mala.CNT_SET_HASH], cb
    # the key-major pass loads a dO tile only for the query tiles it processes
    assert cb[mala.CNT_V_NEEDED] == cb[mala.CNT_V_TILES] >= 0, cb


def _check_train(w, q, k, v, do, tau):
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    assert (bq, bk) == mala.mala_geometry(w.D, mala.PASS_BWD)
    qf, kf, vf, dof = map(bf16_to_f64, (q, k, v, do))
    of = oracle.mala_fwd(qf, kf, vf, scale, f32(tau), bq, bk, want_tiles=True)
    ob = oracle.mala_bwd(qf, kf, vf, of["o"], of["lse"], dof, scale, f32(tau), bq, bk,
                         want_tiles=True)
    Q, K, V, DO = map(dev, (q, k, v, do))
    g = mala.fwd(Q, K, V, scale, tau)
    gb = mala.bwd(Q, K, V, g["o"], g["lse"], DO, scale, tau)
    torch.cuda.synchronize()
    assert_close("O", host(g["o"]), of["o"])
    lse_err = np.abs(host(g["lse"]) - of["lse"]).max()
    assert lse_err <= LSE_DIAG, lse_err
    ex_f = assert_counts("fwd row tiles", host(g["row_tiles"]), of["row_tiles"], tau, ties(of))
    ex_b = assert_counts("bwd row tiles", host(gb["row_tiles"]), ob["row_tiles"], tau, ties(of),
                         ties(ob))
    assert_close("dQ", host(gb["dq"]), ob["dq"])
    assert_close("dK", host(gb["dk"]), ob["dk"])
    assert_close("dV", host(gb["dv"]), ob["dv"])
    B, Hq, Nq, D = q.shape
    Nk = k.shape[2]
    cf, cb = counters(g["counters"]), counters(gb["counters"])
    legal = legal_tiles(B, Hq, Nq, Nk, bq, bk)
    assert cf[mala.CNT_LEGAL] == legal and cb[mala.CNT_LEGAL] == legal
    assert cf[mala.CNT_RETAINED] <= legal and (tau > 0 or cf[mala.CNT_RETAINED] == legal)
    assert 0 < cf[mala.CNT_V_NEEDED] <= cf[mala.CNT_V_TILES]
    assert cf[mala.CNT_RETAINED_KV] == 0 and cf[mala.CNT_SET_HASH_KV] == 0
    _check_backward_passes_agree(cb)
    # outside the tie band the retained sets equal the oracle's tile for tile
    if not ex_f.any():
        assert cf[mala.CNT_RETAINED] == int((of["tile_keep"] == 1).sum())
        assert cf[mala.CNT_SET_HASH] == set_fingerprint(of["tile_keep"])
        # (workgroup, key tile) pairs in which some wavefront retained the tile
        assert cf[mala.CNT_V_NEEDED] == fwd_v_loads(of["tile_keep"])
    if not ex_b.any():
        assert cb[mala.CNT_RETAINED] == int((ob["tile_keep"] == 1).sum())
        assert cb[mala.CNT_SET_HASH] == set_fingerprint(ob["tile_keep"])
        assert cb[mala.CNT_V_TILES] == bwd_do_loads(ob["tile_keep"])
    return ex_f.mean(), ex_b.mean()


@pytest.mark.parametrize("name,tau", [(n, t) for n in TRAIN_CASES for t in TRAIN_TAUS[n]])
def test_train_parity_small(name, tau):
    w, q, k, v, do = _train_case(name, tau)
    _check_train(w, q, k, v, do, tau)


@pytest.mark.parametrize("name,tau,seed", [(n, t, sd) for n in ("gqa_d128_ragged",
                                                                   "local_d64_ragged",
                                                                   "lm_d128_ragged")
                                            for t in (1e-3, 1.0) for sd in (1, 2)])
def test_train_parity_other_seeds(name, tau, seed):
    w, q, k, v, do = _train_case(name, tau, seed=seed)
    _check_train(w, q, k, v, do, tau)


@pytest.mark.parametrize("Nq,tau", [(200, 0.0), (200, 0.05), (77, 1.0)])
def test_prefill_against_longer_cache(Nq, tau):
    w, q, k, v, do = _train_case("gqa_d128_ragged", tau, Nq=Nq)
    _check_train(w, q, k, v, do, tau)


@pytest.mark.parametrize("tau", [1e-3, 1.0])
def test_prefill_with_split_sweeps(tau):
    # 5000 new rows against 12000 keys, 16 query heads on one KV head: the key-block
    # sweeps (from each block's first visible query tile) run in parts
    w, q, k, v, do = _train_case("gqa16_chunks", tau, Nq=5000)
    assert dkdv_splits(1, 16, 1, 5000, 12000)
    _check_train(w, q, k, v, do, tau)


def test_split_cases_split():
    # the parity cases meant for the split sweeps do split under the launch rule
    assert dkdv_splits(1, 16, 1, 12000) and dkdv_splits(2, 8, 1, 6000)


def test_forward_skips_are_exercised():
    # the skip-heavy case must really skip in forward and more in backward
    w, q, k, v, do = _train_case("local_d64_ragged", 1.0)
    Q, K, V, DO = map(dev, (q, k, v, do))
    g = mala.fwd(Q, K, V, f32(w.scale), 1.0)
    gb = mala.bwd(Q, K, V, g["o"], g["lse"], DO, f32(w.scale), 1.0)
    cf, cb = host(g["counters"]), host(gb["counters"])
    assert cf[1] < 0.9 * cf[0]
    assert cb[1] <= cf[1]


def test_fidelity_measurement_matches_oracle():
    # The fidelity figures the benchmark reports (per-head relative L2 errors of
    # tau = 1 against tau = 0, and the omitted mass from the two normalizers),
    # measured through the kernels, equal the oracle's within the kernels' own error.
    import bench
    tau = 1.0
    w, q, k, v, do = _train_case("lm_d128_ragged", tau)
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    qf, kf, vf, dof = map(bf16_to_f64, (q, k, v, do))
    Q, K, V, DO = map(dev, (q, k, v, do))
    ro, rg, tie_rows = {}, {}, None
    for t in (0.0, tau):
        of = oracle.mala_fwd(qf, kf, vf, scale, f32(t), bq, bk)
        ob = oracle.mala_bwd(qf, kf, vf, of["o"], of["lse"], dof, scale, f32(t), bq, bk)
        ro[t] = {x: torch.from_numpy(np.ascontiguousarray(y)) for x, y in
                 (("o", of["o"]), ("lse", of["lse"]), ("dq", ob["dq"]), ("dk", ob["dk"]),
                  ("dv", ob["dv"]))}
        g = mala.fwd(Q, K, V, scale, t)
        gb = mala.bwd(Q, K, V, g["o"], g["lse"], DO, scale, t)
        rg[t] = {"o": g["o"], "lse": g["lse"], "dq": gb["dq"], "dk": gb["dk"], "dv": gb["dv"]}
        if t > 0:
            tie_rows = tie_masks(t, ties(of))[0]
    torch.cuda.synchronize()
    rg = {t: {x: y.cpu().double() for x, y in r.items()} for t, r in rg.items()}
    fo = bench.head_fidelity(ro[0.0], ro[tau])
    fg = bench.head_fidelity(rg[0.0], rg[tau])
    # omitted mass per row: eps = -expm1(lse_t - lse_0) moves by at most the change of
    # the difference, so twice the largest LSE deviation bounds it (tie rows aside)
    delta = max(float((rg[t]["lse"] - ro[t]["lse"]).abs().max()) for t in ro)
    eo = bench.omitted_mass_rows(ro[0.0]["lse"], ro[tau]["lse"]).numpy()
    eg = bench.omitted_mass_rows(rg[0.0]["lse"], rg[tau]["lse"]).numpy()
    dev_rows = np.abs(eg - eo)[~tie_rows]
    print("[fidelity] omitted mass: oracle mean %.3e max %.3e | |gpu-oracle| max %.3e "
          "(bound %.3e, %d tie rows)" % (eo.mean(), eo.max(), dev_rows.max(), 2 * delta,
                                         int(tie_rows.sum())), flush=True)
    assert eo.max() > 0
    assert dev_rows.max() <= 2 * delta + 1e-12
    # per-head relative L2: by the triangle inequality the two measurements differ by
    # at most (e_tau + e_0 (1 + r)) / ||X_0||, e_t = ||X_t(gpu) - X_t(oracle)|| per head
    for x in ("o", "dq", "dk", "dv"):
        norm = lambda a: torch.linalg.vector_norm(a.flatten(2), dim=2).flatten().numpy()
        e_t, e_0 = (norm(rg[t][x] - ro[t][x]) for t in (tau, 0.0))
        bound = (e_t + e_0 * (1 + fo[x])) / norm(rg[0.0][x])
        print("[fidelity] rel-L2 %-2s oracle mean %.3e%% | gpu mean %.3e%% | kernel-error "
              "bound mean %.3e%%" % (x, 100 * fo[x].mean(), 100 * fg[x].mean(),
                                      100 * bound.mean()), flush=True)
        assert (np.abs(fg[x] - fo[x]) <= bound * (1 + 1e-9) + 1e-15).all(), x


# --------------------------------------------------------------------------
# packed variable-length batches
# --------------------------------------------------------------------------
VARLEN_TRAIN_CASES = {
    # ragged lengths, one token, a whole tile, several workgroups, a short tail
    "gqa_d128": (dict(kind="train", B=1, Hq=4, Hkv=2, D=128, beta=2.5, local=2.0),
                 [300, 1, 64, 513, 37]),
    "mha_d64": (dict(kind="train", B=1, Hq=2, Hkv=2, D=64, beta=3.0, local=4.0), [1000, 7, 256]),
}


def _packed(spec, lens, seed=0):
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    w = Workload(dict(spec, N=int(cu[-1])), seed=seed)
    t = w.tensors()
    return w, cu, {x: t[x][0] for x in ("q", "k", "v", "do")}   # [H, total, D]


# (tau = 1 would put a one-token sequence's only entry exactly on its threshold,
# P = 1 = tau / L, where either decision is correct; 0.5 retains it unambiguously)
@pytest.mark.parametrize("name,tau", [(n, t) for n in VARLEN_TRAIN_CASES
                                      for t in (0.0, 1e-3, 0.5)])
def test_varlen_train_parity(name, tau):
    # every packed sequence against the oracle run on that sequence alone
    spec, lens = VARLEN_TRAIN_CASES[name]
    w, cu, t = _packed(spec, lens)
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    Q, K, V, DO = (dev(t[x]) for x in ("q", "k", "v", "do"))
    CU = torch.from_numpy(cu).to("cuda")
    g = mala.fwd_varlen(Q, K, V, CU, max(lens), scale, tau)
    gb = mala.bwd_varlen(Q, K, V, CU, max(lens), g["o"], g["lse"], DO, scale, tau)
    torch.cuda.synchronize()
    o, lse, rt = host(g["o"]), host(g["lse"]), host(g["row_tiles"])
    dq, dk, dv, rtb = host(gb["dq"]), host(gb["dk"]), host(gb["dv"]), host(gb["row_tiles"])
    legal, fp_f, fp_b, any_ex_f, any_ex_b = 0, 0, 0, False, False
    for b, n in enumerate(lens):
        r = slice(int(cu[b]), int(cu[b + 1]))
        qf, kf, vf, dof = (bf16_to_f64(t[x][None, :, r]) for x in ("q", "k", "v", "do"))
        of = oracle.mala_fwd(qf, kf, vf, scale, f32(tau), bq, bk, want_tiles=True)
        ob = oracle.mala_bwd(qf, kf, vf, of["o"], of["lse"], dof, scale, f32(tau), bq, bk,
                             want_tiles=True)
        assert_close("O seq %d (n=%d)" % (b, n), o[:, r], of["o"][0])
        assert np.abs(lse[:, r] - of["lse"][0]).max() <= LSE_DIAG
        ex_f = assert_counts("fwd row tiles seq %d" % b, rt[:, r], of["row_tiles"][0], tau,
                             ties(of, 0))
        ex_b = assert_counts("bwd row tiles seq %d" % b, rtb[:, r], ob["row_tiles"][0], tau,
                             ties(of, 0), ties(ob, 0))
        assert_close("dQ seq %d" % b, dq[:, r], ob["dq"][0])
        assert_close("dK seq %d" % b, dk[:, r], ob["dk"][0])
        assert_close("dV seq %d" % b, dv[:, r], ob["dv"][0])
        legal += legal_tiles(1, w.Hq, n, n, bq, bk)
        fp_f += set_fingerprint(of["tile_keep"], b0=b)
        fp_b += set_fingerprint(ob["tile_keep"], b0=b)
        any_ex_f |= bool(ex_f.any())
        any_ex_b |= bool(ex_b.any())
    cf, cb = counters(g["counters"]), counters(gb["counters"])
    assert cf[mala.CNT_LEGAL] == legal and cb[mala.CNT_LEGAL] == legal
    _check_backward_passes_agree(cb)
    wrap = lambda x: (x + (1 << 63)) % (1 << 64) - (1 << 63)    # sum modulo 2^64, signed
    if not any_ex_f:
        assert cf[mala.CNT_SET_HASH] == wrap(fp_f)
    if not any_ex_b:
        assert cb[mala.CNT_SET_HASH] == wrap(fp_b)


def test_varlen_cut_and_uncovered_rows():
    # a sequence longer than max_seqlen is cut to its first max_seqlen rows, and rows
    # that no sequence covers are left as the caller's zeros
    spec = dict(kind="train", B=1, Hq=2, Hkv=1, N=300, D=128, beta=2.0, local=2.0)
    w = Workload(spec)
    t = {x: y[0] for x, y in w.tensors().items()}
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    cu = np.array([0, 150, 250], dtype=np.int32)          # rows 250..299 uncovered
    Q, K, V, DO = (dev(t[x]) for x in ("q", "k", "v", "do"))
    CU = torch.from_numpy(cu).to("cuda")
    g = mala.fwd_varlen(Q, K, V, CU, 120, scale, 1e-3)    # sequence 0 cut to 120 rows
    gb = mala.bwd_varlen(Q, K, V, CU, 120, g["o"], g["lse"], DO, scale, 1e-3)
    torch.cuda.synchronize()
    o, dq, dk = host(g["o"]), host(gb["dq"]), host(gb["dk"])
    for rows in (slice(120, 150), slice(250, 300)):
        assert (o[:, rows] == 0).all() and (dq[:, rows] == 0).all() and (dk[:, rows] == 0).all()
    for r in (slice(0, 120), slice(150, 250)):
        qf, kf, vf, dof = (bf16_to_f64(t[x][None, :, r]) for x in ("q", "k", "v", "do"))
        of = oracle.mala_fwd(qf, kf, vf, scale, f32(1e-3), bq, bk)
        ob = oracle.mala_bwd(qf, kf, vf, of["o"], of["lse"], dof, scale, f32(1e-3), bq, bk)
        assert_close("O", o[:, r], of["o"][0])
        assert_close("dK", dk[:, r], ob["dk"][0])


@pytest.mark.parametrize("tau", [0.0, 1e-3, 0.5])
def test_varlen_prefill_parity(tau):
    # packed prefill against cached keys: sequence b has lens_k[b] keys and its last
    # lens_q[b] rows as queries (bottom-right aligned); one sequence is skipped
    # because it has more query rows than keys, and its rows stay zero
    lens_k = [300, 64, 513, 40, 3]
    lens_q = [100, 64, 1, 17, 5]
    spec = dict(kind="train", B=1, Hq=4, Hkv=2, D=128, beta=2.5, local=2.0)
    cuk = np.concatenate([[0], np.cumsum(lens_k)]).astype(np.int32)
    cuq = np.concatenate([[0], np.cumsum(lens_q)]).astype(np.int32)
    w = Workload(dict(spec, N=int(cuk[-1])))
    t = {x: y[0] for x, y in w.tensors().items()}
    rows = np.concatenate([np.arange(cuk[b + 1] - nq, cuk[b + 1]) for b, nq in enumerate(lens_q)])
    q = np.ascontiguousarray(t["q"][:, rows])
    do = np.ascontiguousarray(t["do"][:, rows])
    k, v = t["k"], t["v"]
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    Q, K, V, DO = dev(q), dev(k), dev(v), dev(do)
    CUQ, CUK = (torch.from_numpy(c).to("cuda") for c in (cuq, cuk))
    kw = dict(cu_seqlens_k=CUK, max_seqlen_k=max(lens_k))
    g = mala.fwd_varlen(Q, K, V, CUQ, max(lens_q), scale, tau, **kw)
    gb = mala.bwd_varlen(Q, K, V, CUQ, max(lens_q), g["o"], g["lse"], DO, scale, tau, **kw)
    torch.cuda.synchronize()
    o, lse, rt = host(g["o"]), host(g["lse"]), host(g["row_tiles"])
    dq, dk, dv = host(gb["dq"]), host(gb["dk"]), host(gb["dv"])
    legal = 0
    for b, (nq, nk) in enumerate(zip(lens_q, lens_k)):
        rq, rk = slice(int(cuq[b]), int(cuq[b + 1])), slice(int(cuk[b]), int(cuk[b + 1]))
        if nq > nk:
            assert (o[:, rq] == 0).all() and (dq[:, rq] == 0).all() and (dk[:, rk] == 0).all()
            continue
        qf, dof = bf16_to_f64(q[None, :, rq]), bf16_to_f64(do[None, :, rq])
        kf, vf = bf16_to_f64(k[None, :, rk]), bf16_to_f64(v[None, :, rk])
        of = oracle.mala_fwd(qf, kf, vf, scale, f32(tau), bq, bk)
        ob = oracle.mala_bwd(qf, kf, vf, of["o"], of["lse"], dof, scale, f32(tau), bq, bk)
        assert_close("O seq %d (%d of %d)" % (b, nq, nk), o[:, rq], of["o"][0])
        assert np.abs(lse[:, rq] - of["lse"][0]).max() <= LSE_DIAG
        assert_counts("fwd row tiles seq %d" % b, rt[:, rq], of["row_tiles"][0], tau, ties(of, 0))
        assert_close("dQ seq %d" % b, dq[:, rq], ob["dq"][0])
        assert_close("dK seq %d" % b, dk[:, rk], ob["dk"][0])
        assert_close("dV seq %d" % b, dv[:, rk], ob["dv"][0])
        legal += legal_tiles(1, w.Hq, nq, nk, bq, bk)
    cb = counters(gb["counters"])
    assert counters(g["counters"])[mala.CNT_LEGAL] == legal and cb[mala.CNT_LEGAL] == legal
    _check_backward_passes_agree(cb)




@pytest.mark.parametrize("tau", [1e-4, 1.0])
def test_varlen_full_size_equals_per_sequence_calls(tau):
    # 32768 packed tokens of the language-model-like inputs: every sequence's
    # outputs equal, bit for bit, a fixed-length call on that sequence alone (the
    # same tiles from the sequence's first row, the same arithmetic).  Except dK and
    # dV where the fixed-length call splits its key-block sweeps (few key-block
    # workgroups): its parts add their sums afterwards and share the lo-term budgets,
    # so the two agree within the sum of their error bounds (2^-8 x budget x the
    # largest |dO| or scale |Q|, per path)
    lens = [16384, 8192, 4096, 1500, 1024, 1000, 500, 68, 4]
    w, cu, t = _packed(dict(WORKLOADS["lm_like_gqa8x2_32k"], B=1), lens)
    scale = f32(w.scale)
    Q, K, V, DO = (dev(t[x]) for x in ("q", "k", "v", "do"))
    CU = torch.from_numpy(cu).to("cuda")
    print("[varlen full] packed fwd + bwd", flush=True)
    g = mala.fwd_varlen(Q, K, V, CU, max(lens), scale, tau)
    gb = mala.bwd_varlen(Q, K, V, CU, max(lens), g["o"], g["lse"], DO, scale, tau)
    torch.cuda.synchronize()
    for b in range(len(lens)):
        r = slice(int(cu[b]), int(cu[b + 1]))
        q1, k1, v1, do1 = (x[None, :, r].contiguous() for x in (Q, K, V, DO))
        f1 = mala.fwd(q1, k1, v1, scale, tau)
        b1 = mala.bwd(q1, k1, v1, f1["o"], f1["lse"], do1, scale, tau)
        torch.cuda.synchronize()
        pairs = (("o", g["o"], f1["o"]), ("lse", g["lse"], f1["lse"]),
                 ("row_tiles", g["row_tiles"], f1["row_tiles"]), ("dq", gb["dq"], b1["dq"]),
                 ("bwd row_tiles", gb["row_tiles"], b1["row_tiles"]))
        for name, a, ref in pairs:
            assert torch.equal(a[:, r], ref[0]), (b, name)
        split = dkdv_splits(1, w.Hq, w.Hkv, lens[b])
        for name, a, ref in (("dk", gb["dk"], b1["dk"]), ("dv", gb["dv"], b1["dv"])):
            if split:
                err = (a[:, r] - ref[0]).abs().max().item()
                assert err <= 2e-3, (b, name, err)
            else:
                assert torch.equal(a[:, r], ref[0]), (b, name)


DECODE_CASES = [
    (dict(kind="decode", B=2, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4), 1, 0.0),
    (dict(kind="decode", B=2, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4), 4, 1e-4),
    (dict(kind="decode", B=2, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4), 7, 1e-2),
    (dict(kind="decode", B=1, Hq=2, Hkv=2, N=999, D=64, beta=3.0, needles=4), 3, 0.1),
    (dict(kind="decode", B=3, Hq=16, Hkv=1, N=64, D=128, beta=2.0, needles=2), 2, 1e-3),
    (dict(kind="decode", B=1, Hq=4, Hkv=4, N=5, D=64, beta=2.0, needles=1), 1, 1.0),
    # groups of more than 16 query heads (two wavefronts per KV head and split)
    (dict(kind="decode", B=2, Hq=40, Hkv=2, N=1500, D=128, beta=3.0, needles=4), 3, 1e-3),
    (dict(kind="decode", B=1, Hq=32, Hkv=1, N=777, D=64, beta=3.0, needles=4), 2, 0.1),
]


def _decode_v_needed(keep, Hkv):
    """V tiles a decode wavefront consumes, from the oracle's decisions keep [B, Hq, T]:
    one per (sequence, KV head, chunk of up to 16 query heads of its group, key tile)
    in which some head of the chunk retains the tile."""
    keep = np.asarray(keep)
    B, Hq, T = keep.shape
    grp = Hq // Hkv
    n = 0
    for hk in range(Hkv):
        for c0 in range(0, grp, 16):
            heads = slice(hk * grp + c0, hk * grp + min(grp, c0 + 16))
            n += int((keep[:, heads] == 1).any(axis=1).sum())
    return n


def _check_decode_counters(cd, keep_b, ex, Hkv):
    """keep_b: [(b, keep [1, Hq, T_b])] of the oracle; ex: the exempt heads."""
    assert 0 < cd[mala.CNT_V_NEEDED] <= cd[mala.CNT_V_TILES], cd
    assert cd[mala.CNT_RETAINED_KV] == 0 and cd[mala.CNT_SET_HASH_KV] == 0
    if not np.asarray(ex).any():
        fp = sum(set_fingerprint(kp, b0=b) for b, kp in keep_b)
        assert cd[mala.CNT_SET_HASH] == (fp + (1 << 63)) % (1 << 64) - (1 << 63)
        assert cd[mala.CNT_V_NEEDED] == sum(_decode_v_needed(kp, Hkv) for _, kp in keep_b)


@pytest.mark.parametrize("spec,splits,tau", DECODE_CASES)
def test_decode_parity_small(spec, splits, tau):
    w = Workload(spec)
    t = w.tensors()
    scale = f32(w.scale)
    bk = mala.mala_geometry(w.D, mala.PASS_DECODE)[1]
    qf, kf, vf = map(bf16_to_f64, (t["q"], t["k"], t["v"]))
    od = oracle.mala_decode(qf, kf, vf, scale, f32(tau), bk, splits, want_tiles=True)
    g = mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]), scale, tau, splits)
    torch.cuda.synchronize()
    assert_close("decode O", host(g["o"]), od["o"])
    assert np.abs(host(g["lse"]) - od["lse"]).max() <= LSE_DIAG
    ex = assert_counts("decode head tiles", host(g["head_tiles"]), od["tiles"], tau, ties(od))
    cd = counters(g["counters"])
    assert cd[mala.CNT_LEGAL] == w.B * w.Hq * -(-w.N // bk)
    _check_decode_counters(cd, [(b, od["keep"][b:b + 1]) for b in range(w.B)], ex, w.Hkv)


VARLEN_DECODE_CASES = [
    # per-sequence cache lengths: full, ragged, one token, a whole number of tiles,
    # empty, and one past the capacity (clamped to Nk)
    (dict(kind="decode", B=6, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4),
     [3001, 1777, 1, 64, 0, 5000], 4, 1e-4),
    (dict(kind="decode", B=3, Hq=4, Hkv=4, N=999, D=64, beta=3.0, needles=4), [999, 33, 500], 3,
     0.1),
    (dict(kind="decode", B=4, Hq=16, Hkv=1, N=2048, D=128, beta=2.0, needles=2),
     [2048, 1000, 31, 1500], 7, 1.0),
]


@pytest.mark.parametrize("spec,lens,splits,tau", VARLEN_DECODE_CASES)
def test_decode_per_sequence_cache_lengths(spec, lens, splits, tau):
    # each sequence against the oracle on its own valid prefix of the cache
    w = Workload(spec)
    t = w.tensors()
    scale = f32(w.scale)
    bk = mala.mala_geometry(w.D, mala.PASS_DECODE)[1]
    qf, kf, vf = map(bf16_to_f64, (t["q"], t["k"], t["v"]))
    cl = torch.tensor(lens, dtype=torch.int32, device="cuda")
    g = mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]), scale, tau, splits, cache_lens=cl)
    torch.cuda.synchronize()
    o, lse, ht = host(g["o"]), host(g["lse"]), host(g["head_tiles"])
    legal, keeps, exs = 0, [], []
    for b, n in enumerate(lens):
        n = min(max(n, 0), w.N)
        if n == 0:
            assert (o[b] == 0).all() and np.isneginf(lse[b]).all() and (ht[b] == 0).all()
            continue
        od = oracle.mala_decode(qf[b:b + 1], kf[b:b + 1, :, :n], vf[b:b + 1, :, :n], scale,
                                f32(tau), bk, splits, want_tiles=True)
        assert_close("decode O seq %d (n=%d)" % (b, n), o[b], od["o"][0])
        assert np.abs(lse[b] - od["lse"][0]).max() <= LSE_DIAG
        exs.append(assert_counts("decode head tiles seq %d" % b, ht[b:b + 1], od["tiles"], tau,
                                 ties(od)).any())
        keeps.append((b, od["keep"]))
        legal += -(-n // bk) * w.Hq
    cd = counters(g["counters"])
    assert cd[mala.CNT_LEGAL] == legal
    _check_decode_counters(cd, keeps, exs, w.Hkv)


@pytest.mark.parametrize("tau", [0.0, 1e-3])
def test_decode_never_reads_cache_rows_past_a_length(tau):
    # rows at and past a sequence's cache length play no part: filling them with NaN
    # leaves every output and statistic bitwise unchanged (lengths off the 32-key
    # grid, so each sequence ends in a ragged tile, and one sequence shorter than
    # one split's share of the tiles)
    spec = dict(kind="decode", B=3, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4)
    w = Workload(spec)
    t = {x: np.array(y) for x, y in w.tensors().items()}
    lens = [3001, 1000, 37]
    cl = torch.tensor(lens, dtype=torch.int32, device="cuda")

    def run():
        g = mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]), f32(w.scale), tau, 4,
                        cache_lens=cl)
        torch.cuda.synchronize()
        return {x: y.cpu() for x, y in g.items()}

    clean = run()
    for b, n in enumerate(lens):
        t["k"][b, :, n:] = NAN_BITS
        t["v"][b, :, n:] = NAN_BITS
    bad = run()
    assert torch.isfinite(bad["o"]).all()
    for name in clean:
        assert torch.equal(bad[name], clean[name]), name


def test_decode_full_lengths_match_uniform_path():
    # cache_lens all equal to Nk is the uniform decode (bitwise at tau = 0, where
    # the threshold plays no part)
    spec = dict(kind="decode", B=3, Hq=8, Hkv=2, N=1500, D=128, beta=3.0, needles=4)
    w = Workload(spec)
    t = w.tensors()
    q, k, v = dev(t["q"]), dev(t["k"]), dev(t["v"])
    cl = torch.full((w.B,), w.N, dtype=torch.int32, device="cuda")
    for tau in (0.0, 1e-3):
        a = mala.decode(q, k, v, f32(w.scale), tau, 3)
        b = mala.decode(q, k, v, f32(w.scale), tau, 3, cache_lens=cl)
        torch.cuda.synchronize()
        if tau == 0.0:
            assert torch.equal(a["o"], b["o"]) and torch.equal(a["lse"], b["lse"])
        else:
            np.testing.assert_allclose(host(b["o"]), host(a["o"]), atol=1e-5)


def test_decode_splits_cover_dense_at_tau0():
    spec = dict(kind="decode", B=1, Hq=4, Hkv=1, N=2048, D=128, beta=3.0, needles=4)
    w = Workload(spec)
    t = w.tensors()
    outs = [mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]), f32(w.scale), 0.0, s)
            for s in (1, 5, 64)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        np.testing.assert_allclose(host(o["o"]), host(outs[0]["o"]), atol=1e-5)
        assert (host(o["head_tiles"]) == 64).all()


# --------------------------------------------------------------------------
# full-size workloads: sampled outputs in the benchmark's launch configuration
# --------------------------------------------------------------------------
def _full_train(name, tau, sample_heads, sample_fracs, kv, rows_from, key_fracs, seed=0):
    """One workload in the benchmark's launch configuration, against the oracle on:
      * sampled query blocks (sample_fracs of the blocks) of sampled query heads:
        O, LSE, forward and backward retained counts, dQ;
      * one KV head kv = (b, h_kv) with every query head of its GQA group: O, LSE and
        forward counts on every query row from rows_from * N on, then dK and dV on two
        key tiles at each of key_fracs (at or after rows_from * N: such keys are seen
        only by rows the oracle forward covered), accumulated over all those rows and
        heads the way the key-major pass accumulates them;
    and the two backward passes' retained counts and fingerprints against each
    other."""
    w = Workload(name, seed=seed)
    print("[full %s tau=%g] generating inputs" % (name, tau), flush=True)
    t = w.tensors(threads=16)
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    N, D = w.N, w.D
    Q, K, V, DO = map(dev, (t["q"], t["k"], t["v"], t["do"]))
    print("[full %s] gpu fwd+bwd" % name, flush=True)
    g = mala.fwd(Q, K, V, scale, tau)
    gb = mala.bwd(Q, K, V, g["o"], g["lse"], DO, scale, tau)
    torch.cuda.synchronize()
    _check_backward_passes_agree(counters(gb["counters"]))
    o_gpu, lse_gpu, rt_gpu = host(g["o"]), host(g["lse"]), host(g["row_tiles"])
    dq_gpu, rtb_gpu = host(gb["dq"]), host(gb["row_tiles"])
    dk_gpu, dv_gpu = host(gb["dk"]), host(gb["dv"])
    del Q, K, V, DO, g, gb
    Tr, Tc = -(-N // bq), -(-N // bk)
    grp = w.g
    f64 = lambda x, b_, h0, h1: bf16_to_f64(t[x][b_:b_ + 1, h0:h1])
    # sampled query blocks of sampled heads: forward, dQ and counts
    for (b, h) in sample_heads:
        hk = h // grp
        qf, dof = f64("q", b, h, h + 1), f64("do", b, h, h + 1)
        kf, vf = f64("k", b, hk, hk + 1), f64("v", b, hk, hk + 1)
        for i in sorted({min(Tr - 1, int(f * Tr)) for f in sample_fracs}):
            print("[full %s] oracle head %d block %d" % (name, h, i), flush=True)
            rows = slice(i * bq, min(N, (i + 1) * bq))
            of = oracle.mala_fwd(qf, kf, vf, scale, f32(tau), bq, bk, blocks=(i, i + 1))
            ob = oracle.mala_bwd(qf, kf, vf, of["o"], of["lse"], dof, scale, f32(tau), bq, bk,
                                 qblocks=(i, i + 1), kblocks=(0, 0))
            sl = (0, 0, rows)
            assert_close("O blk %d" % i, o_gpu[b, h, rows], of["o"][sl])
            assert np.abs(lse_gpu[b, h, rows] - of["lse"][sl]).max() <= LSE_DIAG
            assert_counts("fwd tiles", rt_gpu[b, h, rows], of["row_tiles"][sl], tau, ties(of, sl))
            assert_counts("bwd tiles", rtb_gpu[b, h, rows], ob["row_tiles"][sl], tau,
                          ties(of, sl), ties(ob, sl))
            assert_close("dQ blk %d" % i, dq_gpu[b, h, rows], ob["dq"][sl])
    # one KV head and its whole query-head group
    b, hk = kv
    h0, h1 = hk * grp, (hk + 1) * grp
    i0 = int(rows_from * Tr)
    r0 = i0 * bq
    qf, dof = f64("q", b, h0, h1), f64("do", b, h0, h1)
    kf, vf = f64("k", b, hk, hk + 1), f64("v", b, hk, hk + 1)
    print("[full %s] oracle forward of kv head %d (%d query heads), rows %d.." %
          (name, hk, grp, r0), flush=True)
    of = oracle.mala_fwd(qf, kf, vf, scale, f32(tau), bq, bk, blocks=(i0, Tr))
    sl = (0, slice(None), slice(r0, N))
    assert_close("O group", o_gpu[b, h0:h1, r0:], of["o"][sl])
    assert np.abs(lse_gpu[b, h0:h1, r0:] - of["lse"][sl]).max() <= LSE_DIAG
    assert_counts("fwd tiles group", rt_gpu[b, h0:h1, r0:], of["row_tiles"][sl], tau,
                  ties(of, sl))
    o_in, lse_in = np.nan_to_num(of["o"]), np.nan_to_num(of["lse"])
    j_lo = -(-r0 // bk)
    for j in sorted({min(Tc - 2, max(j_lo, int(f * Tc))) for f in key_fracs}):
        print("[full %s] oracle dK/dV of key tiles %d-%d (kv head %d)" % (name, j, j + 1, hk),
              flush=True)
        ob = oracle.mala_bwd(qf, kf, vf, o_in, lse_in, dof, scale, f32(tau), bq, bk,
                             qblocks=(0, 0), kblocks=(j, j + 2))
        r = slice(j * bk, min(N, (j + 2) * bk))
        assert_close("dK keys %d.." % (j * bk), dk_gpu[b, hk, r], ob["dk"][0, 0, r])
        assert_close("dV keys %d.." % (j * bk), dv_gpu[b, hk, r], ob["dv"][0, 0, r])


EDGES = (0.0, 0.5, 1.0)   # key tiles at the start, the middle and the end


@pytest.mark.parametrize("tau", [0.0, 1e-4, 1e-3])
def test_full_mha16_8k_sampled(tau):
    _full_train("mha16_8k", tau, [(0, 3), (0, 12)], (0.0, 0.37, 0.999), kv=(0, 5), rows_from=0.0,
                key_fracs=EDGES)


@pytest.mark.parametrize("tau", [0.0, 1e-4, 1.0])
def test_full_gqa32x8_32k_sampled(tau):
    # heads 28..31 of KV head 7; their needle strengths beta_h differ
    _full_train("gqa32x8_32k", tau, [(0, 1), (0, 30)], (0.5, 0.999), kv=(0, 7), rows_from=0.0,
                key_fracs=EDGES)


@pytest.mark.parametrize("tau", [1e-4, 1.0])
def test_full_gqa8x2_128k_sampled(tau):
    # the key tiles from 15/16 of the sequence on accumulate over ~1000 query tiles of
    # each of the 4 query heads of the group
    _full_train("gqa8x2_128k", tau, [(0, 6)], (0.25, 0.999), kv=(0, 1), rows_from=15 / 16,
                key_fracs=(15 / 16, 31 / 32, 1.0))


@pytest.mark.parametrize("tau", [1e-4, 1.0])
def test_full_lm_like_gqa8x2_32k_sampled(tau):
    _full_train("lm_like_gqa8x2_32k", tau, [(0, 2), (0, 7)], (0.3, 0.999), kv=(0, 1), rows_from=0.0,
                key_fracs=EDGES)


@pytest.mark.parametrize("tau", [0.0, 1e-4, 1.0])
def test_full_decode_gqa32x8_128k_sampled(tau):
    w = Workload("decode_gqa32x8_128k")
    print("[full decode_gqa32x8_128k tau=%g] generating inputs" % tau, flush=True)
    t = w.tensors(threads=16)
    scale = f32(w.scale)
    bk = mala.mala_geometry(w.D, mala.PASS_DECODE)[1]
    S = mala.default_num_splits(w.B, w.Hkv, w.N)
    g = mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]), scale, tau, S)
    torch.cuda.synchronize()
    o, lse, ht = host(g["o"]), host(g["lse"]), host(g["head_tiles"])
    rng = np.random.default_rng(5)
    pairs = [(int(rng.integers(w.B)), int(rng.integers(w.Hq))) for _ in range(6)]
    print("[full decode_gqa32x8_128k] oracle on", pairs, "splits", S, flush=True)
    qf = bf16_to_f64(t["q"])
    for b, h in pairs:
        hk = h // w.g
        od = oracle.mala_decode(qf[b:b + 1, h:h + 1], bf16_to_f64(t["k"][b:b + 1, hk:hk + 1]),
                                bf16_to_f64(t["v"][b:b + 1, hk:hk + 1]), scale, f32(tau), bk, S)
        assert_close("decode O", o[b, h], od["o"][0, 0])
        assert abs(lse[b, h] - od["lse"][0, 0]) <= LSE_DIAG
        assert_counts("decode tiles", ht[b:b + 1, h:h + 1], od["tiles"], tau, ties(od))


@pytest.mark.parametrize("tau", [1e-4, 1.0])
def test_full_decode_gqa32x8_128k_ragged_lengths_sampled(tau):
    # the serving case: the 131072-token caches holding ragged valid lengths
    w = Workload("decode_gqa32x8_128k")
    print("[full decode_gqa32x8_128k ragged tau=%g] generating inputs" % tau, flush=True)
    t = w.tensors(threads=16)
    scale = f32(w.scale)
    bk = mala.mala_geometry(w.D, mala.PASS_DECODE)[1]
    S = mala.default_num_splits(w.B, w.Hkv, w.N)
    lens = np.random.default_rng(7).integers(1, w.N + 1, size=w.B).astype(np.int32)
    lens[0], lens[1] = w.N, 1
    cl = torch.from_numpy(lens).to("cuda")
    g = mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]), scale, tau, S, cache_lens=cl)
    torch.cuda.synchronize()
    o, lse, ht = host(g["o"]), host(g["lse"]), host(g["head_tiles"])
    qf = bf16_to_f64(t["q"])
    for b, h in [(0, 5), (1, 0), (2, 17), (9, 31)]:
        n, hk = int(lens[b]), h // w.g
        print("[full decode_gqa32x8_128k ragged] oracle seq %d head %d n=%d splits %d" % (b, h, n, S), flush=True)
        od = oracle.mala_decode(qf[b:b + 1, h:h + 1], bf16_to_f64(t["k"][b:b + 1, hk:hk + 1, :n]),
                                bf16_to_f64(t["v"][b:b + 1, hk:hk + 1, :n]), scale, f32(tau), bk,
                                S)
        assert_close("decode O", o[b, h], od["o"][0, 0])
        assert abs(lse[b, h] - od["lse"][0, 0]) <= LSE_DIAG
        assert_counts("decode tiles", ht[b:b + 1, h:h + 1], od["tiles"], tau, ties(od))


# --------------------------------------------------------------------------
# non-finite inputs: the kernels finish, the outputs that depend on a NaN / Inf
# input are non-finite, and the outputs of tiles that never touch it are bitwise
# those of the clean inputs (tau = 0: every tile is retained, so a row with a NaN
# state cannot change another row's decisions).  Inside a 32 x 32 tile that holds
# the bad value, masked entries may become NaN too (their zero probability meets
# the NaN in an MFMA product), so whole tiles are compared.
# --------------------------------------------------------------------------
def _nonfinite_case():
    w, q, k, v, do = _train_case("gqa_d128_ragged", 0.0)
    return w, [np.array(x) for x in (q, k, v, do)]


def _run_train(w, q, k, v, do, tau=0.0):
    Q, K, V, DO = map(dev, (q, k, v, do))
    g = mala.fwd(Q, K, V, f32(w.scale), tau)
    gb = mala.bwd(Q, K, V, g["o"], g["lse"], DO, f32(w.scale), tau)
    torch.cuda.synchronize()
    return {x: y.cpu() for x, y in list(g.items()) + list(gb.items()) if x != "counters"}


NAN_BITS, INF_BITS = np.uint16(0x7FC0), np.uint16(0x7F80)   # bf16 NaN and +Inf


@pytest.mark.parametrize("tensor", ["q", "do"])
def test_nan_in_a_query_row_propagates(tensor):
    w, (q, k, v, do) = _nonfinite_case()
    clean = _run_train(w, q, k, v, do)
    b, h, r = 1, 3, 333                    # query head 3 reads KV head 1
    x = {"q": q, "do": do}[tensor]
    x[b, h, r, 5] = NAN_BITS
    bad = _run_train(w, q, k, v, do)
    hk = h // w.g
    t0 = r // 32 * 32                        # first row / key of r's 32-row tile
    # the row's own outputs
    assert torch.isnan(bad["dq"][b, h, r]).all()
    if tensor == "q":
        assert torch.isnan(bad["o"][b, h, r]).all() and torch.isnan(bad["lse"][b, h, r])
    # every key up to the row feeds the row's gradient: dK and dV are NaN there
    assert (~torch.isfinite(bad["dk"][b, hk, :r + 1])).any(dim=-1).all()
    assert (~torch.isfinite(bad["dv"][b, hk, :r + 1])).any(dim=-1).all()
    # untouched: the rows of the other 32-row tiles (the rows of r's own tile share
    # its wavefront's rescaling and lo-term ballots, so their last bits may move),
    # keys after r's tile, other KV heads and sequences
    rows = torch.ones(w.N, dtype=torch.bool)
    rows[t0:t0 + 32] = False
    others = [hh for hh in range(w.Hq) if hh != h]
    for name in ("o", "lse", "dq", "row_tiles"):
        if name in ("o", "lse", "row_tiles") and tensor == "do":
            assert torch.equal(bad[name], clean[name]), name     # dO plays no part
            continue
        sel = slice(None) if name == "row_tiles" else rows     # tau = 0: counts unchanged
        assert torch.equal(bad[name][b, h, sel], clean[name][b, h, sel]), name
        assert torch.equal(bad[name][:, others], clean[name][:, others]), name
        assert torch.equal(bad[name][1 - b], clean[name][1 - b]), name
    for name in ("dk", "dv"):
        assert torch.equal(bad[name][b, hk, t0 + 32:], clean[name][b, hk, t0 + 32:]), name
        assert torch.equal(bad[name][b, 1 - hk], clean[name][b, 1 - hk]), name
        assert torch.equal(bad[name][1 - b], clean[name][1 - b]), name


def test_inf_in_a_value_row_propagates():
    w, (q, k, v, do) = _nonfinite_case()
    clean = _run_train(w, q, k, v, do)
    b, hk, c = 0, 1, 250
    v[b, hk, c, 7] = INF_BITS
    bad = _run_train(w, q, k, v, do)
    heads = range(hk * w.g, (hk + 1) * w.g)
    t0 = c // 32 * 32
    for h in heads:
        # every row that sees key c (retained at tau = 0) has a non-finite output
        assert (~torch.isfinite(bad["o"][b, h, c:])).any(dim=-1).all()
        # rows of the query tiles before key c's tile never touch it
        assert torch.equal(bad["o"][b, h, :t0], clean["o"][b, h, :t0])
        assert torch.equal(bad["lse"][b, h], clean["lse"][b, h])   # V plays no part in LSE
    others = [h for h in range(w.Hq) if h not in heads]
    for name in ("o", "lse", "dq", "dk", "dv"):
        assert torch.equal(bad[name][1 - b], clean[name][1 - b]), name
    for name in ("o", "dq"):
        assert torch.equal(bad[name][:, others], clean[name][:, others]), name


def test_nan_in_a_decode_query_propagates():
    spec = dict(kind="decode", B=2, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4)
    w = Workload(spec)
    t = {x: np.array(y) for x, y in w.tensors().items()}
    run = lambda: {x: y.cpu() for x, y in mala.decode(dev(t["q"]), dev(t["k"]), dev(t["v"]),
                                                       f32(w.scale), 0.0, 4).items()}
    clean = run()
    torch.cuda.synchronize()
    t["q"][1, 5, 9] = NAN_BITS
    bad = run()
    torch.cuda.synchronize()
    assert torch.isnan(bad["o"][1, 5]).all() and torch.isnan(bad["lse"][1, 5])
    keep = torch.ones(2, 8, dtype=torch.bool)
    keep[1, 5] = False
    assert torch.equal(bad["o"][keep], clean["o"][keep])
    assert torch.equal(bad["lse"][keep], clean["lse"][keep])


# --------------------------------------------------------------------------
# reproducibility
# --------------------------------------------------------------------------
def test_repeat_runs_bitwise_forward_dk_dv():
    # no kernel accumulates through atomics or in a launch-dependent order, so
    # repeated calls give identical outputs and statistics
    w, q, k, v, do = _train_case("gqa_d128_ragged", 0.1)
    Q, K, V, DO = map(dev, (q, k, v, do))
    r1 = mala.fwd(Q, K, V, f32(w.scale), 0.1)
    r2 = mala.fwd(Q, K, V, f32(w.scale), 0.1)
    b1 = mala.bwd(Q, K, V, r1["o"], r1["lse"], DO, f32(w.scale), 0.1)
    b2 = mala.bwd(Q, K, V, r1["o"], r1["lse"], DO, f32(w.scale), 0.1)
    torch.cuda.synchronize()
    assert torch.equal(r1["o"], r2["o"]) and torch.equal(r1["lse"], r2["lse"])
    assert torch.equal(b1["dk"], b2["dk"]) and torch.equal(b1["dv"], b2["dv"])
    assert torch.equal(b1["dq"], b2["dq"])
    assert torch.equal(b1["row_tiles"], b2["row_tiles"])
    assert torch.equal(r1["row_tiles"], r2["row_tiles"])


@pytest.mark.parametrize("name,tau,Nq", [("gqa_d128_ragged", 0.1, None), ("local_d64_ragged", 0.3, None),
                                         ("tiny_d128", 1e-3, None), ("split_d64_b2", 1e-3, None),
                                         ("lm_d128_ragged", 1.0, None), ("gqa_d128_ragged", 0.05, 77)])
def test_statistics_leave_outputs_unchanged(name, tau, Nq):
    # The optional statistics (row tile counts, counters) take work of their own in
    # the kernels (the key-major pass re-runs the offline test on its tiles only when
    # counters are requested, and masks the scores without it otherwise): the
    # outputs are the same bits either way (also for a prefill of the last Nq rows).
    w, q, k, v, do = _train_case(name, tau, Nq=Nq)
    Q, K, V, DO = map(dev, (q, k, v, do))
    s = f32(w.scale)
    f1 = mala.fwd(Q, K, V, s, tau)
    f0 = mala.fwd(Q, K, V, s, tau, stats=False)
    b1 = mala.bwd(Q, K, V, f1["o"], f1["lse"], DO, s, tau)
    b0 = mala.bwd(Q, K, V, f1["o"], f1["lse"], DO, s, tau, stats=False)
    torch.cuda.synchronize()
    assert torch.equal(f1["o"], f0["o"]) and torch.equal(f1["lse"], f0["lse"])
    for x in ("dq", "dk", "dv"):
        assert torch.equal(b1[x], b0[x]), x


@pytest.mark.parametrize("name", ["gqa_d128_ragged", "split_d64_b2"])
def test_graph_capture_replays_match_eager(name):
    # The library only launches kernels on the caller's stream (counters are
    # cleared by a kernel, not by hipMemsetAsync, and nothing is allocated), so a
    # fwd + bwd + decode step captured in a HIP graph replays to the eager results;
    # every replay is checked, with eager work on the outputs in between (the second
    # case runs the split key-block sweeps and their reduction pass).
    tau = 1e-3
    w, q, k, v, do = _train_case(name, tau)
    Q, K, V, DO = map(dev, (q, k, v, do))
    scale = f32(w.scale)
    B, Hq, N, D = Q.shape
    Hkv = K.shape[1]
    f = dict(dtype=torch.float32, device="cuda")
    i32 = dict(dtype=torch.int32, device="cuda")
    o, lse = torch.empty((B, Hq, N, D), **f), torch.empty((B, Hq, N), **f)
    dq = torch.empty_like(o)
    dk, dv = torch.empty((B, Hkv, N, D), **f), torch.empty((B, Hkv, N, D), **f)
    rt, rtb = torch.empty((B, Hq, N), **i32), torch.empty((B, Hq, N), **i32)
    cf, cb, cd = (torch.empty(mala.NUM_COUNTERS, dtype=torch.int64, device="cuda")
                  for _ in range(3))
    ws = torch.empty(mala.mala_bwd_workspace_size(B, Hq, Hkv, N, N, D), dtype=torch.uint8,
                     device="cuda")
    wd = Workload(dict(kind="decode", B=2, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4))
    td = wd.tensors()
    qd, kd, vd = dev(td["q"]), dev(td["k"]), dev(td["v"])
    S = 4
    od, lsed = torch.empty((2, 8, 128), **f), torch.empty((2, 8), **f)
    ht = torch.empty((2, 8), **i32)
    wsd = torch.empty(mala.mala_decode_workspace_size(2, 8, 128, S), dtype=torch.uint8,
                      device="cuda")
    lens = torch.tensor([3001, 1000], **i32)

    def step():
        mala.mala_fwd(Q, K, V, o, lse, rt, cf, scale, tau)
        mala.mala_bwd(Q, K, V, o, lse, DO, dq, dk, dv, rtb, cb, ws, scale, tau)
        mala.mala_decode(qd, kd, vd, od, lsed, ht, cd, S, wsd, f32(wd.scale), tau,
                         cache_lens=lens)

    outs = (o, lse, rt, cf, dq, dk, dv, rtb, cb, od, lsed, ht, cd)
    step()
    torch.cuda.synchronize()
    ref = [x.clone() for x in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):     # warm-up on a side stream before capture
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for i in range(3):
        for x in outs:
            x.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert torch.equal(a, b), i


@pytest.mark.parametrize("tau", [0.0, 1e-3])
def test_bf16_outputs(tau):
    # O and the gradients stored as bf16 are the fp32 results rounded once at the
    # store (bit for bit); with a bf16 O in D_q = rowsum(O * dO), the gradients meet
    # the bar against the oracle's backward from that same O, and the bf16-stored
    # ones within the bar plus one bf16 rounding
    w, q, k, v, do = _train_case("gqa_d128_ragged", tau)
    Q, K, V, DO = map(dev, (q, k, v, do))
    scale = f32(w.scale)
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    of32 = mala.fwd(Q, K, V, scale, tau)
    ob16 = mala.fwd(Q, K, V, scale, tau, out_dtype=torch.bfloat16)
    gf = mala.bwd(Q, K, V, ob16["o"], ob16["lse"], DO, scale, tau)
    gb = mala.bwd(Q, K, V, ob16["o"], ob16["lse"], DO, scale, tau, grad_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(ob16["o"], of32["o"].to(torch.bfloat16))
    assert torch.equal(ob16["lse"], of32["lse"])
    assert torch.equal(ob16["row_tiles"], of32["row_tiles"])
    for x in ("dq", "dk", "dv"):
        assert torch.equal(gb[x], gf[x].to(torch.bfloat16)), x
    assert torch.equal(gb["row_tiles"], gf["row_tiles"])
    qf, kf, vf, dof = map(bf16_to_f64, (q, k, v, do))
    ofr = oracle.mala_fwd(qf, kf, vf, scale, f32(tau), bq, bk)
    o16 = host(ob16["o"].float())
    obr = oracle.mala_bwd(qf, kf, vf, o16, ofr["lse"], dof, scale, f32(tau), bq, bk)
    rounded = {"O": (o16, ofr["o"])}
    for x, name in (("dq", "dQ"), ("dk", "dK"), ("dv", "dV")):
        assert_close(name + " (bf16 O)", host(gf[x]), obr[x])
        rounded[name] = (host(gb[x].float()), obr[x])
    for name, (got, ref) in rounded.items():
        err = np.abs(got - ref) - 2.0 ** -8 * np.abs(ref)
        assert err.max() <= TOL_MAX, (name, float(err.max()))


@pytest.mark.parametrize("tau", [1e-3, 1.0])
def test_bf16_gradients_with_split_sweeps(tau):
    # split key-block sweeps: the parts' fp32 sums are added by the reduction pass,
    # which rounds once at the store, so bf16 dK / dV are the fp32 ones rounded
    w, q, k, v, do = _train_case("split_d64_b2", tau)
    assert dkdv_splits(2, 8, 1, 6000)
    Q, K, V, DO = map(dev, (q, k, v, do))
    scale = f32(w.scale)
    f = mala.fwd(Q, K, V, scale, tau)
    gf = mala.bwd(Q, K, V, f["o"], f["lse"], DO, scale, tau)
    gb = mala.bwd(Q, K, V, f["o"], f["lse"], DO, scale, tau, grad_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    for x in ("dq", "dk", "dv"):
        assert torch.equal(gb[x], gf[x].to(torch.bfloat16)), x


def test_decode_bf16_output():
    spec = dict(kind="decode", B=2, Hq=8, Hkv=2, N=3001, D=128, beta=3.0, needles=4)
    w = Workload(spec)
    t = w.tensors()
    q, k, v = dev(t["q"]), dev(t["k"]), dev(t["v"])
    a = mala.decode(q, k, v, f32(w.scale), 1e-4, 4)
    b = mala.decode(q, k, v, f32(w.scale), 1e-4, 4, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(b["o"], a["o"].to(torch.bfloat16)) and torch.equal(b["lse"], a["lse"])


def test_concurrent_streams_match_sequential():
    # the library keeps no device state between calls: two forward + backward calls
    # on two streams at once give the results of the calls run one after the other
    tau = 1e-3
    cases = [_train_case("gqa_d128_ragged", tau), _train_case("local_d64_ragged", tau)]
    dev_in = [tuple(map(dev, c[1:])) + (f32(c[0].scale),) for c in cases]

    def run(Q, K, V, DO, scale):
        f = mala.fwd(Q, K, V, scale, tau)
        b = mala.bwd(Q, K, V, f["o"], f["lse"], DO, scale, tau)
        return [f["o"], f["lse"], f["row_tiles"], b["dq"], b["dk"], b["dv"], b["row_tiles"]]

    ref = [run(*a) for a in dev_in]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [None, None]
    for i in range(2):
        streams[i].wait_stream(torch.cuda.current_stream())
    for i, (s, a) in enumerate(zip(streams, dev_in)):
        with torch.cuda.stream(s):
            outs[i] = run(*a)
    torch.cuda.synchronize()
    for r, o in zip(ref, outs):
        for x, y in zip(r, o):
            assert torch.equal(x, y)

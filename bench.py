"""Benchmark of the MALA hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input:
  mala_fwd + mala_bwd on the 131072-token causal workload (one tensor-parallel
  share: batch 1, 8 query heads, 2 KV heads, head_dim 128, tau = 1e-4), then
  mala_decode of 16 one-token queries over 131072-token KV caches (32 query
  heads, 8 KV heads, tau = 1e-4).
Inputs are resident in HBM before the timed region; outputs and workspaces are
preallocated.  The same kernels at tau = 0 (dense attention) and the
32768-token GQA 32/8 workload are timed as well, because the metric asks for
the speed-up over dense at 32K and 128K.

Prints ONE JSON line (rank 0, N = 1).  More than one GPU is not supported.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MALA fwd/bwd ms + speedup vs dense at 32K/128K; decode ms; retained-tile %"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


class Train:
    """Device-resident inputs, outputs and workspace of one fwd+bwd workload."""

    def __init__(self, name, tau, **over):
        import torch
        import paper_2609_32712_amd as mala
        from workloads import Workload
        self.w = Workload(name, **over)
        self.tau = tau
        t0 = time.time()
        t = self.w.tensors(threads=16)
        log("%s %s inputs generated in %.1fs" % (name, over or "", time.time() - t0))
        dev = lambda b: torch.from_numpy(b.view(np.int16)).to("cuda").view(torch.bfloat16)
        self.q, self.k, self.v, self.do = (dev(t[x]) for x in ("q", "k", "v", "do"))
        del t
        w = self.w
        f = dict(dtype=torch.float32, device="cuda")
        self.o = torch.empty((w.B, w.Hq, w.N, w.D), **f)
        self.lse = torch.empty((w.B, w.Hq, w.N), **f)
        self.dq = torch.empty((w.B, w.Hq, w.N, w.D), **f)
        self.dk = torch.empty((w.B, w.Hkv, w.N, w.D), **f)
        self.dv = torch.empty((w.B, w.Hkv, w.N, w.D), **f)
        i32 = dict(dtype=torch.int32, device="cuda")
        self.rt_f = torch.empty((w.B, w.Hq, w.N), **i32)
        self.rt_b = torch.empty((w.B, w.Hq, w.N), **i32)
        self.cnt_f = torch.empty(mala.NUM_COUNTERS, dtype=torch.int64, device="cuda")
        self.cnt_b = torch.empty(mala.NUM_COUNTERS, dtype=torch.int64, device="cuda")
        n = mala.mala_bwd_workspace_size(w.B, w.Hq, w.Hkv, w.N, w.N, w.D)
        self.ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        self.scale = float(np.float32(w.scale))
        self.mala = mala

    # The timed calls leave out the optional statistics (per-row tile counts and the
    # counters); stats() repeats the fwd + bwd pair with them, which takes exactly the
    # same decisions.
    def fwd(self, tau, stats=False):
        self.mala.mala_fwd(self.q, self.k, self.v, self.o, self.lse,
                           self.rt_f if stats else None, self.cnt_f if stats else None,
                           self.scale, tau)

    def bwd(self, tau, stats=False):
        self.mala.mala_bwd(self.q, self.k, self.v, self.o, self.lse, self.do, self.dq, self.dk,
                           self.dv, self.rt_b if stats else None, self.cnt_b if stats else None,
                           self.ws, self.scale, tau)

    def stats(self, tau):
        """The counters of one fwd + bwd pair at tau (with the statistics on)."""
        self.fwd(tau, True)
        self.bwd(tau, True)
        return self.counters()

    def counters(self):
        return self.cnt_f.cpu().numpy(), self.cnt_b.cpu().numpy()

    def outputs(self):
        return {k: getattr(self, k).clone() for k in ("o", "lse", "dq", "dk", "dv")}


class Decode:
    def __init__(self, name, tau, splits=None):
        import torch
        import paper_2609_32712_amd as mala
        from workloads import Workload
        self.w = Workload(name)
        t0 = time.time()
        t = self.w.tensors(threads=16)
        log("%s inputs generated in %.1fs" % (name, time.time() - t0))
        dev = lambda b: torch.from_numpy(b.view(np.int16)).to("cuda").view(torch.bfloat16)
        self.q, self.k, self.v = (dev(t[x]) for x in ("q", "k", "v"))
        del t
        w = self.w
        self.splits = splits or mala.default_num_splits(w.B, w.Hkv, w.N)
        self.o = torch.empty((w.B, w.Hq, w.D), dtype=torch.float32, device="cuda")
        self.lse = torch.empty((w.B, w.Hq), dtype=torch.float32, device="cuda")
        self.ht = torch.empty((w.B, w.Hq), dtype=torch.int32, device="cuda")
        self.cnt = torch.empty(mala.NUM_COUNTERS, dtype=torch.int64, device="cuda")
        n = mala.mala_decode_workspace_size(w.B, w.Hq, w.D, self.splits)
        self.ws = torch.empty(n, dtype=torch.uint8, device="cuda")
        self.scale = float(np.float32(w.scale))
        self.mala = mala

    def run(self, tau, cache_lens=None, stats=False):
        self.mala.mala_decode(self.q, self.k, self.v, self.o, self.lse,
                              self.ht if stats else None, self.cnt if stats else None,
                              self.splits, self.ws, self.scale, tau, cache_lens=cache_lens)

    def stats(self, tau, cache_lens=None):
        """The counters of one decode call at tau (with the statistics on)."""
        self.run(tau, cache_lens, True)
        return self.cnt.cpu().numpy()


def ragged_lengths(B, N, seed=7):
    """Valid cache lengths of a serving batch: uniform on [1, N], the first sequence
    full and the second holding one token."""
    lens = np.random.default_rng(seed).integers(1, N + 1, size=B).astype(np.int32)
    lens[0] = N
    if B > 1:
        lens[1] = 1
    return lens


MIN_WARM_MS = 50.0   # --min-warm-ms


def time_calls(fn, reps, warmup, min_warm_ms=None):
    """Mean and median per-call device time (ms) from HIP events on the current stream.
    The untimed calls run until both `warmup` calls and `min_warm_ms` of wall time have
    passed: a few calls of a sub-millisecond kernel leave the GPU at its idle clock,
    and the first timed calls of such a kernel then run ~10% slow."""
    import torch
    min_warm_ms = MIN_WARM_MS if min_warm_ms is None else min_warm_ms
    t0 = time.time()
    n = 0
    while n < warmup or (time.time() - t0) * 1e3 < min_warm_ms:
        fn()
        n += 1
        if n >= warmup:
            torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    ts = [a.elapsed_time(b) for a, b in ev]
    return float(np.mean(ts)), float(np.median(ts))


def train_flops(cnt_f, cnt_b, D, bq, bk):
    """Algorithmic flops of one fwd and one bwd launch at tile granularity:
    2*d per legal QK slot (score discovery), plus 2*d (fwd PV) or 8*d (bwd dP, dV,
    dK, dQ) per retained slot."""
    slots = bq * bk
    fwd = (cnt_f[0] + cnt_f[1]) * slots * 2 * D
    bwd = (cnt_b[0] * 2 + cnt_b[1] * 8) * slots * D
    return float(fwd), float(bwd)


def dense_do_tiles(B, Hq, Hkv, N, bq=32, bwd_keys=128):
    """The dO tiles the key-major backward pass would load if it retained every tile
    (N_q = N_k = N): a workgroup of bwd_keys keys of one KV head visits every query
    tile of its GQA group's heads from its own first key on.  The denominator of the
    loaded percentage."""
    d = 0
    for k0 in range(0, N, bwd_keys):
        d += (N + bq - 1) // bq - k0 // bq
    return B * Hkv * (Hq // Hkv) * d


def cpu_model():
    """The host CPU's model name (first processor in /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.lower().startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def operator_memory(tr, tau):
    """Device memory (MiB) that one call of each allocating wrapper takes beyond the
    inputs already resident: torch.cuda.max_memory_allocated around the call minus
    the memory allocated before it.  That is the call's outputs and workspace; the
    library itself allocates nothing."""
    import torch
    mala = tr.mala
    mib = lambda x: round(x / 2 ** 20, 2)

    def peak(fn):
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        out = fn()
        torch.cuda.synchronize()
        return out, torch.cuda.max_memory_allocated() - base

    res = {}
    for name, dt in (("fp32_outputs", torch.float32), ("bf16_outputs", torch.bfloat16)):
        f, mf = peak(lambda: mala.fwd(tr.q, tr.k, tr.v, tr.scale, tau, out_dtype=dt))
        b, mb = peak(lambda: mala.bwd(tr.q, tr.k, tr.v, f["o"], f["lse"], tr.do, tr.scale, tau,
                                      grad_dtype=dt))
        res[name] = {"fwd_mib": mib(mf), "bwd_mib": mib(mb)}
        del f, b
    torch.cuda.empty_cache()
    return res


def time_train(tr, taus, timing):
    """fwd and bwd latencies of a Train at each tau, grouped by operator: first every
    forward series, then every backward series (each after an untimed forward at its
    tau, whose O and LSE it takes), so that each series follows the same kind of work
    (a series timed right after seconds of another operator ran at a lower clock).
    timing(tau) gives (reps, warmup).  Returns {tau: (fwd, bwd, cf, cb)}."""
    fw = {t_: time_calls(lambda: tr.fwd(t_), *timing(t_)) for t_ in taus}
    out = {}
    for t_ in taus:
        tr.fwd(t_)
        b = time_calls(lambda: tr.bwd(t_), *timing(t_))
        out[t_] = (fw[t_], b) + tuple(tr.stats(t_))
    return out


def train_workload(name, taus, reps, warmup, supp_taus=(), supp=None, memory=True):
    """One training workload: fwd / bwd latency (HIP events, mean and median of reps
    calls after warmup) at tau = 0 (dense through the same kernels) and at each tau,
    the speed-ups over dense, the retained work and the V / dO loads the retained
    tiles needed, executed and dense-equivalent TFLOP/s, and the operators' device
    memory."""
    import torch
    from workloads import WORKLOADS
    tr = Train(name, 0.0)
    w = tr.w
    mala = tr.mala
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    de_f, de_b = dense_equivalent_flops(w.B, w.Hq, w.N, w.D)
    rows = w.B * w.Hq * w.N
    pct = lambda a, b_: round(100.0 * float(a) / max(1.0, float(b_)), 3)
    do_dense = dense_do_tiles(w.B, w.Hq, w.Hkv, w.N)
    res = time_train(tr, (0.0,) + tuple(x for x in taus if x != 0.0),
                     lambda t_: supp if t_ in supp_taus else (reps, warmup))
    out = {"workload": WORKLOADS[name]["desc"], "shape": [w.B, w.Hq, w.Hkv, w.N, w.D]}
    f0, b0 = res[0.0][0][0], res[0.0][1][0]
    for t_, (f, b, cf, cb) in res.items():
        fl_f, fl_b = train_flops(cf, cb, w.D, bq, bk)
        out["tau=%g" % t_ + (" (supplementary)" if t_ in supp_taus else "")] = {
            "fwd_ms": round(f[0], 4), "fwd_ms_median": round(f[1], 4),
            "bwd_ms": round(b[0], 4), "bwd_ms_median": round(b[1], 4),
            "speedup_fwd": round(f0 / f[0], 4), "speedup_bwd": round(b0 / b[0], 4),
            "retained_tiles_pct_fwd": pct(cf[1], cf[0]),
            "retained_tiles_pct_bwd": pct(cb[1], cb[0]),
            "v_tiles_needed_pct_fwd": pct(cf[5], cf[2]),
            "do_tiles_loaded_pct_bwd": pct(cb[2], do_dense),
            "mean_slots_per_query_fwd": round(float(cf[3]) / rows, 1),
            "mean_slots_per_query_bwd": round(float(cb[3]) / rows, 1),
            "executed_tflops_fwd": round(fl_f / (f[0] * 1e-3) / 1e12, 1),
            "executed_tflops_bwd": round(fl_b / (b[0] * 1e-3) / 1e12, 1),
            "dense_equiv_tflops_fwd": round(de_f / (f[0] * 1e-3) / 1e12, 1),
            "dense_equiv_tflops_bwd": round(de_b / (b[0] * 1e-3) / 1e12, 1),
        }
    if memory:
        out["operator_memory"] = operator_memory(tr, taus[0])
    log("%s dense fwd %.3f bwd %.3f ms | %s" % (
        name, f0, b0, " ".join("tau=%g fwd %.3f bwd %.3f" % (t_, r[0][0], r[1][0])
                                 for t_, r in res.items() if t_)))
    del tr, res
    torch.cuda.empty_cache()
    return out


def dense_equivalent_flops(B, Hq, N, D):
    pairs = B * Hq * N * (N + 1) / 2
    return pairs * 4 * D, pairs * 10 * D


def head_fidelity(ref, out):
    """Operator fidelity of one run against the screening-disabled run (tau = 0) of
    the same operator on the same inputs, per head, following the operator-fidelity
    protocol of the experiments section and its appendix:
      * relative L2 error ||X - X_ref|| / ||X_ref|| of O and dQ per query head and of
        dK and dV per KV head (the norms run over one head's N x d block);
      * the dense softmax mass omitted by each query row, recovered from the two
        normalizers as 1 - exp(lse - lse_ref) (Z_R / (Z_R + Z_O) = exp(lse - lse_ref)),
        averaged over the rows of each query head; also the largest row value.
    ref, out: dicts of tensors o, dq [B, Hq, N, d], dk, dv [B, Hkv, N, d], lse [B, Hq, N]
    (any device).  Returns numpy arrays (fractions, not percent)."""
    import torch

    def rel(k):
        a, b = ref[k].double(), out[k].double()
        num = torch.linalg.vector_norm((b - a).flatten(2), dim=2)
        den = torch.linalg.vector_norm(a.flatten(2), dim=2)
        return (num / den).flatten().cpu().numpy()

    eps = omitted_mass_rows(ref["lse"], out["lse"])
    res = {k: rel(k) for k in ("o", "dq", "dk", "dv")}
    res["omitted_mass"] = eps.mean(dim=2).flatten().cpu().numpy()
    res["omitted_mass_row_max"] = float(eps.max())
    return res


def omitted_mass_rows(lse_ref, lse):
    """Dense softmax mass a row omits, from the screened and the screening-disabled
    normalizers: 1 - Z_R / (Z_R + Z_O) = -expm1(lse - lse_ref), in float64."""
    import torch
    return -torch.expm1(lse.double() - lse_ref.double())


def mean_p95(x):
    """Mean and 95th percentile (linear interpolation) over head-level measurements."""
    x = np.asarray(x, dtype=np.float64)
    return float(x.mean()), float(np.percentile(x, 95))


LM_SWEEP_N = (1024, 2048, 4096, 8192, 16384, 32768)
LM_SWEEP_TOKENS = 32768        # batch = tokens / N, so every length has the same token count
LM_SWEEP_TAUS = (1e-4, 1.0)


def lm_sweep(reps, warmup, lengths=LM_SWEEP_N):
    """The language-model-like workload (8 query / 2 KV heads, head_dim 128) at context
    lengths 1K..32K: fwd/bwd time and retained work at tau = 0, 1e-4 and the canonical
    tau = 1, and the operator fidelity of tau > 0 against tau = 0 (same kernels)."""
    import torch
    rows = []
    for N in lengths:
        tr = Train("lm_like_gqa8x2_32k", 0.0, N=N, B=max(1, LM_SWEEP_TOKENS // N))
        w = tr.w
        nrows = w.B * w.Hq * w.N
        runs = {}
        for t_, (f, b, cf, cb) in time_train(tr, (0.0,) + LM_SWEEP_TAUS,
                                             lambda t_: (reps, warmup)).items():
            tr.stats(t_)   # the outputs at t_ for the fidelity figures
            runs[t_] = dict(fwd=f[0], bwd=b[0], cf=cf, cb=cb, out=tr.outputs())
        d = runs[0.0]
        row = {"N": N, "batch": w.B, "q_heads": w.B * w.Hq, "kv_heads": w.B * w.Hkv,
               "dense_fwd_ms": round(d["fwd"], 4), "dense_bwd_ms": round(d["bwd"], 4)}
        for t_ in LM_SWEEP_TAUS:
            r = runs[t_]
            fid = head_fidelity(d["out"], r["out"])
            pc = lambda x: [round(100 * v, 5) for v in mean_p95(x)]
            row["tau=%g" % t_] = {
                "fwd_ms": round(r["fwd"], 4), "bwd_ms": round(r["bwd"], 4),
                "speedup_fwd": round(d["fwd"] / r["fwd"], 4),
                "speedup_bwd": round(d["bwd"] / r["bwd"], 4),
                "retained_tiles_pct_fwd": round(100.0 * r["cf"][1] / r["cf"][0], 3),
                "retained_tiles_pct_bwd": round(100.0 * r["cb"][1] / r["cb"][0], 3),
                "mean_slots_per_query_fwd": round(float(r["cf"][3]) / nrows, 1),
                "mean_slots_per_query_bwd": round(float(r["cb"][3]) / nrows, 1),
                "omitted_mass_pct_mean_p95": pc(fid["omitted_mass"]),
                "omitted_mass_pct_row_max": round(100 * fid["omitted_mass_row_max"], 5),
                "rel_l2_pct_mean_p95": {k: pc(fid[k]) for k in ("o", "dq", "dk", "dv")},
            }
        log("lm N=%d B=%d dense fwd %.3f bwd %.3f | tau=1 fwd %.3f bwd %.3f ms" % (
            N, w.B, d["fwd"], d["bwd"], runs[1.0]["fwd"], runs[1.0]["bwd"]))
        rows.append(row)
        del tr, runs, d
        torch.cuda.empty_cache()
    return rows


def mfma_probe(reps=5, blocks=256 * 12, iters=4096):
    """The bf16 MFMA rate this machine sustains under a pure MFMA load: libmala_probe.so
    runs chains of v_mfma_f32_32x32x16_bf16 with operands in registers and no memory
    traffic (three wavefronts per SIMD, 256 x 12 workgroups of four), timed with HIP
    events on the current stream; the implied clock is the rate over 1024 flops per
    SIMD per cycle (32x32x16 x 2 flops in 32 cycles) x 1024 SIMDs.  Context for the
    machine's power state, not the roofline's peak.  None if the probe is not built."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_2609_32712_amd", "libmala_probe.so")
    if not os.path.exists(path):
        return None
    lib = ctypes.CDLL(path)
    lib.mala_probe_mfma.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    lib.mala_probe_mfma.restype = ctypes.c_int
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    run = lambda: lib.mala_probe_mfma(ctypes.c_void_p(out.data_ptr()), blocks, iters, st)
    if run() != 0:
        return None
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = float(np.median(times))
    flops = float(blocks) * 4 * iters * 4 * 32768     # waves x MFMAs x flops
    tflops = flops / (ms * 1e-3) / 1e12
    return {"tflops": round(tflops, 1), "frac_of_rated_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
            "implied_mfma_clock_ghz": round(tflops * 1e12 / (1024.0 * 1024.0) / 1e9, 3),
            "ms": round(ms, 3),
            "note": "independent v_mfma_f32_32x32x16_bf16 chains, operands in registers, "
                    "no memory traffic, on every CU: the rate this machine sustains under a pure "
                    "MFMA load (its power management lowers the clock on some machines; the "
                    "attention kernels, at 38-54% MFMA issue, run at ~2.0-2.3 GHz)"}


def source_sha(path):
    with open(path, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


TRAFFIC_FILES = {"bwd": "mala_bwd_traffic_128k.json", "decode": "mala_decode_traffic_128k.json"}


def _traffic(which, kernel_src):
    p = os.path.join(ROOT, "profiles", TRAFFIC_FILES[which])
    if not os.path.exists(p):
        return None
    with open(p) as fh:
        d = json.load(fh)
    if d.get("source_sha") != source_sha(kernel_src):
        return None
    return float(d["bytes_per_launch"])


def traffic_from_profiles(kernel_src):
    """HBM bytes per launch of the backward operator from the committed rocprofv3
    counter summary (FETCH_SIZE and WRITE_SIZE, each scaled by what it reads for a
    plain copy), or None if the kernel source changed since the counters were taken."""
    return _traffic("bwd", kernel_src)


def decode_traffic_from_profiles(kernel_src):
    """HBM bytes per mala_decode call (split + merge kernels) from the committed
    counter summary, or None if the decode source changed since it was taken."""
    return _traffic("decode", kernel_src)


def cpu_baseline(step_ms_model):
    """Time the fp64 oracle on a bounded sample of the same step and scale it up by
    tile counts: the last nb query blocks of one head of the 131072-token workload
    (forward, then the backward's dQ sweep over those blocks), the backward's dK/dV
    sweep over the last nb key blocks (the rows that see them are exactly the rows
    of the sampled forward), and whole decode calls of a few query heads."""
    import oracle
    from workloads import Workload, bf16_to_f64
    import paper_2609_32712_amd as mala
    oracle.build()
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    w = Workload("gqa8x2_128k")
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)
    Tr = -(-w.N // bq)
    nb = min(Tr, 8 * cores)
    i0 = Tr - nb
    qf = bf16_to_f64(w.q_head(0, 0))[None, None]
    kf = bf16_to_f64(w.k_head(0, 0))[None, None]
    vf = bf16_to_f64(w.v_head(0, 0))[None, None]
    dof = bf16_to_f64(w.do_head(0, 0))[None, None]
    scale = float(np.float32(w.scale))
    tau = float(np.float32(1e-4))
    t0 = time.time()
    of = oracle.mala_fwd(qf, kf, vf, scale, tau, bq, bk, blocks=(i0, Tr), heads=[(0, 0)])
    t_f = time.time() - t0
    o_in, lse_in = np.nan_to_num(of["o"]), np.nan_to_num(of["lse"])
    t0 = time.time()
    oracle.mala_bwd(qf, kf, vf, o_in, lse_in, dof, scale, tau, bq, bk, qblocks=(i0, Tr),
                    kblocks=(0, 0))
    t_q = time.time() - t0
    t0 = time.time()
    oracle.mala_bwd(qf, kf, vf, o_in, lse_in, dof, scale, tau, bq, bk, qblocks=(0, 0),
                    kblocks=(i0, Tr))
    t_k = time.time() - t0
    # tiles: query block i sees i + 1 key tiles, key block j is seen by Tr - j query
    # tiles; the whole step has Hq * Tr (Tr + 1) / 2 of them on either side
    q_tiles = sum(i + 1 for i in range(i0, Tr))
    k_tiles = sum(Tr - j for j in range(i0, Tr))
    total_tiles = w.Hq * Tr * (Tr + 1) / 2
    ms_fwd = t_f * 1e3 * total_tiles / q_tiles
    ms_bwd = (t_q / q_tiles + t_k / k_tiles) * 1e3 * total_tiles
    wd = Workload("decode_gqa32x8_128k")
    sd = mala.default_num_splits(wd.B, wd.Hkv, wd.N)
    qd = bf16_to_f64(wd.q_head(0, 0))[None, None]
    kd = bf16_to_f64(wd.k_head(0, 0))[None, None]
    vd = bf16_to_f64(wd.v_head(0, 0))[None, None]
    t0 = time.time()
    nh = 8
    for h in range(nh):
        oracle.mala_decode(qd, kd, vd, scale, tau, mala.mala_geometry(wd.D, mala.PASS_DECODE)[1],
                           sd)
    t_d = (time.time() - t0) / nh
    ms_dec = t_d * 1e3 * wd.B * wd.Hq
    total = ms_fwd + ms_bwd + ms_dec
    return {"value": round(total, 1), "unit": "ms", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": ("fp64 C oracle (OpenMP) on head 0 of the 131072-token workload: forward "
                       "of the last %d query blocks %.1fs, dQ sweep of those blocks %.1fs, dK/dV "
                       "sweep of the last %d key blocks %.1fs, scaled by total / sampled tiles; "
                       "decode of %d query heads (%.2fs each, x%d heads); extrapolated to one "
                       "full step" % (nb, t_f, t_q, nb, t_k, nh, t_d, wd.B * wd.Hq)),
            "fwd_ms": round(ms_fwd, 1), "bwd_ms": round(ms_bwd, 1), "decode_ms": round(ms_dec, 1)}


COUNTER_CMD = ("cd /tmp && export TMPDIR=/tmp && timeout -s KILL 180 rocprofv3 --pmc {c} "
               "--output-format csv -d $OUT/pmc_{d} -o run -- "
               "python $REPO/bench.py --counter-pass")
TRACE_CMD = ("cd /tmp && export TMPDIR=/tmp && timeout -k 10 600 rocprofv3 --kernel-trace --stats "
             "--output-format csv -d $OUT/trace_bench -o bench -- "
             "python $REPO/bench.py --steps 2 --warmup 1 --reps 2 --kernel-warmup 1 "
             "--supp-reps 2 --supp-warmup 1 --no-cpu-baseline --no-32k --no-lm --no-ragged "
             "--no-small --no-memory --min-warm-ms 0 --no-stats-timing")


def counter_pass(which="bwd"):
    """The program the traffic counters are taken on: a plain 512 MiB device copy
    (the calibration kernel), then two mala_fwd + mala_bwd calls of the 131072-token
    workload (which = "bwd") or two mala_decode calls of the 16 x 131072-token decode
    workload (which = "decode"), tau = 1e-4."""
    import torch
    import paper_2609_32712_amd as mala
    mala.load_library()
    x = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    x.fill_(1)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    del x, y
    if which == "decode":
        dec = Decode("decode_gqa32x8_128k", 1e-4)
        for _ in range(2):
            dec.run(1e-4)
    else:
        tr = Train("gqa8x2_128k", 1e-4)
        for _ in range(2):
            tr.fwd(1e-4)
            tr.bwd(1e-4)
    torch.cuda.synchronize()
    log("counter pass done")


SKIP_TAUS = (0.0, 1.0, 1e30)
SKIP_TRACE_CMD = ("cd /tmp && export TMPDIR=/tmp && timeout -k 10 300 rocprofv3 --kernel-trace "
                  "--stats --output-format csv -d $OUT/trace_skip -o skip -- "
                  "python $REPO/bench.py --skip-pass")


def skip_pass():
    """The program of the skip-cost trace: the 32768-token language-model-like
    workload (8 query / 2 KV heads), three mala_fwd + mala_bwd calls at each of
    tau = 0 (dense), 1 (the canonical tolerance) and 1e30 (every backward tile and
    every forward tile but a row's first skipped: the cost floor of the skip path)."""
    import torch
    import paper_2609_32712_amd as mala
    mala.load_library()
    tr = Train("lm_like_gqa8x2_32k", 0.0)
    for tau in SKIP_TAUS:
        for _ in range(3):
            tr.fwd(tau)
            tr.bwd(tau)
        cf, cb = tr.stats(tau)   # a fourth call, with the statistics
        torch.cuda.synchronize()
        log("tau %g: retained tiles fwd %.2f%% bwd %.2f%%" % (
            tau, 100.0 * cf[1] / cf[0], 100.0 * cb[1] / cb[0]))


def summarize_skip_trace(trace_csv):
    """profiles/kernels_lm32k_skip_cost.md from the kernel trace of SKIP_TRACE_CMD
    (every training kernel has 4 dispatches per tau, in the order of SKIP_TAUS: 3
    without the statistics, then 1 with them)."""
    import csv
    import collections
    with open(trace_csv) as fh:
        rows = list(csv.DictReader(fh))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = collections.defaultdict(list)
    for r in rows:
        if "mala_" in r["Kernel_Name"] and "fill_zero" not in r["Kernel_Name"]:
            dur[r["Kernel_Name"]].append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6)
    lines = ["# Cost of skipped tiles: the 32768-token language-model-like workload", "",
             "Command (run from the repository root on one MI355X; `$REPO` is that root, "
             "`$OUT` an output directory):", "",
             "```", SKIP_TRACE_CMD, "python bench.py --summarize-skip-trace "
             "$OUT/trace_skip/skip_kernel_trace.csv", "```", "",
             "Mean kernel durations (ms) over 3 calls per tau (without the optional "
             "statistics).  tau = 1e30 skips every "
             "backward tile and every forward tile but each row's first (the cost floor of "
             "the skip path: score MFMAs, the test, staging and synchronisation); the last "
             "column is that floor as a fraction of the dense time.", "",
             "| kernel | tau 0 (dense) | tau 1 | tau 1e30 (all skipped) | floor / dense |",
             "|---|---|---|---|---|"]
    for k, v in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        # per tau: 3 calls without the statistics, then the one with them (left out)
        if len(v) != 4 * len(SKIP_TAUS):
            lines.append("| `%s` | %d dispatches (unexpected) | | | |" % (k, len(v)))
            continue
        m = [sum(v[4 * i:4 * i + 3]) / 3 for i in range(len(SKIP_TAUS))]
        lines.append("| `%s` | %.3f | %.3f | %.3f | %.2f |" % (k.replace("|", "/"), m[0], m[1],
                                                               m[2], m[2] / m[0]))
    with open(os.path.join(ROOT, "profiles", "kernels_lm32k_skip_cost.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_means(path):
    """Per-kernel mean over dispatches of a rocprofv3 counter CSV (KiB for the
    *_SIZE counters); values of one dispatch are summed first."""
    import csv
    import collections
    per = collections.defaultdict(float)
    names = {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            per[r["Dispatch_Id"]] += float(r["Counter_Value"])
            names[r["Dispatch_Id"]] = r["Kernel_Name"]
    by = collections.defaultdict(list)
    for d, v in per.items():
        by[names[d]].append(v)
    return {k: sum(v) / len(v) for k, v in by.items()}


COUNTED = {
    "bwd": dict(prefix="mala_bwd", src="mala_bwd.hip", flag="--counter-pass",
                summarize="--summarize-counters",
                workload="mala_bwd on the 131072-token share (8 q / 2 kv heads, d 128), tau 1e-4"),
    "decode": dict(prefix="mala_decode", src="mala_decode.hip", flag="--decode-counter-pass",
                   summarize="--summarize-decode-counters",
                   workload="mala_decode, 16 x 32 q / 8 kv heads over 131072-token caches, d 128, "
                            "tau 1e-4, 16 splits (split + merge kernels)"),
}


def summarize_counters(fetch_csv, write_csv, which="bwd"):
    """profiles/mala_<which>_traffic_128k.json: HBM bytes per launch of the backward
    operator (which = "bwd") or of a decode call ("decode") from the FETCH_SIZE and
    WRITE_SIZE passes, each scaled by what the counter reads for the 512 MiB copy of
    the same run."""
    c = COUNTED[which]
    f, w = _counter_means(fetch_csv), _counter_means(write_csv)
    copy = [k for k in f if "copy" in k.lower()]
    if not copy:
        raise SystemExit("no copy kernel in %s" % fetch_csv)
    copy = copy[0]
    kib = 512 * 1024
    fscale, wscale = round(kib / f[copy], 1), round(kib / w[copy], 1)
    kernels, total = {}, 0.0
    for k in sorted(f):
        if c["prefix"] in k or "mala_fill_zero" in k:
            b = (f[k] * fscale + w.get(k, 0.0) * wscale) * 1024
            if c["prefix"] in k:
                total += b
            kernels[k] = {"fetch_kib": f[k], "write_kib": w.get(k, 0.0), "bytes": b}
    cmd = COUNTER_CMD.replace("--counter-pass", c["flag"])
    out = {"source_sha": source_sha(os.path.join(ROOT, "paper_2609_32712_amd", "csrc", c["src"])),
           "bytes_per_launch": total, "fetch_scale": fscale, "write_scale": wscale,
           "kernels": kernels,
           "calibration": {"copy_kernel": copy, "copy_bytes": 512 << 20,
                           "copy_fetch_kib": f[copy], "copy_write_kib": w[copy]},
           "workload": c["workload"],
           "commands": [cmd.format(c="FETCH_SIZE", d="fetch"), cmd.format(c="WRITE_SIZE", d="write"),
                        "python bench.py %s $OUT/pmc_fetch/run_counter_collection.csv "
                        "$OUT/pmc_write/run_counter_collection.csv" % c["summarize"]]}
    with open(os.path.join(ROOT, "profiles", TRAFFIC_FILES[which]), "w") as fh:
        json.dump(out, fh, indent=1)
    print("%s HBM bytes per launch %.3f GB (fetch x%.1f, write x%.1f)"
          % (c["prefix"], total / 1e9, fscale, wscale))


def summarize_trace(trace_csv):
    """profiles/kernels_128k_train_and_decode.md from the rocprofv3 kernel trace of
    TRACE_CMD.  That run calls each operator 3 times at tau = 1e-4 (1 warm-up + 2
    timed steps), then 3 times at each of tau = 1e-4, 0 and 1 (1 warm-up + 2
    event-timed calls), so that dispatches 1-6, 7-9 and 10-12 of every kernel are those
    taus; the dispatches after them (the untimed forwards before the backward
    series, the calls with the statistics) are left out."""
    import csv
    import collections
    with open(trace_csv) as fh:
        rows = list(csv.DictReader(fh))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = collections.defaultdict(list)
    for r in rows:
        dur[r["Kernel_Name"]].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6)
    ms = lambda v: sum(v) / len(v) if v else float("nan")
    lines = ["# Kernel time of one bench run: 131072-token fwd + bwd and decode", "",
             "Command (run from the repository root on one MI355X; `$REPO` is that root, "
             "`$OUT` an output directory):", "",
             "```", TRACE_CMD, "python bench.py --summarize-trace "
             "$OUT/trace_bench/bench_kernel_trace.csv", "```", "",
             "Durations in milliseconds from the rocprofv3 kernel trace.  Dispatches 1-6 "
             "of each kernel are at tau = 1e-4 (the bench step and its event-timed calls), "
             "7-9 at tau = 0 (dense through the same kernels), 10-12 at tau = 1; the "
             "dispatches after them (the untimed forward before each backward series, one "
             "call per tau with the optional statistics) are left out of the means.", "",
             "| kernel | calls | mean ms, tau 1e-4 | mean ms, tau 0 | mean ms, tau 1 | total ms |",
             "|---|---|---|---|---|---|"]
    for k, v in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        n = len(v)
        if n in (15, 18):
            cells = (ms(v[:6]), ms(v[6:9]), ms(v[9:12]))
            lines.append("| `%s` | %d | %.3f | %.3f | %.3f | %.3f |"
                         % ((k.replace("|", "/"), n) + cells + (sum(v),)))
        else:
            lines.append("| `%s` | %d | %.3f (all) | | | %.3f |" % (k.replace("|", "/"), n, ms(v),
                                                                  sum(v)))
    with open(os.path.join(ROOT, "profiles", "kernels_128k_train_and_decode.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_mfma(csv_path):
    """profiles/mfma_util_128k.md from a `rocprofv3 --pmc MfmaUtil MfmaFlopsBF16` pass
    over --counter-pass (rocprofv3's derived counters: MFMA-busy SIMD cycles over
    active cycles x SIMDs, and executed bf16 MFMA flops)."""
    import csv
    import collections
    per = collections.defaultdict(dict)
    names = {}
    with open(csv_path) as fh:
        for r in csv.DictReader(fh):
            d = r["Dispatch_Id"]
            c = r["Counter_Name"]
            per[d][c] = per[d].get(c, 0.0) + float(r["Counter_Value"])
            names[d] = r["Kernel_Name"]
    by = collections.defaultdict(list)
    for d, v in per.items():
        if "mala" in names[d]:
            by[names[d]].append(v)
    cmd = COUNTER_CMD.format(c="MfmaUtil MfmaFlopsBF16", d="mfma")
    lines = ["# MFMA utilisation of the 131072-token fwd + bwd kernels", "",
             "Command (from the repository root on one MI355X; `$REPO` is that root, `$OUT` an "
             "output directory):", "",
             "```", cmd,
             "python bench.py --summarize-mfma $OUT/pmc_mfma/run_counter_collection.csv",
             "```", "",
             "`MfmaUtil` = MFMA-busy cycles summed over SIMDs / (active cycles x SIMDs), %; "
             "`MfmaFlopsBF16` = executed bf16 MFMA flops per dispatch (the hi/lo split and "
             "the dQ pass's recomputation included).  Mean over the dispatches of the run.", "",
             "| kernel | dispatches | MfmaUtil % | executed bf16 MFMA TFLOP per dispatch |",
             "|---|---|---|---|"]
    for k, vs in sorted(by.items()):
        u = sum(v.get("MfmaUtil", 0.0) for v in vs) / len(vs)
        f = sum(v.get("MfmaFlopsBF16", 0.0) for v in vs) / len(vs)
        lines.append("| `%s` | %d | %.1f | %.2f |" % (k.replace("|", "/"), len(vs), u, f / 1e12))
    with open(os.path.join(ROOT, "profiles", "mfma_util_128k.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_pipes(csv_path):
    """profiles/pipe_util_128k.md from a `rocprofv3 --pmc VALUBusy MfmaUtil LdsUtil`
    pass over --counter-pass: how busy each pipe of the CU is during each kernel
    (rocprofv3's derived counters, % of the kernel's active cycles)."""
    import csv
    import collections
    per = collections.defaultdict(dict)
    names = {}
    with open(csv_path) as fh:
        for r in csv.DictReader(fh):
            d = r["Dispatch_Id"]
            c = r["Counter_Name"]
            per[d][c] = per[d].get(c, 0.0) + float(r["Counter_Value"])
            names[d] = r["Kernel_Name"]
    by = collections.defaultdict(list)
    for d, v in per.items():
        if "mala" in names[d] and "fill_zero" not in names[d]:
            by[names[d]].append(v)
    cmd = COUNTER_CMD.format(c="VALUBusy MfmaUtil LdsUtil", d="pipes")
    lines = ["# Pipe utilisation of the 131072-token fwd + bwd kernels", "",
             "Command (from the repository root on one MI355X; `$REPO` is that root, `$OUT` an "
             "output directory):", "",
             "```", cmd,
             "python bench.py --summarize-pipes $OUT/pmc_pipes/run_counter_collection.csv",
             "```", "",
             "`VALUBusy` = cycles issuing vector-ALU instructions per CU / active cycles; "
             "`MfmaUtil` = MFMA-busy cycles per SIMD / active cycles; `LdsUtil` = cycles the "
             "LDS is active per CU / active cycles (all %, mean over the dispatches).", "",
             "| kernel | dispatches | VALUBusy % | MfmaUtil % | LdsUtil % |",
             "|---|---|---|---|---|"]
    for k, vs in sorted(by.items()):
        m = lambda c: sum(v.get(c, 0.0) for v in vs) / len(vs)
        lines.append("| `%s` | %d | %.1f | %.1f | %.1f |" % (k.replace("|", "/"), len(vs),
                                                          m("VALUBusy"), m("MfmaUtil"),
                                                          m("LdsUtil")))
    with open(os.path.join(ROOT, "profiles", "pipe_util_128k.md"), "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--tau", type=float, default=1e-4)
    ap.add_argument("--reps", type=int, default=100,
                    help="event-timed calls per kernel at the measured taus (the paper's 100)")
    ap.add_argument("--kernel-warmup", type=int, default=25,
                    help="untimed calls before them (the paper's 25)")
    ap.add_argument("--supp-reps", type=int, default=20,
                    help="event-timed calls per kernel for the supplementary fields")
    ap.add_argument("--supp-warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--min-warm-ms", type=float, default=50.0,
                    help="untimed calls before each event-timed series: at least this long")
    ap.add_argument("--no-stats-timing", action="store_true",
                    help="leave out the timing of the calls with the optional statistics")
    ap.add_argument("--no-32k", action="store_true")
    ap.add_argument("--no-small", action="store_true",
                    help="skip the 1024- and 8192-token workloads")
    ap.add_argument("--no-memory", action="store_true",
                    help="skip the per-call device memory measurement")
    ap.add_argument("--no-lm", action="store_true",
                    help="skip the language-model-like tau = 1 timing and fidelity sweep")
    ap.add_argument("--no-ragged", action="store_true",
                    help="skip the ragged-cache-length decode timing")
    ap.add_argument("--counter-pass", action="store_true",
                    help="run only the program profiled for the traffic counters")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--decode-counter-pass", action="store_true",
                    help="run only the decode program profiled for the traffic counters")
    ap.add_argument("--summarize-decode-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV")
    ap.add_argument("--skip-pass", action="store_true",
                    help="run only the program of the skip-cost trace")
    ap.add_argument("--summarize-skip-trace", metavar="KERNEL_TRACE_CSV")
    ap.add_argument("--summarize-mfma", metavar="COUNTER_CSV")
    ap.add_argument("--summarize-pipes", metavar="COUNTER_CSV")
    args = ap.parse_args()
    global MIN_WARM_MS
    MIN_WARM_MS = args.min_warm_ms
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return
    if args.summarize_decode_counters:
        summarize_counters(*args.summarize_decode_counters, which="decode")
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_skip_trace:
        summarize_skip_trace(args.summarize_skip_trace)
        return
    if args.summarize_mfma:
        summarize_mfma(args.summarize_mfma)
        return
    if args.summarize_pipes:
        summarize_pipes(args.summarize_pipes)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the MALA operator is built and measured on a "
              "single MI355X (heads and batch shard with no exchange; see the design notes).",
              file=sys.stderr)
        sys.exit(2)
    if args.counter_pass or args.decode_counter_pass:
        counter_pass("decode" if args.decode_counter_pass else "bwd")
        return
    if args.skip_pass:
        skip_pass()
        return
    import torch
    import paper_2609_32712_amd as mala
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    mala.load_library()
    tau = args.tau

    tr = Train("gqa8x2_128k", tau)
    dec = Decode("decode_gqa32x8_128k", tau)
    w = tr.w
    bq, bk = mala.mala_geometry(w.D, mala.PASS_FWD)

    def step():
        tr.fwd(tau)
        tr.bwd(tau)
        dec.run(tau)

    log("warmup")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("timed region: %d steps" % args.steps)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps

    # per-kernel event timings at tau, at tau = 0 (dense through the same kernels) and
    # at the paper's canonical tau = 1 (supplementary), grouped by operator: every
    # forward series, then every backward series (each after an untimed forward at
    # its tau), then every decode series, then one call each with the statistics
    sr, sw = args.supp_reps, args.supp_warmup
    series = (("tau", tau, args.reps, args.kernel_warmup),
              ("dense", 0.0, args.reps, args.kernel_warmup), ("tau1", 1.0, sr, sw))
    res = {name: {} for name, _, _, _ in series}
    for name, t_, n_, w_ in series:
        res[name]["fwd"] = time_calls(lambda: tr.fwd(t_), n_, w_)
    for name, t_, n_, w_ in series:
        tr.fwd(t_)
        res[name]["bwd"] = time_calls(lambda: tr.bwd(t_), n_, w_)
    for name, t_, n_, w_ in series:
        res[name]["dec"] = time_calls(lambda: dec.run(t_), n_, w_)
    for name, t_, _, _ in series:
        res[name]["cf"], res[name]["cb"] = tr.stats(t_)
        res[name]["cd"] = dec.stats(t_)
        log(name, "fwd %.2f bwd %.2f decode %.3f ms" % (res[name]["fwd"][0], res[name]["bwd"][0],
                                                        res[name]["dec"][0]))
    r1 = res.pop("tau1")
    f1, b1, d1, cf1, cb1, cd1 = (r1[x] for x in ("fwd", "bwd", "dec", "cf", "cb", "cd"))
    # the same calls with the optional statistics (per-row tile counts and counters)
    with_stats = None
    if not args.no_stats_timing:
        fs = time_calls(lambda: tr.fwd(tau, True), sr, sw)
        bs = time_calls(lambda: tr.bwd(tau, True), sr, sw)
        ds = time_calls(lambda: dec.run(tau, None, True), sr, sw)
        with_stats = {"note": "the 131072-token fwd / bwd and the decode at tau with row tile "
                              "counts and counters requested (the timed calls above leave "
                              "them out; the statistics come from one extra call each)",
                      "fwd_ms": round(fs[0], 3), "bwd_ms": round(bs[0], 3),
                      "decode_ms": round(ds[0], 4)}
    # supplementary: the same decode batch with ragged valid cache lengths
    ragged = None
    if not args.no_ragged:
        lens = ragged_lengths(dec.w.B, dec.w.N)
        cl = torch.from_numpy(lens).to("cuda")
        dr = time_calls(lambda: dec.run(tau, cl), sr, sw)
        cdr = dec.stats(tau, cl)
        drd = time_calls(lambda: dec.run(0.0, cl), sr, sw)
        # K of every valid key, V of the tiles fetched
        rag_bytes = (float(lens.sum()) * dec.w.Hkv * dec.w.D * 2
                     + float(cdr[mala.CNT_V_TILES]) * 32 * dec.w.D * 2)
        ragged = {
            "lens": "uniform on [1, %d], seed 7, first full, second 1 token; total %d"
                    % (dec.w.N, int(lens.sum())),
            "ms": round(dr[0], 4), "dense_ms": round(drd[0], 4),
            "speedup": round(drd[0] / dr[0], 4),
            "retained_head_tiles_pct": round(100.0 * cdr[1] / max(1, cdr[0]), 3),
            "hbm_gbs_algorithmic": round(rag_bytes / (dr[0] * 1e-3) / 1e9, 1),
        }
    rt, rd = res["tau"], res["dense"]
    fl_f, fl_b = train_flops(rt["cf"], rt["cb"], w.D, bq, bk)
    de_f, de_b = dense_equivalent_flops(w.B, w.Hq, w.N, w.D)
    bwd_ms = rt["bwd"][0]
    achieved = fl_b / (bwd_ms * 1e-3) / 1e12
    cd = rt["cd"]
    dw = dec.w
    tile_bytes = mala.mala_geometry(dw.D, mala.PASS_DECODE)[1] * dw.D * 2
    # K tiles read (one per decode wavefront and tile: nchunk wavefronts per KV head)
    k_tiles = dw.B * dw.Hkv * (-(-dw.g // 16)) * (-(-dw.N // mala.mala_geometry(dw.D, 2)[1]))
    dec_bytes = (k_tiles + cd[mala.CNT_V_TILES]) * tile_bytes
    dec_traffic = decode_traffic_from_profiles(
        os.path.join(ROOT, "paper_2609_32712_amd", "csrc", "mala_decode.hip"))
    pct = lambda a, b_: round(100.0 * float(a) / max(1.0, float(b_)), 3)
    do_dense = dense_do_tiles(w.B, w.Hq, w.Hkv, w.N)

    detail = {
        "128k": {
            "fwd_ms": round(rt["fwd"][0], 3), "fwd_ms_median": round(rt["fwd"][1], 3),
            "bwd_ms": round(rt["bwd"][0], 3), "bwd_ms_median": round(rt["bwd"][1], 3),
            "dense_fwd_ms": round(rd["fwd"][0], 3), "dense_bwd_ms": round(rd["bwd"][0], 3),
            "speedup_fwd": round(rd["fwd"][0] / rt["fwd"][0], 4),
            "speedup_bwd": round(rd["bwd"][0] / rt["bwd"][0], 4),
            "retained_tiles_pct_fwd": pct(rt["cf"][1], rt["cf"][0]),
            "retained_tiles_pct_bwd": pct(rt["cb"][1], rt["cb"][0]),
            "v_tiles_needed_pct_fwd": pct(rt["cf"][5], rt["cf"][2]),
            "do_tiles_loaded_pct_bwd": pct(rt["cb"][2], do_dense),
            "mean_slots_per_query_fwd": round(float(rt["cf"][3]) / (w.B * w.Hq * w.N), 1),
            "mean_slots_per_query_bwd": round(float(rt["cb"][3]) / (w.B * w.Hq * w.N), 1),
            "executed_tflops_fwd": round(fl_f / (rt["fwd"][0] * 1e-3) / 1e12, 1),
            "executed_tflops_bwd": round(achieved, 1),
            "dense_equiv_tflops_fwd": round(de_f / (rt["fwd"][0] * 1e-3) / 1e12, 1),
            "dense_equiv_tflops_bwd": round(de_b / (rt["bwd"][0] * 1e-3) / 1e12, 1),
        },
        "decode": {
            "ms": round(rt["dec"][0], 4), "ms_median": round(rt["dec"][1], 4),
            "dense_ms": round(rd["dec"][0], 4),
            "speedup": round(rd["dec"][0] / rt["dec"][0], 4),
            "num_splits": dec.splits,
            "retained_head_tiles_pct": pct(cd[1], cd[0]),
            "v_tiles_fetched_pct": pct(cd[mala.CNT_V_TILES], k_tiles),
            "v_tiles_consumed_pct": pct(cd[mala.CNT_V_NEEDED], k_tiles),
            "bytes_algorithmic": float(dec_bytes),
            "hbm_gbs_algorithmic": round(dec_bytes / (rt["dec"][0] * 1e-3) / 1e9, 1),
            "hbm_frac_algorithmic": round(dec_bytes / (rt["dec"][0] * 1e-3) / 1e9 / PEAK_HBM_GBS,
                                          4),
            "bytes_counters": dec_traffic,
            "hbm_gbs_counters": (round(dec_traffic / (rt["dec"][0] * 1e-3) / 1e9, 1)
                                 if dec_traffic else None),
            "hbm_frac": round((dec_traffic or dec_bytes) / (rt["dec"][0] * 1e-3) / 1e9
                              / PEAK_HBM_GBS, 4),
            "hbm_frac_source": "counters" if dec_traffic else "algorithmic",
            "ragged_lengths_supplementary": ragged,
        },
        "decision_tile": [bq, bk],
        "timing_protocol": ("HIP events per call; measured taus: mean / median of %d calls after "
                            "%d untimed (and at least %g ms of untimed calls); supplementary "
                            "fields: %d after %d; the timed calls leave out the optional "
                            "statistics, which one extra call per setting records"
                            % (args.reps, args.kernel_warmup, args.min_warm_ms, args.supp_reps,
                               args.supp_warmup)),
        "with_statistics": with_stats,
        "tau1_supplementary": {
            "fwd_ms": round(f1[0], 3), "bwd_ms": round(b1[0], 3), "decode_ms": round(d1[0], 4),
            "speedup_fwd": round(rd["fwd"][0] / f1[0], 4),
            "speedup_bwd": round(rd["bwd"][0] / b1[0], 4),
            "speedup_decode": round(rd["dec"][0] / d1[0], 4),
            "retained_tiles_pct_fwd": pct(cf1[1], cf1[0]),
            "retained_tiles_pct_bwd": pct(cb1[1], cb1[0]),
            "v_tiles_needed_pct_fwd": pct(cf1[5], cf1[2]),
            "do_tiles_loaded_pct_bwd": pct(cb1[2], do_dense),
            "retained_head_tiles_pct_decode": pct(cd1[1], cd1[0]),
            "v_tiles_fetched_pct_decode": pct(cd1[2], k_tiles),
            "v_tiles_consumed_pct_decode": pct(cd1[5], k_tiles),
            "mean_slots_per_query_fwd": round(float(cf1[3]) / (w.B * w.Hq * w.N), 1),
            "mean_slots_per_query_bwd": round(float(cb1[3]) / (w.B * w.Hq * w.N), 1),
        },
    }
    if not args.no_memory:
        detail["128k"]["operator_memory"] = operator_memory(tr, tau)
    del tr
    torch.cuda.empty_cache()
    rw = (args.reps, args.kernel_warmup)
    if not args.no_small:
        # the two smaller workloads at their tolerance sweeps (tau = 0 is measured too)
        detail["needle_1k_d64"] = train_workload("needle_1k_d64", (1e-4, 1e-3), *rw, memory=not args.no_memory)
        detail["mha16_8k"] = train_workload("mha16_8k", (1e-4, 1e-3), *rw, memory=not args.no_memory)
    if not args.no_32k:
        # the 32768-token GQA workload at tau (and the canonical tau = 1, supplementary)
        detail["32k"] = train_workload("gqa32x8_32k", (tau, 1.0), *rw, supp_taus=(1.0,), supp=(sr, sw),
                                     memory=not args.no_memory)
    if not args.no_lm:
        detail["lm_like_sweep"] = {
            "note": ("supplementary: language-model-like inputs (local key alpha=2, needles "
                     "shared by 32-row blocks beta=2, sink 1.5, Rademacher dO), 8 query / 2 KV "
                     "heads, head_dim 128, batch = 32768 / N; fidelity of tau > 0 against "
                     "tau = 0 through the same kernels: mean and P95 over heads, in percent"),
            "rows": lm_sweep(sr, sw),
        }

    line = {
        "metric": METRIC,
        "value": round(ms_per_step, 3),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": ("mala_fwd + mala_bwd, causal, batch 1, 8 query / 2 KV heads, 131072 "
                         "tokens, head_dim 128 (one TP=8 share), planted needles beta=2; then "
                         "mala_decode, batch 16, 32 query / 8 KV heads, 131072-token caches, "
                         "4 needles beta=3"),
            "tau": tau, "seq_len": w.N, "head_dim": w.D, "q_heads": w.Hq, "kv_heads": w.Hkv,
            "decode_batch": dec.w.B, "decode_splits": dec.splits,
        },
        "roofline": {
            "kernel": "mala_bwd (preprocess + dK/dV + dQ kernels)",
            "bound": "mfma",
            "achieved": round(achieved, 1),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic_from_profiles(
                os.path.join(ROOT, "paper_2609_32712_amd", "csrc", "mala_bwd.hip")),
            "flops_per_launch": fl_b,
            "launch_ms": round(bwd_ms, 3),
        },
        "detail": detail,
    }
    probe = mfma_probe()
    if probe is not None:
        detail["mfma_probe"] = probe
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        line["cpu_baseline"] = cpu_baseline(ms_per_step)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

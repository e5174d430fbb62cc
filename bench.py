#!/usr/bin/env python3
"""Throughput of the GTF-DEER hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic input:
  PLRNN workloads: deer_solve (Newton loop: residual + Jacobian masks, chunked MFMA scan,
                   carries, fix-up + max-norm test, until every sequence converged or the
                   fixed iteration count) followed by deer_adjoint (MSE seed, reverse scan
                   with transposed Jacobians, parameter-gradient reductions).
  diagonal SSM:    deer_solve (fused input projection + forward complex scan), then
                   deer_readout_loss (read-out MLP loss, its cotangent dL/dRe h and the
                   read-out gradients), then deer_adjoint on that real cotangent (reverse scan
                   with conj(lambda) + dlambda / dBc reductions).
Inputs are resident in HBM before the timed region.  The value is DEER timesteps per
second: sum over sequences of T x Newton updates, per second of the whole step (a latent
warm-up, --tw, is part of the same Newton iteration, so every update spans the T steps).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 5]

The default workload is the largest one, the M = 64 vanilla PLRNN (B = 32, T = 131072), whose
dense 64 x 64 chunk products are the matrix-core bound part of the path.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

PEAK_HBM_GBS = 8000.0            # MI355X HBM3E
PEAK_FP32_MFMA_TFLOPS = 157.3    # MI355X dense fp32 matrix
# fp32 vector: 256 CUs x 4 SIMDs x 16 lanes x 2 flops (FMA) x 2.4 GHz = 78.6 TFLOP/s.  The
# published 157.3 counts packed fp32 (two FMAs per lane per instruction); the kernels are built
# without packed instructions, so 78.6 is the ceiling they can reach and the peak used here.
PEAK_FP32_VALU_TFLOPS = 78.6
# quasi-DEER gains about one exact leading step per update, so a solve may need up to T + 1
# updates; beyond this many passes per solve the run would not finish in a benchmark's time
QUASI_MAX_PASSES = 20000


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _plrnn_step(D, model, xd, c, ws_s, ws_a, T_w=0):
    res = D.deer_solve(model, xd, c.alpha, c.n_obs, tol=c.tol, max_iter=c.max_iter, fixed_iters=c.fixed_iters,
                       ws=ws_s, check=False, T_w=T_w)
    if res["status"] != 0:
        raise RuntimeError(f"deer_solve returned status {res['status']}: {D.load().deer_last_error()}")
    # the step's outputs are the parameter gradients: the adjoint itself is not stored
    D.deer_adjoint(model, xd, res["z"], c.alpha, c.n_obs, ws=ws_a, want_lam=False, T_w=T_w)
    return sum(res["iters"])


def check_quasi_bound(c, passes):
    """Refuse, before any GPU work, a quasi-DEER solve to tolerance whose pass bound (T + 2:
    about one more exact leading step per update) is too long for a benchmark run; a fixed
    number of passes is always accepted."""
    if passes < 0:
        raise SystemExit("--quasi-passes must be >= 0")
    if passes == 0 and not c.fixed_iters and c.T + 2 > QUASI_MAX_PASSES:
        raise SystemExit(f"quasi-DEER on {c.name}: a solve to tolerance may take up to T + 2 = {c.T + 2} passes "
                         f"(> {QUASI_MAX_PASSES}); pass --quasi-passes K to time K passes per solve instead")


def _quasi_step(D, model, xd, c, ws_s, ws_a, T_w=0):
    # quasi-DEER: one more leading step is exact per update, so T + 1 updates always suffice
    # (check_quasi_bound has refused the workloads where that is too many)
    res = D.deer_solve_quasi(model, xd, c.alpha, c.n_obs, tol=c.tol, max_iter=c.T + 2, fixed_iters=c.fixed_iters,
                             ws=ws_s, check=False, T_w=T_w)
    if res["status"] != 0:
        raise RuntimeError(f"deer_solve_quasi returned status {res['status']}: {D.load().deer_last_error()}")
    D.deer_adjoint_quasi(model, xd, res["z"], c.alpha, c.n_obs, ws=ws_a, want_lam=False, T_w=T_w)
    return sum(res["iters"])


def _train_step(D, model, xd, c, ws, st, T_w):
    # one optimiser step: solve, MSE + MAR loss, gradient, Adam on the parameters in place
    st["step"] += 1
    out = D.deer_train_step(model, xd, c.alpha, c.n_obs, step=st["step"], state=st.get("adam"), lr=1e-4,
                            mar_lambda=1.0, mar_units=max(1, c.M // 4), mar_p=2, mar_gamma_w=1.0 / (3 * c.M),
                            mar_gamma_v=1.0 / (3 * c.M), T_w=T_w, tol=c.tol, max_iter=c.max_iter, ws=ws)
    st["adam"] = out["state"]
    return sum(out["iters"])


def _diag_step(D, model, readout, xd, c, ws_s, ws_r, ws_a, bufs):
    res = D.deer_solve(model, xd, 0.0, 0, ws=ws_s, z=bufs["h"])
    r = D.deer_readout_loss(readout, res["z"], xd, g=bufs["g"], ws=ws_r)
    D.deer_adjoint(model, xd, res["z"], 0.0, 0, g=r["g"], ws=ws_a, want_lam=False)
    return c.B


def kernel_work(c, steps, updates):
    """Algorithmic work of each kernel over the timed region: {name: (bound, total work)};
    work in flop (mfma) or bytes (hbm).  `updates` = Newton updates summed over sequences, each
    over the whole sequence."""
    B, T, M, N = c.B, c.T, c.M, c.n_obs
    W = (M + 31) // 32
    fwd = updates * T                 # (b, t) steps processed by the updates
    adj = steps * B * T               # (b, t) steps of the adjoint passes
    prod = fwd + steps * B * (T - 1)  # chunk-product steps (the adjoint product covers 1..T-1)
    if c.kind == "diag_ssm":
        K = c.n_obs
        elems = steps * B * T * M
        xin = steps * B * T * 4 * K
        return {
            # forward: b formed from x on the fly; the write pass stores y (8 B per element)
            "k_diag_seg_write": ("hbm", elems * 8 + xin),
            # adjoint: real cotangent (4 B) and forward states (8 B) read, dlam / dBc accumulated
            # on the way (the training step does not store the adjoint itself)
            "k_diag_rseg": ("hbm", elems * 12 + xin),
            "k_diag_scan_lb_grads": ("hbm", elems * 12 + xin),
            "k_diag_scan_lb": ("hbm", elems * 12 + xin),
            # read-out: three [rows x 64] x [64 x 128] products (s, g, dWa) on the matrix cores
            "k_readout": ("mfma", steps * B * T * 3 * 2.0 * M * c.params["Wa"].shape[0]),
        }
    out = {}
    if c.kind == "plrnn":
        # forward Newton updates run the fused kernel (residual + masks + product); the
        # adjoint runs the shifted product and a mask pass
        out["k_newton_product_plrnn"] = ("mfma", fwd * 2.0 * M ** 3)
        # M <= 16 with whole blocks of chunks: one kernel per pass (the fix-up of an update and
        # the forward pass of the next); its matrix-core work is the forward pass's
        out["k_newton_pass16"] = ("mfma", fwd * 2.0 * M ** 3)
        # M <= 4 with a fixed update count: the whole solve in one launch on the vector units
        # (the same chunk-map composition, 2 M^3 flops per timestep and update)
        out["k_newton_small"] = ("alu", fwd * 2.0 * M ** 3)
        out["k_chunk_product_plrnn"] = ("mfma", steps * B * (T - 1) * 2.0 * M ** 3)
        out["k_resjac_plrnn"] = ("hbm", adj * (4 * M + 4 * N + 4 * W))
        # quasi-DEER: residual and diagonal (z, x read; r, d written / adjoint: d written),
        # chunk aggregates (d and r, or d and the seed inputs), fix-ups (forward: d, r, z read
        # and the next iterate written; reverse: d read, z and x for the forced inputs)
        out["k_qdeer_resdiag"] = ("hbm", fwd * (12 * M + 4 * N) + adj * (8 * M + 4 * N))
        out["k_qdeer_chunk"] = ("hbm", fwd * 8 * M + adj * (4 * M + 8 * N))
        out["k_qdeer_fixup_fwd"] = ("hbm", fwd * 16 * M)
        out["k_qdeer_fixup_rev"] = ("hbm", adj * (8 * M + 4 * N))
        # the adaptive loop's one-kernel quasi pass: z and x read, the next iterate written (the
        # residual is formed again from them, the chunk aggregates are a few floats per chunk)
        out["k_qdeer_pass"] = ("hbm", fwd * (8 * M + 4 * N))
        if M <= 16:
            # the register-tiled fix-ups form the residual and the masks again from z and x:
            # forward z, x read and the next iterate written; reverse z, x read (the training
            # step keeps the parameter gradients only, so the adjoint is not written)
            out["k_fixup_fwd_plrnn"] = ("hbm", fwd * (8 * M + 4 * N))
            out["k_fixup_rev_plrnn"] = ("hbm", adj * (4 * M + 4 * N))
        else:
            out["k_fixup_fwd_plrnn"] = ("hbm", fwd * (12 * M + 4 * W))
            out["k_fixup_rev_plrnn"] = ("hbm", adj * (8 * M + 4 * N + 4 * W))
    else:
        L = c.L
        LW = (L + 31) // 32
        out["k_jacform_shplrnn"] = ("mfma", (fwd + adj) * 2.0 * M * M * L)
        out["k_chunk_product_dense"] = ("mfma", prod * 2.0 * M ** 3)
        # without a stored Jacobian: J~_t formed (2 M^2 L) and composed (2 M^3) in the chunk
        # products; two matrix-vector products with W1 and W2 (4 M L) per step in the fix-ups
        out["k_chunk_product_shfused"] = ("mfma", fwd * (2.0 * M * M * L + 2.0 * M ** 3))
        out["k_chunk_product_shfused_rev"] = ("mfma", steps * B * (T - 1) * (2.0 * M * M * L + 2.0 * M ** 3))
        out["k_fixup_shjvp"] = ("mfma", fwd * 4.0 * M * L)
        # the Newton passes' residual on the matrix cores: u = W2 z~ and W1 relu(u), 4 M L per step
        out["k_resjac_shmfma"] = ("mfma", fwd * 4.0 * M * L)
        out["k_fixup_shjvp_rev"] = ("mfma", steps * B * (T - 1) * 4.0 * M * L)
        out["k_resjac_shplrnn"] = ("hbm", (fwd + adj) * (8 * M + 4 * N + 4 * LW))
        out["k_fixup_dense_fwd"] = ("hbm", fwd * (4 * M * M + 12 * M))
        out["k_fixup_dense_rev"] = ("hbm", adj * (4 * M * M + 8 * M))
    return out


# HBM bytes per launch measured with rocprofv3 counter passes (FETCH_SIZE, WRITE_SIZE), each
# scaled by the reading of a plain copy of known size in the same run; kept in
# profiles/traffic_<workload>.txt together with the hash of the kernel's source file, and
# reported only while that source is unchanged.
KERNEL_SOURCE = {"k_chunk_product_shfused": "k_shfused.hip", "k_chunk_product_shfused_rev": "k_shfused.hip",
                 "k_fixup_shjvp": "k_shfused.hip", "k_resjac_shmfma": "k_shfused.hip", "k_newton_product_plrnn": "k_plrnn.hip", "k_newton_pass16": "k_plrnn.hip", "k_chunk_product_plrnn": "k_plrnn.hip",
                 "k_fixup_fwd_plrnn": "k_plrnn.hip", "k_jacform_shplrnn": "k_shallow.hip",
                 "k_chunk_product_dense": "k_dense.hip", "k_readout": "k_readout.hip",
                 "k_diag_scan_lb_grads": "k_diag.hip", "k_diag_seg_write": "k_diag.hip",
                 "k_diag_rseg": "k_diag.hip"}
CALIB_COPY_BYTES = 256 << 20


def measured_traffic(workload, kernel):
    import hashlib
    path = os.path.join(HERE, "profiles", f"traffic_{workload}.txt")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCE:
        return None
    rec = {}
    for ln in open(path):
        if ":" in ln and not ln.startswith("#"):
            k, v = ln.split(":", 1)
            rec[k.strip()] = v.strip()
    src = os.path.join(HERE, "paper_2605_12683_amd", "csrc", KERNEL_SOURCE[kernel])
    if rec.get("kernel") != kernel or not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("source_sha256"):
        return None
    return float(rec["traffic_bytes_per_launch"])


def measured_mfma(workload, kernel):
    """Matrix-core activity of the kernel from rocprofv3 counter passes
    (SQ_INSTS_VALU_MFMA_MOPS_F32, SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE), kept in
    profiles/mfma_<workload>.txt with the hash of the kernel's source; None once it changed."""
    import hashlib
    path = os.path.join(HERE, "profiles", f"mfma_{workload}.txt")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCE:
        return None
    rec = {}
    for ln in open(path):
        if ":" in ln and not ln.startswith("#"):
            k, v = ln.split(":", 1)
            rec[k.strip()] = v.strip()
    src = os.path.join(HERE, "paper_2605_12683_amd", "csrc", KERNEL_SOURCE[kernel])
    if rec.get("kernel") != kernel or not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("source_sha256"):
        return None
    tf = float(rec["mfma_counted_tflops"])
    return {"busy_frac": float(rec["mfma_busy_frac"]), "counted_tflops": tf,
            "counted_frac": tf / PEAK_FP32_MFMA_TFLOPS,
            "counted_flops_per_launch": float(rec["mfma_flops_per_dispatch"]),
            "source": f"profiles/mfma_{workload}.txt"}


def roofline_for(name, c, total_ms, launches, steps, updates):
    """Algorithmic work of the dominant kernel over the timed region, divided by its time."""
    work = kernel_work(c, steps, updates)
    base = {"kernel": name, "avg_launch_ms": total_ms / launches, "launches": launches,
            "traffic": measured_traffic(c.name, name)}
    if name not in work:
        base.update({"bound": "unknown", "achieved": None, "peak": None, "unit": None, "frac": None})
        return base
    bound, w = work[name]
    if bound == "mfma":
        ach = w / (total_ms * 1e-3) / 1e12
        base.update({"bound": "mfma", "achieved": ach, "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / PEAK_FP32_MFMA_TFLOPS, "work_per_launch": w / launches,
                     "mfma_counters": measured_mfma(c.name, name)})
    elif bound == "alu":
        ach = w / (total_ms * 1e-3) / 1e12
        base.update({"bound": "alu", "achieved": ach, "peak": PEAK_FP32_VALU_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / PEAK_FP32_VALU_TFLOPS, "work_per_launch": w / launches})
    else:
        ach = w / (total_ms * 1e-3) / 1e9
        base.update({"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": ach / PEAK_HBM_GBS, "work_per_launch": w / launches})
    return base


def _oracle_sample(kind, params, x, alpha, n_obs, tol, max_iter, fixed_iters):
    """One oracle run on a sample: the work one CPU user of the method would do.  PLRNN kinds:
    Newton solve, adjoint and parameter gradients; diagonal SSM: forward scan, read-out,
    reverse scan and gradients.  Returns (timesteps processed, seconds)."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:       # pragma: no cover
        pass
    t0 = time.perf_counter()
    if kind == "diag_ssm":
        O.diag_ssm_step(params, x)
        work = x.shape[0] * (x.shape[1] - 1)
    else:
        m = {"kind": kind, **params}
        res = O.newton(m, x, alpha, n_obs, tol=tol, max_iter=max_iter, fixed_iters=fixed_iters)
        lam = O.adjoint(m, x, res["z"], alpha, n_obs)
        O.param_grads(m, x, res["z"], alpha, n_obs, lam)
        work = float(np.sum(res["iters"])) * (x.shape[1] - 1)
    return work, time.perf_counter() - t0


def _warm_worker(_):
    import oracle  # noqa: F401  (import cost kept out of the timed region)
    return os.getpid()


def _host_cpu():
    """Usable host cores (affinity) and the CPU model name."""
    try:
        ncpu = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        ncpu = os.cpu_count() or 1
    model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:         # pragma: no cover
        pass
    return ncpu, model


def cpu_baseline(c, budget_s=12.0, max_workers=16):
    """The float64 oracle on the host, on a bounded sample of the same workload, twice: on one
    thread, and across the host's cores with one worker process per share of the sequences
    (at most B workers, at most `max_workers`; each worker single-threaded).  Runs in child
    processes of this one, before the GPU is used."""
    import multiprocessing as mp
    ncpu, model = _host_cpu()
    args = (c.kind, c.params, None, c.alpha, c.n_obs, c.tol, c.max_iter, c.fixed_iters)
    if c.kind == "diag_ssm":
        Ts = min(c.T, 1 << 15)
        seqs = list(range(c.B))
        single_x = c.x[:1, :Ts + 1]
        desc = f"first {Ts} of {c.T} steps, forward + read-out + reverse + gradients"
    else:
        # calibrate on a short prefix of the whole batch, then shorten T to fit the budget
        Tc = min(c.T, 256)
        w, dt = _oracle_sample(*args[:2], c.x[:, :Tc + 1], *args[3:])
        per = dt / max(w, 1.0)          # seconds per (b, t, update)
        Ts = c.T
        while Ts > 512 and per * w / Tc * Ts > budget_s:
            Ts //= 2
        seqs = list(range(c.B))
        single_x = c.x[:, :Ts + 1]
        desc = f"first {Ts} of {c.T} steps, Newton solve + adjoint + gradients"
    ctx = mp.get_context("spawn")
    with ctx.Pool(1) as pool:
        w1, dt1 = pool.apply(_oracle_sample, (*args[:2], np.ascontiguousarray(single_x), *args[3:]))
    nw = max(1, min(len(seqs), ncpu, max_workers))
    if c.kind == "diag_ssm":
        shares = [c.x[[b], :Ts + 1] for b in seqs]
        desc_all = f"all {c.B} sequences, " + desc
    else:
        shares = [c.x[seqs[k::nw], :Ts + 1] for k in range(nw)]
        desc_all = f"all {c.B} sequences, " + desc
    with ctx.Pool(nw) as pool:
        pool.map(_warm_worker, range(nw))
        t0 = time.perf_counter()
        res = pool.starmap(_oracle_sample, [(*args[:2], np.ascontiguousarray(x), *args[3:]) for x in shares])
        dtn = time.perf_counter() - t0
    wn = sum(r[0] for r in res)
    single = {"value": w1 / dt1, "cores": 1, "seconds": dt1,
              "sample": (f"1 of {c.B} sequences, " if c.kind == "diag_ssm" else f"all {c.B} sequences, ") + desc}
    return {"value": wn / dtn, "unit": "timesteps/s", "cores": nw, "kind": "oracle", "sample": desc_all,
            "seconds": dtn, "single_thread": single, "host_cpus": ncpu, "cpu_model": model}


def fig1a_sweep(reps: int = 3, inits=("random", "contracting"), Ms=(4, 16, 64, 128), Ts=None):
    """Runtime of one training step (forward + backward with the parameter gradients), GTF-DEER
    against the sequential baseline on the same GPU, over the grid of Fig. 1A: shallow PLRNN
    L = 50, M in (4, 16, 64, 128), B = 1, T = 2^7 ... 2^15, alpha = 0.15, Lorenz-63 data (N = 3).
    Models are not trained: "random" draws the default initialisation (A in [0.5, 0.95], W1, W2
    with variance 1/L), which is not a contraction for M >= 16 and makes DEER take many Newton
    updates; "contracting" rescales W1 so that max A + ||W1|| ||W2|| < 1 (A in [0.5, 0.65],
    ||W1|| ||W2|| = 0.3), the regime GTF is meant to produce.  DEER's iteration counts are those
    of the model at hand.  One JSON line per point."""
    import torch
    import workloads as W
    import paper_2605_12683_amd as D

    L, N, alpha = 50, 3, 0.15

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            t0 = time.perf_counter()
            out = fn()
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts)) * 1e3, out

    Ts = Ts or [1 << lt for lt in range(7, 16)]
    for init in inits:
        for M in Ms:
            _fig1a_model(D, W, init, M, L, N, alpha, timed, Ts)


def _fig1a_model(D, W, init, M, L, N, alpha, timed, Ts):
    import torch
    rng = np.random.default_rng(9000 + M)
    if init == "random":
        params = W.shplrnn_params(M, L, rng)
    else:
        params = W.shplrnn_params(M, L, rng, a_range=(0.5, 0.65))
        W1 = params["W1"].astype(np.float64)
        norm = np.linalg.norm(W1, 2) * np.linalg.norm(params["W2"].astype(np.float64), 2)
        params["W1"] = (W1 * (0.3 / norm)).astype(np.float32)
    model = D._Model({"kind": "shplrnn", **params})
    for T in Ts:
        lt = T.bit_length() - 1
        x = torch.tensor(W.observed_batch("lorenz63", N, 1, T, 9100 + lt), device="cuda")
        ws_q = D._workspace(D.deer_sequential_workspace_bytes(model, 1, T))
        seq_ms, _ = timed(lambda: D.deer_sequential(model, x, alpha, N, ws=ws_q, want_lam=False))
        rec = {"sweep": "fig1a", "model": "shplrnn", "init": init, "M": M, "L": L, "B": 1, "T": T, "alpha": alpha,
               "sequential_ms": round(seq_ms, 4), "deer_ms": None, "newton_updates": None, "speedup": None}
        ws_s = D._workspace(D.deer_workspace_bytes(model, 1, T, 0))
        ws_a = D._workspace(D.deer_workspace_bytes(model, 1, T, 1))

        def step():
            r = D.deer_solve(model, x, alpha, N, tol=1e-5, max_iter=500, ws=ws_s, check=False)
            D.deer_adjoint(model, x, r["z"], alpha, N, ws=ws_a, want_lam=False)
            return r
        deer_ms, r = timed(step)
        rec.update(deer_ms=round(deer_ms, 4), newton_updates=int(sum(r["iters"])),
                   speedup=round(seq_ms / deer_ms, 3), status=int(r["status"]))
        print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=5, help="workload 1..5 (default 5, the M = 64 vanilla PLRNN)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tw", type=int, default=0,
                    help="PLRNN workloads with a tolerance: latent warm-up of this many steps")
    ap.add_argument("--train", action="store_true",
                    help="PLRNN workloads with a tolerance: the whole training step (deer_train_step: loss with "
                         "MAR, gradient, Adam update in place)")
    ap.add_argument("--quasi", action="store_true",
                    help="PLRNN workloads: quasi-DEER (diagonal Jacobians) instead of GTF-DEER")
    ap.add_argument("--quasi-passes", type=int, default=0,
                    help="with --quasi: run exactly this many quasi-DEER updates per solve (no tolerance) and "
                         "report that throughput; required when T + 2 exceeds %d" % QUASI_MAX_PASSES)
    ap.add_argument("--fig1a", action="store_true",
                    help="instead of the workload: the Fig. 1A sweep, GTF-DEER against the sequential baseline")
    ap.add_argument("--fig1a-point", default=None, metavar="INIT,M,T",
                    help="with --fig1a: one point of the grid only (e.g. contracting,128,32768)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)
    if args.fig1a:
        if args.fig1a_point:
            init, M, T = args.fig1a_point.split(",")
            if init not in ("random", "contracting") or int(T) < 1 or int(T) & (int(T) - 1):
                raise SystemExit("--fig1a-point: INIT is random or contracting, T a power of two")
            fig1a_sweep(inits=(init,), Ms=(int(M),), Ts=[int(T)])
        else:
            fig1a_sweep()
        return

    import torch
    import workloads as W
    import paper_2605_12683_amd as D
    from paper_2605_12683_amd import _binding as Bnd

    c = W.make_config(args.config)
    log(f"[bench] workload {c.name}: B={c.B} T={c.T} M={c.M} kind={c.kind}")
    if args.quasi:
        if c.kind != "plrnn":
            print("quasi-DEER is built for the vanilla PLRNN workloads (1, 2, 5)", file=sys.stderr)
            sys.exit(3)
        check_quasi_bound(c, args.quasi_passes)
        if args.quasi_passes > 0:
            c.fixed_iters = args.quasi_passes
    cb = None
    if not args.no_cpu_baseline and not args.quasi:
        # before the GPU is used: the oracle runs in child processes of this one
        log("[bench] timing the CPU oracle on a bounded sample (one thread, then all cores)")
        cb = cpu_baseline(c)
        log(f"[bench] cpu oracle: {cb['single_thread']['value']:.4g} timesteps/s on 1 thread, {cb['value']:.4g} on "
            f"{cb['cores']} processes ({cb['cpu_model']}, {cb['host_cpus']} usable cpus; {cb['sample']})")
    dev = torch.device("cuda:0")
    xd = torch.tensor(c.x, device=dev)
    # a plain device copy of known size: the calibration the counter passes scale by
    calib = torch.empty(CALIB_COPY_BYTES // 4, device=dev)
    torch.empty_like(calib).copy_(calib)
    del calib
    if c.kind == "diag_ssm":
        model = D._Model({"kind": "diag_ssm", "lam": c.params["lam"], "Bc": c.params["Bc"]})
        readout = D._Readout({k: c.params[k] for k in ("Wa", "ca", "Wb", "cb")})
        ws_s = D._workspace(D.deer_workspace_bytes(model, c.B, c.T, Bnd.DEER_OP_SOLVE))
        ws_a = D._workspace(D.deer_workspace_bytes(model, c.B, c.T, Bnd.DEER_OP_ADJOINT))
        ws_r = D._workspace(D.deer_readout_workspace_bytes(readout, c.B, c.T, c.M))
        bufs = {"h": torch.empty(c.B, c.T, c.M, 2, device=dev), "g": torch.empty(c.B, c.T, c.M, device=dev)}
        step = lambda: _diag_step(D, model, readout, xd, c, ws_s, ws_r, ws_a, bufs)   # noqa: E731
    elif c.kind in ("plrnn", "shplrnn"):
        model = D._Model({"kind": c.kind, **c.params})
        if args.train:
            lib = D.load()
            fw = Bnd.deer_forcing(float(c.alpha), int(c.n_obs), int(args.tw))
            ws_t = D._workspace(lib.deer_train_workspace_bytes(ctypes.byref(model.c), ctypes.byref(fw), c.B, c.T, 0))
            tstate = {"step": 0}
            step = lambda: _train_step(D, model, xd, c, ws_t, tstate, args.tw)   # noqa: E731
        elif args.quasi:
            lib = D.load()
            ws_s = D._workspace(lib.deer_quasi_workspace_bytes(ctypes.byref(model.c), c.B, c.T, Bnd.DEER_OP_SOLVE))
            ws_a = D._workspace(lib.deer_quasi_workspace_bytes(ctypes.byref(model.c), c.B, c.T,
                                                               Bnd.DEER_OP_ADJOINT))
            step = lambda: _quasi_step(D, model, xd, c, ws_s, ws_a, args.tw)   # noqa: E731
        else:
            lib = D.load()
            fw = Bnd.deer_forcing(float(c.alpha), int(c.n_obs), int(args.tw))
            ws_s = D._workspace(lib.deer_workspace_bytes_ex(ctypes.byref(model.c), ctypes.byref(fw), c.B, c.T,
                                                            Bnd.DEER_OP_SOLVE, 0))
            ws_a = D._workspace(lib.deer_workspace_bytes_ex(ctypes.byref(model.c), ctypes.byref(fw), c.B, c.T,
                                                            Bnd.DEER_OP_ADJOINT, 0))
            step = lambda: _plrnn_step(D, model, xd, c, ws_s, ws_a, args.tw)   # noqa: E731
    else:
        print(f"workload {c.name}: model kind {c.kind} not supported by this build", file=sys.stderr)
        sys.exit(3)

    t_w = time.perf_counter()
    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done ({time.perf_counter() - t_w:.2f} s)")
    torch.cuda.synchronize()
    # steps long enough to be seen are reported one by one (outside the timed region for short ones)
    slow = args.warmup > 0 and (time.perf_counter() - t_w) / args.warmup > 0.5
    # per-kernel durations: HIP events around every launch on the stream it is launched on,
    # over separate steps (the events add launch overhead, so the timed steps run without them)
    prof_steps = max(1, min(args.steps, 3))
    Bnd.timing_enable(True)
    prof_updates = 0
    for i in range(prof_steps):
        prof_updates += step()
        if slow:
            log(f"[bench] event-timed step {i + 1}/{prof_steps} done")
    torch.cuda.synchronize()
    kt = Bnd.timing_report()
    Bnd.timing_enable(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    updates = 0
    for i in range(args.steps):
        updates += step()
        if slow:
            log(f"[bench] timed step {i + 1}/{args.steps} returned")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    log(f"[bench] {args.steps} timed steps: {(t1 - t0) * 1e3 / args.steps:.3f} ms per step")
    dt = t1 - t0
    iters_per_step = updates / args.steps
    timesteps = updates * c.T
    value = timesteps / dt
    for k, (ms, n) in sorted(kt.items(), key=lambda kv: -kv[1][0]):
        log(f"[bench] {k:28s} {ms:10.3f} ms total  {n:6d} launches  {ms / n:9.4f} ms avg")
    # dominant kernel: the one with the largest share of device time among those with a
    # work model (a latency-bound helper such as the carry pass has none)
    modeled = {k: v for k, v in kt.items() if k in kernel_work(c, 1, 1)}
    dom = max((modeled or kt).items(), key=lambda kv: kv[1][0])
    roof = roofline_for(dom[0], c, dom[1][0], dom[1][1], prof_steps, prof_updates)
    kernels = {k: {"ms_total": ms, "launches": n, **({"frac": r["frac"], "unit": r["unit"], "achieved": r["achieved"]}
                                                      if (r := roofline_for(k, c, ms, n, prof_steps, prof_updates))["frac"]
                                                      is not None else {})}
               for k, (ms, n) in kt.items()}

    out = {
        "metric": "DEER timesteps/sec (B*T*Newton iters)",
        "value": value,
        "unit": "timesteps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Lorenz trajectories, random-init parameters)",
        "config": {"workload": c.name, "kind": c.kind, "B": c.B, "T": c.T, "M": c.M, "N": c.n_obs,
                   "alpha": c.alpha, "tol": c.tol if not c.fixed_iters else None,
                   "fixed_iters": c.fixed_iters or None, "newton_updates_per_step": iters_per_step,
                   "step": ("deer_train_step (solve, MSE + MAR loss, gradient, Adam)" if args.train else
                            "deer_solve_quasi + deer_adjoint_quasi (quasi-DEER: diagonal Jacobians)" if args.quasi
                            else "deer_solve + deer_adjoint"), "latent_warmup": args.tw},
        "roofline": roof,
        "kernels": kernels,
    }
    if cb is not None:
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

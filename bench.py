#!/usr/bin/env python3
"""ALS half-sweep throughput on one MI355X.

One step = one ALS sweep of the paper's order (Sec. 2.2): the item half-sweep
(solve V with U fixed) then the user half-sweep (solve U with V fixed); each
half-sweep's gather also yields the squared residuals of the state it enters,
so every state's training RMSE is produced once. The metric is ratings per
second per half-sweep, 2 * nnz * steps / elapsed, with the rating matrix and
factors resident in HBM before the timed region; per_side gives each side's
median half-sweep time (HIP events) and its ratings per second.

Default workload: the full-scale synthetic stand-in for the paper's data set
(1,000,990 users x 624,961 items x 262,810,175 ratings, Sec. 1), D = 20,
lambda = 0.065 weighted by n_s. --config 4 selects the same matrix at D = 100.

Besides the JSON line's throughput, the script reports the roofline position
of the dominant kernel (HIP-event timing of each of its launches over the timed
region; the other phases are timed on two extra untimed sweeps, so that their
event records stay out of the timed region) and the fp64 CPU oracle's throughput
on a bounded sample of the same half-sweep on this host's cores.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
MFMA_F32_PEAK_TFS = 157.3  # MI355X dense fp32 matrix
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.txt")
CSRC = os.path.join(ROOT, "paper_1108_2580_amd", "csrc")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=None, choices=[1, 2, 3, 4, 5],
                    help="one workload only (default: the D = 20 headline on the full-scale "
                         "matrix, then the same matrix at D = 100 as the d100 leg)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target duration of the CPU oracle sample (0 disables it)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (for HBM counter scaling)")
    ap.add_argument("--phase-sweeps", type=int, default=2,
                    help="untimed sweeps with every phase timed, after the timed ones (0: none; "
                         "phases_ms_per_step is then null)")
    ap.add_argument("--heldout-share", type=int, default=64,
                    help="held-out prediction leg on 1/K of the stored positions (0 disables)")
    ap.add_argument("--weighted", action="store_true",
                    help="weighted ALS: seeded per-rating weights, log-uniform on [0.25, 4)")
    ap.add_argument("--gibbs", action="store_true",
                    help="Bayesian factorisation: one step is a BPMF Gibbs iteration")
    ap.add_argument("--tensor", action="store_true",
                    help="tensor ALS over 6649 seeded time bins: one step updates the items, "
                         "the users and the time bins")
    ap.add_argument("--bptf", action="store_true",
                    help="BPTF: one step is a Gibbs iteration of the tensor model over 6649 "
                         "seeded time bins (alpha, the three hyperparameter draws, then the "
                         "items, users and time bins)")
    args = ap.parse_args()
    if args.gibbs + args.weighted + args.tensor + args.bptf > 1:
        ap.error("--gibbs, --weighted, --tensor and --bptf are exclusive")
    return args


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def copy_calibration():
    import torch

    n = 1 << 30  # 1 Gi floats = 4 GiB each way
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: 3 copies of {4 * n} bytes")


def strip_comments(src):
    """C/C++ source without comments, trailing blanks or empty lines (string and
    character literals are kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        ch = src[i]
        if ch in "\"'":
            j = i + 1
            while j < n and src[j] != ch:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            while i < n and src[i] != "\n":
                i += 1
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(ch)
            i += 1
    lines = (line.rstrip() for line in "".join(out).split("\n"))
    return "\n".join(line for line in lines if line)


def kernel_source_hash():
    """Hash of the device sources with comments removed (the counters are void once the
    code of any of them changes)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            h.update(name.encode())
            h.update(strip_comments(open(os.path.join(CSRC, name)).read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload_name, kernel):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter
    summary, if it was taken on the current device sources for this workload; else None."""
    try:
        for line in open(TRAFFIC_FILE):
            if line.startswith("TRAFFIC_JSON "):
                rec = json.loads(line[len("TRAFFIC_JSON "):])
                if rec.get("src_sha256_16") == kernel_source_hash() and \
                        rec.get("workload") == workload_name and rec.get("kernel") == kernel:
                    return rec.get("bytes_per_launch")
    except OSError:
        pass
    return None


def cpu_baseline(r, side_fixed, target_s, weights=None, gibbs=False, tensor=None):
    """fp64 oracle on a seeded random sample of the user half-sweep's rows (the Gibbs row
    draws with ``gibbs``; the tensor user-mode update with ``tensor`` = (bins, T))."""
    import numpy as np

    import oracle

    deg = np.diff(r.row_ptr)
    rows = np.flatnonzero(deg > 0)
    rng = np.random.default_rng(12345)
    perm = rows[rng.permutation(rows.size)]
    csum = np.cumsum(deg[perm])
    val = r.val.astype(np.float64)
    w = None if weights is None else weights.astype(np.float64)
    fixed = side_fixed.astype(np.float64)
    threads = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))

    def run(n_ratings):
        k = int(np.searchsorted(csum, n_ratings)) + 1
        k = min(k, perm.size)
        sel = np.sort(perm[:k])
        t0 = time.perf_counter()
        if tensor is not None:
            bins, Tf = tensor
            sub_ptr = np.concatenate([[0], np.cumsum(deg[sel])]).astype(np.int64)
            take = np.repeat(r.row_ptr[sel] - sub_ptr[:-1], deg[sel]) + np.arange(sub_ptr[-1])
            t_a = time.perf_counter()
            if gibbs:
                oracle.tensor_gibbs_rows(sub_ptr, r.col[take], bins[take], val[take], fixed, Tf,
                                         BPTF_ALPHA_TYPICAL, np.eye(r.D), np.zeros(r.D),
                                         np.zeros((k, r.D)), np.zeros((k, r.D)), threads=threads)
            else:
                oracle.tensor_rows(sub_ptr, r.col[take], bins[take], val[take], fixed, Tf,
                                   r.lam, np.zeros((k, r.D)), threads=threads)
            return int(deg[sel].sum()), k, time.perf_counter() - t_a
        if gibbs:
            sub_ptr = np.concatenate([[0], np.cumsum(deg[sel])]).astype(np.int64)
            take = np.repeat(r.row_ptr[sel] - sub_ptr[:-1], deg[sel]) + np.arange(sub_ptr[-1])
            Lam, mu = np.eye(r.D), np.zeros(r.D)
            z = np.zeros((k, r.D))
            t_a = time.perf_counter()
            oracle.gibbs_rows(sub_ptr, r.col[take], val[take], fixed, GIBBS_ALPHA, Lam, mu, z,
                              np.zeros((k, r.D)), threads=threads)
            return int(deg[sel].sum()), k, time.perf_counter() - t_a
        oracle.solve_rows(sel, r.row_ptr, r.col, val, fixed, r.lam, threads=threads, w=w)
        dt = time.perf_counter() - t0
        return int(deg[sel].sum()), k, dt

    n0, k0, t0 = run(max(1, r.nnz // 500))
    rate0 = n0 / max(t0, 1e-9)
    target = min(r.nnz, int(rate0 * target_s))
    n1, k1, t1 = run(target)
    return dict(value=n1 / t1, unit="ratings/s", cores=threads, kind="oracle",
                cpu_model=host_cpu(), build=" ".join(["gcc", *oracle.CFLAGS]),
                schedule="rows in descending degree order, dynamic",
                sample=(f"user half-sweep of {r.name}"
                        f"{' (weighted)' if w is not None else ' (Gibbs draws)' if gibbs else ''}"
                        f"{' (tensor user mode)' if tensor is not None else ''}"
                        f"{' (BPTF user draws)' if tensor is not None and gibbs else ''}: "
                        f"{k1} of {rows.size} rows (seeded random), "
                        f"{n1} ratings, D={r.D}, fp64, {t1:.1f} s"))


def host_cpu():
    """The host CPU as lscpu names it (model name, with family / model / stepping when the
    name alone is generic)."""
    import subprocess

    fields = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
        for line in out.splitlines():
            if ":" in line:
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    except (OSError, subprocess.SubprocessError):
        pass
    name = fields.get("Model name", "unknown")
    ident = ", ".join(f"{k.lower()} {fields[k]}" for k in ("CPU family", "Model", "Stepping")
                      if k in fields)
    sockets = fields.get("Socket(s)")
    return f"{name} ({ident}{', ' + sockets + ' socket(s)' if sockets else ''})"


def one_thread_scale():
    """For scale beside the all-threads figure: the fp64 oracle on one host thread over the
    whole user half-sweep of the mid workload (100,000 x 50,000, 10M ratings, D = 20), from
    its seeded initial factors."""
    import numpy as np

    import oracle
    import workload

    m = workload.make_config(2)
    _, V0 = workload.init_factors(m.M, m.N, m.D, m.init_seed)
    rows = np.arange(m.M)
    val = m.val.astype(np.float64)
    t0 = time.perf_counter()
    oracle.solve_rows(rows, m.row_ptr, m.col, val, V0.astype(np.float64), m.lam, threads=1)
    dt = time.perf_counter() - t0
    return dict(value=m.nnz / dt, unit="ratings/s", cores=1,
                sample=(f"whole user half-sweep of {m.name} ({m.M} x {m.N}, {m.nnz} ratings, "
                        f"D={m.D}), fp64, one thread, {dt:.1f} s"))


def heldout_leg(args, k, r, als, U, V, workload_name, reps=20):
    """Held-out predictions r_hat = u . v on a seeded sample of the stored positions (the
    degree distributions of both sides), timed over back-to-back launches of the predict
    kernel; plus the validation RMSE of the same pairs through the registered-set path."""
    import numpy as np
    import torch
    import workload

    n = r.nnz // args.heldout_share
    hu, hi, hr = workload.stored_pairs(r.row_ptr, r.col, r.val, n,
                                       workload.holdout_seed(k))
    dev = U.device
    du = torch.from_numpy(hu).to(dev)
    di = torch.from_numpy(hi).to(dev)
    pred = torch.empty(n, dtype=torch.float32, device=dev)
    als.predict(U, V, du, di, out=pred)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        als.predict(U, V, du, di, out=pred)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    als.set_holdout(hu, hi, hr)
    vr = als.holdout_rmse(U, V)
    # algorithmic bytes, compulsory accounting: per pair two 4-byte indices and the 4-byte
    # prediction written; every distinct user's and item's D-vector once. A gather of the
    # item's row per pair (the per-pair figure, also reported) overstates the bytes that
    # reach memory: the item table (625k rows) is largely served by the caches, and that
    # figure reached 100 % of HBM peak at D = 100.
    n_users = int(np.unique(hu).size)
    n_items = int(np.unique(hi).size)
    alg = n * 12 + (n_users + n_items) * 4 * r.D
    per_pair = n * (12 + 4 * r.D) + n_users * 4 * r.D
    achieved = alg / (ms * 1e-3) / 1e9
    log(f"held-out leg: {n} pairs, {ms:.4f} ms per launch, {achieved:.0f} GB/s algorithmic")
    cpu = None
    if args.cpu_seconds > 0:
        import oracle

        threads = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))
        Uh = U.cpu().numpy().astype(np.float64)
        Vh = V.cpu().numpy().astype(np.float64)
        oracle.predict(hu[:1000], hi[:1000], Uh, Vh, threads=threads)
        # whole passes over the pairs until about a second of host work has been timed
        passes, t0 = 0, time.perf_counter()
        while passes == 0 or time.perf_counter() - t0 < 1.0:
            oracle.predict(hu, hi, Uh, Vh, threads=threads)
            passes += 1
        dt = time.perf_counter() - t0
        cpu = dict(value=passes * n / dt, unit="pairs/s", cores=threads, kind="oracle",
                   sample=f"{passes} passes over all {n} pairs, fp64, {dt:.2f} s")
    return dict(metric="held-out predictions/sec", value=n / (ms * 1e-3), unit="pairs/s",
                pairs=n, launches=reps, ms_per_launch=ms,
                sample=(f"1/{args.heldout_share} of the stored positions of {r.name}, seeded, "
                        f"in CSR order; factors after the timed sweeps"),
                roofline=dict(bound="hbm", achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s",
                              frac=achieved / HBM_PEAK_GBS, kernel="k_predict",
                              alg_per_launch=alg, accounting="compulsory bytes",
                              per_pair_gather_bytes=per_pair,
                              traffic=measured_traffic(workload_name + "_heldout", "k_predict")),
                cpu_baseline=cpu, rmse_same_pairs=vr)


# BPMF Gibbs iteration: the usual hyperprior (mu0 = 0, beta0 = 2, W0 = I, nu0 = D) and a
# rating precision matching noise of standard deviation 10 on the 0..100 scale
GIBBS_ALPHA = 0.01
GIBBS_BETA0 = 2.0


class GibbsSteps:
    """Seeded variates for every Gibbs half-sweep of the run, generated on the device
    before the timed region, and the hyperparameter buffers of both sides."""

    def __init__(self, r, als, n_steps, seed):
        import numpy as np
        import torch

        D = r.D
        dev = torch.device("cuda:0")
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        rng = np.random.default_rng(seed)
        self.z, self.var = {}, {}
        for side, n in (("items", r.N), ("users", r.M)):
            als.set_nw_prior(side, np.zeros(D), GIBBS_BETA0, np.eye(D), float(D))
            self.z[side] = torch.randn((n_steps, n, D), generator=g, device=dev)
            nu_s = D + n
            self.var[side] = [tuple(torch.from_numpy(a).to(dev) for a in (
                rng.chisquare(nu_s - np.arange(D)), rng.normal(size=D * (D - 1) // 2),
                rng.normal(size=D))) for _ in range(n_steps)]
        self.mu = {s: torch.empty(D, dtype=torch.float64, device=dev) for s in self.z}
        self.Lam = {s: torch.empty((D, D), dtype=torch.float64, device=dev) for s in self.z}

    def half(self, als, side, k, fixed, out):
        chi2, offd, zmu = self.var[side][k]
        als.sample_hyper(side, out, chi2, offd, zmu, self.mu[side], self.Lam[side])
        als.gibbs_half_sweep(side, fixed, GIBBS_ALPHA, self.Lam[side], self.mu[side],
                             self.z[side][k], out)


# BPTF: the rating precision's prior W(w0, nu0) (one-dimensional Wishart), the chain's
# hyperprior (mean 1, as the time factors start around 1), and a typical alpha for the
# oracle baseline (noise of standard deviation 30 on the 0..100 scale)
BPTF_ALPHA_W0 = 1.0
BPTF_ALPHA_NU0 = 2.0
BPTF_ALPHA_TYPICAL = 1.0 / 900.0


class BPTFSteps:
    """Seeded variates of every BPTF iteration of the run (device tensors, and the host
    chi-square of each alpha draw), generated before the timed region; the hyperparameter
    buffers of the three modes."""

    def __init__(self, r, als, n_bins, n_steps, seed):
        import numpy as np
        import torch

        D = r.D
        dev = torch.device("cuda:0")
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        rng = np.random.default_rng(seed)
        self.z, self.var = {}, {}
        for mode, n, prior_side in (("items", r.N, "items"), ("users", r.M, "users"),
                                    ("bins", n_bins, "time")):
            als.set_nw_prior(prior_side, np.ones(D) if mode == "bins" else np.zeros(D),
                             GIBBS_BETA0, np.eye(D), float(D))
            self.z[mode] = torch.randn((n_steps, n, D), generator=g, device=dev)
            nu_s = D + n
            self.var[mode] = [tuple(torch.from_numpy(a).to(dev) for a in (
                rng.chisquare(nu_s - np.arange(D)), rng.normal(size=D * (D - 1) // 2),
                rng.normal(size=D))) for _ in range(n_steps)]
        self.chi2_alpha = rng.chisquare(BPTF_ALPHA_NU0 + r.nnz, size=n_steps)
        self.mu = {m: torch.empty(D, dtype=torch.float64, device=dev) for m in self.z}
        self.Lam = {m: torch.empty((D, D), dtype=torch.float64, device=dev) for m in self.z}
        self.alpha = None

    def mode(self, als, mode, k, U, V, T):
        if mode == "items":
            # the iteration starts with alpha and the three hyperparameter draws
            self.alpha = als.tensor_sample_alpha(U, V, T, BPTF_ALPHA_W0, self.chi2_alpha[k])
            for m, X in (("items", V), ("users", U), ("bins", T)):
                chi2, offd, zmu = self.var[m][k]
                als.sample_hyper("time" if m == "bins" else m, X, chi2, offd, zmu, self.mu[m],
                                 self.Lam[m])
        als.tensor_gibbs_half_sweep(mode, U, V, T, self.alpha, self.Lam[mode], self.mu[mode],
                                    self.z[mode][k])


def run_workload(args, k):
    """Warm-up and timed steps of workload k; returns the result record."""
    import numpy as np
    import torch

    import workload
    from paper_1108_2580_amd import ALS

    t_gen = time.perf_counter()
    r = workload.make_config(k)
    U0, V0 = workload.init_factors(r.M, r.N, r.D, r.init_seed)
    log(f"generated {r.name}: nnz={r.nnz} in {time.perf_counter() - t_gen:.1f} s")
    dev = torch.device("cuda:0")
    t_c = time.perf_counter()
    als = ALS(r.M, r.N, r.row_ptr, r.col, r.val, r.D)
    weights = None
    if args.weighted:
        weights = workload.rating_weights(r.nnz, workload.weight_seed(k))
        als.set_weights(weights)
    log(f"als_create (validation, upload, device CSC, schedules): "
        f"{time.perf_counter() - t_c:.1f} s; users {als.plan_stats('users')} "
        f"items {als.plan_stats('items')}")
    U = torch.from_numpy(U0).to(dev)
    V = torch.from_numpy(V0).to(dev)
    gibbs = GibbsSteps(r, als, args.warmup + args.steps, r.init_seed + 77) if args.gibbs else None
    sides = ("items", "users")
    T = bins = None
    bptf = None
    if args.tensor or args.bptf:
        t_b = time.perf_counter()
        nb = workload.N_TIME_BINS
        bins = workload.time_bins(r.row_ptr, nb, workload.time_seed(k))
        als.set_time_bins(nb, bins)
        rng = np.random.default_rng(r.init_seed + 99)
        T = torch.from_numpy((1.0 + 0.1 * rng.standard_normal((nb, r.D))).astype(np.float32)).to(dev)
        sides = ("items", "users", "bins")
        log(f"time bins ({nb}) and their layout: {time.perf_counter() - t_b:.1f} s")
        if args.bptf:
            bptf = BPTFSteps(r, als, nb, args.warmup + args.steps, r.init_seed + 88)

    def half(side, k):
        if bptf is not None:
            bptf.mode(als, side, k, U, V, T)
            return
        if args.tensor:
            als.tensor_half_sweep(side, U, V, T, r.lam)
            return
        fixed, out = (U, V) if side == "items" else (V, U)
        if gibbs is not None:
            gibbs.half(als, side, k, fixed, out)
        else:
            als.half_sweep(side, fixed, r.lam, out)

    for w in range(args.warmup):
        for side in sides:
            half(side, w)
        torch.cuda.synchronize()
        log(f"warmup {w + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    # the timed sweeps carry event records only around the kernels that build the normal
    # equations (the roofline's kernels); each record costs about 3 us of stream time
    als.set_profiling(True, gram_only=True)
    # HIP events around each half-sweep on the stream the library enqueues on
    ev = {side: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in range(args.steps)] for side in sides}
    t0 = time.perf_counter()
    for k in range(args.steps):
        for side in sides:
            ev[side][k][0].record()
            half(side, args.warmup + k)
            ev[side][k][1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    per_side = {}
    for side in sides:
        ms = sorted(a.elapsed_time(b) for a, b in ev[side])
        med = ms[len(ms) // 2] if len(ms) % 2 else 0.5 * (ms[len(ms) // 2 - 1] + ms[len(ms) // 2])
        per_side[side] = {"ms_median": med, "ms_min": ms[0], "ratings_per_s": r.nnz / (med * 1e-3)}
    prof = als.profile()
    als.set_profiling(False)
    elapsed = t1 - t0
    rmse_in = als.rmse_in()
    rmse = als.tensor_rmse(U, V, T) if (args.tensor or args.bptf) else als.rmse(U, V)
    # every phase's time, on extra untimed sweeps with events around every launch
    prof_all = None
    if args.phase_sweeps > 0:
        als.set_profiling(True)
        for _ in range(args.phase_sweeps):
            for side in sides:
                half(side, args.warmup + args.steps - 1)
        prof_all = als.profile()
        als.set_profiling(False)
    gram_share = phase_cycles = None
    if r.D > 20 and not (args.tensor or args.bptf):
        # one extra, untimed half-sweep per side with the row kernel's phase clocks on
        als.set_phase_timing(True)
        half("items", args.warmup + args.steps - 1)
        half("users", args.warmup + args.steps - 1)
        gi, si = als.phase_cycles("items")
        gu, su = als.phase_cycles("users")
        als.set_phase_timing(False)
        gram_share = (gi + gu) / max(gi + si + gu + su, 1.0)
        rows_i = als.plan_stats("items")["rows_with_ratings"]
        rows_u = als.plan_stats("users")["rows_with_ratings"]
        # mean wavefront clock cycles per row in each phase (both waves of a SIMD share it)
        phase_cycles = {"items": {"gram": gi / max(rows_i, 1), "solve": si / max(rows_i, 1)},
                        "users": {"gram": gu / max(rows_u, 1), "solve": su / max(rows_u, 1)}}
    log(f"timed {args.steps} sweeps in {elapsed:.3f} s; timed kernels (ms total, launches): "
        f"{prof}; phases of {args.phase_sweeps} extra sweeps: {prof_all}; "
        f"rmse entering last half-sweep {rmse_in}, final {rmse:.6f}")

    value = len(sides) * r.nnz * args.steps / elapsed
    halves = len(sides) * args.steps
    rows_with = als.plan_stats("users")["rows_with_ratings"] + \
        als.plan_stats("items")["rows_with_ratings"]
    if args.tensor:
        rows_with += int(np.unique(bins).size)
    if args.bptf:
        # every user, item and bin is drawn (rows without ratings from their priors)
        rows_with = r.M + r.N + workload.N_TIME_BINS
    D = r.D
    workload_name = r.name + ("_wals" if args.weighted else "_bpmf" if args.gibbs else
                              "_tensor" if args.tensor else "_bptf" if args.bptf else "")
    tensor_like = args.tensor or args.bptf
    dominant = max(prof_all or prof, key=lambda k: (prof_all or prof)[k][0])
    # per rating: a weight (weighted ALS); the second index and second gathered row, and
    # the product of the two rows (tensor ALS)
    wbytes = 4 if args.weighted else (4 + 4 * D) if tensor_like else 0
    wflops = D if (args.weighted or tensor_like) else 0
    if D <= 20:
        # gather kernel: per rating the index, the rating (and weight) and the gathered fixed
        # row; per solved row the row pointer and the entering value
        k_ms, k_n = prof["gather"]
        alg = halves * r.nnz * (5 + wbytes + 4 * D) + args.steps * rows_with * (8 + 4 * D)
        if tensor_like:
            # per step: every rating twice with one large gathered row (the user and item
            # modes) and once with two (the time-bin mode), plus both indices and the rating
            # each time; the time-bin table (6649 rows) once per user and item mode
            alg = args.steps * (r.nnz * (27 + 16 * D) + 2 * workload.N_TIME_BINS * 4 * D
                                + rows_with * (8 + 4 * D))
        achieved = alg / (k_ms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=achieved, peak=HBM_PEAK_GBS, unit="GB/s",
                    frac=achieved / HBM_PEAK_GBS, kernel="k_gram_ne",
                    whole_step_frac=alg / elapsed / 1e9 / HBM_PEAK_GBS)
    else:
        # fused row kernel + chunk kernel of split rows, priced on the Gram build alone: the
        # SYRK-convention Gram flops D (D + 1) and the right-hand side 2 D per rating (plus
        # the weight or the second factor's product). The residual dot and the Cholesky
        # with its two solves run in the same kernels but are not counted here; the
        # factorisation's own flops are reported beside it.
        k_ms = prof["solve"][0] + prof["gather"][0]
        k_n = prof["solve"][1]
        alg = halves * r.nnz * (D * (D + 1) + 2 * D + wflops)
        achieved = alg / (k_ms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=achieved, peak=MFMA_F32_PEAK_TFS, unit="TFLOP/s",
                    frac=achieved / MFMA_F32_PEAK_TFS, kernel="k_rows+k_gram_chunks",
                    flops="SYRK Gram + right-hand side per rating",
                    whole_step_frac=alg / elapsed / 1e12 / MFMA_F32_PEAK_TFS,
                    chol_flops_per_step=rows_with * (D ** 3 / 3.0 + 2.0 * D * D))
    roof.update(launches=k_n, avg_launch_ms=k_ms / max(k_n, 1), alg_per_launch=alg / max(k_n, 1),
                traffic=measured_traffic(workload_name, roof["kernel"]), dominant_phase=dominant)
    gram_phase = None
    if gram_share is not None:
        # Gram phase: the chunk kernel plus the share of the fused row kernel's wavefront
        # time spent before the factorisation (gather, Gram, RHS, residuals); flops in
        # the SYRK convention plus the right-hand side
        g_ms = (prof["gather"][0] + gram_share * prof["solve"][0]) / args.steps
        g_flops = 2 * r.nnz * (D * (D + 1) + 2 * D + wflops)
        g_tf = g_flops / (g_ms * 1e-3) / 1e12
        gram_phase = dict(ms_per_step=g_ms, flops_per_step=g_flops, achieved=g_tf,
                          peak=MFMA_F32_PEAK_TFS, unit="TFLOP/s", frac=g_tf / MFMA_F32_PEAK_TFS,
                          row_kernel_gram_share=gram_share,
                          cycles_per_row=phase_cycles,
                          method="chunk-kernel time plus the row kernel's time scaled by the "
                                 "share of wavefront clock cycles before the factorisation")

    # (the held-out leg scores u . v pairs: the matrix model's prediction, so not for the
    # three-way models)
    # the factorisation and triangular solves on their own: the one-lane solve kernel at
    # D <= 20; at D > 20 the fused row kernel's time scaled by the share of its wavefront
    # cycles from the factorisation on (phase clocks; plain ALS and BPMF)
    if D <= 20:
        chol_ms = prof_all["solve"][0] / args.phase_sweeps if prof_all else None
    elif gram_share is not None:
        chol_ms = (1.0 - gram_share) * prof["solve"][0] / args.steps
    else:
        chol_ms = None
    heldout = (heldout_leg(args, k, r, als, U, V, workload_name)
               if args.heldout_share > 0 and not tensor_like else None)

    cpu = None
    if args.cpu_seconds > 0:
        log("cpu baseline: fp64 oracle on a sample of the user half-sweep ...")
        cpu = cpu_baseline(r, V.cpu().numpy(), args.cpu_seconds, weights,
                           gibbs=args.gibbs or args.bptf,
                           tensor=(bins, T.cpu().numpy()) if tensor_like else None)
        if not (args.weighted or args.gibbs or tensor_like):
            cpu["one_thread"] = one_thread_scale()
        log(f"cpu baseline: {cpu}")

    out = {
        "metric": ("wALS" if args.weighted else "BPMF Gibbs" if args.gibbs else
                   "tensor ALS" if args.tensor else "BPTF Gibbs" if args.bptf else "ALS")
        + " ratings/sec per half-sweep",
        "value": value,
        "unit": "ratings/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload_name, "n_users": r.M, "n_items": r.N, "nnz": r.nnz, "D": r.D,
                   "weights": ("per rating, log-uniform on [0.25, 4), seeded" if args.weighted
                               else None),
                   "lambda": None if (args.gibbs or args.bptf) else r.lam,
                   "gibbs": (dict(alpha=GIBBS_ALPHA, mu0=0.0, beta0=GIBBS_BETA0, W0="I",
                                  nu0=r.D, variates="seeded, on the device before timing")
                             if args.gibbs else
                             dict(alpha_prior=dict(w0=BPTF_ALPHA_W0, nu0=BPTF_ALPHA_NU0),
                                  mu0="0 (users, items), 1 (time chain)", beta0=GIBBS_BETA0,
                                  W0="I", nu0=r.D, variates="seeded, on the device before timing")
                             if args.bptf else None),
                   "time_bins": workload.N_TIME_BINS if tensor_like else None,
                   "step": ("item side (hyperparameter draw, row draws) + user side"
                            if args.gibbs else "item, user and time-bin mode updates"
                            if args.tensor else
                            "alpha and three hyperparameter draws, then item, user and "
                            "time-bin (even, then odd) draws" if args.bptf else
                            "item half-sweep + user half-sweep"),
                   "parallelism": "single GPU"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "per_side": per_side,
        "gram_phase": gram_phase,
        "chol_ms_per_step": chol_ms,
        "phases_ms_per_step": ({k: v[0] / args.phase_sweeps for k, v in prof_all.items()}
                               if prof_all else None),
        "rmse": rmse,
        "rmse_entering_last_half_sweep": rmse_in,
        "heldout": heldout,
    }
    als.close()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              f"(the half-sweep would shard by rows with an all-gather of the solved side).",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    special = args.weighted or args.gibbs or args.tensor or args.bptf
    out = run_workload(args, args.config or 3)
    if args.config is None and not special:
        # the headline's second width: the same matrix at D = 100, on the fp32 matrix cores
        log("d100 leg: the same matrix at D = 100")
        leg = run_workload(args, 4)
        out["d100"] = {key: leg[key] for key in (
            "value", "unit", "ms_per_step", "config", "roofline", "gram_phase",
            "chol_ms_per_step", "per_side", "phases_ms_per_step", "cpu_baseline", "rmse",
            "rmse_entering_last_half_sweep", "heldout")}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

"""Throughput of one EigenPro 2.0 iteration on one MI355X.

A step is one call of ep_step: gather the batch, the fused kernel-block
contraction F = K(X_t, X) alpha, residual and batch-block update, the
subsample correction K(X_r, X_t) R through the same fused kernel, and the
rank-k update of the fixed block (Algorithm 1 steps 1-5).

Default workload: the ImageNet-feature-shaped synthetic problem (n = 1.28M
centres, d = 2048, l = 1000 one-hot labels, Gaussian bandwidth 20, s = 20000,
k = 200, batch = the analytic m*). Inputs are generated on the host, uploaded
once, and are resident in HBM before timing starts.

Prints one JSON line. ``value`` is kernel entries per second (m * n per
step over the wall time of the timed steps).
"""

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3     # MI355X dense fp32 matrix peak
PEAK_HBM_GBS = 8000.0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


KERNEL_SOURCES = {"kmv_kernel": ["kmv.hip", "ep_device.h"],
                  "kblock_kernel": ["kblock.hip", "ep_device.h"]}


def code_text(src):
    """C++ source with its comments removed and blank space collapsed, so
    that a measurement stays attached to the code it measured when only
    comments change (no string literal in the kernel sources holds a
    comment marker)."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def kernel_source_sha(kernel="kmv_kernel"):
    """sha256[:16] of the kernel's code (comments and blank space removed)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_1806_06144_amd", "csrc", name)) as f:
            h.update(code_text(f.read()).encode())
        h.update(b"\0")
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel="kmv_kernel"):
    """HBM bytes per launch of the dominant kernel from committed rocprofv3
    counter runs, if they were taken on the current kernel source, and where
    the figure comes from: (bytes or None, provenance dict)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    key = f"{workload} | {kernel}"
    prov = {"record": "profiles/hbm_traffic.json", "key": key,
            "kernel_source_sha": kernel_source_sha(kernel),
            "measured_with": "rocprofv3 --pmc FETCH_SIZE and --pmc WRITE_SIZE runs of bench.py "
                             "(counters calibrated against 1 GiB device copies); not this run"}
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None, dict(prov, status="no record")
    entry = rec.get(key)
    if not entry:
        return None, dict(prov, status="no record for this workload")
    if entry.get("source_sha") != prov["kernel_source_sha"]:
        return None, dict(prov, status=f"record taken on other kernel code ({entry.get('source_sha')})")
    return entry.get("bytes_per_launch"), dict(prov, status="record matches the kernel code")


def host_cores():
    """(physical cores by lscpu, CPUs this process may run on, the
    OMP_NUM_THREADS cap or None)."""
    import subprocess
    phys = None
    try:
        out = subprocess.run(["lscpu", "-p=SOCKET,CORE"], capture_output=True, text=True,
                             timeout=20).stdout
        pairs = {line.strip() for line in out.splitlines() if line and not line.startswith("#")}
        phys = len(pairs) or None
    except (OSError, subprocess.SubprocessError):
        phys = None
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS")
    omp = int(omp) if omp and omp.isdigit() else None
    return phys, nproc, omp


def timing_state(X, cfg, seed=0):
    """An oracle state for timing oracle.step on the workload: the
    workload's subsample and shapes, with a seeded orthonormal s x k basis
    and a decreasing spectrum standing in for the eigensystem (the step's
    arithmetic, and so its time, does not depend on their values; the
    oracle's own eigensolve is a setup cost, not part of a step)."""
    import oracle
    import synth
    n = X.shape[0]
    r = synth.subsample_indices(cfg, seed, n=n)
    rng = np.random.default_rng(seed + 99)
    V = np.linalg.qr(rng.standard_normal((cfg.s, cfg.k)))[0] if cfg.k else np.zeros((cfg.s, 0))
    sigma = cfg.s * 0.5 * 0.98 ** np.arange(cfg.k + 1)
    D = (1.0 - sigma[cfg.k] / sigma[:cfg.k]) / sigma[:cfg.k]
    beta = oracle.beta_closed_form(sigma, V)
    lam = sigma[cfg.k] / cfg.s
    m_star = beta / lam
    return oracle.OracleState(X, cfg.kernel_id, float(cfg.bandwidth), r,
                              np.asarray(X[r], dtype=np.float64), sigma, V, D, float(beta),
                              float(lam), float(m_star), int(min(n, max(1, np.floor(m_star)))))


def _timed_rows(fn, n_rows_max, target_s, start=32):
    """Run fn(rows) with a growing row count until one call takes about
    target_s; returns (rows, seconds) of the last call. Each call pays a
    per-centre cost as well as a per-row one, so time grows more slowly
    than the row count and two rescales bring the call near the target."""
    rows = min(start, n_rows_max)
    dt = fn(rows)
    for _ in range(3):
        if dt >= 0.6 * target_s:
            break
        grown = int(min(n_rows_max, rows * target_s / max(dt, 1e-3)))
        if grown <= rows:
            break
        rows = grown
        dt = fn(rows)
    return rows, dt


def cpu_baseline(X, alpha_host, cfg, m, configs=("tiny", "mnist", "cifar", "timit"),
                 target_s=8.0):
    """The float64 oracle timed on the host cores with BLAS pinned to the
    physical core count (capped by the CPUs and OMP_NUM_THREADS this process
    may use): a whole oracle.step (Algorithm 1 steps 1-5) on a bounded batch
    of the headline workload, step 2 alone (F = K(X_t, X) alpha) on it, and
    a whole step on each other workload, each reported as kernel entries per
    second (batch rows x n over the call's time)."""
    import oracle
    import synth
    from threadpoolctl import threadpool_limits

    phys, nproc, omp = host_cores()
    cores = min(x for x in (phys, nproc, omp) if x)
    rng = np.random.default_rng(123)
    out = {"unit": "entries/s", "kind": "oracle", "cores": int(cores),
           "physical_cores": phys, "nproc": nproc, "omp_num_threads": omp}
    with threadpool_limits(limits=cores):
        st = timing_state(X, cfg)
        y_of = lambda t: np.zeros((len(t), alpha_host.shape[1]))

        def whole(rows, st=st, alpha=alpha_host):
            t = rng.choice(st.n, rows, replace=False)
            t0 = time.perf_counter()
            oracle.step(st, alpha, t, y_of(t))
            return time.perf_counter() - t0

        def step2(rows):
            Q = X[rng.choice(X.shape[0], rows, replace=False)]
            t0 = time.perf_counter()
            oracle.predict(X, alpha_host, Q, cfg.kernel_id, cfg.bandwidth)
            return time.perf_counter() - t0

        rows, dt = _timed_rows(whole, min(m, X.shape[0]), 2.0 * target_s)
        n = X.shape[0]
        out["value"] = rows * n / dt
        # an epoch is ceil(n/m) steps of m rows; a step's time is close to
        # linear in its rows (its F and G parts are), so the measured rate
        # carries over to the full batch
        out["s_per_epoch_extrapolated"] = -(-n // m) * dt * (m / rows)
        out["sample"] = (f"oracle.step (Algorithm 1 steps 1-5, float64) on {rows} batch rows of "
                         f"the {cfg.name}-shaped workload (n={n}, d={X.shape[1]}, l={cfg.l}, "
                         f"s={cfg.s}, k={cfg.k}): {dt:.1f} s; the eigensystem is a seeded "
                         f"stand-in (time does not depend on it)")
        rows2, dt2 = _timed_rows(step2, min(m, X.shape[0]), target_s)
        out["step2_value"] = rows2 * n / dt2
        out["step2_sample"] = f"oracle F = K(X_t, X) alpha for {rows2} rows: {dt2:.1f} s"
        per = []
        for name in configs:
            c = synth.get_config(name)
            Xc = synth.features(c, 0)
            stc = timing_state(Xc, c)
            ac = synth.initial_alpha(c.n, c.l, 0)

            def whole_c(rows, stc=stc, ac=ac):
                t = rng.choice(stc.n, rows, replace=False)
                t0 = time.perf_counter()
                oracle.step(stc, ac, t, np.zeros((rows, c.l)))
                return time.perf_counter() - t0

            rc_, dc_ = _timed_rows(whole_c, min(4096, c.n), target_s / 2)
            per.append({"workload": name, "n": c.n, "d": c.d, "l": c.l, "s": c.s, "k": c.k,
                        "batch_rows": rc_, "step_s": dc_, "value": rc_ * c.n / dc_})
            del Xc, stc, ac
        out["per_config"] = per
    return out


def _time_steps(ep, torch, ctx, stream, tl, yl):
    """Median HIP-event time (ms) of ep_step over the given device batches,
    on the library's stream (torch's current stream here)."""
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(tl) + 1)]
    evs[0].record(stream)
    for i, (tb, yb) in enumerate(zip(tl, yl)):
        ep.ep_step(ctx, tb, tb.shape[0], yb)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    return float(np.median([evs[i].elapsed_time(evs[i + 1]) for i in range(len(tl))]))


def study_batch(args):
    """Synthetic analogue of the paper's batch-size / GPU-utilisation study
    (Section 5, Figure 4): time per iteration (a whole ep_step, Algorithm 1
    steps 1-5) and per step-2 pass against batch size on a TIMIT-shaped
    problem (n = 1e5, d = 440, l = 144), the resource batch of Section 3
    Step 1 (the knee of that curve), the Eq. 7 rank for it, and time per
    epoch against n at that batch."""
    import torch
    import synth
    import paper_1806_06144_amd as ep
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    base = synth.get_config("timit")
    out = []
    cfg = synth.get_config("timit", n=100000, s=4000, k=400)
    X = synth.features(cfg, 0)
    labels = synth.class_labels(cfg, X, 0)
    Xd = torch.from_numpy(X).to(dev)
    ctx, info = ep.ep_setup(Xd, cfg.n, cfg.d, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s, cfg.k,
                            sub_idx=synth.subsample_indices(cfg, 0), stream=stream)
    ms = [2 ** j for j in range(4, 15)]
    t = ep.ep_batch_sweep(ctx, ms, reps=3)
    alpha0 = torch.zeros((cfg.n, cfg.l), dtype=torch.float32, device=dev)
    perm = synth.epoch_permutation(cfg.n, 0)
    for m, tm in zip(ms, t):
        # whole iterations on distinct batches of this size, from alpha = 0
        # each time (the timing does not depend on alpha)
        reps = 5
        tl = [torch.from_numpy(perm[(i * m) % cfg.n:(i * m) % cfg.n + m].copy()).to(dev)
              for i in range(reps)]
        tl = [x if x.shape[0] == m else torch.from_numpy(perm[:m].copy()).to(dev) for x in tl]
        yl = [torch.from_numpy(synth.one_hot(labels[x.cpu().numpy()], cfg.l)).to(dev) for x in tl]
        ep.ep_set_alpha(ctx, alpha0)
        ep.ep_step(ctx, tl[0], m, yl[0])
        step_ms = _time_steps(ep, torch, ctx, stream, tl, yl)
        rec = {"study": "time_per_iteration_vs_batch", "n": cfg.n, "d": cfg.d, "l": cfg.l,
               "m": m, "step_ms": step_ms, "fused_pass_ms": tm,
               "entries_per_s": m * cfg.n / (step_ms * 1e-3)}
        out.append(rec)
        log(json.dumps(rec))
    ep.ep_set_alpha(ctx, alpha0)
    m_C, m_S, m_G = ep.ep_resource_batch(ctx, 0.1)
    m_C2 = ep.ep_resource_batch(ctx, 0.1)[0]
    _, knee = ep.ep_batch_knee(ms, t, 0.1)
    ep.ep_set_rank(ctx, 0)
    mstar0 = ep.ep_get_info(ctx).m_star
    ad = ep.ep_adapt(ctx, m_G)
    rec = {"study": "resource_adaptive", "n": cfg.n, "k_max": cfg.k, "m_C": m_C,
           "m_C_second_call": m_C2, "knee_of_this_sweep": knee, "m_S": m_S, "m_G": m_G,
           "chosen_k": ad.k, "m_star_original": mstar0, "m_star_adapted": ad.m_star,
           "beta_adapted": ad.beta, "sigma_1": ad.sigma_1, "sigma_k1": ad.sigma_k1,
           "acceleration": ad.accel, "step_eta": ad.eta}
    out.append(rec)
    log(json.dumps(rec))
    ep.ep_destroy(ctx)
    del Xd
    torch.cuda.empty_cache()
    # time per epoch against n at the adapted batch and rank
    for n in [25000, 100000, 400000, base.n]:
        c = synth.get_config("timit", n=n, s=4000, k=ad.k)
        Xn = synth.features(c, 0)
        labels = synth.class_labels(c, Xn, 0)
        Xd = torch.from_numpy(Xn).to(dev)
        ctx, inf = ep.ep_setup(Xd, c.n, c.d, c.l, c.kernel, c.bandwidth, c.s, c.k,
                               sub_idx=synth.subsample_indices(c, 0))
        m = min(n, m_G)
        batches = synth.epoch_batches(n, m, 0)
        tl = [torch.from_numpy(b).to(dev) for b in batches]
        yl = [torch.from_numpy(synth.one_hot(labels[b], c.l)).to(dev) for b in batches]
        ep.ep_step(ctx, tl[0], len(batches[0]), yl[0])
        ep.ep_sync(ctx)
        t0 = time.perf_counter()
        for tb, yb, b in zip(tl, yl, batches):
            ep.ep_step(ctx, tb, len(b), yb)
        ep.ep_sync(ctx)
        dt = time.perf_counter() - t0
        rec = {"study": "time_per_epoch_vs_n", "n": n, "m": m, "k": c.k, "steps": len(batches),
               "epoch_s": dt}
        out.append(rec)
        log(json.dumps(rec))
        ep.ep_destroy(ctx)
        del Xd, tl, yl
        torch.cuda.empty_cache()
    return out


def _train_to(ep, torch, ctx, Xd, Y, n, m, thr, max_epochs, budget_s, first_epoch=0):
    """Epochs of Algorithm 1 from alpha = 0 at batch m until the training
    MSE (mean over points and labels) falls below thr, or a cap; returns
    (epochs, step seconds, final MSE)."""
    import synth
    dev = Xd.device
    P = torch.empty_like(Y)

    def mse():
        ep.ep_predict(ctx, Xd, n, P)
        ep.ep_sync(ctx)
        return float(((P - Y) ** 2).mean())

    ep.ep_set_alpha(ctx, torch.zeros_like(Y))
    gpu_s, epochs, err = 0.0, 0, mse()
    while err >= thr and epochs < max_epochs and gpu_s < budget_s:
        batches = synth.epoch_batches(n, m, first_epoch + epochs)
        tl = [torch.from_numpy(b).to(dev) for b in batches]
        yl = [Y[b] for b in tl]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for tb, yb in zip(tl, yl):
            ep.ep_step(ctx, tb, tb.shape[0], yb)
        ep.ep_sync(ctx)
        gpu_s += time.perf_counter() - t0
        epochs += 1
        err = mse()
    return epochs, gpu_s, err


def study_convergence(args):
    """Synthetic analogue of the paper's convergence comparison (Section 5,
    Figure 3): epochs and GPU time to bring the training MSE (mean over
    points and labels) below a threshold, against batch size m, for plain
    kernel SGD (rank 0, its own optimal step) and EigenPro 2.0 with the
    kernel adapted to the batch (the Eq. 7 rank for m_G = m, the step size
    of Section 3 Step 3). TIMIT-shaped problem with n = 1e5 and
    threshold 2e-4 (--study convergence), or the MNIST-shaped workload at
    its full size with threshold 1e-4 (--study convergence-mnist, the
    paper's threshold for its MNIST curves)."""
    import torch
    import synth
    import paper_1806_06144_amd as ep
    dev = torch.device("cuda:0")
    if args.study == "convergence-mnist":
        cfg = synth.get_config("mnist", s=4000, k=400)
        thr, max_epochs, budget_s = 1e-4, 200, 30.0
    else:
        cfg = synth.get_config("timit", n=100000, s=4000, k=400)
        thr, max_epochs, budget_s = 2e-4, 40, 60.0
    X = synth.features(cfg, 0)
    labels = synth.class_labels(cfg, X, 0)
    Xd = torch.from_numpy(X).to(dev)
    Y = torch.from_numpy(synth.one_hot(labels, cfg.l)).to(dev)
    ctx, info = ep.ep_setup(Xd, cfg.n, cfg.d, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s, cfg.k,
                            sub_idx=synth.subsample_indices(cfg, 0))
    _, _, m_G = ep.ep_resource_batch(ctx, 0.1)
    k_G = ep.ep_adapt(ctx, m_G).k
    out = []
    for method in ("sgd", "eigenpro"):
        for m in (64, 256, 1024, 4096):
            if method == "sgd":
                ep.ep_set_rank(ctx, 0)
            else:
                ep.ep_adapt(ctx, m)
            inf = ep.ep_get_info(ctx)
            epochs, gpu_s, err = _train_to(ep, torch, ctx, Xd, Y, cfg.n, m, thr, max_epochs,
                                           budget_s)
            rec = {"study": "convergence", "workload": cfg.name, "n": cfg.n, "method": method,
                   "k": inf.k, "m_star": inf.m_star, "m": m, "epochs": epochs,
                   "step_time_s": gpu_s, "train_mse": err, "threshold": thr,
                   "converged": err < thr, "m_G": m_G, "k_at_m_G": k_G}
            out.append(rec)
            log(json.dumps(rec))
    ep.ep_destroy(ctx)
    return out


def study_kernels(args):
    """The paper's remarks on the kernel function (Section 5): with the
    Laplacian kernel training takes fewer epochs, and its critical batch m*
    is larger, than with the Gaussian. Same TIMIT-shaped data (n = 1e5,
    d = 440, l = 144), same bandwidth 15 (Table 5's TIMIT row uses the
    Laplacian kernel at 15), same subsample; for each kernel: m* at ranks
    0, 1, 10, 100 and 400 (Section 3 Step 2), and epochs and GPU time to
    training MSE < 2e-4 for plain kernel SGD at m = 64 and for EigenPro 2.0
    at m = 4096 with the kernel adapted to that batch (Eq. 7)."""
    import torch
    import synth
    import paper_1806_06144_amd as ep
    dev = torch.device("cuda:0")
    cfg = synth.get_config("timit", n=100000, s=4000, k=400)
    X = synth.features(cfg, 0)
    labels = synth.class_labels(cfg, X, 0)
    Xd = torch.from_numpy(X).to(dev)
    Y = torch.from_numpy(synth.one_hot(labels, cfg.l)).to(dev)
    r = synth.subsample_indices(cfg, 0)
    out = []
    for kernel in ("gaussian", "laplacian"):
        ctx, info = ep.ep_setup(Xd, cfg.n, cfg.d, cfg.l, kernel, cfg.bandwidth, cfg.s, cfg.k,
                                sub_idx=r)
        mstar = {}
        for k in (0, 1, 10, 100, 400):
            ep.ep_set_rank(ctx, k)
            mstar[str(k)] = ep.ep_get_info(ctx).m_star
        ep.ep_set_rank(ctx, 0)
        sgd = _train_to(ep, torch, ctx, Xd, Y, cfg.n, 64, 2e-4, 40, 60.0)
        ad = ep.ep_adapt(ctx, 4096)
        epro = _train_to(ep, torch, ctx, Xd, Y, cfg.n, ad.m, 2e-4, 40, 60.0)
        rec = {"study": "kernel_choice", "kernel": kernel, "bandwidth": cfg.bandwidth,
               "n": cfg.n, "sigma_1": info.sigma_1, "m_star_by_rank": mstar,
               "sgd_m": 64, "sgd_epochs": sgd[0], "sgd_step_s": sgd[1], "sgd_mse": sgd[2],
               "eigenpro_m": ad.m, "eq7_rank": ad.k, "m_star_adapted": ad.m_star,
               "eigenpro_epochs": epro[0], "eigenpro_step_s": epro[1], "eigenpro_mse": epro[2],
               "threshold": 2e-4}
        out.append(rec)
        log(json.dumps(rec))
        ep.ep_destroy(ctx)
    return out


def study_setup(args):
    """Setup eigensolve at the subsample size and rank of each workload:
    the full divide-and-conquer eigendecomposition against the
    Chebyshev-filtered subspace iteration (both float64 on the device), on
    s rows drawn from the workload's law (taken as the subsample), with the
    largest eigenvalue difference and the V D V^T difference between them."""
    import torch
    import synth
    import paper_1806_06144_amd as ep
    dev = torch.device("cuda:0")
    out = []
    for name in ["mnist", "cifar", "timit", "imagenet"]:
        base = synth.get_config(name)
        cfg = synth.get_config(name, n=base.s)
        X = synth.features(cfg, 0)
        Xd = torch.from_numpy(X).to(dev)
        r = np.arange(cfg.s, dtype=np.int64)
        res = {}
        for solver in ["dense", "subspace", "dense", "subspace"]:    # second pass timed warm
            ctx, info = ep.ep_setup_ex(Xd, cfg.n, cfg.d, cfg.l, cfg.kernel, cfg.bandwidth,
                                       cfg.s, cfg.k, sub_idx=r,
                                       opts={"solver": solver, "no_fallback": 1})
            sigma, D, V, _ = ep.ep_get_preconditioner(ctx, info)
            ep.ep_destroy(ctx)
            res[solver] = (info, sigma, (V.astype(np.float64) * D) @ V.T.astype(np.float64))
        (i_d, s_d, L_d), (i_s, s_s, L_s) = res["dense"], res["subspace"]
        rec = {"study": "setup_eigensolver", "workload": name, "s": cfg.s, "d": cfg.d,
               "k": cfg.k, "kernel": cfg.kernel,
               "dense_setup_ms": i_d.setup_ms, "subspace_setup_ms": i_s.setup_ms,
               "speedup": i_d.setup_ms / i_s.setup_ms,
               "subspace_iters": i_s.solver_iters, "subspace_matvecs": i_s.solver_matvecs,
               "subspace_eig_residual": i_s.eig_residual,
               "max_rel_sigma_diff": float(np.max(np.abs(s_s - s_d) / s_d)),
               "lowrank_rel_diff": float(np.linalg.norm(L_s - L_d) / np.linalg.norm(L_d)),
               "sigma_1": i_s.sigma_1, "sigma_k1": i_s.sigma_k1}
        out.append(rec)
        log(json.dumps(rec))
        del Xd
        torch.cuda.empty_cache()
    return out


def traffic_summary(fetch_csv, write_csv, workload, kernel, n_step, command_note,
                    out_path=os.path.join(ROOT, "profiles", "hbm_traffic.json")):
    """HBM bytes per launch of the dominant kernel from two rocprofv3 --pmc
    runs (FETCH_SIZE, WRITE_SIZE; KiB per dispatch), each scaled by what the
    same counter reads for the 1 GiB device copies of --calibrate-copy.
    Only the kernel's first n_step dispatches count: those of the warm-up
    and timed steps, whose launches the roofline averages (the prediction
    pass that follows runs the same kernel on other shapes).
    Writes profiles/hbm_traffic.json and returns a text summary."""
    import csv

    def per_kernel(path, counter):
        out = {}
        with open(path, newline="") as f:
            for row in csv.DictReader(f):
                if row["Counter_Name"] != counter:
                    continue
                name = row["Kernel_Name"]
                key = ("kmv_kernel" if "kmv_kernel<" in name else
                       "kmv_subsample_kernel" if "kmv_subsample_kernel<" in name else
                       "kblock_kernel" if "kblock_kernel<" in name else
                       "copy" if "copyBuffer" in name and float(row["Counter_Value"]) > (1 << 18) else
                       None)
                if key:
                    out.setdefault(key, []).append(float(row["Counter_Value"]))
        return out

    fe = per_kernel(fetch_csv, "FETCH_SIZE")
    wr = per_kernel(write_csv, "WRITE_SIZE")
    fe[kernel], wr[kernel] = fe[kernel][:n_step], wr[kernel][:n_step]
    if len(fe[kernel]) != n_step or len(wr[kernel]) != n_step:
        raise SystemExit(f"expected {n_step} {kernel} dispatches in each counter run")
    gib_kib = float(1 << 20)
    rf = gib_kib / np.mean(fe["copy"])
    wf = gib_kib / np.mean(wr["copy"])
    f_kib, w_kib = np.mean(fe[kernel]), np.mean(wr[kernel])
    bytes_launch = (f_kib * rf + w_kib * wf) * 1024.0
    rec = {}
    path = out_path
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        rec = {}
    rec[f"{workload} | {kernel}"] = {
        "source_sha": kernel_source_sha(kernel), "bytes_per_launch": bytes_launch,
        "fetch_kib": f_kib, "write_kib": w_kib, "read_factor": rf, "write_factor": wf}
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
    lines = [f"workload: {workload}", f"kernel: {kernel}",
             f"kernel code sha256[:16] (comments removed): {kernel_source_sha(kernel)}", "",
             command_note, "",
             f"per-dispatch counter values (KiB; {kernel}: its first {n_step} dispatches, "
             "those of the warm-up and timed steps):"]
    for key in [kernel, "kmv_subsample_kernel", "copy"]:
        if not fe.get(key) and not wr.get(key):
            continue
        lines.append(f"  {key:21s} FETCH_SIZE " + ", ".join(f"{v:.6g}" for v in fe.get(key, [])))
        lines.append(f"  {key:21s} WRITE_SIZE " + ", ".join(f"{v:.6g}" for v in wr.get(key, [])))
    lines += ["", "calibration: a 1 GiB copy reads and writes 1048576 KiB;",
              f"  read factor  = 1048576 / {np.mean(fe['copy']):.6g} = {rf:.4f}",
              f"  write factor = 1048576 / {np.mean(wr['copy']):.6g} = {wf:.4f}", "",
              f"{kernel} traffic per launch = ({f_kib:.6g} * {rf:.4f} + {w_kib:.6g} * {wf:.4f}) KiB",
              f"    = {bytes_launch / 1e9:.2f} GB"]
    return "\n".join(lines)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="imagenet")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--contraction", choices=["auto", "fused", "blocked"], default="auto",
                    help="form of F = K(X_t, X) alpha timed for the headline (ep_set_contraction)")
    ap.add_argument("--blocked-compare", action="store_true",
                    help="also time the opt-in blocked form (kernel block written per centre "
                         "chunk) on the same batches, after the headline")
    ap.add_argument("--no-blocked-compare", dest="blocked_compare", action="store_false",
                    help="do not time the blocked form (the default)")
    ap.add_argument("--s", type=int, default=None,
                    help="override the subsample size (experiments only)")
    ap.add_argument("--shard", type=int, default=1,
                    help="run one GPU's share of a G-way split of the centres: the "
                         "first n/G rows of the same workload")
    ap.add_argument("--save-setup", default=None,
                    help="write the subsample and eigensystem to this .npz")
    ap.add_argument("--load-setup", default=None,
                    help="rebuild the context from a saved setup (ep_restore; no eigensolve)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--traffic-summary", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "BENCH_OUT"),
                    help="turn two rocprofv3 --pmc counter_collection.csv files (FETCH_SIZE, "
                         "WRITE_SIZE; runs with --calibrate-copy) into profiles/hbm_traffic.json "
                         "for the workload named in BENCH_OUT (the JSON line of the counted "
                         "run), and print a summary; no GPU needed")
    ap.add_argument("--study", choices=["batch", "convergence", "convergence-mnist", "kernels",
                                        "setup"], default=None,
                    help="run a study instead of the benchmark (JSON lines on stdout)")
    args = ap.parse_args()
    if args.traffic_summary:
        fcsv, wcsv, bout = args.traffic_summary
        with open(bout) as f:
            line = [x for x in f.read().splitlines() if x.startswith("{")][-1]
        rec = json.loads(line)
        workload = rec["config"]["workload"]
        kernel = rec["roofline"]["kernel"].split()[0]
        n_step = (rec["warmup"] + rec["steps"]) * rec["roofline"]["launches"] // rec["steps"]
        print(traffic_summary(fcsv, wcsv, workload, kernel, n_step,
                              "counters from rocprofv3 --pmc FETCH_SIZE / --pmc WRITE_SIZE runs of "
                              "bench.py --calibrate-copy (three 1 GiB device copies)"))
        return
    if args.study:
        fn = {"batch": study_batch, "convergence": study_convergence,
              "convergence-mnist": study_convergence, "kernels": study_kernels,
              "setup": study_setup}[args.study]
        for rec in fn(args):
            print(json.dumps(rec), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); "
              "the library has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_1806_06144_amd as ep

    cfg = synth.get_config(args.config)
    if args.s is not None:
        cfg = synth.get_config(args.config, s=args.s)
    if args.shard > 1:
        cfg = synth.get_config(args.config, n=cfg.n // args.shard, s=cfg.s)
    dev = torch.device("cuda:0")
    log(f"workload {cfg.name}: n={cfg.n} d={cfg.d} l={cfg.l} s={cfg.s} k={cfg.k}")
    t0 = time.perf_counter()
    X = synth.features(cfg, 0)
    labels = synth.class_labels(cfg, X, 0)
    r = synth.subsample_indices(cfg, 0)
    log(f"generated inputs in {time.perf_counter() - t0:.1f} s")
    Xd = torch.from_numpy(X).to(dev)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    if args.load_setup:
        sv = np.load(args.load_setup)
        ctx, info = ep.ep_restore(Xd, cfg.n, cfg.d, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s,
                                  cfg.k, sv["r"], sv["sigma"], sv["V"], stream=stream)
    else:
        ctx, info = ep.ep_setup(Xd, cfg.n, cfg.d, cfg.l, cfg.kernel, cfg.bandwidth, cfg.s,
                                cfg.k, sub_idx=r, stream=stream)
    if args.save_setup:
        sigma, _, V, r_used = ep.ep_get_preconditioner(ctx, info)
        np.savez(args.save_setup, r=r_used, sigma=sigma, V=V)
    ep.ep_set_contraction(ctx, args.contraction)
    m = int(cfg.m) if cfg.m else int(info.m)
    log(f"setup {info.setup_ms / 1e3:.1f} s: m*={info.m_star:.1f} m={m} beta={info.beta:.4f} "
        f"sigma_k+1={info.sigma_k1:.4f} eta={info.eta:.1f}")

    nb = args.warmup + args.steps
    # full batches of successive epochs (the short last batch of each is
    # timed on its own below)
    batches, epoch = [], 0
    while len(batches) < nb:
        batches += [b for b in synth.epoch_batches(cfg.n, m, epoch) if len(b) == m]
        epoch += 1
    batches = batches[:nb]
    t_dev = [torch.from_numpy(b).to(dev) for b in batches]
    y_dev = [torch.from_numpy(synth.one_hot(labels[b], cfg.l)).to(dev) for b in batches]

    for i in range(args.warmup):
        ep.ep_step(ctx, t_dev[i], m, y_dev[i])
    ep.ep_sync(ctx)
    ep.ep_timing_enable(ctx, True)
    # the library works on torch's current stream here, so events recorded
    # between its calls bracket each step on the GPU
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.warmup, nb):
        evs[i - args.warmup].record(stream)
        ep.ep_step(ctx, t_dev[i], m, y_dev[i])
    evs[-1].record(stream)
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    ep.ep_sync(ctx)
    tim = ep.ep_timing_read(ctx)
    ep.ep_timing_enable(ctx, False)
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]

    # the short last batch of an epoch (n mod m rows), for the epoch time
    last_ms = None
    m_last = cfg.n % m
    if m_last:
        tl = synth.epoch_batches(cfg.n, m, 0)[-1]
        tl_dev = torch.from_numpy(tl).to(dev)
        yl_dev = torch.from_numpy(synth.one_hot(labels[tl], cfg.l)).to(dev)
        ep.ep_step(ctx, tl_dev, m_last, yl_dev)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(3):
            ep.ep_step(ctx, tl_dev, m_last, yl_dev)
        ev1.record(stream)
        torch.cuda.synchronize()
        last_ms = ev0.elapsed_time(ev1) / 3

    # prediction (Section 2) of held-out rows with the trained alpha: the
    # same fused pass with m -> n_z, no diagonal rule
    n_z = 10000 if cfg.n > 100000 else 2000
    Z = torch.from_numpy(synth.heldout(cfg, 0, n_z=n_z)).to(dev)
    P = torch.empty((n_z, cfg.l), dtype=torch.float32, device=dev)
    ep.ep_predict(ctx, Z, n_z, P)
    ep.ep_sync(ctx)
    torch.cuda.synchronize()
    p0 = time.perf_counter()
    ep.ep_predict(ctx, Z, n_z, P)
    ep.ep_sync(ctx)
    p1 = time.perf_counter()
    predict = {"n_z": n_z, "ms": (p1 - p0) * 1e3,
               "tflops": 2.0 * n_z * cfg.n * (cfg.d + cfg.l) / (p1 - p0) / 1e12,
               "entries_per_s": n_z * cfg.n / (p1 - p0)}
    log(f"predict {n_z} rows: {predict['ms']:.1f} ms, {predict['tflops']:.1f} TFLOP/s")
    del Z, P

    # the blocked form on the same batches, for comparison (not the headline:
    # it writes the kernel block to memory)
    blocked_form = None
    if args.contraction != "blocked" and args.blocked_compare and cfg.d % 4 == 0:
        ep.ep_set_contraction(ctx, "blocked")
        ep.ep_step(ctx, t_dev[0], m, y_dev[0])
        ep.ep_sync(ctx)
        ep.ep_timing_enable(ctx, True)
        torch.cuda.synchronize()
        b0 = time.perf_counter()
        for i in range(args.warmup, nb):
            ep.ep_step(ctx, t_dev[i], m, y_dev[i])
        torch.cuda.synchronize()
        b1 = time.perf_counter()
        ep.ep_sync(ctx)
        tb = ep.ep_timing_read(ctx)
        ep.ep_timing_enable(ctx, False)
        ep.ep_set_contraction(ctx, args.contraction)
        if tb.kblock_launches > 0:
            kb_tf = 2.0 * m * cfg.n * cfg.d * args.steps / (tb.kblock_ms / 1e3) / 1e12
            blocked_form = {
                "ms_per_step": (b1 - b0) / args.steps * 1e3,
                "value": m * cfg.n / ((b1 - b0) / args.steps),
                "kblock_kernel_tflops": kb_tf,
                "kblock_kernel_frac": kb_tf / PEAK_FP32_MFMA_TFLOPS,
                "kblock_avg_launch_ms": tb.kblock_ms / tb.kblock_launches,
                "kblock_launches": int(tb.kblock_launches),
                "contraction_gemm_tflops":
                    2.0 * m * cfg.n * cfg.l * args.steps / (tb.gemm_ms / 1e3) / 1e12,
                "note": "kernel block written per centre chunk (<= 2 GiB) and contracted "
                        "by rocBLAS float32 GEMMs; same batches, timed after the headline",
            }
            log(f"blocked form: {blocked_form['ms_per_step']:.1f} ms/step, kblock_kernel "
                f"{kb_tf:.1f} TFLOP/s")

    sec_per_step = (t_end - t_start) / args.steps
    n, d, l, s, k = cfg.n, cfg.d, cfg.l, cfg.s, cfg.k
    entries = m * n
    kmv_flops = 2.0 * m * n * (d + l)
    kmv_avg_s = tim.kmv_ms / 1e3 / max(tim.kmv_launches, 1)
    pass_tflops = kmv_flops / kmv_avg_s / 1e12
    blocked = tim.kblock_launches > 0
    # steps 4-5: the fused form keeps the kernel values of the subsample
    # columns from step 2 and needs one s x m x l product; the blocked form
    # recomputes them in a subsample pass (distances and product)
    sub_flops = 2.0 * m * s * (d + l) if blocked else 2.0 * m * s * l
    step_flops = kmv_flops + sub_flops + 4.0 * s * k * l
    if blocked:
        # dominant kernel: the kernel block (distances -> kernel values);
        # its algorithmic work is 2 d flops per entry, over all chunks
        dom = "kblock_kernel"
        dom_label = "kblock_kernel (distance -> kernel block of a centre chunk, step 2, blocked form)"
        launches = int(tim.kblock_launches)
        dom_avg_s = tim.kblock_ms / 1e3 / launches
        dom_flops = 2.0 * m * n * d * args.steps / launches
        gemm_tflops = 2.0 * m * n * l * args.steps / (tim.gemm_ms / 1e3) / 1e12
    else:
        dom = "kmv_kernel"
        dom_label = "kmv_kernel (fused distance -> kernel -> contraction, step 2)"
        launches = int(tim.kmv_launches)
        dom_avg_s = kmv_avg_s
        dom_flops = kmv_flops
        gemm_tflops = None
    achieved = dom_flops / dom_avg_s / 1e12
    workload = f"{cfg.name}-shaped n={n} d={d} l={l} {cfg.kernel} bw={cfg.bandwidth:g} s={s} k={k} m={m}"
    if args.shard > 1:
        workload += f" (1/{args.shard} centre shard)"

    if args.calibrate_copy:
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log("calibration copy: 3 x 1 GiB device-to-device")

    probe_tf, probe_mhz = ep.ep_device_probe()
    log(f"device probe: fp32 MFMA {probe_tf:.1f} TFLOP/s sustained at {probe_mhz:.0f} MHz")

    cpu = None
    if not args.no_cpu_baseline:
        alpha = torch.empty((n, l), dtype=torch.float32, device=dev)
        ep.ep_get_alpha(ctx, alpha)
        ep.ep_sync(ctx)
        log("timing the oracle on bounded samples")
        cpu = cpu_baseline(X, alpha.cpu().numpy(), cfg, m)
    ep.ep_destroy(ctx)

    traffic, traffic_prov = measured_traffic(workload, dom)
    out = {
        "metric": "kernel entries/s (m*n per step)",
        "value": entries / sec_per_step,
        "unit": "entries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": sec_per_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": workload, "n": n, "d": d, "l": l, "s": s, "k": k, "m": m,
                   "kernel": cfg.kernel, "bandwidth": cfg.bandwidth},
        "contraction": "blocked" if blocked else "fused",
        "tflops_step2_pass": pass_tflops,
        "tflops_contraction_gemm": gemm_tflops,
        "tflops_whole_step": step_flops / sec_per_step / 1e12,
        "ms_per_step_median": float(np.median(step_ms)),
        # floor(n/m) full steps at the median time plus the short last batch
        "s_per_epoch": ((n // m) * float(np.median(step_ms)) + (last_ms or 0.0)) / 1e3,
        "last_batch": {"m": int(m_last), "ms": last_ms},
        "setup_s": info.setup_ms / 1e3,
        "roofline": {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_FP32_MFMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_MFMA_TFLOPS,
            "traffic": traffic,
            "traffic_source": traffic_prov,
            "kernel": dom_label,
            "avg_launch_ms": dom_avg_s * 1e3,
            "launches": launches,
            "flops_per_launch": dom_flops,
            "probe_mfma_f32_tflops": probe_tf,
            "probe_shader_clock_mhz": probe_mhz,
            "frac_of_probe": achieved / probe_tf if probe_tf > 0 else None,
        },
        "cpu_baseline": cpu,
        "predict": predict,
        "blocked_form": blocked_form,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

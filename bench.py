"""Throughput of the Shampoo hot path on one MI355X.

Workload (C2): 96 blocks, each with statistics L (1024 x 1024) built from 19
earlier gradients and a current gradient G (1024 x 4096) ~ N(0, 1/4096); a
step is one pass of the whole hot path over the 96 blocks:
    L += G G^T                       (grouped fp32-MFMA SYRK)
    Lr = (L + 1e-6 I)^(-1/4)         (96 roots in one grouped coupled-Newton call)
    P = Lr G                         (grouped fp32-MFMA GEMM; R side not tracked)
    D += G o G, graft, W -= eta P    (two HBM passes)
All inputs are resident in HBM before timing.  Before every step L is restored
to its pristine value L_19 (a device copy inside the timed region, reported
on its own), so every timed step roots the same matrices L_19 + G_20 G_20^T.
`value` is roots completed per second of whole-step time.  After the headline
step the default run also measures the other workloads at full size with a
few steps each (C1 latency, the four C3 root calls, the C4 step and root
refresh, the C5 grouped roots and step) and reports them under "workloads".
One JSON line is printed.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-extra]
       python bench.py --workload {c1,c3,c4,c5,c6} [...]   (one workload alone)
"""
import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "1024² fp32 inverse-4th-roots/sec + stats+precondition step ms; fp32 MFMA util %"
PEAK_F32_MFMA = 157.3   # TFLOP/s, MI355X dense fp32 matrix
PEAK_F64_MFMA = 78.6
PEAK_HBM = 8000.0       # GB/s


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def measured_traffic(name="newton_stage_kernel_c2_counters.txt"):
    """HBM bytes per launch of the Newton kernel from the committed rocprofv3
    counter summary, or None when the kernel sources changed since the
    counters were taken (the summary records a digest of the sources)."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    kv = dict(line.strip().split("=", 1) for line in open(path) if "=" in line and not line.startswith("#"))
    if kv.get("source_code_sha256") != source_code_digest():
        return None
    return float(kv["bytes_per_launch"])


def source_code_digest(src=None):
    """SHA-256 over the kernel sources with comments and white space removed,
    so that an edit of comments alone keeps the counter summary valid while
    any change of the code voids it."""
    import hashlib
    import re
    src = src or os.path.join(ROOT, "paper_2002_09018_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(src)):
        text = open(os.path.join(src, f), encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(f.encode() + b"\0" + " ".join(text.split()).encode())
    return h.hexdigest()


def newton_products(iters, p, power):
    """Symmetric products one matrix takes in a precision phase of `iters`
    iterations: 1 + floor(log2 p) + popcount(p) per iteration, less the
    first X product (X0 is a multiple of I).  The power-bound start adds M0^2
    and M0^4 and turns the first iteration's M-only products of its first
    stage (M1 M1, and M1 M for odd p) into an elementwise pass; at p = 4 the
    whole first M update is one product (M0^2 and M0^4 are known)."""
    per = 1 + (p.bit_length() - 1) + bin(p).count("1")
    stage0 = 2 if (p & 1 and p > 1) else 1
    if iters <= 0:
        return 2 if power else 0
    if power:
        first = 1 if p == 4 else per - 1 - stage0
        return 2 + first + per * (iters - 1)
    return per * iters - 1


def gen_block(i, n, k):
    from synth import configs as cfg
    L = cfg.wishart_bartlett(n, 19 * k, 1.0 / k, cfg.C2, i, 0).astype(np.float32)
    G = cfg.c2_grad(i, n, k, 20)
    D = cfg.c2_adagrad_state(i, n, k, 19)
    W = cfg.c2_weight(i, n, k)
    return L, G, D, W


def cpu_baseline(sample, n, k, p, eps, eta0, budget_s=12.0):
    """The oracle's step (fp64 stats, eigh root, precondition, graft) timed on
    host cores over a bounded sample of the blocks."""
    import oracle.shampoo_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([t.get("num_threads", 1) for t in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count()
    done, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        L, G, D, W = sample[done % len(sample)]
        Ln, _ = O.stats_update(L, None, G)
        Lr, st, _ = O.inv_root(Ln, p, eps)
        P = O.precondition(G, Lr, None)
        O.graft_update(W, D, G, P, eta0)
        done += 1
    dt = time.perf_counter() - t0
    import scipy
    cpu = "unknown"
    try:
        cpu = next(l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name"))
    except Exception:
        pass
    out = dict(value=done / dt, unit="roots/s", cores=int(cores), kind="oracle", cpu_model=cpu,
               numpy=np.__version__, scipy=scipy.__version__,
               sample=f"{done} block-steps cycling over {len(sample)} of the 96 blocks, full fp64 step "
                      f"per block (stats L+GG^T, eigh root, Lr G, graft), {dt:.1f} s")
    # The paper's CPU root service: Algorithm 1 transcribed in fp64 (two
    # roots), and the eigh root on one thread (per-root latency).
    t1 = time.perf_counter()
    its, its4 = [], []
    for L, G, D, W in sample[:2]:
        Ln, _ = O.stats_update(L, None, G)
        its.append(O.coupled_newton(Ln, p, eps=eps, tol=1e-6)["iters"])
    out["newton_transcript_s_per_root"] = (time.perf_counter() - t1) / 2
    out["newton_transcript_iters"] = its          # Algorithm 1 as printed (Frobenius start)
    for L, G, D, W in sample[:2]:
        Ln, _ = O.stats_update(L, None, G)
        its4.append(O.coupled_newton(Ln, p, eps=eps, tol=1e-6, scaling="power4")["iters"])
    out["newton_transcript_iters_power4"] = its4  # the start the GPU uses
    try:
        from threadpoolctl import threadpool_limits
        L, G, D, W = sample[0]
        Ln, _ = O.stats_update(L, None, G)
        with threadpool_limits(limits=1):
            t1 = time.perf_counter()
            O.inv_root(Ln, p, eps)
            out["eigh_root_s_1thread"] = time.perf_counter() - t1
    except Exception as e:  # threadpoolctl missing: no 1-thread figure
        log(f"no 1-thread figure: {e}")
    return out


def warm_measure(torch, B, h, As, X0s, prm, ws, ref=None, sample=4):
    """Warm-started roots (coupled-Newton appendix, warm start) of As from
    X0s: one untimed call (code-object loading), then a timed one with
    kernel timing.  Full products counted as 2 n^3 each: at p = 4 the start
    takes 3 (X0^2, X0^4, X0^4 A_d) and each warm iteration 6 (4 of the
    iteration, 2 of the commutator monitor).  ref: cold roots of the same
    As; the relative Frobenius distance of the warm result from them is
    reported on a sample of matrices."""
    dev = As[0].device
    n_all = len(As)
    info = torch.zeros(8 * n_all, dtype=torch.int32, device=dev)
    wout = torch.zeros(2 * n_all, dtype=torch.int32, device=dev)
    Xw = [x.clone() for x in X0s]
    B.shampoo_inv_root_warm_batched(h, As, Xw, prm, ws, info, wout)
    torch.cuda.synchronize()
    for x, x0 in zip(Xw, X0s):
        x.copy_(x0)
    B.shampoo_timing_enable(h, True)
    for c in range(len(B.KCLASS_NAMES)):
        B.shampoo_timing_read(h, c)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    B.shampoo_inv_root_warm_batched(h, As, Xw, prm, ws, info, wout)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3
    B.shampoo_timing_enable(h, False)
    times = {B.KCLASS_NAMES[c]: B.shampoo_timing_read(h, c) for c in range(len(B.KCLASS_NAMES))}
    w = wout.cpu().numpy().reshape(-1, 2)
    p = prm.p
    prologue = (p.bit_length() - 1) + bin(p).count("1")
    per_iter = (p.bit_length() - 1) + bin(p).count("1") + 1 + 2
    flops = sum(2.0 * a.shape[0] ** 3 * (prologue + per_iter * int(k)) for a, k in zip(As, w[:, 1]))
    wms = times["newton_warm"][0]
    out = {"roots": n_all, "ms": ms, "roots_per_s": n_all / ms * 1e3,
           "kept": int((w[:, 0] == 1).sum()), "given_up": int((w[:, 0] == 2).sum()),
           "warm_iters_mean": float(w[:, 1].mean()),
           "full_products_ms": wms, "full_products_tflops": flops / (wms * 1e-3) / 1e12 if wms else None,
           "phases_ms": {c: v[0] for c, v in times.items() if v[1]}}
    if ref is not None:
        idx = np.linspace(0, n_all - 1, min(sample, n_all)).astype(int)
        errs = [float(torch.linalg.norm(Xw[i].double() - ref[i].double()) / torch.linalg.norm(ref[i].double()))
                for i in idx]
        out["rel_dist_from_cold_root_max"] = max(errs)
        out["rel_dist_sample"] = [int(i) for i in idx]
    return out


def time_steps(torch, B, h, step, K, kernel_timing=True):
    """Times K steps (per-launch HIP events when kernel_timing): elapsed
    seconds and {kernel class: (ms, launches)}."""
    B.shampoo_timing_enable(h, kernel_timing)
    for c in range(len(B.KCLASS_NAMES)):
        B.shampoo_timing_read(h, c)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    B.shampoo_timing_enable(h, False)
    return elapsed, {B.KCLASS_NAMES[c]: B.shampoo_timing_read(h, c) for c in range(len(B.KCLASS_NAMES))}


def step_report(K, el_f, t_f, el_s, t_s, flops_stats, flops_prec, bytes_graft, bytes_pass2):
    """Per-kernel rates from the run with separate preconditioning and graft
    calls (their classes hold exactly those kernels); the whole-step time and
    phases of the fused run beside it."""
    return {
        "phases_ms_per_step": {c: v[0] / K for c, v in t_f.items()},
        "kernels": {"stats_tflops": flops_stats / (t_s["stats"][0] * 1e-3) / 1e12,
                    "precond_tflops": flops_prec / (t_s["precond"][0] * 1e-3) / 1e12,
                    "graft_gbs": bytes_graft / (t_s["graft"][0] * 1e-3) / 1e9,
                    "fused_graft_pass2_gbs": bytes_pass2 / (t_f["graft"][0] * 1e-3) / 1e9 if t_f["graft"][0] else None},
        "split_calls_phases_ms_per_step": {c: v[0] / K for c, v in t_s.items()},
    }


def run_c4(args, torch, B):
    """C4: 24 BERT-Large-shaped layers, 288 blocks of 1024 x 1024 (strided
    views of the Q, K, V, O, FFN-in and FFN-out tensors); a step is the
    two-sided statistics, preconditioning and graft over all blocks.  The
    root refresh (every 100 steps in the workload) is timed separately."""
    from synth import configs as cfg
    dev = torch.device("cuda:0")
    d, nl = 1024, cfg.C4_LAYERS
    shapes = dict(cfg.c4_layer_tensors())
    names = [nm for nm, _ in cfg.c4_layer_tensors()]
    log("generating C4 tensors")
    Wt, Dt, Pt, Gt = {}, {}, {}, {}
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 4)) as ex:
        keys = [(l, t) for l in range(nl) for t in range(len(names))]
        grads = list(ex.map(lambda lt: cfg.c4_grad(lt[0], lt[1], 1, shapes[names[lt[1]]]), keys))
    for (l, t), g in zip(keys, grads):
        sh = shapes[names[t]]
        Gt[l, t] = torch.from_numpy(g).to(dev)
        Wt[l, t] = (0.02 * torch.randn(sh, device=dev, generator=torch.Generator(device=dev).manual_seed(l * 8 + t)))
        Dt[l, t] = torch.zeros(sh, device=dev)
        Pt[l, t] = torch.zeros(sh, device=dev)
    blocks, Ls, Rs, Lrs, Rrs = [], [], [], [], []
    for l in range(nl):
        for (t, r0, c0, rr, cc) in cfg.c4_blocks(d):
            sl = (slice(r0, r0 + rr), slice(c0, c0 + cc))
            L = torch.zeros(rr, rr, device=dev)
            R = torch.zeros(cc, cc, device=dev)
            Lr = torch.zeros(rr, rr, device=dev)
            Rr = torch.zeros(cc, cc, device=dev)
            Ls.append(L); Rs.append(R); Lrs.append(Lr); Rrs.append(Rr)
            blocks.append(B.Block(G=Gt[l, t][sl], W=Wt[l, t][sl], D=Dt[l, t][sl], P=Pt[l, t][sl],
                                  L=L, R=R, Lr=Lr, Rr=Rr))
    nb = len(blocks)
    h = B.shampoo_create(0)
    # root refresh at step 100 of the workload: statistics of 100 gradients
    # N(0, 1e-3) of a 1024 x 1024 block are Wishart(1024, 102400 dof)
    for b in range(nb):
        Ls[b].copy_(cfg.wishart_bartlett_device(d, 100 * d, 1e-3, torch, dev, cfg.C4, 7, b, 0))
        Rs[b].copy_(cfg.wishart_bartlett_device(d, 100 * d, 1e-3, torch, dev, cfg.C4, 7, b, 1))
    prm = B.shampoo_root_params_default(p=4, eps=1e-6)
    As, Xs = Ls + Rs, Lrs + Rrs
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([d] * len(As), prm.precision), dtype=torch.uint8,
                     device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    # one untimed call first (code-object loading, table allocation); the
    # statistics are only read, so the timed call repeats the same work
    B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
    torch.cuda.synchronize()
    root_ms = (time.perf_counter() - t0) * 1e3
    iters = [i["iters"] for i in B.decode_root_info(info)]
    # the same call once more with per-launch events: the Newton products' own time
    _, rtimes = time_steps(torch, B, h, lambda: B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info), 1)
    root_newton_ms = rtimes["newton_f32"][0]
    log(f"root refresh: {len(As)} roots in {root_ms:.1f} ms (Newton products {root_newton_ms:.1f} ms)")
    # the next refresh (step 200) warm-started from these roots: 100 more
    # gradients add an independent Wishart(1024, 102400 dof) draw
    warm = None
    if not args.no_warm:
        As2 = [a + cfg.wishart_bartlett_device(d, 100 * d, 1e-3, torch, dev, cfg.C4, 8, b % nb, b // nb)
               for b, a in enumerate(As)]
        X2 = [torch.zeros(d, d, device=dev) for _ in As]
        B.shampoo_inv_root_batched(h, As2, X2, prm, ws, info)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        B.shampoo_inv_root_batched(h, As2, X2, prm, ws, info)
        torch.cuda.synchronize()
        cold2_ms = (time.perf_counter() - t0) * 1e3
        warm = warm_measure(torch, B, h, As2, Xs, prm, ws, ref=X2)
        warm["cold_ms_same_matrices"] = cold2_ms
        log(f"warm refresh: {warm['ms']:.1f} ms (cold {cold2_ms:.1f} ms), kept {warm['kept']}")
        del As2, X2

    pblocks = B.PackedBlocks(h, blocks)   # checked and packed once for the repeated calls

    def step_fused():
        B.shampoo_update_stats(h, pblocks)
        B.shampoo_precondition_graft(h, pblocks, 6e-3)

    def step_split():
        B.shampoo_update_stats(h, pblocks)
        B.shampoo_precondition(h, pblocks)
        B.shampoo_graft(h, pblocks, 6e-3)

    main_step = step_split if args.split_graft else step_fused
    for _ in range(args.warmup):
        main_step()
    torch.cuda.synchronize()
    K = args.steps
    elapsed, times = time_steps(torch, B, h, main_step, K)
    el_s, t_s = time_steps(torch, B, h, step_split, K)
    B.shampoo_destroy(h)
    flops_stats = K * nb * 2 * d * d * (d + 1)
    flops_prec = K * nb * 4 * d ** 3
    bytes_graft = K * nb * d * d * 28
    roof_ms = (flops_stats / PEAK_F32_MFMA + flops_prec / PEAK_F32_MFMA) / 1e9 / K + bytes_graft / PEAK_HBM / 1e6 / K
    ms_step = elapsed * 1e3 / K
    prods = sum(newton_products(i, 4, True) for i in iters)
    out = {
        "metric": "C4 stats+precondition+graft step ms (288 blocks of 1024^2, two-sided)",
        "value": ms_step, "unit": "ms/step", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": ms_step, "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "C4: 24 layers x 12 blocks of 1024x1024 (BERT-Large shapes), G ~ N(0,1e-3) fp32, "
                               "stats L,R + L^-1/4 G R^-1/4 + AdaGrad graft per step",
                   "blocks": nb, "graft": "separate calls" if args.split_graft else "fused into preconditioning"},
        "phase_roofline_ms": roof_ms, "frac_of_phase_roofline": roof_ms / ms_step,
        **step_report(K, elapsed, times, el_s, t_s, flops_stats, flops_prec, bytes_graft, K * nb * d * d * 12),
        "root_refresh": {"roots": len(As), "ms": root_ms, "roots_per_s": len(As) / root_ms * 1e3,
                         "iters_mean": float(np.mean(iters)),
                         "newton_ms": root_newton_ms,
                         "newton_tflops": prods * d * d * (d + 1) / (root_newton_ms * 1e-3) / 1e12,
                         "call_tflops": prods * d * d * (d + 1) / (root_ms * 1e-3) / 1e12},
        "root_refresh_warm_step200": warm,
    }
    kr = out["kernels"]
    out["roofline"] = {"kernel": "gemm_grouped_kernel (preconditioning, the step's largest phase)", "bound": "mfma",
                       "achieved": kr["precond_tflops"], "peak": PEAK_F32_MFMA, "unit": "TFLOP/s",
                       "frac": kr["precond_tflops"] / PEAK_F32_MFMA,
                       "step_frac_of_phase_roofline": roof_ms / ms_step}
    rr = out["root_refresh"]
    rr["newton_frac"] = rr["newton_tflops"] / PEAK_F32_MFMA
    return out


def run_c6(args, torch, B):
    """C6: an embedding table (vocab x 1024, default 32768 rows: the C5
    embedding) read by 65536 one-hot Zipf lookups per step.  A step is the
    compaction of the lookup gradient, the 1024 x 1024 statistic U^T U over
    the active rows, the one-sided preconditioned rows U R^(-1/2) and the
    grafted update of the active rows.  The root refresh (p = 2) is timed
    separately.  Each step has its own lookups; all are resident in HBM."""
    from synth import configs as cfg
    dev = torch.device("cuda:0")
    vocab, nnz, dim, eta0 = args.vocab, args.lookups, 1024, 1e-2
    nsteps = args.warmup + args.steps
    log(f"generating C6 lookups: {nsteps} steps of {nnz} over {vocab} rows")
    idx_d, dy_d = [], []
    for t in range(nsteps):
        idx, _, _, m = cfg.c6_lookup(t + 1, nnz, vocab)
        idx_d.append(torch.from_numpy(idx).to(dev))
        dy_d.append(torch.from_numpy(cfg.c6_dy(t + 1, m, dim)).to(dev))
    W = 0.02 * torch.randn(vocab, dim, device=dev, generator=torch.Generator(device=dev).manual_seed(6))
    D = torch.zeros(vocab, dim, device=dev)
    R = cfg.wishart_bartlett_device(dim, 100 * nnz, 1e-3, torch, dev, cfg.C6, 8, 0)
    Rr = torch.zeros(dim, dim, device=dev)
    rows = torch.zeros(nnz, dtype=torch.int32, device=dev)
    U = torch.zeros(nnz, dim, device=dev)
    P = torch.zeros(nnz, dim, device=dev)
    counts = torch.zeros(nsteps, 2, dtype=torch.int32, device=dev)
    ws = torch.empty(B.shampoo_embedding_workspace_bytes(nnz, dim), dtype=torch.uint8, device=dev)
    h = B.shampoo_create(0)
    prm = B.shampoo_root_params_default(p=2, eps=1e-6)
    rws = torch.empty(B.shampoo_inv_root_workspace_bytes([dim], prm.precision), dtype=torch.uint8, device=dev)
    info = torch.zeros(8, dtype=torch.int32, device=dev)
    # one untimed call first (code-object loading, table allocation); R is
    # only read, so the timed call repeats the same work
    B.shampoo_inv_root_batched(h, [R], [Rr], prm, rws, info)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    B.shampoo_inv_root_batched(h, [R], [Rr], prm, rws, info)
    torch.cuda.synchronize()
    root_ms = (time.perf_counter() - t0) * 1e3

    def step(t):
        c = counts[t]
        B.shampoo_embedding_rows(h, idx_d[t], None, None, vocab, dy_d[t], rows, U, c, ws)
        B.shampoo_embedding_stats(h, U, c, R, 1.0, ws)
        B.shampoo_embedding_precondition(h, U, c, Rr, P)
        B.shampoo_embedding_graft(h, rows, c, U, P, W, D, eta0)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()
    B.shampoo_timing_enable(h, True)
    for c in range(len(B.KCLASS_NAMES)):
        B.shampoo_timing_read(h, c)
    t0 = time.perf_counter()
    for t in range(args.warmup, nsteps):
        step(t)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    B.shampoo_timing_enable(h, False)
    times = {B.KCLASS_NAMES[c]: B.shampoo_timing_read(h, c) for c in range(len(B.KCLASS_NAMES))}
    B.shampoo_destroy(h)
    K = args.steps
    u = counts[args.warmup:, 0].cpu().numpy().astype(np.float64)
    flops_stats = float(np.sum(u)) * dim * (dim + 1)          # upper triangle of U^T U
    flops_prec = float(np.sum(u)) * 2 * dim * dim
    bytes_graft = float(np.sum(u)) * dim * 28
    bytes_emb = K * nnz * dim * 8.0                          # dy read + U written
    ms_step = elapsed * 1e3 / K
    st_ms, pr_ms = times["stats"][0], times["precond"][0]
    out = {
        "metric": f"C6 embedding step: lookups/s ({vocab} x {dim} table, {nnz} one-hot Zipf lookups per step)",
        "value": K * nnz / elapsed, "unit": "lookups/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"C6: embedding {vocab}x{dim}, {nnz} Zipf(1.07) one-hot lookups/step; compact "
                               "rows + R += U^T U + U R^-1/2 + row-indexed AdaGrad graft",
                   "vocab": vocab, "dim": dim, "lookups": nnz},
        "active_rows_mean": float(np.mean(u)),
        "phases_ms_per_step": {c: v[0] / K for c, v in times.items()},
        "kernels": {"stats_tflops": flops_stats / (st_ms * 1e-3) / 1e12,
                    "precond_tflops": flops_prec / (pr_ms * 1e-3) / 1e12,
                    "graft_gbs": bytes_graft / (times["graft"][0] * 1e-3) / 1e9,
                    "emb_compaction_gbs": bytes_emb / (times["emb"][0] * 1e-3) / 1e9},
        "root_refresh": {"roots": 1, "p": 2, "ms": root_ms, "iters": B.decode_root_info(info)[0]["iters"]},
    }
    return out


def run_c3(args, torch, B):
    """C3: 32 ill-conditioned 2048 x 2048 matrices (log-uniform spectrum in
    [1e-6, 1e2]), scaled damping eps_d * lambda_max with eps_d = 1e-6 (damped
    condition ~1e6, the 1e-3 band) and 1e-8 (~5e7, the 5e-3 band), one grouped
    call per (p, eps_d), p in {2, 4}; AUTO precision (fp32 attempt, fp64
    tail).  Each call is timed on its second run (the first loads code
    objects and sizes the tables)."""
    from synth import configs as cfg
    dev = torch.device("cuda:0")
    n, nm = 2048, 32
    log("generating C3 matrices on the device")
    gen = [cfg.c3_matrix_device(i, torch, dev, n) for i in range(nm)]
    As = [a for a, _ in gen]
    lams = [lam for _, lam in gen]
    Xs = [torch.zeros_like(a) for a in As]
    h = B.shampoo_create(0)
    res = {}
    sym = n * n * (n + 1)
    ws = None
    for p in (2, 4):
        for epsd in (1e-6, 1e-8):
            prm = B.shampoo_root_params_default(p=p, eps=epsd, eps_relative=1)
            if ws is None:
                ws = torch.empty(B.shampoo_inv_root_workspace_bytes([n] * nm, prm.precision), dtype=torch.uint8,
                                 device=dev)
            info = torch.zeros(8 * nm, dtype=torch.int32, device=dev)
            B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
            torch.cuda.synchronize()
            B.shampoo_timing_enable(h, True)
            for c in range(len(B.KCLASS_NAMES)):
                B.shampoo_timing_read(h, c)
            t0 = time.perf_counter()
            B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3
            B.shampoo_timing_enable(h, False)
            times = {B.KCLASS_NAMES[c]: B.shampoo_timing_read(h, c) for c in range(len(B.KCLASS_NAMES))}
            inf = B.decode_root_info(info)
            pr64 = sum(newton_products(i["iters"], p, True) for i in inf if i["precision"] == 64)
            pr32 = sum(newton_products(i["iters_fp32"], p, True) for i in inf)
            t64, t32 = times["newton_f64"][0], times["newton_f32"][0]
            kappa = [float((lam.max() + i["eps_eff"]) / (lam.min() + i["eps_eff"])) for lam, i in zip(lams, inf)]
            r = {
                "p": p, "eps_d": epsd, "ms": ms, "roots_per_s": nm / ms * 1e3,
                "kappa_damped_range": [min(kappa), max(kappa)],
                "iters_fp64_mean": float(np.mean([i["iters"] for i in inf if i["precision"] == 64] or [0])),
                "iters_fp64_max": max([i["iters"] for i in inf if i["precision"] == 64] or [0]),
                "iters_fp32_attempt_mean": float(np.mean([i["iters_fp32"] for i in inf])),
                "n_fp64": sum(1 for i in inf if i["precision"] == 64),
                "status": sorted(set(i["status"] for i in inf)),
                "newton_f64_ms": t64, "newton_f32_ms": t32, "root_aux_ms": times["root_aux"][0],
                "newton_f64_tflops": pr64 * sym / (t64 * 1e-3) / 1e12 if t64 else None,
                "newton_f32_tflops": pr32 * sym / (t32 * 1e-3) / 1e12 if t32 else None,
            }
            r["roofline"] = {"kernel": "newton_stage_kernel<double>", "bound": "mfma", "unit": "TFLOP/s",
                             "achieved": r["newton_f64_tflops"], "peak": PEAK_F64_MFMA,
                             "frac": r["newton_f64_tflops"] / PEAK_F64_MFMA if t64 else None}
            if not args.no_cpu_baseline and args.workload == "c3":
                # accuracy on one matrix: relative error against the oracle
                # (eigh, fed the GPU's lambda_max) and the true residual
                import oracle.shampoo_oracle as O
                q = 0
                Ad = As[q].double() + inf[q]["eps_eff"] * torch.eye(n, device=dev, dtype=torch.float64)
                Rm = torch.linalg.matrix_power(Xs[q].double(), p) @ Ad - torch.eye(n, device=dev,
                                                                                  dtype=torch.float64)
                Xo, _, _ = O.inv_root(As[q].cpu().numpy(), p, epsd, eps_relative=True,
                                      lam_max=inf[q]["lambda_max"])
                Xh = Xs[q].cpu().numpy().astype(np.float64)
                r["accuracy_matrix0"] = {"true_resid_fro": float(torch.linalg.norm(Rm)),
                                         "rel_err_vs_eigh": float(np.linalg.norm(Xh - Xo) / np.linalg.norm(Xo))}
            res[f"p{p}_eps{epsd:g}"] = r
            log(f"C3 p={p} eps_d={epsd:g}: {ms:.1f} ms, fp64 {r['newton_f64_tflops'] or 0:.1f} TFLOP/s")
    warm = c3_warm(torch, B, h, As, ws)
    B.shampoo_destroy(h)
    main = res["p4_eps1e-06"]
    out = {"metric": "C3 ill-conditioned 2048^2 inverse roots (AUTO precision, fp64 tail)", "value": main["ms"],
           "unit": "ms per 32 roots (p=4, eps_d 1e-6)", "n_gpus": 1, "higher_is_better": False,
           "dtype": "f32/f64", "data": "synthetic",
           "config": {"workload": "C3: 32 x 2048^2, lambda log-uniform [1e-6,1e2], eps_d * lambda_max with "
                                  "eps_d in {1e-6, 1e-8}, p in {2,4}"},
           "roofline": main["roofline"], "results": res, "warm_start_drift": warm}
    return out


def c3_warm(torch, B, h, As, ws, drifts=(1e-8, 1e-6, 1e-4)):
    """Warm start (coupled-Newton appendix) where it pays: the ill-conditioned
    C3 matrices, whose cold roots take about 19 fp64 iterations.  Their
    p = 4, eps_d = 1e-6 roots X0 seed the roots of the drifted statistics
    A + s lambda_max u u^T (u a seeded unit vector per matrix, one drift size
    s per case), rooted warm in fp64 and cold (AUTO, the C3 default, and
    fp64) on the same matrices; the warm results are compared with the cold
    fp64 roots (the same policy, so the same MaxSV and damping)."""
    dev = As[0].device
    nm, n = len(As), As[0].shape[0]
    prm_auto = B.shampoo_root_params_default(p=4, eps=1e-6, eps_relative=1)
    prm64 = B.shampoo_root_params_default(p=4, eps=1e-6, eps_relative=1, precision=B.PRECISION_FP64)
    info = torch.zeros(8 * nm, dtype=torch.int32, device=dev)
    X0 = [torch.zeros_like(a) for a in As]
    B.shampoo_inv_root_batched(h, As, X0, prm_auto, ws, info)
    torch.cuda.synchronize()
    lam = [i["lambda_max"] for i in B.decode_root_info(info)]
    g = torch.Generator(device=dev).manual_seed(33)
    us = [torch.randn(n, device=dev, generator=g, dtype=torch.float64) for _ in range(nm)]
    us = [u / torch.linalg.norm(u) for u in us]
    out = {}

    def cold(prm, A2):
        X = [torch.zeros_like(a) for a in A2]
        B.shampoo_inv_root_batched(h, A2, X, prm, ws, info)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        B.shampoo_inv_root_batched(h, A2, X, prm, ws, info)
        torch.cuda.synchronize()
        inf = B.decode_root_info(info)
        return X, (time.perf_counter() - t0) * 1e3, float(np.mean([i["iters"] + i["iters_fp32"] * (
            i["precision"] == 64) for i in inf]))

    for sd in drifts:
        A2 = [(a.double() + (sd * lm) * torch.outer(u, u)).float() for a, lm, u in zip(As, lam, us)]
        Xa, cold_auto_ms, cold_auto_iters = cold(prm_auto, A2)
        del Xa
        Xc, cold64_ms, cold64_iters = cold(prm64, A2)
        w = warm_measure(torch, B, h, A2, X0, prm64, ws, ref=Xc)
        w.update({"cold_auto_ms": cold_auto_ms, "cold_auto_iters_mean": cold_auto_iters,
                  "cold_fp64_ms": cold64_ms, "cold_fp64_iters_mean": cold64_iters})
        out[f"drift{sd:g}"] = w
        log(f"C3 warm, drift {sd:g}: {w['ms']:.1f} ms ({w['warm_iters_mean']:.1f} it, kept {w['kept']}) against "
            f"cold {cold_auto_ms:.1f} ms AUTO / {cold64_ms:.1f} ms fp64")
        del A2, Xc
    return out


def run_c5(args, torch, B):
    """C5: a 32768 x 1024 embedding (32 row blocks of 1024 x 1024) and 200
    square blocks with sides drawn from {128, ..., 2048}, bf16-stored
    gradients N(0, 1e-3) and fp32 statistics L and R for every block.  Ten
    statistics steps build the factors; one grouped call then roots all 464
    factors (p = 4, per-matrix early exit); the call is timed, and each size
    class is also rooted alone.  A step is the statistics, the two-sided
    preconditioning and the graft over the 232 blocks.

    --emb-lookups N > 0: the embedding's gradient is row-sparse instead of
    dense, the rows read by N lookups per step from a Zipf(1.1) token stream
    (embedding appendix: only the looked-up rows carry gradient), so its 64
    factors are rank-deficient and damping-dominated (condition ~1e9) and
    take the fp64 tail while the 400 others stop after a few fp32
    iterations: the case per-matrix early exit is for."""
    from synth import configs as cfg
    dev = torch.device("cuda:0")
    nemb = cfg.C5_EMB_ROWS // cfg.C5_D
    shp = [(cfg.C5_D, cfg.C5_D)] * nemb + [(k, k) for k in cfg.c5_mixed_sizes()]
    nb = len(shp)
    gen = torch.Generator(device=dev).manual_seed(5)
    emb = torch.empty(cfg.C5_EMB_ROWS, cfg.C5_D, dtype=torch.bfloat16, device=dev)
    mixed = [torch.empty(s, dtype=torch.bfloat16, device=dev) for s in shp[nemb:]]
    tensors = [emb] + mixed
    Gv = [emb[i * cfg.C5_D:(i + 1) * cfg.C5_D] for i in range(nemb)] + mixed
    Wt = [0.02 * torch.randn(t.shape, device=dev, generator=gen) for t in tensors]
    Dt = [torch.zeros(t.shape, device=dev) for t in tensors]
    Pt = [torch.zeros(t.shape, device=dev) for t in tensors]

    def view(ts, b):
        return ts[0][b * cfg.C5_D:(b + 1) * cfg.C5_D] if b < nemb else ts[1 + b - nemb]

    Ls = [torch.zeros(m, m, device=dev) for m, _ in shp]
    Rs = [torch.zeros(n, n, device=dev) for _, n in shp]
    Lrs = [torch.zeros_like(a) for a in Ls]
    Rrs = [torch.zeros_like(a) for a in Rs]
    blocks = [B.Block(G=Gv[b], W=view(Wt, b), D=view(Dt, b), P=view(Pt, b), L=Ls[b], R=Rs[b], Lr=Lrs[b],
                      Rr=Rrs[b]) for b in range(nb)]
    h = B.shampoo_create(0)

    sparse = args.emb_lookups > 0
    emb32 = torch.zeros(emb.shape, device=dev) if sparse else None

    def fill_grads(step):
        for t in tensors[1:] if sparse else tensors:
            t.copy_((torch.randn(t.shape, device=dev, generator=gen) * 1e-3 ** 0.5).to(torch.bfloat16))
        if sparse:
            idx = torch.from_numpy(cfg.zipf_rows(args.emb_lookups, emb.shape[0], 1.1, cfg.C5, 3, step)).to(dev)
            dy = torch.randn(args.emb_lookups, emb.shape[1], device=dev, generator=gen) * 1e-3 ** 0.5
            emb32.zero_()
            emb32.index_add_(0, idx.long(), dy)
            emb.copy_(emb32.to(torch.bfloat16))

    log(f"C5: {nb} blocks, 10 statistics steps" + (f", embedding row-sparse ({args.emb_lookups} Zipf lookups/step)"
                                                    if sparse else ""))
    for t in range(10):
        fill_grads(t)
        B.shampoo_update_stats(h, blocks)
    torch.cuda.synchronize()
    As, Xs = Ls + Rs, Lrs + Rrs
    ns = [a.shape[0] for a in As]
    # the row-sparse variant's factors have many zero eigenvalues, and fp32
    # rounding of the statistics leaves them near +-1e-7 lambda_max, far
    # above an absolute 1e-6 ridge: they take the scaled damping
    # eps * lambda_max of Algorithm 1 (MaxSV) instead
    prm = B.shampoo_root_params_default(p=4, eps=1e-6, eps_relative=1 if sparse else 0)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes(ns, prm.precision), dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * len(As), dtype=torch.int32, device=dev)
    B.shampoo_inv_root_batched(h, As[:2], Xs[:2], prm, ws, info)     # warm-up
    torch.cuda.synchronize()
    B.shampoo_timing_enable(h, True)
    for c in range(len(B.KCLASS_NAMES)):
        B.shampoo_timing_read(h, c)
    t0 = time.perf_counter()
    B.shampoo_inv_root_batched(h, As, Xs, prm, ws, info)
    torch.cuda.synchronize()
    root_ms = (time.perf_counter() - t0) * 1e3
    B.shampoo_timing_enable(h, False)
    rt = {B.KCLASS_NAMES[c]: B.shampoo_timing_read(h, c) for c in range(len(B.KCLASS_NAMES))}
    inf = B.decode_root_info(info)
    log(f"grouped roots: {len(As)} in {root_ms:.1f} ms")
    sym = [n * n * (n + 1) for n in ns]
    # executed products: every matrix's fp32 iterations, plus the fp64 tail of
    # the escalated ones; without early exit every matrix of a phase would run
    # that phase's largest iteration count
    prods = [newton_products(i["iters_fp32"], 4, True) for i in inf]
    prods64 = [newton_products(i["iters"], 4, True) if i["precision"] == 64 else 0 for i in inf]
    executed = sum((pq + pq64) * s for pq, pq64, s in zip(prods, prods64, sym))
    esc = [j for j, i in enumerate(inf) if i["precision"] == 64]
    no_exit = newton_products(max(i["iters_fp32"] for i in inf), 4, True) * sum(sym)
    if esc:
        no_exit += newton_products(max(inf[j]["iters"] for j in esc), 4, True) * sum(sym[j] for j in esc)
    classes = {}
    for k in sorted(set(ns)):
        sel = [j for j, n in enumerate(ns) if n == k]
        a_k, x_k = [As[j] for j in sel], [Xs[j] for j in sel]
        info_k = torch.zeros(8 * len(sel), dtype=torch.int32, device=dev)
        B.shampoo_inv_root_batched(h, a_k, x_k, prm, ws, info_k)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        B.shampoo_inv_root_batched(h, a_k, x_k, prm, ws, info_k)
        torch.cuda.synchronize()
        ms_k = (time.perf_counter() - t1) * 1e3
        it_k = [inf[j]["iters"] + (inf[j]["iters_fp32"] if inf[j]["precision"] == 64 else 0) for j in sel]
        classes[str(k)] = {"roots": len(sel), "iters_min": min(it_k), "iters_max": max(it_k),
                           "iters_mean": float(np.mean(it_k)), "alone_ms": ms_k,
                           "alone_roots_per_s": len(sel) / ms_k * 1e3,
                           "alone_newton_tflops": sum((prods[j] + prods64[j]) * sym[j] for j in sel) / (ms_k * 1e-3) / 1e12}
        log(f"  class {k}: {len(sel)} roots alone in {ms_k:.2f} ms")

    pblocks = B.PackedBlocks(h, blocks)   # checked and packed once for the repeated calls

    def step_fused():
        B.shampoo_update_stats(h, pblocks)
        B.shampoo_precondition_graft(h, pblocks, 1e-2)

    def step_split():
        B.shampoo_update_stats(h, pblocks)
        B.shampoo_precondition(h, pblocks)
        B.shampoo_graft(h, pblocks, 1e-2)

    main_step = step_split if args.split_graft else step_fused
    for _ in range(args.warmup):
        main_step()
    torch.cuda.synchronize()
    K = args.steps
    elapsed, times = time_steps(torch, B, h, main_step, K)
    el_s, t_s = time_steps(torch, B, h, step_split, K)
    B.shampoo_destroy(h)
    flops_stats = K * sum(m * (m + 1) * n + n * (n + 1) * m for m, n in shp)
    flops_prec = K * sum(2 * m * m * n + 2 * m * n * n for m, n in shp)
    bytes_graft = K * sum(m * n for m, n in shp) * 26     # bf16 G: 2 + 3 * 4 B pass 1, 3 * 4 B pass 2
    roof_ms = ((flops_stats + flops_prec) / PEAK_F32_MFMA / 1e9 + bytes_graft / PEAK_HBM / 1e6) / K
    ms_step = elapsed * 1e3 / K
    ms_newton = rt["newton_f32"][0] + rt["newton_f64"][0]
    out = {
        "metric": "C5 grouped inverse roots (464 factors, sizes 128..2048) + bf16 stats+precondition+graft step",
        "value": ms_step, "unit": "ms/step", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": ms_step, "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32 (bf16-stored G)", "data": "synthetic",
        "config": {"workload": "C5: embedding 32768x1024 as 32 row blocks + 200 square blocks k in "
                               "{128,256,512,1024,2048}; G ~ N(0,1e-3) stored bf16; 10 stats steps; p=4, "
                               "eps 1e-6" + (f"; embedding gradient row-sparse, {args.emb_lookups} Zipf(1.1) "
                                             "lookups/step; damping eps * lambda_max" if sparse else ""),
                   "blocks": nb, "factors": len(As), "emb_lookups": args.emb_lookups,
                   "graft": "separate calls" if args.split_graft else "fused into preconditioning"},
        "phase_roofline_ms": roof_ms, "frac_of_phase_roofline": roof_ms / ms_step,
        **step_report(K, elapsed, times, el_s, t_s, flops_stats, flops_prec, bytes_graft,
                      K * sum(m * n for m, n in shp) * 12),
        "grouped_roots": {
            "roots": len(As), "ms": root_ms, "roots_per_s": len(As) / root_ms * 1e3,
            "newton_ms": ms_newton, "root_aux_ms": rt["root_aux"][0],
            "newton_tflops": executed / (ms_newton * 1e-3) / 1e12 if ms_newton else None,
            "newton_f32_tflops": (sum(pq * s for pq, s in zip(prods, sym)) / (rt["newton_f32"][0] * 1e-3) / 1e12
                                  if rt["newton_f32"][0] else None),
            "newton_f64_tflops": (sum(pq * s for pq, s in zip(prods64, sym)) / (rt["newton_f64"][0] * 1e-3) / 1e12
                                  if rt["newton_f64"][0] else None),
            "statuses": sorted(set(i["status"] for i in inf)),
            "n_fp64": len(esc),
            "iters_fp32_max": max(i["iters_fp32"] for i in inf),
            "iters_fp64_max": max((inf[j]["iters"] for j in esc), default=0),
            "executed_gflop": executed / 1e9, "no_early_exit_gflop": no_exit / 1e9,
            "early_exit_saving": 1.0 - executed / no_exit,
            "by_size": classes,
        },
    }
    kr = out["kernels"]
    out["roofline"] = {"kernel": "gemm_grouped_kernel (preconditioning, the step's largest phase)", "bound": "mfma",
                       "achieved": kr["precond_tflops"], "peak": PEAK_F32_MFMA, "unit": "TFLOP/s",
                       "frac": kr["precond_tflops"] / PEAK_F32_MFMA,
                       "step_frac_of_phase_roofline": roof_ms / ms_step}
    gr = out["grouped_roots"]
    gr["newton_f32_frac"] = gr["newton_f32_tflops"] / PEAK_F32_MFMA if gr["newton_f32_tflops"] else None
    gr["newton_f64_frac"] = gr["newton_f64_tflops"] / PEAK_F64_MFMA if gr["newton_f64_tflops"] else None
    return out


def run_c1(args, torch, B):
    """C1: one 128 x 128 block, ten steps of gradients N(0, 1/128); each step
    is the two-sided statistics, both inverse 4th roots (one grouped call),
    the preconditioning and the graft.  Latency-bound: the ten steps are run
    `--steps` times from the same initial state and timed per step."""
    from synth import configs as cfg
    dev = torch.device("cuda:0")
    n, nsteps = 128, 10
    Gs = [torch.from_numpy(cfg.c1_grad(t)).to(dev) for t in range(1, nsteps + 1)]
    W0 = torch.from_numpy(cfg.c1_weight()).to(dev)
    G = torch.zeros(n, n, device=dev)
    W, D, P = W0.clone(), torch.zeros(n, n, device=dev), torch.zeros(n, n, device=dev)
    L, R = torch.zeros(n, n, device=dev), torch.zeros(n, n, device=dev)
    Lr, Rr = torch.zeros(n, n, device=dev), torch.zeros(n, n, device=dev)
    blk = [B.Block(G=G, W=W, D=D, P=P, L=L, R=R, Lr=Lr, Rr=Rr)]
    h = B.shampoo_create(0)
    prm = B.shampoo_root_params_default(p=4, eps=1e-6)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([n, n], prm.precision), dtype=torch.uint8, device=dev)
    info = torch.zeros(16, dtype=torch.int32, device=dev)
    iters = []

    def run10(record):
        W.copy_(W0); D.zero_(); L.zero_(); R.zero_()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(nsteps):
            G.copy_(Gs[t])
            B.shampoo_update_stats(h, blk)
            B.shampoo_inv_root_batched(h, [L, R], [Lr, Rr], prm, ws, info)
            B.shampoo_precondition(h, blk)
            B.shampoo_graft(h, blk, 1e-2)
            if record:
                iters.append([i["iters"] for i in B.decode_root_info(info)])
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    for _ in range(args.warmup):
        run10(False)
    ts = [run10(False) for _ in range(args.steps)]
    run10(True)
    B.shampoo_destroy(h)
    us = float(np.median(ts)) / nsteps * 1e6
    out = {
        "metric": "C1 single 128x128 block: us per step (stats L,R + 2 inverse 4th roots + precondition + graft)",
        "value": us, "unit": "us/step", "n_gpus": 1, "steps": args.steps * nsteps, "warmup": args.warmup,
        "ms_per_step": us / 1e3, "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "C1: one 128x128 block, 10 steps of G ~ N(0,1/128), roots every step, p=4, "
                               "eps 1e-6, eta0 1e-2"},
        "us_per_step_min": min(ts) / nsteps * 1e6, "us_per_step_max": max(ts) / nsteps * 1e6,
        "root_iters_per_step": iters,
    }
    # useful flops of the ten steps: statistics (symmetric counting, both
    # sides), preconditioning (two products) and the roots' symmetric
    # products; at the fp32-MFMA peak they take a microsecond or two, so the
    # step is bound by launch and synchronisation latency, not by a unit
    sym = n * n * (n + 1)
    flops = nsteps * (2 * sym + 4 * n ** 3) + sum(newton_products(i, 4, True) * sym for it in iters
                                          for i in it)
    roof_us = flops / nsteps / (PEAK_F32_MFMA * 1e12) * 1e6
    out["roofline"] = {"kernel": "whole step (latency-bound)", "bound": "latency", "achieved": roof_us,
                       "peak": us, "unit": "us at fp32-MFMA peak vs measured us", "frac": roof_us / us}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--blocks", type=int, default=96)
    ap.add_argument("--workload", choices=["c1", "c2", "c3", "c4", "c5", "c6"], default="c2",
                    help="c2 (default): the metric's workload; c1: single-block latency; c3: ill-conditioned "
                         "roots; c4: the transformer-layer step; c5: mixed-size grouped roots and bf16 step; "
                         "c6: the embedding-table step")
    ap.add_argument("--scaling", choices=["power4", "frobenius"], default="power4",
                    help="cold-start scaling of the roots: power4 (library default, bound ||A^4||_F^(1/4)) or "
                         "frobenius (Algorithm 1 as printed)")
    ap.add_argument("--no-compare-scaling", action="store_true",
                    help="skip the comparison roots call under the other scaling (for profiling runs)")
    ap.add_argument("--vocab", type=int, default=32768, help="c6: table rows")
    ap.add_argument("--emb-lookups", type=int, default=0,
                    help="c5: row-sparse embedding gradient from this many Zipf lookups per step (0: dense)")
    ap.add_argument("--lookups", type=int, default=65536, help="c6: lookups per step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--split-graft", action="store_true",
                    help="c2, c4, c5: separate preconditioning and graft calls instead of the fused "
                         "shampoo_precondition_graft")
    ap.add_argument("--no-warm", action="store_true",
                    help="c2, c4: skip the warm-start roots measured after the timed steps")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="c2: no per-launch HIP events in the timed steps (whole-step time only)")
    ap.add_argument("--no-extra", action="store_true",
                    help="c2: skip the other workloads (C1, C3, C4, C5) that the default run reports under "
                         "'workloads' after the headline step")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="before the steps, copy a buffer of this size once (a plain copy kernel of known "
                         "traffic, to scale FETCH_SIZE/WRITE_SIZE counter readings)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this implementation runs on one GPU only (blocks would shard across GPUs "
                                   "with no communication inside the optimizer; that path is not built)",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import torch
    from paper_2002_09018_amd import binding as B

    runners = dict(c1=run_c1, c2=run_c2, c3=run_c3, c4=run_c4, c5=run_c5, c6=run_c6)
    out = runners[args.workload](args, torch, B)
    if args.workload == "c2" and not args.no_extra:
        # The other workloads of the scope table, each at its full size with
        # a bounded number of steps, so that one default run reports them all.
        extra = {}
        for name, steps, warmup in (("c1", 3, 1), ("c3", 0, 0), ("c4", 10, 2), ("c5", 5, 1)):
            torch.cuda.empty_cache()
            a = argparse.Namespace(**vars(args))
            a.workload, a.steps, a.warmup, a.emb_lookups = name, steps, warmup, 0
            t0 = time.perf_counter()
            log(f"workload {name}")
            r = runners[name](a, torch, B)
            r["bench_s"] = time.perf_counter() - t0
            extra[name] = r
            log(f"workload {name} done in {r['bench_s']:.1f} s")
        out["workloads"] = extra
    print(json.dumps(out), flush=True)


def run_c2(args, torch, B):
    """C2 (the metric's workload): 96 blocks, a step is the statistics
    update, 96 inverse 4th roots in one grouped call, the preconditioning and
    the graft.  Before every step the statistics are restored to their
    pristine L_19 (a device copy, timed and reported on its own), so each
    step roots exactly C2's matrices L_19 + G_20 G_20^T, whatever the number
    of steps."""
    dev = torch.device("cuda:0")
    nb, n, k, p, eps, eta0 = args.blocks, 1024, 4096, 4, 1e-6, 1e-2
    log(f"generating {nb} blocks")
    t0 = time.time()
    Ls, Gs, Ds, Ws = [], [], [], []
    sample = []
    # the statistics are views into one allocation, so the restore before
    # every step is one contiguous device copy
    Lall = torch.empty(nb, n, n, device=dev)
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 4)) as ex:
        for i, (L, G, D, W) in enumerate(ex.map(lambda i: gen_block(i, n, k), range(nb))):
            Lall[i].copy_(torch.from_numpy(L))
            Ls.append(Lall[i])
            Gs.append(torch.from_numpy(G).to(dev))
            Ds.append(torch.from_numpy(D).to(dev))
            Ws.append(torch.from_numpy(W).to(dev))
            if i < 24 and not args.no_cpu_baseline:
                sample.append((L, G, D, W))
            if (i + 1) % 24 == 0:
                log(f"  {i + 1}/{nb} blocks resident ({time.time() - t0:.1f} s)")
    if args.calib_copy_mb:
        src = torch.ones(args.calib_copy_mb * 2 ** 18, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.calib_copy_mb} MiB done")
        del src, dst
    L0all = Lall.clone()                   # pristine L_19, restored before every step
    Lrs = [torch.zeros(n, n, device=dev) for _ in range(nb)]
    Ps = [torch.zeros(n, k, device=dev) for _ in range(nb)]
    blocks = [B.Block(G=Gs[i], W=Ws[i], D=Ds[i], P=Ps[i], L=Ls[i], Lr=Lrs[i]) for i in range(nb)]
    h = B.shampoo_create(0)
    scaling = B.SCALING_POWER4 if args.scaling == "power4" else B.SCALING_FROBENIUS
    prm = B.shampoo_root_params_default(p=p, eps=eps, scaling=scaling)
    ws = torch.empty(B.shampoo_inv_root_workspace_bytes([n] * nb, prm.precision), dtype=torch.uint8, device=dev)
    info = torch.zeros(8 * nb, dtype=torch.int32, device=dev)
    infos = []

    restore_ev = []
    # the step's block views and root jobs, checked and packed once (the
    # calls repeat with the same tensors)
    pblocks = B.PackedBlocks(h, blocks)
    pjobs = B.PackedJobs(h, Ls, Lrs)

    def step(record, split=args.split_graft):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        Lall.copy_(L0all)
        e1.record()
        if record:
            restore_ev.append((e0, e1))
        B.shampoo_update_stats(h, pblocks)
        B.shampoo_inv_root_batched(h, pjobs, None, prm, ws, info)
        if record:
            infos.append(info.clone())
        if split:
            B.shampoo_precondition(h, pblocks)
            B.shampoo_graft(h, pblocks, eta0)
        else:  # graft pass 1 runs in the preconditioning GEMM's epilogue
            B.shampoo_precondition_graft(h, pblocks, eta0)

    for w in range(args.warmup):
        step(False)
        torch.cuda.synchronize()
        log(f"warmup step {w + 1}/{args.warmup} done")
    B.shampoo_timing_enable(h, not args.no_kernel_timing)
    for c in range(len(B.KCLASS_NAMES)):
        B.shampoo_timing_read(h, c)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(True)
        log(f"timed step {s + 1}/{args.steps} enqueued")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    B.shampoo_timing_enable(h, False)
    times = {B.KCLASS_NAMES[c]: B.shampoo_timing_read(h, c) for c in range(len(B.KCLASS_NAMES))}
    # The same steps with separate preconditioning and graft calls: the
    # statistics + preconditioning half of the metric and the per-kernel
    # rates (the fused call's preconditioning time also carries graft pass 1).
    el_s, t_s = time_steps(torch, B, h, lambda: step(False, True), args.steps)
    log("split-call steps done")
    other = B.SCALING_FROBENIUS if scaling == B.SCALING_POWER4 else B.SCALING_POWER4
    other_ms, other_iters = None, None
    if not args.no_compare_scaling:
        prm_o = B.shampoo_root_params_default(p=p, eps=eps, scaling=other)
        Xo = [torch.zeros(n, n, device=dev) for _ in range(nb)]
        B.shampoo_inv_root_batched(h, Ls, Xo, prm_o, ws, info)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(3):
            B.shampoo_inv_root_batched(h, Ls, Xo, prm_o, ws, info)
        torch.cuda.synchronize()
        other_ms = (time.perf_counter() - t1) * 1e3 / 3
        other_iters = float(np.mean([i["iters"] for i in B.decode_root_info(info)]))
        del Xo

    # Warm start (coupled-Newton appendix): one more statistics update, then
    # the roots of the new statistics from those of the last timed step,
    # beside the cold call on the same statistics.
    warm = None
    if not args.no_warm:
        # the next step's statistics L_21 = L_20 + G_21 G_21^T (a fresh
        # gradient), rooted warm from L_20's roots and cold
        from synth import configs as cfg
        X0 = [x.clone() for x in Lrs]
        with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 4)) as ex:
            for i, g in enumerate(ex.map(lambda i: cfg.c2_grad(i, n, k, 21), range(nb))):
                Gs[i].copy_(torch.from_numpy(g))
        B.shampoo_update_stats(h, blocks)
        Xc = [torch.zeros(n, n, device=dev) for _ in range(nb)]
        info_c = torch.zeros(8 * nb, dtype=torch.int32, device=dev)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        B.shampoo_inv_root_batched(h, Ls, Xc, prm, ws, info_c)
        torch.cuda.synchronize()
        cold_ms = (time.perf_counter() - t1) * 1e3
        warm = warm_measure(torch, B, h, Ls, X0, prm, ws, ref=Xc)
        warm["cold_ms_same_matrices"] = cold_ms
        warm["cold_iters_mean"] = float(np.mean([i["iters"] for i in B.decode_root_info(info_c)]))
        log(f"warm roots: {warm['ms']:.1f} ms (cold {cold_ms:.1f} ms), kept {warm['kept']}")
        del X0, Xc

    # algorithmic work
    # Products per matrix at p = 4: X M1, M1 M1, (M1^2)^2 and M1^4 M per
    # iteration, except the first, whose X product (X0 a multiple of I) is
    # not a GEMM: 4 iters - 1.  The power-bound scaling adds M0^2 and M0^4
    # and makes the first iteration's M1 M1 elementwise: 4 iters.
    def products(iters):
        return newton_products(iters, p, scaling == B.SCALING_POWER4)
    it32, it64, prod32, prod64 = 0, 0, 0, 0
    iters_per_step = []
    for t in infos:
        dec = B.decode_root_info(t)
        iters_per_step.append(float(np.mean([i["iters_fp32"] for i in dec])))
        for inf in dec:
            it32 += inf["iters_fp32"]
            prod32 += products(inf["iters_fp32"])
            if inf["precision"] == 64:
                it64 += inf["iters"]
                prod64 += products(inf["iters"])
    sym_prod = n * n * (n + 1)                     # symmetric product, upper-triangle counting
    flops_newton32 = prod32 * sym_prod
    flops_newton64 = prod64 * sym_prod
    flops_stats = args.steps * nb * n * (n + 1) * k
    flops_prec = args.steps * nb * 2 * n * n * k
    graft_bytes = args.steps * nb * n * k * 28   # pass 1: G, D, D', P; pass 2: W, P, W'
    ms_newton, launches_newton = times["newton_f32"]
    achieved = flops_newton32 / (ms_newton * 1e-3) / 1e12 if ms_newton > 0 else 0.0
    ms_step = elapsed * 1e3 / args.steps
    stats_prec_ms = (t_s["stats"][0] + t_s["precond"][0]) / args.steps
    out = {
        "metric": METRIC,
        "value": nb * args.steps / elapsed,
        "unit": "roots/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "C2 step: 96 blocks, L 1024x1024 (Wishart, 19x4096 dof) + G 1024x4096 "
                               "N(0,1/4096); stats + 96 inverse 4th roots (grouped coupled Newton, eps 1e-6, "
                               "tol 1e-6, AUTO precision) + L^-1/4 G + AdaGrad graft; L restored to L_19 "
                               "before every step (device copy, inside the timed region)",
                   "blocks": nb, "n": n, "k": k, "p": p, "eps": eps, "root_scaling": args.scaling,
                   "graft": "separate calls" if args.split_graft else "fused into preconditioning"},
        "roofline": {
            "kernel": "newton_stage_kernel<float> (grouped fp32-MFMA Newton products)",
            "bound": "mfma", "achieved": achieved, "peak": PEAK_F32_MFMA, "unit": "TFLOP/s",
            "frac": achieved / PEAK_F32_MFMA,
            "flops_per_launch": flops_newton32 / max(launches_newton, 1),
            "avg_launch_us": ms_newton * 1e3 / max(launches_newton, 1),
            "traffic": measured_traffic(),
            "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
        },
        "stats_precondition_ms_per_step": stats_prec_ms,
        # both passes are fp32-MFMA bound: roofline time of their algorithmic
        # flops (symmetric counting for the statistics) over the measured time
        "stats_precondition_roofline_frac": ((flops_stats + flops_prec) / args.steps / (PEAK_F32_MFMA * 1e12)
                                             / (stats_prec_ms * 1e-3) if stats_prec_ms else None),
        "fp32_mfma_util": achieved / PEAK_F32_MFMA,
        "phases_ms_per_step": {c: v[0] / args.steps for c, v in times.items()},
        "launches_per_step": {c: v[1] / args.steps for c, v in times.items()},
        "split_calls_phases_ms_per_step": {c: v[0] / args.steps for c, v in t_s.items()},
        "kernels": {
            "stats_tflops": flops_stats / (t_s["stats"][0] * 1e-3) / 1e12 if t_s["stats"][0] else None,
            "precond_tflops": flops_prec / (t_s["precond"][0] * 1e-3) / 1e12 if t_s["precond"][0] else None,
            "graft_gbs": graft_bytes / (t_s["graft"][0] * 1e-3) / 1e9 if t_s["graft"][0] else None,
            "fused_graft_pass2_gbs": (args.steps * nb * n * k * 12 / (times["graft"][0] * 1e-3) / 1e9
                                      if times["graft"][0] and not args.split_graft else None),
            "newton_f64_tflops": (flops_newton64 / (times["newton_f64"][0] * 1e-3) / 1e12
                                  if times["newton_f64"][0] else None),
        },
        "newton_iters_mean": it32 / max(1, nb * args.steps),
        "newton_iters_per_step": iters_per_step,
        "newton_iters_sample_blocks": [i["iters_fp32"] for i in B.decode_root_info(infos[-1])][:2],
        "restore_ms_per_step": float(np.mean([a.elapsed_time(b) for a, b in restore_ev])),
        "roots_per_s_root_phase": (nb * args.steps / ((times["newton_f32"][0] + times["newton_f64"][0]
                                                       + times["root_aux"][0]) * 1e-3)
                                   if times["newton_f32"][0] else None),
        "newton_products_per_root": prod32 / max(1, nb * args.steps),
        "other_scaling": None if other_ms is None else {
            "scaling": "frobenius" if scaling == B.SCALING_POWER4 else "power4",
            "roots_call_ms": other_ms, "roots_per_s_roots_call": nb / (other_ms * 1e-3), "iters_mean": other_iters},
        "warm_start_next_step": warm,
    }
    # device copy bandwidth (a plain 1 GiB copy), the practical ceiling of
    # the HBM-bound graft passes
    src = torch.empty(2 ** 28, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    out["hbm_copy_gbs"] = 5 * 2 * src.numel() * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    if not args.no_cpu_baseline:
        log("timing the oracle on a sample")
        out["cpu_baseline"] = cpu_baseline(sample, n, k, p, eps, eta0)
    B.shampoo_destroy(h)
    return out




if __name__ == "__main__":
    main()

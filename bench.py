"""Throughput of the HeteroFold transfer path on one MI355X.

One step = one pass of the whole path over one synthetic batch:
hf_build_alignment (GPU) -> hf_build_layer_map (host) -> hf_transfer_kv (GPU),
with inputs already resident in HBM.  Prints ONE JSON line (rank 0):

  value     receiver KV tokens per second (every receiver token of the batch,
            all layers, K and V), whole step
  roofline  the transfer kernel's achieved bf16 matrix-core TFLOP/s (algorithmic
            flops per launch / mean launch time from HIP events recorded on the
            launch stream over the timed steps) against the MI355X dense bf16 peak
  cpu_baseline  the fp64 CPU oracle on a bounded sample of the same workload

With --workload calib-14b (or calib-small) it times the offline construction
of one map instead: hf_recolor_moments -> hf_recolor_solve -> hf_fold_map over
2^20 synthetic calibration samples, value = samples/s, roofline = the fp64
covariance product against the MI355X fp64 matrix-core peak.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0
PEAK_FP64_TFLOPS = 78.6     # MI355X dense fp64 matrix-core peak
CALIB_METRIC = "calibration samples/sec for one map (moments + Recolor + fold, fp64)"
METRIC = "receiver KV tokens/sec (all layers, K+V) at 32K; % of MFMA/HBM roofline"
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_cost(cfg, seg):
    """Flops and HBM bytes of one transfer kernel launch:
    flops = 2 roles x L_r x 2 n d_r per receiver token, n the map's input size
    (d_in, or 3 d_in for the three-layer neighbourhood); bytes = each sender
    layer the layer map uses read once per role, the receiver cache written
    once, the maps read once."""
    from paper_2609_32259_amd import heterofold as hf
    T_r = int(seg.r_len.sum())
    T_s = int(seg.s_len.sum())
    el = 2 if cfg.dtype == "bf16" else 4
    n = cfg.d_map_in
    flops = 2 * cfg.L_r * 2 * n * cfg.d_r * T_r
    if cfg.layer_map == "neighbor3":
        used = set(hf.hf_build_layer_taps(cfg.L_s, cfg.L_r).reshape(-1).tolist())
    else:
        lo, hi, rem, _ = hf.hf_build_layer_map(cfg.L_s, cfg.L_r)
        used = set(lo.tolist()) | {int(h) for h, r in zip(hi, rem) if r}
    read = len(used) * 2 * T_s * cfg.d_in * el
    write = cfg.L_r * 2 * T_r * cfg.d_r * el
    maps = cfg.L_r * 2 * cfg.d_r * n * el + cfg.L_r * 2 * cfg.d_r * 4
    return flops, read + write + maps


def kernel_name(cfg):
    """The transfer kernel hf_transfer_kv(_taps) launches for this shape."""
    if cfg.dtype != "bf16":
        return "transfer_f32_kernel"
    if cfg.H_r in (4, 8) and cfg.H_s <= 8:
        return f"transfer_bf16_tiled_kernel<{cfg.H_r // 2}, {'true' if cfg.n_taps > 1 else 'false'}>"
    return f"transfer_bf16_direct_kernel<{cfg.H_r}>"


def kernel_traffic(cfg, staged=False):
    """HBM bytes per launch of the dominant kernel from a committed rocprofv3
    counter summary (profiles/*_traffic.json) of this workload and path, or
    None if there is none or the kernel's source changed since it was taken."""
    import glob
    path = "staged" if staged else "fused"
    for fn in sorted(glob.glob(os.path.join(PROFILES, "*_traffic.json"))):
        try:
            with open(fn) as f:
                rec = json.load(f)
            if rec.get("workload_name") != cfg.name or rec.get("path", "fused") != path:
                continue
            with open(os.path.join(ROOT, rec["kernel_source"]), "rb") as f:
                src = hashlib.sha256(f.read()).hexdigest()
            if rec.get("kernel_source_sha256") == src:
                return rec.get("bytes_per_launch")
        except (OSError, ValueError, KeyError):
            continue
    return None


def cpu_model() -> str:
    """The host CPU's model name and logical CPU count, from /proc/cpuinfo."""
    name = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{name}, {os.cpu_count()} logical CPUs"


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return os.cpu_count() or 1


def cpu_baseline_full(wl):
    """The fp64 oracle over the whole step at full length: the alignment of
    the batch and every receiver layer, K and V, each layer from its own sender
    taps (as ``cpu_baseline`` does for one layer).  One run, minutes of CPU."""
    from oracle import alignment as al
    from oracle import layer_map as lm
    from oracle import transfer as tr
    cfg, seg = wl.cfg, wl.seg
    if cfg.layer_map != "interp2" or wl.opts is not None:
        raise SystemExit("--cpu-baseline-full covers the interpolating map without options")
    lt = lm.interp2(cfg.L_s, cfg.L_r)
    t_total = 0.0
    for b in range(seg.batch):
        t0 = time.perf_counter()
        csr = al.build_alignment(*seg.seq(b), "overlap")
        t_total += time.perf_counter() - t0
        T_s = int(seg.s_len[b])
        rp = None if wl.rope is None else dict(wl.rope, pos0_s=0, pos0_r=0)
        for layer in range(cfg.L_r):
            lo, hi = int(lt[0][layer]), int(lt[1][layer])
            taps = [lo] if lt[2][layer] == 0 else [lo, hi]
            sub = (np.array([0]), np.array([len(taps) - 1]), lt[2][layer:layer + 1],
                   lt[3][layer:layer + 1])
            S = wl.S[b, taps, :, :, :T_s, :].float().cpu().numpy().astype(np.float64)
            A = wl.A[layer:layer + 1].float().cpu().numpy().astype(np.float64)
            bias = wl.bias[layer:layer + 1].float().cpu().numpy().astype(np.float64)
            t0 = time.perf_counter()
            tr.transfer(S, sub, csr, A, bias, rp, H_r=cfg.H_r)
            t_total += time.perf_counter() - t0
            del S
            log(f"[bench] oracle b={b} layer {layer}: {t_total:.1f} s so far")
    T_r = int(seg.r_len.sum())
    return {"value": T_r / t_total, "unit": "tokens/s", "cores": blas_threads(),
            "kind": "oracle", "cpu": cpu_model(),
            "sample": (f"fp64 NumPy oracle, the whole step at full length: overlap alignment and "
                       f"all {cfg.L_r} receiver layers, K and V, of {T_r} receiver tokens: "
                       f"{t_total:.1f} s of oracle time in one run (host copies of the cache "
                       f"excluded)")}


def cpu_baseline(wl, budget_s=30.0):
    """Time the fp64 oracle on the host: the full alignment of the batch plus
    one receiver layer (K and V) at full length; scale to the whole step."""
    from oracle import alignment as al
    from oracle import layer_map as lm
    from oracle import transfer as tr
    threads = blas_threads()
    cfg, seg = wl.cfg, wl.seg
    t0 = time.perf_counter()
    csr = [al.build_alignment(*seg.seq(b), "overlap") for b in range(seg.batch)]
    t_align = time.perf_counter() - t0
    layer = 1 if cfg.L_r > 1 else 0
    t_layer = 0.0
    for b in range(seg.batch):
        T_s = int(seg.s_len[b])
        A = wl.A[layer:layer + 1].float().cpu().numpy().astype(np.float64)
        bias = wl.bias[layer:layer + 1].float().cpu().numpy().astype(np.float64)
        rp = None if wl.rope is None else dict(wl.rope, pos0_s=0, pos0_r=0)
        opts = None
        if wl.opts is not None:
            opts = dict(inv_r=wl.opts["inv_r"][layer:layer + 1].cpu().numpy().astype(np.float64),
                        k_norm=wl.opts["k_norm"][layer:layer + 1].cpu().numpy().astype(np.float64),
                        k_norm_eps=wl.opts["k_norm_eps"])
        if cfg.layer_map == "neighbor3":
            taps = lm.neighbor3(cfg.L_s, cfg.L_r)[layer]
            S = wl.S[b, list(taps), :, :, :T_s, :].float().cpu().numpy().astype(np.float64)
            t0 = time.perf_counter()
            tr.transfer_taps(S, np.arange(len(taps))[None, :], csr[b], A, bias, rp, H_r=cfg.H_r,
                             opts=opts)
        else:
            lt = lm.interp2(cfg.L_s, cfg.L_r)
            lo, hi = int(lt[0][layer]), int(lt[1][layer])
            sub = (np.array([0]), np.array([1 if hi != lo else 0]), lt[2][layer:layer + 1],
                   lt[3][layer:layer + 1])
            taps = [lo] if hi == lo else [lo, hi]
            S = wl.S[b, taps, :, :, :T_s, :].float().cpu().numpy().astype(np.float64)
            t0 = time.perf_counter()
            tr.transfer(S, sub, csr[b], A, bias, rp, H_r=cfg.H_r, opts=opts)
        t_layer += time.perf_counter() - t0
        del S
    est = t_align + cfg.L_r * t_layer
    T_r = int(seg.r_len.sum())
    return {"value": T_r / est, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": (f"fp64 NumPy oracle: full overlap alignment of the batch ({t_align:.2f} s) "
                       f"+ receiver layer {layer} K and V at full length ({t_layer:.2f} s), "
                       f"scaled to {cfg.L_r} layers: {est:.1f} s per step of {T_r} receiver tokens")}


def cpu_baseline_calib(x, y, w, p, rank, budget_rows=16384):
    """The fp64 oracle on the host: weighted moments of the first budget_rows
    samples (scaled to all n) plus the Recolor solve and the fold on them."""
    from oracle import recolor as rc
    threads = blas_threads()
    n = int(x.shape[0])
    k = min(n, budget_rows)
    X = x[:k].double().cpu().numpy()
    Y = y[:k].double().cpu().numpy()
    W = w[:k].double().cpu().numpy()
    t0 = time.perf_counter()
    r = rc.sender_rms(X, W)
    mz, my, Szz, Szy, Syy = rc.weighted_moments(X / r, Y, W)
    t_mom = time.perf_counter() - t0
    t0 = time.perf_counter()
    A, b = rc.recolor(mz, my, Szz, Szy, Syy, 1e-6)
    q = A.shape[1]
    rng = np.random.default_rng(0)
    rc.fold(A, b, 0.02 * rng.standard_normal((q, rank)), rng.standard_normal((rank, q)))
    t_solve = time.perf_counter() - t0
    est = t_mom * n / k + t_solve
    return {"value": n / est, "unit": "samples/s", "cores": int(threads), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": (f"fp64 NumPy oracle: weighted moments of {k} samples ({t_mom:.2f} s, "
                       f"scaled to {n}) + Recolor solve and rank-{rank} fold ({t_solve:.2f} s): "
                       f"{est:.1f} s per map")}


def run_calibration(args, cfg):
    import torch
    from paper_2609_32259_amd import heterofold as hf
    from paper_2609_32259_amd import synth

    rank, ridge = 16, 1e-6
    log(f"[bench] workload {cfg.name}: generating samples on the GPU")
    x, y, w = synth.make_calibration(cfg, seed=args.seed, device="cuda")
    p, q, n = cfg.p, cfg.q, cfg.n
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed + 1)
    B = 0.02 * torch.randn((q, rank), generator=g, dtype=torch.float64, device="cuda")
    G = torch.randn((rank, q), generator=g, dtype=torch.float64, device="cuda")
    ws_m = torch.empty(hf.hf_recolor_moments_workspace_bytes(n, p, q), dtype=torch.uint8,
                       device="cuda")
    ws_s = torch.empty(hf.hf_recolor_solve_workspace_bytes(p, q), dtype=torch.uint8,
                       device="cuda")
    ws_f = torch.empty(hf.hf_fold_workspace_bytes(p, rank), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()

    def step():
        r, mu, cov = hf.hf_recolor_moments(x, y, w, workspace=ws_m)
        A, b, info = hf.hf_recolor_solve(mu, cov, p, ridge=ridge, workspace=ws_s)
        hf.hf_fold_map(A, b, B, G, out=(A, b), workspace=ws_f)
        return info

    log(f"[bench] n={n} p={p} q={q}; warmup {args.warmup}")
    info = None
    for _ in range(args.warmup):
        info = step()
    torch.cuda.synchronize()
    if info is not None:
        log(f"[bench] solve convergence {hf.recolor_info(info)}")
    hf.hf_profiler_reset()
    hf.hf_profiler_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        info = step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    hf.hf_profiler_enable(False)
    conv = hf.recolor_info(info)
    ms_step = (t1 - t0) * 1e3 / args.steps
    parts = {}
    for name, kid in (("stats", hf.HF_KERNEL_MOMENTS_STATS), ("cov", hf.HF_KERNEL_MOMENTS_COV),
                      ("solve", hf.HF_KERNEL_RECOLOR_SOLVE), ("fold", hf.HF_KERNEL_FOLD)):
        t, c = hf.hf_profiler_query(kid)
        # the statistics group runs twice per call (column sums, partial-sum reduction)
        parts[name] = t / max(c, 1) * (2 if kid == hf.HF_KERNEL_MOMENTS_STATS else 1)
    log(f"[bench] step {ms_step:.2f} ms; " + ", ".join(f"{k} {v:.2f} ms" for k, v in parts.items()))
    m = p + q
    flops = 2.0 * n * m * (m + 1) / 2   # distinct entries of the symmetric Gram product
    achieved = flops / (parts["cov"] * 1e-3) / 1e12
    roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_FP64_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP64_TFLOPS, 4), "traffic": None,
            "kernel": f"cov_kernel<{'float' if cfg.dtype == 'f32' else 'unsigned short'}>", "kernel_ms": round(parts["cov"], 3),
            "stats_ms": round(parts["stats"], 3), "solve_ms": round(parts["solve"], 3),
            "fold_ms": round(parts["fold"], 3)}
    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline_calib(x, y, w, p, rank)
    out = {
        "metric": CALIB_METRIC,
        "value": round(n / (ms_step * 1e-3), 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": cfg.name, "n": n, "p": p, "q": q, "sample_dtype": cfg.dtype,
                   "ridge": ridge, "rank": rank, "solve_converged": conv["converged"],
                   "solve_iterations": conv["iterations"], "parallelism": "single-gpu"},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def run_gemm_yardstick(args, cfg):
    """A plain library GEMM of the transfer's shape, as a yardstick for what a
    dense bf16 contraction reaches on this chip at the clock it holds: one
    batched product of 2 L_r (layer, role) pairs, [T_r x d_in] x [d_in x d_r]
    each, through torch.bmm (hipBLASLt), operands contiguous.  The features
    are random: nothing of the method is computed here."""
    import torch
    from paper_2609_32259_amd import synth

    seg = synth.make_segmentation(cfg, seed=args.seed)
    M = int(seg.r_len.sum())
    K, N, L = cfg.d_map_in, cfg.d_r, 2 * cfg.L_r
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed)
    X = torch.randn((L, M, K), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    W = (torch.randn((L, K, N), generator=g, device="cuda", dtype=torch.float32)
         / K ** 0.5).to(torch.bfloat16)
    Y = torch.empty((L, M, N), device="cuda", dtype=torch.bfloat16)
    log(f"[yardstick] bmm bf16 {L} x [{M} x {K}] x [{K} x {N}]; warmup {args.warmup}")
    for _ in range(args.warmup):
        torch.bmm(X, W, out=Y)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    for a, b in ev:
        a.record()
        torch.bmm(X, W, out=Y)
        b.record()
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    flops = 2.0 * L * M * K * N
    tf = flops / (ms.mean() * 1e-3) / 1e12
    del X, W, Y
    # The library's best case on this chip: one square 8192^3 product.
    S = 8192
    Xs = torch.randn((S, S), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    Ws = torch.randn((S, S), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    Ys = torch.empty((S, S), device="cuda", dtype=torch.bfloat16)
    for _ in range(args.warmup):
        torch.matmul(Xs, Ws, out=Ys)
    torch.cuda.synchronize()
    ev2 = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, b in ev2:
        a.record()
        torch.matmul(Xs, Ws, out=Ys)
        b.record()
    torch.cuda.synchronize()
    ms2 = np.array([a.elapsed_time(b) for a, b in ev2])
    tf2 = 2.0 * S ** 3 / (ms2.mean() * 1e-3) / 1e12
    out = {"yardstick": "torch.bmm bf16 (hipBLASLt)", "workload": cfg.name,
           "shape": {"batch": L, "M": M, "K": K, "N": N}, "steps": args.steps,
           "ms_mean": round(float(ms.mean()), 4), "ms_median": round(float(np.median(ms)), 4),
           "ms_min": round(float(ms.min()), 4), "tflops": round(tf, 1),
           "frac_of_peak": round(tf / PEAK_BF16_TFLOPS, 4),
           "square_8192": {"ms_mean": round(float(ms2.mean()), 4), "tflops": round(tf2, 1),
                           "frac_of_peak": round(tf2 / PEAK_BF16_TFLOPS, 4)}}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="14b-32k")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--path", choices=("auto", "fused", "staged"), default="auto",
                    help="transfer path: the library's staged path (build the aligned features "
                         "into the workspace, then a separate multiply) where the shape allows "
                         "it (auto), or force one")
    ap.add_argument("--T-s", dest="T_s", type=int, default=None,
                    help="sender tokens per sequence, overriding the workload's (the "
                         "reverse-b4 context sweep: 1024, 4096, 16384, 32768)")
    ap.add_argument("--cpu-baseline-full", action="store_true",
                    help="time the oracle over the whole step at full length instead of "
                         "one layer scaled (minutes of CPU)")
    ap.add_argument("--gemm-yardstick", action="store_true",
                    help="time a plain hipBLASLt bf16 GEMM of the workload's shape instead")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="first run one plain device copy of this many MiB (a known-size "
                         "reference for hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the transfer path is built and timed on a single "
              f"MI355X; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_32259_amd import heterofold as hf
    from paper_2609_32259_amd import synth
    from paper_2609_32259_amd.path import TransferPath

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    hf.lib()
    if args.copy_probe_mib:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device="cuda")
        dst = src.clone()
        torch.cuda.synchronize()
        log(f"[bench] copy probe: {args.copy_probe_mib} MiB read + {args.copy_probe_mib} MiB written")
        del src, dst
    if args.workload in synth.CALIB_CONFIGS:
        run_calibration(args, synth.CALIB_CONFIGS[args.workload])
        return
    cfg = synth.CONFIGS[args.workload]
    if args.T_s is not None:
        import re
        name = re.sub(r" T_s=\d+", "", cfg.name)
        cfg = cfg.with_(T_s=args.T_s, name=f"{name} T_s={args.T_s}")
    if args.gemm_yardstick:
        run_gemm_yardstick(args, cfg)
        return
    log(f"[bench] workload {cfg.name}: generating inputs on the GPU")
    wl = synth.make_workload(cfg, seed=args.seed, device="cuda")
    staged = {"auto": None, "fused": False, "staged": True}[args.path]
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r,
                        layer_map=cfg.layer_map, opts=wl.opts, staged=staged)
    torch.cuda.synchronize()
    T_r = int(wl.seg.r_len.sum())
    T_s = int(wl.seg.s_len.sum())
    log(f"[bench] B={wl.seg.batch} T_s={T_s} T_r={T_r}; warmup {args.warmup}")
    for _ in range(args.warmup):
        path.step()
    torch.cuda.synchronize()

    hf.hf_profiler_reset()
    hf.hf_profiler_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        path.step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    hf.hf_profiler_enable(False)
    ms_step = (t1 - t0) * 1e3 / args.steps
    sg_ms, sg_n = hf.hf_profiler_query(hf.HF_KERNEL_STAGED_GEMM)
    sb_ms, sb_n = hf.hf_profiler_query(hf.HF_KERNEL_STAGED_BUILD)
    ran_staged = sg_n > 0
    # The dominant kernel: the fused transfer kernel, or on the staged path its multiply.
    dom = hf.HF_KERNEL_STAGED_GEMM if ran_staged else hf.HF_KERNEL_TRANSFER
    k_ms, k_n = hf.hf_profiler_query(dom)
    a_ms, a_n = hf.hf_profiler_query(hf.HF_KERNEL_ALIGNMENT)
    r_ms, r_n = hf.hf_profiler_query(hf.HF_KERNEL_ROPE_TABLES)
    g_ms, g_n = hf.hf_profiler_query(hf.HF_KERNEL_TRANSFER_STAGE)
    k_avg = k_ms / max(k_n, 1)
    b_avg = sb_ms / max(sb_n, 1)
    ks = hf.hf_profiler_samples(dom).astype(np.float64)
    k_med, k_min, k_p90 = (float(np.median(ks)), float(ks.min()), float(np.percentile(ks, 90)))
    log(f"[bench] path {'staged' if ran_staged else 'fused'}; step {ms_step:.3f} ms; "
        f"{'multiply' if ran_staged else 'transfer'} kernel mean {k_avg:.3f} ms, median {k_med:.3f}, "
        f"min {k_min:.3f}, p90 {k_p90:.3f} (x{k_n}); "
        + (f"staged build {b_avg:.3f} ms; " if ran_staged else "")
        + f"alignment {a_ms / max(a_n, 1):.3f} ms; rope tables {r_ms / max(r_n, 1):.3f} ms; "
        f"tile staging {g_ms / max(g_n, 1):.3f} ms")

    flops, bytes_alg = algorithmic_cost(cfg, wl.seg)
    traffic = kernel_traffic(cfg, staged=ran_staged)
    # The binding roof: matrix-core time against HBM time of the algorithmic work.
    if bytes_alg / (PEAK_HBM_GBS * 1e9) > flops / (PEAK_BF16_TFLOPS * 1e12):
        bound, unit, peak = "hbm", "GB/s", PEAK_HBM_GBS
        achieved = bytes_alg / (k_avg * 1e-3) / 1e9
    else:
        bound, unit, peak = "mfma", "TFLOP/s", PEAK_BF16_TFLOPS
        achieved = flops / (k_avg * 1e-3) / 1e12
    roof = {"bound": bound, "achieved": round(achieved, 2), "peak": peak,
            "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
            "tflops": round(flops / (k_avg * 1e-3) / 1e12, 2), "algorithmic_flops": flops,
            "kernel": "staged_gemm_kernel" if ran_staged else kernel_name(cfg),
            "kernel_ms": round(k_avg, 4),
            "kernel_ms_median": round(k_med, 4), "kernel_ms_min": round(k_min, 4),
            "kernel_ms_p90": round(k_p90, 4),
            "alignment_ms": round(a_ms / max(a_n, 1), 4),
            "tile_staging_ms": round(g_ms / max(g_n, 1), 4),
            "algorithmic_bytes": bytes_alg,
            "hbm_GBps_algorithmic": round(bytes_alg / (k_avg * 1e-3) / 1e9, 1),
            "path": "staged" if ran_staged else "fused"}
    if ran_staged:  # the build kernel is part of the transfer: the path's own fraction too
        path_ms = k_avg + b_avg
        roof["staged_build_ms"] = round(b_avg, 4)
        roof["transfer_kernels_ms"] = round(path_ms, 4)
        roof["transfer_kernels_frac"] = round(flops / (path_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
    cpu = None
    if args.cpu_baseline_full:
        log("[bench] timing the CPU oracle over the whole step at full length")
        cpu = cpu_baseline_full(wl)
    elif not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(wl)
    out = {
        "metric": METRIC,
        "value": round(T_r / (ms_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "batch": wl.seg.batch, "T_s": T_s, "T_r": T_r,
                   "L_s": cfg.L_s, "L_r": cfg.L_r, "H_s": cfg.H_s, "H_r": cfg.H_r, "d_h": cfg.d_h,
                   "rope": list(cfg.rope) if cfg.rope else None, "alignment": "overlap",
                   "layer_map": cfg.layer_map,
                   "sender_keys": "post-rope" if cfg.sender_keys_post_rope else "pre-rope",
                   "inv_r_and_key_norm": bool(cfg.paper_opts), "parallelism": "single-gpu"},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

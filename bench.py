#!/usr/bin/env python3
"""Throughput of the Partial FC head step on one MI355X class shard.

One step = sampling + remap, gather + normalise, cosine contraction, margin
softmax cross-entropy, backward and the sparse momentum update, for one batch
of synthetic inputs already resident in HBM.  Default workload: the 8M-class
shard (one GPU's share of 64M classes), B = 1024, d = 512, r = 0.1, fp16
weights, ArcFace s = 64, m = 0.5; step t uses sampler seed t.

Prints ONE JSON line (last line of stdout) with the throughput, a roofline
entry for the step's dominant kernel (timed with HIP events inside the timed
region) and the CPU oracle timed on this host on a bounded sample.
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

METRIC = "samples/sec & ms/step, PFC head fwd+bwd+update, C_shard=8M r=0.1; %MFMA/%HBM peak"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {"sample": "sample.hip", "prep": "prep.hip", "fwd_gemm": "fwd.hip",
                  "lse": "fwd.hip", "dx_gemm": "bwd.hip", "dx_final": "bwd.hip",
                  "dw_update": "bwd.hip"}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_sha(name):
    path = os.path.join(ROOT, "paper_2010_05222_amd", "csrc", KERNEL_SOURCES[name])
    h = hashlib.sha256()
    for p in [path] + [os.path.join(ROOT, "paper_2010_05222_amd", "csrc", f)
                       for f in ("pfc_device.h", "pfc_gemm.h")]:
        with open(p, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def algorithmic_work(name, cfg, K):
    """(flops, bytes) the method must spend in one launch of a kernel."""
    from paper_2010_05222_amd import costmodel as cm
    B, d = cfg["B"], cfg["d"]
    if name in ("fwd_gemm", "dx_gemm"):
        return cm.contraction_flops(B, d, K), 0
    if name == "dw_update":
        return cm.contraction_flops(B, d, K), cm.update_bytes(K, d, cfg["dtype"], cfg["master"])
    return 0, 0


def roofline_entry(name, cfg, K, avg_ms, traffic):
    from paper_2010_05222_amd import costmodel as cm
    flops, nbytes = algorithmic_work(name, cfg, K)
    peak_tf = cm.PEAK_TFLOPS[cfg["dtype"]]
    t_mfma = flops / (peak_tf * 1e12)
    t_hbm = nbytes / (cm.PEAK_HBM_GBPS * 1e9)
    sec = avg_ms * 1e-3
    if t_hbm >= t_mfma:
        achieved = nbytes / sec / 1e9
        entry = {"bound": "hbm", "achieved": achieved, "peak": cm.PEAK_HBM_GBPS, "unit": "GB/s"}
    else:
        achieved = flops / sec / 1e12
        entry = {"bound": "mfma", "achieved": achieved, "peak": peak_tf, "unit": "TFLOP/s"}
    entry["frac"] = entry["achieved"] / entry["peak"]
    entry["traffic"] = traffic
    # The HBM rate the counters imply (every byte the kernel moves, its own
    # intermediates included), next to the algorithmic rate above.
    entry["traffic_GBps"] = traffic / sec / 1e9 if traffic else None
    entry["kernel"] = name
    entry["avg_ms"] = avg_ms
    return entry


def contraction_precision(dtype):
    """Operand and accumulator types of the step's three contractions."""
    if dtype == "f32":
        return {"forward": "f32 x f32 -> f32 (FMA)", "dx": "f32 x f32 -> f32 (FMA)",
                "dw": "f32 x f32 -> f32 (FMA)"}
    return {"forward": f"{dtype} x {dtype} -> f32 (MFMA)",
            "dx": (f"{dtype} W x {dtype} coefficients -> f32 (MFMA)"
                   + (", coefficients scaled by a power of two" if dtype == "f16" else "")),
            "dw": "bf16 x_hat x bf16 coefficients -> f32 (MFMA)"}


def gather_entry(cfg, K, stage_ms, traffic):
    """Stage a3 (gather + normalise of the sampled class rows, judged by HBM
    rate).  The gather has no kernel of its own: the forward contraction
    streams the active W rows from HBM straight into LDS.  Its rate is the
    compulsory gathered bytes (|S| rows of d elements, read once) over the
    forward kernel's time.  Also reports how many times a step reads the
    active W rows: the forward gathers them, the feature-gradient
    contraction gathers them again, and the class-gradient kernel reads them
    for the update (compulsory: the update is a read-modify-write)."""
    from paper_2010_05222_amd import costmodel as cm
    elt = cm.DTYPE_BYTES[cfg["dtype"]]
    nbytes = K * cfg["d"] * elt
    sec = stage_ms["fwd_gemm"] * 1e-3
    achieved = nbytes / sec / 1e9
    ent = {"bytes": nbytes, "kernel": "fwd_gemm", "achieved": achieved, "unit": "GB/s",
           "peak": cm.PEAK_HBM_GBPS, "frac": achieved / cm.PEAK_HBM_GBPS,
           "w_row_reads_per_step": 3, "w_row_read_bytes_per_step": 3 * nbytes}
    if traffic:
        ent["counter_read_bytes"] = traffic
    return ent


def measured_traffic_record(name, workload):
    """The committed counter record of a kernel (HBM bytes per launch), if it
    was taken on this workload and the kernel's source has not changed since."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    ent = rec.get(name)
    if not ent or ent.get("workload") != workload:
        return None
    if ent.get("source_sha256") != kernel_source_sha(name):
        return None
    return ent


def measured_traffic(name, workload):
    """HBM bytes per launch from committed counter runs, if they match the current kernel."""
    ent = measured_traffic_record(name, workload)
    return ent.get("bytes_per_launch") if ent else None


def cpu_baseline(cfg, W_dev, rows):
    """The CPU oracle, as it stands, on a bounded sample of the workload.

    Sample: the full shard's sampling (all C classes) and the full update of
    the |S| active rows, plus forward and backward of `rows` batch rows
    against all |S| active classes; the per-row part is scaled to the full
    batch.  Returns the baseline entry (samples/s) and the phase timings."""
    import numpy as np
    import torch
    from oracle import pfc_oracle as O
    import workloads

    X, labels = workloads.make_batch(cfg, 0)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg["dtype"]]
    Xs = torch.from_numpy(X[:rows]).to(tdt).double().numpy()
    Ls = labels[:rows]
    W = W_dev.cpu().numpy() if cfg["dtype"] != "bf16" else W_dev.float().cpu().numpy()
    C, d = cfg["C"], cfg["d"]
    t0 = time.perf_counter()
    active, mapped, _ = O.sample_active(Ls, C, cfg["a"], cfg["r"], 0)
    t1 = time.perf_counter()
    Ws = np.asarray(W[active], dtype=np.float64)
    fw = O.forward(Xs, Ws, mapped, cfg["s"], cfg["m"], cfg["margin"])
    O.grad_x(Xs, Ws, mapped, fw["lse"], rows, cfg["s"], cfg["m"], cfg["margin"])
    g = O.grad_w(Xs, Ws, np.arange(len(active)), mapped, fw["lse"], rows, cfg["s"], cfg["m"],
                 cfg["margin"])
    t2 = time.perf_counter()
    M = np.zeros((C, d), dtype=np.float32)
    O.momentum_update(W, M, active, g, cfg["lr"], cfg["mu"], cfg["dtype"])
    t3 = time.perf_counter()
    t_step = (t1 - t0) + (t3 - t2) + (t2 - t1) * cfg["B"] / rows
    threads = 1
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        threads = max([i.get("num_threads", 1) for i in info] + [1])
    except Exception:  # noqa: BLE001 - threadpoolctl is optional
        pass
    entry = {"value": cfg["B"] / t_step, "unit": "samples/s", "cores": threads, "kind": "oracle",
             "sample": (f"full sampling over C={C} and full update of |S|={len(active)} rows, "
                        f"forward+backward of {rows} of {cfg['B']} rows against all |S| classes, "
                        f"row part scaled x{cfg['B'] // rows}; float64 NumPy, BLAS threads "
                        f"{threads}, host affinity {len(os.sched_getaffinity(0))} cpus"),
             "phase_s": {"sample": t1 - t0, "rows": t2 - t1, "update": t3 - t2},
             "cpu_seconds": t3 - t0}
    return entry


def run_tiered(args, cfg):
    """The same workload with the class bank in pinned host memory: every step
    stages its cold rows over the host link and writes its rows back
    (TieredShard); prints one JSON line of its own."""
    import numpy as np
    import torch
    import workloads
    from paper_2010_05222_amd.head import TieredShard

    dev = torch.device("cuda:0")
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg["dtype"]]
    B, d, C = cfg["B"], cfg["d"], cfg["C"]
    ts = TieredShard(B, d, C, cfg["r"], dtype=cfg["dtype"], class_offset=cfg["a"], s=cfg["s"],
                     m=cfg["m"], margin=cfg["margin"], lr=cfg["lr"], mu=cfg["mu"], device=dev,
                     master=cfg["master"])
    W, master = workloads.make_weights_device(cfg, dev)
    ts.W_bank.copy_(W)
    if master is not None:
        ts.P_bank.copy_(master)
    del W, master
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    wbytes = ts.W_bank.element_size() * d + 4 * d * (2 if cfg["master"] else 1)
    log(f"[bench] tiered: bank of {C} rows in pinned host memory "
        f"({C * wbytes / 2**30:.2f} GiB), {ts.n} slots of {ts.cap} rows")
    n = args.warmup + args.steps
    batches = []
    for t in range(n + 1):
        seed = t - args.warmup if t >= args.warmup else 10**6 + t
        X, L = workloads.make_batch(cfg, seed)
        batches.append((torch.from_numpy(X).to(tdt).to(dev), torch.from_numpy(L).to(dev), seed))
    torch.cuda.synchronize()
    ts.begin(batches[0][1], batches[0][2])
    sets = []
    t0 = None
    for t in range(n):
        if t == args.warmup:
            ts.finish()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
        nxt = batches[t + 1] if t + 1 < n else None
        out = ts.step(batches[t][0], nxt[1] if nxt else None, nxt[2] if nxt else None)
        if t >= args.warmup:
            sets.append((out.active.clone(), out.n_active.clone()))
    ts.finish()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    stale = ts.stale_rows()
    loss = float(out.loss.item())
    ms = elapsed * 1e3 / args.steps
    # Rows over the host link per step: up, the rows of S(t) in none of the
    # sets still held in slots; down, the rows of S(t) not in S(t+1) (those
    # are written back by the next step; the last step writes all).
    acts = [a[:int(k.item())].cpu().numpy() for a, k in sets]
    Ks = [len(a) for a in acts]
    cold, gone = [], []
    for t, a in enumerate(acts):
        held = acts[max(0, t - ts.n + 1):t]
        cold.append(len(np.setdiff1d(a, np.concatenate(held))) if held else len(a))
        gone.append(len(np.setdiff1d(a, acts[t + 1])) if t + 1 < len(acts) else len(a))
    up = float(np.mean(cold[ts.n - 1:] if len(cold) >= ts.n else cold)) * wbytes
    down = float(np.mean(gone[:-1] if len(gone) > 1 else gone)) * wbytes
    peak = 64.0       # PCIe 5.0 x16, one direction
    log(f"[bench] tiered {args.steps} steps: {ms:.2f} ms/step, up {up / 1e9:.2f} GB/step "
        f"({up / ms / 1e6:.1f} GB/s), down {down / 1e9:.2f} GB/step ({down / ms / 1e6:.1f} GB/s), "
        f"stale rows {stale}, last loss {loss:.4f}")
    if stale or not np.isfinite(loss):
        raise RuntimeError("tiered run: stale rows or non-finite loss")
    print(json.dumps({
        "metric": METRIC + " (tiered: class bank in pinned host memory)",
        "value": B * args.steps / elapsed, "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg["dtype"], "data": "synthetic",
        "config": {"workload": f"{cfg['name']} with the class bank in host memory: B={B} d={d} "
                               f"C_shard={C} r={cfg['r']}", "global_batch": B, "d": d,
                   "C_shard": C, "r": cfg["r"], "bank": "pinned host memory",
                   "parallelism": "one class shard on one GPU"},
        "roofline": {"bound": "host-link", "achieved": max(up, down) / ms / 1e6, "peak": peak,
                     "unit": "GB/s", "frac": max(up, down) / ms / 1e6 / peak, "traffic": None,
                     "kernel": "bank stage + write-back"},
        "host_link": {"up_GB_per_step": up / 1e9, "down_GB_per_step": down / 1e9,
                      "up_GBps": up / ms / 1e6, "down_GBps": down / ms / 1e6,
                      "cold_rows_mean": up / wbytes, "written_rows_mean": down / wbytes,
                      "active_mean": float(np.mean(Ks)), "slots": ts.n},
        "last_loss": loss,
    }), flush=True)


def measured_ceilings(dev, dtype):
    """What plain library work reaches on this GPU, next to the published
    peaks: a large 16-bit GEMM (torch.matmul, 8192^3, the library's own MFMA
    kernel) and a 1 GiB device-to-device copy."""
    import torch
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[dtype]
    n = 8192
    a = torch.randn((n, n), device=dev).to(tdt).contiguous()
    b = torch.randn((n, n), device=dev).to(tdt).contiguous()
    for _ in range(3):
        torch.matmul(a, b)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    e0.record()
    for _ in range(reps):
        torch.matmul(a, b)
    e1.record()
    torch.cuda.synchronize()
    gemm_tflops = 2.0 * n ** 3 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del a, b
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbps = 2.0 * (1 << 30) * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return {"gemm_8192_tflops": gemm_tflops, "copy_1GiB_GBps": copy_gbps,
            "gemm_dtype": dtype}


def library_same_shape(dev, dtype, B, d, K, copy_gbps, update_bytes):
    """The library's own GEMM (torch.matmul) on the step's three contraction
    shapes, with contiguous random operands and none of the path's other work
    (no gather, no epilogue, no update): [B,d]x[d,K] with a 16-bit [B,K]
    result (the forward), [B,K]x[K,d] (dX), and [K,B]x[B,d] with the class
    operand stored class-major (dW's contraction).  For dW the library figure
    adds the update's compulsory bytes at the measured copy rate, as a
    separate update kernel would need."""
    import torch
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16}[dtype]
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    X = torch.randn((B, d), device=dev, generator=g).to(tdt)
    W = (torch.randn((K, d), device=dev, generator=g) * 0.05).to(tdt)
    G = (torch.rand((B, K), device=dev, generator=g) * 1e-3).to(tdt)
    Gt = G.t().contiguous()
    out = torch.empty((B, K), device=dev, dtype=tdt)

    def ms_of(f, reps=10):
        for _ in range(2):
            f()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            f()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    res = {"forward_ms": ms_of(lambda: torch.matmul(X, W.t(), out=out)),
           "dx_ms": ms_of(lambda: torch.matmul(G, W)),
           "dw_gemm_ms": ms_of(lambda: torch.matmul(Gt, X))}
    res["dw_gemm_plus_update_ms"] = res["dw_gemm_ms"] + update_bytes / (copy_gbps * 1e9) * 1e3
    res["dtype"] = dtype
    del X, W, G, Gt, out
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="massive")
    ap.add_argument("--kernel-steps", type=int, default=5,
                    help="steps per untimed per-kernel timing pass")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=32)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--tiered", action="store_true",
                    help="keep the class bank in pinned host memory (staged per step)")
    ap.add_argument("--tau", type=float, default=None,
                    help="PFC* conflict threshold (a negative whose cosine exceeds it leaves "
                         "the row's denominator); default: plain PFC")
    ap.add_argument("--serial", action="store_true",
                    help="draw each step's active set in the step itself, rather than on a "
                         "side stream beside the previous step")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU's class shard only (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE {world}); runs over several GPUs are not supported.", flush=True)
        sys.exit(2)

    import numpy as np
    import torch
    import workloads
    from paper_2010_05222_amd import pfc as abi
    from paper_2010_05222_amd.head import PfcPipeline

    cfg = workloads.config(args.workload)
    dev = torch.device("cuda:0")
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg["dtype"]]
    B, d, C = cfg["B"], cfg["d"], cfg["C"]
    log(f"[bench] workload {cfg['name']}: B={B} d={d} C={C} r={cfg['r']} {cfg['dtype']}")
    if args.tiered:
        run_tiered(args, cfg)
        return

    W, master = workloads.make_weights_device(cfg, dev)
    M = torch.zeros((C, d), dtype=torch.float32, device=dev)
    pipe = PfcPipeline(B, d, C, cfg["r"], dtype=cfg["dtype"], class_offset=cfg["a"], s=cfg["s"],
                       m=cfg["m"], margin=cfg["margin"], lr=cfg["lr"], mu=cfg["mu"], device=dev,
                       tau=args.tau)
    shard = pipe.parts[0]
    n_extra = args.warmup + args.kernel_steps * len(abi.KERNEL_NAMES)
    batches = []
    # One batch more than the timed steps: the last step draws the next active
    # set, so the timed region holds exactly `steps` samplings either way.
    for t in range(args.steps + 1):
        X, L = workloads.make_batch(cfg, t)
        batches.append((torch.from_numpy(X).to(tdt).to(dev), torch.from_numpy(L).to(dev), t))
    extra = []
    for i in range(n_extra):
        X, L = workloads.make_batch(cfg, 10**6 + i)
        extra.append((torch.from_numpy(X).to(tdt).to(dev), torch.from_numpy(L).to(dev),
                      10**6 + i))
    torch.cuda.synchronize()
    log(f"[bench] inputs resident: W {W.numel() * W.element_size() / 2**30:.2f} GiB, "
        f"momentum {M.numel() * 4 / 2**30:.2f} GiB, workspace 2 x "
        f"{shard.ws_bytes / 2**30:.2f} GiB")

    serial_shard = shard

    def run(batch):
        X, L, seed = batch
        serial_shard.step(X, L, W, M, seed, master)

    it = iter(extra)
    if args.serial:
        for _ in range(args.warmup):
            run(next(it))
    else:
        # Warm both buffer sets of the pipeline.
        warm = [next(it) for _ in range(args.warmup)]
        if warm:
            pipe.begin(warm[0][1], warm[0][2])
            for i, (X, _, _) in enumerate(warm):
                nxt = warm[i + 1] if i + 1 < len(warm) else None
                pipe.step(X, W, M, nxt[1] if nxt else None, nxt[2] if nxt else None, master)
    torch.cuda.synchronize()
    log("[bench] warm-up done")

    # Untimed per-kernel passes: mean duration of each kernel (HIP events).
    stage_ms = {}
    for kid, name in abi.KERNEL_NAMES.items():
        abi.pfc_timing_begin(kid, args.kernel_steps)
        for _ in range(args.kernel_steps):
            run(next(it))
        torch.cuda.synchronize()
        tot, n = abi.pfc_timing_end()
        stage_ms[name] = tot / max(n, 1)
    K = int(shard.n_active.item())
    contenders = {k: v for k, v in stage_ms.items() if k != "sample"}
    dominant = max(contenders, key=contenders.get)
    dom_id = {v: k for k, v in abi.KERNEL_NAMES.items()}[dominant]
    log(f"[bench] |S|={K}; per-kernel ms: " +
        ", ".join(f"{k}={v:.4f}" for k, v in stage_ms.items()) + f"; dominant {dominant}")

    # Timed region: exactly `steps` steps; the dominant kernel bracketed by HIP events.
    # Per-step HIP events on the step's stream give the median / p99 step time.
    # By default step t+1's active set is drawn on a side stream beside step t
    # (PfcPipeline): the first step's before the region, one past the last
    # inside it.
    timed = batches[:args.steps]
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in timed]
    if not args.serial:
        pipe.begin(batches[0][1], batches[0][2])
    abi.pfc_timing_begin(dom_id, args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t, (e0, e1) in enumerate(ev):
        e0.record()
        if args.serial:
            run(timed[t])
        else:
            X, _, _ = timed[t]
            shard = pipe.step(X, W, M, batches[t + 1][1], batches[t + 1][2], master)
        e1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    step_ms = np.array([e0.elapsed_time(e1) for e0, e1 in ev])
    dom_total, dom_n = abi.pfc_timing_end()
    dom_avg = dom_total / max(dom_n, 1)
    loss = float(shard.loss.item())
    ms_per_step = elapsed * 1e3 / args.steps
    log(f"[bench] timed {args.steps} steps: {ms_per_step:.4f} ms/step, last loss {loss:.4f}, "
        f"{dominant} avg {dom_avg:.4f} ms over {dom_n} launches")
    if not np.isfinite(loss):
        raise RuntimeError("non-finite loss")

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("[bench] copy calibration: 3 x 1 GiB device copies")

    from paper_2010_05222_amd import costmodel as cm
    roof = roofline_entry(dominant, cfg, K, dom_avg, measured_traffic(dominant, cfg["name"]))
    step_fl = cm.step_flops(B, d, K)
    upd_b = cm.update_bytes(K, d, cfg["dtype"], cfg["master"])
    stage_roofs = {}
    for name, ms in stage_ms.items():
        fl, nb = algorithmic_work(name, cfg, K)
        if fl or nb:
            stage_roofs[name] = roofline_entry(name, cfg, K, ms, None)["frac"]
    reads = {}
    for name in ("fwd_gemm", "dx_gemm", "dw_update"):
        rec = measured_traffic_record(name, cfg["name"])
        if rec:
            reads[name] = rec["read_bytes"]
    gather = gather_entry(cfg, K, stage_ms, reads or None)
    stage_roofs["gather"] = gather["frac"]

    ceil = measured_ceilings(dev, cfg["dtype"] if cfg["dtype"] != "f32" else "bf16")
    log(f"[bench] measured ceilings: {ceil['gemm_8192_tflops']:.0f} TFLOP/s "
        f"({ceil['gemm_dtype']} GEMM 8192^3), {ceil['copy_1GiB_GBps']:.0f} GB/s (1 GiB copy)")
    dw_bytes = cm.update_bytes(K, d, cfg["dtype"], cfg["master"])
    vs_ceil = {
        "fwd_gemm": cm.contraction_flops(B, d, K) / (stage_ms["fwd_gemm"] * 1e-3) / 1e12
        / ceil["gemm_8192_tflops"],
        "dx_gemm": cm.contraction_flops(B, d, K) / (stage_ms["dx_gemm"] * 1e-3) / 1e12
        / ceil["gemm_8192_tflops"],
        "dw_update": dw_bytes / (stage_ms["dw_update"] * 1e-3) / 1e9 / ceil["copy_1GiB_GBps"],
    }
    lib = vs_lib = None
    if cfg["dtype"] in ("bf16", "f16"):
        lib = library_same_shape(dev, cfg["dtype"], B, d, K, ceil["copy_1GiB_GBps"], dw_bytes)
        vs_lib = {"fwd_gemm": lib["forward_ms"] / stage_ms["fwd_gemm"],
                  "dx_gemm": lib["dx_ms"] / stage_ms["dx_gemm"],
                  "dw_update": lib["dw_gemm_plus_update_ms"] / stage_ms["dw_update"]}
        log(f"[bench] library GEMM on the same shapes: forward {lib['forward_ms']:.3f} ms, "
            f"dX {lib['dx_ms']:.3f} ms, dW {lib['dw_gemm_ms']:.3f} ms "
            f"(+ update at copy rate {lib['dw_gemm_plus_update_ms']:.3f} ms)")

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle on a bounded sample ({args.cpu_rows} rows)...")
        cpu = cpu_baseline(cfg, W, args.cpu_rows)
        log(f"[bench] CPU oracle: {cpu['value']:.3f} samples/s ({cpu['cpu_seconds']:.1f} s)")

    out = {
        "metric": METRIC,
        "value": B * args.steps / elapsed,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "step_ms_median": float(np.median(step_ms)),
        "step_ms_p99": float(np.percentile(step_ms, 99)),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": f"{cfg['name']}: B={B} d={d} C_shard={C} r={cfg['r']} "
                               f"|S|={K} {cfg['margin']} s={cfg['s']} m={cfg['m']}",
                   "global_batch": B, "d": d, "C_shard": C, "r": cfg["r"], "active": K,
                   "margin": cfg["margin"], "w_dtype": cfg["dtype"], "momentum": "f32",
                   "contractions": contraction_precision(cfg["dtype"]),
                   "tau": args.tau,
                   "sampling": ("in the step" if args.serial else
                                "step t+1's active set drawn on a side stream beside step t"),
                   "parallelism": "one class shard on one GPU"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "stage_ms": stage_ms,
        "stage_roofline_frac": stage_roofs,
        "gather": gather,
        "measured_ceilings": ceil,
        "stage_frac_of_measured_ceiling": vs_ceil,
        "library_same_shape": lib,
        "stage_speed_vs_library_same_shape": vs_lib,
        "step_mfma_frac": step_fl / (ms_per_step * 1e-3) / (cm.PEAK_TFLOPS[cfg["dtype"]] * 1e12),
        "update_hbm_frac": upd_b / (stage_ms["dw_update"] * 1e-3) / (cm.PEAK_HBM_GBPS * 1e9),
        "last_loss": loss,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

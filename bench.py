#!/usr/bin/env python3
"""Benchmark of one training step of the Lattice Network's sparse-dense core
on one MI355X.

A step is one call of lattice_step on one batch: pooled lookups, bottom MLP,
FM interaction, top MLP, masked BCE, full backward, row-coalesced embedding
gradient and row-sparse SGD on the tables.  Default workload: B=8192, 64
tables of 2,000,000 x 128 bf16 (Zipf 1.05 indices, Poisson(20) bags clipped to
[1,128]), dense 64 -> 512 -> 128, FM over 65 vectors with rank 32, top
2208 -> 1024 -> 512 -> 16, 50% masked heads, SGD lr 0.01 on the tables.
Inputs are seeded and synthetic and resident in HBM before timing starts.

Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFS = 2516.6    # MI355X dense bf16 MFMA, TFLOP/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large-emb-fm",
                    help="one of: tiny-dot-f32, mid-dot-bf16, large-emb-fm, multidomain-dot, deep-stack")
    ap.add_argument("--batches", type=int, default=4, help="distinct batches cycled")
    ap.add_argument("--cpu-sample", type=int, default=2048, help="samples in the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--uniform", action="store_true", help="uniform indices (control run)")
    ap.add_argument("--single-stream", action="store_true",
                    help="no side stream: every stage on the step's stream (no overlap)")
    ap.add_argument("--fp8", choices=["precise", "fast"], default=None,
                    help="mixed FP8/BF16 training: the top MLP's hidden-layer forward GEMMs in FP8 e4m3 "
                         "(row-wise scales) with fast accumulation off (precise) or on (fast)")
    ap.add_argument("--top-act", choices=["relu", "swishrn", "hardswishrn"], default="relu",
                    help="activation of the top MLP's hidden layers (SwishRN: RMS-normalised self-gated, "
                         "sigmoid or hard-sigmoid gate)")
    ap.add_argument("--norm-block", type=int, choices=[128, 0], default=128,
                    help="SwishRN groups: 128 (BlockNorm, in the GEMM epilogue) or 0 (whole-row RMSNorm)")
    ap.add_argument("--towers", type=int, default=0,
                    help="per-objective towers: the last hidden top layer becomes T towers of this many "
                         "units each (replacing its width) and every head reads only its tower")
    ap.add_argument("--untie", type=int, default=0,
                    help="multi-domain workloads: the first N top layers hold one parameter set per "
                         "domain (parameter untying; batches grouped by domain)")
    ap.add_argument("--lcb-n", type=int, default=0,
                    help="stacked workloads: output vectors of each fusion block's linear compression "
                         "block (full DHEN/Wukong fusion blocks; 0: FM block only)")
    ap.add_argument("--fp8-proj", choices=["precise", "fast"], default=None,
                    help="stacked workloads: the FM blocks' projection in FP8 e4m3 (row-wise scales)")
    ap.add_argument("--infer", action="store_true",
                    help="time the forward alone (lattice_forward, inference); with --fp8 fast: FP8 serving")
    ap.add_argument("--no-skip-absent", action="store_true",
                    help="multi-domain DOT: compute the slots of absent features too (control run)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the timed steps, stream 1 GiB through a plain elementwise kernel "
                         "(torch.neg, 1 GiB read + 1 GiB written) as a counter calibration point")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def mlp_fwd_flops(dims, B):
    return sum(2.0 * B * dims[i] * dims[i + 1] for i in range(len(dims) - 1))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the training step is not sharded across GPUs)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    from paper_2512_09200_amd import api
    from paper_2512_09200_amd._abi import STAGES

    if args.workload not in synth.WORKLOADS:
        print(f"unknown workload {args.workload!r}; choose from {sorted(synth.WORKLOADS)}", file=sys.stderr)
        sys.exit(2)
    cfg = synth.WORKLOADS[args.workload]
    if args.uniform:
        cfg = cfg.scaled(index_dist=("uniform",))
    if args.towers:
        if args.fp8:
            print("--fp8 needs the dense heads", file=sys.stderr)
            sys.exit(2)
        T = cfg.top[-1]
        cfg = cfg.scaled(top=tuple(cfg.top[:-2]) + (T * args.towers, T), towers=args.towers)
    if args.untie:
        if not cfg.domains or args.fp8:
            print("--untie needs a multi-domain workload and tied FP8 layers", file=sys.stderr)
            sys.exit(2)
        cfg = cfg.scaled(untie=args.untie)
    if args.lcb_n:
        if cfg.interact != "stack":
            print("--lcb-n needs a stacked workload", file=sys.stderr)
            sys.exit(2)
        cfg = cfg.scaled(lcb_n=args.lcb_n)
    if args.fp8_proj:
        if cfg.interact != "stack":
            print("--fp8-proj needs a stacked workload", file=sys.stderr)
            sys.exit(2)
        cfg = cfg.scaled(stack_fp8=args.fp8_proj)
    if args.top_act != "relu":
        if args.fp8:
            print("--fp8 needs ReLU top layers", file=sys.stderr)
            sys.exit(2)
        cfg = cfg.scaled(top_act=args.top_act, norm_block=args.norm_block)
    dev = "cuda"
    sdt = synth.torch_dtype(cfg.dtype)
    t0 = time.time()
    log(f"[bench] {cfg.name}: generating {args.batches} batches")
    batches = []
    for i in range(args.batches):
        b = synth.make_batch(cfg, i)
        batches.append(dict(
            np=b, offsets=torch.from_numpy(b["offsets"]).to(dev),
            indices=torch.from_numpy(b["indices"]).to(dev),
            dense=torch.from_numpy(b["dense"]).to(sdt).to(dev),
            labels=torch.from_numpy(b["labels"]).to(dev), mask=torch.from_numpy(b["mask"]).to(dev),
            nnz=int(b["offsets"][-1]), U=distinct_rows(b, cfg),
            domain_offsets=b["domain_offsets"] if cfg.untie else None))
    row_base = torch.from_numpy(batches[0]["np"]["row_base"]).to(dev)
    log(f"[bench] batches ready ({time.time() - t0:.1f}s); generating tables")
    E = synth.make_tables(cfg, device=dev)
    p = synth.make_dense_params(cfg)

    def lin(W, b):
        return dict(W=torch.from_numpy(W).to(sdt).to(dev), b=torch.from_numpy(b).to(dev),
                    dW=torch.empty(W.shape, device=dev), db=torch.empty(b.shape, device=dev))

    bottom = [lin(W, b) for W, b in p["bottom"]]
    top = [lin(W, b) for W, b in p["top"]]
    for L, (ga, gb) in zip(top, p.get("top_gain", [])):
        L["gain"] = torch.from_numpy(np.stack([ga, gb], axis=-2)).to(dev)
        L["dgain"] = torch.empty(tuple(L["gain"].shape), device=dev)
    fm_W = torch.from_numpy(p["fm_W"]).to(sdt).to(dev) if "fm_W" in p else None
    fm_dW = torch.empty(tuple(fm_W.shape), device=dev) if fm_W is not None else None
    stack = None
    if "stack" in p:
        stack = []
        for lay in p["stack"]:
            d = {k: torch.from_numpy(lay[k]).to(sdt).to(dev) for k in ("W", "A")}
            d["gamma"] = torch.from_numpy(lay["gamma"]).to(dev)
            d["C"] = torch.from_numpy(lay["C"]).to(sdt).to(dev) if lay["C"] is not None else None
            d["L"] = torch.from_numpy(lay["L"]).to(sdt).to(dev) if lay.get("L") is not None else None
            for k in ("W", "A", "gamma", "C", "L"):
                if d[k] is not None:
                    d["d" + k] = torch.empty(tuple(d[k].shape), device=dev)
            stack.append(d)
    # multi-domain batches leave whole features absent: the DOT forward skips them
    skip_absent = cfg.interact == "dot" and cfg.domains is not None and not args.no_skip_absent
    model = api.StepModel(tables=E, row_base=row_base, num_features=cfg.F, dense_in=cfg.dense_in,
                          max_rows=cfg.rows,
                          bottom=bottom, top=top, interact=cfg.interact, fm_W=fm_W, fm_dW=fm_dW,
                          pool=cfg.pool, stack=stack, stack_n=cfg.stack_n, ln_eps=cfg.ln_eps,
                          top_act=cfg.top_act, norm_block=cfg.norm_block, norm_eps=cfg.norm_eps,
                          towers=bool(cfg.towers), n_domains=len(cfg.domains[0]) if cfg.untie else 0,
                          untied_layers=cfg.untie, skip_absent=skip_absent, fp8_proj=cfg.stack_fp8)
    nnz_max = max(b["nnz"] for b in batches)
    lay = api.lattice_step_plan(model, cfg.B, nnz_max, cfg.lr_tables, False, fp8_top=args.fp8)
    ws = torch.empty(lay.total_bytes, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    log(f"[bench] inputs resident ({time.time() - t0:.1f}s); workspace {lay.total_bytes / 2**30:.2f} GiB")

    side = api.SideStream()

    def step(i, events=None, one_stream=args.single_stream):
        b = batches[i % len(batches)]
        api.lattice_step(model, b["offsets"], b["indices"], b["dense"], b["labels"], b["mask"], ws,
                         cfg.lr_tables, False, stage_events=events, nnz_capacity=nnz_max,
                         side=None if one_stream else side, fp8_top=args.fp8,
                         domain_offsets=b["domain_offsets"])

    def forward(i, events=None, one_stream=args.single_stream):
        b = batches[i % len(batches)]
        api.lattice_forward(model, b["offsets"], b["indices"], b["dense"], cfg.B, ws,
                            nnz_capacity=nnz_max, side=None if one_stream else side, fp8_top=args.fp8,
                            domain_offsets=b["domain_offsets"])
        if events is not None:
            raise ValueError("stage events: use the step")

    for i in range(args.warmup):
        (forward if args.infer else step)(i)
    torch.cuda.synchronize()
    log("[bench] warmup done")

    if args.infer:
        # inference: the forward alone (lattice_forward), no labels, no update
        t_start = time.perf_counter()
        for i in range(args.steps):
            forward(args.warmup + i)
        torch.cuda.synchronize()
        ms = 1e3 * (time.perf_counter() - t_start) / args.steps
        print(json.dumps({
            "metric": "inference samples/s (forward) at 1 GPU", "value": round(cfg.B / (ms * 1e-3), 1),
            "unit": "samples/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": cfg.dtype if not args.fp8 else f"{cfg.dtype}+fp8-e4m3(top hidden fwd, {args.fp8} accumulation)",
            "data": "synthetic (seeded; Zipf/Poisson jagged batches, random-init weights)",
            "config": {"workload": cfg.name, "global_batch": cfg.B, "mode": "forward only",
                       "fp8_top": args.fp8, "top_act": cfg.top_act, "towers": cfg.towers or None,
                       "untied_top_layers": cfg.untie or None, "dot_skip_absent": skip_absent or None},
            "roofline": None, "cpu_baseline": None}))
        return

    nst = len(STAGES)

    def make_events(n, stages=None):
        # begin / end event of each stage (all, or those named), recorded on
        # the stream that runs it; None entries are not recorded
        ev = [[torch.cuda.Event(enable_timing=True) if stages is None or STAGES[k // 2] in stages
               else None for k in range(2 * nst)] for _ in range(n)]
        for es in ev:      # create the underlying events before handing them to the library
            for e in es:
                if e is not None:
                    e.record()
        torch.cuda.synchronize()
        return ev

    def stage_times(ev, stages=STAGES):
        return {s: float(np.mean([e[2 * k].elapsed_time(e[2 * k + 1]) for e in ev]))
                for k, s in enumerate(STAGES) if s in stages}

    # Timed region: every event record costs GPU time, so only the kernels
    # reported as roofline lines are bracketed here (live, on their stream).
    timed_stages = ["embbag_fwd", "embbag_reduce"]
    ev = make_events(args.steps, timed_stages)
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, ev[i])
    torch.cuda.synchronize()
    t_total = time.perf_counter() - t_start
    ms_per_step = 1e3 * t_total / args.steps
    timed_ms = stage_times(ev, timed_stages)
    # Attribution after the timed region: every stage bracketed, overlapped
    # as in the timed steps (stage_ms), then on one stream (the kernels' own
    # rates: stages sharing the GPU with the side stream run slower than alone)
    ev_all = make_events(args.steps)
    for i in range(args.steps):
        step(args.warmup + args.steps + i, ev_all[i])
    torch.cuda.synchronize()
    stage_ms = stage_times(ev_all)
    log("[bench] stage ms: " + ", ".join(f"{k}={v:.3f}" for k, v in stage_ms.items()))
    if args.single_stream:
        iso_ms = stage_ms
    else:
        ev_iso = make_events(args.steps)
        for i in range(args.steps):
            step(args.warmup + 2 * args.steps + i, ev_iso[i], one_stream=True)
        torch.cuda.synchronize()
        iso_ms = stage_times(ev_iso)
        log("[bench] stage ms, one stream: " + ", ".join(f"{k}={v:.3f}" for k, v in iso_ms.items()))

    # ---- algorithmic work -------------------------------------------------
    es = 2 if cfg.dtype == "bf16" else 4
    nnz = float(np.mean([b["nnz"] for b in batches]))
    U = float(np.mean([b["U"] for b in batches]))        # distinct rows per batch
    bags = cfg.F * cfg.B
    row_bytes = cfg.d * es
    upd = U * 2 * row_bytes if cfg.lr_tables else U * 4 * cfg.d   # SGD read+write, or fp32 G
    # Compulsory bytes (what the kernel must move at least once): each
    # distinct table row once, each index / offset once, each pooled row or
    # dX row once.
    fwd_bytes = U * row_bytes + nnz * 4 + bags * 4 + bags * cfg.d * es
    red_bytes = nnz * 8 + bags * cfg.d * es + upd
    # Logical bytes (every lookup counted as a row read, every occurrence as
    # a dX row read): the rate the kernels deliver to the arithmetic,
    # including rows re-read from L2 / MALL.
    fwd_logical = nnz * (row_bytes + 4) + bags * 4 + bags * cfg.d * es
    red_logical = nnz * (cfg.d * es + 8) + upd
    # whole sparse-gradient stage, logical (sort and bookkeeping are overhead)
    bwd_bytes = nnz * (cfg.d * es + 4) + bags * 4 + upd
    bwd_stages = ["embbag_sort", "embbag_runs", "embbag_reduce", "embbag_fixup"]
    bwd_ms = sum(iso_ms[s] for s in bwd_stages)

    def gbs(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9

    fwd_gbs = gbs(fwd_bytes, timed_ms["embbag_fwd"])
    red_gbs = gbs(red_bytes, timed_ms["embbag_reduce"])
    bwd_gbs = gbs(bwd_bytes, bwd_ms)
    n = cfg.n_slots
    flops_fwd = mlp_fwd_flops((cfg.dense_in,) + tuple(cfg.bottom), cfg.B) if cfg.has_dense else 0.0
    flops_fwd += mlp_fwd_flops((cfg.top_in,) + tuple(cfg.top[:-1]), cfg.B)
    flops_fwd += 2.0 * cfg.B * cfg.top[-1] * (cfg.towers if cfg.towers else cfg.top[-2])   # heads
    if cfg.interact == "fm":
        flops_fwd += 4.0 * cfg.B * n * cfg.d * cfg.fm_rank
    elif cfg.interact == "dot":
        flops_fwd += 2.0 * cfg.B * cfg.n_pairs * cfg.d
    elif cfg.interact == "stack":
        nl = n
        for l in range(cfg.stack_layers):
            flops_fwd += 4.0 * cfg.B * nl * cfg.d * cfg.fm_rank                      # FM block
            nF = cfg.stack_n - cfg.lcb_n
            flops_fwd += 2.0 * cfg.B * (nl * cfg.fm_rank) * (nF * cfg.d)             # FM projection
            flops_fwd += 2.0 * cfg.B * cfg.lcb_n * nl * cfg.d                        # linear compression block
            if l == 0 and nl != cfg.stack_n:
                flops_fwd += 2.0 * cfg.B * cfg.stack_n * nl * cfg.d                  # residual C X
            nl = cfg.stack_n
    dense_stages = ["bottom_fwd", "interact_fwd", "top_fwd", "loss", "top_bwd", "interact_bwd",
                    "top_wgrad", "bottom_bwd"]
    dense_ms = sum(iso_ms[s] for s in dense_stages)
    mfma_tfs = 3.0 * flops_fwd / (dense_ms * 1e-3) / 1e12
    samples_per_s = cfg.B / (ms_per_step * 1e-3)

    def roof(kernel, stage, nbytes, logical):
        ms = timed_ms[stage]
        t = counted_traffic(cfg.name, kernel)
        r = {"bound": "hbm", "kernel": kernel, "achieved": round(gbs(nbytes, ms), 1),
             "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs(nbytes, ms) / HBM_PEAK_GBS, 4),
             "traffic": t, "bytes_per_launch": int(nbytes), "launch_ms": round(ms, 4),
             "logical_bytes_per_launch": int(logical), "logical_GBps": round(gbs(logical, ms), 1)}
        if t:
            r["dram_GBps"] = round(gbs(t, ms), 1)
            r["dram_frac"] = round(gbs(t, ms) / HBM_PEAK_GBS, 4)
        return r

    # dominant kernel: the segmented reduction of the sparse gradient
    roofline = roof("seg_reduce_kernel", "embbag_reduce", red_bytes, red_logical)
    gather_roofline = roof("embbag_fwd_kernel", "embbag_fwd", fwd_bytes, fwd_logical)

    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # ---- CPU baseline: the oracle on a bounded sample of the same workload ----
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, batches[0]["np"], p, E, args.cpu_sample)

    out = {
        "metric": "train samples/s (fwd+bwd) at 1 GPU; EmbBag HBM GB/s and interaction MFMA util",
        "value": round(samples_per_s, 1), "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype if not args.fp8 else f"{cfg.dtype}+fp8-e4m3(top hidden fwd, {args.fp8} accumulation)",
        "data": "synthetic (seeded; Zipf/Poisson jagged batches, random-init weights)",
        "config": {"workload": cfg.name, "global_batch": cfg.B, "features": cfg.F,
                   "rows_per_table": cfg.rows, "dim": cfg.d,
                   "index_dist": list(cfg.index_dist), "bag_dist": list(cfg.bag_dist),
                   "interaction": cfg.interact, "top": list(cfg.top), "lr_tables": cfg.lr_tables,
                   "nnz_per_step": int(nnz), "distinct_rows_per_step": int(U),
                   "batches_cycled": len(batches), "parallelism": "single-gpu",
                   "fp8_top": args.fp8,
                   "top_act": cfg.top_act,
                   "lcb_n": cfg.lcb_n if cfg.interact == "stack" else None,
                   "towers": cfg.towers or None,
                   "untied_top_layers": cfg.untie or None,
                   "dot_skip_absent": skip_absent or None,
                   "fp8_stack_projection": cfg.stack_fp8,
                   "norm_block": cfg.norm_block if cfg.top_act != "relu" else None,
                   "sparse_sort_stream": "step" if args.single_stream else "side"},
        "roofline": roofline,
        "gather_roofline": gather_roofline,
        "embbag_fwd_GBps": round(fwd_gbs, 1), "embbag_fwd_hbm_frac": round(fwd_gbs / HBM_PEAK_GBS, 4),
        "embbag_bwd_logical_GBps": round(bwd_gbs, 1),
        "embbag_bwd_ms": round(bwd_ms, 4),
        "interaction_mlp_TFLOPs": round(mfma_tfs, 1),
        "interaction_mlp_mfma_frac": round(mfma_tfs / MFMA_BF16_PEAK_TFS, 4),
        "stage_ms": {k: round(x, 4) for k, x in stage_ms.items()},
        "stage_ms_one_stream": {k: round(x, 4) for k, x in iso_ms.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def distinct_rows(batch, cfg):
    """Distinct global table rows a batch touches (host-side bookkeeping of the
    bench's byte counts; the step computes its own on the GPU)."""
    import numpy as np
    lengths = np.diff(batch["offsets"].astype(np.int64))
    feat = np.repeat(np.arange(cfg.F * cfg.B, dtype=np.int64) // cfg.B, lengths)
    keys = batch["row_base"].astype(np.int64)[feat] + batch["indices"].astype(np.int64)
    return int(np.unique(keys).size)


def source_digest(files):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def counted_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    counter summary (FETCH_SIZE + WRITE_SIZE, each scaled by the reading of a
    copy kernel of known size), or None when there is none or the kernel's
    sources have changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.txt")
    try:
        kv = {}
        for line in open(path):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
        files = kv["sources"].split()
        if source_digest(files) != kv["sources_sha256"]:
            return None
        return int(kv["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def cpu_baseline(cfg, batch, params, E, n_samples):
    """Times the CPU oracle (as it stands) on the first n_samples samples of
    the batch, with the touched table rows copied to host memory."""
    import numpy as np
    import torch

    import synth
    from oracle import step as ostep

    Bs = min(n_samples, cfg.B)
    scfg, sub, rows = synth.sub_batch(cfg, batch, np.arange(Bs))
    table = E[torch.from_numpy(rows).to(E.device)].float().cpu().double().numpy()
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 0) for i in threadpool_info()), default=None)
    except Exception:
        pass
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    t = time.perf_counter()
    ostep.step(scfg, params, table, sub)
    dt = time.perf_counter() - t
    return {"value": round(Bs / dt, 3), "unit": "samples/s", "cores": threads or os.cpu_count(),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"first {Bs} of {cfg.B} samples of batch 0 (all {cfg.F} features, "
                      f"{int(sub['offsets'][-1])} lookups, {rows.size} touched rows), fwd+bwd+SGD "
                      "in float64 numpy", "cpu_model": cpu_model, "nproc": os.cpu_count()}


if __name__ == "__main__":
    main()

"""Benchmark of the BaryCache hot path on one MI355X.

One step = one BaryCache sampling run of the whole batch through the full
schedule (every full step runs the block stack, every other step the K-way
forecast; all steps run the final layer and the sampler update), starting
from resident noise.  Default workload: the DiT-XL/2-shaped class-conditional
model (28 blocks, D 1152, 16 x 72 heads, MLP 4608, 256 tokens), batch 16,
50 DDIM steps, K = 3, one full step every 4 (14 of 50), bf16, random-init
weights drawn from seed 2026.

Prints one JSON line: samples/s, the roofline of the dominant kernel (of the
fc2, fc1 and self-attention kernels, the one with the most time per run, each
timed with HIP events on its launch stream; the others follow), the forecast
kernel's HBM bandwidth on [8, 16384, 3072] features, the speedup over the
all-full mask, and the oracle's CPU throughput on a bounded sample.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="dit_xl2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-forecast", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="skip timing the HIP-graph replay of the run")
    ap.add_argument("--no-blockwise", action="store_true", help="skip timing the blockwise-mode run")
    ap.add_argument("--adaptive-ell", type=float, default=0.13,
                    help="threshold of the timed adaptive-schedule run (negative: skip it)")
    ap.add_argument("--kernels-only", action="store_true",
                    help="only launch the roofline kernels (fc2, fc1, self-attention of the workload's block, the "
                         "K = 3 forecast) a few times each through the C ABI, for hardware-counter passes")
    ap.add_argument("--cpu-steps", type=int, default=9, help="oracle sample: first N steps of one sample")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one 1 GiB device copy through the library (counter calibration)")
    return ap.parse_args()


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2608_28670_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counters_traffic(kernel_tag, src_hash, launches_bytes_ref):
    """HBM bytes per launch from committed rocprofv3 counter summaries, or None
    if none exist for the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel_tag}_counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        c = json.load(f)
    if c.get("source_hash") != src_hash:
        return None
    return c.get("hbm_bytes_per_launch")


def forecast_bench(bc, torch, dev, K=3, dtype="bf16", iters=10):
    """HBM bandwidth of the forecast kernel on K cached [8, 16384, 3072] features."""
    import synth
    shape = synth.FORECAST_SHAPE
    n = shape[0] * shape[1] * shape[2]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device=dev)
    g.manual_seed(synth.SEED + K)
    storage = torch.empty((K, n), dtype=tdt, device=dev)
    for j in range(K):
        storage[j].normal_(generator=g)
    ring = bc.CacheRing(K, storage)
    s, t = synth.forecast_times(K)
    for j in reversed(range(K)):
        ring.push(None, float(s[j]))
    w = bc.bary_weights(s, t)
    out = torch.empty(n, dtype=tdt, device=dev)
    for _ in range(2):
        bc.bary_extrapolate(ring, w, out)
    torch.cuda.synchronize()
    bc.profile_enable(bc.PROF_FORECAST, iters)
    for _ in range(iters):
        bc.bary_extrapolate(ring, w, out)
    ms, cnt = bc.profile_collect(bc.PROF_FORECAST)
    esz = 2 if dtype == "bf16" else 4
    bytes_alg = (K + 1) * n * esz
    avg_s = ms / cnt / 1e3
    gbs = bytes_alg / avg_s / 1e9
    del storage, out
    torch.cuda.empty_cache()
    return {"K": K, "dtype": dtype, "shape": list(shape), "bytes_per_launch": bytes_alg,
            "avg_us": round(avg_s * 1e6, 2), "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}


def device_params(cfg, torch, dev):
    """Random-init weights drawn on the GPU (N(0, 1) * param_scale, seeded):
    the multi-billion-parameter video workload would take minutes and tens of
    GB of host memory to draw on the host, and throughput does not depend on
    the values."""
    import synth
    g = torch.Generator(device=dev)
    g.manual_seed(synth.SEED)
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    out = {}
    for name, shape in synth.param_shapes(cfg):
        t = torch.empty(shape, dtype=torch.float32, device=dev)
        t.normal_(0.0, cfg.param_scale, generator=g)
        if name.endswith("_norm"):   # RMSNorm scales sit around 1
            t.add_(1.0)
        out[name] = t.to(dt)
        del t
    return out


def cpu_baseline(cfg, params, labels, xT, mask, nsteps):
    """The oracle on the host cores, on one sample and the first `nsteps` steps
    of the schedule; per-step times composed to the whole schedule."""
    import numpy as np
    from oracle import bary, model as om, sampler as osm
    M = om.Model(cfg, params)
    x = xT[:1].astype(np.float64)
    lab = labels[:1]
    steps = bary.plan(mask, cfg.K)
    tin = osm.model_time(cfg.sampler, cfg.steps, cfg.flow_shift)
    smp = osm.Sampler(cfg.sampler, cfg.steps, cfg.in_ch, cfg.flow_shift)
    ring = bary.Ring(cfg.K)
    t_full, t_fc = [], []
    for k in range(min(nsteps, cfg.steps)):
        t0 = time.perf_counter()
        cond = M.condition(tin[k], 1, lab)
        if mask[k]:
            feat = M.stack(M.embed(x), cond, None)
            ring.push(feat, k)
        else:
            st = steps[k]
            feat = bary.forecast([ring.slots[i] for i in st.slots], st.w)
        out = M.final(feat, cond)
        x = smp.step(k, x, out)
        (t_full if mask[k] else t_fc).append(time.perf_counter() - t0)
    nfull = int(mask.sum())
    per_sample = nfull * np.mean(t_full) + (cfg.steps - nfull) * np.mean(t_fc)
    cores = len(os.sched_getaffinity(0))
    return {"value": round(1.0 / per_sample, 6), "unit": "samples/s", "cores": cores, "kind": "oracle",
            "sample": (f"1 sample, steps 0-{nsteps - 1} of the {cfg.steps}-step schedule "
                       f"({len(t_full)} full at {np.mean(t_full):.2f} s, {len(t_fc)} forecast at "
                       f"{np.mean(t_fc) * 1e3:.1f} ms), composed to {nfull} full + {cfg.steps - nfull} "
                       f"forecast steps; numpy fp64 on {cores} host threads")}


def kernels_only(args):
    """The roofline kernels at the workload's shapes, each launched `args.steps`
    times on synthetic operands (no sampling loop): the program the byte
    counters are collected on."""
    import torch

    import synth
    import paper_2608_28670_amd as bc
    if not os.path.exists(bc.LIB_PATH):
        from paper_2608_28670_amd import build
        build.build()
    dev = "cuda:0"
    cfg = synth.CONFIGS[args.workload]
    M, D, F = cfg.batch * cfg.tokens, cfg.hidden, cfg.mlp
    g = torch.Generator(device=dev)
    g.manual_seed(synth.SEED)

    def rnd(*shape, dt=torch.bfloat16, scale=0.02):
        t = torch.empty(shape, dtype=torch.float32, device=dev)
        t.normal_(0.0, scale, generator=g)
        return t.to(dt)

    h, w1, b1, hm = rnd(M, D), rnd(F, D), rnd(F), torch.empty((M, F), dtype=torch.bfloat16, device=dev)
    w2, b2 = rnd(D, F), rnd(D)
    x, gate = rnd(M, D, dt=torch.float32, scale=1.0), rnd(cfg.batch, D, dt=torch.float32, scale=1.0)
    H, dh, T = cfg.heads, cfg.head_dim, cfg.tokens
    q, k, v = (rnd(cfg.batch, T, H, dh, scale=1.0) for _ in range(3))
    o = torch.empty_like(q)
    for _ in range(args.steps):
        bc.linear(h, w1, b1, hm, bc.EPI_BIAS_GELU)
        bc.linear(hm, w2, b2, x, bc.EPI_GATE_RES, res=x, gate=gate, rows_per_gate=T)
        bc.attention(q, k, v, o)
    torch.cuda.synchronize()
    del h, w1, b1, hm, w2, b2, x, gate, q, k, v, o
    torch.cuda.empty_cache()
    forecast_bench(bc, torch, dev, K=3, dtype="bf16", iters=args.steps)
    if args.calib_copy:
        n = 1 << 29
        src = torch.ones(n, dtype=torch.bfloat16, device=dev)
        store = torch.empty((1, n), dtype=torch.bfloat16, device=dev)
        ring = bc.CacheRing(1, store)
        ring.push(src, 0.0)
        torch.cuda.synchronize()
    print(json.dumps({"kernels_only": args.workload, "launches_each": args.steps}))


def main():
    args = parse()
    if args.kernels_only:
        kernels_only(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    import paper_2608_28670_amd as bc
    from paper_2608_28670_amd import loader

    if not os.path.exists(bc.LIB_PATH):
        from paper_2608_28670_amd import build
        build.build()
    dev = "cuda:0"
    cfg = synth.CONFIGS[args.workload]
    t0 = time.time()
    # Host weights (shared with the oracle's CPU baseline) for the default
    # image workload; GPU-drawn weights for the others.
    host_weights = args.workload == "dit_xl2"
    params = synth.params(cfg) if host_weights else None
    dm = loader.DeviceModel(cfg, params, dev_params=None if host_weights else device_params(cfg, torch, dev))
    B = cfg.batch
    mask = bc.make_mask(cfg.steps, cfg.interval)
    labels = synth.labels(cfg) if cfg.n_classes else None
    text = synth.text(cfg) if cfg.kind != "dit" else None
    xT = synth.latents(cfg)
    x0 = torch.from_numpy(xT).to(dev)
    x = torch.empty_like(x0)
    tl = torch.from_numpy(labels).to(dev) if labels is not None else None
    tt = torch.from_numpy(text).to(dev).to(loader.torch_dtype(cfg)) if text is not None else None
    print(f"setup {time.time() - t0:.1f} s", file=sys.stderr)

    def run(m):
        x.copy_(x0)
        dm.sample(x, m, labels=tl, text=tt)

    for _ in range(args.warmup):
        run(mask)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        run(mask)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed / args.steps * 1e3
    value = B * args.steps / elapsed

    # Kernel classes timed with per-launch HIP events on their launch stream
    # in one extra sampling run (the events ride on the launches themselves),
    # right after the timed runs and in the same state: where a full step's
    # time goes, and the roofline of the dominant kernel.
    nfull = int(mask.sum())
    classes = {"gemm_gelu": bc.PROF_GEMM_GELU, "gemm_down": bc.PROF_GEMM_DOWN, "gemm_gated": bc.PROF_GEMM_GATE,
               "gemm_bias": bc.PROF_GEMM_BIAS, "attention": bc.PROF_ATTENTION, "layernorm": bc.PROF_LAYERNORM}
    cap = 16 * nfull * cfg.depth + 1024
    for c in classes.values():
        bc.profile_enable(c, cap)
    run(mask)
    breakdown, times = {}, {}
    for name, c in classes.items():
        t = bc.profile_times(c, cap).astype(np.float64)
        times[name] = t
        if len(t):
            breakdown[name] = {"ms_per_run": round(float(t.sum()), 3), "launches": len(t),
                               "avg_us": round(float(t.mean()) * 1e3, 2)}
    roofline, others = None, []
    if cfg.kind in ("dit", "pixart"):
        M_rows = B * cfg.tokens
        nb = nfull * cfg.depth
        gemm_hash = source_hash("gemm.hip", "gemm.h", "hip_common.h")
        att_hash = source_hash("attention.hip", "attention.h", "hip_common.h")
        # One launch per block and full step for each candidate.  PixArt's
        # caption MLP (once per run, before the loop) is the first GELU GEMM;
        # its cross-attention follows each self-attention.
        att = times["attention"] if cfg.kind == "dit" else times["attention"][0::2]
        cands = [
            ("gemm fc2 (gated residual, MLP down projection)", times["gemm_down"], "mfma",
             2.0 * M_rows * cfg.hidden * cfg.mlp, [M_rows, cfg.hidden, cfg.mlp], f"gemm_fc2_{cfg.name}", gemm_hash),
            ("gemm fc1 (bias+GELU)", times["gemm_gelu"][-nb:], "mfma",
             2.0 * M_rows * cfg.mlp * cfg.hidden, [M_rows, cfg.mlp, cfg.hidden], f"gemm_fc1_{cfg.name}", gemm_hash),
            ("self-attention", att, "mfma",
             4.0 * B * cfg.heads * cfg.tokens * cfg.tokens * cfg.head_dim,
             [B, cfg.heads, cfg.tokens, cfg.head_dim], f"attention_{cfg.name}", att_hash),
        ]
        recs = []
        for name, t, bound, flops, shape, tag, h in cands:
            assert len(t) == nb, (name, len(t), nb)
            avg_s = float(t.mean()) / 1e3
            achieved = flops / avg_s / 1e12
            recs.append((float(t.sum()), {
                "bound": bound, "kernel": name, "shape": shape, "flops_per_launch": flops,
                "avg_us": round(avg_s * 1e6, 2), "launches": len(t), "ms_per_run": round(float(t.sum()), 3),
                "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": counters_traffic(tag, h, None), "source_hash": h}))
        recs.sort(key=lambda r: -r[0])
        roofline, others = recs[0][1], [r[1] for r in recs[1:]]


    # The same run replayed from a HIP graph captured once (bc_sample_graph_*).
    graph = None
    if not args.no_graph:
        g = dm.sample_graph(x, mask, labels=tl, text=tt)
        for _ in range(max(1, args.warmup)):
            x.copy_(x0)
            g.launch()
        torch.cuda.synchronize()
        tg = time.perf_counter()
        for _ in range(args.steps):
            x.copy_(x0)
            g.launch()
        torch.cuda.synchronize()
        eg = time.perf_counter() - tg
        graph = {"value": round(B * args.steps / eg, 3), "ms_per_step": round(eg / args.steps * 1e3, 3)}
        del g

    # The adaptive schedule (decided during the run from the first block's
    # modulated input; one host read-back per step), timed like `value`.
    adaptive = None
    if args.adaptive_ell >= 0:
        def run_adaptive():
            x.copy_(x0)
            return dm.sample_adaptive(x, cfg.steps, args.adaptive_ell, labels=tl, text=tt)
        for _ in range(max(1, args.warmup)):
            run_adaptive()
        torch.cuda.synchronize()
        ta = time.perf_counter()
        for _ in range(args.steps):
            _, amask, _ = run_adaptive()
        torch.cuda.synchronize()
        ea = time.perf_counter() - ta
        # The fixed-mask loop under the realised mask: the probe's and the
        # read-backs' cost is the difference.
        run(amask)
        torch.cuda.synchronize()
        tfm = time.perf_counter()
        for _ in range(args.steps):
            run(amask)
        torch.cuda.synchronize()
        efm = time.perf_counter() - tfm
        adaptive = {"ell": args.adaptive_ell, "full_steps": int(amask.sum()),
                    "value": round(B * args.steps / ea, 3), "ms_per_step": round(ea / args.steps * 1e3, 3),
                    "ms_fixed_loop_same_mask": round(efm / args.steps * 1e3, 3),
                    "mask": "".join(str(int(v)) for v in amask)}

    # Blockwise mode (Br = 0) under the same mask: every module's output is
    # cached, so the cache is 2 (DiT) or 3 (PixArt) tensors per block instead
    # of one per run; timed like `value`.
    blockwise = None
    if not args.no_blockwise and cfg.kind in ("dit", "pixart"):
        def run_blockwise():
            x.copy_(x0)
            return dm.sample_blockwise(x, mask, labels=tl, text=tt)
        for _ in range(max(1, args.warmup)):
            sites = run_blockwise()
        torch.cuda.synchronize()
        tb = time.perf_counter()
        for _ in range(args.steps):
            sites = run_blockwise()
        torch.cuda.synchronize()
        eb = time.perf_counter() - tb
        blockwise = {"value": round(B * args.steps / eb, 3), "ms_per_step": round(eb / args.steps * 1e3, 3),
                     "sites": int(sites.shape[0]), "cache_bytes": int(sites.numel() * sites.element_size()),
                     "stepwise_cache_bytes": int(cfg.K * B * cfg.tokens * cfg.hidden * sites.element_size())}
        del sites
        dm.release_blockwise()
        torch.cuda.empty_cache()

    # Speedup reference: the same sampler with every step full.
    full = np.ones(cfg.steps, np.uint8)
    run(full)
    torch.cuda.synchronize()
    tf = time.perf_counter()
    nref = max(1, min(3, args.steps))
    for _ in range(nref):
        run(full)
    torch.cuda.synchronize()
    ms_full = (time.perf_counter() - tf) / nref * 1e3

    forecast = None
    if not args.no_forecast:
        del dm
        torch.cuda.empty_cache()
        forecast = forecast_bench(bc, torch, dev, K=3, dtype="bf16")
        fc_hash = source_hash("forecast.hip", "hip_common.h")
        forecast["traffic"] = counters_traffic("forecast_k3_bf16", fc_hash, None)
        forecast["source_hash"] = fc_hash

    if args.calib_copy:
        # A plain copy of known size through the library's 16-byte copy kernel:
        # the reference for scaling HBM byte counters.
        n = 1 << 29
        src = torch.ones(n, dtype=torch.bfloat16, device=dev)
        store = torch.empty((1, n), dtype=torch.bfloat16, device=dev)
        ring = bc.CacheRing(1, store)
        ring.push(src, 0.0)
        torch.cuda.synchronize()
        del src, store, ring

    cpu = None
    if not args.no_cpu_baseline and host_weights:
        cpu = cpu_baseline(cfg, params, labels, xT, mask, args.cpu_steps)

    blocks = (f"{cfg.depth} dual-stream + {cfg.depth_single} single-stream blocks" if cfg.kind == "mmdit"
              else f"{cfg.depth} blocks")
    line = {
        "metric": "end-to-end samples/s at fixed skip schedule; forecast HBM GB/s; block MFMA util",
        "value": round(value, 3), "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {blocks}, D {cfg.hidden}, {cfg.heads}x{cfg.head_dim} heads, "
                               f"MLP {cfg.mlp}, {cfg.tokens} tokens, batch {B}, {cfg.steps} {cfg.sampler} steps, "
                               f"K={cfg.K}, full every {cfg.interval} ({nfull}/{cfg.steps}), random-init weights",
                   "global_batch": B, "parallelism": "none (1 GPU)"},
        "graph_replay": graph,
        "adaptive": adaptive,
        "blockwise": blockwise,
        "speedup_vs_all_full": round(ms_full / ms_per_step, 3),
        "ms_all_full": round(ms_full, 3),
        "roofline": roofline,
        "roofline_others": others,
        "kernel_classes": breakdown,
        "forecast": forecast,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()

"""Benchmark of the BaryCache hot path on one MI355X.

One step = one BaryCache sampling run of the whole batch through the full
schedule (every full step runs the block stack and its last block writes the
stepwise feature into the ring; every other step forecasts it from the ring
with Eq. 13; all steps run the final layer and the sampler update), with the
noise, the weights and the conditioning inputs already resident in HBM.

Headline workload (the largest single-GPU configuration): the HunyuanVideo-
shaped text-to-video model, 20 dual-stream + 40 single-stream blocks, hidden
3072, 24 heads of 128, MLP 12288, QK RMSNorm and 3D RoPE, 14 310 video tokens
(16 x 9 x 60 x 106 latent, patch 2) + 256 text tokens, batch 1, 50 Euler steps
with time shift 7, K = 3, a full step every 5 (11 of 50), bf16, random-init
weights from seed 2026.

The JSON line also carries, measured in the same process:
  * `roofline`: the dominant kernel of the headline run (the kernel and shape
    with the most time per run, from per-launch HIP events on its launch
    stream), its algorithmic FLOPs per launch over its average duration;
  * `kernel_classes`: every kernel class's time per run and its average rate;
  * `workloads`: the DiT-XL/2-shaped (batch 16, DDIM-50) and PixArt-shaped
    (batch 4, DPM-Solver++(2M)-20) workloads measured the same way with
    fewer runs, each with its own roofline;
  * `forecast`: the forecast kernel on [8, 16384, 3072] features for every
    K in {2, 3, 4, 5}, bf16 and fp32, and the ring push's copy path;
  * `cpu_baseline`: the oracle on the host cores, composed from timed pieces
    (see cpu_baseline_video).
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
PAPER_CONTEXT = ("The paper reports end-to-end speedups of up to 3.30x over 50-step DDIM (PixArt-Sigma 1024x1024, "
                 "batch 4, interval N = 6, on an RTX 5090, precision not stated; Table 1, Sec. 4.1); 2.18x on "
                 "DiT-XL/2 (N = 6, RTX 5090; Table 3) and 3.02x on HunyuanVideo (N = 7, A800; Table 2). "
                 "Context only: other hardware, trained weights, other schedules.")

CLASS_NAMES = ["forecast", "gemm_gelu", "gemm_gated", "gemm_bias", "attention", "layernorm", "gemm_down", "copy"]
MFMA_CLASSES = {"gemm_gelu", "gemm_gated", "gemm_bias", "attention", "gemm_down"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="hunyuan", help="headline workload (hunyuan, pixart, dit_xl2, tiny)")
    ap.add_argument("--legs", default="dit_xl2,pixart",
                    help="other workloads measured in the same line (comma list; empty: none)")
    ap.add_argument("--leg-steps", type=int, default=3, help="timed runs of each other workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-forecast", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the graph-replay, adaptive and blockwise runs of the DiT-XL/2 leg")
    ap.add_argument("--adaptive-ell", type=float, default=0.13, help="threshold of the adaptive-schedule run")
    ap.add_argument("--kernels-only", action="store_true",
                    help="launch only the roofline kernels at the workloads' shapes, for hardware-counter passes")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one 1 GiB device copy through the library (counter calibration)")
    ap.add_argument("--launch-log", default=None, help="--kernels-only: write the tag of every launch here")
    ap.add_argument("--summarize-trace", default=None,
                    help="STATS_CSV,LINE_JSON: write profiles/bench_kernel_trace.md from a kernel-trace run")
    ap.add_argument("--loop-counters", action="store_true",
                    help="run the workload's sampling loop --steps times and the 1 GiB calibration copy, nothing "
                         "else (the program of the whole-loop rocprofv3 --pmc passes)")
    ap.add_argument("--summarize-loop-counters", default=None,
                    help="write profiles/sampling_loop_<workload>_counters.md from the --pmc passes in this directory")
    ap.add_argument("--summarize-counters", default=None,
                    help="write profiles/<tag>_counters.json from the rocprofv3 --pmc passes in this directory")
    return ap.parse_args()


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2608_28670_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {"attention": ("attention.hip", "attention.h", "hip_common.h"),
                  "gemm": ("gemm.hip", "gemm.h", "hip_common.h"),
                  "forecast": ("forecast.hip", "hip_common.h")}


def counters_traffic(tag, src_hash):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated) from the
    committed rocprofv3 counter summary of this kernel and shape, or None if
    there is none for the current kernel source."""
    path = os.path.join(ROOT, "profiles", f"{tag}_counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        c = json.load(f)
    if c.get("source_hash") != src_hash:
        return None
    return c.get("hbm_bytes_per_launch")


def ensure_library():
    import paper_2608_28670_amd as bc
    if not bc.is_current():
        from paper_2608_28670_amd import build
        print("libbarycache.so is missing or stale; rebuilding", file=sys.stderr)
        build.build()
    return bc


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# kernel shapes of a workload (to name the launches the profiler records)
# ---------------------------------------------------------------------------

def kernel_shapes(cfg):
    """(class, name, shape, work) of every block kernel of one full step and
    of the conditioning GEMMs that run once per run or per chunk of full
    steps; work = algorithmic FLOPs per launch, which with the class
    identifies a launch."""
    B, D, F, T = cfg.batch, cfg.hidden, cfg.mlp, cfg.tokens
    H, hd = cfg.heads, cfg.head_dim
    out = []

    def gemm(cls, name, M, N, K):
        out.append((cls, name, [M, N, K], 2.0 * M * N * K))

    def att(name, Tq, Tk):
        out.append(("attention", name, [B, H, Tq, Tk, hd], 4.0 * B * H * Tq * Tk * hd))

    if cfg.kind in ("dit", "pixart"):
        M = B * T
        if cfg.dtype == "bf16" and T <= 256 and hd in (32, 64, 72) and D % 64 == 0:
            # one kernel per (sample, head): the QKV projection into LDS, then the attention
            out.append(("attention", "QKV projection + self-attention (one kernel per sample and head)",
                        [B, H, T, T, hd], 2.0 * M * 3 * D * D + 4.0 * B * H * T * T * hd))
        else:
            gemm("gemm_bias", "QKV projection", M, 3 * D, D)
            att("self-attention", T, T)
        if cfg.kind == "pixart":
            # The cross-attention's output projection is a residual GEMM of the
            # same shape as the attention output projection: one group.
            gemm("gemm_gated", "attention and cross-attention output projections + residual", M, D, D)
            gemm("gemm_bias", "cross-attention query projection", M, D, D)
            att("cross-attention", T, cfg.ctx_tokens)
        else:
            gemm("gemm_gated", "attention output projection + gated residual", M, D, D)
        gemm("gemm_gelu", "MLP up projection + GELU", M, F, D)
        gemm("gemm_down", "MLP down projection + gated residual", M, D, F)
    else:
        Tt = cfg.txt_tokens
        L = T + Tt
        for s, M in (("image", B * T), ("text", B * Tt)):
            gemm("gemm_bias", f"dual-stream {s} QKV projection", M, 3 * D, D)
        # The other dual-stream GEMMs run the image and text streams in one
        # launch (the text tiles fill the image grid's last round): one group
        # with the work of B (T + Tt) rows.
        gemm("gemm_gated", "dual-stream output projection + gated residual (image and text)", B * L, D, D)
        gemm("gemm_gelu", "dual-stream MLP up projection + GELU (image and text)", B * L, F, D)
        gemm("gemm_down", "dual-stream MLP down projection + gated residual (image and text)", B * L, D, F)
        gemm("gemm_gelu", "single-stream [qkv | mlp] projection + GELU", B * L, 3 * D + F, D)
        gemm("gemm_down", "single-stream output projection + gated residual", B * L, D, D + F)
        att("joint attention (dual- and single-stream)", L, L)
    # Once per run (or per chunk of full steps): the conditioning GEMMs.
    S = cfg.steps
    nf = sum(1 for k in range(S) if k % cfg.interval == 0 or k == S - 1)
    chunk = max(1, min(S, 256 // B, 64))
    for f0 in range(0, nf, chunk):
        Mc = min(chunk, nf - f0) * B
        if cfg.kind == "dit":
            gemm("gemm_bias", "adaLN modulation of a chunk of full steps (all blocks, one grouped launch)",
                 Mc, cfg.depth * 6 * D, D)
        elif cfg.kind == "pixart":
            gemm("gemm_bias", "t6 projection of a chunk of full steps", Mc, 6 * D, D)
        else:
            gemm("gemm_bias", "dual-stream adaLN modulation of a chunk of full steps (grouped)",
                 Mc, 2 * cfg.depth * 6 * D, D)
            gemm("gemm_bias", "single-stream adaLN modulation of a chunk of full steps (grouped)",
                 Mc, cfg.depth_single * 3 * D, D)
    if cfg.kind != "pixart":
        gemm("gemm_bias", "final-layer modulation of every step", S * B, 2 * D, D)
    return out


def group_launches(records, cfg):
    """Per (class, work) group: launches, time; named from kernel_shapes."""
    import numpy as np
    names = {(c, w): (n, s) for c, n, s, w in kernel_shapes(cfg)}
    groups = []
    for cls, (ms, work) in records.items():
        if not len(ms):
            continue
        for wv in np.unique(work[work > 0]):
            sel = work == wv
            t = ms[sel].astype(np.float64)
            nm = names.get((cls, float(wv)))
            groups.append({"class": cls, "kernel": nm[0] if nm else None, "shape": nm[1] if nm else None,
                           "work": float(wv), "launches": int(sel.sum()), "ms_per_run": float(t.sum()),
                           "avg_us": float(t.mean()) * 1e3})
    groups.sort(key=lambda g: -g["ms_per_run"])
    return groups


# kernel-name prefix of a profiled class's launches (the gated epilogue is template argument 2)
CLASS_KERNEL = {"attention": ("void bc::attention_dma_kernel<",),
                "gemm_gated": ("void bc::gemm_wide_kernel<2,", "void bc::gemm_wide_pair_kernel<2,"),
                "gemm_down": ("void bc::gemm_wide_kernel<2,", "void bc::gemm_wide_pair_kernel<2,"),
                "gemm_gelu": ("void bc::gemm_wide_kernel<0,", "void bc::gemm_wide_pair_kernel<0,"),
                "gemm_bias": ("void bc::gemm_wide_kernel<0,", "void bc::gemm_wide_pair_kernel<0,")}


def loop_traffic(workload, g, src):
    """HBM bytes per launch of a kernel group from the whole-loop counter
    summary of this workload: the one (kernel, grid) group of the class's
    kernel with as many dispatches per run as the group has launches, if the
    kernel source is unchanged since the counters were taken; else None."""
    path = os.path.join(ROOT, "profiles", f"sampling_loop_{workload}_counters.json")
    if not os.path.exists(path) or g["class"] not in CLASS_KERNEL:
        return None
    with open(path) as f:
        c = json.load(f)
    if c.get("source_hashes", {}).get(src) != source_hash(*KERNEL_SOURCES[src]):
        return None
    hits = [r for r in c["groups"] if r["kernel"].startswith(CLASS_KERNEL[g["class"]])
            and abs(r["dispatches_per_run"] - g["launches"]) < 0.5 and "hbm_bytes" in r
            and grid_fits(r["kernel"], r["grid_threads"], g)]
    return hits[0]["hbm_bytes"] if len(hits) == 1 else None


def grid_fits(kernel, grid_threads, g):
    """Whether a dispatch grid is the one the kernel's template arguments give
    for the group's shape (GEMM [M, N, K]: one workgroup per BM x BN tile;
    attention [B, H, Tq, Tk, d]: one per 16 QG NWV queries of a head)."""
    import re
    m = re.search(r"<([^>]*)>", kernel)
    if not m or not g.get("shape"):
        return False
    args = [a.strip() for a in m.group(1).split(",")]
    if "attention" in kernel:
        qg, nwv = int(args[1]), int(args[2])
        B, H, Tq, Tk = g["shape"][0], g["shape"][1], g["shape"][2], g["shape"][3]
        qt = 16 * qg * nwv
        # the streaming key loop (template argument 4) serves more than 256 keys
        # (PixArt's self- and cross-attention share B, H and Tq)
        if (args[4] == "true") != (Tk > 256):
            return False
        return grid_threads == -(-Tq // qt) * H * B * 64 * nwv
    bm, bn, wm, wn, kg = int(args[1]), int(args[2]), int(args[3]), int(args[4]), int(args[7])
    M, N = g["shape"][0], g["shape"][1]
    return grid_threads == -(-M // bm) * -(-N // bn) * 64 * wm * wn * kg


def roofline_of(g, tag=None, src=None, workload=None):
    """Roofline record of a kernel group; traffic from the whole-loop counter
    summary, else from the counter program's summary."""
    avg_s = g["avg_us"] / 1e6
    achieved = g["work"] / avg_s / 1e12
    r = {"bound": "mfma", "kernel": g["kernel"], "class": g["class"], "shape": g["shape"],
         "flops_per_launch": g["work"], "avg_us": round(g["avg_us"], 2), "launches": g["launches"],
         "ms_per_run": round(g["ms_per_run"], 3), "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
         "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4)}
    r["traffic"] = None
    if src is None:
        src = "attention" if g["class"] == "attention" else "gemm" if g["class"].startswith("gemm") else None
    if src is not None:
        h = source_hash(*KERNEL_SOURCES[src])
        r["source_hash"] = h
        lt = loop_traffic(workload, g, src) if workload else None
        if lt is not None:
            r["traffic"], r["traffic_from"] = lt, "sampling loop (profiles/sampling_loop_%s_counters.json)" % workload
        elif tag is not None:
            ct = counters_traffic(tag, h)
            if ct is not None:
                r["traffic"], r["traffic_from"] = ct, "counter program (profiles/%s_counters.json)" % tag
    return r


def counter_tag(cfg, g):
    """The counter-summary tag of a profiled kernel group (matched by its
    class and algorithmic FLOPs among the counter program's kernels: DiT-XL/2's
    MLP up and down projections have the same FLOPs), or None."""
    for k in kernel_tags(cfg):
        if k["class"] == g["class"] and abs(k["flops"] - g["work"]) <= 1e-9 * g["work"]:
            return k["tag"], k["tag"].split("_")[0]
    return None, None


# ---------------------------------------------------------------------------
# one workload
# ---------------------------------------------------------------------------

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


def measure(bc, torch, cfg, steps, warmup, extras=False, adaptive_ell=0.13):
    """Time `steps` sampling runs after `warmup` runs; one more run with every
    kernel class timed per launch; the all-full mask at the same S."""
    import numpy as np

    import synth
    from paper_2608_28670_amd import loader
    dev = "cuda:0"
    t0 = time.time()
    dm = loader.DeviceModel(cfg, None, dev_params=device_params(cfg, torch, dev))
    B = cfg.batch
    mask = bc.make_mask(cfg.steps, cfg.interval)
    labels = synth.labels(cfg) if cfg.n_classes else None
    text = synth.text(cfg) if cfg.kind != "dit" else None
    x0 = torch.from_numpy(synth.latents(cfg)).to(dev)
    x = torch.empty_like(x0)
    tl = torch.from_numpy(labels).to(dev) if labels is not None else None
    tt = torch.from_numpy(text).to(dev).to(loader.torch_dtype(cfg)) if text is not None else None
    torch.cuda.synchronize()
    log(f"[{cfg.name}] setup {time.time() - t0:.1f} s")

    def run(m):
        x.copy_(x0)
        dm.sample(x, m, labels=tl, text=tt)

    for _ in range(warmup):
        run(mask)
    torch.cuda.synchronize()
    log(f"[{cfg.name}] {warmup} warm-up runs done; timing {steps}")
    t_start = time.perf_counter()
    for _ in range(steps):
        run(mask)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    res = {"value": B * steps / elapsed, "ms_per_step": elapsed / steps * 1e3, "mask": mask}
    log(f"[{cfg.name}] {res['value']:.4g} samples/s, {res['ms_per_step']:.1f} ms per run")

    # Per-launch HIP events on the launch stream, in one more run.
    cap = 1 << 16
    for c in range(len(CLASS_NAMES)):
        bc.profile_enable(c, cap)
    run(mask)
    records = {}
    for c, name in enumerate(CLASS_NAMES):
        ms, work = bc.profile_records(c, cap)
        records[name] = (ms, work)
    classes = {}
    for name, (ms, work) in records.items():
        if not len(ms):
            continue
        t = ms.astype(np.float64)
        e = {"ms_per_run": round(float(t.sum()), 3), "launches": int(len(t)), "avg_us": round(float(t.mean()) * 1e3, 2)}
        if name in MFMA_CLASSES and work.sum() > 0:
            e["tflops"] = round(float(work.sum()) / (t.sum() / 1e3) / 1e12, 1)
            e["frac_of_mfma_peak"] = round(e["tflops"] / PEAK_BF16_TFLOPS, 4)
        elif work.sum() > 0:
            e["gbs"] = round(float(work.sum()) / (t.sum() / 1e3) / 1e9, 1)
            e["frac_of_hbm_peak"] = round(e["gbs"] / PEAK_HBM_GBS, 4)
        classes[name] = e
    groups = [g for g in group_launches(records, cfg) if g["class"] in MFMA_CLASSES]
    res["roofline"] = roofline_of(groups[0], *counter_tag(cfg, groups[0]), workload=cfg.name)
    res["roofline_others"] = [roofline_of(g, *counter_tag(cfg, g), workload=cfg.name) for g in groups[1:6]]
    res["kernel_classes"] = classes
    res["profiled_run_ms"] = round(float(sum(float(ms.sum()) for ms, _ in records.values())), 3)

    if extras:
        res.update(extra_runs(bc, torch, cfg, dm, run, mask, x, x0, tl, tt, steps, adaptive_ell))

    # Speedup reference: every step full, same sampler (kernels already warm).
    full = np.ones(cfg.steps, np.uint8)
    nref = 1 if res["ms_per_step"] > 1000 else 2
    if nref > 1:
        run(full)
    torch.cuda.synchronize()
    tf = time.perf_counter()
    for _ in range(nref):
        run(full)
    torch.cuda.synchronize()
    ms_full = (time.perf_counter() - tf) / nref * 1e3
    res["ms_all_full"] = ms_full
    res["speedup_vs_all_full"] = ms_full / res["ms_per_step"]
    res["ideal_speedup"] = cfg.steps / int(mask.sum())
    log(f"[{cfg.name}] all-full mask {ms_full:.1f} ms per run: speedup {res['speedup_vs_all_full']:.3f}")
    del dm, x, x0, tl, tt
    torch.cuda.empty_cache()
    return res


def extra_runs(bc, torch, cfg, dm, run, mask, x, x0, tl, tt, steps, ell):
    """HIP-graph replay, the adaptive schedule and blockwise mode on the same
    workload, each timed like `value`."""
    B = cfg.batch
    out = {}
    g = dm.sample_graph(x, mask, labels=tl, text=tt)
    x.copy_(x0)
    g.launch()
    torch.cuda.synchronize()
    tg = time.perf_counter()
    for _ in range(steps):
        x.copy_(x0)
        g.launch()
    torch.cuda.synchronize()
    eg = time.perf_counter() - tg
    out["graph_replay"] = {"value": round(B * steps / eg, 3), "ms_per_step": round(eg / steps * 1e3, 3)}
    del g

    def run_adaptive():
        x.copy_(x0)
        return dm.sample_adaptive(x, cfg.steps, ell, labels=tl, text=tt)
    run_adaptive()
    torch.cuda.synchronize()
    ta = time.perf_counter()
    for _ in range(steps):
        _, amask, _ = run_adaptive()
    torch.cuda.synchronize()
    ea = time.perf_counter() - ta
    run(amask)
    torch.cuda.synchronize()
    tfm = time.perf_counter()
    for _ in range(steps):
        run(amask)
    torch.cuda.synchronize()
    efm = time.perf_counter() - tfm
    out["adaptive"] = {"ell": ell, "full_steps": int(amask.sum()), "value": round(B * steps / ea, 3),
                       "ms_per_step": round(ea / steps * 1e3, 3),
                       "ms_fixed_loop_same_mask": round(efm / steps * 1e3, 3),
                       "mask": "".join(str(int(v)) for v in amask)}

    if cfg.kind in ("dit", "pixart"):
        def run_blockwise():
            x.copy_(x0)
            return dm.sample_blockwise(x, mask, labels=tl, text=tt)
        sites = run_blockwise()
        torch.cuda.synchronize()
        tb = time.perf_counter()
        for _ in range(steps):
            sites = run_blockwise()
        torch.cuda.synchronize()
        eb = time.perf_counter() - tb
        out["blockwise"] = {"value": round(B * steps / eb, 3), "ms_per_step": round(eb / steps * 1e3, 3),
                            "sites": int(sites.shape[0]), "cache_bytes": int(sites.numel() * sites.element_size()),
                            "stepwise_cache_bytes": int(cfg.K * B * cfg.tokens * cfg.hidden * sites.element_size())}
        del sites
        dm.release_blockwise()
        torch.cuda.empty_cache()
    return out


def workload_desc(cfg, mask):
    nfull = int(mask.sum())
    blocks = (f"{cfg.depth} dual-stream + {cfg.depth_single} single-stream blocks" if cfg.kind == "mmdit"
              else f"{cfg.depth} blocks")
    extra = ""
    if cfg.kind == "mmdit":
        extra = f" + {cfg.txt_tokens} text tokens, QK RMSNorm + 3D RoPE, time shift {cfg.flow_shift:g}"
    elif cfg.kind == "pixart":
        extra = f", cross-attention to {cfg.ctx_tokens} text tokens of width {cfg.ctx_dim}"
    return (f"{cfg.name}: {blocks}, D {cfg.hidden}, {cfg.heads}x{cfg.head_dim} heads, MLP {cfg.mlp}, "
            f"{cfg.tokens} tokens{extra}, batch {cfg.batch}, {cfg.steps} {cfg.sampler} steps, K={cfg.K}, "
            f"full every {cfg.interval} ({nfull}/{cfg.steps}), random-init weights")


# ---------------------------------------------------------------------------
# forecast microbenchmark and the push copy
# ---------------------------------------------------------------------------

def forecast_sweep(bc, torch, iters=5):
    """Forecast kernel HBM bandwidth on K cached [8, 16384, 3072] features for
    K in 2..5, bf16 and fp32 (algorithmic bytes (K + 1) n s per launch), and
    the ring push's copy path on one bf16 feature (2 n s bytes)."""
    import synth
    dev = "cuda:0"
    shape = synth.FORECAST_SHAPE
    n = shape[0] * shape[1] * shape[2]
    out = []
    fc_hash = source_hash(*KERNEL_SOURCES["forecast"])
    for dt in ("bf16", "f32"):
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        esz = 2 if dt == "bf16" else 4
        g = torch.Generator(device=dev)
        g.manual_seed(synth.SEED)
        storage = torch.empty((5, n), dtype=tdt, device=dev)
        for j in range(5):
            storage[j].normal_(generator=g)
        res = torch.empty(n, dtype=tdt, device=dev)
        for K in (2, 3, 4, 5):
            ring = bc.CacheRing(K, storage[:K])
            s, t = synth.forecast_times(K)
            for j in reversed(range(K)):
                ring.push(None, float(s[j]))
            w = bc.bary_weights(s, t)
            bc.bary_extrapolate(ring, w, res)
            torch.cuda.synchronize()
            bc.profile_enable(bc.PROF_FORECAST, iters)
            for _ in range(iters):
                bc.bary_extrapolate(ring, w, res)
            ms, work = bc.profile_records(bc.PROF_FORECAST, iters)
            avg_s = float(ms.mean()) / 1e3
            bytes_alg = (K + 1) * n * esz
            assert abs(work[0] - bytes_alg) < 1
            gbs = bytes_alg / avg_s / 1e9
            out.append({"K": K, "dtype": dt, "shape": list(shape), "bytes_per_launch": bytes_alg,
                        "avg_us": round(avg_s * 1e6, 2), "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                        "traffic": counters_traffic(f"forecast_k{K}_{dt}", fc_hash)})
            del ring
        del storage, res
        torch.cuda.empty_cache()
    # the push's copy path: one bf16 feature into the next ring slot
    src = torch.empty(n, dtype=torch.bfloat16, device=dev).normal_()
    store = torch.empty((3, n), dtype=torch.bfloat16, device=dev)
    ring = bc.CacheRing(3, store)
    ring.push(src, 0.0)
    torch.cuda.synchronize()
    bc.profile_enable(bc.PROF_COPY, iters)
    for i in range(iters):
        ring.push(src, float(i + 1))
    ms, work = bc.profile_records(bc.PROF_COPY, iters)
    avg_s = float(ms.mean()) / 1e3
    gbs = 2 * n * 2 / avg_s / 1e9
    push = {"shape": list(shape), "dtype": "bf16", "bytes_per_launch": 2 * n * 2, "avg_us": round(avg_s * 1e6, 2),
            "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
            "note": "copy path of bc_cache_push; the sampling loop itself pushes with no copy (the last block's "
                    "epilogue writes the ring slot)"}
    del src, store, ring
    torch.cuda.empty_cache()
    return out, push


# ---------------------------------------------------------------------------
# the oracle on the host cores
# ---------------------------------------------------------------------------

def host_info():
    import numpy as np
    cpu = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = "unknown"
    try:
        cfgs = np.show_config(mode="dicts")
        b = cfgs.get("Build Dependencies", {}).get("blas", {})
        blas = f"{b.get('name', '?')} {b.get('version', '')}".strip()
    except Exception:   # older numpy: no dict mode
        pass
    try:
        from threadpoolctl import threadpool_info
        pools = [f"{p.get('internal_api')} {p.get('version')} ({p.get('num_threads')} threads)"
                 for p in threadpool_info() if p.get("user_api") == "blas"]
        if pools:
            blas = "; ".join(pools)
    except Exception:
        pass
    return cpu, blas


def cpu_baseline_video(cfg):
    """The oracle (numpy, fp32 model as the video workload's tests run it)
    timed in pieces on one sample at the full shape and composed to a whole
    sampling run: one dual-stream block and one single-stream block on all
    14 566 tokens, one forecast step (Eq. 13 over K = 3 features) and one final
    layer + Euler update; a run is 11 x (20 dual + 40 single blocks) + 39
    forecasts + 50 final layers and updates (the embedding and conditioning
    are left out: they take well under 1 % of a block)."""
    import numpy as np

    import synth
    from oracle import bary, model as om, sampler as osm
    one = synth.scaled(cfg, depth=1, depth_single=1, batch=1)
    names = [n for n, _ in synth.param_shapes(one)
             if n.startswith(("dual.0.", "single.0.", "final_", "txt_", "t_"))]
    P = synth.params(one, names=names)
    M = om.Model(one, P, dtype=np.float32)
    D, T, Tt = cfg.hidden, cfg.tokens, cfg.txt_tokens
    x = synth.normal("cpu/x", (1, T, D))
    xt = synth.normal("cpu/xt", (1, Tt, D))
    c = {"c": synth.normal("cpu/c", (1, D), 0.5)}
    t0 = time.perf_counter()
    M.dual_block(0, x, xt, c)
    t_dual = time.perf_counter() - t0
    log(f"[cpu] oracle dual-stream block {t_dual:.1f} s")
    t0 = time.perf_counter()
    M.single_block(0, np.concatenate([x, xt], axis=1), c, T)
    t_single = time.perf_counter() - t0
    log(f"[cpu] oracle single-stream block {t_single:.1f} s")
    ring = [synth.normal(f"cpu/ring{j}", (1, T, D)) for j in range(3)]
    w = bary.bary_weights([10.0, 5.0, 0.0], 12.0)
    t0 = time.perf_counter()
    feat = bary.forecast(ring, w)
    t_fc = time.perf_counter() - t0
    smp = osm.Sampler("euler", cfg.steps, cfg.in_ch, cfg.flow_shift)
    lat = synth.latents(one).astype(np.float64)
    t0 = time.perf_counter()
    out = M.final(feat, c)
    smp.step(1, lat, out)
    t_fin = time.perf_counter() - t0
    mask = bary.make_mask(cfg.steps, cfg.interval)
    nfull = int(mask.sum())
    per = nfull * (cfg.depth * t_dual + cfg.depth_single * t_single) + (cfg.steps - nfull) * t_fc + cfg.steps * t_fin
    cores = len(os.sched_getaffinity(0))
    cpu, blas = host_info()
    return {"value": round(cfg.batch / per, 8), "unit": "samples/s", "cores": cores, "kind": "oracle",
            "composed": True, "cpu_model": cpu, "blas": blas,
            "seconds_per_sample": round(per, 1),
            "sample": (f"oracle pieces timed once each on one sample at the full shape (numpy fp32 model, "
                       f"{cores} host threads): dual-stream block {t_dual:.2f} s, single-stream block "
                       f"{t_single:.2f} s (14310 + 256 tokens, D 3072), forecast K=3 {t_fc * 1e3:.0f} ms, final "
                       f"layer + Euler update {t_fin * 1e3:.0f} ms; composed to {nfull} full steps x "
                       f"({cfg.depth} dual + {cfg.depth_single} single blocks) + {cfg.steps - nfull} forecasts + "
                       f"{cfg.steps} final layers")}


def cpu_baseline_image(cfg, nsteps=9):
    """The oracle (numpy fp64) on one sample of an image workload for the
    first `nsteps` steps of its schedule; per-step times composed to the whole
    schedule."""
    import numpy as np

    import synth
    from oracle import bary, model as om, sampler as osm
    one = synth.scaled(cfg, batch=1)
    params = synth.params(one)
    M = om.Model(one, params)
    x = synth.latents(one).astype(np.float64)
    lab = synth.labels(one) if one.n_classes else None
    text = synth.text(one) if one.kind != "dit" else None
    mask = bary.make_mask(cfg.steps, cfg.interval)
    steps = bary.plan(mask, cfg.K)
    tin = osm.model_time(cfg.sampler, cfg.steps, cfg.flow_shift)
    smp = osm.Sampler(cfg.sampler, cfg.steps, cfg.in_ch, cfg.flow_shift)
    ring = bary.Ring(cfg.K)
    ctx = M.context(text) if one.kind != "dit" else None
    t_full, t_fc = [], []
    for k in range(min(nsteps, cfg.steps)):
        t0 = time.perf_counter()
        cond = M.condition(tin[k], 1, lab, text)
        if mask[k]:
            feat = M.stack(M.embed(x), cond, ctx)
            ring.push(feat, k)
        else:
            st = steps[k]
            feat = bary.forecast([ring.slots[i] for i in st.slots], st.w)
        x = smp.step(k, x, M.final(feat, cond))
        (t_full if mask[k] else t_fc).append(time.perf_counter() - t0)
    nfull = int(mask.sum())
    per = nfull * np.mean(t_full) + (cfg.steps - nfull) * np.mean(t_fc)
    cores = len(os.sched_getaffinity(0))
    return {"value": round(1.0 / per, 6), "unit": "samples/s", "cores": cores, "kind": "oracle", "composed": True,
            "sample": (f"1 sample, steps 0-{nsteps - 1} of the {cfg.steps}-step schedule ({len(t_full)} full at "
                       f"{np.mean(t_full):.2f} s, {len(t_fc)} forecast at {np.mean(t_fc) * 1e3:.1f} ms), composed "
                       f"to {nfull} full + {cfg.steps - nfull} forecast steps; numpy fp64 on {cores} host threads")}


def cpu_baseline_tiny(cfg):
    """The oracle (numpy fp64) running the tiny fp32 workload end to end: the
    whole batch through the whole schedule (full steps and forecasts)."""
    import numpy as np

    import synth
    from oracle import bary, model as om, sampler as osm
    M = om.Model(cfg, synth.params(cfg))
    mask = bary.make_mask(cfg.steps, cfg.interval)
    x = synth.latents(cfg).astype(np.float64)
    t0 = time.perf_counter()
    osm.sample(M, x, mask, cfg.K)
    dt = time.perf_counter() - t0
    return {"value": round(cfg.batch / dt, 3), "unit": "samples/s", "kind": "oracle", "composed": False,
            "sample": f"the whole batch of {cfg.batch} through all {cfg.steps} steps ({int(mask.sum())} full), "
                      f"numpy fp64: {dt:.2f} s"}


def cpu_baseline_blocks(cfg):
    """The oracle (numpy fp32 model) on one sample of an image workload, timed
    in pieces at the full shape (one block, with PixArt's cross-attention; one
    forecast step over K features; one final layer + sampler update) and
    composed to a run: #full x depth blocks + #skipped forecasts + every
    step's final layer (the per-run caption context and the embeddings are
    left out)."""
    import numpy as np

    import synth
    from oracle import bary, model as om, sampler as osm
    one = synth.scaled(cfg, depth=1, batch=1)
    M = om.Model(one, synth.params(one), dtype=np.float32)
    D, T = cfg.hidden, cfg.tokens
    x = synth.normal("cpu/bx", (1, T, D))
    c = synth.normal("cpu/bc", (1, D), 0.5)
    if cfg.kind == "pixart":
        t6 = synth.normal("cpu/bt6", (1, 6 * D), 0.5)
        bcond, fcond, ctx = {"t6": t6}, {"t": c, "t6": t6}, M.context(synth.text(one))
    else:
        bcond = fcond = {"c": c}
        ctx = None
    t0 = time.perf_counter()
    M.dit_block(0, x, M.block_mod(0, bcond), ctx)
    t_blk = time.perf_counter() - t0
    ring = [synth.normal(f"cpu/bring{j}", (1, T, D)) for j in range(cfg.K)]
    w = bary.bary_weights([float(10 - 2 * j) for j in range(cfg.K)], 12.0)
    t0 = time.perf_counter()
    feat = bary.forecast(ring, w)
    t_fc = time.perf_counter() - t0
    smp = osm.Sampler(cfg.sampler, cfg.steps, cfg.in_ch, cfg.flow_shift)
    lat = synth.latents(one).astype(np.float64)
    t0 = time.perf_counter()
    smp.step(0, lat, M.final(feat, fcond))
    t_fin = time.perf_counter() - t0
    mask = bary.make_mask(cfg.steps, cfg.interval)
    nfull = int(mask.sum())
    per = nfull * cfg.depth * t_blk + (cfg.steps - nfull) * t_fc + cfg.steps * t_fin
    what = "block with cross-attention" if cfg.kind == "pixart" else "block"
    return {"value": round(1.0 / per, 6), "unit": "samples/s", "kind": "oracle", "composed": True,
            "sample": (f"oracle pieces on one sample at the full shape (numpy fp32 model): {what} "
                       f"{t_blk:.2f} s ({T} tokens, D {D}), forecast K={cfg.K} {t_fc * 1e3:.0f} ms, final layer + "
                       f"update {t_fin * 1e3:.0f} ms; composed to {nfull} full steps x {cfg.depth} blocks + "
                       f"{cfg.steps - nfull} forecasts + {cfg.steps} final layers")}


def cpu_baseline_forecast():
    """The oracle's Eq. 13 (fp64 accumulation) on fp32 K = 3 features of the
    forecast microbenchmark shape, timed on a 1/64 slice of it and scaled to
    the whole [8, 16384, 3072] tensor."""
    import synth
    from oracle import bary
    K, shape = 3, synth.FORECAST_SHAPE
    rows = 2048                       # of the 8 x 16384 rows: 1/64 of the tensor
    feats = synth.forecast_features(K, (1, rows, shape[2]))
    s, t = synth.forecast_times(K)
    w = bary.bary_weights(s, t)
    t0 = time.perf_counter()
    bary.forecast([feats[j] for j in range(K)], w)
    scale = shape[0] * shape[1] // rows
    dt = (time.perf_counter() - t0) * scale
    n = shape[0] * shape[1] * shape[2]
    return {"value": round((K * 4 + 4) * n / dt / 1e9, 2), "unit": "GB/s", "kind": "oracle", "composed": True,
            "sample": f"K = 3 fp32 features [1, {rows}, {shape[2]}] (1/{scale} of [8, 16384, 3072]), scaled "
                      f"x{scale}: {dt:.2f} s for the whole tensor"}


# ---------------------------------------------------------------------------
# counter program
# ---------------------------------------------------------------------------

def kernel_tags(cfg):
    """Counter tags, shapes and algorithmic bytes / FLOPs of the kernels the
    counter program launches for a workload (in launch order per block)."""
    B, T, D, F, H, hd = cfg.batch, cfg.tokens, cfg.hidden, cfg.mlp, cfg.heads, cfg.head_dim
    bf = 2
    def gemm(tag, cls, M, N, K, gated):
        # A and W read once, output written once (+ the fp32 residual read for
        # the gated epilogue: res read and out written as fp32)
        byt = (M * K + N * K) * bf + (M * N * 8 if gated else M * N * bf)
        return {"tag": f"gemm_{tag}_{cfg.name}", "class": cls, "shape": [M, N, K], "flops": 2.0 * M * N * K,
                "bytes": byt}
    def att(L):
        return {"tag": f"attention_{cfg.name}", "class": "attention", "shape": [B, H, L, hd],
                "flops": 4.0 * B * H * L * L * hd, "bytes": 4 * B * L * H * hd * bf}
    if cfg.kind == "mmdit":
        L = T + cfg.txt_tokens
        return [gemm("single_in", "gemm_gelu", B * L, 3 * D + F, D, False), att(L),
                gemm("single_out", "gemm_down", B * L, D, D + F, True)]
    M = B * T
    return [gemm("qkv", "gemm_bias", M, 3 * D, D, False), att(T), gemm("proj", "gemm_gated", M, D, D, True),
            gemm("fc1", "gemm_gelu", M, F, D, False), gemm("fc2", "gemm_down", M, D, F, True)]


def kernels_only(args):
    """The roofline kernels at the workloads' shapes, launched through the C
    ABI without the sampling loop: the program the rocprofv3 counter passes
    run on.  Per workload, `steps` rounds over as many distinct weight sets as
    the model has blocks (so weights arrive from HBM, as in the loop): for
    DiT-XL/2 the QKV, out-projection, MLP up and down projections and
    self-attention; for the video model the single-stream block's projections
    and the joint attention over 14 566 tokens.  Then the K = 3 bf16 forecast
    and, with --calib-copy, one 1 GiB copy of known size.  With --launch-log
    the tag of every library launch is written there, in launch order."""
    import torch

    import synth
    bc = ensure_library()
    dev = "cuda:0"
    g = torch.Generator(device=dev)
    g.manual_seed(synth.SEED)
    log_tags = []

    def rnd(*shape, dt=torch.bfloat16, scale=0.02):
        t = torch.empty(shape, dtype=torch.float32, device=dev)
        t.normal_(0.0, scale, generator=g)
        return t.to(dt)

    for name in args.workload.split(","):
        cfg = synth.CONFIGS[name]
        tags = [k["tag"] for k in kernel_tags(cfg)]
        B, T, D, F, H, hd = cfg.batch, cfg.tokens, cfg.hidden, cfg.mlp, cfg.heads, cfg.head_dim
        if cfg.kind == "mmdit":
            L = T + cfg.txt_tokens
            nb = 4
            w1 = [rnd(3 * D + F, D) for _ in range(nb)]
            w2 = [rnd(D, D + F) for _ in range(nb)]
            b1, b2 = rnd(3 * D + F), rnd(D)
            h = rnd(B * L, D)
            y = torch.empty((B * L, 3 * D + F), dtype=torch.bfloat16, device=dev)
            z = rnd(B * L, D + F)
            xs, gate = rnd(B * L, D, dt=torch.float32, scale=1.0), rnd(B, D, dt=torch.float32, scale=1.0)
            q, k, v = (rnd(B, L, H, hd, scale=1.0) for _ in range(3))
            o = torch.empty_like(q)
            for r in range(args.steps):
                for i in range(nb):
                    bc.linear(h, w1[i], b1, y, bc.EPI_BIAS_GELU)
                    bc.attention(q, k, v, o)
                    bc.linear(z, w2[i], b2, xs, bc.EPI_GATE_RES, res=xs, gate=gate, rows_per_gate=L)
                    log_tags += tags
            torch.cuda.synchronize()
            del w1, w2, h, y, z, xs, q, k, v, o
        else:
            M = B * T
            nb = cfg.depth
            wq = [rnd(3 * D, D) for _ in range(nb)]
            wo = [rnd(D, D) for _ in range(nb)]
            w1 = [rnd(F, D) for _ in range(nb)]
            w2 = [rnd(D, F) for _ in range(nb)]
            bq, bo, b1, b2 = rnd(3 * D), rnd(D), rnd(F), rnd(D)
            h = rnd(M, D)
            qkv = torch.empty((M, 3 * D), dtype=torch.bfloat16, device=dev)
            a = rnd(M, D)
            hm = torch.empty((M, F), dtype=torch.bfloat16, device=dev)
            x, gate = rnd(M, D, dt=torch.float32, scale=1.0), rnd(B, D, dt=torch.float32, scale=1.0)
            q, k, v = (rnd(B, T, H, hd, scale=1.0) for _ in range(3))
            o = torch.empty_like(q)
            for r in range(args.steps):
                for i in range(nb):
                    bc.linear(h, wq[i], bq, qkv, bc.EPI_BIAS)
                    bc.attention(q, k, v, o)
                    bc.linear(a, wo[i], bo, x, bc.EPI_GATE_RES, res=x, gate=gate, rows_per_gate=T)
                    bc.linear(h, w1[i], b1, hm, bc.EPI_BIAS_GELU)
                    bc.linear(hm, w2[i], b2, x, bc.EPI_GATE_RES, res=x, gate=gate, rows_per_gate=T)
                    log_tags += tags
            torch.cuda.synchronize()
            del wq, wo, w1, w2, h, qkv, a, hm, x, q, k, v, o
        torch.cuda.empty_cache()
    shape = synth.FORECAST_SHAPE
    n = shape[0] * shape[1] * shape[2]
    storage = torch.empty((3, n), dtype=torch.bfloat16, device=dev).normal_(generator=g)
    ring = bc.CacheRing(3, storage)
    s, t = synth.forecast_times(3)
    for j in reversed(range(3)):
        ring.push(None, float(s[j]))
    out = torch.empty(n, dtype=torch.bfloat16, device=dev)
    w = bc.bary_weights(s, t)
    for _ in range(args.steps):
        bc.bary_extrapolate(ring, w, out)
        log_tags.append("forecast_k3_bf16")
    torch.cuda.synchronize()
    del storage, out, ring
    if args.calib_copy:
        nn = 1 << 29
        src = torch.ones(nn, dtype=torch.bfloat16, device=dev)
        store = torch.empty((1, nn), dtype=torch.bfloat16, device=dev)
        ring = bc.CacheRing(1, store)
        ring.push(src, 0.0)
        log_tags.append("calib_copy_1gib")
        torch.cuda.synchronize()
    if args.launch_log:
        with open(args.launch_log, "w") as f:
            json.dump(log_tags, f)
    print(json.dumps({"kernels_only": args.workload, "rounds": args.steps, "launches": len(log_tags)}), flush=True)


def summarize_counters(args):
    """Per-kernel summaries of rocprofv3 --pmc passes over the counter program
    (--kernels-only): each directory under args.summarize_counters holds one
    pass's run_counter_collection.csv; launches.json the program's launch log.
    HBM bytes: FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by
    the ratio of known bytes to the counter's reading on the 1 GiB copy.
    Writes profiles/<tag>_counters.json."""
    import csv
    import glob
    import statistics

    import synth
    root = args.summarize_counters
    tags = json.load(open(os.path.join(root, "launches.json")))
    per = {}   # counter -> list per library dispatch (in order)
    for path in sorted(glob.glob(os.path.join(root, "*", "run_counter_collection.csv"))):
        rows = list(csv.DictReader(open(path)))
        vals, names = {}, {}
        for r in rows:
            d = int(r["Dispatch_Id"])
            names[d] = r["Kernel_Name"]
            vals.setdefault(d, {}).setdefault(r["Counter_Name"], 0.0)
            vals[d][r["Counter_Name"]] += float(r["Counter_Value"])
        lib = [d for d in sorted(names) if names[d].startswith(("void bc::", "bc::"))]
        if len(lib) != len(tags):
            raise SystemExit(f"{path}: {len(lib)} library dispatches, launch log has {len(tags)}")
        for d, tag in zip(lib, tags):
            for c, v in vals[d].items():
                per.setdefault(tag, {}).setdefault(c, []).append(v)
            per[tag].setdefault("_kernel", set()).add(names[d])
    calib = per.get("calib_copy_1gib")
    if not calib:
        raise SystemExit("no calibration copy in the launch log")
    nbytes = float(1 << 30)
    f_fetch = nbytes / (calib["FETCH_SIZE"][0] * 1024.0)
    f_write = nbytes / (calib["WRITE_SIZE"][0] * 1024.0)
    known = {}
    for name in args.workload.split(","):
        for k in kernel_tags(synth.CONFIGS[name]):
            known[k["tag"]] = k
    n = synth.FORECAST_SHAPE[0] * synth.FORECAST_SHAPE[1] * synth.FORECAST_SHAPE[2]
    known["forecast_k3_bf16"] = {"tag": "forecast_k3_bf16", "shape": list(synth.FORECAST_SHAPE), "bytes": 4 * n * 2}
    src_for = {"attention": KERNEL_SOURCES["attention"], "gemm": KERNEL_SOURCES["gemm"],
               "forecast": KERNEL_SOURCES["forecast"]}
    written = []
    for tag, c in per.items():
        if tag == "calib_copy_1gib":
            continue
        med = {k: statistics.median(v) for k, v in c.items() if k != "_kernel"}
        info = known[tag]
        rec = {"tag": tag, "kernel": sorted(c["_kernel"]), "shape": info["shape"], "dispatches": len(c.get("FETCH_SIZE", [])),
               "source_hash": source_hash(*src_for[tag.split("_")[0]]),
               "command": "rocprofv3 --pmc <counters> -d <dir>/<pass> -o run --output-format csv -- python3 bench.py "
                          f"--kernels-only --workload {args.workload} --steps {args.steps} --calib-copy "
                          "--launch-log <dir>/launches.json  (passes: FETCH_SIZE; WRITE_SIZE; SQ counters)",
               "calibration": {"copy_bytes": int(nbytes), "fetch_factor": round(f_fetch, 4),
                               "write_factor": round(f_write, 4)},
               "counters_median_per_dispatch": {k: round(v, 1) for k, v in med.items()}}
        if "FETCH_SIZE" in med and "WRITE_SIZE" in med:
            rec["hbm_fetch_bytes"] = int(med["FETCH_SIZE"] * 1024 * f_fetch)
            rec["hbm_write_bytes"] = int(med["WRITE_SIZE"] * 1024 * f_write)
            rec["hbm_bytes_per_launch"] = rec["hbm_fetch_bytes"] + rec["hbm_write_bytes"]
            rec["algorithmic_bytes"] = int(info["bytes"])
            rec["traffic_over_algorithmic"] = round(rec["hbm_bytes_per_launch"] / info["bytes"], 3)
        if "SQ_VALU_MFMA_BUSY_CYCLES" in med and "GRBM_GUI_ACTIVE" in med:
            # GRBM_GUI_ACTIVE is reported per XCD (8 instances summed), MFMA busy per SIMD (1024 summed)
            rec["mfma_busy_frac"] = round(med["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / (med["GRBM_GUI_ACTIVE"] / 8), 4)
            if "SQ_VALU_MFMA_COEXEC_CYCLES" in med:
                rec["mfma_valu_coexec_frac"] = round(med["SQ_VALU_MFMA_COEXEC_CYCLES"] / 1024 / (med["GRBM_GUI_ACTIVE"] / 8), 4)
            if "SQ_LDS_BANK_CONFLICT" in med and "SQ_LDS_IDX_ACTIVE" in med:
                rec["lds_bank_conflict_over_active"] = round(med["SQ_LDS_BANK_CONFLICT"] / max(med["SQ_LDS_IDX_ACTIVE"], 1), 4)
        if "flops" in info:
            rec["flops_per_launch"] = info["flops"]
        out = os.path.join(ROOT, "profiles", f"{tag}_counters.json")
        with open(out, "w") as f:
            json.dump(rec, f, indent=1)
        written.append(out)
    print(json.dumps({"written": written}))


def loop_counters(args):
    """The whole sampling loop of --workload, --steps runs back to back, then
    one 1 GiB copy through the library's push path (counter calibration):
    what the whole-loop counter passes profile."""
    import torch

    import synth
    from paper_2608_28670_amd import loader
    bc = ensure_library()
    dev = "cuda:0"
    cfg = synth.CONFIGS[args.workload]
    dm = loader.DeviceModel(cfg, None, dev_params=device_params(cfg, torch, dev))
    mask = bc.make_mask(cfg.steps, cfg.interval)
    labels = synth.labels(cfg) if cfg.n_classes else None
    text = synth.text(cfg) if cfg.kind != "dit" else None
    x = torch.from_numpy(synth.latents(cfg)).to(dev)
    tl = torch.from_numpy(labels).to(dev) if labels is not None else None
    tt = torch.from_numpy(text).to(dev).to(loader.torch_dtype(cfg)) if text is not None else None
    for r in range(args.steps):
        dm.sample(x, mask, labels=tl, text=tt)
        torch.cuda.synchronize()
        log(f"[{cfg.name}] sampling run {r + 1} of {args.steps} done")
    del dm
    torch.cuda.empty_cache()
    nn = 1 << 29
    src = torch.ones(nn, dtype=torch.bfloat16, device=dev)
    store = torch.empty((1, nn), dtype=torch.bfloat16, device=dev)
    ring = bc.CacheRing(1, store)
    ring.push(src, 0.0)
    torch.cuda.synchronize()
    print(json.dumps({"loop_counters": args.workload, "runs": args.steps, "full_steps": int(mask.sum())}), flush=True)


def summarize_loop_counters(args):
    """profiles/sampling_loop_<workload>_counters.{md,json} from rocprofv3
    --pmc passes over `bench.py --loop-counters` (one run_counter_collection.csv
    per pass directory under args.summarize_loop_counters): per kernel and grid
    size, the dispatches of one sampling run, HBM bytes per dispatch
    (FETCH_SIZE and WRITE_SIZE scaled by the calibration copy, the last library
    dispatch) and MFMA-busy / VALU-active fractions of the dispatch's cycles.
    The JSON is what the roofline's `traffic` is read from."""
    import csv
    import glob
    import statistics
    root = args.summarize_loop_counters
    per = {}      # (kernel, grid) -> counter -> [values per dispatch]
    calib = {}
    passes = []
    for path in sorted(glob.glob(os.path.join(root, "*", "run_counter_collection.csv"))):
        vals, names = {}, {}
        for r in csv.DictReader(open(path)):
            d = int(r["Dispatch_Id"])
            names[d] = (r["Kernel_Name"], int(r["Grid_Size"]))
            vals.setdefault(d, {}).setdefault(r["Counter_Name"], 0.0)
            vals[d][r["Counter_Name"]] += float(r["Counter_Value"])
        lib = [d for d in sorted(names) if names[d][0].startswith(("void bc::", "bc::"))]
        passes.append(os.path.basename(os.path.dirname(path)) + ": " + ", ".join(sorted(vals[lib[0]])))
        for c, v in vals[lib[-1]].items():
            calib[c] = v
        for d in lib[:-1]:
            for c, v in vals[d].items():
                per.setdefault(names[d], {}).setdefault(c, []).append(v)
    nbytes = float(1 << 30)
    f_fetch = nbytes / (calib["FETCH_SIZE"] * 1024.0) if "FETCH_SIZE" in calib else None
    f_write = nbytes / (calib["WRITE_SIZE"] * 1024.0) if "WRITE_SIZE" in calib else None
    runs = args.steps
    rows = []
    for (name, grid), c in per.items():
        n = max(len(v) for v in c.values())
        med = {k: statistics.median(v) for k, v in c.items()}
        tot = {k: sum(v) for k, v in c.items()}
        r = {"kernel": name, "grid_threads": grid, "dispatches_per_run": n / runs}
        if f_fetch and "FETCH_SIZE" in med:
            r["fetch_bytes"] = int(med["FETCH_SIZE"] * 1024 * f_fetch)
        if f_write and "WRITE_SIZE" in med:
            r["write_bytes"] = int(med["WRITE_SIZE"] * 1024 * f_write)
        if "fetch_bytes" in r and "write_bytes" in r:
            r["hbm_bytes"] = r["fetch_bytes"] + r["write_bytes"]
        if "GRBM_GUI_ACTIVE" in tot:
            cyc = tot["GRBM_GUI_ACTIVE"] / 8          # per XCD, summed over the 8
            r["cycles_per_run"] = cyc / runs
            if "SQ_VALU_MFMA_BUSY_CYCLES" in tot:
                r["mfma_busy"] = round(tot["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / cyc, 4)
            if "SQ_ACTIVE_INST_VALU" in tot:
                r["valu_active"] = round(tot["SQ_ACTIVE_INST_VALU"] * 4 / 1024 / cyc, 4)
        rows.append(r)
    rows.sort(key=lambda r: -r.get("cycles_per_run", 0.0))
    total_cyc = sum(r.get("cycles_per_run", 0.0) for r in rows)
    cmd = (f"rocprofv3 --pmc <counters> -d <dir>/<pass> -o run --output-format csv -- "
           f"python3 bench.py --loop-counters --workload {args.workload} --steps {runs}")
    rec = {"workload": args.workload, "runs": runs, "command": cmd, "passes": passes,
           "source_hashes": {k: source_hash(*v) for k, v in KERNEL_SOURCES.items()},
           "calibration": {"copy_bytes": int(nbytes), "fetch_factor": round(f_fetch, 4) if f_fetch else None,
                           "write_factor": round(f_write, 4) if f_write else None},
           "groups": rows}
    with open(os.path.join(ROOT, "profiles", f"sampling_loop_{args.workload}_counters.json"), "w") as fh:
        json.dump(rec, fh, indent=1)
    out = [f"# Hardware counters over the whole sampling loop: {args.workload}", "",
           "Commands (from a shell in `/tmp`, `TMPDIR=/tmp`), one pass per counter set:", "",
           "    " + cmd,
           f"    python3 bench.py --summarize-loop-counters <dir> --workload {args.workload} --steps {runs}", "",
           "Passes: " + "; ".join(passes) + ".", "",
           "Counter runs serialise the dispatches, so cycles are each dispatch's own duration "
           "(GRBM_GUI_ACTIVE, summed over the 8 XCDs and divided by 8). HBM bytes: FETCH_SIZE and WRITE_SIZE "
           "(KiB per dispatch, medians) times the factor that makes the 1 GiB calibration copy read its known "
           f"size (fetch x{f_fetch:.4f}, write x{f_write:.4f})." if f_fetch and f_write else "",
           "MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES over the 1024 SIMDs' cycles; VALU active: SQ_ACTIVE_INST_VALU "
           "(counted per 4 cycles) over the same. One row per kernel and grid size.", "",
           "| kernel | grid (threads) | dispatches per run | share of cycles | fetch MB | write MB | MFMA busy | VALU active |",
           "|---|---|---|---|---|---|---|---|"]

    def f(r, k, fmt, scale=1.0):
        return format(r[k] * scale, fmt) if k in r else "-"
    for r in rows[:40]:
        share = r.get("cycles_per_run", 0.0) / total_cyc if total_cyc else 0.0
        out.append(f"| `{r['kernel'][:140]}` | {r['grid_threads']} | {r['dispatches_per_run']:.0f} | {share:.1%} | "
                   f"{f(r, 'fetch_bytes', '.1f', 1e-6)} | {f(r, 'write_bytes', '.1f', 1e-6)} | "
                   f"{f(r, 'mfma_busy', '.1%')} | {f(r, 'valu_active', '.1%')} |")
    path = os.path.join(ROOT, "profiles", f"sampling_loop_{args.workload}_counters.md")
    with open(path, "w") as fh:
        fh.write("\n".join(out) + "\n")
    print(path)


def summarize_trace(args):
    """profiles/bench_kernel_trace.md from a rocprofv3 --kernel-trace --stats
    run of the default bench command (run_kernel_stats.csv) and the JSON line
    that run printed."""
    import csv
    stats_path, line_path = args.summarize_trace.split(",")
    rows = list(csv.DictReader(open(stats_path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    line = json.load(open(line_path))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    out = ["# Kernel trace of the default benchmark command", "",
           "Command (from a shell in `/tmp`, `TMPDIR=/tmp`):", "",
           "    rocprofv3 --kernel-trace --stats -d <dir> -o run --output-format csv -- "
           f"python3 bench.py --gpus 1 --steps {line['steps']} --warmup {line['warmup']}", "",
           f"The run covers everything the command does: the video workload ({line['warmup']} warm-up, "
           f"{line['steps']} timed and one "
           "event-timed sampling runs, then one all-full-mask run), the DiT-XL/2 and PixArt legs, the forecast sweep, "
           "the push copy.  Per-call averages are the figures to compare with the JSON line's per-launch averages "
           "(which come from HIP events in the same process).", "",
           f"JSON line of this traced run: value {line['value']} samples/s, {line['ms_per_step']} ms per sampling run; "
           f"roofline kernel `{line['roofline']['kernel']}` avg {line['roofline']['avg_us']} us "
           f"-> {line['roofline']['achieved']} TFLOP/s = {line['roofline']['frac']} of {line['roofline']['peak']}.", "",
           "| kernel | calls | total ms | avg us | share |", "|---|---|---|---|---|"]
    for r in rows[:30]:
        out.append(f"| `{r['Name'][:150]}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.1f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['TotalDurationNs']) / total:.1%} |")
    path = os.path.join(ROOT, "profiles", "bench_kernel_trace.md")
    with open(path, "w") as f:
        f.write("\n".join(out) + "\n")
    print(path)


# ---------------------------------------------------------------------------

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    if args.kernels_only:
        kernels_only(args)
        return
    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.loop_counters:
        loop_counters(args)
        return
    if args.summarize_loop_counters:
        summarize_loop_counters(args)
        return
    if args.summarize_trace:
        summarize_trace(args)
        return
    import torch

    import synth
    bc = ensure_library()
    cfg = synth.CONFIGS[args.workload]
    head = measure(bc, torch, cfg, args.steps, args.warmup, extras=not args.no_extras and cfg.kind == "dit",
                   adaptive_ell=args.adaptive_ell)
    legs = {}
    for name in [w for w in args.legs.split(",") if w and w != args.workload]:
        lc = synth.CONFIGS[name]
        r = measure(bc, torch, lc, args.leg_steps, 1, extras=not args.no_extras and lc.kind == "dit",
                    adaptive_ell=args.adaptive_ell)
        leg = {"config": workload_desc(lc, r.pop("mask")), "value": round(r.pop("value"), 3), "unit": "samples/s",
               "ms_per_step": round(r.pop("ms_per_step"), 3), "steps": args.leg_steps, "warmup": 1,
               "speedup_vs_all_full": round(r.pop("speedup_vs_all_full"), 3),
               "ms_all_full": round(r.pop("ms_all_full"), 3), "ideal_speedup": round(r.pop("ideal_speedup"), 3)}
        leg.update(r)
        legs[name] = leg
    forecast, push = (None, None) if args.no_forecast else forecast_sweep(bc, torch)
    cpu = None
    others = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline_video(cfg) if cfg.kind == "mmdit" else cpu_baseline_image(cfg)
        # The other configurations' oracle timings (context for their legs).
        others = {"tiny": cpu_baseline_tiny(synth.CONFIGS["tiny"]),
                  "dit_xl2": cpu_baseline_blocks(synth.CONFIGS["dit_xl2"]),
                  "pixart": cpu_baseline_blocks(synth.CONFIGS["pixart"]),
                  "forecast_k3_f32": cpu_baseline_forecast()}
        log("[cpu] other configurations: " + ", ".join(f"{k} {v['value']} {v['unit']}" for k, v in others.items()))

    mask = head.pop("mask")
    line = {
        "metric": "end-to-end samples/s at fixed skip schedule; forecast HBM GB/s; block MFMA util",
        "value": round(head["value"], 4), "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(head["ms_per_step"], 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": workload_desc(cfg, mask), "global_batch": cfg.batch, "seq_len": cfg.tokens,
                   "parallelism": "none (1 GPU)"},
        "speedup_vs_all_full": round(head["speedup_vs_all_full"], 3),
        "ms_all_full": round(head["ms_all_full"], 3),
        "ideal_speedup": round(head["ideal_speedup"], 3),
        "roofline": head["roofline"],
        "roofline_others": head["roofline_others"],
        "kernel_classes": head["kernel_classes"],
        "profiled_run_ms": head["profiled_run_ms"],
        "workloads": legs,
        "forecast": forecast,
        "push_copy": push,
        "cpu_baseline": cpu,
        "cpu_baselines_other": others,
        "paper_context": PAPER_CONTEXT,
    }
    for k in ("graph_replay", "adaptive", "blockwise"):
        if k in head:
            line[k] = head[k]
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

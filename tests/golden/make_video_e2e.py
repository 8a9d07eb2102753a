"""Write tests/golden/video_e2e_sampled.txt: the oracle's final latent of the
video workload at its real width and full token count (hidden 3072, 24 heads
of 128, MLP 12288, 14 310 image + 256 text tokens, batch 1, 50 shift-7 Euler
steps, K = 3, a full step every 5th) with the depth reduced to one dual-stream
and one single-stream block, at 4096 seeded element positions.

Calls only the oracle (fp32) and the seeded input generators.  Takes about
15-30 minutes on 8 host cores:

    python tests/golden/make_video_e2e.py
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import bary, model as om, sampler as osm  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "video_e2e_sampled.txt")
N_SAMPLED = 4096


def config():
    return synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, batch=1)


def positions(n_total):
    idx = np.sort(np.random.default_rng(2026).choice(n_total, N_SAMPLED - 2, replace=False))
    return np.unique(np.concatenate([[0], idx, [n_total - 1]]))


def main():
    cfg = config()
    t0 = time.time()
    P = synth.params(cfg)
    M = om.Model(cfg, P, dtype=np.float32)
    xT = synth.latents(cfg)
    text = synth.text(cfg)
    mask = bary.make_mask(cfg.steps, cfg.interval)
    trace = {}
    x = osm.sample(M, xT.astype(np.float64), mask, cfg.K, text=text, trace=trace)
    idx = positions(x.size)
    flat = np.asarray(x, dtype=np.float64).reshape(-1)
    with open(OUT, "w") as f:
        f.write("# The oracle's final latent (fp32 model, fp64 sampler state) of the video workload at real width\n"
                "# and full token count, one dual-stream and one single-stream block, 50 shift-7 Euler steps, K = 3,\n"
                f"# full steps {''.join(map(str, mask))}; inputs from synth (seed {synth.SEED}).\n"
                "# Written by tests/golden/make_video_e2e.py (oracle only).\n"
                f"# latent shape {list(x.shape)}; whole-tensor L2 norm {np.linalg.norm(flat):.9e}, "
                f"mean {flat.mean():.9e}\n"
                "# flat index, value\n")
        for i in idx:
            f.write(f"{int(i)} {flat[i]:.9e}\n")
    print(f"wrote {OUT}: {len(idx)} values in {time.time() - t0:.0f} s")


if __name__ == "__main__":
    main()

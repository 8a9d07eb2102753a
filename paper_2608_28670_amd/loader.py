"""Upload a DiT-family model's weights to the GPU and drive bc_sample.

Marshalling only: host arrays become device tensors of the model dtype, their
addresses fill the C descriptors of include/bc.h, and sampling is one call of
bc_sample.  `cfg` is any object with the workload fields (kind, depth,
depth_single, hidden, heads, head_dim, mlp, in_ch, out_ch, patch, latent,
n_classes, ctx_tokens, ctx_dim, txt_tokens, freq_dim, dtype, K, tokens).
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

from . import (BF16, BLOCK_DIT, BLOCK_DUAL, BLOCK_PIXART, BLOCK_SINGLE, F32, MODEL_DIT, MODEL_MMDIT,
               MODEL_PIXART, BlockWeights, CacheRing, Model, ModelDesc, SampleGraph, block_weights, sample,
               sample_adaptive, sample_blockwise, sample_cfg)

_KIND = {"dit": MODEL_DIT, "pixart": MODEL_PIXART, "mmdit": MODEL_MMDIT}


def torch_dtype(cfg):
    import torch
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def upload(params: Dict[str, np.ndarray], cfg, device="cuda:0"):
    import torch
    dt = torch_dtype(cfg)
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(device=device).to(dt) for k, v in params.items()}


def model_desc(cfg) -> ModelDesc:
    d = ModelDesc()
    d.kind = _KIND[cfg.kind]
    d.depth, d.depth_single = cfg.depth, cfg.depth_single
    d.D, d.heads, d.head_dim, d.mlp = cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp
    d.in_ch, d.out_ch, d.patch = cfg.in_ch, cfg.out_ch, cfg.p
    if len(cfg.latent) == 3:
        d.frames, d.height, d.width = 1, cfg.latent[1], cfg.latent[2]
    else:
        d.frames, d.height, d.width = cfg.latent[1], cfg.latent[2], cfg.latent[3]
    d.n_classes = cfg.n_classes
    d.ctx_tokens, d.ctx_dim, d.txt_tokens = cfg.ctx_tokens, cfg.ctx_dim, cfg.txt_tokens
    d.freq_dim = cfg.freq_dim
    d.dtype = BF16 if cfg.dtype == "bf16" else F32
    d.rope_theta = getattr(cfg, "rope_theta", 0.0) if cfg.kind == "mmdit" else 0.0
    d.flow_shift = getattr(cfg, "flow_shift", 1.0)
    return d


def rope_grid(cfg):
    """(frames, rows, columns, theta) of the image-token grid for block
    descriptors, or None when the model has no rotary embedding."""
    if cfg.kind != "mmdit" or not getattr(cfg, "rope_theta", 0.0):
        return None
    f = 1 if len(cfg.latent) == 3 else cfg.latent[1]
    return f, cfg.latent[-2] // cfg.p, cfg.latent[-1] // cfg.p, cfg.rope_theta


def _stream(P, pre):
    return {"w_mod": P.get(pre + "w_mod", P.get(pre + "table")), "b_mod": P.get(pre + "b_mod"),
            "w_qkv": P.get(pre + "w_qkv"), "b_qkv": P.get(pre + "b_qkv"),
            "w_o": P.get(pre + "w_o"), "b_o": P.get(pre + "b_o"),
            "w_fc1": P.get(pre + "w_fc1"), "b_fc1": P.get(pre + "b_fc1"),
            "w_fc2": P.get(pre + "w_fc2"), "b_fc2": P.get(pre + "b_fc2"),
            "q_norm": P.get(pre + "q_norm"), "k_norm": P.get(pre + "k_norm")}


def block_list(cfg, P) -> List[BlockWeights]:
    out = []
    if cfg.kind in ("dit", "pixart"):
        for l in range(cfg.depth):
            pre = f"blocks.{l}."
            cross = None
            if cfg.kind == "pixart":
                cross = {k: P[pre + k] for k in ("wx_q", "bx_q", "wx_kv", "bx_kv", "wx_o", "bx_o")}
            out.append(block_weights(_stream(P, pre), None, cross))
    else:
        for l in range(cfg.depth):
            out.append(block_weights(_stream(P, f"dual.{l}.img."), _stream(P, f"dual.{l}.txt.")))
        for l in range(cfg.depth_single):
            pre = f"single.{l}."
            out.append(block_weights({"w_mod": P[pre + "w_mod"], "b_mod": P[pre + "b_mod"],
                                      "w_qkv": P[pre + "w_1"], "b_qkv": P[pre + "b_1"],
                                      "w_o": P[pre + "w_2"], "b_o": P[pre + "b_2"],
                                      "q_norm": P.get(pre + "q_norm"), "k_norm": P.get(pre + "k_norm")}))
    return out


def model_weights(cfg, P) -> Dict[str, object]:
    w = {k: P.get(k) for k in ("t_w1", "t_b1", "t_w2", "t_b2", "patch_w", "patch_b", "pos", "y_table", "t6_w",
                               "t6_b", "cap_w1", "cap_b1", "cap_w2", "cap_b2", "txt_w", "txt_b", "final_w",
                               "final_b")}
    if cfg.kind == "pixart":
        w["final_w_mod"], w["final_b_mod"] = P["final_table"], None
    else:
        w["final_w_mod"], w["final_b_mod"] = P["final_w_mod"], P["final_b_mod"]
    return w


class DeviceModel:
    """A model resident on one GPU with its bc_model handle."""

    def __init__(self, cfg, params: Dict[str, np.ndarray], device="cuda:0", dev_params=None):
        self.cfg = cfg
        self.device = device
        self.P = dev_params if dev_params is not None else upload(params, cfg, device)
        self.model = Model(model_desc(cfg), model_weights(cfg, self.P), block_list(cfg, self.P))
        self._ws = {}
        self._ring = {}
        self._sites = {}

    def workspace(self, B: int, S: int):
        """bc_sample's workspace for batch B and S steps (allocated once, reused)."""
        import torch
        if (B, S) not in self._ws:
            n = self.model.workspace_size(B, S)
            self._ws[(B, S)] = torch.empty(n, dtype=torch.uint8, device=self.device)
        return self._ws[(B, S)]

    def buffers(self, B: int, K: int, S: int):
        """Workspace and ring storage for batch B and S steps (allocated once, reused)."""
        return self.workspace(B, S), self.ring(B, K)

    def ring(self, B: int, K: int) -> CacheRing:
        """Ring of K slots of B*T*D elements (allocated once, reused)."""
        import torch
        key = (B, K)
        if key not in self._ring:
            numel = B * self.cfg.tokens * self.cfg.hidden
            storage = torch.empty((K, numel), dtype=torch_dtype(self.cfg), device=self.device)
            self._ring[key] = CacheRing(K, storage)
        return self._ring[key]

    def sample_graph(self, x, mask, K: Optional[int] = None, labels=None, text=None, p=None):
        """The same run captured as a HIP graph on x's buffer; .launch() replays it in place."""
        K = K or self.cfg.K
        B = x.shape[0]
        ws, ring = self.buffers(B, K, len(mask))
        return SampleGraph(self.model, B, self.cfg.sampler, mask, K, ring, x, ws, labels=labels, text=text, p=p)

    def sample_blockwise(self, x, mask, K: Optional[int] = None, labels=None, text=None, p=None, stream=None):
        """Blockwise-mode sampling in place on x; returns the site storage
        [sites, K, B*T*D] (allocated once per (B, K) and reused)."""
        import torch
        K = K or self.cfg.K
        B = x.shape[0]
        ws = self.workspace(B, len(mask))
        key = (B, K)
        if key not in self._sites:
            n = self.model.blockwise_sites()
            self._sites[key] = torch.empty((n, K, B * self.cfg.tokens * self.cfg.hidden), dtype=torch_dtype(self.cfg),
                                           device=self.device)
        sample_blockwise(self.model, B, self.cfg.sampler, mask, K, self._sites[key], x, ws, labels=labels,
                         text=text, p=p, stream=stream)
        return self._sites[key]

    def release_blockwise(self):
        """Drop the blockwise site storage (it is sites * K times the stepwise ring)."""
        self._sites.clear()

    def sample_adaptive(self, x, S: int, ell: float, K: Optional[int] = None, labels=None, text=None, p=None,
                        stream=None):
        """Adaptive-schedule sampling in place on x; returns (ring, mask, changes)."""
        import torch
        K = K or self.cfg.K
        B = x.shape[0]
        key = ("adaptive", B, S)
        if key not in self._ws:
            self._ws[key] = torch.empty(self.model.adaptive_workspace_size(B, S), dtype=torch.uint8,
                                        device=self.device)
        ring = self.ring(B, K)
        mask, change = sample_adaptive(self.model, B, self.cfg.sampler, S, ell, K, ring, x, self._ws[key],
                                       labels=labels, text=text, p=p, stream=stream)
        return ring, mask, change

    def sample_cfg(self, x, mask, labels, cfg_scale: float, K: Optional[int] = None, p=None, stream=None):
        """Classifier-free guided sampling in place on x (B latents; model batch 2B)."""
        K = K or self.cfg.K
        B = x.shape[0]
        ws, ring = self.buffers(2 * B, K, len(mask))
        sample_cfg(self.model, B, self.cfg.sampler, mask, K, ring, x, ws, labels, cfg_scale, p=p, stream=stream)
        return ring

    def sample(self, x, mask, K: Optional[int] = None, labels=None, text=None, p=None, stream=None):
        """BaryCache sampling in place on x (fp32 device latents [B, ...])."""
        K = K or self.cfg.K
        B = x.shape[0]
        ws, ring = self.buffers(B, K, len(mask))
        sample(self.model, B, self.cfg.sampler, mask, K, ring, x, ws, labels=labels, text=text, p=p,
               stream=stream)
        return ring

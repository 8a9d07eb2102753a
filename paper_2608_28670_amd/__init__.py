"""Python binding of libbarycache (the C ABI in include/bc.h).

Argument marshalling only: every step of the hot path runs in the library's
HIP kernels.  Device buffers are torch tensors (used for device memory and
streams only); host arrays are numpy.  There is no fallback: if the built
library is missing, loading fails with an error that says how to build it.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libbarycache.so")

OK, ERR_INVALID_ARG, ERR_DEGENERATE, ERR_STATE, ERR_HIP, ERR_UNSUPPORTED = range(6)
F32, BF16 = 0, 1
NODES_TRAPEZOID, NODES_LAGRANGE = 0, 1
BLEND_RECENT, BLEND_LITERAL = 0, 1
BLOCK_DIT, BLOCK_PIXART, BLOCK_DUAL, BLOCK_SINGLE = range(4)
MODEL_DIT, MODEL_PIXART, MODEL_MMDIT = range(3)
SAMPLER_DDIM, SAMPLER_DPMPP2M, SAMPLER_EULER = range(3)
EPI_BIAS, EPI_BIAS_GELU, EPI_GATE_RES = range(3)
PROF_FORECAST, PROF_GEMM_GELU, PROF_GEMM_GATE, PROF_GEMM_BIAS, PROF_ATTENTION, PROF_LAYERNORM, PROF_GEMM_DOWN, \
    PROF_COPY = range(8)
SAMPLERS = {"ddim": SAMPLER_DDIM, "dpmpp2m": SAMPLER_DPMPP2M, "euler": SAMPLER_EULER}


class BCError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


# ---------------------------------------------------------------------------
# C structures (mirror include/bc.h)
# ---------------------------------------------------------------------------

class BaryParams(C.Structure):
    _fields_ = [("nodes", C.c_int), ("clip_C", C.c_double), ("eta", C.c_double),
                ("delta", C.c_double), ("lambda_", C.c_double), ("blend", C.c_int)]


class PlanStep(C.Structure):
    _fields_ = [("is_full", C.c_int), ("count", C.c_int), ("head", C.c_int),
                ("slots", C.c_int * 8), ("w", C.c_double * 8)]


class BlockDesc(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("kind", "B", "T", "D", "heads", "head_dim", "mlp",
                                       "T_txt", "T_ctx", "dtype", "rope_f", "rope_h", "rope_w")] + \
               [("rope_theta", C.c_double)]


_STREAM_FIELDS = ("w_mod", "b_mod", "w_qkv", "b_qkv", "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2",
                  "q_norm", "k_norm")


class StreamWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _STREAM_FIELDS]


class BlockWeights(C.Structure):
    _fields_ = [("img", StreamWeights), ("txt", StreamWeights)] + \
               [(n, C.c_void_p) for n in ("wx_q", "bx_q", "wx_kv", "bx_kv", "wx_o", "bx_o")]


class ModelDesc(C.Structure):
    _fields_ = [(n, C.c_int) for n in ("kind", "depth", "depth_single", "D", "heads", "head_dim", "mlp",
                                       "in_ch", "out_ch", "patch", "frames", "height", "width",
                                       "n_classes", "ctx_tokens", "ctx_dim", "txt_tokens", "freq_dim",
                                       "dtype")] + [("rope_theta", C.c_double), ("flow_shift", C.c_double)]


_MODEL_PTRS = ("t_w1", "t_b1", "t_w2", "t_b2", "patch_w", "patch_b", "pos", "y_table", "t6_w", "t6_b",
               "cap_w1", "cap_b1", "cap_w2", "cap_b2", "txt_w", "txt_b", "final_w_mod", "final_b_mod",
               "final_w", "final_b")


class ModelWeights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _MODEL_PTRS] + [("blocks", C.POINTER(BlockWeights))]


# ---------------------------------------------------------------------------
# library loading
# ---------------------------------------------------------------------------

_lib: Optional[C.CDLL] = None

_SIGS = {
    "bc_status_str": (C.c_char_p, [C.c_int]),
    "bc_last_error": (C.c_char_p, []),
    "bc_version": (C.c_int, []),
    "bc_build_id": (C.c_char_p, []),
    "bc_bary_params_default": (None, [C.POINTER(BaryParams)]),
    "bc_bary_weights": (C.c_int, [C.c_void_p, C.c_int, C.c_double, C.c_void_p]),
    "bc_bary_weights_ex": (C.c_int, [C.c_void_p, C.c_int, C.c_double, C.POINTER(BaryParams), C.c_void_p]),
    "bc_make_mask": (C.c_int, [C.c_int, C.c_int, C.c_int, C.c_void_p]),
    "bc_plan": (C.c_int, [C.c_int, C.c_void_p, C.c_void_p, C.c_int, C.POINTER(BaryParams),
                          C.POINTER(PlanStep)]),
    "bc_cache_create": (C.c_int, [C.c_int, C.c_int64, C.c_int, C.c_void_p, C.POINTER(C.c_void_p)]),
    "bc_cache_destroy": (C.c_int, [C.c_void_p]),
    "bc_cache_reset": (C.c_int, [C.c_void_p]),
    "bc_cache_next_slot": (C.c_int, [C.c_void_p, C.POINTER(C.c_void_p)]),
    "bc_cache_push": (C.c_int, [C.c_void_p, C.c_void_p, C.c_double, C.c_void_p]),
    "bc_cache_state": (C.c_int, [C.c_void_p, C.POINTER(C.c_int), C.POINTER(C.c_int), C.c_void_p, C.c_void_p]),
    "bc_bary_extrapolate": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_int, C.c_void_p]),
    "bc_block_workspace_size": (C.c_int, [C.POINTER(BlockDesc), C.POINTER(C.c_size_t)]),
    "bc_dit_block_forward": (C.c_int, [C.POINTER(BlockDesc), C.POINTER(BlockWeights), C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                       C.c_void_p]),
    "bc_dit_block_forward_noalloc": (C.c_int, [C.POINTER(BlockDesc), C.POINTER(BlockWeights), C.c_void_p,
                                               C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]),
    "bc_noalloc_scratch_bytes": (C.c_size_t, []),
    "bc_model_create": (C.c_int, [C.POINTER(ModelDesc), C.POINTER(ModelWeights), C.POINTER(C.c_void_p)]),
    "bc_model_destroy": (C.c_int, [C.c_void_p]),
    "bc_make_schedule": (C.c_int, [C.c_int, C.c_int, C.c_void_p, C.c_void_p]),
    "bc_make_schedule_shifted": (C.c_int, [C.c_int, C.c_int, C.c_double, C.c_void_p, C.c_void_p]),
    "bc_sample_workspace_size": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.POINTER(C.c_size_t)]),
    "bc_sample": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int,
                            C.POINTER(BaryParams), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                            C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_sample_cfg": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int,
                                C.POINTER(BaryParams), C.c_void_p, C.c_void_p, C.c_void_p, C.c_float,
                                C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_blockwise_sites": (C.c_int, [C.c_void_p, C.POINTER(C.c_int)]),
    "bc_sample_blockwise": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int,
                                      C.POINTER(BaryParams), C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p,
                                      C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_sample_adaptive_workspace_size": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.POINTER(C.c_size_t)]),
    "bc_sample_adaptive": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_double, C.c_int,
                                     C.POINTER(BaryParams), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                     C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p, C.c_void_p]),
    "bc_sample_graph_create": (C.c_int, [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int,
                                         C.POINTER(BaryParams), C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                         C.c_void_p, C.c_size_t, C.c_void_p, C.POINTER(C.c_void_p)]),
    "bc_sample_graph_launch": (C.c_int, [C.c_void_p, C.c_void_p]),
    "bc_sample_graph_destroy": (C.c_int, [C.c_void_p]),
    "bc_linear": (C.c_int, [C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                            C.c_int, C.c_void_p, C.c_void_p, C.c_int, C.c_int, C.c_void_p]),
    "bc_attention": (C.c_int, [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p,
                               C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_attention_prescaled": (C.c_int, [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p,
                               C.c_void_p, C.c_void_p, C.c_int, C.c_void_p, C.c_size_t, C.c_void_p]),
    "bc_attention_workspace_size": (C.c_int, [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                                              C.POINTER(C.c_size_t)]),
    "bc_profile_enable": (C.c_int, [C.c_int, C.c_int]),
    "bc_profile_collect": (C.c_int, [C.c_int, C.POINTER(C.c_double), C.POINTER(C.c_int)]),
    "bc_profile_times": (C.c_int, [C.c_int, C.POINTER(C.c_float), C.c_int, C.POINTER(C.c_int)]),
    "bc_profile_records": (C.c_int, [C.c_int, C.POINTER(C.c_float), C.POINTER(C.c_double), C.c_int,
                                     C.POINTER(C.c_int)]),
}


def built_id() -> Optional[str]:
    """The source hash the built library reports, without loading it into
    this process for use (None if it is missing)."""
    if not os.path.exists(LIB_PATH):
        return None
    L = C.CDLL(LIB_PATH)
    fn = L.bc_build_id
    fn.restype = C.c_char_p
    return fn().decode()


def is_current() -> bool:
    """True if the built library was built from the sources in this tree."""
    from . import build
    return built_id() == build.source_hash()


def lib() -> C.CDLL:
    """The loaded library.  Raises if it has not been built, or if it was
    built from other sources than those in this tree."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; "
                              f"g.build()'` or `python paper_2608_28670_amd/build.py`")
        from . import build
        L = C.CDLL(LIB_PATH)
        L.bc_build_id.restype = C.c_char_p
        have, want = L.bc_build_id().decode(), build.source_hash()
        if have != want:
            raise ImportError(f"{LIB_PATH} was built from other sources (build id {have}, sources {want}): "
                              f"rebuild it with `python paper_2608_28670_amd/build.py`")
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def exported_symbols() -> List[str]:
    return list(_SIGS)


def _check(rc: int):
    if rc != OK:
        L = lib()
        raise BCError(rc, f"{L.bc_status_str(rc).decode()}: {L.bc_last_error().decode()}")


# ---------------------------------------------------------------------------
# helpers
# ---------------------------------------------------------------------------

def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def dev_ptr(t) -> Optional[int]:
    """Device address of a torch tensor (None for None)."""
    if t is None:
        return None
    return t.data_ptr()


def dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def stream_handle(stream=None) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def params(nodes: str = "trapezoid", clip_C: float = 10.0, eta: float = 1e-12, delta: Optional[float] = None,
           lam: float = 0.0, blend: str = "recent") -> BaryParams:
    p = BaryParams()
    p.nodes = NODES_TRAPEZOID if nodes == "trapezoid" else NODES_LAGRANGE
    p.clip_C = clip_C
    p.eta = eta
    p.delta = -1.0 if delta is None else delta
    p.lambda_ = lam
    p.blend = BLEND_RECENT if blend == "recent" else BLEND_LITERAL
    return p


def default_params() -> BaryParams:
    p = BaryParams()
    lib().bc_bary_params_default(C.byref(p))
    return p


# ---------------------------------------------------------------------------
# host plan
# ---------------------------------------------------------------------------

def bary_weights(t_nodes: Sequence[float], t_query: float, p: Optional[BaryParams] = None) -> np.ndarray:
    s = _f64(t_nodes)
    w = np.zeros(len(s), dtype=np.float64)
    _check(lib().bc_bary_weights_ex(_ptr(s), len(s), float(t_query), C.byref(p) if p else None, _ptr(w)))
    return w


def make_mask(S: int, interval: int, force_last: bool = True) -> np.ndarray:
    m = np.zeros(S, dtype=np.uint8)
    _check(lib().bc_make_mask(S, interval, int(force_last), _ptr(m)))
    return m


def plan(mask, K: int, coords=None, p: Optional[BaryParams] = None) -> List[PlanStep]:
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    c = _f64(coords) if coords is not None else None
    out = (PlanStep * len(m))()
    _check(lib().bc_plan(len(m), _ptr(m), _ptr(c) if c is not None else None, K,
                         C.byref(p) if p else None, out))
    return list(out)


def make_schedule(sampler: str, S: int, flow_shift: float = 1.0):
    tau = np.zeros(S, dtype=np.int32)
    tm = np.zeros(S, dtype=np.float64)
    _check(lib().bc_make_schedule_shifted(SAMPLERS[sampler], S, float(flow_shift), _ptr(tau), _ptr(tm)))
    return tau, tm


# ---------------------------------------------------------------------------
# cache ring and forecast
# ---------------------------------------------------------------------------

class CacheRing:
    """Ring of K feature slots over a caller-owned device tensor [K, numel]."""

    def __init__(self, K: int, storage):
        self.storage = storage
        self.K = K
        self.numel = storage.numel() // K
        h = C.c_void_p()
        _check(lib().bc_cache_create(K, self.numel, dtype_code(storage), dev_ptr(storage), C.byref(h)))
        self.h = h

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.bc_cache_destroy(self.h)
            self.h = None

    def reset(self):
        _check(lib().bc_cache_reset(self.h))

    def next_slot(self) -> int:
        p = C.c_void_p()
        _check(lib().bc_cache_next_slot(self.h, C.byref(p)))
        return p.value

    def push(self, feat, t: float, stream=None):
        _check(lib().bc_cache_push(self.h, dev_ptr(feat), float(t), stream_handle(stream)))

    def state(self):
        cnt, head = C.c_int(), C.c_int()
        tn = np.zeros(8, dtype=np.float64)
        sl = np.zeros(8, dtype=np.int32)
        _check(lib().bc_cache_state(self.h, C.byref(cnt), C.byref(head), _ptr(tn), _ptr(sl)))
        return cnt.value, head.value, tn[:cnt.value].copy(), sl[:cnt.value].copy()


def bary_extrapolate(ring: CacheRing, w: Sequence[float], out, stream=None):
    wa = _f64(w)
    _check(lib().bc_bary_extrapolate(ring.h, _ptr(wa), len(wa), dev_ptr(out), dtype_code(out),
                                     stream_handle(stream)))


# ---------------------------------------------------------------------------
# building blocks
# ---------------------------------------------------------------------------

def linear(A, W, bias, out, epilogue: int = EPI_BIAS, res=None, gate=None, rows_per_gate: int = 1,
           stream=None):
    M, K = A.shape
    N = W.shape[0]
    _check(lib().bc_linear(M, N, K, dev_ptr(A), dev_ptr(W), dev_ptr(bias), dev_ptr(out), epilogue,
                           dev_ptr(res), dev_ptr(gate), rows_per_gate, dtype_code(A), stream_handle(stream)))


def attention_workspace_size(B, H, Tq, Tk, d, dtype) -> int:
    n = C.c_size_t()
    _check(lib().bc_attention_workspace_size(B, H, Tq, Tk, d, dtype, C.byref(n)))
    return n.value


def attention(q, k, v, out, ws=None, stream=None, prescaled=False):
    """prescaled: q already holds q * log2(e) / sqrt(d) (bc_attention_prescaled)."""
    B, Tq, H, d = q.shape
    Tk = k.shape[1]
    fn = lib().bc_attention_prescaled if prescaled else lib().bc_attention
    _check(fn(B, H, Tq, Tk, d, dev_ptr(q), dev_ptr(k), dev_ptr(v), dev_ptr(out),
              dtype_code(q), dev_ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
              stream_handle(stream)))


def block_desc(kind, B, T, D, heads, head_dim, mlp, dtype, T_txt=0, T_ctx=0, rope=None) -> BlockDesc:
    """rope: (frames, rows, columns, theta) of the image-token grid, or None."""
    d = BlockDesc()
    d.kind, d.B, d.T, d.D, d.heads, d.head_dim, d.mlp = kind, B, T, D, heads, head_dim, mlp
    d.T_txt, d.T_ctx, d.dtype = T_txt, T_ctx, dtype
    if rope is not None:
        d.rope_f, d.rope_h, d.rope_w, d.rope_theta = rope
    return d


def stream_weights(t: Dict[str, object]) -> StreamWeights:
    s = StreamWeights()
    for n in _STREAM_FIELDS:
        setattr(s, n, dev_ptr(t.get(n)))
    return s


def block_weights(img: Dict[str, object], txt: Optional[Dict[str, object]] = None,
                  cross: Optional[Dict[str, object]] = None) -> BlockWeights:
    w = BlockWeights()
    w.img = stream_weights(img)
    w.txt = stream_weights(txt or {})
    for n in ("wx_q", "bx_q", "wx_kv", "bx_kv", "wx_o", "bx_o"):
        setattr(w, n, dev_ptr((cross or {}).get(n)))
    return w


def block_workspace_size(desc: BlockDesc) -> int:
    n = C.c_size_t()
    _check(lib().bc_block_workspace_size(C.byref(desc), C.byref(n)))
    return n.value


def dit_block_forward(desc: BlockDesc, w: BlockWeights, x, c, ws, x_txt=None, ctx=None, stream=None):
    _check(lib().bc_dit_block_forward(C.byref(desc), C.byref(w), dev_ptr(x), dev_ptr(x_txt), dev_ptr(c),
                                      dev_ptr(ctx), dev_ptr(ws), ws.numel() * ws.element_size(),
                                      stream_handle(stream)))


def dit_block_forward_noalloc(desc: BlockDesc, w: BlockWeights, x, c, x_txt=None, ctx=None, stream=None):
    """bc_dit_block_forward with the library's own static workspace (no
    allocation; calls on one GPU share it and must not overlap)."""
    _check(lib().bc_dit_block_forward_noalloc(C.byref(desc), C.byref(w), dev_ptr(x), dev_ptr(x_txt), dev_ptr(c),
                                              dev_ptr(ctx), stream_handle(stream)))


def noalloc_scratch_bytes() -> int:
    return int(lib().bc_noalloc_scratch_bytes())


# ---------------------------------------------------------------------------
# whole model and sampling loop
# ---------------------------------------------------------------------------

class Model:
    """A bc_model handle over device weights (dict name -> tensor) of a
    synthetic DiT-family model; keeps the tensors alive."""

    def __init__(self, desc: ModelDesc, weights: Dict[str, object], blocks: List[BlockWeights]):
        self.desc = desc
        self.weights = weights
        self._blocks = (BlockWeights * max(1, len(blocks)))(*blocks)
        mw = ModelWeights()
        for n in _MODEL_PTRS:
            setattr(mw, n, dev_ptr(weights.get(n)))
        mw.blocks = C.cast(self._blocks, C.POINTER(BlockWeights))
        self._mw = mw
        h = C.c_void_p()
        _check(lib().bc_model_create(C.byref(desc), C.byref(mw), C.byref(h)))
        self.h = h

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.bc_model_destroy(self.h)
            self.h = None

    def workspace_size(self, B: int, S: int) -> int:
        n = C.c_size_t()
        _check(lib().bc_sample_workspace_size(self.h, B, S, C.byref(n)))
        return n.value

    def blockwise_sites(self) -> int:
        n = C.c_int()
        _check(lib().bc_blockwise_sites(self.h, C.byref(n)))
        return n.value

    def adaptive_workspace_size(self, B: int, S: int) -> int:
        n = C.c_size_t()
        _check(lib().bc_sample_adaptive_workspace_size(self.h, B, S, C.byref(n)))
        return n.value


def sample(model: Model, B: int, sampler: str, mask, K: int, ring: CacheRing, latents, ws,
           labels=None, text=None, p: Optional[BaryParams] = None, stream=None):
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    _check(lib().bc_sample(model.h, B, SAMPLERS[sampler], len(m), _ptr(m), K, C.byref(p) if p else None,
                           ring.h, dev_ptr(latents), dev_ptr(labels), dev_ptr(text), dev_ptr(ws),
                           ws.numel() * ws.element_size(), stream_handle(stream)))


def sample_cfg(model: Model, B: int, sampler: str, mask, K: int, ring: CacheRing, latents, ws, labels,
               cfg_scale: float, p: Optional[BaryParams] = None, stream=None):
    """Guided sampling (bc_sample_cfg): ring slots and workspace for a model batch of 2B."""
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    _check(lib().bc_sample_cfg(model.h, B, SAMPLERS[sampler], len(m), _ptr(m), K, C.byref(p) if p else None,
                               ring.h, dev_ptr(latents), dev_ptr(labels), float(cfg_scale), dev_ptr(ws),
                               ws.numel() * ws.element_size(), stream_handle(stream)))


def sample_blockwise(model: Model, B: int, sampler: str, mask, K: int, site_storage, latents, ws, labels=None,
                     text=None, p: Optional[BaryParams] = None, stream=None):
    """Blockwise-mode sampling (bc_sample_blockwise) in place on latents."""
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    _check(lib().bc_sample_blockwise(model.h, B, SAMPLERS[sampler], len(m), _ptr(m), K, C.byref(p) if p else None,
                                     dev_ptr(site_storage), site_storage.numel() * site_storage.element_size(),
                                     dev_ptr(latents), dev_ptr(labels), dev_ptr(text),
                                     dev_ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)))


def sample_adaptive(model: Model, B: int, sampler: str, S: int, ell: float, K: int, ring: CacheRing, latents,
                    ws, labels=None, text=None, p: Optional[BaryParams] = None, stream=None):
    """Adaptive-schedule sampling (bc_sample_adaptive); returns (mask, changes)
    as numpy arrays.  Synchronises the stream at every step."""
    mask = np.zeros(S, dtype=np.uint8)
    change = np.zeros(S, dtype=np.float64)
    _check(lib().bc_sample_adaptive(model.h, B, SAMPLERS[sampler], S, float(ell), K, C.byref(p) if p else None,
                                    ring.h, dev_ptr(latents), dev_ptr(labels), dev_ptr(text), dev_ptr(ws),
                                    ws.numel() * ws.element_size(), stream_handle(stream), _ptr(mask),
                                    _ptr(change)))
    return mask, change


class SampleGraph:
    """A sampling run captured once as a HIP graph (bc_sample_graph_create);
    launch() replays it.  Every buffer the capture saw (latents, labels, text,
    workspace, ring storage, weights) must stay alive and in place."""

    def __init__(self, model: Model, B: int, sampler: str, mask, K: int, ring: CacheRing, latents, ws,
                 labels=None, text=None, p: Optional[BaryParams] = None, stream=None):
        import torch
        self.stream = stream if stream is not None else torch.cuda.Stream()
        self._keep = (model, ring, latents, ws, labels, text)
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        h = C.c_void_p()
        # The capture stream must see the caller's pending work before the run is recorded.
        self.stream.wait_stream(torch.cuda.current_stream())
        _check(lib().bc_sample_graph_create(model.h, B, SAMPLERS[sampler], len(m), _ptr(m), K,
                                            C.byref(p) if p else None, ring.h, dev_ptr(latents),
                                            dev_ptr(labels), dev_ptr(text), dev_ptr(ws),
                                            ws.numel() * ws.element_size(), self.stream.cuda_stream, C.byref(h)))
        self.h = h

    def launch(self, stream=None):
        _check(lib().bc_sample_graph_launch(self.h, stream_handle(stream)))

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.bc_sample_graph_destroy(self.h)
            self.h = None


def profile_enable(kernel_class: int, max_launches: int):
    _check(lib().bc_profile_enable(kernel_class, max_launches))


def profile_collect(kernel_class: int):
    ms, n = C.c_double(), C.c_int()
    _check(lib().bc_profile_collect(kernel_class, C.byref(ms), C.byref(n)))
    return ms.value, n.value


def profile_times(kernel_class: int, max_launches: int) -> np.ndarray:
    """Per-launch durations (ms) of an enabled class, in launch order; disables it."""
    ms = np.zeros(max_launches, np.float32)
    n = C.c_int()
    _check(lib().bc_profile_times(kernel_class, ms.ctypes.data_as(C.POINTER(C.c_float)), max_launches, C.byref(n)))
    return ms[:n.value]


def profile_records(kernel_class: int, max_launches: int):
    """(durations in ms, algorithmic work) of an enabled class's launches, in
    launch order; disables it.  Work: FLOPs (GEMM, attention) or bytes
    (forecast, LayerNorm, copy); 0 for a launch that is not the first of its
    library call."""
    ms = np.zeros(max_launches, np.float32)
    work = np.zeros(max_launches, np.float64)
    n = C.c_int()
    _check(lib().bc_profile_records(kernel_class, ms.ctypes.data_as(C.POINTER(C.c_float)),
                                    work.ctypes.data_as(C.POINTER(C.c_double)), max_launches, C.byref(n)))
    return ms[:n.value], work[:n.value]

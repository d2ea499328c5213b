"""ctypes binding of libeb.so (C ABI in include/eb_layer.h).

Argument marshalling only: torch tensors become device pointers, numpy
length arrays become host pointers, the current torch stream becomes the
hipStream_t.  Every computation runs in the library's HIP kernels.  Loading
raises if the library has not been built; nothing here falls back to another
implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libeb.so")

EB_OK = 0
STATUS = {0: "EB_OK", -1: "EB_ERR_NULL", -2: "EB_ERR_CONFIG", -3: "EB_ERR_BATCH", -4: "EB_ERR_MODE",
          -5: "EB_ERR_PAGES", -6: "EB_ERR_WORKSPACE", -7: "EB_ERR_LIMITS", -8: "EB_ERR_HIP"}
MODES = {"decode": 0, "prefill": 1, "mixed": 2}
EPILOGUES = {"store": 0, "residual": 1, "silu_mul": 2}

# every symbol include/eb_layer.h declares
SYMBOLS = ("eb_create", "eb_destroy", "eb_workspace_bytes", "eb_layer_step_decode", "eb_layer_step_prefill",
           "eb_layer_step_mixed", "eb_validate", "eb_status_str", "eb_last_error", "eb_op_rmsnorm",
           "eb_op_gemm_workspace_bytes", "eb_op_gemm", "eb_op_gemm_w8", "eb_op_moe_ffn_workspace_bytes", "eb_op_moe_ffn", "eb_op_rope_kv_append", "eb_op_attention",
           "eb_op_gather_kv", "eb_profile", "eb_profile_read", "eb_profile_stage_name", "eb_stack_workspace_bytes",
           "eb_stack_step", "eb_workspace_offset", "eb_noalloc_scratch_bytes", "eb_layer_step_mixed_noalloc",
           "eb_packed_weight_bytes", "eb_pack_weight")


class EbError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class LayerConfig(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32), ("expert_ffn", ctypes.c_int32),
                ("moe_renormalize", ctypes.c_int32), ("qk_norm", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")] + \
        [("w_dtype", ctypes.c_int32)] + [(n, ctypes.c_void_p) for n in ("s_qkv", "s_o", "s_gate_up", "s_down")] + \
        [(n, ctypes.c_void_p) for n in ("w_router", "w_experts_gate_up", "w_experts_down", "q_norm", "k_norm")] + \
        [(n, ctypes.c_void_p) for n in ("p_qkv", "p_o", "p_gate_up", "p_down")]


W_BF16, W_FP8_E4M3 = 0, 1


class KvCache(ctypes.Structure):
    _fields_ = [("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p), ("num_pages", ctypes.c_int32),
                ("block_tables", ctypes.c_void_p), ("max_pages_per_seq", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("k_scale", ctypes.c_float), ("v_scale", ctypes.c_float)]


KV_BF16, KV_FP8_E4M3 = 0, 1
_CODE_DTYPES = (torch.uint8,) + ((torch.float8_e4m3fn,) if hasattr(torch, "float8_e4m3fn") else ())


class Batch(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("context_lens_host", ctypes.c_void_p), ("chunk_lens_host", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libeb.so (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, SZ, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p
    sig = {
        "eb_create": (I32, [P(LayerConfig), I32, I32, P(VP)]),
        "eb_destroy": (None, [VP]),
        "eb_workspace_bytes": (SZ, [VP, P(Batch), I32]),
        "eb_workspace_offset": (SZ, [VP, P(Batch), I32, I32]),
        "eb_noalloc_scratch_bytes": (SZ, []),
        "eb_layer_step_mixed_noalloc": (I32, [VP, P(LayerWeights), P(KvCache), P(Batch), VP, VP, VP]),
        "eb_validate": (I32, [P(LayerConfig), P(Batch), VP, I32, I32, I32]),
        "eb_status_str": (ctypes.c_char_p, [I32]),
        "eb_last_error": (ctypes.c_char_p, []),
        "eb_op_rmsnorm": (I32, [VP, VP, VP, VP, I32, VP]),
        "eb_op_gemm_workspace_bytes": (SZ, [I32, I32, I32]),
        "eb_op_gemm": (I32, [VP, VP, VP, VP, I32, I32, I32, I32, VP, SZ, VP]),
        "eb_op_gemm_w8": (I32, [VP, VP, VP, VP, VP, I32, I32, I32, I32, VP, SZ, VP]),
        "eb_packed_weight_bytes": (SZ, [ctypes.c_int, ctypes.c_int]),
        "eb_pack_weight": (I32, [VP, VP, ctypes.c_int, ctypes.c_int, VP]),
        "eb_op_moe_ffn_workspace_bytes": (SZ, [I32, I32, I32, I32, I32]),
        "eb_op_moe_ffn": (I32, [VP, VP, VP, VP, VP, I32, I32, I32, I32, I32, I32, VP, VP, VP, VP, SZ, VP]),
        "eb_op_rope_kv_append": (I32, [VP, VP, P(KvCache), P(Batch), VP, SZ, VP]),
        "eb_op_attention": (I32, [VP, VP, P(KvCache), P(Batch), VP, VP, SZ, I32, VP]),
        "eb_op_gather_kv": (I32, [VP, P(KvCache), P(Batch), VP, VP, VP, SZ, VP]),
        "eb_profile": (I32, [VP, I32, ctypes.c_uint32]),
        "eb_profile_read": (I32, [VP, P(ctypes.c_float), I32]),
        "eb_profile_stage_name": (ctypes.c_char_p, [I32]),
        "eb_stack_workspace_bytes": (SZ, [VP, P(Batch), I32]),
        "eb_stack_step": (I32, [VP, I32, I32, P(LayerWeights), P(KvCache), P(Batch), VP, VP, VP, SZ, VP]),
    }
    for name in ("eb_layer_step_decode", "eb_layer_step_prefill", "eb_layer_step_mixed"):
        sig[name] = (I32, [VP, P(LayerWeights), P(KvCache), P(Batch), VP, VP, VP, SZ, VP])
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(status: int):
    if status != EB_OK:
        raise EbError(status, lib().eb_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def config_of(shape) -> LayerConfig:
    """LayerConfig from any object with the layer-shape attributes."""
    return LayerConfig(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn,
                       getattr(shape, "page_size", 16), float(shape.rms_eps), float(shape.rope_theta),
                       getattr(shape, "n_experts", 0), getattr(shape, "top_k", 0), getattr(shape, "expert_ffn", 0),
                       1 if getattr(shape, "moe_renormalize", True) else 0, 1 if getattr(shape, "qk_norm", False) else 0)


class HostBatch:
    """Holds the host int32 length arrays alive for the duration of a call."""

    def __init__(self, context_lens, chunk_lens):
        self.ctx = np.ascontiguousarray(context_lens, dtype=np.int32)
        self.chk = np.ascontiguousarray(chunk_lens, dtype=np.int32)
        self.c = Batch(len(self.ctx), int(self.chk.sum()), self.ctx.ctypes.data, self.chk.ctypes.data)


def kv_struct(k_cache: torch.Tensor, v_cache: torch.Tensor, block_tables: torch.Tensor,
              kv_scales=None) -> KvCache:
    """bf16 caches, or 8-bit E4M3 code caches (uint8 / float8_e4m3fn) with
    kv_scales = (k_scale, v_scale)."""
    assert block_tables.dtype == torch.int32 and block_tables.dim() == 2
    assert k_cache.dtype == v_cache.dtype
    if k_cache.dtype in _CODE_DTYPES:
        if kv_scales is None:
            raise ValueError("an 8-bit cache needs kv_scales = (k_scale, v_scale)")
        return KvCache(_ptr(k_cache), _ptr(v_cache), int(k_cache.shape[0]), _ptr(block_tables),
                       int(block_tables.shape[1]), KV_FP8_E4M3, float(kv_scales[0]), float(kv_scales[1]))
    assert k_cache.dtype == torch.bfloat16
    return KvCache(_ptr(k_cache), _ptr(v_cache), int(k_cache.shape[0]), _ptr(block_tables),
                   int(block_tables.shape[1]), KV_BF16, 1.0, 1.0)


def weights_struct(w: dict) -> LayerWeights:
    """Weights dict -> struct: bf16 projections, or uint8 / float8_e4m3fn
    codes with float32 row scales under s_qkv, s_o, s_gate_up, s_down;
    a mixture-of-experts layer brings w_router, w_experts_gate_up and
    w_experts_down instead of w_gate_up and w_down; a layer with q/k norms
    brings their gains under q_norm and k_norm; fragment-packed copies of
    the bf16 projections (eb_pack_weight) go under p_qkv, p_o, p_gate_up,
    p_down."""
    lw = LayerWeights(*[_ptr(w.get(k)) for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")])
    for k in ("w_router", "w_experts_gate_up", "w_experts_down", "q_norm", "k_norm", "p_qkv", "p_o", "p_gate_up",
              "p_down"):
        if k in w:
            setattr(lw, k, _ptr(w[k]))
    if w["w_qkv"].dtype in _CODE_DTYPES:
        lw.w_dtype = W_FP8_E4M3
        for k in ("s_qkv", "s_o", "s_gate_up", "s_down"):
            if w[k].dtype != torch.float32 or not w[k].is_contiguous():
                raise ValueError(f"{k} must be contiguous float32")
            setattr(lw, k, _ptr(w[k]))
    return lw


class Handle:
    """eb_create / eb_destroy."""

    def __init__(self, shape, max_seqs: int, max_tokens: int):
        self.shape = shape
        self.cfg = config_of(shape)
        h = ctypes.c_void_p()
        _check(lib().eb_create(ctypes.byref(self.cfg), int(max_seqs), int(max_tokens), ctypes.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            lib().eb_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def eb_workspace_bytes(h: Handle, context_lens, chunk_lens, mode: str) -> int:
    hb = HostBatch(context_lens, chunk_lens)
    return int(lib().eb_workspace_bytes(h.h, ctypes.byref(hb.c), MODES[mode]))


WS_BUFFERS = {"qkv": 0, "attn": 1, "h1": 2, "mlp": 3, "norm": 4}


def eb_workspace_offset(h: Handle, context_lens, chunk_lens, mode: str, which: str) -> int:
    """Byte offset of an intermediate buffer inside a step's workspace (-1:
    none)."""
    hb = HostBatch(context_lens, chunk_lens)
    off = int(lib().eb_workspace_offset(h.h, ctypes.byref(hb.c), MODES[mode], WS_BUFFERS[which]))
    return -1 if off == (1 << 64) - 1 else off


def workspace_intermediates(h: Handle, ws: torch.Tensor, context_lens, chunk_lens, mode: str) -> dict:
    """Views of the intermediate buffers a layer step left in ``ws``: bf16
    qkv [T, (nq + 2 nkv) hd] (q normalised and rotated in place), attn
    [T, nq hd], h1 [T, d], mlp [T, ffn] (dense layers), norm [T, d]."""
    s = h.shape
    T = int(np.asarray(chunk_lens).sum())
    cols = {"qkv": (s.n_q_heads + 2 * s.n_kv_heads) * s.head_dim, "attn": s.n_q_heads * s.head_dim,
            "h1": s.hidden, "mlp": s.ffn, "norm": s.hidden}
    out = {}
    for name, c in cols.items():
        off = eb_workspace_offset(h, context_lens, chunk_lens, mode, name)
        if off < 0:
            continue
        out[name] = ws[off:off + T * c * 2].view(torch.bfloat16).view(T, c)
    return out


def alloc_workspace(nbytes: int, device="cuda") -> torch.Tensor:
    # torch's caching allocator returns 256-byte (or better) aligned blocks
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _step(name, h: Handle, weights: dict, k_cache, v_cache, block_tables, context_lens, chunk_lens,
          x: torch.Tensor, y: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, stream=None,
          kv_scales=None):
    hb = HostBatch(context_lens, chunk_lens)
    mode = {"eb_layer_step_decode": "decode", "eb_layer_step_prefill": "prefill",
            "eb_layer_step_mixed": "mixed"}[name]
    if y is None:
        y = torch.empty_like(x)
    if ws is None:
        ws = alloc_workspace(lib().eb_workspace_bytes(h.h, ctypes.byref(hb.c), MODES[mode]), x.device)
    kv = kv_struct(k_cache, v_cache, block_tables, kv_scales)
    w = weights_struct(weights)
    _check(getattr(lib(), name)(h.h, ctypes.byref(w), ctypes.byref(kv), ctypes.byref(hb.c), _ptr(x), _ptr(y),
                                _ptr(ws), ws.numel(), _stream(stream)))
    return y


def eb_layer_step_decode(h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x, y=None, ws=None,
                         stream=None, kv_scales=None):
    return _step("eb_layer_step_decode", h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x,
                 y, ws, stream, kv_scales)


def eb_layer_step_prefill(h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x, y=None, ws=None,
                          stream=None, kv_scales=None):
    return _step("eb_layer_step_prefill", h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x,
                 y, ws, stream, kv_scales)


def eb_layer_step_mixed(h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x, y=None, ws=None,
                        stream=None, kv_scales=None):
    return _step("eb_layer_step_mixed", h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x,
                 y, ws, stream, kv_scales)


def eb_noalloc_scratch_bytes() -> int:
    return int(lib().eb_noalloc_scratch_bytes())


def eb_layer_step_mixed_noalloc(h, weights, k_cache, v_cache, block_tables, context_lens, chunk_lens, x, y=None,
                                stream=None, kv_scales=None):
    """The mixed step on the library's fixed scratch (no workspace argument;
    y must be given by callers that cannot allocate)."""
    hb = HostBatch(context_lens, chunk_lens)
    if y is None:
        y = torch.empty_like(x)
    kv = kv_struct(k_cache, v_cache, block_tables, kv_scales)
    w = weights_struct(weights)
    _check(lib().eb_layer_step_mixed_noalloc(h.h, ctypes.byref(w), ctypes.byref(kv), ctypes.byref(hb.c), _ptr(x),
                                             _ptr(y), _stream(stream)))
    return y


def eb_stack_workspace_bytes(h: Handle, context_lens, chunk_lens, mode: str) -> int:
    hb = HostBatch(context_lens, chunk_lens)
    return int(lib().eb_stack_workspace_bytes(h.h, ctypes.byref(hb.c), MODES[mode]))


def eb_stack_step(h: Handle, mode: str, weights: list, caches: list, context_lens, chunk_lens, x: torch.Tensor,
                  y: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, stream=None):
    """n = len(weights) layers; caches[l] = (k_cache, v_cache, block_tables)
    of layer l, plus (k_scale, v_scale) for an 8-bit cache (entries may
    repeat the same tensors)."""
    n = len(weights)
    if len(caches) != n:
        raise ValueError("one cache entry per layer")
    hb = HostBatch(context_lens, chunk_lens)
    if y is None:
        y = torch.empty_like(x)
    if ws is None:
        ws = alloc_workspace(lib().eb_stack_workspace_bytes(h.h, ctypes.byref(hb.c), MODES[mode]), x.device)
    ws_arr = (LayerWeights * n)(*[weights_struct(w) for w in weights])
    kv_arr = (KvCache * n)(*[kv_struct(*c) for c in caches])
    _check(lib().eb_stack_step(h.h, MODES[mode], n, ws_arr, kv_arr, ctypes.byref(hb.c), _ptr(x), _ptr(y), _ptr(ws),
                               ws.numel(), _stream(stream)))
    return y


def eb_validate(shape, context_lens, chunk_lens, block_tables_host: np.ndarray, num_pages: int, mode: str) -> int:
    """Host-only validation; returns the status code (0 = EB_OK)."""
    cfg = config_of(shape)
    hb = HostBatch(context_lens, chunk_lens)
    bt = np.ascontiguousarray(block_tables_host, dtype=np.int32)
    mp = bt.shape[1] if bt.ndim == 2 else 0
    return int(lib().eb_validate(ctypes.byref(cfg), ctypes.byref(hb.c), bt.ctypes.data if bt.size else None,
                                 int(num_pages), int(mp), MODES.get(mode, mode) if isinstance(mode, str) else mode))


def eb_last_error() -> str:
    return lib().eb_last_error().decode()


def eb_status_str(status: int) -> str:
    return lib().eb_status_str(int(status)).decode()


def eb_op_rmsnorm(h: Handle, x: torch.Tensor, gamma: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    out = torch.empty_like(x) if out is None else out
    _check(lib().eb_op_rmsnorm(h.h, _ptr(x), _ptr(gamma), _ptr(out), int(x.shape[0]), _stream(stream)))
    return out


def eb_op_gemm(A: torch.Tensor, W: torch.Tensor, epilogue: str = "store", residual: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None, stream=None):
    M, K = A.shape
    N = W.shape[0]
    ncol = N // 2 if epilogue == "silu_mul" else N
    out = torch.empty(M, ncol, dtype=torch.bfloat16, device=A.device) if out is None else out
    nb = int(lib().eb_op_gemm_workspace_bytes(M, N, K))
    ws = alloc_workspace(nb, A.device)
    _check(lib().eb_op_gemm(_ptr(A), _ptr(W), _ptr(out), _ptr(residual), M, N, K, EPILOGUES[epilogue], _ptr(ws),
                            ws.numel(), _stream(stream)))
    return out


def eb_packed_weight_bytes(rows: int, cols: int) -> int:
    return int(lib().eb_packed_weight_bytes(rows, cols))


def eb_pack_weight(W: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Fragment-packed copy of a bf16 [rows, cols] weight matrix (a flat
    bf16 tensor of rows * cols elements)."""
    if W.dtype != torch.bfloat16 or W.dim() != 2:
        raise ValueError("W must be a 2-D bf16 tensor")
    rows, cols = W.shape
    out = torch.empty(rows * cols, dtype=torch.bfloat16, device=W.device) if out is None else out
    if out.numel() * 2 < eb_packed_weight_bytes(rows, cols):
        raise ValueError("out is smaller than the packed copy")
    _check(lib().eb_pack_weight(_ptr(W), _ptr(out), rows, cols, _stream(stream)))
    return out


def pack_layer_weights(w: dict, stream=None) -> dict:
    """The weights dict plus packed copies of its bf16 projections (those
    whose shape has a packed form)."""
    out = dict(w)
    if w.get("w_qkv") is None or w["w_qkv"].dtype != torch.bfloat16:
        return out
    for src, dst in (("w_qkv", "p_qkv"), ("w_o", "p_o"), ("w_gate_up", "p_gate_up"), ("w_down", "p_down")):
        t = w.get(src)
        if t is not None and eb_packed_weight_bytes(*t.shape) > 0:
            out[dst] = eb_pack_weight(t, stream=stream)
    return out


def eb_op_gemm_w8(A: torch.Tensor, W: torch.Tensor, w_scale: torch.Tensor, epilogue: str = "store",
                  residual: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None, stream=None):
    """W: uint8 E4M3 codes [N, K]; w_scale: float32 [N], one scale per row."""
    if W.dtype not in _CODE_DTYPES or w_scale.dtype != torch.float32 or not w_scale.is_contiguous():
        raise TypeError("W must hold uint8 codes and w_scale contiguous float32 row scales")
    M, K = A.shape
    N = W.shape[0]
    if w_scale.numel() != N:
        raise ValueError("w_scale needs one scale per row of W")
    ncol = N // 2 if epilogue == "silu_mul" else N
    out = torch.empty(M, ncol, dtype=torch.bfloat16, device=A.device) if out is None else out
    nb = int(lib().eb_op_gemm_workspace_bytes(M, N, K))
    ws = alloc_workspace(nb, A.device)
    _check(lib().eb_op_gemm_w8(_ptr(A), _ptr(W), _ptr(w_scale), _ptr(out), _ptr(residual), M, N, K,
                               EPILOGUES[epilogue], _ptr(ws), ws.numel(), _stream(stream)))
    return out


def eb_op_moe_ffn(b: torch.Tensor, w_router: torch.Tensor, w_gate_up: torch.Tensor, w_down: torch.Tensor,
                  top_k: int, residual: Optional[torch.Tensor] = None, renormalize: bool = True,
                  out: Optional[torch.Tensor] = None, return_routing: bool = False,
                  ws: Optional[torch.Tensor] = None, stream=None):
    """MoE feed-forward block: b [T, d], w_router [E, d], w_gate_up [E, 2F, d],
    w_down [E, d, F], all bf16; returns out [T, d] (and the int32 expert ids
    and fp32 weights [T, top_k] with ``return_routing``)."""
    for t in (b, w_router, w_gate_up, w_down) + ((residual,) if residual is not None else ()):
        if t.dtype != torch.bfloat16 or not t.is_contiguous():
            raise TypeError("MoE operands must be contiguous bf16")
    T, d = b.shape
    E = w_router.shape[0]
    F = w_gate_up.shape[1] // 2
    if w_router.shape != (E, d) or w_gate_up.shape != (E, 2 * F, d) or w_down.shape != (E, d, F):
        raise ValueError("MoE weight shapes do not match")
    out = torch.empty(T, d, dtype=torch.bfloat16, device=b.device) if out is None else out
    ids = torch.empty(T, top_k, dtype=torch.int32, device=b.device) if return_routing else None
    wts = torch.empty(T, top_k, dtype=torch.float32, device=b.device) if return_routing else None
    if ws is None:
        ws = alloc_workspace(int(lib().eb_op_moe_ffn_workspace_bytes(T, d, E, top_k, F)), b.device)
    _check(lib().eb_op_moe_ffn(_ptr(b), _ptr(residual), _ptr(w_router), _ptr(w_gate_up), _ptr(w_down), T, d, E,
                               int(top_k), F, 1 if renormalize else 0, _ptr(out), _ptr(ids), _ptr(wts), _ptr(ws),
                               ws.numel(), _stream(stream)))
    return (out, ids, wts) if return_routing else out


def _op_ws(h, hb, mode="mixed", device="cuda"):
    return alloc_workspace(lib().eb_workspace_bytes(h.h, ctypes.byref(hb.c), MODES[mode]), device)


def eb_op_rope_kv_append(h: Handle, qkv: torch.Tensor, k_cache, v_cache, block_tables, context_lens, chunk_lens,
                         stream=None, kv_scales=None):
    hb = HostBatch(context_lens, chunk_lens)
    ws = _op_ws(h, hb, device=qkv.device)
    kv = kv_struct(k_cache, v_cache, block_tables, kv_scales)
    _check(lib().eb_op_rope_kv_append(h.h, _ptr(qkv), ctypes.byref(kv), ctypes.byref(hb.c), _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return qkv


def eb_op_attention(h: Handle, qkv: torch.Tensor, k_cache, v_cache, block_tables, context_lens, chunk_lens,
                    mode: str = "mixed", out: Optional[torch.Tensor] = None, stream=None, kv_scales=None):
    hb = HostBatch(context_lens, chunk_lens)
    s = h.shape
    T = int(hb.chk.sum())
    out = torch.empty(T, s.n_q_heads * s.head_dim, dtype=torch.bfloat16, device=qkv.device) if out is None else out
    ws = _op_ws(h, hb, mode if mode in MODES else "mixed", qkv.device)
    kv = kv_struct(k_cache, v_cache, block_tables, kv_scales)
    _check(lib().eb_op_attention(h.h, _ptr(qkv), ctypes.byref(kv), ctypes.byref(hb.c), _ptr(out), _ptr(ws),
                                 ws.numel(), MODES[mode], _stream(stream)))
    return out


def eb_op_gather_kv(h: Handle, k_cache, v_cache, block_tables, context_lens, chunk_lens, stream=None,
                    kv_scales=None):
    """Dense copies of every cached position (raw elements: bf16, or the
    8-bit codes of an 8-bit cache)."""
    hb = HostBatch(context_lens, chunk_lens)
    s = h.shape
    total = int((hb.ctx.astype(np.int64) + hb.chk).sum())
    ok = torch.empty(total, s.n_kv_heads, s.head_dim, dtype=k_cache.dtype, device=k_cache.device)
    ov = torch.empty_like(ok)
    ws = _op_ws(h, hb, device=k_cache.device)
    kv = kv_struct(k_cache, v_cache, block_tables, kv_scales if kv_scales is not None else (1.0, 1.0))
    _check(lib().eb_op_gather_kv(h.h, ctypes.byref(kv), ctypes.byref(hb.c), _ptr(ok), _ptr(ov), _ptr(ws), ws.numel(),
                                 _stream(stream)))
    return ok, ov


def eb_profile(h: Handle, enable: bool = True, steps: int = 1, stages=None):
    """Record the stage events of the following steps (a ring of `steps`
    slots; `stages`: names of the stages to bracket, all if None), or stop
    recording."""
    mask = 0
    if stages is not None:
        names = [lib().eb_profile_stage_name(i).decode() for i in range(32) if lib().eb_profile_stage_name(i)]
        for n in stages:
            mask |= 1 << names.index(n)
    _check(lib().eb_profile(h.h, int(steps) if enable else 0, mask))


def eb_profile_read(h: Handle) -> dict:
    """Stage name -> ms, averaged over the recorded steps on this handle."""
    buf = (ctypes.c_float * 32)()
    n = lib().eb_profile_read(h.h, buf, 32)
    if n < 0:
        raise EbError(-8, "eb_profile_read failed")
    return {lib().eb_profile_stage_name(i).decode(): float(buf[i]) for i in range(n)}

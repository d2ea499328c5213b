"""Plain CPU definition of one decoder-layer step over a paged-KV token batch.

TEST INFRASTRUCTURE ONLY: only tests, the package smoke check and the
benchmark's CPU-baseline leg call this.  It shares no code with the HIP path.

What is computed.  The paper's scheduling model prices one iteration of the
serving loop, T_iter = alpha + beta * n_tok, over a batch whose rows are
prefill chunks and decode tokens (Sec. 1; Sec. 3.1 "Timing Model"); its
engine runs every model in BF16 with paged attention left unchanged
(Sec. 4.1 "Implementation").  The decode context of a request is the number of
tokens already in its KV cache, all of which a decode token streams during
attention (App. A.2, "Effect of decode context length").  The paper does not
write the layer itself down, so this module writes out the standard pre-norm
Llama decoder layer that the workloads name (RMSNorm, GQA, RoPE, SwiGLU):

  a   = RMSNorm(x) * g1
  q,k,v = a Wq^T, a Wk^T, a Wv^T;  q,k rotated by RoPE at pos = c_i + j
  K/V of the new rows are rounded to bf16 and appended to the paged cache
  o_h = softmax(q_h K^T / sqrt(hd)) V  over keys 0..pos of kv head h // G
  h1  = x + concat(o) Wo^T
  m   = SiLU(RMSNorm(h1) * g2 Wg^T) * (RMSNorm(h1) * g2 Wu^T)
  y   = h1 + m Wd^T

Arithmetic runs in float32 (selectable float64 for the self-checks); the only
rounding to bf16 is the cache write, because the attention of the same step
reads the appended keys and values back from the cache.

Parity pins (tests/test_oracle.py): brute-force dense attention in fp64 and
torch's scaled_dot_product_attention; the transformers Llama decoder layer in
fp64; closed forms (c=0 single token, equal keys, RoPE identities, RMSNorm
scale invariance); softmax sums; causal, batch and page-relabelling
invariances.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

from . import fp8


@dataclasses.dataclass(frozen=True)
class LayerCfg:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    page_size: int = 16
    rms_eps: float = 1e-5
    rope_theta: float = 1e4
    n_experts: int = 0          # > 0: mixture-of-experts feed-forward (oracle/moe.py)
    top_k: int = 0
    expert_ffn: int = 0
    moe_renormalize: bool = True
    qk_norm: bool = False       # RMSNorm of every q and k head (gains q_norm, k_norm) before RoPE

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


# ----------------------------------------------------------------------------
# bf16 storage format
# ----------------------------------------------------------------------------

def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32, exactly (bf16 is the top half of fp32)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bits with round-to-nearest-even; NaN -> quiet NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r[np.isnan(x)] = 0x7FC0
    return r


# ----------------------------------------------------------------------------
# elementwise pieces
# ----------------------------------------------------------------------------

def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gamma along the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + x.dtype.type(eps)) * gamma


def rope(u: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing (t, t + hd/2), freq theta^(-2t/hd).

    u: [..., heads, hd] with a leading row axis matching ``pos`` (scalar or
    [rows]).  Angles are formed in float64 and their cos/sin cast to the
    working precision.
    """
    hd = u.shape[-1]
    half = hd // 2
    t = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * t / hd)
    pos = np.asarray(pos, dtype=np.float64)
    ang = pos[..., None] * inv_freq                      # [rows, half] or [half]
    cos = np.cos(ang).astype(u.dtype)
    sin = np.sin(ang).astype(u.dtype)
    if pos.ndim == 1:                                   # broadcast over heads
        cos = cos[:, None, :]
        sin = sin[:, None, :]
    a, b = u[..., :half], u[..., half:]
    return np.concatenate([a * cos - b * sin, a * sin + b * cos], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (z.dtype.type(1) + np.exp(-z))


# ----------------------------------------------------------------------------
# paged KV
# ----------------------------------------------------------------------------

def gather_positions(cache_bits: np.ndarray, bt_row: np.ndarray, npos: int, page: int,
                     dtype=np.float32, scale: Optional[float] = None) -> np.ndarray:
    """Positions 0..npos-1 of one request from the paged cache.

    cache_bits: [num_pages, n_kv, page, hd] bf16 bits, or 8-bit E4M3 codes
    when ``scale`` is given (values decode(code) * scale).  Logical position
    p of the request lives in physical page bt_row[p // page], slot p % page.
    Returns [npos, n_kv, hd].
    """
    p = np.arange(npos)
    phys = np.asarray(bt_row)[p // page]
    slot = p % page
    if scale is not None:
        return fp8.dequantize(cache_bits[phys, :, slot, :], scale).astype(dtype)
    return bf16_bits_to_f32(cache_bits[phys, :, slot, :]).astype(dtype)


def append_kv(cache_bits: np.ndarray, bt_row: np.ndarray, positions: np.ndarray, vals: np.ndarray,
              page: int, scale: Optional[float] = None) -> None:
    """Write vals [rows, n_kv, hd] (rounded to bf16) at the given positions;
    with ``scale``, the cache holds 8-bit codes of the bf16 values divided by
    the scale."""
    positions = np.asarray(positions)
    phys = np.asarray(bt_row)[positions // page]
    b = f32_to_bf16_bits(vals.astype(np.float32))
    if scale is not None:
        cache_bits[phys, :, positions % page, :] = fp8.quantize_cache_value(bf16_bits_to_f32(b), scale)
    else:
        cache_bits[phys, :, positions % page, :] = b


def attend_one(q: np.ndarray, keys: np.ndarray, vals: np.ndarray) -> np.ndarray:
    """softmax(q . k_t / sqrt(hd)) weighted sum of v_t for one query vector."""
    hd = q.shape[-1]
    s = keys @ q / q.dtype.type(np.sqrt(hd))
    s = s - s.max()
    p = np.exp(s)
    p = p / p.sum()
    return p @ vals


def paged_attention_row(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray, bt_row: np.ndarray,
                        pos: int, page: int, group: int, kv_scales=None) -> np.ndarray:
    """Attention of one query row at position pos over keys 0..pos.

    q: [n_q, hd].  Query head h reads kv head h // group.  Returns [n_q, hd].
    """
    ks, vs = kv_scales if kv_scales is not None else (None, None)
    K = gather_positions(k_cache, bt_row, pos + 1, page, q.dtype, ks)
    V = gather_positions(v_cache, bt_row, pos + 1, page, q.dtype, vs)
    out = np.empty_like(q)
    for h in range(q.shape[0]):
        g = h // group
        out[h] = attend_one(q[h], K[:, g, :], V[:, g, :])
    return out


def causal_attention_seq(q: np.ndarray, K: np.ndarray, V: np.ndarray, positions: np.ndarray,
                         group: int) -> np.ndarray:
    """Batched form for one request: q [n, n_q, hd], K/V [L, n_kv, hd].

    Row j (position positions[j]) sees keys t <= positions[j]; masked scores
    get probability exactly zero.  Returns [n, n_q, hd].
    """
    n, nq, hd = q.shape
    L = K.shape[0]
    out = np.empty_like(q)
    visible = np.arange(L)[None, :] <= np.asarray(positions)[:, None]         # [n, L]
    scale = q.dtype.type(1.0 / np.sqrt(hd))
    for h in range(nq):
        g = h // group
        s = (q[:, h, :] @ K[:, g, :].T) * scale                              # [n, L]
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ V[:, g, :]
    return out


# ----------------------------------------------------------------------------
# the layer step
# ----------------------------------------------------------------------------

def prepare_weights(w_bits: Dict[str, np.ndarray], cfg: LayerCfg, dtype=np.float32) -> dict:
    """bf16 weight bits -> working-precision arrays, split into named parts.

    w_qkv rows: q heads, k heads, v heads; w_gate_up rows: gate then up.
    A projection given as 8-bit E4M3 codes (uint8) comes with its per-row
    scales under "s_" + the name without "w_" (s_qkv, s_o, s_gate_up,
    s_down): its weights are decode(code) * scale of the row, formed in
    float64.  The norm gains are always bf16 (q_norm, k_norm [head_dim]
    when cfg.qk_norm).
    """
    nq, nkv, hd, f = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn

    def cv(k):
        w = w_bits[k]
        if w.dtype == np.uint8:
            return fp8.dequantize_rows(w, w_bits["s_" + k[2:]]).astype(dtype)
        return bf16_bits_to_f32(w).astype(dtype)
    qkv = cv("w_qkv")
    W = {"g1": cv("attn_norm"), "g2": cv("mlp_norm"),
         "wq": qkv[: nq * hd], "wk": qkv[nq * hd: (nq + nkv) * hd], "wv": qkv[(nq + nkv) * hd:], "wo": cv("w_o")}
    if cfg.qk_norm:
        W["gq"], W["gk"] = cv("q_norm"), cv("k_norm")
    if cfg.n_experts:
        # the MoE block works from the bf16 weights themselves
        W["moe"] = (w_bits["w_router"], w_bits["w_experts_gate_up"], w_bits["w_experts_down"])
        return W
    gu = cv("w_gate_up")
    W.update({"wg": gu[:f], "wu": gu[f:], "wd": cv("w_down")})
    return W


def feed_forward(cfg: LayerCfg, W: dict, h1: np.ndarray):
    """(y, m): y = h1 + FFN(RMSNorm(h1) * g2) for rows h1 [n, d] (or one row
    [d]).  Dense: m = SiLU(b Wg^T) * (b Wu^T), y = h1 + m Wd^T.  Mixture of
    experts: the block of oracle/moe.py on b rounded to bf16 (the input the
    layer hands the block), m = None."""
    b = rmsnorm(h1, W["g2"], cfg.rms_eps)
    if cfg.n_experts:
        from . import moe
        rows = np.atleast_2d(b)
        y = moe.moe_ffn(f32_to_bf16_bits(rows.astype(np.float32)), *W["moe"], cfg.top_k, cfg.moe_renormalize)
        return h1 + y.reshape(h1.shape).astype(h1.dtype), None
    m = silu(b @ W["wg"].T) * (b @ W["wu"].T)
    return h1 + m @ W["wd"].T, m


def layer_step(cfg: LayerCfg, W: dict, k_cache: np.ndarray, v_cache: np.ndarray,
               block_tables: np.ndarray, context_lens: Sequence[int], chunk_lens: Sequence[int],
               x_bits: np.ndarray, mode: str = "batched", seqs: Optional[Sequence[int]] = None,
               intermediates: bool = False, kv_scales: Optional[Tuple[float, float]] = None):
    """One decoder-layer step.  Mutates k_cache / v_cache (bf16 bits, or
    8-bit E4M3 codes when kv_scales = (k_scale, v_scale) is given) in place.

    Rows of request i are x rows off_i .. off_i + n_i - 1 (off = exclusive
    prefix sum of chunk_lens) at positions c_i .. c_i + n_i - 1.  ``seqs``
    restricts the work to some requests (requests share no pages, so a subset
    yields the same rows as the whole batch); other rows of y are NaN.

    mode 'exact': one row at a time with matrix-vector products, rows of a
    request in order (append the row's K/V, then attend).  mode 'batched': the
    same definition with one matrix product per request and an explicit
    causal mask.  With cfg.qk_norm every q and k head is RMS-normalised
    over its head_dim values and scaled by its gain before RoPE (the Qwen3
    attention block).  Returns y [T, hidden] and, if asked, a dict of the
    intermediates q, k, v (after RoPE), attn, h1, m.
    """
    ks, vs = kv_scales if kv_scales is not None else (None, None)
    dtype = W["wq"].dtype
    nq, nkv, hd, G, P = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.group, cfg.page_size
    ctx = np.asarray(context_lens, np.int64)
    chk = np.asarray(chunk_lens, np.int64)
    off = np.concatenate([[0], np.cumsum(chk)])
    T = int(off[-1])
    x = bf16_bits_to_f32(x_bits).astype(dtype)
    y = np.full((T, cfg.hidden), np.nan, dtype=dtype)
    inter = {k: np.full((T,) + s, np.nan, dtype=dtype) for k, s in
             (("q", (nq, hd)), ("k", (nkv, hd)), ("v", (nkv, hd)), ("attn", (nq * hd,)),
              ("h1", (cfg.hidden,)), ("m", (cfg.ffn,)))} if intermediates else None
    todo = range(len(ctx)) if seqs is None else seqs

    def head_norm(u, gain):
        return rmsnorm(u, W[gain], cfg.rms_eps) if cfg.qk_norm else u
    for i in todo:
        r0, n, c = int(off[i]), int(chk[i]), int(ctx[i])
        bt = block_tables[i]
        if mode == "exact":
            for j in range(n):
                r, pos = r0 + j, c + j
                a = rmsnorm(x[r], W["g1"], cfg.rms_eps)
                q = rope(head_norm((W["wq"] @ a).reshape(nq, hd), "gq"), pos, cfg.rope_theta)
                k = rope(head_norm((W["wk"] @ a).reshape(nkv, hd), "gk"), pos, cfg.rope_theta)
                v = (W["wv"] @ a).reshape(nkv, hd)
                append_kv(k_cache, bt, np.array([pos]), k[None], P, ks)
                append_kv(v_cache, bt, np.array([pos]), v[None], P, vs)
                o = paged_attention_row(q, k_cache, v_cache, bt, pos, P, G, kv_scales).reshape(-1)
                h1 = x[r] + W["wo"] @ o
                y[r], m = feed_forward(cfg, W, h1)
                if inter is not None:
                    for key, val in (("q", q), ("k", k), ("v", v), ("attn", o), ("h1", h1), ("m", m)):
                        if val is not None:
                            inter[key][r] = val
        elif mode == "batched":
            rows = slice(r0, r0 + n)
            pos = c + np.arange(n)
            a = rmsnorm(x[rows], W["g1"], cfg.rms_eps)
            q = rope(head_norm((a @ W["wq"].T).reshape(n, nq, hd), "gq"), pos, cfg.rope_theta)
            k = rope(head_norm((a @ W["wk"].T).reshape(n, nkv, hd), "gk"), pos, cfg.rope_theta)
            v = (a @ W["wv"].T).reshape(n, nkv, hd)
            append_kv(k_cache, bt, pos, k, P, ks)
            append_kv(v_cache, bt, pos, v, P, vs)
            K = gather_positions(k_cache, bt, c + n, P, dtype, ks)
            V = gather_positions(v_cache, bt, c + n, P, dtype, vs)
            o = causal_attention_seq(q, K, V, pos, G).reshape(n, nq * hd)
            h1 = x[rows] + o @ W["wo"].T
            y[rows], m = feed_forward(cfg, W, h1)
            if inter is not None:
                for key, val in (("q", q), ("k", k), ("v", v), ("attn", o), ("h1", h1), ("m", m)):
                    if val is not None:
                        inter[key][rows] = val
        else:
            raise ValueError(mode)
    return (y, inter) if intermediates else y


def stack_step(cfg: LayerCfg, Ws: Sequence[dict], k_caches: Sequence[np.ndarray], v_caches: Sequence[np.ndarray],
               block_tables: Sequence[np.ndarray], context_lens: Sequence[int], chunk_lens: Sequence[int],
               x_bits: np.ndarray, mode: str = "batched", seqs: Optional[Sequence[int]] = None,
               kv_scales: Optional[Sequence[Tuple[float, float]]] = None) -> np.ndarray:
    """A model step: the layers one after another over the same batch.

    The paper's iteration is a pass of the whole model over the batch
    (Sec. 1; Sec. 3.1 "Timing Model"); every layer sees the same requests at
    the same positions.  Layer l takes the previous layer's output as bf16
    (the layer interface carries bf16 activations), appends into its own
    cache (k_caches[l], v_caches[l], mutated in place; entries may be the
    same arrays, in which case each layer overwrites the new slots in turn)
    and the last layer's output is returned in working precision.  With
    kv_scales[l] the caches of layer l hold 8-bit codes.
    """
    xb = x_bits
    y = None
    for l, W in enumerate(Ws):
        y = layer_step(cfg, W, k_caches[l], v_caches[l], block_tables[l], context_lens, chunk_lens, xb,
                       mode=mode, seqs=seqs, kv_scales=None if kv_scales is None else kv_scales[l])
        if l + 1 < len(Ws):
            xb = f32_to_bf16_bits(y.astype(np.float32))
    return y

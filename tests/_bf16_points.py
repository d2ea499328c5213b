"""CPU model of where the HIP layer step rounds to bf16, for error budgets.

The oracle stays in fp32 apart from the cache write.  The HIP step keeps
bf16 tensors between its stages: a = RMSNorm(x) g1, the q/k/v projection
output, q after RoPE, the probabilities entering the P.V product, the
attention output, h1, b = RMSNorm(h1) g2, m and y.  This module runs the
same layer definition with those roundings (and only those), so a test can
measure how far bf16 intermediates alone move the result for a given input
distribution, before it fixes a tolerance against the fp32 oracle.  It is a
test helper: the oracle does not use it and it shares nothing with the HIP
path.
"""
from __future__ import annotations

import numpy as np

from oracle import layer as OL


def rb(x):
    """Round fp32 values to bf16 (nearest even) and back."""
    return OL.bf16_bits_to_f32(OL.f32_to_bf16_bits(np.asarray(x, np.float32)))


def _attention_rounded_p(q, K, V, positions, group):
    """Causal attention with the probabilities rounded to bf16 for the P.V
    product and the normaliser summed from the unrounded values (the prefill
    kernels sum the rounded ones; the two normalisers differ by far less
    than the bounds the model is used for)."""
    n, nq, hd = q.shape
    L = K.shape[0]
    visible = np.arange(L)[None, :] <= np.asarray(positions)[:, None]
    scale = np.float32(1.0 / np.sqrt(hd))
    out = np.empty_like(q)
    for h in range(nq):
        g = h // group
        s = (q[:, h, :] @ K[:, g, :].T) * scale
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        out[:, h, :] = (rb(p) @ V[:, g, :]) / p.sum(axis=1, keepdims=True)
    return out


def layer_step_bf16_points(cfg, W, k_cache, v_cache, block_tables, context_lens, chunk_lens, x_bits,
                           round_qkv=True, round_rest=True):
    """The oracle's batched layer step with the HIP path's bf16 rounding
    points: round_qkv rounds the projection output and the rotated q;
    round_rest rounds a, P, the attention output, h1, b, m and y.  Dense
    layers without q/k norms only.  Mutates the caches like the oracle."""
    assert not cfg.n_experts and not cfg.qk_norm
    nq, nkv, hd, G, P = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.group, cfg.page_size
    ident = lambda t: t  # noqa: E731
    rq = rb if round_qkv else ident
    rr = rb if round_rest else ident
    ctx = np.asarray(context_lens, np.int64)
    chk = np.asarray(chunk_lens, np.int64)
    off = np.concatenate([[0], np.cumsum(chk)])
    x = OL.bf16_bits_to_f32(x_bits).astype(np.float32)
    y = np.empty((int(off[-1]), cfg.hidden), np.float32)
    for i in range(len(ctx)):
        r0, n, c = int(off[i]), int(chk[i]), int(ctx[i])
        bt = block_tables[i]
        rows = slice(r0, r0 + n)
        pos = c + np.arange(n)
        a = rr(OL.rmsnorm(x[rows], W["g1"], cfg.rms_eps))
        q = rq(OL.rope(rq(a @ W["wq"].T).reshape(n, nq, hd), pos, cfg.rope_theta))
        k = OL.rope(rq(a @ W["wk"].T).reshape(n, nkv, hd), pos, cfg.rope_theta)
        v = rq(a @ W["wv"].T).reshape(n, nkv, hd)
        OL.append_kv(k_cache, bt, pos, k, P)
        OL.append_kv(v_cache, bt, pos, v, P)
        K = OL.gather_positions(k_cache, bt, c + n, P)
        V = OL.gather_positions(v_cache, bt, c + n, P)
        if round_rest:
            o = _attention_rounded_p(q, K, V, pos, G)
        else:
            o = OL.causal_attention_seq(q, K, V, pos, G)
        o = rr(o.reshape(n, nq * hd))
        h1 = rr(x[rows] + o @ W["wo"].T)
        b = rr(OL.rmsnorm(h1, W["g2"], cfg.rms_eps))
        m = rr(OL.silu(b @ W["wg"].T) * (b @ W["wu"].T))
        y[rows] = rr(h1 + m @ W["wd"].T)
    return y

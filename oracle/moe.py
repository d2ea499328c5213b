"""Mixture-of-experts feed-forward block for the oracle.

TEST INFRASTRUCTURE ONLY: only tests, the package smoke check and the
benchmark's CPU-baseline leg call this.  It shares no code with the HIP path.

The paper's primary models include an MoE one, Qwen3-30B-A3B (Sec. 4.1
"Models"); its kernel breakdown finds the routing and expert computation
dominating that model's step time while staying insensitive to the batch's
decode share, like the dense GEMMs (App. A.2, "Kernel breakdown").  The paper
does not write the block down; this module writes out the standard sparse
MoE feed-forward block of that model family, in place of the dense SwiGLU:

  logits[t]  = b[t] W_r^T                       (W_r: [E, d], one row per expert)
  S(t)       = the k largest logits of token t  (equal logits: lower expert first)
  w[t, e]    = exp(logits[t, e]) / sum_{e' in S(t)} exp(logits[t, e'])   for e in S(t)
               (renormalised top-k: the softmax over all E restricted to S(t)
               and divided by its sum), or the plain softmax over all E
               restricted to S(t) when renormalisation is off
  m_e(t)     = SiLU(b[t] Wg_e^T) * (b[t] Wu_e^T)  (Wgu_e: [2F, d], rows gate then up)
  moe(t)     = sum_{e in S(t)} w[t, e] * m_e(t) Wd_e^T   (Wd_e: [d, F])

with b the block's (already normalised) bf16 input.  Arithmetic runs in
float64 here; the weights and b are bf16 numbers.  Where the HIP path's
floating point decides which experts a token takes (near-equal logits), its
tests check that the choice is a valid top-k of these logits and evaluate
this block under that choice (`ids` / `weights` arguments).
"""
from __future__ import annotations

from typing import Optional, Tuple

import numpy as np

from .layer import bf16_bits_to_f32, silu


def router_logits(b_bits: np.ndarray, w_router_bits: np.ndarray) -> np.ndarray:
    """[T, E] logits b W_r^T in float64."""
    b = bf16_bits_to_f32(b_bits).astype(np.float64)
    wr = bf16_bits_to_f32(w_router_bits).astype(np.float64)
    return b @ wr.T


def top_k_experts(logits: np.ndarray, k: int) -> np.ndarray:
    """[T, k] expert ids, largest logit first, equal logits by lower id."""
    T, E = logits.shape
    ids = np.empty((T, k), np.int64)
    for t in range(T):
        # sort by (-logit, id): a stable sort of the negated logits keeps the
        # lower id first among equals
        order = np.argsort(-logits[t], kind="stable")
        ids[t] = order[:k]
    return ids


def routing_weights(logits: np.ndarray, ids: np.ndarray, renormalize: bool) -> np.ndarray:
    """[T, k] weights of the chosen experts: softmax over all E at the chosen
    ids, divided by their sum when ``renormalize``."""
    mx = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - mx)
    p = p / p.sum(axis=1, keepdims=True)
    w = np.take_along_axis(p, ids, axis=1)
    if renormalize:
        w = w / w.sum(axis=1, keepdims=True)
    return w


def route(b_bits: np.ndarray, w_router_bits: np.ndarray, k: int,
          renormalize: bool = True) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(ids [T, k], weights [T, k], logits [T, E])."""
    logits = router_logits(b_bits, w_router_bits)
    ids = top_k_experts(logits, k)
    return ids, routing_weights(logits, ids, renormalize), logits


def moe_ffn(b_bits: np.ndarray, w_router_bits: np.ndarray, w_gate_up_bits: np.ndarray,
            w_down_bits: np.ndarray, k: int, renormalize: bool = True,
            ids: Optional[np.ndarray] = None, weights: Optional[np.ndarray] = None) -> np.ndarray:
    """[T, d] float64 output of the MoE block (no residual).  ``ids`` and
    ``weights`` replace the block's own routing when given."""
    if ids is None:
        ids, weights, _ = route(b_bits, w_router_bits, k, renormalize)
    b = bf16_bits_to_f32(b_bits).astype(np.float64)
    T, d = b.shape
    F = w_gate_up_bits.shape[1] // 2
    out = np.zeros((T, d), np.float64)
    for e in np.unique(ids):
        rows, slots = np.nonzero(ids == e)
        wgu = bf16_bits_to_f32(w_gate_up_bits[e]).astype(np.float64)
        wd = bf16_bits_to_f32(w_down_bits[e]).astype(np.float64)
        x = b[rows]
        g = x @ wgu[:F].T
        u = x @ wgu[F:].T
        m = silu(g) * u
        out[rows] += weights[rows, slots][:, None] * (m @ wd.T)
    return out

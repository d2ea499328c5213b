"""Seeded synthetic inputs for one decoder-layer step over a token batch.

This module only draws numbers and lays them out; it performs none of the
layer arithmetic.  Both the HIP path (through the binding) and the CPU oracle
consume what it produces, so it is the one piece of code they share.

Workload shapes follow the per-iteration batch that the paper's scheduler
forms (Sec. 3.1 "Timing Model": prefill rows and decode rows of requests whose
KV is preserved; App. A.1: at most B rows per iteration under chunked
prefill).  Layer shapes are Llama-style decoders (tiny, 8B-shaped,
70B-shaped).  Readings of points the paper leaves open (seeds, gains, RoPE
theta for the larger shapes, length-draw rules) are listed with each helper.

Everything bf16 is held as torch.bfloat16 tensors; ``bits()`` gives the raw
uint16 patterns the oracle works on.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np
import torch

PAGE_SIZE = 16
BASE_SEED = 0


@dataclasses.dataclass(frozen=True)
class LayerShape:
    name: str
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rope_theta: float
    rms_eps: float = 1e-5
    page_size: int = PAGE_SIZE
    # mixture-of-experts feed-forward when n_experts > 0 (ffn then unused)
    n_experts: int = 0
    top_k: int = 0
    expert_ffn: int = 0
    # per-head RMSNorm of q and k before RoPE (Qwen3), gains [head_dim] each
    qk_norm: bool = False

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def weight_bytes(self) -> int:
        d, f = self.hidden, self.ffn
        if self.n_experts:
            n = self.qkv_rows * d + d * self.n_q_heads * self.head_dim + 2 * d + self.n_experts * d + \
                self.n_experts * 3 * self.expert_ffn * d
            return 2 * n + (4 * self.head_dim if self.qk_norm else 0)
        n = self.qkv_rows * d + d * self.n_q_heads * self.head_dim + 2 * f * d + d * f + 2 * d
        return 2 * n


# Tiny layer: hidden 256, GQA 4/2, head_dim 64, SwiGLU 688, RoPE theta 1e4.
TINY = LayerShape("tiny", 256, 4, 2, 64, 688, 1e4)
# Llama-3-8B-shaped layer.  RoPE theta 5e5 follows the Llama-3 convention
# (the workload description does not state it).
L8B = LayerShape("llama3-8b", 4096, 32, 8, 128, 14336, 5e5)
# Llama-3-70B-shaped layer, same theta reading.
L70B = LayerShape("llama3-70b", 8192, 64, 8, 128, 28672, 5e5)
# Mixture-of-experts layers: attention as in the dense layers (no q/k norms),
# the feed-forward replaced by the MoE block.  Qwen3-30B-A3B shapes: hidden
# 2048, 32 q / 4 kv heads of 128, 128 experts, 8 per token, width 768, RoPE
# theta 1e6; and a tiny one for the parity tests.
Q30B = LayerShape("qwen3-30b-a3b", 2048, 32, 4, 128, 0, 1e6, n_experts=128, top_k=8, expert_ffn=768,
                   qk_norm=True)
TINY_MOE = LayerShape("tiny-moe", 256, 4, 2, 64, 0, 1e4, n_experts=16, top_k=4, expert_ffn=128, qk_norm=True)
# the dense tiny layer with the Qwen3 q/k norms
TINY_QKN = LayerShape("tiny-qk-norm", 256, 4, 2, 64, 688, 1e4, qk_norm=True)

SHAPES = {s.name: s for s in (TINY, L8B, L70B, Q30B, TINY_MOE)}


def seeds(base: int = BASE_SEED) -> dict:
    """Four independent integer seeds: weights, kv, batch, x."""
    children = np.random.SeedSequence(base).spawn(4)
    names = ("weights", "kv", "batch", "x")
    return {n: int(c.generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF)
            for n, c in zip(names, children)}


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def bits(t: torch.Tensor) -> np.ndarray:
    """Raw bf16 bit patterns of a bf16 tensor as a uint16 numpy array."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

def make_weights(shape: LayerShape, seed: Optional[int] = None, device="cpu",
                 proj_std: float = 0.02) -> dict:
    """Layer weights in the [out, in] layout, bf16.

    Projections ~ N(0, proj_std), 0.02 by default; a larger spread makes the
    attention scores peaky, which some self-checks need.  Norm gains ~ 1 + 0.1 N(0, 1): a gain of exactly
    one would hide a dropped gain, and N(0, 0.02) gains would shrink the
    residual stream fifty-fold.
    w_qkv rows: q heads, then k heads, then v heads.  w_gate_up rows: gate then up.
    """
    if seed is None:
        seed = seeds()["weights"]
    g = _gen(device, seed)
    d, hd = shape.hidden, shape.head_dim
    f = shape.ffn

    def proj(rows, cols):
        w = torch.empty(rows, cols, dtype=torch.bfloat16, device=device)
        # chunked draw keeps the fp32 temporary small for 70B-sized matrices
        step = max(1, (1 << 26) // cols)
        for r0 in range(0, rows, step):
            r1 = min(rows, r0 + step)
            w[r0:r1] = (torch.randn(r1 - r0, cols, generator=g, device=device) * proj_std).to(torch.bfloat16)
        return w

    def gain(n=d):
        return (1.0 + 0.1 * torch.randn(n, generator=g, device=device)).to(torch.bfloat16)

    def with_qk_norm(w):
        if shape.qk_norm:
            w.update({"q_norm": gain(hd), "k_norm": gain(hd)})
        return w

    if shape.n_experts:  # attention as above, a mixture-of-experts feed-forward
        w = {"attn_norm": gain(), "w_qkv": proj(shape.qkv_rows, d), "w_o": proj(d, shape.n_q_heads * hd),
             "mlp_norm": gain()}
        moe = make_moe_weights(MoeShape(shape.name, d, shape.n_experts, shape.top_k, shape.expert_ffn),
                               seed=seed + 1, device=device, proj_std=proj_std)
        w.update({"w_router": moe["w_router"], "w_experts_gate_up": moe["w_gate_up"],
                  "w_experts_down": moe["w_down"]})
        return with_qk_norm(w)
    return with_qk_norm({
        "attn_norm": gain(),
        "w_qkv": proj(shape.qkv_rows, d),
        "w_o": proj(d, shape.n_q_heads * hd),
        "mlp_norm": gain(),
        "w_gate_up": proj(2 * f, d),
        "w_down": proj(d, f),
    })


# ----------------------------------------------------------------------------
# batches
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Batch:
    """One step's requests.

    context_lens[i]: tokens already in the cache before the step.
    chunk_lens[i]:  new rows this step (1 for a decode request).
    Rows of request i are contiguous and requests are in list order.
    """
    context_lens: np.ndarray
    chunk_lens: np.ndarray
    label: str = ""

    @property
    def num_seqs(self) -> int:
        return int(self.context_lens.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.chunk_lens.sum())

    @property
    def row_offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.chunk_lens)]).astype(np.int64)

    @property
    def num_decode(self) -> int:
        return int((self.chunk_lens == 1).sum())

    def subset(self, idx: Sequence[int]) -> "Batch":
        idx = np.asarray(idx, dtype=np.int64)
        return Batch(self.context_lens[idx].copy(), self.chunk_lens[idx].copy(), self.label + "[subset]")

    def concat(self, other: "Batch") -> "Batch":
        return Batch(np.concatenate([self.context_lens, other.context_lens]),
                     np.concatenate([self.chunk_lens, other.chunk_lens]),
                     self.label + "+" + other.label)


def _uniform_int(rng, lo, hi, n):
    """Inclusive discrete uniform on [lo, hi]."""
    return rng.integers(lo, hi + 1, size=n).astype(np.int32)


def batch_decode(n: int, ctx_lo: int, ctx_hi: int, rng) -> Batch:
    c = _uniform_int(rng, ctx_lo, ctx_hi, n)
    return Batch(c, np.ones(n, dtype=np.int32), f"decode{n}")


def batch_tiny(seed: Optional[int] = None, mode: str = "mixed") -> Batch:
    """4 decode requests with contexts U{64..256} plus one 128-token prefill
    chunk with no prior prefix.  mode: 'decode' | 'prefill' | 'mixed'."""
    rng = np.random.default_rng(seeds()["batch"] if seed is None else seed)
    dec = batch_decode(4, 64, 256, rng)
    pre = Batch(np.zeros(1, np.int32), np.full(1, 128, np.int32), "prefill128")
    return {"decode": dec, "prefill": pre, "mixed": dec.concat(pre)}[mode]


def batch_8b_decode(seed: Optional[int] = None) -> Batch:
    """64 decode requests, contexts U{512..4096}."""
    rng = np.random.default_rng(seeds()["batch"] if seed is None else seed)
    return batch_decode(64, 512, 4096, rng)


def batch_8b_prefill(seed: Optional[int] = None, cap: int = 8192) -> Batch:
    """8 prompts, lengths U{256..2048}, walked in order and cut so the total is
    at most ``cap`` (a prompt that would overflow is truncated to the remainder,
    later ones are dropped); no prior KV."""
    rng = np.random.default_rng(seeds()["batch"] if seed is None else seed)
    lens = _uniform_int(rng, 256, 2048, 8)
    out, left = [], cap
    for L in lens:
        if left <= 0:
            break
        take = int(min(L, left))
        out.append(take)
        left -= take
    n = np.asarray(out, np.int32)
    return Batch(np.zeros_like(n), n, "prefill8")


def batch_mixed_budget(r: float, budget: int, rng, dec_ctx=(1024, 8192),
                       chunk=(256, 1024), prefix=(0, 2048)) -> Batch:
    """Mixed step at a fixed token budget B and decode share r.

    n_d = round(r B) decode rows (one per request) come first; prefill chunks
    drawn from U{chunk} fill the remaining B - n_d rows, the last one cut to
    what is left, each with a prior prefix drawn from U{prefix}.
    """
    n_d = int(round(r * budget))
    dec = batch_decode(n_d, dec_ctx[0], dec_ctx[1], rng) if n_d else Batch(np.zeros(0, np.int32), np.zeros(0, np.int32))
    left = budget - n_d
    cl, pl = [], []
    while left > 0:
        L = int(min(rng.integers(chunk[0], chunk[1] + 1), left))
        cl.append(L)
        pl.append(int(rng.integers(prefix[0], prefix[1] + 1)))
        left -= L
    pre = Batch(np.asarray(pl, np.int32), np.asarray(cl, np.int32), "prefill")
    b = dec.concat(pre) if n_d else pre
    b.label = f"mb_r{r:.2f}_B{budget}"
    return b


def batch_8b_mixed(r: float, budget: int = 2048, seed: Optional[int] = None, **kw) -> Batch:
    """The 8B-shaped mixed sweep point at decode share r (budget 2048)."""
    s = seeds()["batch"] if seed is None else seed
    rng = np.random.default_rng([s, int(round(r * 1000)), budget])
    return batch_mixed_budget(r, budget, rng, **kw)


def batch_70b_decode(seed: Optional[int] = None) -> Batch:
    """256 decode requests, contexts U{2048..16384} (the 70B-shaped step)."""
    rng = np.random.default_rng([seeds()["batch"] if seed is None else seed, 70])
    return batch_decode(256, 2048, 16384, rng)


def batch_70b_mixed(r: float, budget: int = 4096, seed: Optional[int] = None) -> Batch:
    """The 70B-shaped mixed step at decode share r: decode contexts
    U{2048..16384}; prefill chunks and prefixes as in the 8B sweep."""
    s = seeds()["batch"] if seed is None else seed
    rng = np.random.default_rng([s, 70, int(round(r * 1000)), budget])
    return batch_mixed_budget(r, budget, rng, dec_ctx=(2048, 16384))


# ----------------------------------------------------------------------------
# paged KV pool
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class KVPool:
    k_cache: torch.Tensor          # [num_pages, n_kv, page, hd] bf16
    v_cache: torch.Tensor
    block_tables: torch.Tensor     # [num_seqs, max_pages_per_seq] int32 (-1 = unused)
    num_pages: int
    max_pages_per_seq: int

    def clone(self) -> "KVPool":
        return KVPool(self.k_cache.clone(), self.v_cache.clone(), self.block_tables.clone(),
                      self.num_pages, self.max_pages_per_seq)

    def to(self, device) -> "KVPool":
        return KVPool(self.k_cache.to(device), self.v_cache.to(device), self.block_tables.to(device),
                      self.num_pages, self.max_pages_per_seq)


def pages_needed(batch: Batch, page: int = PAGE_SIZE) -> np.ndarray:
    return (batch.context_lens.astype(np.int64) + batch.chunk_lens + page - 1) // page


def make_block_tables(batch: Batch, spare_pages: int, seed: int, page: int = PAGE_SIZE,
                      max_pages_per_seq: Optional[int] = None):
    """A seeded permutation of the pool's page ids dealt out, in order, to the
    (request, logical page) pairs; no page is shared.  Returns (tables, pool)."""
    need = pages_needed(batch, page)
    total = int(need.sum())
    pool = total + spare_pages
    rng = np.random.default_rng(seed)
    perm = rng.permutation(pool).astype(np.int32)
    mp = int(need.max()) if max_pages_per_seq is None else max_pages_per_seq
    assert mp >= int(need.max()) if batch.num_seqs else True
    bt = np.full((batch.num_seqs, max(mp, 1)), -1, np.int32)
    k = 0
    for i, n in enumerate(need):
        bt[i, :n] = perm[k:k + n]
        k += n
    return bt, pool


def _fp8_codes(g, rows: int, cols: int, device) -> torch.Tensor:
    """Random E4M3 codes: random sign, exponent field 4..9, random mantissa."""
    w = torch.empty(rows, cols, dtype=torch.uint8, device=device)
    step = max(1, (1 << 26) // cols)
    for r0 in range(0, rows, step):
        r1 = min(rows, r0 + step)
        n = (r1 - r0, cols)
        sign = torch.randint(0, 2, n, generator=g, device=device) << 7
        ex = torch.randint(4, 10, n, generator=g, device=device) << 3
        man = torch.randint(0, 8, n, generator=g, device=device)
        w[r0:r1] = (sign | ex | man).to(torch.uint8)
    return w


def _row_scales(g, rows: int, proj_std: float, device) -> torch.Tensor:
    return (proj_std / 2.3) * (0.5 + torch.rand(rows, generator=g, device=device))


def make_weights_fp8(shape: LayerShape, seed: Optional[int] = None, device="cpu",
                     proj_std: float = 0.02) -> dict:
    """Layer weights with the four projections as 8-bit E4M3 codes (uint8,
    [out, in]) and one float32 scale per output row (keys s_qkv, s_o,
    s_gate_up, s_down); norm gains bf16 as in make_weights.

    Codes are random bytes with a random sign bit, an exponent field in 4..9
    and a random 3-bit mantissa (values 1/8 .. 7.5 in magnitude, RMS about
    2.3); row scales are proj_std / 2.3 times U[0.5, 1.5], so the weights
    they stand for have about proj_std spread and every row a scale of its own.
    """
    if seed is None:
        seed = seeds()["weights"]
    g = _gen(device, seed)
    d, hd = shape.hidden, shape.head_dim
    f = shape.ffn

    def codes(rows, cols):
        return _fp8_codes(g, rows, cols, device)

    def scales(rows):
        return _row_scales(g, rows, proj_std, device)

    def gain():
        return (1.0 + 0.1 * torch.randn(d, generator=g, device=device)).to(torch.bfloat16)

    return {
        "attn_norm": gain(),
        "w_qkv": codes(shape.qkv_rows, d), "s_qkv": scales(shape.qkv_rows),
        "w_o": codes(d, shape.n_q_heads * hd), "s_o": scales(d),
        "mlp_norm": gain(),
        "w_gate_up": codes(2 * f, d), "s_gate_up": scales(2 * f),
        "w_down": codes(d, f), "s_down": scales(d),
    }


def make_fp8_matrix(rows: int, cols: int, seed: int, device="cpu", proj_std: float = 0.02):
    """One [rows, cols] weight matrix as (uint8 E4M3 codes, float32 row
    scales), drawn as the projections of make_weights_fp8 are."""
    g = _gen(device, seed)
    return _fp8_codes(g, rows, cols, device), _row_scales(g, rows, proj_std, device)


@dataclasses.dataclass(frozen=True)
class MoeShape:
    name: str
    hidden: int
    n_experts: int
    top_k: int
    expert_ffn: int

    def expert_bytes(self) -> int:
        """bf16 bytes of one expert's gate/up and down projections."""
        return 2 * (2 * self.expert_ffn * self.hidden + self.hidden * self.expert_ffn)


# Qwen3-30B-A3B's MoE feed-forward block: hidden 2048, 128 experts, 8 per
# token, expert SwiGLU width 768, renormalised top-k weights.
MOE30B = MoeShape("qwen3-30b-a3b-moe", 2048, 128, 8, 768)
MOE_TINY = MoeShape("moe-tiny", 256, 16, 4, 128)


def make_moe_weights(shape: MoeShape, seed: Optional[int] = None, device="cpu", proj_std: float = 0.02) -> dict:
    """bf16 MoE block weights: router [E, d] ~ N(0, 1 / d) (logits of
    N(0, 1) inputs spread about 1), gate/up [E, 2F, d] (per expert F gate
    rows, then F up rows) and down [E, d, F] ~ N(0, proj_std)."""
    if seed is None:
        seed = seeds()["weights"] + 7
    g = _gen(device, seed)
    E, d, F = shape.n_experts, shape.hidden, shape.expert_ffn

    def draw(*sz, std):
        w = torch.empty(*sz, dtype=torch.bfloat16, device=device)
        for e in range(sz[0]):   # one expert at a time keeps the fp32 temporary small
            w[e] = (torch.randn(*sz[1:], generator=g, device=device) * std).to(torch.bfloat16)
        return w
    return {"w_router": (torch.randn(E, d, generator=g, device=device) / d ** 0.5).to(torch.bfloat16),
            "w_gate_up": draw(E, 2 * F, d, std=proj_std), "w_down": draw(E, d, F, std=proj_std)}


def weight_arrays(w: dict) -> dict:
    """Host numpy form of a weight dict: bf16 bit patterns, 8-bit codes and
    float32 row scales as they are."""
    out = {}
    for k, v in w.items():
        if v.dtype == torch.bfloat16:
            out[k] = bits(v)
        else:
            out[k] = v.detach().contiguous().cpu().numpy()
    return out


def _pool_tensor(shape4, fill, dtype, device, store):
    """A [pool, nkv, P, hd] tensor filled with ``fill``: fresh, or the leading
    elements of the flat byte buffer ``store`` (so that a caller can keep one
    allocation, and one physical placement, across many pools)."""
    if store is None:
        return torch.full(shape4, fill, dtype=dtype, device=device)
    n = int(np.prod(shape4)) * torch.empty((), dtype=dtype).element_size()
    if store.numel() < n or store.dtype != torch.uint8:
        raise ValueError("pool storage too small")
    return store[:n].view(dtype).view(shape4).fill_(fill)


def make_kv_pool(shape: LayerShape, batch: Batch, seed: Optional[int] = None, device="cpu",
                 spare_pages: int = 0, poison: bool = True,
                 max_pages_per_seq: Optional[int] = None, store=None) -> KVPool:
    """Paged bf16 K/V pool holding each request's prior context.

    Prior positions (< context_len) hold bf16 N(0, 1).  With ``poison`` every
    other slot (spare pages, the slots the step will append to, and slots past
    the end of each request) holds bf16 NaN, so any read outside the block
    table or past a request's length shows up as NaN in the output.  ``store``
    (optional): two flat uint8 device buffers the K and V pools are laid in.
    """
    if seed is None:
        seed = seeds()["kv"]
    bt, pool = make_block_tables(batch, spare_pages, seed, shape.page_size, max_pages_per_seq)
    nkv, P, hd = shape.n_kv_heads, shape.page_size, shape.head_dim
    g = _gen(device, seed)
    fill = float("nan") if poison else 0.0
    kc = _pool_tensor((pool, nkv, P, hd), fill, torch.bfloat16, device, store[0] if store else None)
    vc = _pool_tensor((pool, nkv, P, hd), fill, torch.bfloat16, device, store[1] if store else None)
    bt_t = torch.from_numpy(bt).to(device)
    for i in range(batch.num_seqs):
        c = int(batch.context_lens[i])
        if c == 0:
            continue
        npg = (c + P - 1) // P
        pages = bt_t[i, :npg].long()
        kvals = torch.randn(npg * P, nkv, hd, generator=g, device=device).to(torch.bfloat16)
        vvals = torch.randn(npg * P, nkv, hd, generator=g, device=device).to(torch.bfloat16)
        if poison and c % P:
            kvals[c:] = float("nan")
            vvals[c:] = float("nan")
        # [npg*P, nkv, hd] -> [npg, nkv, P, hd]
        kc[pages] = kvals.view(npg, P, nkv, hd).permute(0, 2, 1, 3)
        vc[pages] = vvals.view(npg, P, nkv, hd).permute(0, 2, 1, 3)
    return KVPool(kc, vc, bt_t, pool, bt.shape[1])


def make_kv_pool_codes(shape: LayerShape, batch: Batch, seed: Optional[int] = None, device="cpu",
                       spare_pages: int = 0, poison: bool = True,
                       max_pages_per_seq: Optional[int] = None, store=None) -> KVPool:
    """Paged 8-bit K/V pool (uint8 E4M3 codes) holding each request's prior
    context: random bytes with a random sign bit, an exponent field in 4..9
    and a random 3-bit mantissa (code values 1/8 .. 7.5 in magnitude).  With
    ``poison`` every other slot holds the NaN code 0x7F."""
    if seed is None:
        seed = seeds()["kv"]
    bt, pool = make_block_tables(batch, spare_pages, seed, shape.page_size, max_pages_per_seq)
    nkv, P, hd = shape.n_kv_heads, shape.page_size, shape.head_dim
    g = _gen(device, seed)
    fill = 0x7F if poison else 0
    kc = _pool_tensor((pool, nkv, P, hd), fill, torch.uint8, device, store[0] if store else None)
    vc = _pool_tensor((pool, nkv, P, hd), fill, torch.uint8, device, store[1] if store else None)
    bt_t = torch.from_numpy(bt).to(device)

    def codes(n):
        sign = torch.randint(0, 2, (n, nkv, hd), generator=g, device=device) << 7
        ex = torch.randint(4, 10, (n, nkv, hd), generator=g, device=device) << 3
        man = torch.randint(0, 8, (n, nkv, hd), generator=g, device=device)
        return (sign | ex | man).to(torch.uint8)

    for i in range(batch.num_seqs):
        c = int(batch.context_lens[i])
        if c == 0:
            continue
        npg = (c + P - 1) // P
        pages = bt_t[i, :npg].long()
        kvals, vvals = codes(npg * P), codes(npg * P)
        if poison and c % P:
            kvals[c:] = 0x7F
            vvals[c:] = 0x7F
        kc[pages] = kvals.view(npg, P, nkv, hd).permute(0, 2, 1, 3)
        vc[pages] = vvals.view(npg, P, nkv, hd).permute(0, 2, 1, 3)
    return KVPool(kc, vc, bt_t, pool, bt.shape[1])


def make_x(shape: LayerShape, num_tokens: int, seed: Optional[int] = None, device="cpu") -> torch.Tensor:
    """Activations entering the layer: bf16 N(0, 1), [num_tokens, hidden]."""
    if seed is None:
        seed = seeds()["x"]
    g = _gen(device, seed)
    return torch.randn(num_tokens, shape.hidden, generator=g, device=device).to(torch.bfloat16)


def relabel_pages(pool: KVPool, seed: int) -> KVPool:
    """The same logical cache under a different physical page numbering."""
    rng = np.random.default_rng(seed)
    perm = torch.from_numpy(rng.permutation(pool.num_pages).astype(np.int64))
    inv = torch.empty_like(perm)
    inv[perm] = torch.arange(pool.num_pages)
    kc = torch.empty_like(pool.k_cache)
    vc = torch.empty_like(pool.v_cache)
    kc[perm.to(kc.device)] = pool.k_cache
    vc[perm.to(vc.device)] = pool.v_cache
    bt = pool.block_tables.clone().long()
    m = bt >= 0
    bt[m] = perm.to(bt.device)[bt[m]]
    return KVPool(kc, vc, bt.to(torch.int32), pool.num_pages, pool.max_pages_per_seq)

"""The transformers Llama decoder layer in fp64, fed the oracle's inputs: an
independent reference for the oracle's layer step (CPU only)."""
import numpy as np
import torch

from oracle import layer as L


def hf_layer(shape, w_bits):
    """The Llama decoder layer, or for a shape with q/k norms the Qwen3 one."""
    if shape.qk_norm:
        from transformers import Qwen3Config as Config
        from transformers.models.qwen3.modeling_qwen3 import Qwen3DecoderLayer as Layer
        from transformers.models.qwen3.modeling_qwen3 import Qwen3RotaryEmbedding as Rotary
    else:
        from transformers import LlamaConfig as Config
        from transformers.models.llama.modeling_llama import LlamaDecoderLayer as Layer
        from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding as Rotary
    cfg = Config(hidden_size=shape.hidden, intermediate_size=shape.ffn,
                      num_attention_heads=shape.n_q_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta,
                      attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "sdpa"  # the eager path takes its softmax in fp32
    layer = Layer(cfg, layer_idx=0).double()
    rot = Rotary(cfg).double()
    # the library forms its frequencies in fp32; recompute them in fp64
    hd = shape.head_dim
    rot.inv_freq = shape.rope_theta ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    def f(k):
        # bf16 bits, or 8-bit codes with row scales decoded by torch's float8_e4m3fn
        w = w_bits[k]
        if w.dtype == np.uint8:
            s = torch.from_numpy(np.asarray(w_bits["s_" + k[2:]], np.float64))
            return torch.from_numpy(np.ascontiguousarray(w)).view(torch.float8_e4m3fn).double() * s[:, None]
        return torch.from_numpy(L.bf16_bits_to_f32(w).astype(np.float64))
    nq, nkv, hd, ff = shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn
    qkv, gu = f("w_qkv"), f("w_gate_up")
    # the library's RMSNorm module computes in fp32; use torch's in fp64
    layer.input_layernorm = torch.nn.RMSNorm(shape.hidden, eps=shape.rms_eps, dtype=torch.float64)
    layer.post_attention_layernorm = torch.nn.RMSNorm(shape.hidden, eps=shape.rms_eps, dtype=torch.float64)
    if shape.qk_norm:
        layer.self_attn.q_norm = torch.nn.RMSNorm(shape.head_dim, eps=shape.rms_eps, dtype=torch.float64)
        layer.self_attn.k_norm = torch.nn.RMSNorm(shape.head_dim, eps=shape.rms_eps, dtype=torch.float64)
    with torch.no_grad():
        layer.self_attn.q_proj.weight.copy_(qkv[: nq * hd])
        layer.self_attn.k_proj.weight.copy_(qkv[nq * hd:(nq + nkv) * hd])
        layer.self_attn.v_proj.weight.copy_(qkv[(nq + nkv) * hd:])
        layer.self_attn.o_proj.weight.copy_(f("w_o"))
        layer.mlp.gate_proj.weight.copy_(gu[:ff])
        layer.mlp.up_proj.weight.copy_(gu[ff:])
        layer.mlp.down_proj.weight.copy_(f("w_down"))
        layer.input_layernorm.weight.copy_(f("attn_norm"))
        layer.post_attention_layernorm.weight.copy_(f("mlp_norm"))
        if shape.qk_norm:
            layer.self_attn.q_norm.weight.copy_(f("q_norm"))
            layer.self_attn.k_norm.weight.copy_(f("k_norm"))
    return layer, rot


def bf16_store(t):
    """An appended K/V row as a bf16 cache holds it (rounded through fp32)."""
    return t.float().to(torch.bfloat16).double()


def e4m3_store(scale):
    """An appended K/V row as an 8-bit cache with this scale holds it, with
    torch's own conversions: bf16, divided by the scale in fp32, converted to
    float8_e4m3fn (values stay within its range here), read back times the
    scale."""
    return lambda t: (bf16_store(t).float() / scale).to(torch.float8_e4m3fn).double() * scale


def e4m3_values(codes, scale):
    """The values 8-bit cache codes stand for, by torch's float8_e4m3fn."""
    return torch.from_numpy(np.ascontiguousarray(codes)).view(torch.float8_e4m3fn).double().numpy() * scale


class RoundingCache:
    """Minimal KV cache for the library layer: holds a request's prior K/V and
    stores each appended K/V through the cache's element rounding; returns
    everything stored so far."""

    def __init__(self, k_prior, v_prior, store_k, store_v):
        self.k, self.v = k_prior, v_prior            # [1, n_kv, c, hd] fp64
        self.store_k, self.store_v = store_k, store_v

    def update(self, k, v, layer_idx, cache_kwargs=None):
        self.k = torch.cat([self.k, self.store_k(k)], dim=2)
        self.v = torch.cat([self.v, self.store_v(v)], dim=2)
        return self.k, self.v


def hf_reference(shape, o, seq, kv_scales=None):
    """The library decoder layer in fp64 on request ``seq`` of an oracle input
    set: returns (h1 - x, y - h1, y) for that request's rows.  With
    ``kv_scales`` = (k_scale, v_scale) the caches of ``o`` hold 8-bit E4M3
    codes, read and written through torch's float8_e4m3fn conversions."""
    layer, rot = hf_layer(shape, o["w_bits"])
    c, n = int(o["context_lens"][seq]), int(o["chunk_lens"][seq])
    r0 = int(np.sum(o["chunk_lens"][:seq]))
    bt = o["block_tables"][seq]
    pos = np.arange(c)
    kraw, vraw = o["k_cache"][bt[pos // 16], :, pos % 16, :], o["v_cache"][bt[pos // 16], :, pos % 16, :]
    if kv_scales is None:
        kp = L.bf16_bits_to_f32(kraw).astype(np.float64)
        vp = L.bf16_bits_to_f32(vraw).astype(np.float64)
        stores = (bf16_store, bf16_store)
    else:
        kp, vp = e4m3_values(kraw, kv_scales[0]), e4m3_values(vraw, kv_scales[1])
        stores = (e4m3_store(kv_scales[0]), e4m3_store(kv_scales[1]))
    cache = RoundingCache(torch.from_numpy(kp).permute(1, 0, 2)[None], torch.from_numpy(vp).permute(1, 0, 2)[None],
                          *stores)
    x = torch.from_numpy(L.bf16_bits_to_f32(o["x_bits"][r0:r0 + n]).astype(np.float64))[None]
    p = torch.arange(c, c + n)[None]
    mask = torch.zeros(n, c + n, dtype=torch.float64)
    mask[torch.arange(c + n)[None, :] > (c + torch.arange(n))[:, None]] = float("-inf")
    # the library's rotary module forms angles in fp32; give the layer fp64
    # cos/sin in its own (duplicated-halves) format instead
    ang = p[0].double()[:, None] * rot.inv_freq[None, :]
    emb = torch.cat([ang, ang], dim=-1)[None]
    pe = (emb.cos(), emb.sin())
    with torch.no_grad():
        a = layer.input_layernorm(x)
        attn_branch = layer.self_attn(a, attention_mask=mask[None, None], position_ids=p,
                                      position_embeddings=pe, past_key_values=cache)[0]
        h1 = x + attn_branch
        mlp_branch = layer.mlp(layer.post_attention_layernorm(h1))
    return attn_branch[0].numpy(), mlp_branch[0].numpy(), (h1 + mlp_branch)[0].numpy()

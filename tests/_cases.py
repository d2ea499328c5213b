"""Test cases assembled from the seeded generators, in the forms both the HIP
path (torch tensors) and the oracle (numpy bf16 bit arrays) take."""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

from paper_2606_00516_amd import inputs as gen
import oracle


def oracle_cfg(shape: gen.LayerShape) -> oracle.LayerCfg:
    return oracle.LayerCfg(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn,
                           shape.page_size, shape.rms_eps, shape.rope_theta, shape.n_experts, shape.top_k,
                           shape.expert_ffn, qk_norm=shape.qk_norm)


@dataclasses.dataclass
class Case:
    shape: gen.LayerShape
    weights: dict            # name -> bf16 tensor
    batch: gen.Batch
    pool: gen.KVPool
    x: torch.Tensor          # [T, d] bf16

    def oracle_inputs(self):
        return dict(
            cfg=oracle_cfg(self.shape),
            w_bits={k: gen.bits(v) for k, v in self.weights.items()},
            k_cache=gen.bits(self.pool.k_cache).copy(),
            v_cache=gen.bits(self.pool.v_cache).copy(),
            block_tables=self.pool.block_tables.cpu().numpy(),
            context_lens=self.batch.context_lens,
            chunk_lens=self.batch.chunk_lens,
            x_bits=gen.bits(self.x),
        )

    def run_oracle(self, mode="batched", dtype=np.float32, seqs=None, intermediates=False, W=None):
        o = self.oracle_inputs()
        if W is None:
            W = oracle.prepare_weights(o["w_bits"], o["cfg"], dtype)
        res = oracle.layer_step(o["cfg"], W, o["k_cache"], o["v_cache"], o["block_tables"],
                                o["context_lens"], o["chunk_lens"], o["x_bits"], mode=mode, seqs=seqs,
                                intermediates=intermediates)
        return res, o


def make_case(shape: gen.LayerShape, batch: gen.Batch, spare_pages: int = 3, poison: bool = True,
              device="cpu", weights=None, x_seed=None, kv_seed=None) -> Case:
    w = gen.make_weights(shape, device=device) if weights is None else weights
    pool = gen.make_kv_pool(shape, batch, seed=kv_seed, device=device, spare_pages=spare_pages, poison=poison)
    x = gen.make_x(shape, batch.num_tokens, seed=x_seed, device=device)
    return Case(shape, w, batch, pool, x)


def tiny_case(mode="mixed", **kw) -> Case:
    return make_case(gen.TINY, gen.batch_tiny(mode=mode), **kw)

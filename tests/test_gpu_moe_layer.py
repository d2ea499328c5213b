"""Layer steps whose feed-forward part is the mixture-of-experts block,
through the C ABI against the oracle: the three step entry points on a tiny
MoE layer, a stack of two such layers, the Qwen3-30B-A3B-shaped layer on the
full 8B-style decode, prefill and mixed batches with sampled requests
recomputed by the oracle (tokens route independently, so a request's rows
do not depend on the rest of the batch), and the weight checks.

The block's input reaches the router through the layer's bf16 activations,
which the oracle does not round the same way, so the logits of the two sides
differ at the 1e-3 level; a token whose k-th and (k+1)-th logits are closer
than that may take a different but equally valid expert.  At full size the
comparison therefore covers the tokens whose top-k is unambiguous (oracle
logit margin at least 1 % of the token's largest logit); the block's own
tests check the routing of the rest for validity."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from oracle import layer as OL
from oracle import moe as MO
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import make_case, oracle_cfg
from tests._gpu import DevCase, maxrel, per_request_maxrel, to_f32
from tests.test_gpu_layer import STEP, _sampled_parity, sub_pool_for_oracle

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_tiny_moe_layer_vs_oracle(mode):
    case = make_case(gen.TINY_MOE, gen.batch_tiny(mode=mode))
    d = DevCase(case)
    b = case.batch
    h = B.Handle(case.shape, 8, 512)
    y = STEP[mode](h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    torch.cuda.synchronize()
    ref, _ = case.run_oracle()
    got = to_f32(y)
    assert np.isfinite(got).all()
    errs = per_request_maxrel(got, ref, b.row_offsets)
    assert max(errs) < TOL, errs


def test_tiny_moe_stack_vs_oracle():
    shape = gen.TINY_MOE
    batch = gen.batch_tiny(mode="mixed")
    case = make_case(shape, batch)
    Ws = [gen.make_weights(shape, seed=300 + l) for l in range(2)]
    pools = [gen.make_kv_pool(shape, batch, seed=400 + l, spare_pages=3) for l in range(2)]
    h = B.Handle(shape, 8, 512)
    y = B.eb_stack_step(h, "mixed", [{k: t.cuda() for k, t in w.items()} for w in Ws],
                        [(p.k_cache.cuda(), p.v_cache.cuda(), p.block_tables.cuda()) for p in pools],
                        batch.context_lens, batch.chunk_lens, case.x.cuda())
    torch.cuda.synchronize()
    cfg = oracle_cfg(shape)
    Wo = [oracle.prepare_weights({k: gen.bits(t) for k, t in w.items()}, cfg) for w in Ws]
    ref = OL.stack_step(cfg, Wo, [gen.bits(p.k_cache).copy() for p in pools],
                        [gen.bits(p.v_cache).copy() for p in pools], [p.block_tables.numpy() for p in pools],
                        batch.context_lens, batch.chunk_lens, gen.bits(case.x))
    errs = per_request_maxrel(to_f32(y), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


@pytest.fixture(scope="module")
def wq30():
    w = gen.make_weights(gen.Q30B)
    Wo = oracle.prepare_weights({k: gen.bits(v) for k, v in w.items()}, oracle_cfg(gen.Q30B))
    return {k: v.cuda() for k, v in w.items()}, Wo


def test_q30b_layer_decode_full_size_sampled(wq30):
    w, Wo = wq30
    _sampled_parity(gen.Q30B, gen.batch_8b_decode(), w, Wo, "decode", [0, 21, 63])


def _moe_sampled_parity(shape, batch, w, Wo, mode, sample, margin=1e-2, min_kept=0.6):
    """Sampled requests against the oracle, rows with an unambiguous top-k."""
    pool = gen.make_kv_pool(shape, batch, device="cuda")
    kb, vb, bt = sub_pool_for_oracle(pool, batch, sample)
    x = gen.make_x(shape, batch.num_tokens)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    y = STEP[mode](h, w, pool.k_cache, pool.v_cache, pool.block_tables, batch.context_lens, batch.chunk_lens,
                   x.cuda())
    torch.cuda.synchronize()
    y = to_f32(y)
    assert np.isfinite(y).all()
    del pool
    cfg = oracle_cfg(shape)
    sub = batch.subset(sample)
    off, so = batch.row_offsets, sub.row_offsets
    xs = np.concatenate([gen.bits(x)[off[i]:off[i + 1]] for i in sample])
    ref, inter = oracle.layer_step(cfg, Wo, kb, vb, bt, sub.context_lens, sub.chunk_lens, xs, intermediates=True)
    b = OL.rmsnorm(inter["h1"], Wo["g2"], cfg.rms_eps)
    logits = MO.router_logits(OL.f32_to_bf16_bits(b.astype(np.float32)), Wo["moe"][0])
    top = -np.sort(-logits, axis=1)
    keep = (top[:, cfg.top_k - 1] - top[:, cfg.top_k]) >= margin * np.abs(top[:, 0])
    got = np.concatenate([y[off[i]:off[i + 1]] for i in sample])
    errs = []
    for k in range(len(sample)):
        rows = slice(so[k], so[k + 1])
        kk = keep[rows]
        if kk.any():
            errs.append(maxrel(got[rows][kk], ref[rows][kk]))
    print(f"{mode} {batch.label}: {int(keep.sum())} of {keep.size} rows with an unambiguous top-k; max-rel {errs}")
    assert keep.mean() >= min_kept, keep.mean()
    assert max(errs) < TOL, errs


def test_q30b_layer_prefill_full_size_sampled(wq30):
    # 8192 tokens: the expert products on the 256 x 256 kernel
    w, Wo = wq30
    batch = gen.batch_8b_prefill()
    _moe_sampled_parity(gen.Q30B, batch, w, Wo, "prefill", [int(np.argmin(batch.chunk_lens))])


def test_q30b_layer_mixed_budget_sampled(wq30):
    w, Wo = wq30
    batch = gen.batch_8b_mixed(0.5)
    dec = [int(i) for i in np.nonzero(batch.chunk_lens == 1)[0][:2]]
    pre = [int(i) for i in np.nonzero(batch.chunk_lens > 1)[0]]
    pre = [min(pre, key=lambda i: batch.chunk_lens[i])] if pre else []
    _moe_sampled_parity(gen.Q30B, batch, w, Wo, "mixed", dec + pre)


def test_moe_layer_weight_checks_enqueue_nothing():
    shape = gen.TINY_MOE
    case = make_case(shape, gen.batch_tiny(mode="decode"))
    d = DevCase(case)
    b = case.batch
    h = B.Handle(shape, 8, 512)
    hb = B.HostBatch(b.context_lens, b.chunk_lens)
    kv = B.kv_struct(d.k, d.v, d.bt)
    y = torch.empty_like(d.x)
    ws = B.alloc_workspace(B.lib().eb_workspace_bytes(h.h, ctypes.byref(hb.c), B.MODES["decode"]), "cuda")

    def run(lw):
        return B.lib().eb_layer_step_decode(h.h, ctypes.byref(lw), ctypes.byref(kv), ctypes.byref(hb.c),
                                            d.x.data_ptr(), y.data_ptr(), ws.data_ptr(), ws.numel(), None)
    lw = B.weights_struct(d.w)
    lw.w_router = None
    assert run(lw) == -1                      # EB_ERR_NULL
    lw = B.weights_struct(d.w)
    lw.w_dtype = B.W_FP8_E4M3
    assert run(lw) == -2                      # 8-bit weights in an MoE layer: EB_ERR_CONFIG
    assert run(B.weights_struct(d.w)) == 0
    torch.cuda.synchronize()

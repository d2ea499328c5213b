"""Layers with the Qwen3 per-head q/k RMSNorm before RoPE, through the C ABI
against the oracle: the dense tiny layer (head_dim 64, four threads per head
in the kernel's sum of squares) in the three step modes with a bf16 and with
an 8-bit cache, the keys the step writes to the cache (normalised, then
rotated), a stack of two such layers, and the checks of the entry points.
The mixture-of-experts layer tests run the norms as well: the Qwen3-30B-A3B
shape (head_dim 128, eight threads per head) carries them."""
import ctypes
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import make_case, oracle_cfg
from tests._gpu import DevCase, maxrel, per_request_maxrel, to_f32
from tests.test_gpu_fp8 import KS, VS, _oracle_step, code_case
from tests.test_gpu_layer import STEP

pytestmark = pytest.mark.gpu
TOL = 2e-2
SHAPE = gen.TINY_QKN


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_qk_norm_layer_vs_oracle(mode):
    case = make_case(SHAPE, gen.batch_tiny(mode=mode))
    d = DevCase(case)
    b = case.batch
    h = B.Handle(SHAPE, 8, 512)
    y = STEP[mode](h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    torch.cuda.synchronize()
    (ref, inter), _ = case.run_oracle(intermediates=True)
    got = to_f32(y)
    assert np.isfinite(got).all()
    errs = per_request_maxrel(got, ref, b.row_offsets)
    assert max(errs) < TOL, errs
    # the new keys in the cache: the oracle's normalised and rotated k
    kc = OL.bf16_bits_to_f32(gen.bits(d.k.cpu()))
    bt = case.pool.block_tables.numpy()
    off = b.row_offsets
    rows = [(off[i] + j, int(b.context_lens[i]) + j, i) for i in range(b.num_seqs) for j in range(int(b.chunk_lens[i]))]
    got_k = np.stack([kc[bt[i, p // SHAPE.page_size], :, p % SHAPE.page_size, :] for _, p, i in rows])
    assert maxrel(got_k, np.stack([inter["k"][r] for r, _, _ in rows])) < TOL
    # and the norms matter: without them the keys are far from these (the
    # output moves less, the residual dominates it)
    plain = make_case(dataclasses.replace(SHAPE, qk_norm=False), b, weights=case.weights)
    (_, inter0), _ = plain.run_oracle(intermediates=True)
    assert maxrel(got_k, np.stack([inter0["k"][r] for r, _, _ in rows])) > 0.5


@pytest.mark.parametrize("mode", ["decode", "mixed"])
def test_qk_norm_layer_8bit_cache_vs_oracle(mode):
    case = code_case(SHAPE, gen.batch_tiny(mode=mode))
    b = case.batch
    k, v, bt = case.pool.k_cache.cuda(), case.pool.v_cache.cuda(), case.pool.block_tables.cuda()
    h = B.Handle(SHAPE, 8, 512)
    y = STEP[mode](h, {kk: t.cuda() for kk, t in case.weights.items()}, k, v, bt, b.context_lens, b.chunk_lens,
                   case.x.cuda(), kv_scales=(KS, VS))
    torch.cuda.synchronize()
    ref, _, _ = _oracle_step(case, (KS, VS))
    errs = per_request_maxrel(to_f32(y), ref, b.row_offsets)
    assert max(errs) < TOL, errs


def test_qk_norm_stack_vs_oracle():
    batch = gen.batch_tiny(mode="mixed")
    case = make_case(SHAPE, batch)
    Ws = [gen.make_weights(SHAPE, seed=500 + l) for l in range(2)]
    pools = [gen.make_kv_pool(SHAPE, batch, seed=600 + l, spare_pages=3) for l in range(2)]
    h = B.Handle(SHAPE, 8, 512)
    y = B.eb_stack_step(h, "mixed", [{k: t.cuda() for k, t in w.items()} for w in Ws],
                        [(p.k_cache.cuda(), p.v_cache.cuda(), p.block_tables.cuda()) for p in pools],
                        batch.context_lens, batch.chunk_lens, case.x.cuda())
    torch.cuda.synchronize()
    cfg = oracle_cfg(SHAPE)
    Wo = [oracle.prepare_weights({k: gen.bits(t) for k, t in w.items()}, cfg) for w in Ws]
    ref = OL.stack_step(cfg, Wo, [gen.bits(p.k_cache).copy() for p in pools],
                        [gen.bits(p.v_cache).copy() for p in pools], [p.block_tables.numpy() for p in pools],
                        batch.context_lens, batch.chunk_lens, gen.bits(case.x))
    errs = per_request_maxrel(to_f32(y), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


def test_qk_norm_entry_checks():
    case = make_case(SHAPE, gen.batch_tiny(mode="decode"))
    d = DevCase(case)
    b = case.batch
    h = B.Handle(SHAPE, 8, 512)
    hb = B.HostBatch(b.context_lens, b.chunk_lens)
    kv = B.kv_struct(d.k, d.v, d.bt)
    y = torch.empty_like(d.x)
    ws = B.alloc_workspace(B.lib().eb_workspace_bytes(h.h, ctypes.byref(hb.c), B.MODES["decode"]), "cuda")

    def run(lw):
        return B.lib().eb_layer_step_decode(h.h, ctypes.byref(lw), ctypes.byref(kv), ctypes.byref(hb.c),
                                            d.x.data_ptr(), y.data_ptr(), ws.data_ptr(), ws.numel(), None)
    lw = B.weights_struct(d.w)
    lw.k_norm = None
    assert run(lw) == -1                      # EB_ERR_NULL, nothing enqueued
    assert run(B.weights_struct(d.w)) == 0
    # the single RoPE entry has no gains: a handle with q/k norms is refused
    qkv = torch.zeros(b.num_tokens, SHAPE.qkv_rows, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(Exception) as e:
        B.eb_op_rope_kv_append(h, qkv, d.k, d.v, d.bt, b.context_lens, b.chunk_lens)
    assert getattr(e.value, "status", None) == -2   # EB_ERR_CONFIG
    torch.cuda.synchronize()

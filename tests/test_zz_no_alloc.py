"""The entry point that allocates nothing (eb_layer_step_mixed_noalloc): its
output equals eb_layer_step_mixed's on the same inputs, on two calls in a
row (the second over a smaller batch, so the fixed scratch still holds the
first call's larger contents), and a batch whose workspace exceeds the
fixed scratch is refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import oracle_cfg, tiny_case
from tests._gpu import DevCase, cache_bits, maxrel, per_request_maxrel, to_f32
from tests.test_gpu_layer import sub_pool_for_oracle

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _both(h, w, pool, batch, x):
    """y of the regular mixed step, then y of the no-allocation step, on the
    same inputs (the step rewrites the same cache slots with the same
    values, so the second sees the first's cache)."""
    args = (h, w, pool.k_cache, pool.v_cache, pool.block_tables, batch.context_lens, batch.chunk_lens, x)
    y_ref = B.eb_layer_step_mixed(*args)
    torch.cuda.synchronize()
    k_after = cache_bits(pool.k_cache)
    y_na = B.eb_layer_step_mixed_noalloc(*args)
    torch.cuda.synchronize()
    assert np.array_equal(cache_bits(pool.k_cache), k_after), "the two calls wrote different K"
    return to_f32(y_ref), to_f32(y_na)


def test_noalloc_equals_mixed_step_two_calls_8b():
    shape = gen.L8B
    w = {k: v.cuda() for k, v in gen.make_weights(shape).items()}
    big = gen.batch_8b_decode()
    small = big.subset(list(range(0, 64, 3)))
    h = B.Handle(shape, big.num_seqs, big.num_tokens)
    need_big = B.eb_workspace_bytes(h, big.context_lens, big.chunk_lens, "mixed")
    need_small = B.eb_workspace_bytes(h, small.context_lens, small.chunk_lens, "mixed")
    assert need_small < need_big <= B.eb_noalloc_scratch_bytes()
    Wo = oracle.prepare_weights({k: gen.bits(v.cpu()) for k, v in w.items()}, oracle_cfg(shape))
    for batch, sample in ((big, [0, 63]), (small, [0, small.num_seqs - 1])):
        pool = gen.make_kv_pool(shape, batch, device="cuda")
        kb, vb, bt = sub_pool_for_oracle(pool, batch, sample)
        x = gen.make_x(shape, batch.num_tokens).cuda()
        y_ref, y_na = _both(h, w, pool, batch, x)
        print(f"{batch.num_seqs} requests: bitwise equal {np.array_equal(y_ref, y_na)}")
        assert np.array_equal(y_ref, y_na)
        # and the oracle on sampled requests
        sub = batch.subset(sample)
        off = batch.row_offsets
        xs = np.concatenate([gen.bits(x.cpu())[off[i]:off[i + 1]] for i in sample])
        ref = oracle.layer_step(oracle_cfg(shape), Wo, kb, vb, bt, sub.context_lens, sub.chunk_lens, xs)
        so = sub.row_offsets
        errs = [maxrel(y_na[off[i]:off[i + 1]], ref[so[k]:so[k + 1]]) for k, i in enumerate(sample)]
        assert max(errs) < TOL, errs
        del pool


def test_noalloc_equals_mixed_step_tiny_modes():
    # a mixed batch, then its decode rows alone (smaller), on one handle
    case = tiny_case("mixed")
    d = DevCase(case)
    b = case.batch
    h = B.Handle(case.shape, b.num_seqs, b.num_tokens)
    pool = gen.KVPool(d.k, d.v, d.bt, case.pool.num_pages, case.pool.max_pages_per_seq)
    y_ref, y_na = _both(h, d.w, pool, b, d.x)
    assert np.array_equal(y_ref, y_na)
    ref, _ = case.run_oracle()
    assert max(per_request_maxrel(y_na, ref, b.row_offsets)) < TOL
    dec = np.nonzero(b.chunk_lens == 1)[0]
    sub = b.subset(dec)
    off = b.row_offsets
    xs = torch.cat([d.x[off[i]:off[i + 1]] for i in dec])
    pool2 = gen.KVPool(d.k, d.v, d.bt[torch.as_tensor(dec, device="cuda")].contiguous(), case.pool.num_pages,
                       case.pool.max_pages_per_seq)
    y_ref2, y_na2 = _both(h, d.w, pool2, sub, xs)
    assert np.array_equal(y_ref2, y_na2)


def test_noalloc_refuses_a_batch_beyond_the_scratch():
    shape = gen.L8B
    batch = gen.batch_8b_prefill()
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    assert B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, "mixed") > B.eb_noalloc_scratch_bytes()
    w = {k: torch.zeros(1, dtype=torch.bfloat16, device="cuda") for k in
         ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")}
    k = torch.zeros(1, shape.n_kv_heads, 16, shape.head_dim, dtype=torch.bfloat16, device="cuda")
    bt = torch.zeros(batch.num_seqs, 1, dtype=torch.int32, device="cuda")
    x = torch.zeros(batch.num_tokens, shape.hidden, dtype=torch.bfloat16, device="cuda")
    y = torch.full_like(x, 7.0)
    with pytest.raises(B.EbError) as ei:
        B.eb_layer_step_mixed_noalloc(h, w, k, k.clone(), bt, batch.context_lens, batch.chunk_lens, x, y=y)
    assert ei.value.status == -6
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())

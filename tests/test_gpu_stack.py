"""Model steps through the stack entry point: a batch through several
decoder layers, each with its own weights and paged cache (or one cache
shared by all), planned once.

* bitwise equal to the same layers run one after another through the single
  layer entry points (the stack only chains the layer bodies);
* against the oracle's stack (bf16 hand-off between layers) on the tiny
  shape, with separate and with shared caches;
* 70B-shaped layers: a full 256-request decode batch, sampled requests
  against the oracle, and the stack-equals-chained-layers property at that
  size;
* argument errors."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import oracle_cfg
from tests._gpu import cache_bits, check_cache_update, maxrel, per_request_maxrel, to_f32

pytestmark = pytest.mark.gpu
TOL = 2e-2
STEP = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill, "mixed": B.eb_layer_step_mixed}


def _layers(shape, batch, n, shared=False, proj_std=0.02, device="cuda"):
    ws = [{k: v.to(device) for k, v in gen.make_weights(shape, seed=500 + l, proj_std=proj_std).items()}
          for l in range(n)]
    pools = [gen.make_kv_pool(shape, batch, seed=600 + (0 if shared else l), spare_pages=3, device=device)
             for l in range(1 if shared else n)]
    x = gen.make_x(shape, batch.num_tokens, device=device)
    return ws, pools, x


def _same_bits(a: torch.Tensor, b: torch.Tensor) -> bool:
    # caches hold NaN poison outside the requests' slots: compare bit patterns
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def _caches(pools, n):
    return [(p.k_cache, p.v_cache, p.block_tables) for p in (pools * n if len(pools) == 1 else pools)]


@pytest.mark.parametrize("n", [1, 2, 3])
@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_stack_equals_chained_layer_steps(mode, n):
    shape = gen.TINY
    batch = gen.batch_tiny(mode=mode)
    ws, pools, x = _layers(shape, batch, n)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    chain = [p.clone() for p in pools]
    y = B.eb_stack_step(h, mode, ws, _caches(pools, n), batch.context_lens, batch.chunk_lens, x)
    cur = x
    for l in range(n):
        p = chain[l]
        cur = STEP[mode](h, ws[l], p.k_cache, p.v_cache, p.block_tables, batch.context_lens, batch.chunk_lens, cur)
    torch.cuda.synchronize()
    assert torch.equal(y, cur)
    for a, b in zip(pools, chain):
        assert _same_bits(a.k_cache, b.k_cache) and _same_bits(a.v_cache, b.v_cache)


@pytest.mark.parametrize("shared", [False, True])
def test_stack_vs_oracle(shared):
    shape = gen.TINY
    batch = gen.batch_tiny(mode="mixed")
    n = 3
    ws, pools, x = _layers(shape, batch, n, shared=shared, proj_std=0.05)
    cfg = oracle_cfg(shape)
    Ws = [oracle.prepare_weights({k: gen.bits(v) for k, v in w.items()}, cfg) for w in ws]
    kcs = [gen.bits(p.k_cache).copy() for p in pools]
    vcs = [gen.bits(p.v_cache).copy() for p in pools]
    bts = [p.block_tables.cpu().numpy() for p in pools]
    before_k = [k.copy() for k in kcs]
    idx = [0] * n if shared else list(range(n))
    ref = oracle.stack_step(cfg, Ws, [kcs[i] for i in idx], [vcs[i] for i in idx], [bts[i] for i in idx],
                            batch.context_lens, batch.chunk_lens, gen.bits(x))
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    y = to_f32(B.eb_stack_step(h, "mixed", ws, _caches(pools, n), batch.context_lens, batch.chunk_lens, x))
    torch.cuda.synchronize()
    errs = per_request_maxrel(y, ref, batch.row_offsets)
    print("per-request max-rel after", n, "layers:", errs)
    assert max(errs) < TOL, errs
    for p, kb, kr, bt in zip(pools, before_k, kcs, bts):
        check_cache_update(kb, cache_bits(p.k_cache), kr, batch, bt)


def test_stack_profile_sums_layers():
    shape = gen.TINY
    batch = gen.batch_tiny(mode="mixed")
    ws, pools, x = _layers(shape, batch, 4, shared=True)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    B.eb_profile(h, True)
    B.eb_stack_step(h, "mixed", ws, _caches(pools, 4), batch.context_lens, batch.chunk_lens, x)
    st = B.eb_profile_read(h)
    B.eb_profile(h, False)
    assert len(st) == 9 and all(v > 0 for v in st.values()), st


def test_stack_errors():
    shape = gen.TINY
    batch = gen.batch_tiny(mode="mixed")
    ws, pools, x = _layers(shape, batch, 2)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    with pytest.raises(ValueError):
        B.eb_stack_step(h, "mixed", ws, _caches(pools, 2)[:1], batch.context_lens, batch.chunk_lens, x)
    with pytest.raises(B.EbError) as ei:
        B.eb_stack_step(h, "mixed", [], [], batch.context_lens, batch.chunk_lens, x)
    assert ei.value.status == -2
    bad = dict(ws[1])
    bad["w_o"] = None
    with pytest.raises(B.EbError) as ei:
        B.eb_stack_step(h, "mixed", [ws[0], bad], _caches(pools, 2), batch.context_lens, batch.chunk_lens, x)
    assert ei.value.status == -1 and "layer 1" in str(ei.value)
    with pytest.raises(B.EbError) as ei:
        B.eb_stack_step(h, "decode", ws, _caches(pools, 2), batch.context_lens, batch.chunk_lens, x)
    assert ei.value.status == -4
    with pytest.raises(B.EbError) as ei:
        B.eb_stack_step(h, "mixed", ws, _caches(pools, 2), batch.context_lens, batch.chunk_lens, x,
                        ws=torch.empty(256, dtype=torch.uint8, device="cuda"))
    assert ei.value.status == -6
    # the single-layer workspace is one activation buffer short for a stack
    one = B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, "mixed")
    assert B.eb_stack_workspace_bytes(h, batch.context_lens, batch.chunk_lens, "mixed") > one


# ---------------------------------------------------------------- 70B shape

@pytest.fixture(scope="module")
def decode70():
    shape = gen.L70B
    batch = gen.batch_70b_decode()
    w = {k: v.cuda() for k, v in gen.make_weights(shape, seed=700).items()}
    pool = gen.make_kv_pool(shape, batch, device="cuda")
    x = gen.make_x(shape, batch.num_tokens, device="cuda")
    yield shape, batch, w, pool, x
    del w, pool, x
    torch.cuda.empty_cache()


def test_70b_decode_layer_full_size_sampled(decode70):
    from tests.test_gpu_layer import sub_pool_for_oracle
    shape, batch, w, pool, x = decode70
    sample = [0, 100, int(np.argmax(batch.context_lens)), 255]
    kb, vb, bt = sub_pool_for_oracle(pool, batch, sample)
    work = pool.clone()
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    y = to_f32(B.eb_layer_step_decode(h, w, work.k_cache, work.v_cache, work.block_tables, batch.context_lens,
                                      batch.chunk_lens, x))
    torch.cuda.synchronize()
    del work
    assert np.isfinite(y).all()
    Wo = oracle.prepare_weights({k: gen.bits(v) for k, v in w.items()}, oracle_cfg(shape))
    sub = batch.subset(sample)
    xs = gen.bits(x)[sample]
    ref = oracle.layer_step(oracle_cfg(shape), Wo, kb, vb, bt, sub.context_lens, sub.chunk_lens, xs)
    errs = [maxrel(y[i], ref[k]) for k, i in enumerate(sample)]
    print("70B decode sampled requests", sample, "ctx", list(sub.context_lens), "max-rel", errs)
    assert max(errs) < TOL, errs


def test_70b_decode_stack_equals_chained_layers(decode70):
    # three layers sharing one full-size cache, same weights in every layer
    # (the stack's chaining does not depend on which weights a layer has)
    shape, batch, w, pool, x = decode70
    n = 3
    a, b = pool.clone(), pool.clone()
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    y = B.eb_stack_step(h, "decode", [w] * n, [(a.k_cache, a.v_cache, a.block_tables)] * n, batch.context_lens,
                        batch.chunk_lens, x)
    cur = x
    for _ in range(n):
        cur = B.eb_layer_step_decode(h, w, b.k_cache, b.v_cache, b.block_tables, batch.context_lens,
                                     batch.chunk_lens, cur)
    torch.cuda.synchronize()
    assert torch.equal(y, cur)
    assert _same_bits(a.k_cache, b.k_cache) and _same_bits(a.v_cache, b.v_cache)
    assert torch.isfinite(y.float()).all()

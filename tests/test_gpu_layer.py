"""Whole-step parity of the three C-ABI entry points against the CPU oracle:
the tiny layer in all modes, EB-vs-MB per-request agreement, and the
8B-shaped workloads at full size with sampled requests checked by the
oracle (requests share no pages, so a subset is computed exactly as in the
whole batch)."""
import numpy as np
import pytest
import torch

import oracle
from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import Case, make_case, oracle_cfg, tiny_case
from tests._gpu import DevCase, cache_bits, check_cache_update, maxrel, per_request_maxrel, to_f32

pytestmark = pytest.mark.gpu
TOL = 2e-2
STEP = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill, "mixed": B.eb_layer_step_mixed}


def run_gpu(case: Case, mode: str, handle=None):
    d = DevCase(case)
    b = case.batch
    h = handle or B.Handle(case.shape, max(b.num_seqs, 1), max(b.num_tokens, 1))
    before_k, before_v = cache_bits(d.k), cache_bits(d.v)
    y = STEP[mode](h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    torch.cuda.synchronize()
    return to_f32(y), d, before_k, before_v


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_tiny_step_vs_oracle(mode):
    case = tiny_case(mode)
    y, d, bk, bv = run_gpu(case, mode)
    ref, o = case.run_oracle(mode="batched")
    assert np.isfinite(y).all()
    assert maxrel(y, ref) < TOL
    errs = per_request_maxrel(y, ref, case.batch.row_offsets)
    assert max(errs) < TOL, errs
    bt = case.pool.block_tables.numpy()
    check_cache_update(bk, cache_bits(d.k), o["k_cache"], case.batch, bt)
    check_cache_update(bv, cache_bits(d.v), o["v_cache"], case.batch, bt)


def test_tiny_step_sharp_attention():
    # Projections N(0, 0.08) give attention scores of standard deviation ~1.6
    # (q, k entries ~ 0.08 * sqrt(256)), so the softmax is far from uniform
    # and attention errors are not averaged away.  Much larger spreads make
    # the step ill-conditioned for bf16 intermediates: with scores of ~10 a
    # 2^-9 rounding of q alone moves single probabilities by several percent.
    shape = gen.TINY
    case = make_case(shape, gen.batch_tiny(mode="mixed"), weights=gen.make_weights(shape, proj_std=0.08))
    y, d, bk, bv = run_gpu(case, "mixed")
    ref, o = case.run_oracle(mode="batched")
    errs = per_request_maxrel(y, ref, case.batch.row_offsets)
    print("per-request max-rel", errs)
    assert max(errs) < TOL, errs


def test_eb_and_mb_agree_per_request():
    # each request's rows and written KV are the same whether it runs in an
    # exclusive batch (decode-only / prefill-only) or in the mixed batch
    mixed = gen.batch_tiny(mode="mixed")
    shape = gen.TINY
    case = make_case(shape, mixed)
    y_mb, d_mb, _, _ = run_gpu(case, "mixed")
    off = mixed.row_offsets
    dec_idx = np.nonzero(mixed.chunk_lens == 1)[0]
    pre_idx = np.nonzero(mixed.chunk_lens > 1)[0]
    bitwise = 0
    for idx, mode in ((dec_idx, "decode"), (pre_idx, "prefill")):
        sub = mixed.subset(idx)
        xs = torch.cat([case.x[off[i]:off[i + 1]] for i in idx])
        pool = gen.KVPool(case.pool.k_cache.clone(), case.pool.v_cache.clone(), case.pool.block_tables[idx].clone(),
                          case.pool.num_pages, case.pool.max_pages_per_seq)
        sc = Case(shape, case.weights, sub, pool, xs)
        y_eb, d_eb, _, _ = run_gpu(sc, mode)
        so = sub.row_offsets
        for k, i in enumerate(idx):
            a, b = y_eb[so[k]:so[k + 1]], y_mb[off[i]:off[i + 1]]
            assert maxrel(a, b) < TOL
            bitwise += int(np.array_equal(a, b))
        # written KV of those requests
        bt = case.pool.block_tables.numpy()
        for i in idx:
            for p in range(int(mixed.context_lens[i]), int(mixed.context_lens[i] + mixed.chunk_lens[i])):
                pg, sl = bt[i][p // 16], p % 16
                ke = cache_bits(d_eb.k)[pg, :, sl]
                km = cache_bits(d_mb.k)[pg, :, sl]
                assert maxrel(OL.bf16_bits_to_f32(ke), OL.bf16_bits_to_f32(km)) < TOL
    print(f"requests bitwise equal EB vs MB: {bitwise}/{mixed.num_seqs}")


def test_empty_batch_is_a_noop():
    shape = gen.TINY
    h = B.Handle(shape, 4, 64)
    w = {k: v.cuda() for k, v in gen.make_weights(shape).items()}
    e = np.zeros(0, np.int32)
    k = torch.zeros(2, shape.n_kv_heads, 16, shape.head_dim, dtype=torch.bfloat16, device="cuda")
    bt = torch.zeros(1, 1, dtype=torch.int32, device="cuda")
    x = torch.empty(0, shape.hidden, dtype=torch.bfloat16, device="cuda")
    for f in STEP.values():
        y = f(h, w, k, k.clone(), bt, e, e, x)
        assert y.shape == (0, shape.hidden)


def test_profile_ring_over_steps():
    # stage events of several steps in a ring of slots: a read averages the
    # recorded steps (here after the ring wrapped), off means nothing to read
    case = tiny_case("mixed")
    d = DevCase(case)
    b = case.batch
    h = B.Handle(case.shape, b.num_seqs, b.num_tokens)
    assert B.eb_profile_read(h) == {}
    B.eb_profile(h, True, steps=3)
    assert B.eb_profile_read(h) == {}
    for _ in range(5):
        STEP["mixed"](h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    st = B.eb_profile_read(h)
    assert len(st) == 9 and st["attention"] > 0 and st["qkv_gemm"] > 0, st
    assert all(v >= 0 for v in st.values()), st
    # one stage only: the others read 0
    B.eb_profile(h, True, steps=2, stages=["attention"])
    for _ in range(2):
        STEP["mixed"](h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    one = B.eb_profile_read(h)
    assert one["attention"] > 0 and all(v == 0 for k, v in one.items() if k != "attention"), one
    B.eb_profile(h, False)
    assert B.eb_profile_read(h) == {}
    assert B.lib().eb_profile(h.h, -1, 0) == -2  # EB_ERR_CONFIG
    assert B.lib().eb_profile(h.h, 1, 1 << 9) == -2


def test_step_errors_enqueue_nothing():
    shape = gen.TINY
    case = tiny_case("mixed")
    d = DevCase(case)
    b = case.batch
    h = B.Handle(shape, 8, 512)
    with pytest.raises(B.EbError) as ei:
        B.eb_layer_step_decode(h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    assert ei.value.status == -4
    with pytest.raises(B.EbError) as ei:
        B.eb_layer_step_mixed(h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x,
                              ws=torch.empty(256, dtype=torch.uint8, device="cuda"))
    assert ei.value.status == -6
    small = B.Handle(shape, 2, 512)
    with pytest.raises(B.EbError) as ei:
        B.eb_layer_step_mixed(small, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
    assert ei.value.status == -7


# ---------------------------------------------------------------- 8B shape

@pytest.fixture(scope="module")
def w8b():
    w = gen.make_weights(gen.L8B)
    Wo = oracle.prepare_weights({k: gen.bits(v) for k, v in w.items()}, oracle_cfg(gen.L8B))
    wd = {k: v.cuda() for k, v in w.items()}
    return wd, Wo


def sub_pool_for_oracle(pool: gen.KVPool, batch: gen.Batch, idx, codes: bool = False):
    """The pages of requests ``idx`` copied to the host under compact ids
    (``codes``: an 8-bit pool, copied as its uint8 codes)."""
    need = gen.pages_needed(batch)
    bt_host = pool.block_tables.cpu().numpy()
    pages, rows = [], []
    for i in idx:
        ids = bt_host[i, :need[i]]
        rows.append(np.arange(len(pages), len(pages) + len(ids)))
        pages.extend(ids.tolist())
    sel = torch.as_tensor(pages, dtype=torch.long, device=pool.k_cache.device)
    host = (lambda t: t.cpu().numpy()) if codes else gen.bits
    kb = host(pool.k_cache.index_select(0, sel))
    vb = host(pool.v_cache.index_select(0, sel))
    bt = np.full((len(idx), max(len(r) for r in rows)), -1, np.int32)
    for k, r in enumerate(rows):
        bt[k, :len(r)] = r
    return kb.copy(), vb.copy(), bt


def _sampled_parity(shape, batch, w, Wo, mode, sample, tol=TOL):
    pool = gen.make_kv_pool(shape, batch, device="cuda")
    # the sampled requests' pages as they are before the step
    kb, vb, bt = sub_pool_for_oracle(pool, batch, sample)
    x = gen.make_x(shape, batch.num_tokens)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    y = STEP[mode](h, w, pool.k_cache, pool.v_cache, pool.block_tables, batch.context_lens, batch.chunk_lens,
                   x.cuda())
    torch.cuda.synchronize()
    y = to_f32(y)
    assert np.isfinite(y).all()
    del pool
    # the sampled requests alone through the oracle
    sub = batch.subset(sample)
    off = batch.row_offsets
    xs = np.concatenate([gen.bits(x)[off[i]:off[i + 1]] for i in sample])
    ref = oracle.layer_step(oracle_cfg(shape), Wo, kb, vb, bt, sub.context_lens, sub.chunk_lens, xs)
    so = sub.row_offsets
    errs = [maxrel(y[off[i]:off[i + 1]], ref[so[k]:so[k + 1]]) for k, i in enumerate(sample)]
    print(f"{mode} {batch.label}: sampled requests {list(sample)} max-rel {errs}")
    assert max(errs) < tol, errs
    return errs


def test_8b_decode_full_size_sampled(w8b):
    w, Wo = w8b
    _sampled_parity(gen.L8B, gen.batch_8b_decode(), w, Wo, "decode", [0, 17, 40, 63])


def test_8b_prefill_full_size_sampled(w8b):
    w, Wo = w8b
    batch = gen.batch_8b_prefill()
    _sampled_parity(gen.L8B, batch, w, Wo, "prefill", [int(np.argmin(batch.chunk_lens))])


@pytest.mark.parametrize("r", [0.0, 0.5, 1.0])
def test_8b_mixed_budget_sampled(w8b, r):
    w, Wo = w8b
    batch = gen.batch_8b_mixed(r)
    dec = [int(i) for i in np.nonzero(batch.chunk_lens == 1)[0][:3]]
    pre = [int(i) for i in np.nonzero(batch.chunk_lens > 1)[0]]
    pre = [min(pre, key=lambda i: batch.chunk_lens[i])] if pre else []
    _sampled_parity(gen.L8B, batch, w, Wo, "mixed", dec + pre)


def test_debug_validate_reports_bad_block_tables(monkeypatch):
    # with EB_DEBUG_VALIDATE set when the handle is created, every step reads
    # its device block tables back and refuses bad ids and shared pages
    # before it enqueues anything; without it the same step runs
    case = tiny_case("mixed")
    d = DevCase(case)
    b = case.batch
    monkeypatch.setenv("EB_DEBUG_VALIDATE", "1")
    h = B.Handle(case.shape, b.num_seqs, b.num_tokens)
    monkeypatch.delenv("EB_DEBUG_VALIDATE")
    y = torch.full_like(d.x, 3.0)
    B.eb_layer_step_mixed(h, d.w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x, y=y)
    torch.cuda.synchronize()
    assert not bool((y == 3.0).all())
    for bad_value in ("out_of_range", "shared"):
        bt = d.bt.clone()
        if bad_value == "out_of_range":
            bt[1, 0] = case.pool.num_pages
        else:
            bt[1, 0] = bt[0, 0]
        y = torch.full_like(d.x, 3.0)
        k_before = cache_bits(d.k)
        with pytest.raises(B.EbError) as ei:
            B.eb_layer_step_mixed(h, d.w, d.k, d.v, bt, b.context_lens, b.chunk_lens, d.x, y=y)
        assert ei.value.status == -5, bad_value
        torch.cuda.synchronize()
        assert bool((y == 3.0).all()) and np.array_equal(cache_bits(d.k), k_before)
    # a release handle does not read the tables back
    h2 = B.Handle(case.shape, b.num_seqs, b.num_tokens)
    bt = d.bt.clone()
    bt[1, 0] = bt[0, 0]
    B.eb_layer_step_mixed(h2, d.w, d.k.clone(), d.v.clone(), bt, b.context_lens, b.chunk_lens, d.x)
    torch.cuda.synchronize()

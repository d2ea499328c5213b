"""8-bit (E4M3) KV cache through the C ABI against the oracle: the append
writes the codes the oracle computes (values bit-exact; rotated keys to
within one code where the bf16 rotation itself differs by an ulp), pure
paging of codes is bit-exact, attention in the three launch plans and whole
steps and stacks agree with the oracle run on the dequantized cache, and a
mixed launch equals separate launches bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fp8 as F
from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import Case, oracle_cfg
from tests._gpu import maxrel, per_request_maxrel, to_f32, written_slots

pytestmark = pytest.mark.gpu
TOL = 2e-2
KS, VS = 0.37, 0.61  # not powers of two: the append's fp32 division rounds


def _bf(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).to(torch.bfloat16)


def _codes(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().numpy().astype(np.uint8)


def code_case(shape, batch, poison=True, spare_pages=3, weights=None) -> Case:
    w = gen.make_weights(shape) if weights is None else weights
    pool = gen.make_kv_pool_codes(shape, batch, spare_pages=spare_pages, poison=poison)
    return Case(shape, w, batch, pool, gen.make_x(shape, batch.num_tokens))


def _fill_new_positions(case, seed=31):
    """Random codes (exponent field 4..9, as in the prior context) at the
    step's new positions, so attention can run without an append."""
    s, b = case.shape, case.batch
    kc, vc = _codes(case.pool.k_cache).copy(), _codes(case.pool.v_cache).copy()
    bt = case.pool.block_tables.numpy()
    rng = np.random.default_rng(seed)
    for i in range(b.num_seqs):
        c, n = int(b.context_lens[i]), int(b.chunk_lens[i])
        pos = c + np.arange(n)
        for arr in (kc, vc):
            v = (rng.integers(0, 2, (n, s.n_kv_heads, s.head_dim)) << 7) | \
                (rng.integers(4, 10, (n, s.n_kv_heads, s.head_dim)) << 3) | rng.integers(0, 8, (n, s.n_kv_heads, s.head_dim))
            arr[bt[i][pos // 16], :, pos % 16, :] = v.astype(np.uint8).transpose(0, 1, 2)
    case.pool.k_cache = torch.from_numpy(kc)
    case.pool.v_cache = torch.from_numpy(vc)
    return case


def _oracle_attention(case, qkv_bits):
    s, b = case.shape, case.batch
    nq, hd = s.n_q_heads, s.head_dim
    q = OL.bf16_bits_to_f32(qkv_bits)[:, :nq * hd].reshape(-1, nq, hd)
    kc, vc = _codes(case.pool.k_cache), _codes(case.pool.v_cache)
    bt = case.pool.block_tables.numpy()
    off = b.row_offsets
    out = np.zeros((b.num_tokens, nq * hd), np.float32)
    for i in range(b.num_seqs):
        c, n = int(b.context_lens[i]), int(b.chunk_lens[i])
        K = OL.gather_positions(kc, bt[i], c + n, 16, np.float32, KS)
        V = OL.gather_positions(vc, bt[i], c + n, 16, np.float32, VS)
        out[off[i]:off[i + 1]] = OL.causal_attention_seq(q[off[i]:off[i + 1]], K, V, c + np.arange(n),
                                                         s.group).reshape(n, -1)
    return out


ATT = {
    "tiny-decode": (gen.TINY, lambda: gen.batch_tiny(mode="decode")),
    "tiny-ragged": (gen.TINY, lambda: gen.Batch(np.array([0, 5, 31, 700, 1100, 16, 0], np.int32),
                                                 np.array([1, 37, 1, 1, 90, 16, 3], np.int32))),
    "8b-mixed-small": (gen.L8B, lambda: gen.Batch(np.array([1500, 0, 33, 2047, 517], np.int32),
                                                   np.array([1, 77, 1, 130, 1], np.int32))),
    "70b-shape-small": (gen.L70B, lambda: gen.Batch(np.array([600, 12, 1030], np.int32),
                                                     np.array([1, 40, 1], np.int32))),
}


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_rope_kv_append_codes(mode):
    case = code_case(gen.TINY, gen.batch_tiny(mode=mode))
    s, b = case.shape, case.batch
    k, v, bt_d = case.pool.k_cache.cuda(), case.pool.v_cache.cuda(), case.pool.block_tables.cuda()
    qkv = _bf((b.num_tokens, s.qkv_rows), 4)
    h = B.Handle(s, 8, 512)
    before_k, before_v = _codes(k), _codes(v)
    B.eb_op_rope_kv_append(h, qkv.cuda(), k, v, bt_d, b.context_lens, b.chunk_lens, kv_scales=(KS, VS))
    torch.cuda.synchronize()
    q32 = OL.bf16_bits_to_f32(gen.bits(qkv))
    nq, nkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
    kc, vc = before_k.copy(), before_v.copy()
    bt = case.pool.block_tables.numpy()
    off = b.row_offsets
    for i in range(b.num_seqs):
        rows = slice(off[i], off[i + 1])
        pos = b.context_lens[i] + np.arange(b.chunk_lens[i])
        kk = OL.rope(q32[rows, nq * hd:(nq + nkv) * hd].reshape(-1, nkv, hd), pos, s.rope_theta)
        vv = q32[rows, (nq + nkv) * hd:].reshape(-1, nkv, hd)
        OL.append_kv(kc, bt[i], pos, kk, 16, KS)
        OL.append_kv(vc, bt[i], pos, vv, 16, VS)
    got_k, got_v = _codes(k), _codes(v)
    slots = written_slots(b, bt)
    mask = np.zeros((before_k.shape[0], before_k.shape[2]), bool)
    for pg, sl in slots:
        mask[pg, sl] = True
    full = np.broadcast_to(mask[:, None, :, None], before_k.shape)
    for before, got in ((before_k, got_k), (before_v, got_v)):
        assert np.array_equal(before[~full], got[~full]), "cache bytes outside the new slots changed"
    # values are a plain copy: their codes are exact
    assert np.array_equal(got_v[full], vc[full])
    # rotated keys: the bf16 rotation may differ by an ulp, which can move a
    # code to its neighbour
    gk, rk = got_k[full].astype(np.int64), kc[full].astype(np.int64)
    diff = np.abs(gk - rk)
    assert np.all((diff == 0) | ((diff == 1) & ((gk & 0x80) == (rk & 0x80)))), "key code off by more than one step"
    assert np.mean(diff != 0) < 0.02


def test_gather_codes_bit_exact():
    case = code_case(gen.TINY, gen.batch_tiny(mode="mixed"), poison=False)
    b = case.batch
    h = B.Handle(case.shape, 8, 512)
    ok, ov = B.eb_op_gather_kv(h, case.pool.k_cache.cuda(), case.pool.v_cache.cuda(), case.pool.block_tables.cuda(),
                               b.context_lens, b.chunk_lens, kv_scales=(KS, VS))
    torch.cuda.synchronize()
    kc, vc = _codes(case.pool.k_cache), _codes(case.pool.v_cache)
    bt = case.pool.block_tables.numpy()
    refk, refv = [], []
    for i in range(b.num_seqs):
        p = np.arange(int(b.context_lens[i] + b.chunk_lens[i]))
        refk.append(kc[bt[i][p // 16], :, p % 16, :])
        refv.append(vc[bt[i][p // 16], :, p % 16, :])
    assert np.array_equal(_codes(ok), np.concatenate(refk))
    assert np.array_equal(_codes(ov), np.concatenate(refv))


@pytest.mark.parametrize("name", ["tiny-ragged", "8b-mixed-small", "70b-shape-small"])
@pytest.mark.parametrize("mode", ["prefill", "mixed"])
def test_attention_codes_vs_oracle(name, mode):
    shape, mk = ATT[name]
    batch = mk()
    case = _fill_new_positions(code_case(shape, batch, weights={}))
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 5)
    h = B.Handle(shape, 16, 1024)
    got = B.eb_op_attention(h, qkv.cuda(), case.pool.k_cache.cuda(), case.pool.v_cache.cuda(),
                            case.pool.block_tables.cuda(), batch.context_lens, batch.chunk_lens, mode=mode,
                            kv_scales=(KS, VS))
    torch.cuda.synchronize()
    ref = _oracle_attention(case, gen.bits(qkv))
    g = to_f32(got)
    assert np.isfinite(g).all(), "poisoned codes reached the output"
    errs = per_request_maxrel(g, ref, batch.row_offsets)
    assert max(errs) < TOL, errs


@pytest.mark.parametrize("name", ["tiny-decode", "8b-mixed-small", "70b-shape-small"])
def test_attention_codes_decode_plan(name):
    shape, mk = ATT[name]
    batch = mk()
    batch = batch.subset(np.nonzero(batch.chunk_lens == 1)[0])
    case = _fill_new_positions(code_case(shape, batch, weights={}))
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 6)
    h = B.Handle(shape, 16, 1024)
    got = B.eb_op_attention(h, qkv.cuda(), case.pool.k_cache.cuda(), case.pool.v_cache.cuda(),
                            case.pool.block_tables.cuda(), batch.context_lens, batch.chunk_lens, mode="decode",
                            kv_scales=(KS, VS))
    torch.cuda.synchronize()
    errs = per_request_maxrel(to_f32(got), _oracle_attention(case, gen.bits(qkv)), batch.row_offsets)
    assert max(errs) < TOL, errs


def test_mixed_launch_equals_separate_launches_codes():
    shape, mk = ATT["8b-mixed-small"]
    batch = mk()
    case = _fill_new_positions(code_case(shape, batch, weights={}))
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 9).cuda()
    args = (case.pool.k_cache.cuda(), case.pool.v_cache.cuda(), case.pool.block_tables.cuda(), batch.context_lens,
            batch.chunk_lens)
    h = B.Handle(shape, 16, 1024)
    a = B.eb_op_attention(h, qkv, *args, mode="mixed", kv_scales=(KS, VS))
    b = B.eb_op_attention(h, qkv, *args, mode="prefill", kv_scales=(KS, VS))
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


STEP = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill, "mixed": B.eb_layer_step_mixed}


def _oracle_step(case, kv_scales, mode="batched"):
    cfg = oracle_cfg(case.shape)
    W = oracle.prepare_weights({k: gen.bits(v) for k, v in case.weights.items()}, cfg)
    kc, vc = _codes(case.pool.k_cache).copy(), _codes(case.pool.v_cache).copy()
    y = OL.layer_step(cfg, W, kc, vc, case.pool.block_tables.numpy(), case.batch.context_lens,
                      case.batch.chunk_lens, gen.bits(case.x), mode=mode, kv_scales=kv_scales)
    return y, kc, vc


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_step_codes_vs_oracle(mode):
    case = code_case(gen.TINY, gen.batch_tiny(mode=mode))
    b = case.batch
    k, v, bt = case.pool.k_cache.cuda(), case.pool.v_cache.cuda(), case.pool.block_tables.cuda()
    h = B.Handle(case.shape, 8, 512)
    y = STEP[mode](h, {kk: t.cuda() for kk, t in case.weights.items()}, k, v, bt, b.context_lens, b.chunk_lens,
                   case.x.cuda(), kv_scales=(KS, VS))
    torch.cuda.synchronize()
    ref, kc, vc = _oracle_step(case, (KS, VS))
    got = to_f32(y)
    assert np.isfinite(got).all()
    errs = per_request_maxrel(got, ref, b.row_offsets)
    assert max(errs) < TOL, errs
    # every cached code decodes to the oracle's value to within one code step
    # plus the step's tolerance relative to the largest value: the kernels
    # round q/k/v to bf16 after the projection and again after RoPE, the
    # oracle once, and rotation can cancel most of a key's magnitude
    for got_c, ref_c in ((_codes(k), kc), (_codes(v), vc)):
        gk, rk = F.e4m3_decode(got_c), F.e4m3_decode(ref_c)
        assert np.array_equal(np.isnan(gk), np.isnan(rk)), \
            f"NaN codes differ at {np.argwhere(np.isnan(gk) != np.isnan(rk))[:8].tolist()}"
        fin = np.isfinite(rk)
        slack = TOL * np.max(np.abs(rk[fin]))
        bad = np.abs(gk[fin] - rk[fin]) > np.abs(rk[fin]) / 8 + 2.0 ** -9 + slack
        assert not bad.any(), (int(bad.sum()), gk[fin][bad][:8], rk[fin][bad][:8])


def test_step_codes_8b_decode_sampled():
    # 8B-shaped layer over 32 decode requests (contexts up to 4096): all rows
    # checked against the oracle on an 8-bit cache
    rng = np.random.default_rng(7)
    ctx = rng.integers(300, 4096, 32).astype(np.int32)
    batch = gen.Batch(ctx, np.ones(32, np.int32))
    case = code_case(gen.L8B, batch, spare_pages=2)
    k, v, bt = case.pool.k_cache.cuda(), case.pool.v_cache.cuda(), case.pool.block_tables.cuda()
    h = B.Handle(case.shape, 64, 64)
    y = B.eb_layer_step_decode(h, {kk: t.cuda() for kk, t in case.weights.items()}, k, v, bt, batch.context_lens,
                               batch.chunk_lens, case.x.cuda(), kv_scales=(KS, VS))
    torch.cuda.synchronize()
    ref, _, _ = _oracle_step(case, (KS, VS))
    errs = per_request_maxrel(to_f32(y), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


def test_stack_codes_vs_oracle():
    shape = gen.TINY
    batch = gen.batch_tiny(mode="mixed")
    case = code_case(shape, batch)
    n = 3
    Ws = [gen.make_weights(shape, seed=100 + l) for l in range(n)]
    scales = [(KS, VS), (0.5, 0.25), (1.3, 0.9)]
    pools = [gen.make_kv_pool_codes(shape, batch, seed=200 + l, spare_pages=3) for l in range(n)]
    caches = [(p.k_cache.cuda(), p.v_cache.cuda(), p.block_tables.cuda(), sc) for p, sc in zip(pools, scales)]
    h = B.Handle(shape, 8, 512)
    y = B.eb_stack_step(h, "mixed", [{k: t.cuda() for k, t in w.items()} for w in Ws], caches, batch.context_lens,
                        batch.chunk_lens, case.x.cuda())
    torch.cuda.synchronize()
    cfg = oracle_cfg(shape)
    Wo = [oracle.prepare_weights({k: gen.bits(t) for k, t in w.items()}, cfg) for w in Ws]
    ref = OL.stack_step(cfg, Wo, [_codes(p.k_cache).copy() for p in pools], [_codes(p.v_cache).copy() for p in pools],
                        [p.block_tables.numpy() for p in pools], batch.context_lens, batch.chunk_lens,
                        gen.bits(case.x), kv_scales=scales)
    errs = per_request_maxrel(to_f32(y), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


@pytest.mark.parametrize("scales", [(0.0, 1.0), (1.0, -1.0), (float("inf"), 1.0), (float("nan"), 1.0)])
def test_bad_scales_rejected(scales):
    case = code_case(gen.TINY, gen.batch_tiny(mode="decode"))
    b = case.batch
    h = B.Handle(case.shape, 8, 512)
    with pytest.raises(B.EbError):
        B.eb_layer_step_decode(h, {kk: t.cuda() for kk, t in case.weights.items()}, case.pool.k_cache.cuda(),
                               case.pool.v_cache.cuda(), case.pool.block_tables.cuda(), b.context_lens, b.chunk_lens,
                               case.x.cuda(), kv_scales=scales)

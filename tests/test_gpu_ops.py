"""Op-level parity of the HIP kernels against the CPU oracle, through the C
ABI: GEMM epilogues, RMSNorm, RoPE + paged append, dense KV gather
(bit-exact), attention in the three launch plans, one-hot attention
(bit-exact paging), poisoned pages."""
import numpy as np
import pytest
import torch

import oracle
from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import make_case, tiny_case
from tests._gpu import DevCase, cache_bits, maxrel, per_request_maxrel, to_f32

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _bf(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).to(torch.bfloat16)


# ---------------------------------------------------------------- GEMM

@pytest.mark.parametrize("M,N,K", [(1, 256, 256), (4, 512, 256), (64, 1376, 256), (37, 256, 688), (64, 6144, 4096),
                                   (130, 512, 256), (256, 688, 264), (512, 1024, 512), (300, 1376, 256),
                                   # 256-row weight streaming (70B-shaped decode batch), ragged rows
                                   (256, 10240, 8192), (200, 4104, 1024),
                                   # 256 x 256 LDS-streamed tiles: aligned, and ragged in M, N and F
                                   (1024, 8192, 1024), (1000, 8200, 512), (2048, 6144, 4096),
                                   # 256 x 256 tiles splitting K (few tiles): uneven splits, ragged M, N and F,
                                   # the 70B-shaped down projection
                                   (300, 1032, 2048), (256, 8192, 28672),
                                   # odd counts of 64-wide K tiles per block, and blocks of one or two K
                                   # tiles: one K range, and split K with uneven splits
                                   (512, 1032, 576), (768, 2048, 192), (272, 1024, 1344), (512, 1024, 128),
                                   (512, 1024, 64),
                                   # decode-sized row counts: one K stage, ragged N and F, split K, the
                                   # 8B-shaped down projection
                                   (63, 4104, 128), (17, 1032, 384), (1, 8200, 1152), (64, 4096, 14336)])
@pytest.mark.parametrize("epi", ["store", "residual", "silu_mul"])
def test_gemm(M, N, K, epi):
    A = _bf((M, K), 1)
    W = _bf((N, K), 2, 0.05)
    R = _bf((M, N), 3)
    a32 = OL.bf16_bits_to_f32(gen.bits(A))
    w32 = OL.bf16_bits_to_f32(gen.bits(W))
    prod = a32 @ w32.T
    if epi == "store":
        ref = prod
    elif epi == "residual":
        ref = prod + OL.bf16_bits_to_f32(gen.bits(R))
    else:
        F = N // 2
        ref = OL.silu(prod[:, :F]) * prod[:, F:]
    got = B.eb_op_gemm(A.cuda(), W.cuda(), epi, residual=R.cuda() if epi == "residual" else None)
    torch.cuda.synchronize()
    err = maxrel(to_f32(got), ref)
    assert err < TOL, err
    # rows are independent: a row's result does not depend on the others
    assert np.isfinite(to_f32(got)).all()


def test_gemm_empty_rows():
    A = torch.empty(0, 256, dtype=torch.bfloat16, device="cuda")
    W = _bf((256, 256), 2).cuda()
    out = B.eb_op_gemm(A, W)
    assert out.shape == (0, 256)


# ---------------------------------------------------------------- RMSNorm

@pytest.mark.parametrize("shape,rows", [(gen.TINY, 1), (gen.TINY, 133), (gen.L8B, 64)])
def test_rmsnorm(shape, rows):
    h = B.Handle(shape, 4, 256)
    x = _bf((rows, shape.hidden), 7)
    g = (1 + 0.1 * _bf((shape.hidden,), 8).float()).to(torch.bfloat16)
    got = to_f32(B.eb_op_rmsnorm(h, x.cuda(), g.cuda()))
    ref = OL.rmsnorm(OL.bf16_bits_to_f32(gen.bits(x)), OL.bf16_bits_to_f32(gen.bits(g)), shape.rms_eps)
    assert maxrel(got, ref) < 8e-3


# ---------------------------------------------------------------- paging

def _qkv_for(case, seed=11):
    s = case.shape
    return _bf((case.batch.num_tokens, s.qkv_rows), seed)


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_rope_kv_append(mode):
    case = tiny_case(mode)
    s, b = case.shape, case.batch
    d = DevCase(case)
    qkv = _qkv_for(case)
    h = B.Handle(s, 8, 512)
    before_k, before_v = cache_bits(d.k), cache_bits(d.v)
    q_dev = qkv.cuda()
    B.eb_op_rope_kv_append(h, q_dev, d.k, d.v, d.bt, b.context_lens, b.chunk_lens)
    torch.cuda.synchronize()
    # oracle: rotate q, k at their positions; append k, v
    off = b.row_offsets
    q32 = OL.bf16_bits_to_f32(gen.bits(qkv))
    nq, nkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
    ref_q = np.empty((b.num_tokens, nq, hd), np.float32)
    kc, vc = before_k.copy(), before_v.copy()
    bt = case.pool.block_tables.numpy()
    for i in range(b.num_seqs):
        rows = slice(off[i], off[i + 1])
        pos = b.context_lens[i] + np.arange(b.chunk_lens[i])
        ref_q[rows] = OL.rope(q32[rows, :nq * hd].reshape(-1, nq, hd), pos, s.rope_theta)
        k = OL.rope(q32[rows, nq * hd:(nq + nkv) * hd].reshape(-1, nkv, hd), pos, s.rope_theta)
        v = q32[rows, (nq + nkv) * hd:].reshape(-1, nkv, hd)
        OL.append_kv(kc, bt[i], pos, k, 16)
        OL.append_kv(vc, bt[i], pos, v, 16)
    got_q = to_f32(q_dev)[:, :nq * hd].reshape(-1, nq, hd)
    assert maxrel(got_q, ref_q) < 8e-3
    from tests._gpu import check_cache_update
    check_cache_update(before_k, cache_bits(d.k), kc, b, bt, tol=8e-3)
    check_cache_update(before_v, cache_bits(d.v), vc, b, bt, tol=0.0)   # v is a plain copy: exact


def test_gather_kv_bit_exact():
    case = tiny_case("mixed", poison=False)
    b = case.batch
    d = DevCase(case)
    h = B.Handle(case.shape, 8, 512)
    ok, ov = B.eb_op_gather_kv(h, d.k, d.v, d.bt, b.context_lens, b.chunk_lens)
    torch.cuda.synchronize()
    kb, vb = gen.bits(case.pool.k_cache), gen.bits(case.pool.v_cache)
    bt = case.pool.block_tables.numpy()
    refk, refv = [], []
    for i in range(b.num_seqs):
        n = int(b.context_lens[i] + b.chunk_lens[i])
        p = np.arange(n)
        refk.append(kb[bt[i][p // 16], :, p % 16, :])
        refv.append(vb[bt[i][p // 16], :, p % 16, :])
    assert np.array_equal(cache_bits(ok), np.concatenate(refk))
    assert np.array_equal(cache_bits(ov), np.concatenate(refv))


# ---------------------------------------------------------------- attention

def _oracle_attention(case, qkv_bits, k_bits, v_bits):
    """Oracle attention of every row from given roped q and a filled cache."""
    s, b = case.shape, case.batch
    nq, nkv, hd = s.n_q_heads, s.n_kv_heads, s.head_dim
    q = OL.bf16_bits_to_f32(qkv_bits)[:, :nq * hd].reshape(-1, nq, hd)
    bt = case.pool.block_tables.numpy()
    off = b.row_offsets
    out = np.zeros((b.num_tokens, nq * hd), np.float32)
    for i in range(b.num_seqs):
        c, n = int(b.context_lens[i]), int(b.chunk_lens[i])
        K = OL.gather_positions(k_bits, bt[i], c + n, 16)
        V = OL.gather_positions(v_bits, bt[i], c + n, 16)
        out[off[i]:off[i + 1]] = OL.causal_attention_seq(q[off[i]:off[i + 1]], K, V, c + np.arange(n),
                                                         s.group).reshape(n, -1)
    return out


def _filled_case(shape, batch, seed=21, poison=True):
    """A case whose cache already holds K/V for the step's new positions."""
    case = make_case(shape, batch, poison=poison, weights={})
    kb, vb = gen.bits(case.pool.k_cache).copy(), gen.bits(case.pool.v_cache).copy()
    bt = case.pool.block_tables.numpy()
    rng = np.random.default_rng(seed)
    for i in range(batch.num_seqs):
        c, n = int(batch.context_lens[i]), int(batch.chunk_lens[i])
        pos = c + np.arange(n)
        OL.append_kv(kb, bt[i], pos, rng.standard_normal((n, shape.n_kv_heads, shape.head_dim)).astype(np.float32), 16)
        OL.append_kv(vb, bt[i], pos, rng.standard_normal((n, shape.n_kv_heads, shape.head_dim)).astype(np.float32), 16)
    case.pool.k_cache = torch.from_numpy(kb.view(np.int16)).view(torch.bfloat16)
    case.pool.v_cache = torch.from_numpy(vb.view(np.int16)).view(torch.bfloat16)
    return case


ATT_BATCHES = {
    "tiny-decode": (gen.TINY, lambda: gen.batch_tiny(mode="decode")),
    "tiny-prefill": (gen.TINY, lambda: gen.batch_tiny(mode="prefill")),
    "tiny-mixed": (gen.TINY, lambda: gen.batch_tiny(mode="mixed")),
    # ragged tails, prefixes, a request at c = 0 and single-key decode,
    # long contexts with several splits
    "tiny-ragged": (gen.TINY, lambda: gen.Batch(np.array([0, 5, 31, 700, 1100, 16, 0], np.int32),
                                                 np.array([1, 37, 1, 1, 90, 16, 3], np.int32))),
    "8b-mixed-small": (gen.L8B, lambda: gen.Batch(np.array([1500, 0, 33, 2047, 517], np.int32),
                                                   np.array([1, 77, 1, 130, 1], np.int32))),
    "70b-shape-small": (gen.L70B, lambda: gen.Batch(np.array([600, 12, 1030], np.int32),
                                                     np.array([1, 40, 1], np.int32))),
    # decode work-order edges: last splits exactly full (512 and 1024 keys),
    # the short / split boundary (64 and 65 keys), last splits of 1 and 31
    # pages, and requests listed out of size order
    "8b-decode-edges": (gen.L8B, lambda: gen.Batch(np.array([511, 63, 64, 1023, 512, 1007, 3, 2000], np.int32),
                                                    np.ones(8, np.int32))),
}


@pytest.mark.parametrize("name", list(ATT_BATCHES))
@pytest.mark.parametrize("mode", ["prefill", "mixed"])
def test_attention_vs_oracle(name, mode):
    shape, mk = ATT_BATCHES[name]
    batch = mk()
    if mode == "decode" and (batch.chunk_lens != 1).any():
        pytest.skip("decode plan needs n = 1")
    case = _filled_case(shape, batch)
    d = DevCase(case)
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 5)
    h = B.Handle(shape, 16, 1024)
    got = B.eb_op_attention(h, qkv.cuda(), d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode=mode)
    torch.cuda.synchronize()
    ref = _oracle_attention(case, gen.bits(qkv), gen.bits(case.pool.k_cache), gen.bits(case.pool.v_cache))
    g = to_f32(got)
    assert np.isfinite(g).all()
    errs = per_request_maxrel(g, ref, batch.row_offsets)
    assert max(errs) < TOL, errs


@pytest.mark.parametrize("name", ["tiny-decode", "8b-mixed-small", "8b-decode-edges"])
def test_attention_decode_plan(name):
    shape, mk = ATT_BATCHES[name]
    batch = mk()
    batch = batch.subset(np.nonzero(batch.chunk_lens == 1)[0])
    case = _filled_case(shape, batch)
    d = DevCase(case)
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 6)
    h = B.Handle(shape, 16, 1024)
    got = B.eb_op_attention(h, qkv.cuda(), d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode="decode")
    torch.cuda.synchronize()
    ref = _oracle_attention(case, gen.bits(qkv), gen.bits(case.pool.k_cache), gen.bits(case.pool.v_cache))
    errs = per_request_maxrel(to_f32(got), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


@pytest.mark.parametrize("name", ["tiny-ragged", "8b-mixed-small", "70b-shape-small"])
def test_mixed_launch_equals_separate_launches(name):
    # the single mixed grid runs the same device code per item (its prefill
    # items hold 64 rows, the prefill-only launch's 128): bitwise equal
    shape, mk = ATT_BATCHES[name]
    batch = mk()
    case = _filled_case(shape, batch)
    d = DevCase(case)
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 9).cuda()
    h = B.Handle(shape, 16, 1024)
    a = B.eb_op_attention(h, qkv, d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode="mixed")
    b = B.eb_op_attention(h, qkv, d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode="prefill")
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("shape", [gen.TINY, gen.L8B, gen.L70B], ids=lambda s: s.name)
@pytest.mark.parametrize("target", [0, 15, 16, 17, 511, 512, 513, 700])
def test_one_hot_attention_bit_exact(shape, target):
    # q = e0 * 100 for every head, key `target` = e0 * 100, all other keys
    # = -e0 * 100: the score gap is far past fp32 exp underflow, so every row
    # that can see the target returns exactly that key's value vector.
    # long decode (2 splits), prefill from 0, prefill with a prefix, and a
    # short decode request (at most 64 keys: one wavefront per kv head)
    batch = gen.Batch(np.array([720, 0, 690, 40], np.int32), np.array([1, 64, 30, 1], np.int32))
    case = _filled_case(shape, batch)
    nq, nkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    kb = gen.bits(case.pool.k_cache).copy()
    bt = case.pool.block_tables.numpy()
    hundred = OL.f32_to_bf16_bits(np.array([100.0], np.float32))[0]
    minus = OL.f32_to_bf16_bits(np.array([-100.0], np.float32))[0]
    for i in range(batch.num_seqs):
        n_pos = int(batch.context_lens[i] + batch.chunk_lens[i])
        for p in range(n_pos):
            pg, sl = bt[i][p // 16], p % 16
            kb[pg, :, sl, :] = 0
            kb[pg, :, sl, 0] = hundred if p == target else minus
    case.pool.k_cache = torch.from_numpy(kb.view(np.int16)).view(torch.bfloat16)
    d = DevCase(case)
    qkv = torch.zeros(batch.num_tokens, shape.qkv_rows, dtype=torch.bfloat16)
    for hq in range(nq):
        qkv[:, hq * hd] = 100.0
    h = B.Handle(shape, 16, 1024)
    got = cache_bits(B.eb_op_attention(h, qkv.cuda(), d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens,
                                       mode="mixed"))
    torch.cuda.synchronize()
    vb = gen.bits(case.pool.v_cache)
    off = batch.row_offsets
    checked = 0
    for i in range(batch.num_seqs):
        c, n = int(batch.context_lens[i]), int(batch.chunk_lens[i])
        if target >= c + n:
            continue
        vt = vb[bt[i][target // 16], :, target % 16, :]          # [nkv, hd]
        want = np.concatenate([vt[hq // shape.group] for hq in range(nq)])
        for j in range(n):
            if c + j >= target:
                assert np.array_equal(got[off[i] + j], want), (i, j)
                checked += 1
    assert checked > 0 or target >= 720


def test_poisoned_pages_give_finite_output():
    # every slot outside the requests' positions holds NaN
    shape, mk = ATT_BATCHES["tiny-ragged"]
    batch = mk()
    case = _filled_case(shape, batch, poison=True)
    d = DevCase(case)
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 13).cuda()
    h = B.Handle(shape, 16, 1024)
    for mode in ("prefill", "mixed"):
        got = B.eb_op_attention(h, qkv, d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode=mode)
        torch.cuda.synchronize()
        assert torch.isfinite(got.float()).all()

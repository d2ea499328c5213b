"""8-bit (E4M3) weights with one scale per output row through the C ABI
against the oracle: the projection GEMM with every epilogue on every kernel
it can take (weight streaming with and without split K, more rows than a
streaming block holds, 256 x 256 tiles with and without split K), then whole
layer steps in the three modes, full-size 8B-shaped steps on sampled
requests, 8-bit weights over an 8-bit cache, and a stack whose layers mix the
two weight types."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from oracle import fp8 as F
from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import oracle_cfg
from tests._gpu import maxrel, per_request_maxrel, to_f32
from tests.test_gpu_layer import STEP, _sampled_parity

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _bf(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).to(torch.bfloat16)


_PROD = {}


def _reference_product(M, N, K):
    """A W^T in float32 with W = decode(code) * row scale (the oracle's
    reading of 8-bit weights), cached per shape across the epilogues."""
    key = (M, N, K)
    if key not in _PROD:
        _PROD.clear()
        A = _bf((M, K), 1)
        codes, scales = gen.make_fp8_matrix(N, K, seed=2)
        a32 = OL.bf16_bits_to_f32(gen.bits(A))
        c, s = codes.numpy(), scales.numpy()
        prod = np.empty((M, N), np.float32)
        step = max(1, (1 << 24) // K)   # dequantize a band of rows at a time
        for n0 in range(0, N, step):
            w = F.dequantize_rows(c[n0:n0 + step], s[n0:n0 + step]).astype(np.float32)
            prod[:, n0:n0 + step] = a32 @ w.T
        _PROD[key] = (A, codes, scales, prod)
    return _PROD[key]


@pytest.mark.parametrize("M,N,K", [
    # weight streaming: one row, ragged rows and K, split K, the 256-row 70B-shaped decode batch
    (1, 256, 256), (37, 256, 688), (64, 6144, 4096), (200, 4104, 1024), (256, 10240, 8192),
    # more rows than one streaming block, K not a multiple of the 64-wide tiles
    (300, 1376, 264), (520, 1024, 520),
    # 256 x 256 tiles: aligned, ragged in M, N and F
    (1024, 8192, 1024), (1000, 8200, 512), (2048, 6144, 4096),
    # 256 x 256 tiles splitting K: uneven splits and ragged shapes, the 70B-shaped down projection
    (300, 1032, 2048), (256, 8192, 28672),
    # decode-sized row counts: one K stage, ragged N and F, split K, the 8B-shaped down projection
    (63, 4104, 256), (17, 1032, 768), (5, 520, 512), (64, 4096, 14336)])
@pytest.mark.parametrize("epi", ["store", "residual", "silu_mul"])
def test_gemm_w8(M, N, K, epi):
    A, codes, scales, prod = _reference_product(M, N, K)
    R = _bf((M, N), 3)
    if epi == "store":
        ref = prod
    elif epi == "residual":
        ref = prod + OL.bf16_bits_to_f32(gen.bits(R))
    else:
        Fh = N // 2
        ref = OL.silu(prod[:, :Fh]) * prod[:, Fh:]
    got = B.eb_op_gemm_w8(A.cuda(), codes.cuda(), scales.cuda(), epi,
                          residual=R.cuda() if epi == "residual" else None)
    torch.cuda.synchronize()
    got = to_f32(got)
    assert np.isfinite(got).all()
    err = maxrel(got, ref)
    assert err < TOL, err


def test_gemm_w8_matches_scaled_bf16_product():
    # codes whose values times the scale are exact in bf16 (scales powers of
    # two): the 8-bit GEMM and the bf16 GEMM of the weights those codes stand
    # for form the same products, so they agree to accumulation order only
    M, N, K = 64, 512, 1024
    A = _bf((M, K), 5)
    codes, _ = gen.make_fp8_matrix(N, K, seed=6)
    scales = torch.from_numpy((2.0 ** np.random.default_rng(7).integers(-9, -4, N)).astype(np.float32))
    w = torch.from_numpy(F.dequantize_rows(codes.numpy(), scales.numpy()).astype(np.float32)).to(torch.bfloat16)
    assert np.array_equal(w.float().numpy(), F.dequantize_rows(codes.numpy(), scales.numpy()).astype(np.float32))
    got8 = to_f32(B.eb_op_gemm_w8(A.cuda(), codes.cuda(), scales.cuda()))
    got16 = to_f32(B.eb_op_gemm(A.cuda(), w.cuda()))
    torch.cuda.synchronize()
    assert maxrel(got8, got16) < 8e-3


def test_gemm_w8_empty_rows():
    A = torch.empty(0, 256, dtype=torch.bfloat16, device="cuda")
    codes, scales = gen.make_fp8_matrix(256, 256, seed=2)
    out = B.eb_op_gemm_w8(A, codes.cuda(), scales.cuda())
    assert out.shape == (0, 256)


def test_gemm_w8_argument_errors():
    # host-side checks: nothing is launched
    M, N, K = 4, 256, 256
    A = _bf((M, K), 1).cuda()
    codes, scales = gen.make_fp8_matrix(N, K, seed=2)
    codes = codes.cuda()
    sc = torch.zeros(N + 4, dtype=torch.float32, device="cuda")
    out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    lib = B.lib()
    args = lambda s: (ctypes.c_void_p(A.data_ptr()), ctypes.c_void_p(codes.data_ptr()), s,
                      ctypes.c_void_p(out.data_ptr()), None, M, N, K, 0, None, 0, None)
    assert lib.eb_op_gemm_w8(*args(None)) == -1                                    # EB_ERR_NULL
    assert lib.eb_op_gemm_w8(*args(ctypes.c_void_p(sc.data_ptr() + 4))) == -2     # misaligned: EB_ERR_CONFIG
    assert lib.eb_op_gemm_w8(*args(ctypes.c_void_p(sc.data_ptr()))) == 0
    torch.cuda.synchronize()


# ---------------------------------------------------------------- layer steps

def _oracle_weights(w, shape):
    return oracle.prepare_weights(gen.weight_arrays(w), oracle_cfg(shape))


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
def test_tiny_step_w8_vs_oracle(mode):
    shape = gen.TINY
    batch = gen.batch_tiny(mode=mode)
    w = gen.make_weights_fp8(shape)
    pool = gen.make_kv_pool(shape, batch, spare_pages=3)
    x = gen.make_x(shape, batch.num_tokens)
    h = B.Handle(shape, 8, 512)
    y = STEP[mode](h, {k: t.cuda() for k, t in w.items()}, pool.k_cache.cuda(), pool.v_cache.cuda(),
                   pool.block_tables.cuda(), batch.context_lens, batch.chunk_lens, x.cuda())
    torch.cuda.synchronize()
    ref = oracle.layer_step(oracle_cfg(shape), _oracle_weights(w, shape), gen.bits(pool.k_cache).copy(),
                            gen.bits(pool.v_cache).copy(), pool.block_tables.numpy(), batch.context_lens,
                            batch.chunk_lens, gen.bits(x))
    got = to_f32(y)
    assert np.isfinite(got).all()
    errs = per_request_maxrel(got, ref, batch.row_offsets)
    assert max(errs) < TOL, errs


def test_tiny_step_w8_over_fp8_cache():
    shape = gen.TINY
    batch = gen.batch_tiny(mode="mixed")
    ks, vs = 0.37, 0.61
    w = gen.make_weights_fp8(shape)
    pool = gen.make_kv_pool_codes(shape, batch, spare_pages=3)
    x = gen.make_x(shape, batch.num_tokens)
    h = B.Handle(shape, 8, 512)
    y = B.eb_layer_step_mixed(h, {k: t.cuda() for k, t in w.items()}, pool.k_cache.cuda(), pool.v_cache.cuda(),
                              pool.block_tables.cuda(), batch.context_lens, batch.chunk_lens, x.cuda(),
                              kv_scales=(ks, vs))
    torch.cuda.synchronize()
    kc = pool.k_cache.numpy().astype(np.uint8).copy()
    vc = pool.v_cache.numpy().astype(np.uint8).copy()
    ref = OL.layer_step(oracle_cfg(shape), _oracle_weights(w, shape), kc, vc, pool.block_tables.numpy(),
                        batch.context_lens, batch.chunk_lens, gen.bits(x), kv_scales=(ks, vs))
    errs = per_request_maxrel(to_f32(y), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


@pytest.fixture(scope="module")
def w8b_fp8():
    w = gen.make_weights_fp8(gen.L8B)
    Wo = _oracle_weights(w, gen.L8B)
    return {k: v.cuda() for k, v in w.items()}, Wo


def test_8b_decode_full_size_w8_sampled(w8b_fp8):
    w, Wo = w8b_fp8
    _sampled_parity(gen.L8B, gen.batch_8b_decode(), w, Wo, "decode", [0, 17, 40, 63])


def test_8b_prefill_full_size_w8_sampled(w8b_fp8):
    # thousands of rows: every projection on the 256 x 256 tiles
    w, Wo = w8b_fp8
    batch = gen.batch_8b_prefill()
    _sampled_parity(gen.L8B, batch, w, Wo, "prefill", [int(np.argmin(batch.chunk_lens))])


def test_8b_mixed_budget_w8_sampled(w8b_fp8):
    w, Wo = w8b_fp8
    batch = gen.batch_8b_mixed(0.5)
    dec = [int(i) for i in np.nonzero(batch.chunk_lens == 1)[0][:2]]
    pre = [int(i) for i in np.nonzero(batch.chunk_lens > 1)[0]]
    pre = [min(pre, key=lambda i: batch.chunk_lens[i])] if pre else []
    _sampled_parity(gen.L8B, batch, w, Wo, "mixed", dec + pre)


def test_stack_mixed_weight_types_vs_oracle():
    # layers 0 and 2 on 8-bit weights, layer 1 on bf16: each layer reads its own type
    shape = gen.TINY
    batch = gen.batch_tiny(mode="mixed")
    Ws = [gen.make_weights_fp8(shape, seed=100), gen.make_weights(shape, seed=101),
          gen.make_weights_fp8(shape, seed=102)]
    pools = [gen.make_kv_pool(shape, batch, seed=200 + l, spare_pages=3) for l in range(3)]
    x = gen.make_x(shape, batch.num_tokens)
    h = B.Handle(shape, 8, 512)
    caches = [(p.k_cache.cuda(), p.v_cache.cuda(), p.block_tables.cuda()) for p in pools]
    y = B.eb_stack_step(h, "mixed", [{k: t.cuda() for k, t in w.items()} for w in Ws], caches, batch.context_lens,
                        batch.chunk_lens, x.cuda())
    torch.cuda.synchronize()
    Wo = [_oracle_weights(w, shape) for w in Ws]
    ref = OL.stack_step(oracle_cfg(shape), Wo, [gen.bits(p.k_cache).copy() for p in pools],
                        [gen.bits(p.v_cache).copy() for p in pools], [p.block_tables.numpy() for p in pools],
                        batch.context_lens, batch.chunk_lens, gen.bits(x))
    errs = per_request_maxrel(to_f32(y), ref, batch.row_offsets)
    assert max(errs) < TOL, errs


def test_w8_weight_errors_enqueue_nothing():
    # a missing or misaligned row scale and an unknown weight type fail the
    # host checks before anything is enqueued
    shape = gen.TINY
    batch = gen.batch_tiny(mode="decode")
    w = {k: t.cuda() for k, t in gen.make_weights_fp8(shape).items()}
    pool = gen.make_kv_pool(shape, batch, spare_pages=3)
    x = gen.make_x(shape, batch.num_tokens).cuda()
    y = torch.empty_like(x)
    h = B.Handle(shape, 8, 512)
    hb = B.HostBatch(batch.context_lens, batch.chunk_lens)
    kv = B.kv_struct(pool.k_cache.cuda(), pool.v_cache.cuda(), pool.block_tables.cuda())
    ws = B.alloc_workspace(B.lib().eb_workspace_bytes(h.h, ctypes.byref(hb.c), B.MODES["decode"]), "cuda")

    def run(lw):
        return B.lib().eb_layer_step_decode(h.h, ctypes.byref(lw), ctypes.byref(kv), ctypes.byref(hb.c),
                                            x.data_ptr(), y.data_ptr(), ws.data_ptr(), ws.numel(), None)
    lw = B.weights_struct(w)
    lw.s_down = None
    assert run(lw) == -1                      # EB_ERR_NULL
    lw = B.weights_struct(w)
    lw.s_o = lw.s_o + 4
    assert run(lw) == -2                      # misaligned: EB_ERR_CONFIG
    lw = B.weights_struct(w)
    lw.w_dtype = 7
    assert run(lw) == -2                      # unknown type: EB_ERR_CONFIG
    assert run(B.weights_struct(w)) == 0
    torch.cuda.synchronize()

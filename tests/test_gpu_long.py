"""Long contexts (the paper's 128K-input runs, App. A.1) and operands past
the 32-bit buffer range, through the C ABI against the oracle."""
import numpy as np
import pytest
import torch

from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._gpu import DevCase, maxrel, per_request_maxrel, to_f32
from tests.test_gpu_ops import _bf, _filled_case, _oracle_attention

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.mark.parametrize("mode", ["decode", "mixed"])
def test_decode_attention_near_128k(mode):
    # two decode requests with contexts of 131000 and 70000 tokens (256 and
    # 137 splits of 512 keys, combined by the log-sum-exp kernel)
    shape = gen.L8B
    batch = gen.Batch(np.array([131000, 70000], np.int32), np.array([1, 1], np.int32))
    case = _filled_case(shape, batch, poison=True)
    d = DevCase(case)
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 31)
    h = B.Handle(shape, 4, 64)
    got = B.eb_op_attention(h, qkv.cuda(), d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode=mode)
    torch.cuda.synchronize()
    ref = _oracle_attention(case, gen.bits(qkv), gen.bits(case.pool.k_cache), gen.bits(case.pool.v_cache))
    g = to_f32(got)
    assert np.isfinite(g).all()
    errs = per_request_maxrel(g, ref, batch.row_offsets)
    print("128K decode per-request max-rel", errs)
    assert max(errs) < TOL, errs


def test_prefill_chunk_over_a_100k_prefix():
    # a 96-row chunk whose queries see a 100000-token paged prefix, with a
    # decode request alongside in the mixed launch
    shape = gen.L8B
    batch = gen.Batch(np.array([100000, 3000], np.int32), np.array([96, 1], np.int32))
    case = _filled_case(shape, batch, poison=True)
    d = DevCase(case)
    qkv = _bf((batch.num_tokens, shape.qkv_rows), 32)
    h = B.Handle(shape, 4, 256)
    for mode in ("prefill", "mixed"):
        got = B.eb_op_attention(h, qkv.cuda(), d.k, d.v, d.bt, batch.context_lens, batch.chunk_lens, mode=mode)
        torch.cuda.synchronize()
        ref = _oracle_attention(case, gen.bits(qkv), gen.bits(case.pool.k_cache), gen.bits(case.pool.v_cache))
        errs = per_request_maxrel(to_f32(got), ref, batch.row_offsets)
        assert max(errs) < TOL, (mode, errs)


@pytest.mark.parametrize("epi", ["store", "residual"])
def test_gemm_with_activations_past_2gib(epi):
    # A = 75000 x 14336 bf16 (2.15 GB, the down projection of a
    # single-iteration 75K-token prompt): the 256x256-tile kernel runs in row
    # chunks that each fit a 32-bit buffer range; rows on both sides of the
    # chunk boundary and at the ends are checked against fp64
    M, K, N = 75000, 14336, 256
    g = torch.Generator(device="cuda").manual_seed(41)
    A = torch.randn(M, K, generator=g, device="cuda").to(torch.bfloat16)
    W = (torch.randn(N, K, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    R = torch.randn(M, N, generator=g, device="cuda").to(torch.bfloat16)
    out = B.eb_op_gemm(A, W, epi, residual=R if epi == "residual" else None)
    torch.cuda.synchronize()
    chunk = ((2 ** 31 - 1) // (K * 2)) // 256 * 256
    rows = [0, 1, chunk - 1, chunk, chunk + 1, M - 2, M - 1]
    a = OL.bf16_bits_to_f32(gen.bits(A[rows])).astype(np.float64)
    w = OL.bf16_bits_to_f32(gen.bits(W)).astype(np.float64)
    ref = a @ w.T
    if epi == "residual":
        ref = ref + OL.bf16_bits_to_f32(gen.bits(R[rows])).astype(np.float64)
    got = to_f32(out[rows])
    assert maxrel(got, ref) < TOL
    del A, W, R, out
    torch.cuda.empty_cache()

"""The mixture-of-experts block through the C ABI against the oracle.

The routing is an integer decision taken from floating-point logits, so the
HIP path's choice is checked for validity instead of identity: every chosen
expert's oracle logit reaches the token's k-th largest oracle logit (up to
the fp32 summation error), the ids are distinct and in logit order, and the
weights equal the oracle's weights for that choice.  The block's output is
then compared element by element with the oracle evaluated under the same
choice.  Cases: ragged token counts (one token, fewer tokens than a tile,
several tiles per expert, enough rows per expert for the 256 x 256 kernel),
the Qwen3-30B-A3B shape at a decode and a prefill batch, routing
that sends every token to the same experts (empty experts, one expert with
many row tiles), plain softmax weights, and argument errors."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import moe as MO
from oracle import layer as OL
from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._gpu import maxrel, to_f32

pytestmark = pytest.mark.gpu
TOL = 2e-2


def _case(shape, T, seed=0):
    w = gen.make_moe_weights(shape, seed=seed)
    g = torch.Generator().manual_seed(seed + 1)
    b = torch.randn(T, shape.hidden, generator=g).to(torch.bfloat16)
    res = torch.randn(T, shape.hidden, generator=g).to(torch.bfloat16)
    return w, b, res


def _check(shape, w, b, res, renormalize=True, min_same=0.9):
    k = shape.top_k
    out, ids, wts = B.eb_op_moe_ffn(b.cuda(), w["w_router"].cuda(), w["w_gate_up"].cuda(), w["w_down"].cuda(), k,
                                    residual=res.cuda() if res is not None else None, renormalize=renormalize,
                                    return_routing=True)
    torch.cuda.synchronize()
    ids = ids.cpu().numpy().astype(np.int64)
    wts = wts.cpu().numpy().astype(np.float64)
    bb, wr = gen.bits(b), gen.bits(w["w_router"])
    logits = MO.router_logits(bb, wr)
    T = b.shape[0]
    # a valid top-k of the oracle's logits
    slack = 1e-4 * max(1.0, float(np.max(np.abs(logits))))
    kth = -np.sort(-logits, axis=1)[:, k - 1]
    chosen = np.take_along_axis(logits, ids, axis=1)
    assert ids.min() >= 0 and ids.max() < shape.n_experts
    assert all(len(set(r)) == k for r in ids), "repeated expert in a token's choice"
    assert np.all(chosen >= kth[:, None] - slack), "an expert outside the top k"
    assert np.all(np.diff(chosen, axis=1) <= slack), "experts not in logit order"
    same = np.mean(np.all(ids == MO.top_k_experts(logits, k), axis=1))
    assert same >= min_same, same
    # weights: the oracle's for that choice
    ref_w = MO.routing_weights(logits, ids, renormalize)
    assert np.allclose(wts, ref_w, rtol=1e-4, atol=1e-6), np.max(np.abs(wts - ref_w))
    # the block under that choice
    ref = MO.moe_ffn(bb, wr, gen.bits(w["w_gate_up"]), gen.bits(w["w_down"]), k, renormalize, ids=ids,
                     weights=ref_w)
    if res is not None:
        ref = ref + OL.bf16_bits_to_f32(gen.bits(res))
    got = to_f32(out)
    assert np.isfinite(got).all()
    err = maxrel(got, ref)
    assert err < TOL, err
    return ids, err


@pytest.mark.parametrize("T", [1, 7, 100, 333,
                               # 128 or more rows per expert: the 256 x 256 kernel on tiles of up to 256 rows
                               600, 1500])
def test_moe_small_vs_oracle(T):
    w, b, res = _case(gen.MOE_TINY, T)
    _check(gen.MOE_TINY, w, b, res)


def test_moe_plain_softmax_weights_no_residual():
    w, b, _ = _case(gen.MOE_TINY, 50, seed=3)
    _check(gen.MOE_TINY, w, b, None, renormalize=False)


def test_moe_30b_shape_decode_batch():
    # Qwen3-30B-A3B block at a 64-token decode batch: almost every expert hit
    w, b, res = _case(gen.MOE30B, 64, seed=5)
    ids, _ = _check(gen.MOE30B, w, b, res)
    assert len(np.unique(ids)) > 100


def test_moe_30b_shape_prefill_batch():
    # 2048 tokens, 128 rows per expert on average: the 256 x 256 kernel
    w, b, res = _case(gen.MOE30B, 2048, seed=9)
    _check(gen.MOE30B, w, b, res)


@pytest.mark.parametrize("T", [300, 600])
def test_moe_every_token_to_the_same_experts(T):
    # a constant input feature and a router that scores experts 0..k-1 far
    # above the rest on it: each of them receives every token (300: five
    # 64-row tiles; 600: three tiles of up to 256 rows), twelve receive none
    shape = gen.MOE_TINY
    w, b, res = _case(shape, T, seed=7)
    b[:, 0] = 8.0
    wr = (w["w_router"].float() * 1e-3)
    wr[:, 0] = -4.0
    wr[:shape.top_k, 0] = torch.arange(shape.top_k, 0, -1, dtype=torch.float32)
    w["w_router"] = wr.to(torch.bfloat16)
    ids, _ = _check(shape, w, b, res, min_same=1.0)
    assert np.array_equal(np.sort(np.unique(ids)), np.arange(shape.top_k))


def test_moe_empty_and_argument_errors():
    shape = gen.MOE_TINY
    w, b, res = _case(shape, 4)
    wd = {k: v.cuda() for k, v in w.items()}
    empty = torch.empty(0, shape.hidden, dtype=torch.bfloat16, device="cuda")
    assert B.eb_op_moe_ffn(empty, wd["w_router"], wd["w_gate_up"], wd["w_down"], shape.top_k).shape == (0, shape.hidden)
    L = B.lib()
    out = torch.empty(4, shape.hidden, dtype=torch.bfloat16, device="cuda")
    bc = b.cuda()

    def call(E, k, d=shape.hidden, F=shape.expert_ffn, ptr=True):
        return L.eb_op_moe_ffn(bc.data_ptr() if ptr else None, None, wd["w_router"].data_ptr(),
                               wd["w_gate_up"].data_ptr(), wd["w_down"].data_ptr(), 4, d, E, k, F, 1,
                               out.data_ptr(), None, None, None, 0, None)
    assert call(20, 4) == -2          # E not a multiple of 16
    assert call(16, 17) == -2         # top_k above E
    assert call(16, 4, d=200) == -2   # d not a multiple of 32
    assert call(16, 4, ptr=False) == -1
    assert call(16, 4) == -6          # no workspace
    torch.cuda.synchronize()

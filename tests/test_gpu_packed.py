"""Fragment-packed weights.  The packed copy against its definition (each
16 x 32 block of W as one 1 KiB run in the lane order of the 16x16x32 bf16
matrix-core operand: lane l holds row 16 g + l % 16, columns
32 c + 8 (l / 16) .. + 7), and layer steps whose weight-streaming GEMMs read
packed copies against the same steps on the row-major matrices: the kernels
take the same operands in the same order, so the outputs must agree bit for
bit; the packed steps also against the oracle."""
import numpy as np
import pytest
import torch

from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen
from tests._cases import make_case
from tests._gpu import DevCase, cache_bits, maxrel, per_request_maxrel, to_f32

pytestmark = pytest.mark.gpu
STEP = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill, "mixed": B.eb_layer_step_mixed}
# every projection of this shape has a packed form (the tiny layer's down
# projection, K = 688, has none and stays on the row-major path)
MID = gen.LayerShape("mid", 1024, 8, 2, 128, 2048, 1e6)


def packed_by_loops(W: np.ndarray) -> np.ndarray:
    rows, cols = W.shape
    out = np.empty(rows * cols, np.uint16)
    q = 0
    for g in range(rows // 16):
        for c in range(cols // 32):
            for lane in range(64):
                r, k = 16 * g + lane % 16, 32 * c + 8 * (lane // 16)
                out[q:q + 8] = W[r, k:k + 8]
                q += 8
    return out


def packed_by_reshape(W: np.ndarray) -> np.ndarray:
    rows, cols = W.shape
    return W.reshape(rows // 16, 16, cols // 32, 4, 8).transpose(0, 2, 3, 1, 4).reshape(-1)


def bits16(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("rows,cols", [(16, 32), (48, 96), (64, 4096), (6144, 4096)])
def test_pack_weight_layout(rows, cols):
    g = torch.Generator().manual_seed(rows * 7 + cols)
    W = (torch.randn(rows, cols, generator=g) * 0.02).to(torch.bfloat16)
    P = B.eb_pack_weight(W.cuda())
    torch.cuda.synchronize()
    Wb = bits16(W).reshape(rows, cols)
    ref = packed_by_reshape(Wb)
    if rows * cols <= 48 * 96:
        assert np.array_equal(packed_by_loops(Wb), ref)
    assert np.array_equal(bits16(P), ref)


def _steps(shape, batch, mode):
    """The step on row-major weights and on packed copies, each on a fresh
    copy of the same inputs: (y, k, v) bits of both, the oracle's y, and the
    packed-weights dict."""
    case = make_case(shape, batch)
    outs = []
    for packed in (False, True):
        d = DevCase(case)
        w = B.pack_layer_weights(d.w) if packed else d.w
        b = case.batch
        h = B.Handle(case.shape, b.num_seqs, b.num_tokens)
        y = STEP[mode](h, w, d.k, d.v, d.bt, b.context_lens, b.chunk_lens, d.x)
        torch.cuda.synchronize()
        outs.append((bits16(y), cache_bits(d.k), cache_bits(d.v), to_f32(y), w))
    ref, _ = case.run_oracle(mode="batched")
    return outs, ref, case


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed"])
@pytest.mark.parametrize("shape", [gen.TINY, MID], ids=["tiny", "mid"])
def test_packed_step_bitwise_and_vs_oracle(shape, mode):
    ((y0, k0, v0, _, _), (y1, k1, v1, yf, w)), ref, case = _steps(shape, gen.batch_tiny(mode=mode), mode)
    packed = {k for k in ("p_qkv", "p_o", "p_gate_up", "p_down") if k in w}
    assert packed == ({"p_qkv", "p_o", "p_gate_up"} if shape is gen.TINY else {"p_qkv", "p_o", "p_gate_up", "p_down"})
    assert np.array_equal(y0, y1)
    assert np.array_equal(k0, k1) and np.array_equal(v0, v1)
    assert maxrel(yf, ref) < 2e-2
    assert max(per_request_maxrel(yf, ref, case.batch.row_offsets)) < 2e-2


@pytest.mark.parametrize("mode", ["decode", "mixed"])
def test_packed_8b_full_size_bitwise(mode):
    # the 8B-shaped decode batch (qkv with the first RMSNorm folded in, o and
    # down split over K, gate/up unsplit) and a 192-row mixed step (steps of
    # 256 rows and more take the 256 x 256 tiled GEMMs on row-major weights)
    shape = gen.L8B
    batch = gen.batch_8b_decode() if mode == "decode" else gen.batch_8b_mixed(0.1, budget=192)
    assert batch.num_tokens < 256
    w = {k: v.cuda() for k, v in gen.make_weights(shape).items()}
    wp = B.pack_layer_weights(w)
    assert all(k in wp for k in ("p_qkv", "p_o", "p_gate_up", "p_down"))
    pool = gen.make_kv_pool(shape, batch, device="cuda")
    x = gen.make_x(shape, batch.num_tokens).cuda()
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    ys = []
    for ww in (w, wp, w):  # the step rewrites the same cache slots with the same values
        y = STEP[mode](h, ww, pool.k_cache, pool.v_cache, pool.block_tables, batch.context_lens, batch.chunk_lens, x)
        torch.cuda.synchronize()
        ys.append(bits16(y))
    assert np.array_equal(ys[0], ys[2])
    assert np.array_equal(ys[0], ys[1])
    assert np.isfinite(to_f32(y)).all()


def test_packed_stack_bitwise():
    # a two-layer model step with one layer packed and one not
    shape = MID
    batch = gen.batch_tiny(mode="mixed")
    outs = []
    cases = [make_case(shape, batch, weights=gen.make_weights(shape, seed=100 + layer), kv_seed=200 + layer)
             for layer in range(2)]
    for pack in ((False, False), (True, False), (False, True)):
        ws, caches = [], []
        for layer in range(2):
            d = DevCase(cases[layer])  # fresh cache copies for every run
            ws.append(B.pack_layer_weights(d.w) if pack[layer] else d.w)
            caches.append((d.k, d.v, d.bt))
        h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
        x = d.x
        y = B.eb_stack_step(h, "mixed", ws, caches, batch.context_lens, batch.chunk_lens, x)
        torch.cuda.synchronize()
        outs.append(bits16(y))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])

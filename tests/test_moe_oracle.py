"""Pins of the oracle's mixture-of-experts block (oracle/moe.py) to things
other than itself: the transformers Qwen3-MoE sparse block in float64 (the
model family the paper measures, Sec. 4.1 "Models"), with and without
renormalised top-k weights; one expert reducing to the transformers dense
MLP; the top-k rule on equal logits; invariance under relabelling experts;
and planted mistakes that must fail the transformers pin."""
import numpy as np
import pytest
import torch

from oracle import moe as MO
from oracle import layer as OL

pytestmark = pytest.mark.filterwarnings("ignore")


def _bits(rng, shape, scale):
    return OL.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def _inputs(T=9, d=64, E=16, F=32, seed=0):
    rng = np.random.default_rng(seed)
    return dict(b=_bits(rng, (T, d), 1.0), wr=_bits(rng, (E, d), 0.3),
                wgu=_bits(rng, (E, 2 * F, d), 0.1), wd=_bits(rng, (E, d, F), 0.1))


def _f64(bits):
    return torch.from_numpy(OL.bf16_bits_to_f32(bits).astype(np.float64))


def _hf_block(o, k, renormalize):
    from transformers.models.qwen3_moe.configuration_qwen3_moe import Qwen3MoeConfig
    from transformers.models.qwen3_moe import modeling_qwen3_moe as m
    E, twoF, d = o["wgu"].shape
    cfg = Qwen3MoeConfig(hidden_size=d, num_experts=E, num_experts_per_tok=k, moe_intermediate_size=twoF // 2,
                         norm_topk_prob=renormalize, hidden_act="silu")
    cfg._experts_implementation = "eager"
    blk = m.Qwen3MoeSparseMoeBlock(cfg).double()
    with torch.no_grad():
        blk.gate.weight.copy_(_f64(o["wr"]))
        blk.experts.gate_up_proj.copy_(_f64(o["wgu"]))
        blk.experts.down_proj.copy_(_f64(o["wd"]))
    return blk


def _hf(o, k, renormalize):
    blk = _hf_block(o, k, renormalize)
    x = _f64(o["b"])
    with torch.no_grad():
        _, w, ids = blk.gate(x)
        y = blk(x[None])[0]
    return ids.numpy(), w.numpy(), y.numpy()


@pytest.mark.parametrize("k,renormalize", [(4, True), (4, False), (1, True), (16, True)])
def test_block_matches_transformers(k, renormalize):
    o = _inputs()
    ids_hf, w_hf, y_hf = _hf(o, k, renormalize)
    ids, w, _ = MO.route(o["b"], o["wr"], k, renormalize)
    # the same experts in the same order (random logits: no ties), the same
    # weights (transformers takes the softmax in float32 whatever the input
    # type, hence 1e-6)
    assert np.array_equal(ids, ids_hf)
    assert np.allclose(w, w_hf, rtol=1e-6, atol=0)
    y = MO.moe_ffn(o["b"], o["wr"], o["wgu"], o["wd"], k, renormalize)
    assert np.max(np.abs(y - y_hf)) <= 1e-6 * np.max(np.abs(y_hf))
    # and exactly the block given transformers' own routing
    y2 = MO.moe_ffn(o["b"], o["wr"], o["wgu"], o["wd"], k, renormalize, ids=ids_hf, weights=w_hf)
    assert np.max(np.abs(y2 - y_hf)) <= 1e-12 * np.max(np.abs(y_hf))


def test_one_expert_is_the_dense_mlp():
    from transformers.models.qwen3_moe.configuration_qwen3_moe import Qwen3MoeConfig
    from transformers.models.qwen3_moe import modeling_qwen3_moe as m
    o = _inputs(E=1)
    F = o["wgu"].shape[1] // 2
    cfg = Qwen3MoeConfig(hidden_size=64, intermediate_size=F, hidden_act="silu")
    mlp = m.Qwen3MoeMLP(cfg, intermediate_size=F).double()
    with torch.no_grad():
        mlp.gate_proj.weight.copy_(_f64(o["wgu"][0, :F]))
        mlp.up_proj.weight.copy_(_f64(o["wgu"][0, F:]))
        mlp.down_proj.weight.copy_(_f64(o["wd"][0]))
        ref = mlp(_f64(o["b"])).numpy()
    y = MO.moe_ffn(o["b"], o["wr"], o["wgu"], o["wd"], 1, True)
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_equal_logits_take_the_lower_expert():
    o = _inputs(E=8)
    wr = o["wr"].copy()
    wr[5] = wr[2]          # experts 2 and 5 always score the same
    wr[7] = wr[2]
    logits = MO.router_logits(o["b"], wr)
    ids = MO.top_k_experts(logits, 8)
    for t in range(ids.shape[0]):
        pos = {e: i for i, e in enumerate(ids[t])}
        assert pos[2] < pos[5] < pos[7]
        assert np.all(np.diff(logits[t, ids[t]]) <= 0)


def test_weights_renormalised_sum_to_one_and_follow_the_logits():
    o = _inputs()
    ids, w, logits = MO.route(o["b"], o["wr"], 4, True)
    assert np.allclose(w.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    # renormalised top-k weights are the softmax over the chosen logits
    sel = np.take_along_axis(logits, ids, axis=1)
    ref = np.exp(sel - sel.max(axis=1, keepdims=True))
    assert np.allclose(w, ref / ref.sum(axis=1, keepdims=True), rtol=1e-13, atol=0)
    _, w_all, _ = MO.route(o["b"], o["wr"], 16, False)
    assert np.allclose(w_all.sum(axis=1), 1.0, rtol=0, atol=1e-14)


def test_relabelling_experts_changes_nothing():
    o = _inputs(seed=3)
    perm = np.random.default_rng(4).permutation(16)
    y = MO.moe_ffn(o["b"], o["wr"], o["wgu"], o["wd"], 4)
    yp = MO.moe_ffn(o["b"], o["wr"][perm], o["wgu"][perm], o["wd"][perm], 4)
    assert np.max(np.abs(y - yp)) <= 1e-12 * np.max(np.abs(y))


def test_planted_mistakes_fail_the_transformers_pin(monkeypatch):
    o = _inputs(seed=5)
    _, _, y_hf = _hf(o, 4, True)
    tol = 1e-4 * np.max(np.abs(y_hf))
    good_w, good_k = MO.routing_weights, MO.top_k_experts
    plants = {
        "no renormalisation": ("routing_weights", lambda lg, ids, r: good_w(lg, ids, False)),
        "smallest logits": ("top_k_experts", lambda lg, k: good_k(-lg, k)),
        "equal weights": ("routing_weights", lambda lg, ids, r: np.full(ids.shape, 1.0 / ids.shape[1])),
    }
    for name, (fn, bad) in plants.items():
        with monkeypatch.context() as mp:
            mp.setattr(MO, fn, bad)
            y = MO.moe_ffn(o["b"], o["wr"], o["wgu"], o["wd"], 4, True)
        assert np.max(np.abs(y - y_hf)) > tol, name
    # gate and up halves swapped in the weights the oracle is given
    F = o["wgu"].shape[1] // 2
    swapped = np.concatenate([o["wgu"][:, F:], o["wgu"][:, :F]], axis=1)
    y = MO.moe_ffn(o["b"], o["wr"], swapped, o["wd"], 4, True)
    assert np.max(np.abs(y - y_hf)) > tol


# ---------------------------------------------------------------- MoE layer

def _moe_layer_case(identical=False):
    from paper_2606_00516_amd import inputs as gen
    from tests._cases import make_case, oracle_cfg
    shape = gen.TINY_MOE
    case = make_case(shape, gen.batch_tiny(mode="mixed"), spare_pages=2)
    if identical:
        # every expert the same SwiGLU: the renormalised weights sum to one,
        # so the block is that SwiGLU whatever the routing
        for k in ("w_experts_gate_up", "w_experts_down"):
            case.weights[k] = case.weights[k][:1].repeat(shape.n_experts, 1, 1)
    return shape, case, oracle_cfg(shape)


def test_moe_layer_with_identical_experts_is_the_dense_layer():
    import dataclasses
    shape, case, cfg = _moe_layer_case(identical=True)
    y_moe, _ = case.run_oracle(dtype=np.float64)
    dense_cfg = dataclasses.replace(cfg, ffn=shape.expert_ffn, n_experts=0, top_k=0, expert_ffn=0)
    o = case.oracle_inputs()
    wb = dict(o["w_bits"])
    wb["w_gate_up"] = wb.pop("w_experts_gate_up")[0]
    wb["w_down"] = wb.pop("w_experts_down")[0]
    W = oracle_prepare(wb, dense_cfg)
    y_dense = OL.layer_step(dense_cfg, W, o["k_cache"], o["v_cache"], o["block_tables"], o["context_lens"],
                            o["chunk_lens"], o["x_bits"])
    # the MoE block sees its input rounded to bf16, the dense feed-forward
    # does not: the two agree to that rounding
    assert np.max(np.abs(y_moe - y_dense)) <= 1e-2 * np.max(np.abs(y_dense))
    assert np.max(np.abs(y_moe - y_dense)) > 0


def test_moe_layer_is_attention_then_the_pinned_block():
    shape, case, cfg = _moe_layer_case()
    (y, inter), o = case.run_oracle(dtype=np.float64, intermediates=True)
    W = oracle_prepare(o["w_bits"], cfg, np.float64)
    b = OL.rmsnorm(inter["h1"], W["g2"], cfg.rms_eps)
    blk = MO.moe_ffn(OL.f32_to_bf16_bits(b.astype(np.float32)), o["w_bits"]["w_router"],
                     o["w_bits"]["w_experts_gate_up"], o["w_bits"]["w_experts_down"], shape.top_k)
    assert np.max(np.abs(y - (inter["h1"] + blk))) <= 1e-12 * np.max(np.abs(y))


def oracle_prepare(w_bits, cfg, dtype=np.float64):
    return OL.prepare_weights(w_bits, cfg, dtype)

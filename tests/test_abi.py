"""The C ABI without a GPU: the library loads, exports every declared symbol,
and its host-side validation returns the documented status for each kind of
bad input.  No compute call is made."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_00516_amd import binding as B
from paper_2606_00516_amd import inputs as gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eb_layer.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(eb_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = B.lib()
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(B.SYMBOLS)


def test_status_strings():
    for code, name in B.STATUS.items():
        assert B.eb_status_str(code) == name


def _ok_case():
    b = gen.batch_tiny(mode="mixed")
    bt, pool = gen.make_block_tables(b, spare_pages=2, seed=5)
    return b, bt, pool


def test_validate_accepts_generated_batches():
    b, bt, pool = _ok_case()
    assert B.eb_validate(gen.TINY, b.context_lens, b.chunk_lens, bt, pool, "mixed") == 0
    assert B.eb_validate(gen.TINY, b.context_lens, b.chunk_lens, bt, pool, "prefill") == 0
    d = gen.batch_tiny(mode="decode")
    bt, pool = gen.make_block_tables(d, spare_pages=0, seed=1)
    assert B.eb_validate(gen.TINY, d.context_lens, d.chunk_lens, bt, pool, "decode") == 0
    for r in (0.0, 0.3, 1.0):
        mb = gen.batch_8b_mixed(r)
        bt, pool = gen.make_block_tables(mb, spare_pages=0, seed=3)
        assert B.eb_validate(gen.L8B, mb.context_lens, mb.chunk_lens, bt, pool, "mixed") == 0
        assert mb.num_tokens == 2048


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("n_kv_heads", 3), ("page_size", 32), ("hidden", 252),
                                         ("ffn", 690), ("n_q_heads", 24)])
def test_validate_rejects_unsupported_shapes(field, value):
    import dataclasses
    shape = dataclasses.replace(gen.TINY, **{field: value})
    b, bt, pool = _ok_case()
    assert B.eb_validate(shape, b.context_lens, b.chunk_lens, bt, pool, "mixed") == -2
    assert B.eb_last_error()


def test_validate_moe_layers():
    # the mixture-of-experts layer shapes validate; each rule of the MoE
    # config fails with EB_ERR_CONFIG (n_experts a multiple of 16 up to 256,
    # 1 <= top_k <= min(n_experts, 64), expert_ffn a positive multiple of 8,
    # hidden a multiple of 32; the dense ffn may then be 0, not otherwise)
    import dataclasses
    b, bt, pool = _ok_case()
    assert B.eb_validate(gen.TINY_MOE, b.context_lens, b.chunk_lens, bt, pool, "mixed") == 0
    assert B.eb_validate(gen.Q30B, b.context_lens, b.chunk_lens, bt, pool, "mixed") == 0
    for field, value in (("n_experts", 20), ("n_experts", 272), ("top_k", 0), ("top_k", 17), ("expert_ffn", 100),
                         ("expert_ffn", 0), ("hidden", 264)):
        shape = dataclasses.replace(gen.TINY_MOE, **{field: value})
        assert B.eb_validate(shape, b.context_lens, b.chunk_lens, bt, pool, "mixed") == -2, (field, value)
    assert B.eb_validate(dataclasses.replace(gen.TINY, ffn=0), b.context_lens, b.chunk_lens, bt, pool,
                         "mixed") == -2


def test_validate_batch_errors():
    b, bt, pool = _ok_case()
    ctx, chk = b.context_lens.copy(), b.chunk_lens.copy()
    # chunk_len 0
    c2 = chk.copy()
    c2[1] = 0
    assert B.eb_validate(gen.TINY, ctx, c2, bt, pool, "mixed") == -3
    # negative context
    x2 = ctx.copy()
    x2[0] = -1
    assert B.eb_validate(gen.TINY, x2, chk, bt, pool, "mixed") == -3
    # num_tokens != sum
    cfg = B.config_of(gen.TINY)
    hb = B.HostBatch(ctx, chk)
    hb.c.num_tokens += 1
    btc = np.ascontiguousarray(bt)
    st = B.lib().eb_validate(ctypes.byref(cfg), ctypes.byref(hb.c), btc.ctypes.data, pool, bt.shape[1], 2)
    assert st == -3
    # decode mode with a prefill chunk
    assert B.eb_validate(gen.TINY, ctx, chk, bt, pool, "decode") == -4
    # unknown mode
    assert B.eb_validate(gen.TINY, ctx, chk, bt, pool, 7) == -4
    # NULL length arrays
    hb = B.HostBatch(ctx, chk)
    hb.c.context_lens_host = None
    st = B.lib().eb_validate(ctypes.byref(cfg), ctypes.byref(hb.c), btc.ctypes.data, pool, bt.shape[1], 2)
    assert st == -1
    # NULL config
    hb = B.HostBatch(ctx, chk)
    st = B.lib().eb_validate(None, ctypes.byref(hb.c), btc.ctypes.data, pool, bt.shape[1], 2)
    assert st == -1


def test_validate_page_errors():
    b, bt, pool = _ok_case()
    ctx, chk = b.context_lens, b.chunk_lens
    # id beyond the pool
    bad = bt.copy()
    bad[0, 0] = pool
    assert B.eb_validate(gen.TINY, ctx, chk, bad, pool, "mixed") == -5
    # negative id in a needed slot
    bad = bt.copy()
    bad[2, 1] = -1
    assert B.eb_validate(gen.TINY, ctx, chk, bad, pool, "mixed") == -5
    # a page shared by two requests
    bad = bt.copy()
    bad[1, 0] = bad[0, 0]
    assert B.eb_validate(gen.TINY, ctx, chk, bad, pool, "mixed") == -5
    # table too short for context + chunk
    short = bt[:, :2]
    assert B.eb_validate(gen.TINY, ctx, chk, short, pool, "mixed") == -5
    # -1 entries past a request's needed pages are ignored
    ok = bt.copy()
    need = gen.pages_needed(b)
    for i, n in enumerate(need):
        ok[i, n:] = -1
    assert B.eb_validate(gen.TINY, ctx, chk, ok, pool, "mixed") == 0


def test_validate_empty_batch():
    e = np.zeros(0, np.int32)
    assert B.eb_validate(gen.TINY, e, e, np.zeros((0, 1), np.int32), 1, "mixed") == 0


def test_create_rejects_bad_config_before_touching_the_gpu():
    import dataclasses
    cfg = B.config_of(dataclasses.replace(gen.TINY, head_dim=80))
    h = ctypes.c_void_p()
    assert B.lib().eb_create(ctypes.byref(cfg), 4, 64, ctypes.byref(h)) == -2
    assert not h.value
    cfg = B.config_of(gen.TINY)
    assert B.lib().eb_create(ctypes.byref(cfg), 0, 64, ctypes.byref(h)) == -7
    assert B.lib().eb_create(ctypes.byref(cfg), 4, 64, None) == -1


def test_packed_weight_shapes_host_only():
    # the size of a packed copy and the shapes without one; a rejected shape
    # returns before any device call
    L = B.lib()
    assert L.eb_packed_weight_bytes(16, 32) == 16 * 32 * 2
    assert L.eb_packed_weight_bytes(28672, 4096) == 28672 * 4096 * 2
    for rows, cols in [(0, 32), (16, 0), (17, 32), (16, 48), (8, 32), (-16, 32), (32768, 32768)]:
        assert L.eb_packed_weight_bytes(rows, cols) == 0, (rows, cols)
    fake = ctypes.c_void_p(0x1000)
    code = {name: c for c, name in B.STATUS.items()}
    assert L.eb_pack_weight(fake, fake, 16, 48, None) == code["EB_ERR_CONFIG"]
    assert L.eb_pack_weight(None, fake, 16, 32, None) == code["EB_ERR_NULL"]

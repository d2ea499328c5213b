#!/usr/bin/env python
"""Benchmark of one decoder-layer step on one MI355X.

Default workload: the Llama-3-8B-shaped layer, pure-decode exclusive step, 64
decode requests with contexts uniform in 512..4096, paged bf16 KV (page 16,
seeded random block tables).  A step is the whole layer (RMSNorm, QKV GEMM,
RoPE + KV append, split-K decode attention + combine, O GEMM + residual,
RMSNorm, gate/up GEMM + SiLU*mul, down GEMM + residual) through the C ABI,
with every input resident in HBM before the timed region.

Prints one JSON line.  Other workloads: --workload prefill8b (8 prompts,
lengths 256..2048 capped at 8192 tokens), mixed8b --r R (2048-token step at
decode share R), sweep8b (the mixed step at decode shares 0, 0.1, ..., 1 and
several token budgets, with the exclusive endpoints, K(r), kappa, the
per-share linear fits and the crossover share), decode70b (one
Llama-3-70B-shaped layer, 256 decode requests with contexts 2048..16384),
stack70b (the 70B-shaped model step: --layers decoder layers, 80 by default,
as an exclusive decode step and as 4096-token mixed steps), copy (a plain
device copy of known size, used to calibrate the HBM byte counters).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "step latency vs decode share; decode HBM GB/s; prefill MFMA TFLOP/s"
HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2516.6
ATTN_SRC = os.path.join(ROOT, "paper_2606_00516_amd", "csrc", "k_attention.hip")
GEMM_SRC = os.path.join(ROOT, "paper_2606_00516_amd", "csrc", "k_gemm.hip")
COUNTERS = os.path.join(ROOT, "profiles", "hbm_counters.json")


def sha_of(path: str) -> str:
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="decode8b",
                    choices=["decode8b", "prefill8b", "mixed8b", "sweep8b", "decode70b", "stack70b", "policy8b",
                             "long8b", "moe30b", "q30b", "copy", "oracle_cpu"])
    ap.add_argument("--calib-out", default=None, help="policy8b: write the calibrated step-cost profile here")
    ap.add_argument("--shape", default="l8b", choices=["l8b", "q30b"],
                    help="layer of the sweep8b / policy8b workloads: the llama3-8b layer, or the "
                         "qwen3-30b-a3b-shaped mixture-of-experts layer")
    ap.add_argument("--layers", type=int, default=80, help="decoder layers of the stack70b model step")
    ap.add_argument("--stack-r", default="0.2,0.5,0.8", help="decode shares of the stack70b mixed steps")
    ap.add_argument("--budgets", default="1024,2048", help="token budgets of the sweep (for alpha/beta fits)")
    ap.add_argument("--ctx16", action="store_true", help="sweep with every decode context = 16 instead")
    ap.add_argument("--dec-ctx", default=None, help="decode context range lo,hi of the sweep (default 1024,8192)")
    ap.add_argument("--r", type=float, default=0.5, help="decode share for mixed8b")
    ap.add_argument("--budget", type=int, default=2048, help="token budget for mixed8b")
    ap.add_argument("--kv", default="bf16", choices=["bf16", "fp8"],
                    help="KV cache element: bf16, or 8-bit E4M3 codes with per-tensor k/v scales")
    ap.add_argument("--weights", default="bf16", choices=["bf16", "fp8"],
                    help="projection weights: bf16, or 8-bit E4M3 codes with one fp32 scale per output row")
    ap.add_argument("--packed-weights", default="on", choices=["on", "off"],
                    help="single-layer workloads: give the step fragment-packed copies of the bf16 projections "
                         "(made once, before timing; read by the weight-streaming GEMMs of steps under 256 rows)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="decode8b: skip the prefill step and the MB sweep that the default line carries")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU time of the oracle sample")
    ap.add_argument("--json-out", default=None)
    return ap.parse_args()


# ----------------------------------------------------------------------------
# algorithmic work of a step (each byte / flop counted once)
# ----------------------------------------------------------------------------

def weight_bytes(shape, kind="bf16"):
    """Bytes of one layer's weights: bf16, or 8-bit projection codes plus one
    fp32 scale per projection row (norm gains bf16 either way)."""
    if kind == "bf16":
        return shape.weight_bytes()
    d, f = shape.hidden, shape.ffn
    codes = shape.qkv_rows * d + d * shape.n_q_heads * shape.head_dim + 2 * f * d + d * f
    rows = shape.qkv_rows + d + 2 * f + d
    return codes + 4 * rows + 2 * 2 * d


def step_work(shape, batch, kv_elem=2, w_kind="bf16"):
    """Bytes and FLOPs a step must move / compute at minimum (``kv_elem``:
    bytes per cached K or V element, 2 for bf16, 1 for 8-bit codes;
    ``w_kind``: the projection weights' type)."""
    import numpy as np
    nkv, hd, nq, d = shape.n_kv_heads, shape.head_dim, shape.n_q_heads, shape.hidden
    c = batch.context_lens.astype(np.int64)
    n = batch.chunk_lens.astype(np.int64)
    dec = n == 1
    kv_bytes_dec = int(((c[dec] + 1) * nkv * hd * 2 * kv_elem).sum())
    kv_bytes_pf = int(((c[~dec] + n[~dec]) * nkv * hd * 2 * kv_elem).sum())
    T = int(n.sum())
    w_bytes = weight_bytes(shape, w_kind)
    act_bytes = T * d * 2 * 2
    gemm_flops = 2 * T * (shape.qkv_rows * d + d * nq * hd + 2 * shape.ffn * d + d * shape.ffn)
    attn_flops_dec = int((4 * nq * hd * (c[dec] + 1)).sum())
    attn_flops_pf = int((4 * nq * hd * (n[~dec] * c[~dec] + n[~dec] * (n[~dec] + 1) // 2)).sum())
    return dict(T=T, kv_bytes_decode=kv_bytes_dec, kv_bytes_prefill=kv_bytes_pf, weight_bytes=w_bytes,
                act_bytes=act_bytes, gemm_flops=gemm_flops, attn_flops_decode=attn_flops_dec,
                attn_flops_prefill=attn_flops_pf)


def workload(args):
    from paper_2606_00516_amd import inputs as gen
    if args.workload == "decode8b":
        return "llama3-8b-layer decode EB: 64 requests, ctx U[512,4096], page 16", gen.L8B, gen.batch_8b_decode(), \
            "decode"
    if args.workload == "prefill8b":
        return "llama3-8b-layer prefill EB: 8 prompts U[256,2048] capped at 8192 tokens", gen.L8B, \
            gen.batch_8b_prefill(), "prefill"
    if args.workload == "decode70b":
        return "llama3-70b-layer decode EB (one layer): 256 requests, ctx U[2048,16384], page 16", gen.L70B, \
            gen.batch_70b_decode(), "decode"
    b = gen.batch_8b_mixed(args.r, args.budget)
    return (f"llama3-8b-layer MB: {args.budget}-token step, decode share {args.r:.2f}, decode ctx U[1024,8192], "
            f"chunks U[256,1024] with prefix U[0,2048]"), gen.L8B, b, "mixed"


# ----------------------------------------------------------------------------
# CPU oracle baseline
# ----------------------------------------------------------------------------

# per-tensor scales of the 8-bit cache: the synthetic codes span 1/8 .. 7.5 in
# magnitude, so cached values span about 0.06 .. 3.75 like the bf16 N(0, 1) pool
FP8_SCALES = (0.5, 0.5)
KV_LABEL = {"bf16": "bf16", "fp8": "fp8-e4m3 codes, per-tensor k/v scales"}
W_LABEL = {"bf16": "bf16", "fp8": "fp8-e4m3 codes, one fp32 scale per output row"}


def make_w(gen, shape, kind, **kw):
    """One layer's random-init weights of type ``kind``."""
    return gen.make_weights_fp8(shape, **kw) if kind == "fp8" else gen.make_weights(shape, **kw)


def make_pool(gen, shape, batch, kv, **kw):
    """(paged K/V pool, kv_scales or None) for cache element ``kv``."""
    if kv == "fp8":
        return gen.make_kv_pool_codes(shape, batch, **kw), FP8_SCALES
    return gen.make_kv_pool(shape, batch, **kw), None


def cpu_baseline(shape, batch, w, pool, x, mode, target_s, kv_scales=None):
    """The oracle as it is, on the host's cores, over as many requests of the
    same workload as fit in about ``target_s`` seconds."""
    import numpy as np
    import torch

    import oracle
    from paper_2606_00516_amd import inputs as gen
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    cfg = oracle.LayerCfg(shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn,
                          shape.page_size, shape.rms_eps, shape.rope_theta)
    W = oracle.prepare_weights(gen.weight_arrays(w), cfg)
    w_kind = "fp8" if w["w_qkv"].dtype == torch.uint8 else "bf16"
    need = gen.pages_needed(batch)
    bt_host = pool.block_tables.cpu().numpy()
    off = batch.row_offsets
    xb = gen.bits(x)
    done, spent, rows, kv_bytes = [], 0.0, 0, 0
    # cheapest requests first; passes over the whole workload repeat until
    # about target_s seconds of oracle time have been spent (at most 64 passes)
    order = list(np.argsort(batch.chunk_lens, kind="stable"))
    staged = {}
    passes = 0
    while spent < target_s and passes < 64:
        for i in order:
            if i not in staged:
                ids = torch.as_tensor(bt_host[i, :need[i]].astype(np.int64), device=pool.k_cache.device)
                host = (lambda t: t.cpu().numpy().copy()) if kv_scales is not None else \
                    (lambda t: gen.bits(t).copy())
                staged[i] = (host(pool.k_cache.index_select(0, ids)), host(pool.v_cache.index_select(0, ids)))
            kb0, vb0 = staged[i]
            kb, vb = kb0.copy(), vb0.copy()
            bt = np.arange(need[i], dtype=np.int32)[None]
            xs = xb[off[i]:off[i + 1]]
            t0 = time.perf_counter()
            oracle.layer_step(cfg, W, kb, vb, bt, batch.context_lens[i:i + 1], batch.chunk_lens[i:i + 1], xs,
                              kv_scales=kv_scales)
            spent += time.perf_counter() - t0
            done.append(int(i))
            rows += int(batch.chunk_lens[i])
            c, n = int(batch.context_lens[i]), int(batch.chunk_lens[i])
            kv_bytes += (c + n) * shape.n_kv_heads * shape.head_dim * (2 if kv_scales is not None else 4)
            if spent >= target_s:
                break
        passes += 1
    # algorithmic bytes of the step-equivalents done: the weights once per
    # whole-workload step (rows / T of them) plus each request's K/V
    gbps = (kv_bytes + weight_bytes(shape, w_kind) * rows / batch.num_tokens) / spent / 1e9
    return {"value": round(gbps, 4), "unit": "GB/s", "cores": int(threads), "kind": "oracle", **host_facts(),
            "tokens_per_s": round(rows / spent, 3), "seconds": round(spent, 2),
            "sample": f"{len(done)} request-steps ({rows} rows; {passes} pass(es) over the {batch.num_seqs} requests "
                      f"of the same workload), fp32 numpy oracle in batched mode, one request per call"}


# ----------------------------------------------------------------------------
# timing
# ----------------------------------------------------------------------------

FLUSH_BYTES = 512 << 20
_FLUSH = {}


def flush_caches(device):
    """Write a 512 MiB scratch buffer: more than the 256 MB Infinity Cache and
    the L2s together, so the next step finds none of its operands cached."""
    import torch
    buf = _FLUSH.get(str(device))
    if buf is None:
        buf = _FLUSH[str(device)] = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=device)
    buf.zero_()


def stats_of(times_ms):
    import numpy as np
    t = np.asarray(times_ms, np.float64)
    return {"mean_ms": round(float(t.mean()), 5), "median_ms": round(float(np.median(t)), 5),
            "p10_ms": round(float(np.percentile(t, 10)), 5), "p90_ms": round(float(np.percentile(t, 90)), 5),
            "n": int(t.size)}


def measure(B, h, step_fn, w, pool, batch, x, y, ws, steps, warmup, kv_scales=None, timed_stage=None):
    """(mean ms per step, per-stage ms, ms of ``timed_stage``, timing stats).

    Every timed step is preceded by a 512 MiB cache flush outside its own
    pair of HIP events (recorded on the step's stream), so each step starts
    cold and the flush is not timed; the stats give the mean, median, p10
    and p90 of the per-step times and the wall time per step of the whole
    bracketed region (flushes included).  In the timed steps the library
    also brackets ``timed_stage`` with HIP events of its own (two markers
    per step, in a ring of ``steps`` slots created before the region), so its
    mean comes from the timed steps themselves; the full per-stage breakdown
    (a marker at every stage boundary) comes from a second pass of as many
    steps, flushed the same way."""
    import torch
    call = lambda: step_fn(h, w, pool.k_cache, pool.v_cache, pool.block_tables, batch.context_lens,  # noqa: E731
                           batch.chunk_lens, x, y=y, ws=ws, kv_scales=kv_scales)
    for _ in range(warmup):
        flush_caches(x.device)
        call()
    if timed_stage:
        B.eb_profile(h, True, steps=steps, stages=[timed_stage])
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in evs:
        flush_caches(x.device)
        a.record()
        call()
        b.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) / steps * 1e3
    st = stats_of([a.elapsed_time(b) for a, b in evs])
    st["wall_ms_per_step_incl_flush"] = round(wall_ms, 5)
    timed = B.eb_profile_read(h)[timed_stage] if timed_stage else None
    B.eb_profile(h, True, steps=steps)
    for _ in range(steps):
        flush_caches(x.device)
        call()
    stages = B.eb_profile_read(h)
    B.eb_profile(h, False)
    return st["mean_ms"], stages, timed, st


def sweep(args, dev, budgets=None, w=None, store=None):
    """Mixed step of the chosen layer (the 8B one by default) over decode
    shares 0, 0.1, .., 1 at several budgets (``budgets``, else --budgets)."""
    import numpy as np
    import torch

    from paper_2606_00516_amd import analysis as AN
    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen
    shape = gen.Q30B if args.shape == "q30b" else gen.L8B
    if w is None:
        w = gen.make_weights(shape, device=dev)
    if budgets is None:
        budgets = [int(b) for b in args.budgets.split(",")]
    rs = [round(0.1 * i, 1) for i in range(11)]
    dec_ctx = (16, 16) if args.ctx16 else (1024, 8192)
    if args.dec_ctx:
        lo, hi = (int(v) for v in args.dec_ctx.split(","))
        dec_ctx = (lo, hi)
    pts = []

    def run(batch, mode):
        pool, kvs = make_pool(gen, shape, batch, args.kv, device=dev, poison=False, store=store)
        x = gen.make_x(shape, batch.num_tokens, device=dev)
        y = torch.empty_like(x)
        h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
        ws = B.alloc_workspace(B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, mode), dev)
        fn = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill,
              "mixed": B.eb_layer_step_mixed}[mode]
        ms, st, _, tst = measure(B, h, fn, w, pool, batch, x, y, ws, args.steps, args.warmup, kv_scales=kvs)
        del pool, x, y, ws, h
        torch.cuda.empty_cache()
        gemm = sum(v for k, v in st.items() if k.endswith("gemm"))
        attn = st.get("attention", 0.0) + st.get("attention_combine", 0.0)
        wk = step_work(shape, batch, 1 if args.kv == "fp8" else 2)
        kv_b = wk["kv_bytes_decode"] + wk["kv_bytes_prefill"]
        a_ms = st.get("attention", 0.0)
        return {"ms": ms, "median_ms": tst["median_ms"], "p10_ms": tst["p10_ms"], "p90_ms": tst["p90_ms"],
                "gemm_ms": gemm, "attention_ms": attn, "other_ms": sum(st.values()) - gemm - attn,
                "kv_bytes_decode": wk["kv_bytes_decode"], "kv_bytes": kv_b,
                "attention_kernel_hbm_frac": round(kv_b / (a_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4) if a_ms else None,
                "gemm_tflops": round(wk["gemm_flops"] / (gemm / 1e3) / 1e12, 1) if gemm else None,
                "n_tok": wk["T"], "n_decode": batch.num_decode}

    for bud in budgets:
        for r in rs:
            s0 = gen.seeds()["batch"]
            rng = np.random.default_rng([s0, int(round(r * 1000)), bud])
            batch = gen.batch_mixed_budget(r, bud, rng, dec_ctx=dec_ctx)
            p = run(batch, "mixed")
            p.update(r=r, budget=bud, mode="mixed")
            pts.append(p)
            print(f"# B={bud} r={r:.1f} ms={p['ms']:.4f} attn={p['attention_ms']:.4f} gemm={p['gemm_ms']:.4f}",
                  file=sys.stderr, flush=True)
            if r in (0.0, 1.0):
                q = run(batch, "prefill" if r == 0.0 else "decode")
                q.update(r=r, budget=bud, mode="prefill" if r == 0.0 else "decode")
                pts.append(q)
    # analysis at the largest budget: K(r), EB line, kappa
    big = max(budgets)
    mb = sorted([p for p in pts if p["budget"] == big and p["mode"] == "mixed"], key=lambda p: p["r"])
    r_arr = [p["r"] for p in mb]
    K = [p["median_ms"] for p in mb]  # per share: the median step (one slow step does not bend the curve)
    Ka = [p["attention_ms"] for p in mb]
    rep = AN.sweep_report(r_arr, K)
    rep_attn = AN.sweep_report(r_arr, Ka)
    out = {"budget": big, "r": r_arr, "K_ms": K, "attention_ms": Ka, "gemm_ms": [p["gemm_ms"] for p in mb],
           "other_ms": [p["other_ms"] for p in mb], "K_bar_ms": list(AN.eb_line(r_arr, K[0], K[-1])),
           "fit": rep, "attention_fit": rep_attn,
           "eb_endpoints_ms": {p["mode"]: p["ms"] for p in pts if p["budget"] == big and p["mode"] != "mixed"},
           "eb_favoured_r": AN.eb_favoured(r_arr, K, 0.02 * max(K))}
    # per-share linear fits over budgets and the crossover share
    if len(budgets) >= 2:
        betas, alphas, r2s = [], [], []
        for r in rs:
            ps = [p for p in pts if p["r"] == r and p["mode"] == "mixed"]
            a, b_, r2 = AN.linear_fit([p["n_tok"] for p in ps], [p["ms"] for p in ps])
            alphas.append(a)
            betas.append(b_)
            r2s.append(r2)
        out.update(alpha_ms=alphas, beta_ms_per_token=betas, r2=r2s,
                   crossover_r=AN.crossover_primary(rs, betas))
    return out, pts


def stack70b(args, dev):
    """The 70B-shaped model step: ``args.layers`` decoder layers with their own
    random-init bf16 weights, as an exclusive decode step (256 requests,
    contexts U[2048,16384]) and as 4096-token mixed steps at the given decode
    shares.  The KV pool of one layer is as large as the batch needs; as many
    distinct pools as fit in the HBM left after the weights are allocated and
    layer l reads pool l mod n_pools (every pool is far larger than the
    caches, so each layer streams its context from HBM either way)."""
    import numpy as np
    import torch

    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen
    shape = gen.L70B
    L = args.layers
    s0 = gen.seeds()
    t0 = time.perf_counter()
    weights = [make_w(gen, shape, args.weights, seed=s0["weights"] + l, device=dev) for l in range(L)]
    torch.cuda.synchronize()
    print(f"# {L} layers of weights generated in {time.perf_counter() - t0:.1f} s "
          f"({L * weight_bytes(shape, args.weights) / 1e9:.1f} GB)", file=sys.stderr, flush=True)
    points = [("decode", gen.batch_70b_decode(), "decode")]
    for r in [float(v) for v in args.stack_r.split(",") if v]:
        points.append((f"mixed r={r:.1f}", gen.batch_70b_mixed(r), "mixed"))
    out = []
    for name, batch, mode in points:
        h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
        nbytes = B.eb_stack_workspace_bytes(h, batch.context_lens, batch.chunk_lens, mode)
        ws = B.alloc_workspace(nbytes, dev)
        kv_elem = 1 if args.kv == "fp8" else 2
        pool_bytes = int(gen.pages_needed(batch).sum()) * shape.n_kv_heads * shape.page_size * shape.head_dim * \
            2 * kv_elem
        free = torch.cuda.mem_get_info()[0]
        n_pools = max(1, min(L, int((free - (4 << 30)) // max(pool_bytes, 1))))
        t1 = time.perf_counter()
        made = [make_pool(gen, shape, batch, args.kv, seed=s0["kv"] + i, device=dev, poison=False)
                for i in range(n_pools)]
        pools = [m[0] for m in made]
        x = gen.make_x(shape, batch.num_tokens, device=dev)
        y = torch.empty_like(x)
        caches = [(pools[l % n_pools].k_cache, pools[l % n_pools].v_cache, pools[l % n_pools].block_tables) +
                  ((made[0][1],) if made[0][1] is not None else ()) for l in range(L)]
        torch.cuda.synchronize()
        print(f"# {name}: {batch.num_seqs} requests, {batch.num_tokens} rows, {n_pools} pool(s) of "
              f"{pool_bytes / 1e9:.1f} GB in {time.perf_counter() - t1:.1f} s", file=sys.stderr, flush=True)
        call = lambda: B.eb_stack_step(h, mode, weights, caches, batch.context_lens, batch.chunk_lens, x,  # noqa
                                       y=y, ws=ws)
        for _ in range(args.warmup):
            call()
        # the attention stage bracketed by events in the timed steps (the
        # library creates them here, for the warm-up's layer count); the full
        # per-stage breakdown from one more step with every stage's events
        B.eb_profile(h, True, steps=args.steps, stages=["attention"])
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            call()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t1) / args.steps * 1e3
        attn_timed = B.eb_profile_read(h)["attention"]
        B.eb_profile(h, True)
        call()
        st = B.eb_profile_read(h)
        B.eb_profile(h, False)
        wk = step_work(shape, batch, kv_elem, args.weights)
        kv = wk["kv_bytes_decode"] + wk["kv_bytes_prefill"]
        gemm_ms = sum(v for k, v in st.items() if k.endswith("gemm"))
        attn_ms = attn_timed
        pt = {"point": name, "mode": mode, "n_tok": wk["T"], "n_decode": batch.num_decode,
              "decode_share": round(batch.num_decode / wk["T"], 4), "ms_per_step": round(ms, 3),
              "tokens_per_s": round(wk["T"] / (ms / 1e3), 1),
              "step_bytes": L * (kv + wk["weight_bytes"] + wk["act_bytes"]),
              "step_flops": L * (wk["gemm_flops"] + wk["attn_flops_decode"] + wk["attn_flops_prefill"]),
              "kv_bytes_per_layer": kv, "kv_pools": n_pools,
              "stage_ms_sum_over_layers": {k: round(v, 3) for k, v in st.items()},
              "gemm_ms": round(gemm_ms, 3), "attention_ms": round(attn_ms, 3),
              "gemm_tflops": round(L * wk["gemm_flops"] / (gemm_ms / 1e3) / 1e12, 1) if gemm_ms else None}
        if mode == "decode":
            pt["attention_hbm_gbps"] = round(L * wk["kv_bytes_decode"] / (attn_ms / 1e3) / 1e9, 1)
        pt["whole_step_gbps"] = round(pt["step_bytes"] / (ms / 1e3) / 1e9, 1)
        print(f"# {name}: {ms:.2f} ms/step, attention {attn_ms:.1f} ms, GEMMs {gemm_ms:.1f} ms", file=sys.stderr,
              flush=True)
        out.append(pt)
        del made, pools, caches, x, y, ws, h, call
        torch.cuda.empty_cache()
    return out


def policy8b(args, dev):
    """The batching decision on this GPU: calibrate the linear step-cost model
    from an 8B-layer MB sweep whose decode contexts (512..1024) match the
    paper's synthetic mixes, evaluate the crossover condition and theta_0 for
    those mixes, and run the serving-loop simulator (EB(k0*), MB, EB+) priced
    by the measured coefficients."""
    from paper_2606_00516_amd import cost_model as CM
    from paper_2606_00516_amd import scheduler_sim as SIM
    args.dec_ctx = args.dec_ctx or "512,1024"
    args.budgets = args.budgets if args.budgets != "1024,2048" else "512,1024,2048,4096"
    sw, pts = sweep(args, dev)
    layer = "qwen3-30b-a3b-shaped MoE layer" if args.shape == "q30b" else "llama3-8b layer"
    c = CM.calibrate(pts, label=f"MI355X {layer}, decode ctx U[{args.dec_ctx}]")
    prof = {"hardware": "MI355X", "shape": layer, "decode_ctx": args.dec_ctx,
            "budgets": args.budgets, "costs": c.to_dict()}
    if args.calib_out:
        with open(args.calib_out, "w") as f:
            json.dump(prof, f, indent=1)
    table = CM.evaluate(c, Ns=(64, 256, 1024, 4096))
    sims = []
    for mu_L, mu_O in CM.PAPER_MIXES:
        wl = SIM.Workload(SIM.fixed_inputs(mu_L), SIM.geometric_outputs(mu_O), f"{mu_L}/{mu_O}")
        for N in (256, 1024):
            th0 = CM.solve_theta0(c.alpha_p / (c.alpha_d * mu_O))
            k0 = max(1, int(th0 * N))
            row = {"mix": f"{mu_L}/{mu_O}", "N": N, "theta0": th0, "k0": k0}
            for pol in ("eb", "mb", "ebplus"):
                r = SIM.Simulator(c, wl, SIM.SimCfg(N=N, k=k0, B=8192, policy=pol, max_completions=3000,
                                                    warmup=300), seed=0).run()
                row[pol] = {"requests_per_s_per_layer": round(r.throughput, 3),
                            "eb_iteration_share": round(r.eb_iterations / max(1, r.iterations), 3)}
            d = CM.compare(c, mu_L, mu_O, N)
            row["condition_favours"] = "MB" if d.mb_favoured else "EB"
            sims.append(row)
            print(f"# mix {mu_L}/{mu_O} N={N}: theta0={th0:.3f} EB {row['eb']['requests_per_s_per_layer']} "
                  f"MB {row['mb']['requests_per_s_per_layer']} EB+ {row['ebplus']['requests_per_s_per_layer']} "
                  f"(condition: {row['condition_favours']})", file=sys.stderr, flush=True)
    return {"calibration": prof, "sweep": {k: sw[k] for k in ("budget", "r", "K_ms", "fit", "crossover_r")
                                           if k in sw}, "decisions": table, "simulated": sims}


def long8b(args, dev):
    """Long contexts on the 8B-shaped layer, after the paper's 128K-input /
    64-output runs (App. A.1): (a) decode steps of 4 requests at contexts
    near 128K; (b) the 16 chunked-prefill steps of one 128K prompt under an
    8192-token budget, each chunk attending over the chunks before it;
    (c) single-iteration prefill of one prompt of 1K..128K tokens (the
    paper's stress test beyond the budget) with the R^2 of the linear model
    over the practical range (<= 8K) and over the whole range."""
    import numpy as np
    import torch

    from paper_2606_00516_amd import analysis as AN
    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen
    shape = gen.L8B
    w = gen.make_weights(shape, device=dev)
    steps = max(2, args.steps // 5)

    def run(batch, mode):
        pool, kvs = make_pool(gen, shape, batch, args.kv, device=dev, poison=False)
        x = gen.make_x(shape, batch.num_tokens, device=dev)
        y = torch.empty_like(x)
        h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
        ws = B.alloc_workspace(B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, mode), dev)
        fn = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill}[mode]
        ms, st, _, _ = measure(B, h, fn, w, pool, batch, x, y, ws, steps, 1, kv_scales=kvs)
        del pool, x, y, ws, h
        torch.cuda.empty_cache()
        wk = step_work(shape, batch, 1 if args.kv == "fp8" else 2)
        return ms, st, wk

    out = {}
    c = np.array([131072 - 64 + 16 * j for j in range(4)], np.int32)
    ms, st, wk = run(gen.Batch(c, np.ones(4, np.int32), "decode128k"), "decode")
    out["decode_128k"] = {"ms": round(ms, 4), "attention_ms": round(st["attention"], 4),
                          "attention_hbm_gbps": round(wk["kv_bytes_decode"] / (st["attention"] / 1e3) / 1e9, 1),
                          "kv_bytes": wk["kv_bytes_decode"]}
    print(f"# decode at 128K: {ms:.3f} ms/step, attention {st['attention']:.3f} ms "
          f"({out['decode_128k']['attention_hbm_gbps']} GB/s)", file=sys.stderr, flush=True)
    chunks = []
    for i in (0, 4, 8, 12, 15):
        ms, st, wk = run(gen.Batch(np.array([8192 * i], np.int32), np.array([8192], np.int32), f"chunk{i}"), "prefill")
        fl = wk["attn_flops_prefill"]
        chunks.append({"chunk": i, "prefix": 8192 * i, "ms": round(ms, 4), "attention_ms": round(st["attention"], 4),
                       "attention_tflops": round(fl / (st["attention"] / 1e3) / 1e12, 1),
                       "gemm_ms": round(sum(v for k, v in st.items() if k.endswith("gemm")), 4)})
        print(f"# chunk {i} (prefix {8192 * i}): {ms:.3f} ms, attention {st['attention']:.3f} ms "
              f"({chunks[-1]['attention_tflops']} TFLOP/s)", file=sys.stderr, flush=True)
    out["chunked_prefill_128k"] = chunks
    single = []
    for n in (1024, 2048, 4096, 8192, 16384, 32768, 65536, 131072):
        ms, st, wk = run(gen.Batch(np.zeros(1, np.int32), np.array([n], np.int32), f"prompt{n}"), "prefill")
        single.append({"n_tok": n, "ms": round(ms, 4), "attention_ms": round(st["attention"], 4),
                       "gemm_ms": round(sum(v for k, v in st.items() if k.endswith("gemm")), 4)})
        print(f"# single prompt {n}: {ms:.3f} ms (attention {st['attention']:.3f})", file=sys.stderr, flush=True)
    xs = [p["n_tok"] for p in single]
    ys = [p["ms"] for p in single]
    small = [i for i, v in enumerate(xs) if v <= 8192]
    a8, b8, r2_8 = AN.linear_fit([xs[i] for i in small], [ys[i] for i in small])
    aa, ba, r2_all = AN.linear_fit(xs, ys)
    out["single_prompt"] = single
    out["linear_fit"] = {"r2_le_8k": r2_8, "r2_all": r2_all, "beta_ms_per_token_le_8k": b8,
                         "beta_ms_per_token_all": ba}
    return out


def moe30b(args, dev):
    """The Qwen3-30B-A3B mixture-of-experts feed-forward block (128 experts,
    8 per token, expert width 768, hidden 2048) on a 64-token decode batch
    (weight streaming: most experts are hit, each read once) and an
    8192-token prefill batch (about 512 rows per expert, MFMA work)."""
    import torch

    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen
    shape = gen.MOE30B
    E, d, k, F = shape.n_experts, shape.hidden, shape.top_k, shape.expert_ffn
    w = gen.make_moe_weights(shape, device=dev)
    pts = []
    for name, T in (("decode", 64), ("prefill", 8192)):
        g = torch.Generator(device=dev).manual_seed(11 + T)
        b = torch.randn(T, d, generator=g, device=dev).to(torch.bfloat16)
        res = torch.randn(T, d, generator=g, device=dev).to(torch.bfloat16)
        y = torch.empty_like(b)
        ws = B.alloc_workspace(int(B.lib().eb_op_moe_ffn_workspace_bytes(T, d, E, k, F)), dev)
        _, ids, _ = B.eb_op_moe_ffn(b, w["w_router"], w["w_gate_up"], w["w_down"], k, residual=res, out=y, ws=ws,
                                    return_routing=True)
        torch.cuda.synchronize()
        hit = int(torch.unique(ids).numel())
        call = lambda: B.eb_op_moe_ffn(b, w["w_router"], w["w_gate_up"], w["w_down"], k, residual=res,  # noqa
                                       out=y, ws=ws)
        for _ in range(args.warmup):
            call()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            call()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        # algorithmic work: the router and every expert hit read once, the
        # activations in and out; products over the T k assignments
        wbytes = E * d * 2 + hit * shape.expert_bytes()
        act = 3 * T * d * 2
        flops = 2 * T * E * d + 2 * T * k * 3 * F * d
        pt = {"point": name, "tokens": T, "experts_hit": hit, "ms": round(ms, 5),
              "tokens_per_s": round(T / (ms / 1e3), 1), "weight_bytes": wbytes,
              "hbm_gbps": round((wbytes + act) / (ms / 1e3) / 1e9, 1),
              "tflops": round(flops / (ms / 1e3) / 1e12, 1)}
        pts.append(pt)
        print(f"# moe {name}: {ms:.3f} ms, {hit} experts hit, {pt['hbm_gbps']} GB/s, {pt['tflops']} TFLOP/s",
              file=sys.stderr, flush=True)
        del b, res, y, ws
    return pts


def q30b(args, dev):
    """The Qwen3-30B-A3B-shaped layer (attention of 32 q / 4 kv heads, the
    mixture-of-experts feed-forward) on the 8B-style batches: 64 decode
    requests, 8 prompts of prefill, and a 2048-token mixed step at r = 0.5."""
    import torch

    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen
    shape = gen.Q30B
    w = gen.make_weights(shape, device=dev)
    pts = []
    for name, batch, mode in (("decode", gen.batch_8b_decode(), "decode"),
                              ("prefill", gen.batch_8b_prefill(), "prefill"),
                              ("mixed r=0.5", gen.batch_8b_mixed(0.5), "mixed")):
        step_fn = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill,
                   "mixed": B.eb_layer_step_mixed}[mode]
        pool, _ = make_pool(gen, shape, batch, "bf16", device=dev, poison=False)
        x = gen.make_x(shape, batch.num_tokens, device=dev)
        y = torch.empty_like(x)
        h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
        ws = B.alloc_workspace(B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, mode), dev)
        ms, stages, t_att, _ = measure(B, h, step_fn, w, pool, batch, x, y, ws, args.steps, args.warmup,
                                    timed_stage="attention")
        wk = step_work(shape, batch)
        pt = {"point": name, "mode": mode, "tokens": wk["T"], "ms_per_step": round(ms, 5),
              "tokens_per_s": round(wk["T"] / (ms / 1e3), 1), "attention_ms": round(t_att, 5),
              "stage_ms": {k: round(v, 5) for k, v in stages.items()}}
        if mode == "decode":
            pt["attention_hbm_gbps"] = round(wk["kv_bytes_decode"] / (t_att / 1e3) / 1e9, 1)
        pts.append(pt)
        print(f"# q30b {name}: {ms:.3f} ms/step, attention {t_att:.3f} ms", file=sys.stderr, flush=True)
        del pool, x, y, ws, h
        torch.cuda.empty_cache()
    return pts


def prefill_part(args, dev, w):
    """The exclusive-prefill step of the 8B layer (8 prompts U[256,2048]
    capped at 8192 tokens): step TFLOP/s, the gate/up GEMM and the prefill
    attention kernel against the bf16 MFMA peak."""
    import torch

    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen
    shape, batch = gen.L8B, gen.batch_8b_prefill()
    pool, kvs = make_pool(gen, shape, batch, "bf16", device=dev)
    x = gen.make_x(shape, batch.num_tokens, device=dev)
    y = torch.empty_like(x)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    ws = B.alloc_workspace(B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, "prefill"), dev)
    ms, st, g_ms, tst = measure(B, h, B.eb_layer_step_prefill, w, pool, batch, x, y, ws, args.steps, args.warmup,
                                timed_stage="gate_up_gemm")
    del pool, x, y, ws, h
    torch.cuda.empty_cache()
    wk = step_work(shape, batch)
    flops = wk["gemm_flops"] + wk["attn_flops_prefill"]
    gemm_ms = sum(v for k, v in st.items() if k.endswith("gemm"))
    fl_gu = 2 * wk["T"] * 2 * shape.ffn * shape.hidden
    a_ms = st["attention"]
    return {"workload": "llama3-8b-layer prefill EB: 8 prompts U[256,2048] capped at 8192 tokens, "
                        f"lengths {batch.chunk_lens.tolist()}",
            "ms_per_step": ms, **{k: v for k, v in tst.items() if k != "mean_ms"},
            "step_tflops": round(flops / (ms / 1e3) / 1e12, 1),
            "step_frac_of_mfma_peak": round(flops / (ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "gemm_ms": round(gemm_ms, 5), "gemm_tflops": round(wk["gemm_flops"] / (gemm_ms / 1e3) / 1e12, 1),
            "gemm_frac": round(wk["gemm_flops"] / (gemm_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4),
            "stage_ms": {k: round(v, 5) for k, v in st.items()},
            "roofline": {"kernel": "k_gemm_big (gate/up projection + SiLU*mul, 256x256 tiles)", "bound": "mfma",
                         "achieved": round(fl_gu / (g_ms / 1e3) / 1e12, 1), "peak": BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(fl_gu / (g_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS, 4),
                         "avg_launch_ms": round(g_ms, 5), "flops_per_launch": fl_gu},
            "attention_roofline": {"kernel": "k_prefill (causal prefill attention, MFMA)", "bound": "mfma",
                                   "achieved": round(wk["attn_flops_prefill"] / (a_ms / 1e3) / 1e12, 1),
                                   "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                   "frac": round(wk["attn_flops_prefill"] / (a_ms / 1e3) / 1e12 / BF16_PEAK_TFLOPS,
                                                 4),
                                   "avg_launch_ms": round(a_ms, 5), "flops_per_launch": wk["attn_flops_prefill"]}}


def sweep_store(shape, budgets, dec_ctx, kv, dev):
    """One K and one V buffer sized for the largest pool of a sweep over
    ``budgets``: every point lays its pool in them, so all points and repeats
    read the same physical memory (separate allocations of a multi-GB pool
    moved a point by up to 10 % between repeats)."""
    import numpy as np
    import torch

    from paper_2606_00516_amd import inputs as gen
    most = 0
    for bud in budgets:
        for i in range(11):
            r = round(0.1 * i, 1)
            rng = np.random.default_rng([gen.seeds()["batch"], int(round(r * 1000)), bud])
            most = max(most, int(gen.pages_needed(gen.batch_mixed_budget(r, bud, rng, dec_ctx=dec_ctx)).sum()))
    n = most * shape.n_kv_heads * shape.page_size * shape.head_dim * (1 if kv == "fp8" else 2)
    return (torch.empty(n, dtype=torch.uint8, device=dev), torch.empty(n, dtype=torch.uint8, device=dev))


def sweep_part(args, dev, w, repeats=5):
    """The 8B MB sweep at the 2048-token budget (decode ctx U[1024,8192],
    r = 0, 0.1, .., 1) ``repeats`` times, for K(r) and the spread of kappa,
    and once at budgets 512, 1024 and 4096 for the per-share linear fits
    T = alpha + beta n_tok and the crossover share."""
    import copy

    import numpy as np

    from paper_2606_00516_amd import analysis as AN
    a = copy.copy(args)
    a.shape, a.ctx16, a.dec_ctx, a.kv = "l8b", False, None, "bf16"
    runs, pts_all = [], []
    from paper_2606_00516_amd import inputs as gen
    store = sweep_store(gen.L8B, [512, 1024, 2048, 4096], (1024, 8192), a.kv, dev)
    for _ in range(repeats):
        out, pts = sweep(a, dev, budgets=[2048], w=w, store=store)
        runs.append(out)
        pts_all += pts
        print(f"# sweep B=2048 kappa {out['fit']['kappa']:.4f}", file=sys.stderr, flush=True)
    _, pts_other = sweep(a, dev, budgets=[512, 1024, 4096], w=w, store=store)
    r = runs[0]["r"]
    K = np.median(np.array([o["K_ms"] for o in runs]), axis=0)
    kappas = [o["fit"]["kappa"] for o in runs]
    rep = AN.sweep_report(r, K)
    # per-share fits over the four budgets (the 2048 point: median of the repeats)
    betas, alphas, r2s = [], [], []
    for i, rr in enumerate(r):
        ns = [2048] + [p["n_tok"] for p in pts_other if p["r"] == rr and p["mode"] == "mixed"]
        ts = [float(K[i])] + [p["ms"] for p in pts_other if p["r"] == rr and p["mode"] == "mixed"]
        al, be, r2 = AN.linear_fit(ns, ts)
        alphas.append(round(al, 5))
        betas.append(round(be * 1e3, 5))
        r2s.append(round(r2, 5))
    mixed0 = [p for p in pts_all if p["mode"] == "mixed"][:len(r)]
    eb = {}
    for mode in ("prefill", "decode"):
        v = [p["ms"] for p in pts_all if p["mode"] == mode]
        eb[mode] = round(float(np.median(v)), 5) if v else None
    return {"workload": "llama3-8b-layer MB sweep: 2048-token steps at r = 0, 0.1, .., 1, decode ctx U[1024,8192], "
                        "chunks U[256,1024] with prefix U[0,2048]; budgets 512/1024/4096 once for the fits",
            "r": r, "K_ms": [round(float(k), 5) for k in K],
            "K_ms_runs": [[round(k, 5) for k in o["K_ms"]] for o in runs],
            "K_bar_ms": [round(float(k), 5) for k in AN.eb_line(r, K[0], K[-1])],
            "eb_endpoints_ms": eb,
            "attention_ms": [round(p["attention_ms"], 5) for p in mixed0],
            "gemm_ms": [round(p["gemm_ms"], 5) for p in mixed0],
            "attention_kernel_hbm_frac": [p["attention_kernel_hbm_frac"] for p in mixed0],
            "kappa": round(float(np.median(kappas)), 4), "kappa_runs": [round(k, 4) for k in kappas],
            "kappa_spread": round(float(max(kappas) - min(kappas)), 4), "fit_of_median": rep,
            "alpha_ms": alphas, "beta_us_per_token": betas, "fit_r2": r2s,
            "crossover_r": AN.crossover_primary(r, betas),
            "eb_favoured_r": AN.eb_favoured(r, K, 0.02 * float(max(K))),
            "paper_crossover_context": {"H200 (4.8 TB/s)": 0.8, "RTX PRO 6000 (1.792 TB/s)": 0.2,
                                        "note": "the paper's crossovers were measured with every decode context "
                                                "at 16 tokens (Sec. 1, Fig. marginal_cost); this sweep uses "
                                                "contexts U[1024,8192]"}}


def oracle_cpu(args, dev, per_run_s=4.0, runs=3):
    """The CPU oracle (as it stands, on this host's cores) on every workload it
    can run: the tiny layer in its three modes, the 8B decode and prefill
    steps and the 2048-token MB step at r = 0, 0.5 and 1, each as the median
    of ``runs`` bounded runs of about ``per_run_s`` seconds of oracle time
    (cheapest requests first, as in the default line's baseline)."""
    import torch

    from paper_2606_00516_amd import inputs as gen
    cases = [("tiny decode EB (4 requests, ctx U[64,256])", gen.TINY, gen.batch_tiny(mode="decode"), "decode"),
             ("tiny prefill EB (128-token chunk)", gen.TINY, gen.batch_tiny(mode="prefill"), "prefill"),
             ("tiny MB (4 decode rows + a 128-token chunk)", gen.TINY, gen.batch_tiny(mode="mixed"), "mixed"),
             ("llama3-8b decode EB (64 requests, ctx U[512,4096])", gen.L8B, gen.batch_8b_decode(), "decode"),
             ("llama3-8b prefill EB (8 prompts U[256,2048])", gen.L8B, gen.batch_8b_prefill(), "prefill")]
    for r in (0.0, 0.5, 1.0):
        cases.append((f"llama3-8b MB, 2048 tokens, r = {r:.1f}", gen.L8B, gen.batch_8b_mixed(r), "mixed"))
    out = []
    weights = {}
    for label, shape, batch, mode in cases:
        if shape.name not in weights:
            weights[shape.name] = gen.make_weights(shape, device=dev)
        w = weights[shape.name]
        pool, _ = make_pool(gen, shape, batch, "bf16", device=dev, poison=False)
        x = gen.make_x(shape, batch.num_tokens, device=dev)
        res = [cpu_baseline(shape, batch, w, pool, x, mode, per_run_s) for _ in range(runs)]
        del pool, x
        torch.cuda.empty_cache()
        tps = sorted(r_["tokens_per_s"] for r_ in res)
        gbps = sorted(r_["value"] for r_ in res)
        med_tps = tps[len(tps) // 2]
        out.append({"workload": label, "mode": mode, "tokens_per_s_median": med_tps, "tokens_per_s_runs": tps,
                    "gbps_median": gbps[len(gbps) // 2],
                    "sample": res[len(res) // 2]["sample"], "seconds_per_run": res[0]["seconds"]})
        print(f"# {label}: {med_tps} tokens/s (runs {tps})", file=sys.stderr, flush=True)
    return out


def host_facts():
    """The host the CPU oracle runs on: logical CPUs, model, BLAS."""
    import platform
    model = platform.processor() or ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')} ({info[0].get('num_threads')} threads)"
    except Exception:  # pragma: no cover
        pass
    return {"os_cpu_count": os.cpu_count(), "cpu_model": model, "blas": blas,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: --gpus {args.gpus} is not supported (the layer step has no "
              f"multi-GPU path; data-parallel replicas would each run this same single-GPU step)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2606_00516_amd import binding as B
    from paper_2606_00516_amd import inputs as gen

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.workload == "copy":
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            dst.copy_(src)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / args.steps
        print(json.dumps({"workload": "copy", "bytes_read": n, "bytes_written": n, "ms": dt * 1e3,
                          "GBps": 2 * n / dt / 1e9}))
        return

    if args.workload == "oracle_cpu":
        t0 = time.perf_counter()
        pts = oracle_cpu(args, dev)
        line = {"metric": "CPU oracle throughput", "value": pts[3]["tokens_per_s_median"], "unit": "tokens/s",
                "n_gpus": 0, "steps": 3, "warmup": 0, "ms_per_step": None, "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
                "config": {"workload": "the CPU oracle on the tiny, 8B decode / prefill and 8B MB (r = 0, 0.5, 1) "
                                       "inputs; value: the 8B decode step's median tokens/s"},
                "host": host_facts(), "points": pts, "wall_s": round(time.perf_counter() - t0, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    if args.workload == "sweep8b":
        t0 = time.perf_counter()
        out, pts = sweep(args, dev)
        wall = time.perf_counter() - t0
        big = out["budget"]
        line = {"metric": METRIC, "value": round(out["fit"]["kappa"], 4), "unit": "kappa (dimensionless)",
                "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
                "ms_per_step": round(out["K_ms"][-1], 5), "higher_is_better": False, "scaling": "weak",
                "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                "config": {"workload": f"llama3-8b-layer MB sweep, budgets {args.budgets}, decode ctx "
                                       f"{args.dec_ctx or ('16' if args.ctx16 else '1024,8192')}, r = 0..1 step 0.1",
                           "kv_cache": KV_LABEL[args.kv], "parallelism": "single-gpu"},
                "sweep": out, "points": pts, "wall_s": round(wall, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    if args.workload == "long8b":
        t0 = time.perf_counter()
        out = long8b(args, dev)
        d = out["decode_128k"]
        line = {"metric": METRIC, "value": d["attention_hbm_gbps"], "unit": "GB/s", "n_gpus": 1,
                "steps": args.steps, "warmup": 1, "ms_per_step": d["ms"], "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                "config": {"workload": "llama3-8b layer, 128K contexts: decode of 4 requests, chunked prefill of a "
                                       "128K prompt (8192-token chunks), single-iteration prompts 1K..128K",
                           "kv_cache": KV_LABEL[args.kv], "parallelism": "single-gpu"},
                **out, "wall_s": round(time.perf_counter() - t0, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    if args.workload == "policy8b":
        t0 = time.perf_counter()
        out = policy8b(args, dev)
        line = {"metric": METRIC, "value": out["sweep"].get("crossover_r"), "unit": "crossover decode share",
                "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": None,
                "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
                "data": "synthetic",
                "config": {"workload": f"{'qwen3-30b-a3b-shaped MoE' if args.shape == 'q30b' else 'llama3-8b'}-layer cost model: MB sweep budgets {args.budgets}, decode ctx "
                                       f"{args.dec_ctx}; decisions and simulated EB / MB / EB+ for the paper's "
                                       f"mixes", "kv_cache": KV_LABEL[args.kv], "parallelism": "single-gpu"},
                **out, "wall_s": round(time.perf_counter() - t0, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    if args.workload == "moe30b":
        t0 = time.perf_counter()
        pts = moe30b(args, dev)
        dec, pre = pts
        line = {"metric": METRIC, "value": dec["hbm_gbps"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
                "warmup": args.warmup, "ms_per_step": dec["ms"], "higher_is_better": True, "scaling": "weak",
                "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                "config": {"workload": "qwen3-30b-a3b MoE feed-forward block (E=128, k=8, F=768, d=2048): decode "
                                       "64 tokens, prefill 8192 tokens", "parallelism": "single-gpu"},
                "roofline": {"kernel": "eb_op_moe_ffn (router, plan, grouped gate/up and down GEMMs, combine) on "
                                       "the decode batch", "bound": "hbm", "achieved": dec["hbm_gbps"],
                             "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                             "frac": round(dec["hbm_gbps"] / HBM_PEAK_GBPS, 4), "traffic": None},
                "prefill_roofline": {"bound": "mfma", "achieved": pre["tflops"], "peak": BF16_PEAK_TFLOPS,
                                     "unit": "TFLOP/s", "frac": round(pre["tflops"] / BF16_PEAK_TFLOPS, 4)},
                "points": pts, "wall_s": round(time.perf_counter() - t0, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    if args.workload == "q30b":
        t0 = time.perf_counter()
        pts = q30b(args, dev)
        dec = pts[0]
        line = {"metric": METRIC, "value": dec["attention_hbm_gbps"], "unit": "GB/s", "n_gpus": 1,
                "steps": args.steps, "warmup": args.warmup, "ms_per_step": dec["ms_per_step"],
                "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
                "data": "synthetic",
                "config": {"workload": "qwen3-30b-a3b-shaped layer (attention + MoE feed-forward): decode EB 64 "
                                       "requests ctx U[512,4096]; prefill EB 8 prompts; MB 2048 tokens at r = 0.5",
                           "parallelism": "single-gpu"},
                "roofline": {"kernel": "k_decode_mfma (decode attention, G = 8)", "bound": "hbm",
                             "achieved": dec["attention_hbm_gbps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                             "frac": round(dec["attention_hbm_gbps"] / HBM_PEAK_GBPS, 4), "traffic": None},
                "points": pts, "wall_s": round(time.perf_counter() - t0, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    if args.workload == "stack70b":
        t0 = time.perf_counter()
        pts = stack70b(args, dev)
        dec = pts[0]
        line = {"metric": METRIC, "value": dec["whole_step_gbps"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
                "warmup": args.warmup, "ms_per_step": dec["ms_per_step"], "higher_is_better": True,
                "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
                "config": {"workload": f"llama3-70b-shaped model step, {args.layers} layers: decode EB 256 requests "
                                       f"ctx U[2048,16384]; MB 4096-token steps at r = {args.stack_r}",
                           "kv_cache": KV_LABEL[args.kv], "weights": W_LABEL[args.weights],
                           "parallelism": "single-gpu"},
                "roofline": {"kernel": "k_decode_mfma (decode attention, summed over layers)", "bound": "hbm",
                             "achieved": dec["attention_hbm_gbps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                             "frac": round(dec["attention_hbm_gbps"] / HBM_PEAK_GBPS, 4), "traffic": None},
                "points": pts, "wall_s": round(time.perf_counter() - t0, 1)}
        js = json.dumps(line)
        print(js)
        if args.json_out:
            with open(args.json_out, "w") as f:
                f.write(js + "\n")
        return

    label, shape, batch, mode = workload(args)
    step_fn = {"decode": B.eb_layer_step_decode, "prefill": B.eb_layer_step_prefill,
               "mixed": B.eb_layer_step_mixed}[mode]
    # inputs generated on the GPU and left resident in HBM
    w = make_w(gen, shape, args.weights, device=dev)
    packed = args.packed_weights == "on" and args.weights == "bf16"
    if packed:
        w = B.pack_layer_weights(w)
        torch.cuda.synchronize()
    pool, kvs = make_pool(gen, shape, batch, args.kv, device=dev)
    x = gen.make_x(shape, batch.num_tokens, device=dev)
    y = torch.empty_like(x)
    h = B.Handle(shape, batch.num_seqs, batch.num_tokens)
    ws = B.alloc_workspace(B.eb_workspace_bytes(h, batch.context_lens, batch.chunk_lens, mode), dev)
    timed_stage = "gate_up_gemm" if mode == "prefill" else "attention"
    ms, stages, t_ms, tstats = measure(B, h, step_fn, w, pool, batch, x, y, ws, args.steps, args.warmup, kv_scales=kvs,
                               timed_stage=timed_stage)

    wk = step_work(shape, batch, 1 if args.kv == "fp8" else 2, args.weights)
    step_bytes = wk["kv_bytes_decode"] + wk["kv_bytes_prefill"] + wk["weight_bytes"] + wk["act_bytes"]
    step_flops = wk["gemm_flops"] + wk["attn_flops_decode"] + wk["attn_flops_prefill"]
    gemm_ms = sum(v for k, v in stages.items() if k.endswith("gemm"))
    attn_ms = stages.get("attention", 0.0) + stages.get("attention_combine", 0.0)

    if mode == "decode":
        unit = "GB/s"
        value = step_bytes / (ms / 1e3) / 1e9
        a_ms = t_ms
        achieved = wk["kv_bytes_decode"] / (a_ms / 1e3) / 1e9
        roof = {"kernel": "k_decode_mfma (split-K paged decode attention on MFMA, LDS page ring)", "bound": "hbm",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "avg_launch_ms": round(a_ms, 5),
                "bytes_per_launch": wk["kv_bytes_decode"], "traffic": None}
    elif mode == "mixed":
        # the step is dominated by the single mixed attention launch, whose
        # decode items stream the requests' K/V from HBM
        unit = "TFLOP/s"
        value = step_flops / (ms / 1e3) / 1e12
        a_ms = t_ms
        kv_b = wk["kv_bytes_decode"] + wk["kv_bytes_prefill"]
        achieved = kv_b / (a_ms / 1e3) / 1e9
        roof = {"kernel": "k_mixed_mfma (prefill tiles + decode splits in one launch)", "bound": "hbm",
                "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "avg_launch_ms": round(a_ms, 5),
                "bytes_per_launch": kv_b, "prefill_attention_flops": wk["attn_flops_prefill"], "traffic": None}
    else:
        unit = "TFLOP/s"
        value = step_flops / (ms / 1e3) / 1e12
        g_ms = t_ms
        fl = 2 * wk["T"] * 2 * shape.ffn * shape.hidden
        achieved = fl / (g_ms / 1e3) / 1e12
        roof = {"kernel": "k_gemm_big (gate/up projection + SiLU*mul, 256x256 tiles" +
                          (", 8-bit weights converted to bf16 in LDS)" if args.weights == "fp8" else ")"),
                "bound": "mfma",
                "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "avg_launch_ms": round(g_ms, 5),
                "flops_per_launch": fl, "traffic": None}
    # HBM traffic from committed counter runs, only if the kernel is unchanged
    try:
        cnt = json.load(open(COUNTERS))
        key = {"decode8b": "decode_attention_8b", "decode70b": "decode_attention_70b"}.get(args.workload)
        if args.workload == "mixed8b" and args.r == 0.5 and args.budget == 2048:
            key = "mixed_attention_8b"  # (counters taken at the default share and budget only)
        key = key + "_fp8" if key and args.kv == "fp8" else key
        ent = cnt.get(key) if key else None
        if ent and ent.get("source_sha") == sha_of(ATTN_SRC):
            roof["traffic"] = ent["bytes_per_dispatch"]
    except (OSError, ValueError):
        pass

    line = {
        "metric": METRIC, "value": round(value, 3), "unit": unit, "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": label, "kv_cache": KV_LABEL[args.kv], "weights": W_LABEL[args.weights],
                   "packed_weights": packed,
                   "num_tokens": wk["T"],
                   "num_requests": batch.num_seqs,
                   "decode_share": round(batch.num_decode / max(wk["T"], 1), 4), "kv_cache": KV_LABEL[args.kv],
                   "parallelism": "single-gpu"},
        "tokens_per_s": round(wk["T"] / (ms / 1e3), 1),
        "timing": {**tstats, "protocol": "per-step HIP events on the library's stream; a 512 MiB cache flush "
                                         "before every step, outside its events; ms_per_step is the mean"},
        "step_bytes": step_bytes, "step_flops": step_flops,
        "stage_ms": {k: round(v, 5) for k, v in stages.items()},
        "gemm_ms": round(gemm_ms, 5), "attention_ms": round(attn_ms, 5),
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(shape, batch, w, pool, x, mode, args.cpu_seconds, kvs)
    if args.workload == "decode8b" and args.kv == "bf16" and args.weights == "bf16" and not args.no_extras:
        # the metric's other two parts on the same line: the prefill EB step
        # (MFMA TFLOP/s) and the MB sweep (step latency vs decode share)
        del pool, ws, x, y
        torch.cuda.empty_cache()
        t1 = time.perf_counter()
        line["prefill_8b"] = prefill_part(args, dev, w)
        print(f"# prefill part {time.perf_counter() - t1:.1f} s", file=sys.stderr, flush=True)
        line["mb_sweep_8b"] = sweep_part(args, dev, w)
        print(f"# prefill + sweep parts {time.perf_counter() - t1:.1f} s", file=sys.stderr, flush=True)
    out = json.dumps(line)
    print(out)
    if args.json_out:
        with open(args.json_out, "w") as f:
            f.write(out + "\n")


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the position-independent cache-hit path on one MI355X.

One step = one pass of the whole path over one batch of requests:
  plan (host) -> copy of the gather blocks to the device -> compose all layers (re-rotate +
  gather) -> suffix prefill attention layer by layer -> one decode token layer by layer.
The first four are the cache-hit TTFT region, timed like the paper's TTFT boundary (App. C.2):
device-synchronised at both ends, starting right before layout construction; projections,
MLP and LM head have no weights here, so the region holds only the attention path.

Inputs are synthetic (N(0,1), seeded) with the workload's shapes and already resident in HBM
when timing starts.  Prints one JSON line.  Per-kernel times come from HIP events recorded on
the stream the kernels run on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFS = 2500.0    # MI355X dense bf16 MFMA
METRIC = "composed-cache TTFT (ms/request); prefill attn TFLOP/s; rerotate+decode HBM GB/s"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="c3", help="c1..c5 or a workload name")
    p.add_argument("--decode-tokens", type=int, default=1, help="decode tokens per step")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget-s", type=float, default=12.0)
    p.add_argument("--copy-calib-gib", type=float, default=0.0,
                   help="also run a plain device copy of this size per step (counter calibration)")
    return p.parse_args()


# ------------------------------------------------------------------------------------------
# algorithmic work (bytes / flops the method must move or compute)
# ------------------------------------------------------------------------------------------

def compose_bytes(w, ctx, n_layers):
    # K and V rows: read from the pool and written to the cache, D elements each
    return int(sum(ctx)) * w.n_kv_heads * n_layers * 4 * w.head_dim * w.elem_bytes


def prefill_flops(w, ctx):
    # 4 * Hq * D per visible (query, key) pair: QK^T and PV, 2 flops per multiply-add
    Ls = w.n_suffix
    pairs = sum(Ls * c + Ls * (Ls + 1) // 2 for c in ctx)
    return 4 * w.n_q_heads * w.head_dim * pairs


def decode_bytes(w, n_vis):
    # every visible K and V row is read once per layer
    return int(sum(n_vis)) * w.n_kv_heads * 2 * w.head_dim * w.elem_bytes


# ------------------------------------------------------------------------------------------
# CPU oracle baseline (bounded sample)
# ------------------------------------------------------------------------------------------

def cpu_baseline(w, budget_s):
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import pic_oracle as O
    from synth import inputs as S

    lay = S.pool_layout(w)
    inp = S.host_layer(w, lay, 0)
    maps = O.plan_layout(lay.requests[:1], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)
    samples = []
    t_end = time.perf_counter() + budget_s
    b = 0
    while True:
        t0 = time.perf_counter()
        m = O.plan_layout([lay.requests[b % w.batch]], lay.doc_offset, lay.doc_len,
                          lay.doc_compile_pos)[0]
        K, V = O.compose_request(inp["pool_k_raw"], inp["pool_v"], m, w.rope_theta, w.dtype)
        if w.n_suffix:
            O.suffix_prefill(K, V, inp["q"][b % w.batch], inp["k_suf"][b % w.batch],
                             inp["v_suf"][b % w.batch])
        samples.append(time.perf_counter() - t0)
        b += 1
        if time.perf_counter() > t_end or b >= w.batch:
            break
    per_req_layer = sum(samples) / len(samples)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    del maps
    return {
        "value": per_req_layer * w.n_layers * 1e3, "unit": "ms/request", "cores": int(threads),
        "kind": "oracle",
        "sample": f"{len(samples)} request(s) x 1 layer of {w.name} (plan + compose + suffix prefill, "
                  f"fp64 numpy), scaled x{w.n_layers} layers; {sum(samples):.1f} s of CPU work",
    }


# ------------------------------------------------------------------------------------------

def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2607_28069_amd as pic
    import synth
    from synth import inputs as S

    pic.load()   # raises if libpic.so is missing: there is no fallback
    w = synth.get(args.workload)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    L, B, Hq, Hkv, D, Ls = w.n_layers, w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_suffix
    n_dec = max(args.decode_tokens, 0)

    # ---- setup, outside any timed region ("model loading" and cache store)
    lay = S.pool_layout(w)
    ctx_host = S.context_lengths(lay)
    max_ctx = int(ctx_host.max())
    cap = max_ctx + Ls + n_dec
    model = pic.Model.of(L, Hq, Hkv, D, w.dtype, w.rope_theta)
    m1 = model.with_layers(1)

    def per_layer(tensor, shape):
        t = torch.empty((L,) + tuple(shape), dtype=dt, device=dev)
        for l in range(L):
            t[l] = S.device_normal(w, tensor, shape, l, dev, dt)
        return t

    pool_k = per_layer("pool_k", (Hkv, lay.pool_tokens, D))
    pool_v = per_layer("pool_v", (Hkv, lay.pool_tokens, D))
    q = per_layer("q", (B, Ls, Hq, D))
    k_suf = per_layer("k_suf", (B, Ls, Hkv, D))
    v_suf = per_layer("v_suf", (B, Ls, Hkv, D))
    dq = per_layer("dq", (B, Hq, D))
    dk = per_layer("dk", (B, Hkv, D))
    dv = per_layer("dv", (B, Hkv, D))
    cache_k = torch.zeros((L, B, Hkv, cap, D), dtype=dt, device=dev)
    cache_v = torch.zeros_like(cache_k)
    out = torch.empty((L, B, Ls, Hq, D), dtype=dt, device=dev)
    dout = torch.empty((L, B, Hq, D), dtype=dt, device=dev)
    mad = cap
    table = torch.empty(pic.pic_rope_table_bytes(model, mad) // 4, dtype=torch.float32, device=dev)
    pic.pic_rope_table_init(model, mad, table)
    ctx_dev = torch.from_numpy(ctx_host.astype(np.int32)).to(dev)
    base_dev = torch.from_numpy((ctx_host + Ls).astype(np.int32)).to(dev)
    max_base = max_ctx + Ls
    ws_pre = torch.empty(max(pic.pic_prefill_workspace_bytes(m1, B, Ls, max_ctx), 16), dtype=torch.uint8, device=dev)
    ws_dec = torch.empty(max(pic.pic_decode_workspace_bytes(m1, B, max_base + n_dec, 0), 16),
                         dtype=torch.uint8, device=dev)
    n_blocks_max = sum((int(n) + 63) // 64 for r in lay.requests for n in lay.doc_len[r])
    blocks_pinned = torch.empty(n_blocks_max * 5, dtype=torch.int32, pin_memory=True)
    blocks_dev = torch.empty(n_blocks_max * 5, dtype=torch.int32, device=dev)
    calib = None
    if args.copy_calib_gib > 0:
        n = int(args.copy_calib_gib * (1 << 30)) // 2
        calib = (torch.empty(n, dtype=torch.bfloat16, device=dev).normal_(), torch.empty(n, dtype=torch.bfloat16, device=dev))
    stream = torch.cuda.current_stream()

    ev = lambda: torch.cuda.Event(enable_timing=True)
    rec = {"compose": [], "prefill": [], "decode": [], "ttft": [], "step": []}

    def step(timing: bool):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        # -- TTFT region
        blocks, ctx = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len,
                                          lay.doc_compile_pos, lay.pool_tokens)
        nb = len(blocks)
        blocks_pinned[: nb * 5].copy_(torch.from_numpy(blocks.view(np.int32)))
        blocks_dev[: nb * 5].copy_(blocks_pinned[: nb * 5], non_blocking=True)
        e0, e1 = ev(), ev()
        e0.record(stream)
        pic.pic_compose(model, pool_k, pool_v, lay.pool_tokens, blocks_dev, nb, table, mad,
                        cache_k, cache_v, B, cap)
        e1.record(stream)
        pre = []
        for l in range(L):
            a, b = ev(), ev()
            a.record(stream)
            pic.pic_suffix_prefill_attn(m1, q[l], k_suf[l], v_suf[l], cache_k[l], cache_v[l], B, cap,
                                        ctx_dev, max_ctx, Ls, out[l], ws_pre)
            b.record(stream)
            pre.append((a, b))
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        # -- decode
        dec = []
        for t in range(n_dec):
            for l in range(L):
                a, b = ev(), ev()
                a.record(stream)
                pic.pic_decode_attn(m1, dq[l], dk[l], dv[l], cache_k[l], cache_v[l], B, cap, base_dev, t,
                                    max_base, dout[l], ws_dec)
                b.record(stream)
                dec.append((a, b))
        if calib is not None:
            calib[1].copy_(calib[0])
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        if timing:
            rec["ttft"].append((t1 - t0) * 1e3)
            rec["step"].append((t2 - t0) * 1e3)
            rec["compose"].append(e0.elapsed_time(e1))
            rec["prefill"] += [a.elapsed_time(b) for a, b in pre]
            rec["decode"] += [a.elapsed_time(b) for a, b in dec]
        return ctx

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    total_ms = (time.perf_counter() - t_start) * 1e3

    mean = lambda x: float(sum(x) / len(x)) if x else 0.0
    ctx = [int(c) for c in ctx_host]
    ttft_ms = mean(rec["ttft"])
    comp_ms, pre_ms, dec_ms = mean(rec["compose"]), mean(rec["prefill"]), mean(rec["decode"])
    comp_b = compose_bytes(w, ctx, L)
    pre_f_layer = prefill_flops(w, ctx)
    dec_b_layer = decode_bytes(w, [c + Ls + 1 for c in ctx])   # step 0 sees ctx + Ls + 1 slots
    kernels = {
        "compose": {"bound": "hbm", "achieved": comp_b / (comp_ms * 1e-3) / 1e9 if comp_ms else None,
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "ms_per_launch": comp_ms,
                    "per_launch": comp_b, "launches_per_step": 1},
        "suffix_prefill_attn": {"bound": "mfma",
                                "achieved": pre_f_layer / (pre_ms * 1e-3) / 1e12 if pre_ms else None,
                                "peak": BF16_MFMA_PEAK_TFS, "unit": "TFLOP/s", "ms_per_launch": pre_ms,
                                "per_launch": pre_f_layer, "launches_per_step": L},
        "decode_attn": {"bound": "hbm", "achieved": dec_b_layer / (dec_ms * 1e-3) / 1e9 if dec_ms else None,
                        "peak": HBM_PEAK_GBS, "unit": "GB/s", "ms_per_launch": dec_ms,
                        "per_launch": dec_b_layer, "launches_per_step": L * n_dec},
    }
    for k in kernels.values():
        k["frac"] = (k["achieved"] / k["peak"]) if k["achieved"] else None
        k["ms_per_step"] = k["ms_per_launch"] * k["launches_per_step"]
    dom_name = max(kernels, key=lambda k: kernels[k]["ms_per_step"])
    dom = kernels[dom_name]
    roofline = {"kernel": dom_name, "bound": dom["bound"], "achieved": dom["achieved"], "peak": dom["peak"],
                "unit": dom["unit"], "frac": dom["frac"], "traffic": None}

    res = {
        "metric": METRIC,
        "value": ttft_ms / B,
        "unit": "ms/request",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "q_heads": Hq, "kv_heads": Hkv, "head_dim": D,
                   "rope_theta": w.rope_theta, "batch": B, "context_tokens": ctx[0] if len(set(ctx)) == 1 else ctx,
                   "suffix_tokens": Ls, "decode_tokens_per_step": n_dec, "pool_docs": w.pool_docs,
                   "docs_per_request": w.docs_per_request},
        "ttft_ms_batch": ttft_ms,
        "prefill_attn_tflops": kernels["suffix_prefill_attn"]["achieved"],
        "rerotate_compose_gbps": kernels["compose"]["achieved"],
        "decode_gbps": kernels["decode_attn"]["achieved"],
        "roofline": roofline,
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_budget_s)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

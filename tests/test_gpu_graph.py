"""Graph capture of the cache-hit path.

Every library call is a pure stream operation (no allocation, synchronisation or memset inside
the library), so a serving loop can record a whole request once -- composition of the documents
(Eq. 3 re-rotation), every layer's suffix prefill, the zero-copy paged prefill and split decode
steps -- and replay it.  Each replay must reproduce the eager results bit for bit; the caches
and outputs are cleared by eager work between replays, so nothing carries over from one run to
the next.
"""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from synth import inputs as S

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager():
    w = synth.get("llama8b_1layer")
    L, steps = 3, 2
    dev, dt = torch.device("cuda", 0), torch.bfloat16
    B, Hq, Hkv, D, Ls = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.n_suffix
    lay = S.pool_layout(w)
    model = pic.Model.of(L, Hq, Hkv, D, "bf16", w.rope_theta)
    m1 = model.with_layers(1)
    blocks, ctx = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                      lay.pool_tokens)
    max_ctx = int(ctx.max())
    cap = max_ctx + Ls + steps
    print(f"graph capture: {w.name} x {L} layers, batch {B}, ctx {max_ctx}, {steps} decode steps",
          flush=True)

    def per_layer(name, shape):
        return torch.stack([S.device_normal(w, name, shape, l, dev, dt) for l in range(L)])

    pool_k, pool_v = per_layer("pool_k", (Hkv, lay.pool_tokens, D)), per_layer("pool_v", (Hkv, lay.pool_tokens, D))
    q, k_suf, v_suf = (per_layer("q", (B, Ls, Hq, D)), per_layer("k_suf", (B, Ls, Hkv, D)),
                       per_layer("v_suf", (B, Ls, Hkv, D)))
    dq, dk, dv = (per_layer("dq", (steps, B, Hq, D)), per_layer("dk", (steps, B, Hkv, D)),
                  per_layer("dv", (steps, B, Hkv, D)))
    cache_k = torch.zeros((L, B, Hkv, cap, D), dtype=dt, device=dev)
    cache_v = torch.zeros_like(cache_k)
    out, pout, rout = (torch.zeros((L, B, Ls, Hq, D), dtype=dt, device=dev) for _ in range(3))
    dout = torch.zeros((L, steps, B, Hq, D), dtype=dt, device=dev)
    table = torch.empty(pic.pic_rope_table_bytes(model, cap) // 4, dtype=torch.float32, device=dev)
    pic.pic_rope_table_init(model, cap, table)
    blocks_dev = torch.from_numpy(blocks.view(np.int32).reshape(-1).copy()).to(dev)
    ctx_dev = torch.from_numpy(ctx).to(dev)
    base_dev = ctx_dev + Ls
    ws_pre = torch.empty(max(pic.pic_prefill_workspace_bytes(m1, B, Ls, max_ctx), 16), dtype=torch.uint8,
                         device=dev)
    ws_dec = torch.empty(max(pic.pic_decode_workspace_bytes(m1, B, max_ctx + Ls + steps, 2), 16),
                         dtype=torch.uint8, device=dev)
    slot_src = torch.empty((B, max_ctx), dtype=torch.int32, device=dev)
    slot_delta = torch.empty_like(slot_src)
    tile_map = torch.empty((B, pic.pic_slot_map_tiles(max_ctx), 2), dtype=torch.int32, device=dev)
    assert pic.pic_prefill_workspace_bytes(m1, B, Ls, max_ctx) > 0   # the split-K combine is recorded too

    def path():
        pic.pic_compose(model, pool_k, pool_v, lay.pool_tokens, blocks_dev, len(blocks), table, cap, cache_k,
                        cache_v, B, cap)
        pic.pic_build_slot_map(blocks_dev, len(blocks), B, max_ctx, slot_src, slot_delta, tile_map)
        for l in range(L):
            pic.pic_suffix_prefill_attn(m1, q[l], k_suf[l], v_suf[l], cache_k[l], cache_v[l], B, cap, ctx_dev,
                                        max_ctx, Ls, out[l], ws_pre)
            pic.pic_paged_prefill_attn(m1, pool_k[l], pool_v[l], lay.pool_tokens, slot_src, slot_delta, max_ctx,
                                       table, cap, q[l], k_suf[l], v_suf[l], cache_k[l], cache_v[l], B, cap,
                                       ctx_dev, max_ctx, Ls, pout[l], ws_pre)
            pic.pic_paged_prefill_attn(m1, pool_k[l], pool_v[l], lay.pool_tokens, slot_src, slot_delta, max_ctx,
                                       table, cap, q[l], k_suf[l], v_suf[l], cache_k[l], cache_v[l], B, cap,
                                       ctx_dev, max_ctx, Ls, rout[l], ws_pre, tile_map=tile_map)
        for t in range(steps):
            for l in range(L):
                pic.pic_decode_attn(m1, dq[l][t], dk[l][t], dv[l][t], cache_k[l], cache_v[l], B, cap, base_dev,
                                    t, max_ctx + Ls, dout[l][t], ws_dec, n_splits=2)

    results = (out, pout, rout, dout, cache_k, cache_v, tile_map)
    path()
    torch.cuda.synchronize()
    ref = [x.clone() for x in results]
    assert torch.equal(ref[0], ref[1])            # paged prefill == compose + prefill
    assert (ref[6][..., 0] >= 0).any()            # whole-run tiles were recorded
    assert ref[3].abs().sum().item() > 0

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        path()
    torch.cuda.synchronize()
    for replay in range(3):
        for x in results:                         # eager work between replays
            x.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, x, y in zip(("out", "paged out", "paged out (whole-run tiles)", "decode out", "cache_k",
                               "cache_v", "tile map"), results, ref):
            assert torch.equal(x, y), f"replay {replay}: {name} differs from the eager run"
        print(f"replay {replay} matches", flush=True)

"""GPU parity of the zero-copy (paged) suffix prefill: attention reading the documents' K/V
straight from the pool through the gather blocks (App. C.1 token map; Sec. 2, Eq. 3).

* Without a tile map every key is turned on load with the float32 arithmetic and bf16
  rounding of compose, so the outputs must be bit-identical to compose + suffix prefill.
* With the tile map, key tiles that are one pool run under one shift are read unturned and the
  queries are turned by -shift instead (RoPE's relative property); the outputs must then be
  within the attention tolerance of compose + prefill and of the oracle.  The tile map itself
  is checked entry by entry.
In both modes the suffix rows stored into the cache are bit-exact.  Without a tile map the
composed document slots stay untouched; with it, the context tiles that are not whole runs are
composed into the cache first (bit-identical to compose, so the prefill reads them from there)
and the whole-run tiles stay untouched.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from oracle import pic_oracle as O
from synth import inputs as S

from gpu_path import (DEV, assert_attn_close, assert_keys_close, gpu_compose, gpu_prefill, host, oracle_prefill,
                      setup, tdtype, to_dev)

pytestmark = pytest.mark.gpu


def _expected_tile_map(sm, dm, map_cap):
    """(src, shift) of every 64-slot tile that is one pool run under one shift, else (-1, 0)."""
    B, T = sm.shape[0], pic.pic_slot_map_tiles(map_cap)
    out = np.tile(np.array([-1, 0], np.int32), (B, T, 1))
    for b in range(B):
        for t in range(T):
            k0 = 64 * t
            if k0 + 64 > map_cap:
                continue
            src, d = int(sm[b, k0]), int(dm[b, k0])
            if src >= 0 and np.array_equal(sm[b, k0:k0 + 64], src + np.arange(64)) and (dm[b, k0:k0 + 64] == d).all():
                out[b, t] = (src, d)
    return out


def _paged(r, model=None, cache_k=None, cache_v=None, pool_k=None, pool_v=None, layers=1, runs=False, scale=0.0):
    """Slot map + paged prefill of run r on fresh (zeroed) caches; returns (out, cache_k, cache_v).
    runs: also build the tile map and pass it (whole-run tiles turn the queries)."""
    w, d, dt = r.w, r.dev, tdtype(r.w)
    m = model or r.model
    shape = (layers, w.batch, w.n_kv_heads, r.cap, w.head_dim)
    ck = torch.zeros(shape, dtype=dt, device=DEV) if cache_k is None else cache_k
    cv = torch.zeros(shape, dtype=dt, device=DEV) if cache_v is None else cache_v
    out = torch.zeros((layers, w.batch, w.n_suffix, w.n_q_heads, w.head_dim), dtype=dt, device=DEV)
    max_ctx = int(r.ctx.max())
    map_cap = max_ctx + 7                                   # any capacity >= max_ctx
    smap = torch.full((w.batch, map_cap), -5, dtype=torch.int32, device=DEV)
    dmap = torch.full((w.batch, map_cap), 123, dtype=torch.int32, device=DEV)
    tmap = (torch.full((w.batch, pic.pic_slot_map_tiles(map_cap), 2), 77, dtype=torch.int32, device=DEV)
            if runs else None)
    pic.pic_build_slot_map(d["blocks"], d["blocks"].numel() // 5, w.batch, map_cap, smap, dmap, tmap)
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m, w.batch, w.n_suffix, max_ctx), 16),
                     dtype=torch.uint8, device=DEV)
    pic.pic_paged_prefill_attn(m, d["pool_k"] if pool_k is None else pool_k,
                               d["pool_v"] if pool_v is None else pool_v, r.lay.pool_tokens, smap, dmap, map_cap,
                               d["table"], d["mad"], d["q"], d["k_suf"], d["v_suf"], ck, cv, w.batch, r.cap,
                               d["ctx"], max_ctx, w.n_suffix, out, ws, scale=scale, tile_map=tmap)
    # the map: pool token and shift of every composed slot, 0 / 0 past each context
    sm, dm = smap.cpu().numpy(), dmap.cpu().numpy()
    for b, mp in enumerate(r.maps):
        n = mp.ctx_len
        assert np.array_equal(sm[b, :n], mp.src_token) and np.array_equal(dm[b, :n], mp.logical_pos - mp.compile_pos)
        assert not sm[b, n:].any() and not dm[b, n:].any()
    if runs:
        tm = tmap.cpu().numpy()
        assert np.array_equal(tm, _expected_tile_map(sm, dm, map_cap)), "tile map"
        _paged.runs = int((tm[..., 0] >= 0).sum()), int((tm[..., 0] < 0).sum())
        _paged.tmap = tm
    return out, ck, cv


def _check_against_materialized(r, out_p, ck_p, cv_p, ck_m, cv_m, out_m, exact=True, tmap=None):
    """tmap (whole-run mode): context tiles marked as runs stay untouched, the others hold the
    composed rows bit for bit."""
    w = r.w
    if exact:
        assert torch.equal(out_p, out_m), "paged outputs differ from compose + prefill"
    else:
        assert_attn_close(host(out_p), host(out_m), "bf16")
    for b in range(w.batch):
        c = int(r.ctx[b])
        sl = slice(c, c + w.n_suffix)
        assert torch.equal(ck_p[:, b, :, sl], ck_m[:, b, :, sl]) and torch.equal(cv_p[:, b, :, sl], cv_m[:, b, :, sl])
        if tmap is None:
            assert not ck_p[:, b, :, :c].any() and not cv_p[:, b, :, :c].any(), "document slots were written"
            continue
        for t in range((c + 63) // 64):
            ts = slice(64 * t, min(64 * t + 64, c))
            if tmap[b, t, 0] >= 0:
                assert not ck_p[:, b, :, ts].any() and not cv_p[:, b, :, ts].any(), f"run tile {t} written"
            else:
                assert torch.equal(ck_p[:, b, :, ts], ck_m[:, b, :, ts]) and \
                    torch.equal(cv_p[:, b, :, ts], cv_m[:, b, :, ts]), f"tile {t} not composed"


@pytest.mark.parametrize("runs", [False, True], ids=["per-key", "whole-runs"])
@pytest.mark.parametrize("name", ["c2", "ragged", "mixed", "joint"])
def test_paged_prefill_equals_compose_then_prefill(name, runs):
    if name in ("c2", "joint"):   # joint: a shared 8-token header before every 520-token document
        w = synth.get("c2" if name == "c2" else "llama8b_joint_1layer")
        r = setup(w)
    else:   # uneven contexts, a prefix-only request, n_rep 7, tails that are not tile multiples;
            # ragged: documents of 7..81 tokens (no tile is one run), mixed: 151..238 tokens
            # (whole-run tiles inside documents, mixed tiles at their boundaries)
        w = dataclasses.replace(synth.get("c2"), name=name, n_q_heads=28, n_kv_heads=4, pool_docs=5,
                                doc_len=77, docs_per_request=4, n_suffix=37, prefix_len=13, batch=3,
                                doc_len_jitter=(1, 150) if name == "ragged" else (60, 300))
        lay = S.pool_layout(w)
        r = setup(w, requests=[[lay.prefix_entry, 3, 0, 4], [lay.prefix_entry], [2, 1, 0, 3, 4]], extra_cap=5)
    gpu_compose(r)
    out_m = gpu_prefill(r).clone()
    out_p, ck_p, cv_p = _paged(r, runs=runs)
    torch.cuda.synchronize()
    _check_against_materialized(r, out_p, ck_p, cv_p, r.dev["cache_k"], r.dev["cache_v"], out_m, exact=not runs,
                                tmap=_paged.tmap if runs else None)
    got = host(out_p)[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(got[b], ref, "bf16")
    if runs:   # c2: context tiles are whole runs; ragged: none is; mixed: both kinds
        n_run, n_other = _paged.runs
        assert (n_run > 0 or name == "ragged") and (n_other > 0 or name == "c2"), _paged.runs
    print(f"[{name}] paged ({'whole-run tiles ' + str(_paged.runs) if runs else 'per-key'}) vs materialized "
          f"and oracle ok (ctx {[int(c) for c in r.ctx]})", flush=True)


@pytest.mark.parametrize("runs", [False, True], ids=["per-key", "whole-runs"])
@pytest.mark.parametrize("pairing", ["half", "interleaved"])
@pytest.mark.parametrize("layout", ["c2", "mixed", "mixed_hd64"])
def test_paged_prefill_with_rotary_variants(pairing, runs, layout):
    # two layers with their own frequencies in one call; pool layer 1 differs from layer 0.
    # mixed: documents of 60..300 tokens, so with the tile map some context tiles are composed
    # into the cache first (both pairings, per-layer tables) and the others read from the pool;
    # mixed_hd64: the same at head_dim 64 (rotate-half partners 4 chunks apart)
    if layout == "c2":
        w = synth.get("c2")
        r = setup(w)
    else:
        w = dataclasses.replace(synth.get("c2"), name=layout, n_q_heads=28, n_kv_heads=4, pool_docs=5,
                                doc_len=77, docs_per_request=4, n_suffix=37, prefix_len=13, batch=3,
                                doc_len_jitter=(60, 300), head_dim=64 if layout == "mixed_hd64" else 128)
        lay = S.pool_layout(w)
        r = setup(w, requests=[[lay.prefix_entry, 3, 0, 4], [lay.prefix_entry], [2, 1, 0, 3, 4]], extra_cap=5)
    d = gpu_compose(r)
    D = w.head_dim
    m2 = pic.Model.of(2, w.n_q_heads, w.n_kv_heads, D, "bf16", w.rope_theta, pairing=pairing,
                      per_layer_tables=True)
    f = np.stack([pic.pic_rope_llama3_freq(D, 5e5), O.inv_freq(D, 1e4)])
    mad = d["mad"]
    table = torch.empty(pic.pic_rope_table_bytes(m2, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init_freq(m2, f, mad, table)
    pk = torch.cat([d["pool_k"], d["pool_k"].flip(-1)], 0).contiguous()
    pv = torch.cat([d["pool_v"], d["pool_v"] * 2], 0).contiguous()
    dt = tdtype(w)
    for name in ("q", "k_suf", "v_suf"):
        d[name] = torch.cat([to_dev(r.inp[name][None], dt)] * 2, 0).contiguous()
    shape = (2, w.batch, w.n_kv_heads, r.cap, D)
    ck_m, cv_m = torch.zeros(shape, dtype=dt, device=DEV), torch.zeros(shape, dtype=dt, device=DEV)
    pic.pic_compose(m2, pk, pv, r.lay.pool_tokens, d["blocks"], d["blocks"].numel() // 5, table, mad, ck_m, cv_m,
                    w.batch, r.cap)
    out_m = torch.zeros((2, w.batch, w.n_suffix, w.n_q_heads, D), dtype=dt, device=DEV)
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m2, w.batch, w.n_suffix, int(r.ctx.max())), 16),
                     dtype=torch.uint8, device=DEV)
    pic.pic_suffix_prefill_attn(m2, d["q"], d["k_suf"], d["v_suf"], ck_m, cv_m, w.batch, r.cap, d["ctx"],
                                int(r.ctx.max()), w.n_suffix, out_m, ws)
    d["table"] = table
    out_p, ck_p, cv_p = _paged(r, model=m2, pool_k=pk, pool_v=pv, layers=2, runs=runs)
    torch.cuda.synchronize()
    _check_against_materialized(r, out_p, ck_p, cv_p, ck_m, cv_m, out_m, exact=not runs,
                                tmap=_paged.tmap if runs else None)
    # and against the oracle: each layer's own frequencies (the oracle's Llama-3.1 scaling and
    # plain base 1e4) and the pairing, over that layer's pool rows
    fo = [O.llama3_inv_freq(D, 5e5), O.inv_freq(D, 1e4)]
    pk_h, pv_h, got = host(pk), host(pv), host(out_p)
    for l in range(2):
        for b in range(w.batch):
            K, V = O.compose_request(pk_h[l], pv_h[l], r.maps[b], w.rope_theta, "bf16", pairing=pairing,
                                     freqs=fo[l])
            ref, _, _ = O.suffix_prefill(K, V, r.inp["q"][b], r.inp["k_suf"][b], r.inp["v_suf"][b])
            assert_attn_close(got[l, b], ref, "bf16")
    if runs and layout != "c2":   # both kinds of context tile occur: some were composed first
        tm = _paged.tmap
        ctx_tiles = [(b, t) for b in range(w.batch) for t in range((int(r.ctx[b]) + 63) // 64)]
        assert any(tm[b, t, 0] >= 0 for b, t in ctx_tiles) and any(tm[b, t, 0] < 0 for b, t in ctx_tiles)
    print(f"[{pairing}, {layout}, {'tile map' if runs else 'per-key'}] two layers with their own "
          f"frequencies: paged == compose + prefill", flush=True)


@pytest.mark.parametrize("head_dim", [128, 64])
@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_tiles_composed_ahead_then_prefill_without_slot_map(pairing, head_dim):
    # pic_compose_tiles for both layers in one launch, then the paged prefill with the tile map
    # and no slot map, against the paged prefill that composes its own tiles: identical caches
    # and outputs (documents of 60..300 tokens, so both kinds of context tile occur; two layers
    # with their own frequencies)
    w = dataclasses.replace(synth.get("c2"), name="mixed", n_q_heads=28, n_kv_heads=4, pool_docs=5,
                            doc_len=77, docs_per_request=4, n_suffix=37, prefix_len=13, batch=3,
                            doc_len_jitter=(60, 300), head_dim=head_dim)
    lay = S.pool_layout(w)
    r = setup(w, requests=[[lay.prefix_entry, 3, 0, 4], [lay.prefix_entry], [2, 1, 0, 3, 4]], extra_cap=5)
    d = gpu_compose(r)
    D, L = w.head_dim, 2
    m2 = pic.Model.of(L, w.n_q_heads, w.n_kv_heads, D, "bf16", w.rope_theta, pairing=pairing,
                      per_layer_tables=True)
    f = np.stack([pic.pic_rope_llama3_freq(D, 5e5), O.inv_freq(D, 1e4)])
    table = torch.empty(pic.pic_rope_table_bytes(m2, d["mad"]) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init_freq(m2, f, d["mad"], table)
    pk = torch.cat([d["pool_k"], d["pool_k"].flip(-1)], 0).contiguous()
    pv = torch.cat([d["pool_v"], d["pool_v"] * 2], 0).contiguous()
    dt = tdtype(w)
    q, ks, vs = (torch.cat([to_dev(r.inp[n][None], dt)] * 2, 0).contiguous() for n in ("q", "k_suf", "v_suf"))
    max_ctx = int(r.ctx.max())
    map_cap = max_ctx + 7
    smap = torch.empty((w.batch, map_cap), dtype=torch.int32, device=DEV)
    dmap = torch.empty_like(smap)
    tmap = torch.empty((w.batch, pic.pic_slot_map_tiles(map_cap), 2), dtype=torch.int32, device=DEV)
    pic.pic_build_slot_map(d["blocks"], d["blocks"].numel() // 5, w.batch, map_cap, smap, dmap, tmap)
    tm = tmap.cpu().numpy()
    assert (tm[..., 0] >= 0).any() and (tm[..., 0] < 0).any()
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m2, w.batch, w.n_suffix, max_ctx), 16),
                     dtype=torch.uint8, device=DEV)
    res = []
    for ahead in (False, True):
        shape = (L, w.batch, w.n_kv_heads, r.cap, D)
        ck, cv = torch.zeros(shape, dtype=dt, device=DEV), torch.zeros(shape, dtype=dt, device=DEV)
        out = torch.zeros((L, w.batch, w.n_suffix, w.n_q_heads, D), dtype=dt, device=DEV)
        if ahead:
            pic.pic_compose_tiles(m2, pk, pv, r.lay.pool_tokens, smap, dmap, map_cap, tmap, table, d["mad"],
                                  d["ctx"], max_ctx, ck, cv, w.batch, r.cap)
        pic.pic_paged_prefill_attn(m2, pk, pv, r.lay.pool_tokens, None if ahead else smap, None if ahead else dmap,
                                   map_cap, table, d["mad"], q, ks, vs, ck, cv, w.batch, r.cap, d["ctx"], max_ctx,
                                   w.n_suffix, out, ws, tile_map=tmap)
        torch.cuda.synchronize()
        res.append((out, ck, cv))
    for a, b in zip(*res):
        assert torch.equal(a, b), "composing the tiles ahead changed the result"
    print(f"[{pairing}, D {head_dim}] tiles composed ahead for both layers: caches and outputs identical", flush=True)


def test_paged_prefill_on_the_largest_pool_head():
    # A pool head of 2^24 - 1 tokens: the most the paged prefill addresses with 32-bit byte
    # offsets from a head's base (a larger pool fails with PIC_ERR_UNSUPPORTED).  The request
    # places a 64-token entry from the bottom of the pool and a 1000-token entry ending at its
    # last token, moved by 64 positions.  Per-key mode bit-identical to compose + prefill; whole-run
    # mode (the tile map) and both against the oracle, which composes the same pool rows.
    w = dataclasses.replace(synth.get("c2"), name="largest_pool", n_q_heads=4, n_kv_heads=1, batch=1, n_suffix=16)
    T = (1 << 24) - 1
    Ls, Hq, D = w.n_suffix, w.n_q_heads, w.head_dim
    m = pic.Model.of(1, Hq, 1, D, "bf16", w.rope_theta)
    bf = torch.bfloat16
    gen = lambda name, shape: S.device_normal(w, name, shape, 0, DEV, bf)
    pool_k, pool_v = gen("pool_k", (1, 1, T, D)), gen("pool_v", (1, 1, T, D))
    q, ks, vs = gen("q", (1, 1, Ls, Hq, D)), gen("k_suf", (1, 1, Ls, 1, D)), gen("v_suf", (1, 1, Ls, 1, D))
    offs, lens = [0, T - 1000], [64, 1000]
    blocks, ctx_h = pic.pic_plan_layout([[0, 1]], offs, lens, [0, 0], T)
    ctx = int(ctx_h[0])
    assert ctx == 1064
    cap = ctx + Ls
    mad = cap
    table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init(m, mad, table)
    blk = torch.from_numpy(blocks.view(np.int32).reshape(-1).copy()).to(DEV)
    ctx_dev = torch.tensor([ctx], dtype=torch.int32, device=DEV)
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m, 1, Ls, ctx), 16), dtype=torch.uint8, device=DEV)
    with pytest.raises(pic.PicError, match="exceeds") as err:
        pic.pic_paged_prefill_attn(m, pool_k, pool_v, T + 1, ctx_dev, ctx_dev, ctx, table, mad, q, ks, vs,
                                   pool_k, pool_v, 1, cap, ctx_dev, ctx, Ls, q, ws)
    assert err.value.status == -2                      # PIC_ERR_UNSUPPORTED

    def caches():
        return (torch.zeros((1, 1, 1, cap, D), dtype=bf, device=DEV), torch.zeros((1, 1, 1, cap, D), dtype=bf, device=DEV))

    # compose + prefill
    ck_m, cv_m = caches()
    out_m = torch.zeros((1, 1, Ls, Hq, D), dtype=bf, device=DEV)
    pic.pic_compose(m, pool_k, pool_v, T, blk, len(blocks), table, mad, ck_m, cv_m, 1, cap)
    pic.pic_suffix_prefill_attn(m, q, ks, vs, ck_m, cv_m, 1, cap, ctx_dev, ctx, Ls, out_m, ws)
    # paged, per key and with the tile map
    smap = torch.zeros((1, ctx), dtype=torch.int32, device=DEV)
    dmap = torch.zeros((1, ctx), dtype=torch.int32, device=DEV)
    tmap = torch.zeros((1, pic.pic_slot_map_tiles(ctx), 2), dtype=torch.int32, device=DEV)
    pic.pic_build_slot_map(blk, len(blocks), 1, ctx, smap, dmap, tmap)
    outs = {}
    for runs in (False, True):
        ck, cv = caches()
        o = torch.zeros((1, 1, Ls, Hq, D), dtype=bf, device=DEV)
        pic.pic_paged_prefill_attn(m, pool_k, pool_v, T, smap, dmap, ctx, table, mad, q, ks, vs, ck, cv, 1, cap,
                                   ctx_dev, ctx, Ls, o, ws, tile_map=tmap if runs else None)
        torch.cuda.synchronize()
        assert torch.equal(ck[..., ctx:, :], ck_m[..., ctx:, :]) and torch.equal(cv[..., ctx:, :], cv_m[..., ctx:, :])
        outs[runs] = o
    tm = tmap.cpu().numpy()
    assert np.array_equal(tm[0, :16, 0], np.r_[0, T - 1000 + 64 * np.arange(15)]) and (tm[0, 16] == [-1, 0]).all()
    assert torch.equal(outs[False], out_m), "per-key paged prefill differs from compose + prefill"

    # the oracle, from the pool rows the request reads (bottom 64 and top 1000 tokens)
    pk = np.concatenate([host(pool_k[0, :, :64]), host(pool_k[0, :, T - 1000:])], axis=1)
    pv = np.concatenate([host(pool_v[0, :, :64]), host(pool_v[0, :, T - 1000:])], axis=1)
    rmap = O.plan_layout([[0, 1]], [0, 64], lens, [0, 0])[0]
    K, V = O.compose_request(pk, pv, rmap, w.rope_theta, "bf16")
    assert_keys_close(host(ck_m[0, 0])[:, :ctx], K, "bf16")
    assert np.array_equal(host(cv_m[0, 0])[:, :ctx], V)
    ref, _, _ = O.suffix_prefill(K, V, host(q)[0, 0], host(ks)[0, 0], host(vs)[0, 0])
    for runs in (False, True):
        assert_attn_close(host(outs[runs])[0, 0], ref, "bf16")


@pytest.mark.parametrize("runs", [False, True], ids=["per-key", "whole-runs"])
def test_paged_prefill_with_an_empty_context(runs):
    # a request that composes nothing (every key of its suffix comes from k_suf) beside one that
    # composes three documents: per-key mode bit-identical to compose + prefill, both modes
    # against the oracle
    w = dataclasses.replace(synth.get("c2"), name="paged_empty", pool_docs=3, doc_len=200, docs_per_request=3,
                            n_suffix=40, prefix_len=0, batch=2)
    r = setup(w, requests=[[], [2, 0, 1]])
    assert list(r.ctx) == [0, 600]
    gpu_compose(r)
    out_m = gpu_prefill(r).clone()
    out_p, ck_p, cv_p = _paged(r, runs=runs)
    torch.cuda.synchronize()
    _check_against_materialized(r, out_p, ck_p, cv_p, r.dev["cache_k"], r.dev["cache_v"], out_m, exact=not runs,
                                tmap=_paged.tmap if runs else None)
    got = host(out_p)[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(got[b], ref, "bf16")

"""bf16 caches at head_dim 64 (every attention call on the matrix-core kernels templated on the head
dim) against the oracle: composition, suffix prefill (split and unsplit launches, one to eight query
heads per kv head, ragged tiles, the suffix rows stored into the cache) and decode (with the
no-workspace entry point), the general frontier layout, zero-copy (paged) prefill bit-identical to
compose + prefill per key and within bf16 rounding of it with the tile map, and fused RoPE of
request-time tokens bit-identical to turning them first.

Tolerances as in test_gpu_parity: values bit-exact, bf16 keys within 1 bf16 ulp (+1e-5),
attention within 2e-2 + 1e-2 |ref| with relative Frobenius error <= 1e-2.
"""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from oracle import pic_oracle as O

from gpu_path import (DEV, assert_attn_close, assert_keys_close, gpu_compose, gpu_decode, gpu_frontier, gpu_prefill,
                      host, oracle_compose, oracle_prefill, setup, setup_frontier, to_dev)
from test_gpu_frontier import _check_cache_and_out, _decode_after
from test_gpu_paged import _check_against_materialized, _paged

pytestmark = pytest.mark.gpu


def _w(name="c2", **kw):
    return dataclasses.replace(synth.get(name), name=name + "_hd64", head_dim=64, **{"n_q_heads": 16, "n_kv_heads": 4, **kw})


def test_hd64_compose_prefill_decode():
    w = _w(decode_steps=3, pool_docs=6, doc_len=300, docs_per_request=4, prefix_len=13, n_suffix=45, batch=3)
    r = setup(w)
    gpu_compose(r)
    ck, cv = host(r.dev["cache_k"][0]), host(r.dev["cache_v"][0])
    for b in range(w.batch):
        K, V = oracle_compose(r, b)
        n = int(r.ctx[b])
        assert np.array_equal(cv[b][:, :n].view(np.uint32), V.view(np.uint32))
        assert assert_keys_close(ck[b][:, :n], K, "bf16") > 0.999
    # 12 (request, kv head) units on 256 compute units: the launch splits key ranges
    assert pic.pic_prefill_workspace_bytes(r.model, w.batch, w.n_suffix, int(r.ctx.max())) > 0
    out = host(gpu_prefill(r))[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(out[b], ref, "bf16")
    ck0, cv0 = r.dev["cache_k"].clone(), r.dev["cache_v"].clone()
    outs = [host(o)[0] for o in gpu_decode(r, w.decode_steps)]
    for b in range(w.batch):
        _, K, V = oracle_prefill(r, b)
        length = int(r.ctx[b]) + w.n_suffix
        for t in range(w.decode_steps):
            ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
            length += 1
            assert_attn_close(outs[t][b], ref, "bf16")
    # the no-workspace decode on the prefilled caches: bit-identical
    base = torch.from_numpy((r.ctx + w.n_suffix).astype(np.int32)).to(DEV)
    max_base = int((r.ctx + w.n_suffix).max())
    for t in range(w.decode_steps):
        o = torch.zeros((1, w.batch, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device=DEV)
        pic.pic_decode_attn_noalloc(r.model, *(to_dev(r.inp[k][t][None], torch.bfloat16) for k in ("dq", "dk", "dv")),
                                    ck0, cv0, w.batch, r.cap, base, t, max_base, o)
        torch.cuda.synchronize()
        assert np.array_equal(host(o)[0], outs[t])
    assert torch.equal(ck0, r.dev["cache_k"]) and torch.equal(cv0, r.dev["cache_v"])


def test_hd64_frontier():
    w = _w("llama8b_frontier_1layer", batch=2, pool_docs=6, docs_per_request=3)
    r = setup_frontier(w)
    out, n_inl = gpu_frontier(r)
    torch.cuda.synchronize()
    Ks, Vs = {}, {}
    for b, K, V in _check_cache_and_out(r, out, n_inl):
        Ks[b], Vs[b] = K, V
    _decode_after(r, 2, Ks, Vs)


@pytest.mark.parametrize("runs", [False, True], ids=["per-key", "with-tile-map"])
def test_hd64_paged_against_compose_then_prefill(runs):
    # per key: bit-identical to compose + prefill, the document slots of the cache untouched; with
    # the tile map: whole-run tiles read from the pool with the queries turned, the other context
    # tiles composed into the cache first, outputs within bf16 rounding
    w = _w(pool_docs=5, doc_len=150, docs_per_request=4, prefix_len=13, n_suffix=37, batch=3,
           doc_len_jitter=(60, 300))
    r = setup(w, extra_cap=5)
    gpu_compose(r)
    out_m = gpu_prefill(r).clone()
    out_p, ck_p, cv_p = _paged(r, runs=runs)
    torch.cuda.synchronize()
    _check_against_materialized(r, out_p, ck_p, cv_p, r.dev["cache_k"], r.dev["cache_v"], out_m, exact=not runs,
                                tmap=_paged.tmap if runs else None)
    if runs:
        assert _paged.runs[0] > 0 and _paged.runs[1] > 0, _paged.runs   # both kinds of tile
    got = host(out_p)[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(got[b], ref, "bf16")


@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_hd64_fused_rope(pairing):
    rng = np.random.default_rng(64)
    D, HQ, HKV, L, B, Ls = 64, 16, 4, 2, 3, 21
    ctx = np.array([300, 1201, 1], np.int32)
    max_ctx = int(ctx.max())
    cap, mad = max_ctx + Ls + 3, max_ctx + Ls + 2
    m = pic.Model.of(L, HQ, HKV, D, "bf16", 1e4, pairing=pairing, per_layer_tables=True)
    m1 = m.with_layers(1)
    freqs = np.stack([O.inv_freq(D, 1e4), O.inv_freq(D, 1e6)])
    table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init_freq(m, freqs, mad, table)
    block = (mad + 1) * (D // 2) * 2
    bf = lambda shape: O.store(rng.standard_normal(shape), "bf16")
    ck = to_dev(bf((L, B, HKV, cap, D)), torch.bfloat16)
    cv = to_dev(bf((L, B, HKV, cap, D)), torch.bfloat16)
    q_raw, k_raw, v = bf((L, B, Ls, HQ, D)), bf((L, B, Ls, HKV, D)), bf((L, B, Ls, HKV, D))
    dq, dk, dv = (to_dev(x, torch.bfloat16) for x in (q_raw, k_raw, v))
    ctx_d = torch.from_numpy(ctx).to(DEV)

    def turned(x, H, pos):
        out = []
        for l in range(L):
            y = x[l].reshape(-1, H, D).contiguous()
            z = torch.empty_like(y)
            pic.pic_rerotate_keys(m1, y, z, y.shape[0], H, torch.from_numpy(pos.astype(np.int32)).to(DEV),
                                  table[l * block:], mad)
            out.append(z.reshape(x[l].shape))
        return torch.stack(out)

    ck_a, cv_a, ck_b, cv_b = ck.clone(), cv.clone(), ck.clone(), cv.clone()
    out_a = torch.zeros((L, B, Ls, HQ, D), dtype=torch.bfloat16, device=DEV)
    out_b = torch.zeros_like(out_a)
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m, B, Ls, max_ctx), 16), dtype=torch.uint8, device=DEV)
    pic.pic_suffix_prefill_attn_rope(m, dq, dk, dv, ck_a, cv_a, B, cap, ctx_d, max_ctx, Ls, table, mad, out_a, ws)
    pos = (ctx[:, None] + np.arange(Ls)[None, :]).reshape(-1)
    pic.pic_suffix_prefill_attn(m, turned(dq, HQ, pos), turned(dk, HKV, pos), dv, ck_b, cv_b, B, cap, ctx_d,
                                max_ctx, Ls, out_b, ws)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b) and torch.equal(ck_a, ck_b) and torch.equal(cv_a, cv_b)
    got, ckh, cvh = host(out_a), host(ck), host(cv)
    for l, b in ((0, 0), (1, 1), (1, 2)):
        n = int(ctx[b])
        p = n + np.arange(Ls)
        qr = O.rope(np.transpose(q_raw[l, b], (1, 0, 2)), p, 0.0, pairing, freqs[l])
        kr = O.store(O.rope(np.transpose(k_raw[l, b], (1, 0, 2)), p, 0.0, pairing, freqs[l]), "bf16")
        Kf = np.concatenate([ckh[l, b][:, :n], kr], axis=1)
        Vf = np.concatenate([cvh[l, b][:, :n], np.transpose(v[l, b], (1, 0, 2))], axis=1)
        assert_attn_close(np.transpose(got[l, b], (1, 0, 2)), O.attention(qr, p, Kf, Vf, np.arange(n + Ls)), "bf16")
    # one fused-RoPE decode step after the prefill, against turn-then-decode
    base = torch.from_numpy((ctx + Ls).astype(np.int32)).to(DEV)
    q1, k1, v1 = bf((L, B, HQ, D)), bf((L, B, HKV, D)), bf((L, B, HKV, D))
    d_q, d_k, d_v = (to_dev(x, torch.bfloat16) for x in (q1, k1, v1))
    o_a, o_b = torch.zeros((L, B, HQ, D), dtype=torch.bfloat16, device=DEV), torch.zeros((L, B, HQ, D),
                                                                                        dtype=torch.bfloat16, device=DEV)
    dws = torch.empty(max(pic.pic_decode_workspace_bytes(m, B, int(max_ctx + Ls) + 1), 16), dtype=torch.uint8,
                      device=DEV)
    pic.pic_decode_attn_rope(m, d_q, d_k, d_v, ck_a, cv_a, B, cap, base, 0, int(max_ctx + Ls), table, mad, o_a, dws)
    dpos = ctx + Ls
    pic.pic_decode_attn(m, turned(d_q[:, :, None], HQ, dpos)[:, :, 0], turned(d_k[:, :, None], HKV, dpos)[:, :, 0],
                        d_v, ck_b, cv_b, B, cap, base, 0, int(max_ctx + Ls), o_b, dws)
    torch.cuda.synchronize()
    assert torch.equal(o_a, o_b) and torch.equal(ck_a, ck_b)


@pytest.mark.parametrize("n_rep,batch,n_suffix", [(1, 1, 130), (2, 2, 29), (4, 32, 64), (8, 1, 77), (3, 5, 200)],
                         ids=["mha-lone", "rep2-split", "rep4-unsplit", "rep8-lone", "rep3-ragged"])
def test_hd64_matrix_core_prefill(n_rep, batch, n_suffix):
    # the matrix-core prefill at head_dim 64: rows of 8 chunks, 8 rows per load instruction, 4 k
    # steps per score product and 2 output blocks.  A lone request splits key ranges (combine at
    # 8 lanes per row), 128 units run unsplit; contexts and suffixes end mid-tile.  Every token
    # and head against the oracle, and the suffix rows stored into the cache bit for bit.
    w = _w(n_q_heads=4 * n_rep, pool_docs=6, doc_len=300, docs_per_request=4, prefix_len=13, n_suffix=n_suffix,
           batch=batch, doc_len_jitter=(37, 700))
    r = setup(w)
    gpu_compose(r)
    ws = pic.pic_prefill_workspace_bytes(r.model, w.batch, w.n_suffix, int(r.ctx.max()))
    assert (ws > 0) == (batch < 32), ws
    out = host(gpu_prefill(r))[0]
    ck, cv = host(r.dev["cache_k"][0]), host(r.dev["cache_v"][0])
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(out[b], ref, "bf16")
        c = int(r.ctx[b])
        assert np.array_equal(ck[b][:, c:c + n_suffix], np.transpose(host(r.dev["k_suf"][0, b]), (1, 0, 2)))
        assert np.array_equal(cv[b][:, c:c + n_suffix], np.transpose(host(r.dev["v_suf"][0, b]), (1, 0, 2)))

"""Degenerate and extreme cases on the GPU, against the oracle: a request that composes
nothing (empty context: the suffix attends only to itself), a single-token suffix, a single
suffix token with a one-token context, keys moved by the largest supported shift, calls that
have nothing to do (they launch nothing and leave outputs untouched), decode with more than 16
query heads per kv head (plain, allocation-free and fused RoPE), and the largest cache stream the
prefill addresses."""
import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from oracle import pic_oracle as O
from synth import inputs as S

from gpu_path import (DEV, assert_attn_close, assert_keys_close, gpu_compose, gpu_decode, gpu_prefill, host,
                      oracle_prefill, setup, to_dev)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_suffix", [1, 37])
def test_empty_and_tiny_contexts(n_suffix):
    w = dataclasses.replace(synth.get("c2"), name="edges", pool_docs=3, doc_len=1, docs_per_request=1,
                            n_suffix=n_suffix, prefix_len=0, batch=3, decode_steps=2)
    r = setup(w, requests=[[], [0], [2, 1, 0]])          # contexts 0, 1 and 3 tokens
    assert list(r.ctx) == [0, 1, 3]
    gpu_compose(r)
    out = host(gpu_prefill(r))[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(out[b], ref, "bf16")
    outs = [host(o)[0] for o in gpu_decode(r, 2)]
    for b in range(w.batch):
        _, K, V = oracle_prefill(r, b)
        length = r.ctx[b] + w.n_suffix
        for t in range(2):
            ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
            length += 1
            assert_attn_close(outs[t][b], ref, "bf16")


def test_largest_shift():
    # keys compiled at position 0 and moved to positions near the table's limit (2^20)
    for dtype, D in (("f32", 64), ("bf16", 128)):
        m = pic.Model.of(1, 4, 2, D, dtype, 5e5)
        mad = 1 << 20
        n, H = 64, 2
        rng = np.random.default_rng(11)
        k = O.store(rng.standard_normal((n, H, D)), dtype)
        a = np.zeros(n, np.int64)
        b = mad - rng.integers(0, 1000, n)
        b[::2] *= -1                                       # also the largest negative shifts
        table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
        pic.pic_rope_table_init(m, mad, table)
        dt = torch.float32 if dtype == "f32" else torch.bfloat16
        kin = to_dev(k, dt)
        kout = torch.empty_like(kin)
        pic.pic_rerotate_keys(m, kin, kout, n, H, torch.from_numpy((b - a).astype(np.int32)).to(DEV), table, mad)
        ref = O.store(O.rerotate_keys(np.transpose(k, (1, 0, 2)), a, b, 5e5), dtype)
        assert_keys_close(np.transpose(host(kout), (1, 0, 2)), ref, dtype)


def test_calls_with_nothing_to_do_leave_outputs_untouched():
    w = synth.get("c2")
    m = pic.Model.of(1, w.n_q_heads, w.n_kv_heads, w.head_dim, "bf16", w.rope_theta)
    out = torch.full((1, 2, 4, w.n_q_heads, w.head_dim), 3.0, dtype=torch.bfloat16, device=DEV)
    ck = torch.full((1, 2, w.n_kv_heads, 16, w.head_dim), 5.0, dtype=torch.bfloat16, device=DEV)
    cv = ck.clone()
    ctx = torch.zeros(2, dtype=torch.int32, device=DEV)
    pic.pic_suffix_prefill_attn(m, out, out, out, ck, cv, 2, 16, ctx, 4, 0, out)      # no suffix tokens
    pic.pic_suffix_prefill_attn(m, out, out, out, ck, cv, 0, 16, ctx, 4, 4, out)      # empty batch
    pic.pic_compose(m, ck, cv, 16, ctx, 0, ctx, 16, ck, cv, 2, 16)                    # no blocks
    torch.cuda.synchronize()
    assert torch.all(out == 3.0) and torch.all(ck == 5.0) and torch.all(cv == 5.0)


@pytest.mark.parametrize("n_q_heads,n_splits", [(40, 0), (40, 3), (64, 1)])
def test_decode_more_than_16_query_heads_per_kv_head(n_q_heads, n_splits):
    # 20 and 32 query heads per kv head: the decode serves them in groups of 16 (one workgroup
    # per group, each streaming the context), with and without key splits; every head of every
    # request against the oracle, and the no-workspace entry point bit-identical
    w = dataclasses.replace(synth.get("c2"), name="wide_gqa", n_q_heads=n_q_heads, n_kv_heads=2, pool_docs=4,
                            doc_len=300, docs_per_request=3, n_suffix=5, prefix_len=0, batch=3, decode_steps=2)
    r = setup(w)
    gpu_compose(r)
    out = host(gpu_prefill(r))[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(out[b], ref, "bf16")
    ck0, cv0 = r.dev["cache_k"].clone(), r.dev["cache_v"].clone()
    outs = [host(o)[0] for o in gpu_decode(r, 2, n_splits=n_splits)]
    for b in range(w.batch):
        _, K, V = oracle_prefill(r, b)
        length = r.ctx[b] + w.n_suffix
        for t in range(2):
            ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
            length += 1
            assert_attn_close(outs[t][b], ref, "bf16")
    # the same two steps through pic_decode_attn_noalloc on the prefilled caches
    ck, cv = ck0, cv0
    base = torch.from_numpy((r.ctx + w.n_suffix).astype(np.int32)).to(DEV)
    max_base = int((r.ctx + w.n_suffix).max())
    for t in range(2):
        q = to_dev(r.inp["dq"][t][None], torch.bfloat16)
        k = to_dev(r.inp["dk"][t][None], torch.bfloat16)
        v = to_dev(r.inp["dv"][t][None], torch.bfloat16)
        o = torch.zeros((1, w.batch, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device=DEV)
        pic.pic_decode_attn_noalloc(r.model, q, k, v, ck, cv, w.batch, r.cap, base, t, max_base, o,
                                    n_splits=n_splits)
        torch.cuda.synchronize()
        assert np.array_equal(host(o)[0], outs[t]), t
    assert torch.equal(ck, r.dev["cache_k"]) and torch.equal(cv, r.dev["cache_v"])


def test_largest_cache_stream():
    # One (request, kv head) cache stream of 2^24 - 1 rows of 256 bytes: the most the matrix-core
    # prefill addresses with 32-bit byte offsets from a stream's base (larger caches fail with
    # PIC_ERR_UNSUPPORTED).  The context fills every slot before the suffix and one decode step
    # writes and reads the very last slot; sampled suffix tokens (all heads) and the decode step
    # against the oracle, the stored suffix rows bit-exact.
    w = dataclasses.replace(synth.get("c2"), name="largest_stream", n_q_heads=4, n_kv_heads=1, batch=1,
                            n_suffix=16)
    cap = (1 << 24) - 1
    Ls, Hq, D = w.n_suffix, w.n_q_heads, w.head_dim
    ctx = cap - 1 - Ls
    m = pic.Model.of(1, Hq, 1, D, "bf16", w.rope_theta)
    with pytest.raises(pic.PicError, match="exceeds") as err:
        pic.pic_suffix_prefill_attn(m, *([torch.empty(16, dtype=torch.bfloat16, device=DEV)] * 5), 1, cap + 1,
                                    torch.zeros(1, dtype=torch.int32, device=DEV), ctx, Ls,
                                    torch.empty(16, dtype=torch.bfloat16, device=DEV))
    assert err.value.status == -2                      # PIC_ERR_UNSUPPORTED
    bf = torch.bfloat16
    gen = lambda name, shape: S.device_normal(w, name, shape, 0, DEV, bf)
    ck, cv = gen("cache_k", (1, 1, 1, cap, D)), gen("cache_v", (1, 1, 1, cap, D))
    q, ks, vs = gen("q", (1, 1, Ls, Hq, D)), gen("k_suf", (1, 1, Ls, 1, D)), gen("v_suf", (1, 1, Ls, 1, D))
    dq, dk, dv = gen("dq", (1, 1, Hq, D)), gen("dk", (1, 1, 1, D)), gen("dv", (1, 1, 1, D))
    # the oracle's keys and values: the generated context, then the suffix and decode inputs
    K = host(ck[0, 0]).astype(np.float64)
    V = host(cv[0, 0]).astype(np.float64)
    K[0, ctx:ctx + Ls], V[0, ctx:ctx + Ls] = host(ks[0, 0, :, 0]), host(vs[0, 0, :, 0])
    K[0, cap - 1], V[0, cap - 1] = host(dk[0, 0, 0]), host(dv[0, 0, 0])
    print(f"[largest stream] cap={cap} ctx={ctx} Ls={Ls}", flush=True)

    ctx_dev = torch.tensor([ctx], dtype=torch.int32, device=DEV)
    out = torch.zeros((1, 1, Ls, Hq, D), dtype=bf, device=DEV)
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m, 1, Ls, ctx), 16), dtype=torch.uint8, device=DEV)
    pic.pic_suffix_prefill_attn(m, q, ks, vs, ck, cv, 1, cap, ctx_dev, ctx, Ls, out, ws)
    base = torch.tensor([ctx + Ls], dtype=torch.int32, device=DEV)
    dout = torch.zeros((1, 1, Hq, D), dtype=bf, device=DEV)
    dws = torch.empty(max(pic.pic_decode_workspace_bytes(m, 1, ctx + Ls + 1), 16), dtype=torch.uint8, device=DEV)
    pic.pic_decode_attn(m, dq, dk, dv, ck, cv, 1, cap, base, 0, ctx + Ls, dout, dws)
    torch.cuda.synchronize()
    assert torch.equal(ck[0, 0, 0, ctx:ctx + Ls], ks[0, 0, :, 0]) and torch.equal(cv[0, 0, 0, ctx:ctx + Ls], vs[0, 0, :, 0])
    assert torch.equal(ck[0, 0, 0, cap - 1], dk[0, 0, 0]) and torch.equal(cv[0, 0, 0, cap - 1], dv[0, 0, 0])

    toks = np.array([0, Ls - 1])
    qh = np.transpose(host(q)[0, 0][toks], (1, 0, 2))                       # [Hq][2][D]
    ref = O.attention(qh, ctx + toks, K, V, np.arange(cap))
    assert_attn_close(np.transpose(host(out)[0, 0][toks], (1, 0, 2)), ref, "bf16")
    ref = O.attention(host(dq)[0, 0][:, None], [cap - 1], K, V, np.arange(cap))[:, 0]
    assert_attn_close(host(dout)[0, 0], ref, "bf16")


@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_fused_rope_decode_more_than_16_query_heads_per_kv_head(pairing):
    # 20 query heads per kv head (two head groups, each streaming the context; only the first
    # stores the new token) with fused RoPE, split and unsplit: bit-identical to turning q and
    # the new key with pic_rerotate_keys and calling the plain decode
    Hq, Hkv, D, B, steps = 40, 2, 128, 3, 2
    base = np.array([900, 33, 2100], np.int32)
    max_base = int(base.max())
    cap, mad = max_base + steps + 3, max_base + steps
    m = pic.Model.of(1, Hq, Hkv, D, "bf16", 5e5, pairing=pairing)
    table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init(m, mad, table)
    rng = np.random.default_rng(5)
    bf = lambda shape: to_dev(O.store(rng.standard_normal(shape), "bf16"), torch.bfloat16)
    ck, cv = bf((1, B, Hkv, cap, D)), bf((1, B, Hkv, cap, D))
    base_d = torch.from_numpy(base).to(DEV)

    def turned(x, pos):
        y = torch.empty_like(x)
        pic.pic_rerotate_keys(m, x, y, x.shape[0], x.shape[1], torch.from_numpy(pos.astype(np.int32)).to(DEV),
                              table, mad)
        return y

    for split in (0, 3):
        ck_a, cv_a, ck_b, cv_b = ck.clone(), cv.clone(), ck.clone(), cv.clone()
        ws = torch.zeros(max(pic.pic_decode_workspace_bytes(m, B, max_base + steps, split), 16), dtype=torch.uint8,
                         device=DEV)
        for t in range(steps):
            q, k, v = bf((1, B, Hq, D)), bf((1, B, Hkv, D)), bf((1, B, Hkv, D))
            out_a = torch.zeros((1, B, Hq, D), dtype=torch.bfloat16, device=DEV)
            pic.pic_decode_attn_rope(m, q, k, v, ck_a, cv_a, B, cap, base_d, t, max_base, table, mad, out_a, ws,
                                     n_splits=split)
            out_b = torch.zeros_like(out_a)
            pos = base + t
            pic.pic_decode_attn(m, turned(q[0], pos)[None], turned(k[0], pos)[None], v, ck_b, cv_b, B, cap, base_d,
                                t, max_base, out_b, ws, n_splits=split)
            torch.cuda.synchronize()
            assert torch.equal(out_a, out_b), (split, t)
            assert torch.equal(ck_a, ck_b) and torch.equal(cv_a, cv_b), (split, t)


def test_empty_context_beside_a_long_one():
    # one request composes nothing while the other composes 6 documents: the prefill launch is
    # split over key ranges for the long request, so most of the empty request's ranges see no
    # key at all (their partials carry a -inf maximum the combine must drop); decode likewise,
    # split and unsplit
    w = dataclasses.replace(synth.get("c2"), name="empty_and_long", pool_docs=6, doc_len=1000, docs_per_request=6,
                            n_suffix=45, prefix_len=0, batch=2, decode_steps=2)
    r = setup(w, requests=[[], [5, 0, 3, 1, 4, 2]])
    assert list(r.ctx) == [0, 6000]
    gpu_compose(r)
    out = host(gpu_prefill(r))[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(out[b], ref, "bf16")
    ck0, cv0 = r.dev["cache_k"].clone(), r.dev["cache_v"].clone()
    for n_splits in (0, 7):
        r.dev["cache_k"], r.dev["cache_v"] = ck0.clone(), cv0.clone()
        outs = [host(o)[0] for o in gpu_decode(r, 2, n_splits=n_splits)]
        for b in range(w.batch):
            _, K, V = oracle_prefill(r, b)
            length = int(r.ctx[b]) + w.n_suffix
            for t in range(2):
                ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
                length += 1
                assert_attn_close(outs[t][b], ref, "bf16")


@pytest.mark.parametrize("n_rep", [1, 2, 3, 5, 8])
def test_query_heads_per_kv_head(n_rep):
    # the matrix-core prefill packs the n_rep query heads of a kv head into its rows (row r is
    # token r / n_rep, head r % n_rep, by a multiply-shift division) and decode puts them along
    # N: plain multi-head attention (n_rep 1) and ratios that do not divide a 256-row tile,
    # prefill split and unsplit, decode split and unsplit, every head against the oracle
    for batch, n_suffix in ((2, 29), (32, 64)):
        w = dataclasses.replace(synth.get("c2"), name=f"rep{n_rep}", n_q_heads=4 * n_rep, n_kv_heads=4, pool_docs=5,
                                doc_len=300, docs_per_request=3, n_suffix=n_suffix, prefix_len=7, batch=batch,
                                decode_steps=2)
        r = setup(w)
        gpu_compose(r)
        out = host(gpu_prefill(r))[0]
        for b in range(w.batch):
            ref, _, _ = oracle_prefill(r, b)
            assert_attn_close(out[b], ref, "bf16")
        outs = [host(o)[0] for o in gpu_decode(r, 2, n_splits=3 if batch == 2 else 1)]
        for b in range(w.batch):
            _, K, V = oracle_prefill(r, b)
            length = int(r.ctx[b]) + w.n_suffix
            for t in range(2):
                ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
                length += 1
                assert_attn_close(outs[t][b], ref, "bf16")

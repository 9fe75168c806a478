"""Full-size GPU parity: the workloads at their real shapes, run through the same driver and
launch configuration the benchmark times (one compose launch over all layers, per-layer prefill
and decode calls), checked against the CPU oracle: every request's composed cache on one layer,
and attention (every head of the sampled tokens) plus decode steps on sampled (layer, request)
pairs spanning the first, middle and last layers.

Tolerances as in test_gpu_parity: values bit-exact, bf16 keys within 1 bf16 ulp (+1e-5),
bf16 attention within 2e-2 + 1e-2 |ref| and relative Frobenius error <= 1e-2.
"""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from bench import DeviceWorkload
from oracle import pic_oracle as O

from gpu_path import assert_attn_close, assert_keys_close

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _host(t):
    return t.detach().float().cpu().numpy()


def _rope(w, l):
    """The oracle's rotary transform of layer l of workload w (pairing and frequencies)."""
    if w.rope_scaling == "llama3":
        f = O.llama3_inv_freq(w.head_dim, w.rope_theta)
    else:
        f = O.inv_freq(w.head_dim, w.layer_theta(l))
    return {"pairing": w.rope_pairing, "freqs": f}


def _check_request(wl, l, r, tokens=None, decode_steps=0):
    w = wl.w
    lay = wl.lay
    m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
    pool_k, pool_v = _host(wl.pool_k[l]), _host(wl.pool_v[l])
    K, V = O.compose_request(pool_k, pool_v, m, w.rope_theta, w.dtype, **_rope(w, l))
    n = m.ctx_len
    ck = _host(wl.cache_k[l, r])
    cv = _host(wl.cache_v[l, r])
    assert np.array_equal(cv[:, :n].view(np.uint32), V.view(np.uint32)), "values not bit-exact"
    frac = assert_keys_close(ck[:, :n], K, w.dtype)
    assert frac > 0.999, frac
    Ls = w.n_suffix
    if Ls:
        ks = _host(wl.k_suf[l, r])
        vs = _host(wl.v_suf[l, r])
        Kf = np.concatenate([K, np.transpose(ks, (1, 0, 2))], axis=1)
        Vf = np.concatenate([V, np.transpose(vs, (1, 0, 2))], axis=1)
        assert np.array_equal(ck[:, n:n + Ls].view(np.uint32), Kf[:, n:].view(np.uint32))
        toks = np.arange(Ls) if tokens is None else np.asarray(tokens)
        q = np.transpose(_host(wl.q[l, r])[toks], (1, 0, 2))           # [Hq][nt][D]
        ref = O.attention(q, n + toks, Kf, Vf, np.arange(n + Ls))     # [Hq][nt][D]
        got = np.transpose(_host(wl.out[l, r])[toks], (1, 0, 2))
        assert_attn_close(got, ref, w.dtype)
    else:
        Kf, Vf = K, V
    length = n + Ls
    for t in range(decode_steps):
        ref, Kf, Vf = O.decode_step(Kf, Vf, length, _host(wl.dq[l, r]), _host(wl.dk[l, r]),
                                    _host(wl.dv[l, r]))
        length += 1
        assert_attn_close(_host(wl.dout[t, l, r]), ref, w.dtype)


def test_llama8b_32layer_bench_configuration():
    w = synth.get("c3")
    wl = DeviceWorkload(w, DEV, n_dec=1)
    wl.step()
    torch.cuda.synchronize()
    print(f"[c3] ctx={wl.max_ctx} cap={wl.cap} layers={wl.L}", flush=True)
    for l, r in ((0, 0), (31, 15), (17, 6)):
        _check_request(wl, l, r, decode_steps=1)
        print(f"[c3] layer {l} request {r} ok", flush=True)


def test_llama8b_joint_bench_configuration():
    # Learned block boundaries: the shared header composed before each of the 10 documents
    # (11 placements per request with the prefix), every layer in one compose launch.
    w = synth.get("llama8b_joint")
    wl = DeviceWorkload(w, DEV, n_dec=1)
    wl.step()
    torch.cuda.synchronize()
    print(f"[joint] ctx={wl.max_ctx} cap={wl.cap} layers={wl.L}", flush=True)
    for l, r in ((0, 3), (31, 12)):
        _check_request(wl, l, r, tokens=[0, 63, 127], decode_steps=1)
        print(f"[joint] layer {l} request {r} ok", flush=True)


def test_llama8b_decode_full_per_layer_shape():
    # 64 requests x 16K composed context from a 256-document pool; 2 of the 32 identical
    # layers (per-layer launches are the same) and 3 of the 256 decode steps.
    w = synth.get("c4")
    wl = DeviceWorkload(w, DEV, n_dec=3, layers=2)
    wl.step()
    torch.cuda.synchronize()
    print(f"[c4] ctx={wl.max_ctx} cap={wl.cap}", flush=True)
    for l, r in ((0, 0), (1, 63), (0, 37)):
        _check_request(wl, l, r, decode_steps=3)
        print(f"[c4] layer {l} request {r} ok", flush=True)


def _check_compose_all_requests(wl, l):
    """Every request's composed K/V on layer l, all elements: V bit-exact, K within 1 bf16 ulp."""
    w, lay = wl.w, wl.lay
    pool_k, pool_v = _host(wl.pool_k[l]), _host(wl.pool_v[l])
    for r in range(w.batch):
        m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
        K, V = O.compose_request(pool_k, pool_v, m, w.rope_theta, w.dtype, **_rope(w, l))
        n = m.ctx_len
        assert np.array_equal(_host(wl.cache_v[l, r])[:, :n].view(np.uint32), V.view(np.uint32)), r
        assert assert_keys_close(_host(wl.cache_k[l, r])[:, :n], K, w.dtype) > 0.999, r


@pytest.mark.parametrize("name,layers", [("c3", 2), ("c4", 1), ("c5", 2)])
def test_compose_shared_equals_per_block_full_size(name, layers):
    # The bench's compose (blocks grouped by document run, each run read once) against
    # pic_compose over the blocks as planned, at full per-layer shape: identical caches.
    w = synth.get(name)
    a = DeviceWorkload(w, DEV, n_dec=1, layers=layers)
    b = DeviceWorkload(w, DEV, n_dec=1, layers=layers, shared_compose=False)
    for wl in (a, b):
        lay = wl.lay
        blocks = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                     lay.pool_tokens)[0]
        nb, ng = wl.upload(blocks, wl.blocks_pinned, wl.blocks_dev, wl.groups_dev)
        wl.compose(wl.blocks_dev, wl.groups_dev, nb, ng, wl.cache_k, wl.cache_v, w.batch)
    torch.cuda.synchronize()
    assert torch.equal(a.pool_k, b.pool_k) and torch.equal(a.pool_v, b.pool_v)
    assert torch.equal(a.cache_k, b.cache_k) and torch.equal(a.cache_v, b.cache_v)
    print(f"[{name}] {nb} blocks in {ng} groups: shared compose == per-block compose, {layers} layer(s)",
          flush=True)


def test_llama8b_32layer_compose_all_requests():
    # The bench configuration again: every request's composed cache on the last layer, and
    # attention (all suffix tokens and heads) of one request on the middle layer.
    w = synth.get("c3")
    wl = DeviceWorkload(w, DEV, n_dec=1)
    wl.step()
    torch.cuda.synchronize()
    _check_compose_all_requests(wl, wl.L - 1)
    print(f"[c3] layer {wl.L - 1}: all {w.batch} requests composed correctly", flush=True)
    _check_request(wl, wl.L // 2, 3, decode_steps=1)
    print(f"[c3] layer {wl.L // 2} request 3 ok", flush=True)


def test_qwen7b_32k_all_layers():
    # 8 requests x ~32K context (32 jittered documents in per-request order), 256 suffix
    # tokens, all 28 layers: every request's composed cache on the last layer; attention of
    # every suffix token (all 7 m-tiles of 256 query rows, every head) and one decode step on
    # the first, middle and last layers.
    w = synth.get("c5")
    wl = DeviceWorkload(w, DEV, n_dec=1)
    wl.step()
    torch.cuda.synchronize()
    print(f"[c5] ctx={[int(c) for c in wl.ctx_host]} cap={wl.cap} layers={wl.L}", flush=True)
    _check_compose_all_requests(wl, wl.L - 1)
    print(f"[c5] layer {wl.L - 1}: all {w.batch} requests composed correctly", flush=True)
    for l, r in ((0, 0), (wl.L // 2, 5), (wl.L - 1, 7)):
        _check_request(wl, l, r, decode_steps=1)
        print(f"[c5] layer {l} request {r} ok (all {w.n_suffix} suffix tokens)", flush=True)


def test_llama8b_decode_256_steps_all_layers():
    # The whole decode workload: 64 requests x 16K composed context x 32 layers, 256 decode
    # steps.  The appended region of every request's cache is bit-exact on the first and the
    # last layer; attention at steps 0, 1, 127 and 255 is checked against the oracle for
    # requests {0, 63} on layers {0, 31} plus one more request on the last layer.
    torch.cuda.empty_cache()
    w = synth.get("c4")
    n_dec = w.decode_steps
    wl = DeviceWorkload(w, DEV, n_dec=n_dec)
    wl.step()
    torch.cuda.synchronize()
    L, Ls = wl.L, w.n_suffix
    assert Ls == 0   # the decode workload has no suffix: decoding starts right after the context
    print(f"[c4] ctx={wl.max_ctx} cap={wl.cap} layers={L} steps={n_dec}", flush=True)
    for l in (0, L - 1):
        for r in range(w.batch):
            c = int(wl.ctx_host[r]) + Ls
            for cache, new in ((wl.cache_k, wl.dk), (wl.cache_v, wl.dv)):
                app = cache[l, r, :, c:c + n_dec]
                assert torch.equal(app, new[l, r][:, None, :].expand_as(app)), (l, r)
    print("[c4] appended regions bit-exact", flush=True)
    lay = wl.lay
    for l in (0, L // 2, L - 1):                       # composed context, sampled requests
        pool_k, pool_v = _host(wl.pool_k[l]), _host(wl.pool_v[l])
        for r in (5, 21, 42):
            m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
            K, V = O.compose_request(pool_k, pool_v, m, w.rope_theta, w.dtype, **_rope(w, l))
            n = m.ctx_len
            assert np.array_equal(_host(wl.cache_v[l, r])[:, :n].view(np.uint32), V.view(np.uint32))
            assert assert_keys_close(_host(wl.cache_k[l, r])[:, :n], K, w.dtype) > 0.999
    print("[c4] composed contexts of layers 0/15/31 x requests 5/21/42 ok", flush=True)
    for l, reqs in ((0, (0, 63)), (L - 1, (0, 63, 17))):
        pool_k, pool_v = _host(wl.pool_k[l]), _host(wl.pool_v[l])
        for r in reqs:
            m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
            K, V = O.compose_request(pool_k, pool_v, m, w.rope_theta, w.dtype)
            n = m.ctx_len + Ls
            q, dk, dv = _host(wl.dq[l, r]), _host(wl.dk[l, r]), _host(wl.dv[l, r])
            for t in (0, 1, 127, n_dec - 1):
                Kt = np.concatenate([K, np.repeat(dk[:, None, :], t + 1, axis=1)], axis=1)
                Vt = np.concatenate([V, np.repeat(dv[:, None, :], t + 1, axis=1)], axis=1)
                ref = O.attention(q[:, None, :], np.asarray([n + t]), Kt, Vt, np.arange(n + t + 1))[:, 0]
                assert_attn_close(_host(wl.dout[t, l, r]), ref, w.dtype)
            print(f"[c4] layer {l} request {r} steps 0/1/127/{n_dec - 1} ok", flush=True)


def test_llama8b_frontier_32layer_bench_shape():
    # The 32-layer Llama shape in the general frontier layout (inline 128-token prefix, a
    # 32-token inline span after each of the 10 documents, 128 query tokens): every inline
    # token's K/V at its slot, composed documents around them, and attention of sampled inline
    # tokens (prefix, spans, query) on the first, middle and last layers, plus a decode step.
    w = synth.get("llama8b_frontier")
    wl = DeviceWorkload(w, DEV, n_dec=1)
    wl.step()
    torch.cuda.synchronize()
    lay = wl.lay
    print(f"[frontier] lengths={sorted(set(int(x) for x in wl.length_host))} inline={wl.Ls}", flush=True)
    toks = np.array([0, 127, 128, 140, 159, 300, 447, 448, 500, 575])
    for l, r in ((0, 0), (wl.L // 2, 9), (wl.L - 1, 15)):
        pool_k, pool_v = _host(wl.pool_k[l]), _host(wl.pool_v[l])
        f = O.plan_frontier([lay.items[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
        Kc, Vc = O.compose_request(pool_k, pool_v, f.cached, w.rope_theta, w.dtype)
        ks, vs = _host(wl.k_suf[l, r]), _host(wl.v_suf[l, r])
        T = f.total_len
        ck, cv = _host(wl.cache_k[l, r]), _host(wl.cache_v[l, r])
        assert np.array_equal(cv[:, f.cached.logical_pos].view(np.uint32), Vc.view(np.uint32))
        assert assert_keys_close(ck[:, f.cached.logical_pos], Kc, w.dtype) > 0.999
        assert np.array_equal(ck[:, f.inline_pos].view(np.uint32),
                              np.transpose(ks, (1, 0, 2)).view(np.uint32))
        assert np.array_equal(cv[:, f.inline_pos].view(np.uint32),
                              np.transpose(vs, (1, 0, 2)).view(np.uint32))
        # the full cache by position from the oracle's composed rows and the inline inputs
        K = np.empty((w.n_kv_heads, T, w.head_dim), np.float32)
        V = np.empty_like(K)
        K[:, f.cached.logical_pos], V[:, f.cached.logical_pos] = Kc, Vc
        K[:, f.inline_pos], V[:, f.inline_pos] = np.transpose(ks, (1, 0, 2)), np.transpose(vs, (1, 0, 2))
        q = np.transpose(_host(wl.q[l, r])[toks], (1, 0, 2))
        ref = O.attention(q, f.inline_pos[toks], K, V, np.arange(T))
        assert_attn_close(np.transpose(_host(wl.out[l, r])[toks], (1, 0, 2)), ref, w.dtype)
        dref, _, _ = O.decode_step(K, V, T, _host(wl.dq[l, r]), _host(wl.dk[l, r]), _host(wl.dv[l, r]))
        assert_attn_close(_host(wl.dout[0, l, r]), dref, w.dtype)
        print(f"[frontier] layer {l} request {r} ok", flush=True)


@pytest.mark.parametrize("name", ["llama31_32layer", "interleaved_localglobal_32layer"])
def test_rotary_variant_workloads(name):
    # The 32-layer Llama shape with Llama-3.1 frequency scaling, or with interleaved pairing and
    # per-layer bases: every request's composed cache on a local and on a global layer, and
    # attention of one request on the global layer.
    w = synth.get(name)
    wl = DeviceWorkload(w, DEV, n_dec=1)
    wl.step()
    torch.cuda.synchronize()
    for l in (0, 5):
        _check_compose_all_requests(wl, l)
        print(f"[{name}] layer {l} (base {w.layer_theta(l):g}): all requests composed correctly", flush=True)
    _check_request(wl, 5, 11, decode_steps=1)
    print(f"[{name}] layer 5 request 11 ok", flush=True)


@pytest.mark.parametrize("name", ["c3", "c5"])
def test_paged_prefill_full_size(name):
    # The bench's zero-copy TTFT path at full size (whole-run tiles read from the pool with the
    # queries turned; the others composed into the cache first and read from there): every
    # layer's paged prefill output within the attention tolerance of the
    # suffix prefill over the cache composed afterwards; sampled requests against the oracle.
    import paper_2607_28069_amd as pic
    from gpu_path import host
    w = synth.get(name)
    wl = DeviceWorkload(w, DEV, n_dec=1, layers=4 if name == "c5" else None, paged=True)
    wl.step()
    torch.cuda.synchronize()
    tm = wl.tile_map.cpu().numpy()
    n_run = int((tm[..., 0] >= 0).sum())
    print(f"[{name} paged] whole-run tiles {n_run} of {tm.shape[0] * tm.shape[1]}", flush=True)
    assert n_run > 0
    paged = wl.out.clone()
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(wl.m1, w.batch, w.n_suffix, wl.max_ctx), 16),
                     dtype=torch.uint8, device=DEV)
    for l in range(wl.L):
        pic.pic_suffix_prefill_attn(wl.m1, wl.q[l], wl.k_suf[l], wl.v_suf[l], wl.cache_k[l], wl.cache_v[l],
                                    w.batch, wl.cap, wl.ctx_dev, wl.max_ctx, w.n_suffix, wl.out[l], ws)
    torch.cuda.synchronize()
    for l in range(wl.L):
        assert_attn_close(host(paged[l]), host(wl.out[l]), w.dtype)
    print(f"[{name} paged] all {wl.L} layers within tolerance of compose + prefill", flush=True)
    wl.out.copy_(paged)
    for l, r in ((0, 0), (wl.L - 1, w.batch - 1)):
        _check_request(wl, l, r, tokens=[0, 1, 64, w.n_suffix - 1], decode_steps=1)
        print(f"[{name} paged] layer {l} request {r} ok", flush=True)


def test_llama8b_single_request_path():
    # A request served alone (batch 1) has 16 (m-tile, kv head) units, so its prefill runs
    # split over ~15 key ranges with a combine (the batched launch needs none).  The
    # benchmark's single-request path -- eager, then replayed from a recorded graph -- on two
    # layers of the 32-layer shape, against the oracle on every suffix token and head.
    from bench import single_request_ttft
    w = synth.get("c3")
    wl = DeviceWorkload(w, DEV, n_dec=1, layers=2)
    assert wl.ws_pre.numel() >= 16
    import paper_2607_28069_amd as pic
    assert pic.pic_prefill_workspace_bytes(wl.m1, 1, w.n_suffix, wl.max_ctx) > 0
    wl.out.zero_()
    single_request_ttft(wl, n_requests=1, reps=1, chunks=[0])
    torch.cuda.synchronize()
    lay, r, Ls = wl.lay, 0, w.n_suffix
    m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
    toks = np.arange(Ls)
    for l in range(2):
        K, V = O.compose_request(_host(wl.pool_k[l]), _host(wl.pool_v[l]), m, w.rope_theta, w.dtype,
                                 **_rope(w, l))
        n = m.ctx_len
        Kf = np.concatenate([K, np.transpose(_host(wl.k_suf[l, r]), (1, 0, 2))], axis=1)
        Vf = np.concatenate([V, np.transpose(_host(wl.v_suf[l, r]), (1, 0, 2))], axis=1)
        q = np.transpose(_host(wl.q[l, r])[toks], (1, 0, 2))
        ref = O.attention(q, n + toks, Kf, Vf, np.arange(n + Ls))
        got = np.transpose(_host(wl.out[l, r])[toks], (1, 0, 2))
        assert_attn_close(got, ref, w.dtype)
        print(f"[c3 single request] layer {l} ok", flush=True)


def test_fused_rope_full_size():
    # The 32-layer Llama shape with unrotated request-time tokens (`bench.py --fused-rope`), two
    # layers: prefill outputs, caches and a decode step bit-identical to turning q / k with the
    # re-rotation kernel first and running the plain calls.
    import paper_2607_28069_amd as pic
    w = synth.get("c3")
    wl = DeviceWorkload(w, DEV, n_dec=1, layers=2, fused_rope=True)
    wl.step()
    torch.cuda.synchronize()
    out_f, dout_f = wl.out.clone(), wl.dout.clone()
    ck_f, cv_f = wl.cache_k.clone(), wl.cache_v.clone()
    B, Ls, Hq, Hkv, D = w.batch, w.n_suffix, w.n_q_heads, w.n_kv_heads, w.head_dim
    pos = (wl.ctx_host.astype(np.int64)[:, None] + np.arange(Ls)[None, :]).reshape(-1).astype(np.int32)
    pos_d = torch.from_numpy(pos).to(DEV)
    dpos_d = torch.from_numpy(wl.length_host.astype(np.int32)).to(DEV)   # decode step 0
    wl.fused_rope = False
    for name, shape, p in (("q", (B * Ls, Hq, D), pos_d), ("k_suf", (B * Ls, Hkv, D), pos_d),
                           ("dq", (B, Hq, D), dpos_d), ("dk", (B, Hkv, D), dpos_d)):
        t = getattr(wl, name)
        for l in range(wl.L):
            x = t[l].reshape(shape).contiguous()
            pic.pic_rerotate_keys(wl.m1, x, x, shape[0], shape[1], p, wl.table, wl.mad)
            t[l].copy_(x.reshape(t[l].shape))
    wl.step()
    torch.cuda.synchronize()
    assert torch.equal(out_f, wl.out), "fused-RoPE prefill differs from turn-then-prefill"
    assert torch.equal(dout_f, wl.dout), "fused-RoPE decode differs from turn-then-decode"
    assert torch.equal(ck_f, wl.cache_k) and torch.equal(cv_f, wl.cache_v), "caches differ"
    print("[c3 fused rope] 2 layers bit-identical to turned inputs + plain calls", flush=True)
    _check_request(wl, 1, 5, tokens=[0, 127], decode_steps=1)   # the turned-input run vs the oracle

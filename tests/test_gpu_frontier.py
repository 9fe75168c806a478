"""GPU parity of the general frontier layout (App. C.1; Sec. 2 canonical order P, D_1, S_1, ...,
D_m, S_m, Q with an inline prefix and inline spans between the documents): plan, compose and
frontier prefill through the C ABI against the oracle, then decode steps on the completed cache.

Tolerances as in test_gpu_parity: the plan and copied values bit-exact, bf16 keys within 1 bf16
ulp (+1e-5), attention within 2e-2 + 1e-2 |ref| with relative Frobenius error <= 1e-2 for bf16
and 1e-5 for float32.
"""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from oracle import pic_oracle as O
from synth import inputs as S

from gpu_path import (DEV, assert_attn_close, assert_keys_close, gpu_frontier, gpu_prefill, gpu_compose,
                      host, oracle_frontier, setup, setup_frontier, tdtype, to_dev)

pytestmark = pytest.mark.gpu


def _check_cache_and_out(r, out, n_inl):
    w = r.w
    ck, cv = host(r.dev["cache_k"][0]), host(r.dev["cache_v"][0])
    for b in range(w.batch):
        f = r.fmaps[b]
        ref, K, V = oracle_frontier(r, b)
        T = f.total_len
        assert np.array_equal(cv[b][:, :T].view(np.uint32), V.view(np.uint32)), b
        ip, cp = f.inline_pos, f.cached.logical_pos
        assert np.array_equal(ck[b][:, ip].view(np.uint32), K[:, ip].view(np.uint32)), b
        assert_keys_close(ck[b][:, cp], K[:, cp], w.dtype)
        n = int(n_inl[b])
        got = np.transpose(host(out[0, b, :n]), (1, 0, 2))
        assert_attn_close(got, np.transpose(ref, (1, 0, 2)), w.dtype)
        yield b, K, V


def _decode_after(r, steps, Ks, Vs):
    """Decode steps on the completed frontier cache vs the oracle, every request."""
    w, dt, d = r.w, tdtype(r.w), r.dev
    base = r.ctx.astype(np.int32)
    base_dev = torch.from_numpy(base).to(DEV)
    max_base = int(base.max())
    nbytes = pic.pic_decode_workspace_bytes(r.model, w.batch, max_base + steps, 0)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    dq = S.normal_f32(w, "dq_frontier", (steps, w.batch, w.n_q_heads, w.head_dim))
    dk = S.normal_f32(w, "dk_frontier", (steps, w.batch, w.n_kv_heads, w.head_dim))
    dv = S.normal_f32(w, "dv_frontier", (steps, w.batch, w.n_kv_heads, w.head_dim))
    if w.dtype == "bf16":
        dq, dk, dv = (S.bf16_bits_to_f32(S.f32_to_bf16_bits(x)) for x in (dq, dk, dv))
    lengths = [int(x) for x in base]
    for t in range(steps):
        out = torch.zeros((1, w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=DEV)
        pic.pic_decode_attn(r.model, to_dev(dq[t][None], dt), to_dev(dk[t][None], dt), to_dev(dv[t][None], dt),
                            d["cache_k"], d["cache_v"], w.batch, r.cap, base_dev, t, max_base, out, ws)
        got = host(out[0])
        for b in range(w.batch):
            ref, Ks[b], Vs[b] = O.decode_step(Ks[b], Vs[b], lengths[b], dq[t][b], dk[t][b], dv[t][b])
            lengths[b] += 1
            assert_attn_close(got[b], ref, w.dtype)


@pytest.mark.parametrize("name", ["tiny_frontier_f32", "llama8b_frontier_1layer"])
def test_frontier_workloads(name):
    w = synth.get(name)
    r = setup_frontier(w)
    out, n_inl = gpu_frontier(r)
    torch.cuda.synchronize()
    assert list(n_inl) == [w.n_inline] * w.batch
    Ks, Vs = {}, {}
    for b, K, V in _check_cache_and_out(r, out, n_inl):
        Ks[b], Vs[b] = K, V
    print(f"[{name}] totals {[int(x) for x in r.ctx]}: cache and {w.n_inline} inline tokens ok", flush=True)
    _decode_after(r, 2, Ks, Vs)


def test_frontier_ragged_requests_and_split_keys():
    # Requests with different inline layouts (and so different inline counts, padded to the
    # largest): rows past a request's count stay untouched; the shape runs the key-range split
    # path (checked through the workspace the call asks for).
    w = synth.get("llama8b_frontier_1layer")
    # (at most 100 inline tokens: 2 m-tiles x 4 requests x 8 kv heads = 64 units, so the
    # launch is split over key ranges)
    items = [[-40, 0, -10, 1, -20, 2, -30], [3, 4, -64], [-5, 5, -3, 6, -1], [7, 8, 9, -100]]
    r = setup_frontier(w, items=items, n_inline_cap=100)
    m1 = r.model
    assert pic.pic_frontier_workspace_bytes(m1, w.batch, 100, int(r.ctx.max())) > 0
    out, n_inl = gpu_frontier(r, sentinel=7.0)
    torch.cuda.synchronize()
    assert list(n_inl) == [100, 64, 9, 100]
    for _ in _check_cache_and_out(r, out, n_inl):
        pass
    o = host(out[0])
    for b, n in enumerate(n_inl):
        assert np.all(o[b, n:] == 7.0), b
    print(f"[ragged] totals {[int(x) for x in r.ctx]} inline {[int(x) for x in n_inl]} ok", flush=True)


def test_frontier_call_equals_suffix_call_on_the_plain_layout():
    # The plain layout (documents back to back, query span last) through both entry points:
    # same cache, bit-identical attention outputs.
    w = synth.get("c2")
    r = setup(w)
    gpu_compose(r)
    out_a = gpu_prefill(r).clone()
    ck_a, cv_a = r.dev["cache_k"].clone(), r.dev["cache_v"].clone()
    lay = r.lay
    items = [list(req) + [-w.n_suffix] for req in lay.requests]
    blocks, total, inl, n_inl = pic.pic_plan_frontier(items, lay.doc_offset, lay.doc_len,
                                                      lay.doc_compile_pos, lay.pool_tokens)
    assert np.array_equal(total, r.ctx + w.n_suffix)
    assert np.array_equal(inl, r.ctx[:, None] + np.arange(w.n_suffix)[None, :])
    d = r.dev
    d["cache_k"].zero_()
    d["cache_v"].zero_()
    dt = tdtype(w)
    gpu_compose(r, blocks=blocks)
    out_b = torch.zeros_like(out_a)
    max_len = int(total.max())
    nbytes = pic.pic_frontier_workspace_bytes(r.model, w.batch, w.n_suffix, max_len)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    pic.pic_frontier_prefill_attn(r.model, d["q"], d["k_suf"], d["v_suf"], d["cache_k"], d["cache_v"],
                                  w.batch, r.cap, torch.from_numpy(inl).to(DEV),
                                  torch.from_numpy(n_inl).to(DEV), w.n_suffix, max_len, out_b, ws)
    torch.cuda.synchronize()
    assert torch.equal(d["cache_k"], ck_a) and torch.equal(d["cache_v"], cv_a)
    assert torch.equal(out_a, out_b)

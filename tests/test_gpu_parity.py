"""GPU parity of the cache-hit path against the CPU oracle, through the C ABI.

Tolerances: gather/index results and copied values are bit-exact; float32 re-rotated keys
within 1e-5 absolute; bf16 keys within 1 bf16 ulp of the oracle (which rounds the exact
result once, the kernel rounds its float32 result) plus the float32 bound 1e-5; float32 attention within 1e-5 absolute;
bf16 attention within 2e-2 + 1e-2 |ref| elementwise and a relative Frobenius error <= 1e-2.
"""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
import synth
from oracle import pic_oracle as O
from synth import inputs as S

from gpu_path import (DEV, assert_attn_close, assert_keys_close, gpu_compose, gpu_decode, gpu_prefill,
                      host, oracle_compose, oracle_prefill, setup, tdtype, to_dev)

pytestmark = pytest.mark.gpu


def _check_compose(r, d):
    ck, cv = host(d["cache_k"])[0], host(d["cache_v"])[0]
    fracs = []
    for b in range(r.w.batch):
        K, V = oracle_compose(r, b)
        n = r.ctx[b]
        assert np.array_equal(cv[b][:, :n].view(np.uint32), V.view(np.uint32)), "V not bit-exact"
        fracs.append(assert_keys_close(ck[b][:, :n], K, r.w.dtype))
    return min(fracs)


@pytest.mark.parametrize("name", ["c1", "c2", "llama8b_joint_1layer"])
def test_compose_and_prefill_small_workloads(name):
    w = synth.get(name)
    r = setup(w)
    print(f"[{name}] ctx={list(r.ctx)} cap={r.cap}", flush=True)
    d = gpu_compose(r)
    frac = _check_compose(r, d)
    print(f"[{name}] compose ok, bit-identical keys {frac:.6f}", flush=True)
    if w.dtype == "bf16":
        assert frac > 0.999
    # the prefix is placed where it was compiled: keys bit-identical
    if w.prefix_len:
        ck = host(d["cache_k"])[0]
        pk = r.pool_k[:, r.lay.doc_offset[r.lay.prefix_entry]:][:, : w.prefix_len]
        for b in range(w.batch):
            assert np.array_equal(ck[b][:, : w.prefix_len].view(np.uint32), pk.view(np.uint32))
    out = host(gpu_prefill(r))[0]
    ck, cv = host(d["cache_k"])[0], host(d["cache_v"])[0]
    for b in range(w.batch):
        ref, K2, V2 = oracle_prefill(r, b)
        n = r.ctx[b] + w.n_suffix
        assert np.array_equal(ck[b][:, r.ctx[b]:n].view(np.uint32), K2[:, r.ctx[b]:].view(np.uint32))
        assert np.array_equal(cv[b][:, r.ctx[b]:n].view(np.uint32), V2[:, r.ctx[b]:].view(np.uint32))
        assert_attn_close(out[b], ref, w.dtype)
    print(f"[{name}] prefill ok", flush=True)


def test_composed_keys_equal_keys_rotated_in_place():
    # Full-recompute equivalence in one layer: relocated keys equal raw keys rotated directly
    # at their logical positions (float32 workload, 1e-5).
    w = synth.get("c1")
    r = setup(w)
    d = gpu_compose(r)
    ck = host(d["cache_k"])[0]
    m = r.maps[0]
    direct = O.rope(r.inp["pool_k_raw"][:, m.src_token], m.logical_pos, w.rope_theta)
    assert np.abs(ck[0][:, : m.ctx_len] - direct).max() <= 1e-5


@pytest.mark.parametrize("name", ["c1", "c2", "llama8b_joint_1layer"])
def test_decode_steps(name):
    w = synth.get(name)
    import dataclasses
    w = dataclasses.replace(w, decode_steps=5)
    r = setup(w)
    gpu_compose(r)
    gpu_prefill(r)
    outs = [host(o)[0] for o in gpu_decode(r, 5)]
    for b in range(w.batch):
        _, K, V = oracle_prefill(r, b)
        length = r.ctx[b] + w.n_suffix
        for t in range(5):
            ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
            length += 1
            assert_attn_close(outs[t][b], ref, w.dtype)
    print(f"[{name}] decode ok", flush=True)


def test_rerotate_keys_standalone():
    for dtype, D in (("f32", 64), ("bf16", 128), ("f32", 128), ("bf16", 64)):
        m = pic.Model.of(1, 8, 2, D, dtype, 5e5)
        n, H = 300, 2
        rng = np.random.default_rng(7)
        k = O.store(rng.standard_normal((n, H, D)) * 2, dtype)
        a = rng.integers(0, 20000, n)
        b = rng.integers(0, 20000, n)
        delta = (b - a).astype(np.int32)
        mad = 20000
        table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
        pic.pic_rope_table_init(m, mad, table)
        dt = torch.float32 if dtype == "f32" else torch.bfloat16
        kin = to_dev(k, dt)
        kout = torch.empty_like(kin)
        pic.pic_rerotate_keys(m, kin, kout, n, H, torch.from_numpy(delta).to(DEV), table, mad)
        ref = O.store(O.rerotate_keys(np.transpose(k, (1, 0, 2)), a, b, 5e5), dtype)
        assert_keys_close(np.transpose(host(kout), (1, 0, 2)), ref, dtype)
        # in place gives the same keys as out of place
        kin2 = kin.clone()
        pic.pic_rerotate_keys(m, kin2, kin2, n, H, torch.from_numpy(delta).to(DEV), table, mad)
        assert torch.equal(kin2, kout)
        # delta 0 leaves keys bit-identical
        zero = torch.zeros(n, dtype=torch.int32, device=DEV)
        pic.pic_rerotate_keys(m, kin, kin, n, H, zero, table, mad)
        assert np.array_equal(host(kin).view(np.uint32), k.view(np.uint32))
        # R(d) then R(-d) comes back (float32: 1e-5)
        if dtype == "f32":
            back = torch.empty_like(kout)
            pic.pic_rerotate_keys(m, kout, back, n, H, torch.from_numpy(-delta).to(DEV), table, mad)
            assert np.abs(host(back) - k).max() <= 1e-5


def test_rope_table_values():
    for D, theta in ((64, 1e4), (128, 5e5), (128, 1e6)):
        m = pic.Model.of(1, 4, 2, D, "bf16", theta)
        mad = 40000
        table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
        pic.pic_rope_table_init(m, mad, table)
        t = host(table).reshape(mad + 1, D // 2, 2)
        rows = np.array([0, 1, 2, 777, 33000, 40000])
        ang = rows[:, None].astype(np.float64) * np.power(theta, -2.0 * np.arange(D // 2) / D)[None]
        assert np.array_equal(t[rows, :, 0], np.cos(ang).astype(np.float32)) or \
            np.abs(t[rows, :, 0] - np.cos(ang)).max() <= 6e-8
        assert np.abs(t[rows, :, 1] - np.sin(ang)).max() <= 6e-8
        assert np.all(t[0, :, 0] == 1.0) and np.all(t[0, :, 1] == 0.0)


def test_structured_inputs_bf16():
    """needle, sink, V = 1 and Q = 0 on the 1-layer Llama-shaped workload."""
    w = synth.get("c2")

    def needle(inp, lay):
        # a key of document 3 aligned with the first suffix query of head 0 (raw key; the
        # query is already at its position, so the planted score is only approximately large)
        inp["pool_k_raw"][0, lay.doc_offset[3] + 100] = 6 * inp["q"][0, 0, 0] / np.linalg.norm(inp["q"][0, 0, 0]) * 11.3

    def sink(inp, lay):
        qm = inp["q"].mean(axis=(0, 1, 2))
        qm = qm / np.linalg.norm(qm) * 11.3 * 4
        for e in range(w.pool_docs):
            inp["pool_k_raw"][:, lay.doc_offset[e]] = qm

    def v_one(inp, lay):
        inp["pool_v"][:] = 1.0
        inp["v_suf"][:] = 1.0

    def q_zero(inp, lay):
        inp["q"][:] = 0.0

    for name, mut in (("needle", needle), ("sink", sink), ("v_one", v_one), ("q_zero", q_zero)):
        def mutate(inp, lay, mut=mut):
            mut(inp, lay)
            for k in inp:
                inp[k] = S.bf16_bits_to_f32(S.f32_to_bf16_bits(inp[k]))
        r = setup(w, mutate=mutate)
        gpu_compose(r)
        out = host(gpu_prefill(r))[0]
        for b in range(w.batch):
            ref, _, _ = oracle_prefill(r, b)
            assert_attn_close(out[b], ref, "bf16")
        if name == "v_one":
            assert np.all(np.abs(out - 1.0) <= 2 ** -8)
        print(f"[structured {name}] ok", flush=True)


def test_negative_controls_fail():
    """A GPU result must NOT match the oracle of a wrong layout: document order swapped,
    every shift set to 0, or the frontier moved by one position."""
    w = synth.get("c1")
    r = setup(w)
    d = gpu_compose(r)
    out = host(gpu_prefill(r))[0][0]
    ck = host(d["cache_k"])[0][0]
    good, _, _ = oracle_prefill(r, 0)
    assert np.abs(out - good).max() <= 1e-5
    # (1) wrong document order
    wrong = O.plan_layout([[2, 1, 0]], r.lay.doc_offset, r.lay.doc_len, r.lay.doc_compile_pos)[0]
    Kw, _ = O.compose_request(r.pool_k, r.inp["pool_v"], wrong, w.rope_theta, "f32")
    assert np.abs(ck[:, :272] - Kw).max() > 1e-2
    # (2) no re-rotation (shift 0 everywhere)
    K0 = r.pool_k[:, r.maps[0].src_token]
    assert np.abs(ck[:, 16:272] - K0[:, 16:]).max() > 1e-2
    # (3) frontier off by one: query i sees one key fewer
    K, V = oracle_compose(r, 0)
    Kf = np.concatenate([K, np.transpose(r.inp["k_suf"][0], (1, 0, 2))], axis=1)
    Vf = np.concatenate([V, np.transpose(r.inp["v_suf"][0], (1, 0, 2))], axis=1)
    qs = np.transpose(r.inp["q"][0], (1, 0, 2))
    off = O.attention(qs, 272 + np.arange(16) - 1, Kf, Vf, np.arange(288))
    assert np.abs(out - np.transpose(off, (1, 0, 2))).max() > 1e-3


def test_determinism_bitwise():
    w = synth.get("c2")
    r = setup(w)
    gpu_compose(r)
    a = host(gpu_prefill(r)).copy()
    gpu_compose(r)
    b = host(gpu_prefill(r))
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_ragged_shapes_bf16():
    """Context and suffix lengths that are not tile multiples, uneven requests, a request with
    only the prefix, n_rep = 7 (Qwen-like), and decode with an explicit split count."""
    import dataclasses
    w = dataclasses.replace(synth.get("c2"), name="ragged", n_q_heads=28, n_kv_heads=4,
                            pool_docs=5, doc_len=77, docs_per_request=4, n_suffix=37, prefix_len=13, batch=3,
                            decode_steps=3, doc_len_jitter=(1, 150))
    lay = S.pool_layout(w)
    reqs = [[lay.prefix_entry, 3, 0, 4], [lay.prefix_entry], [2, 1, 0, 3, 4]]
    r = setup(w, requests=reqs, extra_cap=5)
    print(f"[ragged] ctx={list(r.ctx)}", flush=True)
    d = gpu_compose(r)
    _check_compose(r, d)
    out = host(gpu_prefill(r))[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b)
        assert_attn_close(out[b], ref, "bf16")
    outs = [host(o)[0] for o in gpu_decode(r, 3, n_splits=3)]
    for b in range(w.batch):
        _, K, V = oracle_prefill(r, b)
        length = r.ctx[b] + w.n_suffix
        for t in range(3):
            ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b])
            length += 1
            assert_attn_close(outs[t][b], ref, "bf16")


def test_non_default_stream_and_layer_batching():
    """Two layers in one call equal two single-layer calls; work runs on a side stream."""
    w = synth.get("c2")
    r = setup(w)
    d = gpu_compose(r)
    m2 = r.model.with_layers(2)
    dt = tdtype(w)
    pk = torch.cat([d["pool_k"], d["pool_k"].flip(-1)], 0).contiguous()
    pv = torch.cat([d["pool_v"], d["pool_v"] * 2], 0).contiguous()
    shape = (2, w.batch, w.n_kv_heads, r.cap, w.head_dim)
    ck = torch.zeros(shape, dtype=dt, device=DEV)
    cv = torch.zeros(shape, dtype=dt, device=DEV)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        pic.pic_compose(m2, pk, pv, r.lay.pool_tokens, d["blocks"], d["blocks"].numel() // 5,
                        d["table"], d["mad"], ck, cv, w.batch, r.cap)
    s.synchronize()
    for l in range(2):
        ck1 = torch.zeros_like(ck[:1])
        cv1 = torch.zeros_like(cv[:1])
        pic.pic_compose(r.model, pk[l:l + 1].contiguous(), pv[l:l + 1].contiguous(), r.lay.pool_tokens,
                        d["blocks"], d["blocks"].numel() // 5, d["table"], d["mad"], ck1, cv1,
                        w.batch, r.cap)
        assert torch.equal(ck1[0], ck[l]) and torch.equal(cv1[0], cv[l])


@pytest.mark.parametrize("name", ["c1", "c2", "llama8b_joint_1layer", "llama8b_frontier_1layer", "ragged"])
def test_compose_shared_equals_compose(name):
    """pic_compose_shared over pic_plan_shared's groups writes the cache pic_compose writes, bit
    for bit, slots no block covers included (both start from the same random contents); and
    the blocks taken in any order give that cache too."""
    import dataclasses
    if name == "ragged":
        w = dataclasses.replace(synth.get("c2"), name="ragged", n_q_heads=28, n_kv_heads=4, pool_docs=5,
                                doc_len=77, docs_per_request=4, n_suffix=37, prefix_len=13, batch=3,
                                doc_len_jitter=(1, 150))
    else:
        w = synth.get(name)
    lay = S.pool_layout(w)
    if w.frontier:
        blocks = pic.pic_plan_frontier(lay.items, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                       lay.pool_tokens)[0]
    else:
        blocks = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                     lay.pool_tokens)[0]
    L, dt = 2, tdtype(w)
    m = pic.Model.of(L, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype, w.rope_theta)
    cap = int(max(b["dst_slot"] + b["n_tokens"] for b in blocks)) + 5
    g = torch.Generator(device=DEV).manual_seed(3)
    pk = torch.randn((L, w.n_kv_heads, lay.pool_tokens, w.head_dim), device=DEV, generator=g).to(dt)
    pv = torch.randn(pk.shape, device=DEV, generator=g).to(dt)
    init = torch.randn((L, w.batch, w.n_kv_heads, cap, w.head_dim), device=DEV, generator=g).to(dt)
    table = torch.empty(pic.pic_rope_table_bytes(m, cap) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init(m, cap, table)
    dev_blocks = lambda b: torch.from_numpy(np.ascontiguousarray(b).view(np.int32).reshape(-1).copy()).to(DEV)
    ck, cv = init.clone(), init.clone()
    pic.pic_compose(m, pk, pv, lay.pool_tokens, dev_blocks(blocks), len(blocks), table, cap, ck, cv, w.batch, cap)
    rng = np.random.default_rng(1)
    for order in (np.arange(len(blocks)), rng.permutation(len(blocks))):
        sb, gs = pic.pic_plan_shared(blocks[order])
        ck2, cv2 = init.clone(), init.clone()
        pic.pic_compose_shared(m, pk, pv, lay.pool_tokens, dev_blocks(sb), len(sb), torch.from_numpy(gs).to(DEV),
                               len(gs) - 1, table, cap, ck2, cv2, w.batch, cap)
        torch.cuda.synchronize()
        assert torch.equal(ck, ck2) and torch.equal(cv, cv2), name
    print(f"[{name}] {len(blocks)} blocks in {len(gs) - 1} groups: shared compose == compose", flush=True)


def test_compose_shared_skips_blocks_outside_their_group():
    """A group whose later block names another source run or an out-of-range destination: that
    block is skipped (its slots keep their contents), the others are written."""
    w = synth.get("c2")
    lay = S.pool_layout(w)
    blocks = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos, lay.pool_tokens)[0]
    sb, gs = pic.pic_plan_shared(blocks)
    big = int(np.argmax(np.diff(gs)))               # a group with several blocks
    i0, i1 = int(gs[big]), int(gs[big + 1])
    assert i1 - i0 >= 2
    bad = sb.copy()
    bad[i0 + 1]["src_token"] += 1                   # reads another run: skipped
    bad[i1 - 1]["dst_slot"] = 1 << 30               # destination out of range: skipped
    m = pic.Model.of(1, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype, w.rope_theta)
    cap = int(max(b["dst_slot"] + b["n_tokens"] for b in blocks)) + 1
    pk = torch.randn((1, w.n_kv_heads, lay.pool_tokens, w.head_dim), device=DEV).to(torch.bfloat16)
    pv = torch.randn(pk.shape, device=DEV).to(torch.bfloat16)
    table = torch.empty(pic.pic_rope_table_bytes(m, cap) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init(m, cap, table)
    outs = []
    for lst in (sb, bad):
        ck = torch.full((1, w.batch, w.n_kv_heads, cap, w.head_dim), 7.0, dtype=torch.bfloat16, device=DEV)
        cv = ck.clone()
        pic.pic_compose_shared(m, pk, pv, lay.pool_tokens,
                               torch.from_numpy(lst.view(np.int32).reshape(-1).copy()).to(DEV), len(lst),
                               torch.from_numpy(gs).to(DEV), len(gs) - 1, table, cap, ck, cv, w.batch, cap)
        outs.append((host(ck)[0], host(cv)[0]))
    torch.cuda.synchronize()
    for j, (ref, got) in enumerate(zip(outs[0], outs[1])):
        for i in range(len(sb)):
            b = sb[i]
            sl = np.s_[int(b["request"]), :, int(b["dst_slot"]):int(b["dst_slot"]) + int(b["n_tokens"])]
            if i in (i0 + 1, i1 - 1):
                assert np.all(got[sl] == 7.0), (j, i)
            else:
                assert np.array_equal(got[sl].view(np.uint32), ref[sl].view(np.uint32)), (j, i)

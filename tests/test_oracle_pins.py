"""Pins of the CPU oracle against facts fixed by the mathematics, by brute force and by
independent library routines.  None of these checks retypes the oracle's own formula.

The paper prints no worked numeric example for the cache-hit path, so every pin is one
of: a closed form, an identity of rotations (Eq. 3), a property of softmax attention, an
explicit-loop brute force on tiny inputs, or a third-party implementation of a special
case (torch's bf16 cast, HF transformers' rotary embedding, torch SDPA).
"""
import math

import numpy as np
import pytest
import torch
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import pic_oracle as O

rng = np.random.default_rng(1234)


# ------------------------------------------------------------------------------------
# storage rounding
# ------------------------------------------------------------------------------------

def test_round_to_bf16_matches_torch_cast():
    x = rng.standard_normal(200000).astype(np.float32) * np.float32(3.0)
    # exact halfway cases between neighbouring bf16 values (both parities)
    bits = rng.integers(0x3F000000, 0x40800000, size=5000, dtype=np.uint32)
    ties = ((bits & 0xFFFF0000) | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, -ties, np.float32([0.0, 1.0, -2.5, 1e-30, 3e30])])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = O.round_to_bf16(x.astype(np.float64))
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


# ------------------------------------------------------------------------------------
# the rotary transform and Eq. 3
# ------------------------------------------------------------------------------------

@pytest.mark.parametrize("p", [0, 1, 7, 1000, 33000, 200000])
def test_rope_head_dim_2_closed_form(p):
    # D = 2: theta_0 = base^0 = 1, so R(p) is the plane rotation by p radians.
    e1 = O.rope(np.array([[1.0, 0.0]]), [p], 5e5)[0]
    e2 = O.rope(np.array([[0.0, 1.0]]), [p], 5e5)[0]
    assert e1 == pytest.approx([math.cos(p), math.sin(p)], abs=1e-12)
    assert e2 == pytest.approx([-math.sin(p), math.cos(p)], abs=1e-12)


def test_rope_frequencies_and_pairing_match_hf_transformers():
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding, apply_rotary_pos_emb

    for D, theta in [(64, 1e4), (128, 5e5), (128, 1e6)]:
        cfg = LlamaConfig(hidden_size=4 * D, num_attention_heads=4, num_key_value_heads=2,
                          head_dim=D, rope_parameters={"rope_type": "default", "rope_theta": theta})
        emb = LlamaRotaryEmbedding(cfg)
        pos = np.array([0, 1, 2, 5, 17, 100, 513])
        x = rng.standard_normal((2, len(pos), D))
        xt = torch.from_numpy(x)[None]                                   # [1, H, n, D]
        cos, sin = emb(xt, torch.from_numpy(pos)[None])
        _, ref = apply_rotary_pos_emb(xt, xt, cos, sin)
        got = O.rope(x, pos, theta)
        # HF builds its angles in float32; positions are kept small so that is ~1e-5
        np.testing.assert_allclose(got, ref[0].numpy(), atol=2e-4, rtol=0)


@settings(max_examples=60, deadline=None)
@given(half=st.integers(1, 64), p=st.integers(0, 100000), d=st.integers(-100000, 100000),
       theta=st.sampled_from([1e4, 5e5, 1e6]))
def test_rerotation_composition_identity(half, p, d, theta):
    # R(p + d) = R(d) R(p): re-rotating a key compiled at p to p + d equals rotating the
    # raw key at p + d directly.
    D = 2 * half
    k = rng.standard_normal((3, D))
    compiled = O.rope(k, [p] * 3, theta)
    moved = O.rerotate_keys(compiled, [p] * 3, [p + d] * 3, theta)
    direct = O.rope(k, [p + d] * 3, theta)
    np.testing.assert_allclose(moved, direct, atol=1e-9, rtol=0)


def test_rerotation_zero_delta_is_bit_identical_after_storage_rounding():
    # a single document placed where it was compiled (a = b) comes back unchanged
    for dtype in ("f32", "bf16"):
        k = O.store(rng.standard_normal((4, 300, 128)) * 2, dtype)
        pos = np.arange(300) + 77
        out = O.store(O.rerotate_keys(k, pos, pos, 5e5), dtype)
        assert np.array_equal(out.view(np.uint32), k.view(np.uint32))


def test_rerotation_inverse_and_norm():
    k = rng.standard_normal((2, 50, 128))
    a = rng.integers(0, 40000, 50)
    b = rng.integers(0, 40000, 50)
    there = O.rerotate_keys(k, a, b, 1e6)
    back = O.rerotate_keys(there, b, a, 1e6)
    np.testing.assert_allclose(back, k, atol=1e-10)
    # each rotated pair keeps its 2-norm
    n0 = k[..., :64] ** 2 + k[..., 64:] ** 2
    n1 = there[..., :64] ** 2 + there[..., 64:] ** 2
    np.testing.assert_allclose(n1, n0, rtol=1e-12, atol=1e-12)


@settings(max_examples=40, deadline=None)
@given(m=st.integers(0, 50000), n=st.integers(0, 50000))
def test_relative_position_property(m, n):
    # <R(m) q, R(n) k> = <q, R(n - m) k>: attention scores depend on positions only through
    # their difference, which is why a relocated key behaves as if compiled in place.
    q = rng.standard_normal((1, 128))
    k = rng.standard_normal((1, 128))
    lhs = float(O.rope(q, [m], 5e5)[0] @ O.rope(k, [n], 5e5)[0])
    rhs = float(q[0] @ O.rope(k, [n - m], 5e5)[0])
    assert lhs == pytest.approx(rhs, abs=1e-9)


# ------------------------------------------------------------------------------------
# layout
# ------------------------------------------------------------------------------------

def test_layout_tiny_workload_hand_computed():
    # Two 128-token documents (pool entries 0 and 1, compiled from position 0) behind a
    # 16-token prefix (entry 2, stored at position 0): the documents land at offsets 16
    # and 144, so their keys move by 16 and 144, and the context is 272 tokens long.
    doc_offset = np.array([0, 128, 256])
    doc_len = np.array([128, 128, 16])
    compile_pos = np.array([0, 0, 0])
    (m,) = O.plan_layout([[2, 0, 1]], doc_offset, doc_len, compile_pos)
    assert m.ctx_len == 272
    assert np.array_equal(m.src_token[:16], np.arange(256, 272))
    assert np.array_equal(m.logical_pos, np.arange(272))
    delta = m.logical_pos - m.compile_pos
    assert np.all(delta[:16] == 0) and np.all(delta[16:144] == 16) and np.all(delta[144:] == 144)
    assert np.array_equal(m.src_token[16:144], np.arange(0, 128))
    assert np.array_equal(m.src_token[144:], np.arange(128, 256))


@settings(max_examples=50, deadline=None)
@given(st.data())
def test_layout_is_a_bijection(data):
    n_pool = data.draw(st.integers(1, 12))
    lens = np.array(data.draw(st.lists(st.integers(1, 40), min_size=n_pool, max_size=n_pool)))
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]])
    cpos = np.array(data.draw(st.lists(st.integers(0, 500), min_size=n_pool, max_size=n_pool)))
    reqs = [data.draw(st.permutations(range(n_pool)))[: data.draw(st.integers(1, n_pool))]
            for _ in range(3)]
    for r, m in zip(reqs, O.plan_layout(reqs, offs, lens, cpos)):
        assert m.ctx_len == lens[r].sum()
        assert np.array_equal(np.sort(m.logical_pos), np.arange(m.ctx_len))      # no gaps/overlap
        assert len(np.unique(m.src_token)) == m.ctx_len                         # each token once
        expect = np.concatenate([np.arange(offs[e], offs[e] + lens[e]) for e in r])
        assert np.array_equal(m.src_token, expect)                              # request order
        # within a document the delta is constant (one rotation per document)
        start = 0
        for e in r:
            d = (m.logical_pos - m.compile_pos)[start:start + lens[e]]
            assert np.all(d == d[0]) and d[0] == start - cpos[e]
            start += lens[e]


# ------------------------------------------------------------------------------------
# attention
# ------------------------------------------------------------------------------------

def _brute_attention(q, q_pos, k, v, k_pos, scale):
    Hq, nq, D = q.shape
    n_rep = Hq // k.shape[0]
    out = np.zeros_like(q, dtype=np.float64)
    for h in range(Hq):
        g = h // n_rep
        for i in range(nq):
            scores = {}
            for j in range(k.shape[1]):
                if k_pos[j] <= q_pos[i]:
                    acc = 0.0
                    for d in range(D):
                        acc += float(q[h, i, d]) * float(k[g, j, d])
                    scores[j] = acc * scale
            mx = max(scores.values())
            z = sum(math.exp(s - mx) for s in scores.values())
            for d in range(D):
                out[h, i, d] = sum(math.exp(s - mx) * float(v[g, j, d]) for j, s in scores.items()) / z
    return out


def test_attention_brute_force_tiny():
    q = rng.standard_normal((4, 5, 8))
    k = rng.standard_normal((2, 11, 8))
    v = rng.standard_normal((2, 11, 8))
    k_pos = rng.permutation(11)              # physical slot order is arbitrary
    q_pos = np.array([3, 6, 8, 9, 10])
    got = O.attention(q, q_pos, k, v, k_pos, 0.37)
    ref = _brute_attention(q, q_pos, k, v, k_pos, 0.37)
    np.testing.assert_allclose(got, ref, atol=1e-12)


def test_attention_rows_sum_to_one_and_zero_query_is_visible_mean():
    q = rng.standard_normal((6, 9, 16)) * 3
    k = rng.standard_normal((3, 40, 16)) * 3
    q_pos = np.arange(31, 40)
    ones = np.ones((3, 40, 16))
    np.testing.assert_allclose(O.attention(q, q_pos, k, ones, np.arange(40)), 1.0, atol=1e-13)
    v = rng.standard_normal((3, 40, 16))
    out = O.attention(np.zeros_like(q), q_pos, k, v, np.arange(40))
    for i, p in enumerate(q_pos):        # query at position p sees exactly p + 1 keys
        np.testing.assert_allclose(out[:, i], np.repeat(v[:, : p + 1].mean(axis=1), 2, axis=0),
                                   atol=1e-13)


def test_attention_matches_torch_sdpa_gqa():
    Hq, Hkv, nq, nk, D = 8, 2, 7, 50, 32
    q = rng.standard_normal((Hq, nq, D))
    k = rng.standard_normal((Hkv, nk, D))
    v = rng.standard_normal((Hkv, nk, D))
    q_pos = np.arange(nk - nq, nk)
    mask = torch.from_numpy(np.arange(nk)[None, :] <= q_pos[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(np.repeat(k, Hq // Hkv, 0))[None],
        torch.from_numpy(np.repeat(v, Hq // Hkv, 0))[None], attn_mask=mask)[0].numpy()
    np.testing.assert_allclose(O.attention(q, q_pos, k, v, np.arange(nk)), ref, atol=1e-12)


def test_needle_key_returns_its_value():
    D = 64
    q = rng.standard_normal((2, 1, D))
    k = rng.standard_normal((1, 300, D)) * 0.1
    v = rng.standard_normal((1, 300, D))
    k[0, 123] = 8 * q[0, 0] / np.linalg.norm(q[0, 0]) * np.sqrt(D)
    out = O.attention(q[:1], [299], k, v, np.arange(300))
    np.testing.assert_allclose(out[0, 0], v[0, 123], atol=1e-6)


def test_translation_invariance_of_rotated_attention():
    Hq, Hkv, D = 4, 2, 64
    qr = rng.standard_normal((Hq, 6, D))
    kr = rng.standard_normal((Hkv, 30, D))
    v = rng.standard_normal((Hkv, 30, D))
    kp, qp = np.arange(30), np.arange(24, 30)
    base = O.attention(O.rope(qr, qp, 1e4), qp, O.rope(kr, kp, 1e4), v, kp)
    for c in (1, 999, 31337):
        moved = O.attention(O.rope(qr, qp + c, 1e4), qp + c, O.rope(kr, kp + c, 1e4), v, kp + c)
        np.testing.assert_allclose(moved, base, atol=1e-9)


def test_composed_cache_equals_full_recompute_single_layer():
    # Model-free analogue of the teacher/student pair (Eqs. 1-2): keys compiled per
    # document at positions 0.., relocated by the link operator, must equal keys rotated
    # directly at their logical positions in the concatenated prompt; attention of the
    # suffix over either cache is then the same (here vs torch SDPA as an outside check).
    Hq, Hkv, D, theta = 4, 2, 64, 1e4
    lens = np.array([37, 64, 16])           # doc 0, doc 1, prefix (entry 2)
    offs = np.array([0, 37, 101])
    raw_k = rng.standard_normal((Hkv, 117, D)).astype(np.float32)
    raw_v = rng.standard_normal((Hkv, 117, D)).astype(np.float32)
    cpos = np.concatenate([np.arange(37), np.arange(64), np.arange(16)])
    pool_k = O.round_to_f32(O.rope(raw_k, cpos, theta))
    (m,) = O.plan_layout([[2, 1, 0]], offs, lens, np.zeros(3, int))
    K, V = O.compose_request(pool_k, raw_v, m, theta, "f32")
    direct = O.rope(raw_k[:, m.src_token], m.logical_pos, theta)
    np.testing.assert_allclose(K, direct, atol=1e-5, rtol=0)
    assert np.array_equal(V, raw_v[:, m.src_token])

    Ls = 5
    qr = rng.standard_normal((Ls, Hq, D))
    ks = rng.standard_normal((Ls, Hkv, D))
    vs = rng.standard_normal((Ls, Hkv, D))
    sp = m.ctx_len + np.arange(Ls)
    q = np.transpose(O.rope(np.transpose(qr, (1, 0, 2)), sp, theta), (1, 0, 2))
    k_suf = np.transpose(O.rope(np.transpose(ks, (1, 0, 2)), sp, theta), (1, 0, 2))
    out, Kf, Vf = O.suffix_prefill(K, V, q, k_suf, vs)
    full_k = np.concatenate([direct, np.transpose(k_suf, (1, 0, 2))], axis=1)
    full_v = np.concatenate([raw_v[:, m.src_token], np.transpose(vs, (1, 0, 2))], axis=1)
    nk = full_k.shape[1]
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(np.transpose(q, (1, 0, 2)))[None],
        torch.from_numpy(np.repeat(full_k, 2, 0))[None],
        torch.from_numpy(np.repeat(full_v, 2, 0).astype(np.float64))[None],
        attn_mask=torch.from_numpy(np.arange(nk)[None, :] <= sp[:, None]))[0].numpy()
    np.testing.assert_allclose(np.transpose(out, (1, 0, 2)), ref, atol=2e-5)


def test_boundary_layout_hand_computed_and_equal_to_full_recompute():
    # Learned block boundaries (KV Packet / Joint): one shared header entry, compiled at
    # positions 0..2, is placed before every document; each document (with its trailer) was
    # compiled after the header, from position 3.  Request [prefix, H, B, H, A]:
    #   prefix [0, 2) delta 0 | H [2, 5) delta 2 | B [5, 11) delta 2 | H [11, 14) delta 11 |
    #   A [14, 21) delta 11,
    # and the composed keys equal the raw keys rotated at their logical positions, the
    # header's at both of its places.
    Hkv, D, theta = 2, 64, 1e4
    lens = np.array([7, 6, 2, 3])                 # A (5 + trailer 2), B (4 + 2), prefix, header
    offs = np.array([0, 7, 13, 15])
    cpos_e = np.array([3, 3, 0, 0])
    (m,) = O.plan_layout([[2, 3, 1, 3, 0]], offs, lens, cpos_e)
    assert m.ctx_len == 21 and np.array_equal(m.logical_pos, np.arange(21))
    assert np.array_equal(m.src_token, np.r_[13:15, 15:18, 7:13, 15:18, 0:7])
    assert np.array_equal(m.logical_pos - m.compile_pos, np.r_[[0] * 2, [2] * 3, [2] * 6, [11] * 3, [11] * 7])
    raw_k = rng.standard_normal((Hkv, 18, D))
    raw_v = rng.standard_normal((Hkv, 18, D)).astype(np.float32)
    cpos_t = np.concatenate([np.arange(3, 10), np.arange(3, 9), np.arange(2), np.arange(3)])
    pool_k = O.round_to_f32(O.rope(raw_k, cpos_t, theta))
    K, V = O.compose_request(pool_k, raw_v, m, theta, "f32")
    direct = O.rope(raw_k[:, m.src_token], m.logical_pos, theta)
    np.testing.assert_allclose(K, direct, atol=1e-5, rtol=0)
    assert np.array_equal(V, raw_v[:, m.src_token])
    # the two copies of the header differ (rotated 9 positions apart) but carry the same values
    assert not np.allclose(K[:, 2:5], K[:, 11:14]) and np.array_equal(V[:, 2:5], V[:, 11:14])


# ------------------------------------------------------------------------------------
# reader-side rotary variants: scaled frequencies, interleaved pairing, per-layer transforms
# ------------------------------------------------------------------------------------

def test_llama3_scaled_frequencies_match_hf_transformers():
    from transformers import LlamaConfig
    from transformers.modeling_rope_utils import ROPE_INIT_FUNCTIONS
    for theta, factor, lo, hi, orig in ((5e5, 8.0, 1.0, 4.0, 8192), (1e4, 4.0, 2.0, 8.0, 4096)):
        cfg = LlamaConfig(hidden_size=4096, num_attention_heads=32, rope_theta=theta,
                          max_position_embeddings=131072,
                          rope_scaling={"rope_type": "llama3", "factor": factor, "low_freq_factor": lo,
                                        "high_freq_factor": hi, "original_max_position_embeddings": orig})
        ref, _ = ROPE_INIT_FUNCTIONS["llama3"](cfg, "cpu")
        got = O.llama3_inv_freq(128, theta, factor, lo, hi, orig)
        np.testing.assert_allclose(got, ref.double().numpy(), rtol=2e-6, atol=0)
        # all three regimes occur: kept, divided, blended
        base = O.inv_freq(128, theta)
        assert np.any(got == base) and np.any(np.isclose(got, base / factor, rtol=1e-12, atol=0))
        assert np.any((got < base) & ~np.isclose(got, base / factor, rtol=1e-12, atol=0))


def test_interleaved_pairing_matches_complex_multiplication():
    # pairs (x_2i, x_2i+1) as complex numbers x_2i + i x_2i+1, turned by e^{i p theta_i}
    D, theta = 64, 1e4
    x = rng.standard_normal((3, 7, D))
    pos = np.array([0, 1, 5, 100, 2049, 31337, 7])
    f = O.llama3_inv_freq(D, theta, 4.0, 1.0, 4.0, 1024)
    xc = torch.view_as_complex(torch.from_numpy(x).reshape(3, 7, D // 2, 2).contiguous())
    ang = torch.from_numpy(pos.astype(np.float64))[:, None] * torch.from_numpy(f)[None, :]
    ref = torch.view_as_real(xc * torch.polar(torch.ones_like(ang), ang)).reshape(3, 7, D).numpy()
    np.testing.assert_allclose(O.rope(x, pos, theta, "interleaved", f), ref, atol=1e-12)
    assert not np.allclose(O.rope(x, pos, theta, "half", f), ref, atol=1e-3)


@settings(max_examples=40, deadline=None)
@given(st.sampled_from(["half", "interleaved"]), st.integers(0, 5000), st.integers(-3000, 3000),
       st.sampled_from([1e4, 5e5, 1e6]), st.booleans())
def test_rerotation_identity_for_every_variant(pairing, p, d, theta, scaled):
    f = O.llama3_inv_freq(64, theta) if scaled else None
    k = rng.standard_normal((2, 1, 64))
    moved = O.rerotate_keys(O.rope(k, [p], theta, pairing, f), [p], [p + d], theta, pairing, f)
    np.testing.assert_allclose(moved, O.rope(k, [p + d], theta, pairing, f), atol=1e-9)
    q = rng.standard_normal(64)
    lhs = O.rope(q[None], [p], theta, pairing, f)[0] @ O.rope(k[0], [p + d], theta, pairing, f)[0]
    rhs = q @ O.rope(k[0], [d], theta, pairing, f)[0]
    assert abs(lhs - rhs) < 1e-9 * (1 + abs(rhs))


# ------------------------------------------------------------------------------------
# general frontier layout (inline prefix and inline spans between documents)
# ------------------------------------------------------------------------------------

def test_frontier_layout_hand_computed():
    # P (4 inline), D_0 (8 cached), S_1 (2 inline), D_1 (5 cached), Q (3 inline)
    (m,) = O.plan_frontier([[-4, 0, -2, 1, -3]], [0, 8], [8, 5], [0, 0])
    assert m.total_len == 22
    assert m.inline_pos.tolist() == [0, 1, 2, 3, 12, 13, 19, 20, 21]
    assert m.cached.logical_pos.tolist() == list(range(4, 12)) + list(range(14, 19))
    assert m.cached.src_token.tolist() == list(range(0, 8)) + list(range(8, 13))
    assert m.cached.compile_pos.tolist() == list(range(8)) + list(range(5))


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_frontier_layout_is_a_bijection(data):
    n_docs = data.draw(st.integers(1, 5))
    lens = np.asarray(data.draw(st.lists(st.integers(1, 40), min_size=n_docs, max_size=n_docs)))
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]])
    items = data.draw(st.lists(st.one_of(st.integers(0, n_docs - 1), st.integers(-9, -1)),
                               min_size=1, max_size=8))
    (m,) = O.plan_frontier([items], offs, lens, np.zeros(n_docs, int))
    both = np.concatenate([m.cached.logical_pos, m.inline_pos])
    assert sorted(both.tolist()) == list(range(m.total_len))
    assert np.all(np.diff(m.inline_pos) > 0)
    assert m.inline_pos.size == -sum(i for i in items if i < 0)


def test_frontier_without_inner_spans_reduces_to_suffix_prefill():
    Hq, Hkv, D, theta, Ls = 4, 2, 32, 1e4, 6
    lens, offs = np.array([20, 13]), np.array([0, 20])
    pool_k = rng.standard_normal((Hkv, 33, D)).astype(np.float32)
    pool_v = rng.standard_normal((Hkv, 33, D)).astype(np.float32)
    (m,) = O.plan_layout([[1, 0]], offs, lens, np.zeros(2, int))
    (f,) = O.plan_frontier([[1, 0, -Ls]], offs, lens, np.zeros(2, int))
    K, V = O.compose_request(pool_k, pool_v, m, theta, "f32")
    Kc, Vc = O.compose_request(pool_k, pool_v, f.cached, theta, "f32")
    assert np.array_equal(K, Kc) and np.array_equal(V, Vc)
    q = rng.standard_normal((Ls, Hq, D))
    ks = rng.standard_normal((Ls, Hkv, D)).astype(np.float32)
    vs = rng.standard_normal((Ls, Hkv, D)).astype(np.float32)
    a, Ka, Va = O.suffix_prefill(K, V, q, ks, vs)
    b, Kb, Vb = O.frontier_prefill(Kc, Vc, f, q, ks, vs)
    assert np.array_equal(a, b) and np.array_equal(Ka, Kb) and np.array_equal(Va, Vb)


def test_frontier_prefill_equals_full_causal_recompute():
    # Inline prefix, a span between the documents and a query span: composing the cached
    # documents and prefilling every inline token must equal plain causal attention over the
    # whole prompt with every key and query rotated directly at its logical position
    # (torch SDPA with a causal mask as the outside computation).
    Hq, Hkv, D, theta = 4, 2, 64, 1e4
    lens, offs = np.array([30, 21]), np.array([0, 30])
    items = [-5, 1, -4, 0, -6]
    (f,) = O.plan_frontier([items], offs, lens, np.zeros(2, int))
    T, n_inl = f.total_len, f.inline_pos.size
    raw_k = rng.standard_normal((Hkv, T, D))           # by logical position
    raw_v = rng.standard_normal((Hkv, T, D)).astype(np.float32)
    raw_q = rng.standard_normal((Hq, T, D))
    # the offline compiler's output: each document's keys rotated from position 0
    pool_k = np.zeros((Hkv, 51, D), np.float32)
    pool_v = np.zeros((Hkv, 51, D), np.float32)
    pool_k[:, f.cached.src_token] = O.round_to_f32(
        O.rope(raw_k[:, f.cached.logical_pos], f.cached.compile_pos, theta))
    pool_v[:, f.cached.src_token] = raw_v[:, f.cached.logical_pos]
    Kc, Vc = O.compose_request(pool_k, pool_v, f.cached, theta, "f32")
    ip = f.inline_pos
    q = np.transpose(O.rope(raw_q[:, ip], ip, theta), (1, 0, 2))
    k_inl = np.transpose(O.round_to_f32(O.rope(raw_k[:, ip], ip, theta)), (1, 0, 2))
    v_inl = np.transpose(raw_v[:, ip], (1, 0, 2))
    out, K, V = O.frontier_prefill(Kc, Vc, f, q, k_inl, v_inl)
    assert not np.isnan(K).any() and not np.isnan(V).any()

    def rot_half(x, pos):   # textbook rotate-half RoPE in torch, float64
        x = torch.from_numpy(np.asarray(x, np.float64))
        inv = 1.0 / theta ** (torch.arange(0, D, 2, dtype=torch.float64) / D)
        ang = torch.from_numpy(np.asarray(pos, np.float64))[:, None] * inv[None, :]
        cos, sin = torch.cat([ang.cos(), ang.cos()], -1), torch.cat([ang.sin(), ang.sin()], -1)
        x1, x2 = x[..., : D // 2], x[..., D // 2:]
        return x * cos + torch.cat([-x2, x1], -1) * sin

    allpos = np.arange(T)
    qf = rot_half(raw_q, allpos)
    kf = rot_half(raw_k, allpos).repeat_interleave(Hq // Hkv, 0)
    vf = torch.from_numpy(raw_v.astype(np.float64)).repeat_interleave(Hq // Hkv, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(qf[None], kf[None], vf[None],
                                                           is_causal=True)[0].numpy()
    np.testing.assert_allclose(np.transpose(out, (1, 0, 2)), ref[:, ip], atol=2e-5)
    assert n_inl == 15


def test_frontier_mask_hides_later_documents():
    # The span after the first document must not see the second document: making the
    # second document's values huge changes only queries at or after its positions.
    Hq, Hkv, D = 2, 1, 16
    lens, offs = np.array([10, 10]), np.array([0, 10])
    (f,) = O.plan_frontier([[0, -3, 1, -2]], offs, lens, np.zeros(2, int))
    Kc = rng.standard_normal((Hkv, 20, D)).astype(np.float32)
    Vc = rng.standard_normal((Hkv, 20, D)).astype(np.float32)
    q = rng.standard_normal((5, Hq, D))
    ks = rng.standard_normal((5, Hkv, D)).astype(np.float32)
    vs = rng.standard_normal((5, Hkv, D)).astype(np.float32)
    a, _, _ = O.frontier_prefill(Kc, Vc, f, q, ks, vs)
    Vc2 = Vc.copy()
    Vc2[:, 10:] = 1e6                                  # second document (positions 13..22)
    b, _, _ = O.frontier_prefill(Kc, Vc2, f, q, ks, vs)
    assert f.inline_pos.tolist() == [10, 11, 12, 23, 24]
    assert np.array_equal(a[:3], b[:3])
    assert np.abs(b[3:]).max() > 1e3


def test_decode_step_equals_prefill_row():
    Hq, Hkv, D = 4, 2, 32
    K = rng.standard_normal((Hkv, 40, D)).astype(np.float32)
    V = rng.standard_normal((Hkv, 40, D)).astype(np.float32)
    q = rng.standard_normal((3, Hq, D))
    ks = rng.standard_normal((3, Hkv, D)).astype(np.float32)
    vs = rng.standard_normal((3, Hkv, D)).astype(np.float32)
    pre, _, _ = O.suffix_prefill(K, V, q, ks, vs)
    Kd, Vd, length = K, V, 40
    for i in range(3):
        o, Kd, Vd = O.decode_step(Kd, Vd, length, q[i], ks[i], vs[i])
        length += 1
        np.testing.assert_allclose(o, pre[i], atol=1e-13)


# ------------------------------------------------------------------------------------
# planted mistakes: each must be caught by one of the pins above
# ------------------------------------------------------------------------------------

def test_planted_mistakes_are_caught(monkeypatch):
    k = rng.standard_normal((1, 4, 64))

    # (1) inverse taken as R(p) instead of R(p)^T: the composition identity breaks
    with monkeypatch.context() as mp:
        mp.setattr(O, "rope_inverse", O.rope)
        moved = O.rerotate_keys(O.rope(k, [5] * 4, 1e4), [5] * 4, [9] * 4, 1e4)
        assert not np.allclose(moved, O.rope(k, [9] * 4, 1e4), atol=1e-3)

    # (2) pairing (2i, 2i+1) instead of (i, i + D/2): the HF cross-check breaks
    def interleaved(x, pos, theta):
        x = np.asarray(x, np.float64)
        c, s = O._cos_sin(pos, x.shape[-1], theta)
        out = np.empty_like(x)
        out[..., 0::2] = x[..., 0::2] * c - x[..., 1::2] * s
        out[..., 1::2] = x[..., 0::2] * s + x[..., 1::2] * c
        return out
    std = O.rope(k, np.arange(4), 1e4)
    assert not np.allclose(interleaved(k, np.arange(4), 1e4), std, atol=1e-3)

    # (3) frontier off by one (strict <): the zero-query mean check breaks
    q = np.zeros((2, 1, 8))
    kk = rng.standard_normal((1, 10, 8))
    v = rng.standard_normal((1, 10, 8))
    good = O.attention(q, [5], kk, v, np.arange(10))
    bad = O.attention(q, [4], kk, v, np.arange(10))     # what "<" would see at position 5
    assert np.allclose(good[0, 0], v[0, :6].mean(0)) and not np.allclose(bad[0, 0], v[0, :6].mean(0))

    # (4) values rotated as well as keys: the full-recompute check on V breaks
    lens, offs = np.array([8]), np.array([0])
    (m,) = O.plan_layout([[0]], offs, lens, np.array([3]))
    vv = rng.standard_normal((1, 8, 64)).astype(np.float32)
    _, Vc = O.compose_request(vv, vv, m, 1e4, "f32")
    assert np.array_equal(Vc, vv) and not np.allclose(
        O.rerotate_keys(vv, m.compile_pos, m.logical_pos, 1e4), vv, atol=1e-3)

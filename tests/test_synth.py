"""The seeded input generator: determinism, encodings and the workloads' derived sizes."""
import numpy as np
import torch

import synth
from synth import inputs as S


def test_streams_are_deterministic_and_distinct():
    w = synth.get("c1")
    a = S.normal_f32(w, "q", (4, 5))
    b = S.normal_f32(w, "q", (4, 5))
    c = S.normal_f32(w, "k_suf", (4, 5))
    d = S.normal_f32(w, "q", (4, 5), layer=1)
    assert np.array_equal(a, b) and not np.allclose(a, c) and not np.allclose(a, d)


def test_bf16_encoding_is_round_to_nearest_even():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(S.f32_to_bf16_bits(x), ref)


def test_workload_context_lengths():
    expect = {"c1": [272], "c2": [4160] * 4, "c3": [10368] * 16, "c4": [16384] * 64}
    for name, ctx in expect.items():
        lay = S.pool_layout(synth.get(name))
        assert list(S.context_lengths(lay)) == ctx
    w5 = synth.get("c5")
    lay = S.pool_layout(w5)
    ctx = S.context_lengths(lay)
    assert np.all(ctx == ctx[0]) and 32 * 768 <= ctx[0] <= 32 * 1280
    assert np.all((lay.doc_len >= 768) & (lay.doc_len <= 1280))
    for r in lay.requests:                       # every request is a permutation of all 32
        assert sorted(r) == list(range(32))


def test_requests_draw_distinct_documents():
    for name in ("c2", "c3", "c4"):
        w = synth.get(name)
        lay = S.pool_layout(w)
        for r in lay.requests:
            docs = [e for e in r if e != lay.prefix_entry]
            assert len(docs) == w.docs_per_request == len(set(docs))
            assert all(0 <= e < w.pool_docs for e in docs)
        if w.prefix_len:
            assert all(r[0] == lay.prefix_entry for r in lay.requests)


def test_boundary_layouts_put_the_shared_header_before_every_document():
    w = synth.get("llama8b_joint")
    lay = S.pool_layout(w)
    h, tr = w.boundary
    H, P = lay.header_entry, lay.prefix_entry
    assert lay.doc_len[H] == h and lay.doc_compile_pos[H] == 0
    assert lay.doc_len[P] == w.prefix_len and lay.doc_compile_pos[P] == 0
    docs = [e for e in range(len(lay.doc_len)) if e not in (H, P)]
    assert len(docs) == w.pool_docs
    assert np.all(lay.doc_len[docs] == w.doc_len + tr) and np.all(lay.doc_compile_pos[docs] == h)
    for r in lay.requests:
        assert r[0] == P and r[1::2] == [H] * w.docs_per_request
        assert len(set(r[2::2])) == w.docs_per_request and H not in r[2::2]
    assert list(S.context_lengths(lay)) == [w.prefix_len + w.docs_per_request * (h + w.doc_len + tr)] * w.batch

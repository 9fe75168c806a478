"""Host-side checks of the C ABI: the library loads and exports every declared symbol, the
layout planner matches the oracle's slot map bit for bit, and every argument check fails
with its status code before anything is enqueued (so these run without a GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import paper_2607_28069_amd as pic
from oracle import pic_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pic.LIB_PATH):
        from paper_2607_28069_amd.build import build
        build()
    return pic.load()


def test_library_exports_every_declared_symbol(lib):
    header = open(os.path.join(ROOT, "include", "pic.h")).read()
    declared = set(re.findall(r"\b(pic_[a-z0-9_]+)\s*\(", header))
    assert declared == set(pic.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert pic.pic_status_string(-6) == "PIC_ERR_RANGE"


def _expand(blocks, batch):
    """Per request: slot -> (src token, delta) from the planner's gather blocks."""
    out = [dict() for _ in range(batch)]
    for b in blocks:
        assert 1 <= b["n_tokens"] <= pic.PIC_BLOCK_TOKENS
        for t in range(b["n_tokens"]):
            slot = int(b["dst_slot"]) + t
            assert slot not in out[b["request"]]
            out[b["request"]][slot] = (int(b["src_token"]) + t, int(b["delta"]))
    return out


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_planner_matches_oracle_layout(lib, data):
    n_pool = data.draw(st.integers(1, 10))
    lens = np.array(data.draw(st.lists(st.integers(1, 200), min_size=n_pool, max_size=n_pool)))
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    cpos = np.array(data.draw(st.lists(st.integers(0, 3000), min_size=n_pool, max_size=n_pool)))
    batch = data.draw(st.integers(1, 4))
    # requests of distinct entries, or with repeats (a shared header placed before every
    # document, as the boundary layouts do)
    reqs = [list(data.draw(st.permutations(range(n_pool)))[: data.draw(st.integers(0, n_pool))])
            if data.draw(st.booleans()) else data.draw(st.lists(st.integers(0, n_pool - 1), max_size=8))
            for _ in range(batch)]
    blocks, ctx = pic.pic_plan_layout(reqs, offs, lens, cpos, int(lens.sum()))
    maps = O.plan_layout(reqs, offs, lens, cpos)
    got = _expand(blocks, batch)
    for b, m in enumerate(maps):
        assert ctx[b] == m.ctx_len
        assert sorted(got[b]) == list(range(m.ctx_len))
        src = np.array([got[b][s][0] for s in range(m.ctx_len)], dtype=np.int64)
        delta = np.array([got[b][s][1] for s in range(m.ctx_len)], dtype=np.int64)
        assert np.array_equal(src, m.src_token)
        assert np.array_equal(delta, m.logical_pos - m.compile_pos)


def test_planner_boundary_workload_matches_oracle(lib):
    import synth
    from synth import inputs as S
    lay = S.pool_layout(synth.get("llama8b_joint"))
    blocks, ctx = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                      lay.pool_tokens)
    got = _expand(blocks, len(lay.requests))
    for b, m in enumerate(O.plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos)):
        assert ctx[b] == m.ctx_len == 10528
        src = np.array([got[b][s][0] for s in range(m.ctx_len)], dtype=np.int64)
        delta = np.array([got[b][s][1] for s in range(m.ctx_len)], dtype=np.int64)
        assert np.array_equal(src, m.src_token) and np.array_equal(delta, m.logical_pos - m.compile_pos)


def test_planner_tiny_workload(lib):
    blocks, ctx = pic.pic_plan_layout([[2, 0, 1]], [0, 128, 256], [128, 128, 16], [0, 0, 0], 272)
    assert list(ctx) == [272]
    rows = [tuple(int(x) for x in b) for b in blocks]
    assert rows == [(0, 256, 0, 16, 0), (0, 0, 16, 64, 16), (0, 64, 80, 64, 16),
                    (0, 128, 144, 64, 144), (0, 192, 208, 64, 144)]


def test_planner_errors(lib):
    with pytest.raises(pic.PicError) as e:
        pic.pic_plan_layout([[0, 3]], [0, 10], [10, 10], [0, 0], 20)
    assert e.value.status == -6                          # entry id out of range
    with pytest.raises(pic.PicError) as e:
        pic.pic_plan_layout([[0]], [0, 15], [10, 10], [0, 0], 20)
    assert e.value.status == -6                          # entry outside the pool
    with pytest.raises(pic.PicError) as e:
        pic.pic_plan_layout([[0]], [0], [0], [0], 20)
    assert e.value.status == -1                          # empty entry
    n = ctypes.c_int32(0)
    ctx = np.zeros(1, np.int32)
    one = np.array([1], np.int32)
    z = np.array([0], np.int32)
    ln = np.array([200], np.int32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    blk = np.zeros(2, pic.BLOCK_DTYPE)
    st_ = lib.pic_plan_layout(1, P(one), P(z), 1, P(z), P(ln), P(z), 200, P(blk), 2, ctypes.byref(n), P(ctx))
    assert st_ == -4 and n.value == 4                    # capacity: 4 blocks needed
    assert "4 blocks needed" in pic.pic_last_error()


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_frontier_planner_matches_oracle_layout(lib, data):
    n_pool = data.draw(st.integers(1, 8))
    lens = np.array(data.draw(st.lists(st.integers(1, 150), min_size=n_pool, max_size=n_pool)))
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    cpos = np.array(data.draw(st.lists(st.integers(0, 3000), min_size=n_pool, max_size=n_pool)))
    batch = data.draw(st.integers(1, 4))
    items = [data.draw(st.lists(st.one_of(st.integers(0, n_pool - 1), st.integers(-70, -1)),
                                max_size=7)) for _ in range(batch)]
    blocks, total, inl, n_inl = pic.pic_plan_frontier(items, offs, lens, cpos, int(lens.sum()))
    maps = O.plan_frontier(items, offs, lens, cpos)
    got = _expand(blocks, batch)
    for b, m in enumerate(maps):
        assert total[b] == m.total_len
        assert n_inl[b] == m.inline_pos.size
        assert np.array_equal(inl[b, : n_inl[b]], m.inline_pos)
        assert np.all(inl[b, n_inl[b]:] == -1)
        slots = np.array(sorted(got[b]), dtype=np.int64)
        assert np.array_equal(slots, m.cached.logical_pos)
        src = np.array([got[b][s][0] for s in slots], dtype=np.int64)
        delta = np.array([got[b][s][1] for s in slots], dtype=np.int64)
        assert np.array_equal(src, m.cached.src_token)
        assert np.array_equal(delta, m.cached.logical_pos - m.cached.compile_pos)


def test_frontier_planner_hand_layout_and_errors(lib):
    blocks, total, inl, n_inl = pic.pic_plan_frontier([[-4, 0, -2, 1, -3]], [0, 8], [8, 5], [0, 0], 13)
    assert list(total) == [22] and list(n_inl) == [9]
    assert inl[0].tolist() == [0, 1, 2, 3, 12, 13, 19, 20, 21]
    assert [tuple(int(x) for x in b) for b in blocks] == [(0, 0, 4, 8, 4), (0, 8, 14, 5, 14)]
    with pytest.raises(pic.PicError) as e:
        pic.pic_plan_layout([[-3, 0]], [0], [8], [0], 8)   # inline spans only in the frontier planner
    assert e.value.status == -6
    n, tot, ninl = ctypes.c_int32(0), np.zeros(1, np.int32), np.zeros(1, np.int32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    pos = np.zeros(2, np.int32)
    st_ = lib.pic_plan_frontier(1, P(np.array([2], np.int32)), P(np.array([-3, 0], np.int32)), 1,
                                P(np.array([0], np.int32)), P(np.array([8], np.int32)),
                                P(np.array([0], np.int32)), 8, None, 0, ctypes.byref(n), P(tot),
                                P(pos), 2, P(ninl))
    assert st_ == -4 and "3 inline tokens, room for 2" in pic.pic_last_error()


FAKE = 0x10000          # an aligned, never-dereferenced device address
MIS = 0x10008           # misaligned


def _model(**kw):
    base = dict(n_layers=1, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16", rope_theta=5e5)
    base.update(kw)
    return pic.Model.of(**base)


def _compose(lib, m, **kw):
    a = dict(pool_k=FAKE, pool_v=FAKE, pool_tokens=1000, blocks=FAKE, n_blocks=4, table=FAKE,
             max_abs_delta=100, cache_k=FAKE, cache_v=FAKE, batch=2, cache_cap=1000)
    a.update(kw)
    return lib.pic_compose(ctypes.byref(m), a["pool_k"], a["pool_v"], a["pool_tokens"], a["blocks"],
                           a["n_blocks"], a["table"], a["max_abs_delta"], a["cache_k"], a["cache_v"],
                           a["batch"], a["cache_cap"], None)


def _prefill(lib, m, ws_bytes=0, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, ck=FAKE, cv=FAKE, batch=2, cap=600, ctx=FAKE, max_ctx=500,
             ns=64, scale=0.0, out=FAKE)
    a.update(kw)
    return lib.pic_suffix_prefill_attn(ctypes.byref(m), a["q"], a["k"], a["v"], a["ck"], a["cv"],
                                       a["batch"], a["cap"], a["ctx"], a["max_ctx"], a["ns"],
                                       a["scale"], a["out"], None, ws_bytes, None)


def _decode(lib, m, ws=FAKE, ws_bytes=1 << 30, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, ck=FAKE, cv=FAKE, batch=2, cap=600, base=FAKE, step=0,
             max_base=500, scale=0.0, splits=0, out=FAKE)
    a.update(kw)
    return lib.pic_decode_attn(ctypes.byref(m), a["q"], a["k"], a["v"], a["ck"], a["cv"], a["batch"],
                               a["cap"], a["base"], a["step"], a["max_base"], a["scale"], a["splits"],
                               a["out"], ws, ws_bytes, None)


def _frontier(lib, m, ws_bytes=0, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, ck=FAKE, cv=FAKE, batch=2, cap=600, pos=FAKE, nv=FAKE, n=64,
             max_len=600, scale=0.0, out=FAKE)
    a.update(kw)
    return lib.pic_frontier_prefill_attn(ctypes.byref(m), a["q"], a["k"], a["v"], a["ck"], a["cv"],
                                         a["batch"], a["cap"], a["pos"], a["nv"], a["n"],
                                         a["max_len"], a["scale"], a["out"], None, ws_bytes, None)


def _paged(lib, m, ws_bytes=1 << 30, **kw):
    a = dict(pool_k=FAKE, pool_v=FAKE, pool_tokens=1000, smap=FAKE, dmap=FAKE, map_cap=500, tmap=FAKE,
             table=FAKE, mad=600, q=FAKE, k=FAKE, v=FAKE, ck=FAKE, cv=FAKE, batch=2, cap=600, ctx=FAKE,
             max_ctx=500, ns=64, scale=0.0, out=FAKE, ws=FAKE)
    a.update(kw)
    return lib.pic_paged_prefill_attn(ctypes.byref(m), a["pool_k"], a["pool_v"], a["pool_tokens"], a["smap"],
                                      a["dmap"], a["map_cap"], a["tmap"], a["table"], a["mad"], a["q"], a["k"],
                                      a["v"], a["ck"], a["cv"], a["batch"], a["cap"], a["ctx"], a["max_ctx"],
                                      a["ns"], a["scale"], a["out"], a["ws"], ws_bytes, None)


def test_argument_checks_fail_before_any_launch(lib):
    m = _model()
    assert _compose(lib, _model(head_dim=96)) == -2
    assert _compose(lib, _model(n_q_heads=30)) == -1
    assert _compose(lib, _model(dtype=7)) == -2
    assert _compose(lib, m, pool_k=None) == -1
    assert _compose(lib, m, cache_v=MIS) == -5
    assert _compose(lib, m, max_abs_delta=-1) == -6
    assert _compose(lib, m, batch=-1) == -1
    assert _compose(lib, m, n_blocks=0) == 0            # nothing to do, nothing launched

    assert _prefill(lib, m, max_ctx=580) == -4           # 580 + 64 > cache_cap 600
    assert _prefill(lib, m, q=MIS) == -5
    assert _prefill(lib, m, ctx=None) == -1
    assert _prefill(lib, m, scale=-1.0) == -1
    assert _prefill(lib, _model(head_dim=64)) != -2      # bf16 at head_dim 64: the row-wise kernel
    assert _prefill(lib, m, ns=0) == 0

    assert _frontier(lib, m, max_len=601) == -4          # longer than the cache
    assert _frontier(lib, m, pos=None) == -1
    assert _frontier(lib, m, nv=None) == -1
    assert _frontier(lib, m, k=MIS) == -5
    assert _frontier(lib, m, n=-1) == -1
    assert _frontier(lib, m, scale=float("nan")) == -1
    assert _frontier(lib, _model(head_dim=64)) != -2
    assert _frontier(lib, m, n=0) == 0

    assert _paged(lib, m, map_cap=499) == -4             # the map must cover max_ctx
    assert _paged(lib, m, max_ctx=580) == -4             # 580 + 64 > cache_cap 600
    assert _paged(lib, m, smap=None) == -1
    assert _paged(lib, m, ctx=None) == -1
    assert _paged(lib, m, mad=-1) == -6
    assert _paged(lib, m, pool_tokens=0) == -6           # documents but no pool
    assert _paged(lib, m, q=MIS) == -5
    assert _paged(lib, m, tmap=MIS) == -5
    assert lib.pic_build_slot_map(FAKE, 4, 2, 500, FAKE, FAKE, MIS, None) == -5
    assert _paged(lib, _model(dtype="f32")) == -2
    assert _paged(lib, m, ws=None, ws_bytes=0, max_ctx=4000, map_cap=4000, cap=5000) == -3   # split-K
    assert _paged(lib, m, batch=0) == 0
    # the prefill kernels use 32-bit byte offsets: a cache stream, a request's suffix rows and
    # a pool head each stay below 2^24 rows of 256 bytes
    assert _prefill(lib, m, cap=1 << 24) == -2
    assert _frontier(lib, m, cap=1 << 24) == -2
    assert _paged(lib, m, cap=1 << 24) == -2
    assert _paged(lib, m, pool_tokens=1 << 24) == -2
    assert _paged(lib, m, pool_tokens=(1 << 24) - 1) != -2
    assert lib.pic_build_slot_map(FAKE, 4, 2, 500, None, FAKE, FAKE, None) == -1
    assert lib.pic_build_slot_map(None, 4, 2, 500, FAKE, FAKE, None, None) == -1
    assert lib.pic_build_slot_map(FAKE, -1, 2, 500, FAKE, FAKE, None, None) == -1
    assert lib.pic_build_slot_map(FAKE, 4, 0, 500, FAKE, FAKE, FAKE, None) == 0   # empty map

    # fused RoPE: the table must cover every position the call turns
    rp = lambda mm, table=FAKE, mad=600, ws_bytes=1 << 30: lib.pic_suffix_prefill_attn_rope(
        ctypes.byref(mm), FAKE, FAKE, FAKE, FAKE, FAKE, 2, 600, FAKE, 500, 64, table, mad, 0.0, FAKE, FAKE,
        ws_bytes, None)
    assert rp(m, mad=562) == -6                          # positions up to 563
    assert rp(m, table=None) == -1
    assert rp(m, table=MIS) == -5
    assert rp(_model(dtype="f32", head_dim=64)) == -2
    rd = lambda table=FAKE, mad=600: lib.pic_decode_attn_rope(
        ctypes.byref(m), FAKE, FAKE, FAKE, FAKE, FAKE, 2, 600, FAKE, 3, 500, table, mad, 0.0, 0, FAKE, FAKE,
        1 << 30, None)
    assert rd(mad=502) == -6                             # position 503
    assert rd(table=None) == -1

    assert _decode(lib, m, step=100) == -4               # 500 + 100 + 1 > 600
    assert _decode(lib, m, ws=None) == -3
    assert _decode(lib, m, ws_bytes=16) == -3
    assert _decode(lib, _model(n_q_heads=136, n_kv_heads=8)) != -2   # 17 heads per kv head: two head groups
    assert _decode(lib, m, base=None) == -1
    assert "base_len" in pic.pic_last_error()

    assert lib.pic_rerotate_keys(ctypes.byref(m), FAKE, FAKE, 10, 8, None, FAKE, 10, None) == -1
    assert lib.pic_rerotate_keys(ctypes.byref(m), MIS, FAKE, 10, 8, FAKE, FAKE, 10, None) == -5
    assert lib.pic_rerotate_keys(ctypes.byref(m), FAKE, FAKE, 1 << 62, 8, FAKE, FAKE, 10, None) == -6
    assert lib.pic_rope_table_init(ctypes.byref(m), 10, FAKE, 16, None) == -4
    assert lib.pic_rope_table_init(ctypes.byref(_model(rope_theta=0.5)), 10, FAKE, 1 << 20, None) == -1


def test_sizes(lib):
    m = _model()
    assert pic.pic_rope_table_bytes(m, 65535) == 65536 * 64 * 8
    assert pic.pic_rope_table_bytes(m, -1) == 0
    assert pic.pic_rope_table_bytes(m, (1 << 20) + 1) == 0
    s = pic.pic_decode_auto_splits(m, 64, 16640)
    assert s >= 1
    # fp32 partials (head_dim outputs + max + denominator) per split; none without a split
    assert pic.pic_decode_workspace_bytes(m, 64, 16640, 0) == (0 if s == 1 else 64 * 32 * s * 130 * 4)
    assert pic.pic_decode_workspace_bytes(m, 64, 16640, 1) == 0
    assert pic.pic_decode_workspace_bytes(m, 64, 16640, 3) == 64 * 32 * 3 * 130 * 4
    assert pic.pic_decode_auto_splits(m, 1, 16640) > 1
    assert pic.pic_prefill_workspace_bytes(_model(dtype="f32", head_dim=64), 1, 16, 272) == 0
    # bf16 prefill splits: per split and query row, the normalised output in bf16 (256 bytes)
    # and the (max, sum) pair in fp32 (8 bytes); a lone 32-layer-Llama-shaped request splits
    # (16 (m-tile, kv head) units), a batch of 16 does not
    m32 = _model(n_layers=1, n_q_heads=32, n_kv_heads=8)
    rows = 1 * 128 * 32
    ws = pic.pic_prefill_workspace_bytes(m32, 1, 128, 10368)
    assert ws > 0 and ws % (rows * 264) == 0 and 2 <= ws // (rows * 264) <= 32, ws
    assert pic.pic_prefill_workspace_bytes(m32, 16, 128, 10368) == 0


def test_plan_shared_groups_blocks_by_source():
    """pic_plan_shared: a stable permutation of the blocks in which every group reads one pool
    run (equal src_token and n_tokens) and different groups read different runs; on the
    workloads every document chunk a batch places several times becomes one group."""
    import synth
    from synth import inputs as S
    for name in ("c1", "c2", "c3", "llama8b_joint_1layer", "llama8b_frontier_1layer"):
        w = synth.get(name)
        lay = S.pool_layout(w)
        if w.frontier:
            blocks = pic.pic_plan_frontier(lay.items, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                           lay.pool_tokens)[0]
        else:
            blocks = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                         lay.pool_tokens)[0]
        sb, gs = pic.pic_plan_shared(blocks)
        key = lambda b: (int(b["src_token"]), int(b["n_tokens"]))
        # stable permutation: sorting the input by source run gives the output exactly
        order = sorted(range(len(blocks)), key=lambda i: key(blocks[i]))
        assert np.array_equal(sb, blocks[order])
        assert gs[0] == 0 and gs[-1] == len(blocks) and np.all(np.diff(gs) > 0)
        runs = [key(sb[gs[g]]) for g in range(len(gs) - 1)]
        for g in range(len(gs) - 1):
            assert all(key(b) == runs[g] for b in sb[gs[g]:gs[g + 1]])
        # one group per distinct run, split into groups of at most 8 blocks
        counts = {}
        for b in blocks:
            counts[key(b)] = counts.get(key(b), 0) + 1
        assert np.all(np.diff(gs) <= 8)
        assert len(runs) == sum((c + 7) // 8 for c in counts.values())
        assert all(runs[g] != runs[g + 1] or gs[g + 1] - gs[g] == 8 for g in range(len(runs) - 1))
    # requests sharing documents share groups: 16 requests x 10 of 64 documents
    w = synth.get("c3")
    lay = S.pool_layout(w)
    blocks = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos, lay.pool_tokens)[0]
    assert len(blocks) / (len(pic.pic_plan_shared(blocks)[1]) - 1) > 2
    assert len(pic.pic_plan_shared(blocks[:0])[0]) == 0


def test_compose_shared_argument_checks(lib):
    m = _model()
    n = ctypes.c_int32(0)
    starts = (ctypes.c_int32 * 4)()
    assert lib.pic_plan_shared(None, 3, None, starts, ctypes.byref(n)) == -1
    assert lib.pic_plan_shared(None, -1, None, starts, ctypes.byref(n)) == -1
    a = dict(pool_k=FAKE, pool_v=FAKE, pool_tokens=1000, blocks=FAKE, n_blocks=4, starts=FAKE, n_groups=2,
             table=FAKE, mad=100, ck=FAKE, cv=FAKE, batch=2, cap=1000)
    call = lambda **kw: lib.pic_compose_shared(ctypes.byref(m), *{**a, **kw}.values(), None)
    assert call(n_groups=5) == -1                  # more groups than blocks
    assert call(starts=None) == -1
    assert call(pool_k=MIS) == -5
    assert call(mad=1 << 30) == -6
    assert call(n_groups=0) == 0                   # nothing to do: nothing launched


def test_rotary_variant_arguments(lib):
    m = _model(n_layers=3)
    one = pic.pic_rope_table_bytes(m, 100)
    assert one == 101 * 64 * 8
    per_layer = pic.Model.of(3, 32, 8, 128, "bf16", 5e5, per_layer_tables=True)
    assert pic.pic_rope_table_bytes(per_layer, 100) == 3 * one
    assert per_layer.with_layers(1).rope_tables == 1
    bad = pic.Model.of(3, 32, 8, 128, "bf16", 5e5)
    bad.rope_tables = 2                                   # neither 1 nor n_layers
    assert pic.pic_rope_table_bytes(bad, 100) == 0
    assert _compose(lib, bad) == -1
    bad = pic.Model.of(1, 32, 8, 128, "bf16", 5e5)
    bad.rope_pairing = 2
    assert _compose(lib, bad) == -1
    f = np.full(64, 0.5)
    f[3] = np.nan
    st_ = lib.pic_rope_table_init_freq(ctypes.byref(m), f.ctypes.data_as(ctypes.c_void_p), 10, FAKE,
                                       1 << 20, None)
    assert st_ == -1 and "inv_freq[3]" in pic.pic_last_error()
    with pytest.raises(pic.PicError):
        pic.pic_rope_llama3_freq(128, 5e5, 8.0, 4.0, 1.0)  # high_freq_factor <= low_freq_factor


def test_llama3_frequencies_match_transformers_and_oracle(lib):
    from transformers import LlamaConfig
    from transformers.modeling_rope_utils import ROPE_INIT_FUNCTIONS
    cfg = LlamaConfig(hidden_size=4096, num_attention_heads=32, rope_theta=5e5,
                      max_position_embeddings=131072,
                      rope_scaling={"rope_type": "llama3", "factor": 8.0, "low_freq_factor": 1.0,
                                    "high_freq_factor": 4.0, "original_max_position_embeddings": 8192})
    ref, _ = ROPE_INIT_FUNCTIONS["llama3"](cfg, "cpu")
    got = pic.pic_rope_llama3_freq(128, 5e5)
    np.testing.assert_allclose(got, ref.double().numpy(), rtol=2e-6, atol=0)
    np.testing.assert_allclose(got, O.llama3_inv_freq(128, 5e5), rtol=1e-14, atol=0)


def test_binding_refuses_host_and_strided_buffers(lib):
    # The library reads every tensor argument as a dense device array: the binding stops a
    # host tensor or a strided view before any call is made.
    import torch
    m = pic.Model.of(1, 4, 2, 64, "f32", 1e4)
    host = torch.zeros(16, 64)
    with pytest.raises(ValueError, match="host tensor"):
        pic.pic_rerotate_keys(m, host, host, 16, 1, None, None, 0)
    with pytest.raises(ValueError, match="host tensor"):
        pic._ptr(host[::2])
    assert pic._ptr(None) is None


def test_compose_tiles_argument_checks(lib):
    """pic_compose_tiles and the paged prefill without a slot map: refused before any launch."""
    m = _model()
    args = dict(pool_k=FAKE, pool_v=FAKE, pool_tokens=1000, slot_src=FAKE, slot_delta=FAKE, map_cap=600,
                tile_map=FAKE, table=FAKE, max_abs_delta=100, ctx_len=FAKE, max_ctx=500, cache_k=FAKE,
                cache_v=FAKE, batch=2, cache_cap=600)

    def call(model, **kw):
        a = dict(args, **kw)
        return lib.pic_compose_tiles(ctypes.byref(model), *[a[k] for k in (
            "pool_k", "pool_v", "pool_tokens", "slot_src", "slot_delta", "map_cap", "tile_map", "table",
            "max_abs_delta", "ctx_len", "max_ctx", "cache_k", "cache_v", "batch", "cache_cap")], None)

    assert call(m, tile_map=None) == -1
    assert call(m, slot_src=None) == -1
    assert call(m, ctx_len=None) == -1
    assert call(m, map_cap=400) == -4                   # the map must cover max_ctx
    assert call(m, max_ctx=700) == -4                   # longer than the cache
    assert call(m, max_abs_delta=-1) == -6
    assert call(_model(dtype="f32")) == -2              # built for bf16 caches
    assert call(m, batch=0) == 0                        # nothing to do, nothing launched
    # the paged prefill: no slot map needs a tile map; one map alone is refused
    common = [FAKE, FAKE, 1000]
    tail = [FAKE, 100, FAKE, FAKE, FAKE, FAKE, FAKE, 2, 600, FAKE, 500, 64, ctypes.c_float(0.0), FAKE, None,
            ctypes.c_size_t(0), None]
    assert lib.pic_paged_prefill_attn(ctypes.byref(m), *common, None, None, 600, None, *tail) == -1
    assert lib.pic_paged_prefill_attn(ctypes.byref(m), *common, FAKE, None, 600, FAKE, *tail) == -1
    # head_dim 64 takes the tile-map-only form too: the call gets past the slot-map check and stops
    # at the missing ctx_len (nothing launched)
    no_ctx = tail[:9] + [None] + tail[10:]
    assert lib.pic_paged_prefill_attn(ctypes.byref(_model(head_dim=64)), *common, None, None, 600, FAKE,
                                      *no_ctx) == -1
    assert b"ctx_len" in lib.pic_last_error()


def test_noalloc_decode_argument_checks(lib):
    # The allocation-free decode checks like pic_decode_attn and refuses, before any launch or
    # scratch lookup, split partials larger than its per-GPU scratch array.
    m = _model()
    nd = lambda mm=m, batch=2, step=0, max_base=500, splits=0, q=FAKE, base=FAKE, cap=600: \
        lib.pic_decode_attn_noalloc(ctypes.byref(mm), q, FAKE, FAKE, FAKE, FAKE, batch, cap, base, step,
                                    max_base, 0.0, splits, FAKE, None)
    assert nd(step=100) == -4                            # 500 + 100 + 1 > 600
    assert nd(q=MIS) == -5
    assert nd(base=None) == -1
    assert nd(_model(n_q_heads=136, n_kv_heads=8)) != -2   # two groups of query heads
    assert nd(batch=0) == 0                              # nothing to do
    # 64 requests x 32 heads x 64 splits of (128 + 2) floats: 68 MB > the 8 MiB array
    need = pic.pic_decode_workspace_bytes(m, 64, 502, 64)
    assert need > pic.PIC_DECODE_SCRATCH_BYTES
    assert nd(batch=64, splits=64) == -3
    assert "allocation-free" in pic.pic_last_error()

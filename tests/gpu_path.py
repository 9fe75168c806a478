"""Helpers for the GPU parity tests: build a workload's inputs on the host, run the cache-hit
path through the C ABI (via the Python binding), and compute the oracle's answer for the same
inputs.  Not collected by pytest (no test_ prefix)."""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

import paper_2607_28069_amd as pic
from oracle import pic_oracle as O
from synth import inputs as S
from synth.configs import Workload

DEV = "cuda"


def tdtype(w: Workload):
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def to_dev(x, dtype):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV).to(dtype)


def host(t) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def pool_compile_positions(lay: S.PoolLayout) -> np.ndarray:
    pos = np.zeros(lay.pool_tokens, np.int64)
    for e in range(len(lay.doc_len)):
        o, n = int(lay.doc_offset[e]), int(lay.doc_len[e])
        pos[o:o + n] = int(lay.doc_compile_pos[e]) + np.arange(n)
    return pos


@dataclass
class Run:
    w: Workload
    lay: S.PoolLayout
    inp: dict
    pool_k: np.ndarray            # [Hkv][T][D] compiled keys (rotated at compile positions)
    ctx: np.ndarray
    cap: int
    model: pic.Model = None
    dev: dict = field(default_factory=dict)
    maps: list = None
    fmaps: list = None            # general frontier layout: the oracle's per-request maps


def setup(w: Workload, requests=None, extra_cap: int = 0, mutate=None) -> Run:
    """Host inputs of layer 0; pool keys are raw keys rotated to their compile positions by the
    oracle's R (the format a cache compiler hands over).  `mutate(inp)` may plant structure."""
    lay = S.pool_layout(w)
    if requests is not None:
        lay.requests = requests
    inp = S.host_layer(w, lay, 0)
    if mutate is not None:
        mutate(inp, lay)
    pool_k = O.store(O.rope(inp["pool_k_raw"], pool_compile_positions(lay), w.rope_theta), w.dtype)
    maps = O.plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos)
    ctx = np.array([m.ctx_len for m in maps], np.int32)
    cap = int(ctx.max()) + w.n_suffix + max(w.decode_steps, 0) + extra_cap
    r = Run(w, lay, inp, pool_k, ctx, cap)
    r.maps = maps
    r.model = pic.Model.of(1, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype, w.rope_theta)
    return r


def gpu_compose(r: Run, max_abs_delta=None, blocks=None):
    w, dt = r.w, tdtype(r.w)
    if blocks is None:
        blocks, ctx = pic.pic_plan_layout(r.lay.requests, r.lay.doc_offset, r.lay.doc_len,
                                          r.lay.doc_compile_pos, r.lay.pool_tokens)
        assert np.array_equal(ctx, r.ctx)
    mad = int(max(r.cap, 1)) if max_abs_delta is None else max_abs_delta
    table = torch.empty(pic.pic_rope_table_bytes(r.model, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init(r.model, mad, table)
    d = r.dev
    d["table"], d["mad"] = table, mad
    d["pool_k"] = to_dev(r.pool_k[None], dt)
    d["pool_v"] = to_dev(r.inp["pool_v"][None], dt)
    d["blocks"] = torch.from_numpy(blocks.view(np.int32).reshape(-1).copy()).to(DEV)
    shape = (1, w.batch, w.n_kv_heads, r.cap, w.head_dim)
    d["cache_k"] = torch.zeros(shape, dtype=dt, device=DEV)
    d["cache_v"] = torch.zeros(shape, dtype=dt, device=DEV)
    pic.pic_compose(r.model, d["pool_k"], d["pool_v"], r.lay.pool_tokens, d["blocks"], len(blocks),
                    table, mad, d["cache_k"], d["cache_v"], w.batch, r.cap)
    d["ctx"] = torch.from_numpy(r.ctx).to(DEV)
    return d


def gpu_prefill(r: Run, scale: float = 0.0):
    w, dt, d = r.w, tdtype(r.w), r.dev
    d["q"] = to_dev(r.inp["q"][None], dt)
    d["k_suf"] = to_dev(r.inp["k_suf"][None], dt)
    d["v_suf"] = to_dev(r.inp["v_suf"][None], dt)
    d["out"] = torch.zeros((1, w.batch, w.n_suffix, w.n_q_heads, w.head_dim), dtype=dt, device=DEV)
    nbytes = pic.pic_prefill_workspace_bytes(r.model, w.batch, w.n_suffix, int(r.ctx.max()))
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    pic.pic_suffix_prefill_attn(r.model, d["q"], d["k_suf"], d["v_suf"], d["cache_k"], d["cache_v"],
                                w.batch, r.cap, d["ctx"], int(r.ctx.max()), w.n_suffix, d["out"], ws, scale=scale)
    return d["out"]


def gpu_decode(r: Run, steps: int, n_splits: int = 0, scale: float = 0.0):
    """Decode steps after the prefilled suffix; returns list of [B][Hq][D] outputs."""
    w, dt, d = r.w, tdtype(r.w), r.dev
    base = r.ctx + w.n_suffix
    d["base"] = torch.from_numpy(base.astype(np.int32)).to(DEV)
    max_base = int(base.max())
    nbytes = pic.pic_decode_workspace_bytes(r.model, w.batch, max_base + steps, n_splits)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    outs = []
    for t in range(steps):
        q = to_dev(r.inp["dq"][t][None], dt)
        k = to_dev(r.inp["dk"][t][None], dt)
        v = to_dev(r.inp["dv"][t][None], dt)
        out = torch.zeros((1, w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=DEV)
        pic.pic_decode_attn(r.model, q, k, v, d["cache_k"], d["cache_v"], w.batch, r.cap, d["base"], t,
                            max_base, out, ws, n_splits=n_splits, scale=scale)
        outs.append(out)
    return outs


def oracle_compose(r: Run, b: int):
    return O.compose_request(r.pool_k, r.inp["pool_v"], r.maps[b], r.w.rope_theta, r.w.dtype)


def oracle_prefill(r: Run, b: int, scale: float | None = None):
    K, V = oracle_compose(r, b)
    out, K2, V2 = O.suffix_prefill(K, V, r.inp["q"][b], r.inp["k_suf"][b], r.inp["v_suf"][b], scale)
    return out, K2, V2


# ------------------------------------------------------------------------------------------
# general frontier layout (inline prefix and spans between documents)
# ------------------------------------------------------------------------------------------

def setup_frontier(w: Workload, items=None, n_inline_cap=None, mutate=None) -> Run:
    """Like setup() for a frontier workload: lay.items mixes pool entries with inline spans
    (-n); the inline tokens' q/k/v are the workload's q/k_suf/v_suf rows, in position order."""
    lay = S.pool_layout(w)
    if items is not None:
        lay.items = items
    inp = S.host_layer(w, lay, 0)
    if n_inline_cap is not None:   # ragged layouts: more inline rows than the workload's
        for name, h in (("q", w.n_q_heads), ("k_suf", w.n_kv_heads), ("v_suf", w.n_kv_heads)):
            x = S.normal_f32(w, name + "_ragged", (w.batch, n_inline_cap, h, w.head_dim))
            inp[name] = S.bf16_bits_to_f32(S.f32_to_bf16_bits(x)) if w.dtype == "bf16" else x
    if mutate is not None:
        mutate(inp, lay)
    pool_k = O.store(O.rope(inp["pool_k_raw"], pool_compile_positions(lay), w.rope_theta), w.dtype)
    fmaps = O.plan_frontier(lay.items, lay.doc_offset, lay.doc_len, lay.doc_compile_pos)
    total = np.array([m.total_len for m in fmaps], np.int32)
    cap = int(total.max()) + max(w.decode_steps, 0) + 3
    r = Run(w, lay, inp, pool_k, total, cap)
    r.fmaps = fmaps
    r.model = pic.Model.of(1, w.n_q_heads, w.n_kv_heads, w.head_dim, w.dtype, w.rope_theta)
    return r


def gpu_frontier(r: Run, sentinel: float = 0.0, scale: float = 0.0):
    """Plan (C ABI), compose, frontier prefill; returns (out [1][B][n][Hq][D], n_inline)."""
    w, dt = r.w, tdtype(r.w)
    blocks, total, inl, n_inl = pic.pic_plan_frontier(r.lay.items, r.lay.doc_offset, r.lay.doc_len,
                                                      r.lay.doc_compile_pos, r.lay.pool_tokens)
    assert np.array_equal(total, r.ctx)
    d = gpu_compose(r, blocks=blocks)
    n = r.inp["q"].shape[1]
    assert inl.shape[1] <= n
    pos = np.full((w.batch, n), -1, np.int32)
    pos[:, : inl.shape[1]] = inl
    d["pos"] = torch.from_numpy(pos).to(DEV)
    d["n_valid"] = torch.from_numpy(n_inl.astype(np.int32)).to(DEV)
    d["q"] = to_dev(r.inp["q"][None], dt)
    d["k_inl"] = to_dev(r.inp["k_suf"][None], dt)
    d["v_inl"] = to_dev(r.inp["v_suf"][None], dt)
    d["out"] = torch.full((1, w.batch, n, w.n_q_heads, w.head_dim), sentinel, dtype=dt, device=DEV)
    max_len = int(total.max())
    nbytes = pic.pic_frontier_workspace_bytes(r.model, w.batch, n, max_len)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=DEV)
    pic.pic_frontier_prefill_attn(r.model, d["q"], d["k_inl"], d["v_inl"], d["cache_k"], d["cache_v"],
                                  w.batch, r.cap, d["pos"], d["n_valid"], n, max_len, d["out"], ws, scale=scale)
    return d["out"], n_inl


def oracle_frontier(r: Run, b: int, scale: float | None = None):
    """(out [n_b][Hq][D], K, V [Hkv][total][D]) of request b from the oracle."""
    f = r.fmaps[b]
    Kc, Vc = O.compose_request(r.pool_k, r.inp["pool_v"], f.cached, r.w.rope_theta, r.w.dtype)
    n = f.inline_pos.size
    return O.frontier_prefill(Kc, Vc, f, r.inp["q"][b][:n], r.inp["k_suf"][b][:n], r.inp["v_suf"][b][:n], scale)


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    ax = np.abs(x.astype(np.float64))
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    return np.where(ax > 0, 2.0 ** (e - 7), 2.0 ** -133)


def assert_attn_close(got: np.ndarray, ref: np.ndarray, dtype: str):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if dtype == "f32":
        err = np.abs(got - ref).max()
        assert err <= 1e-5, f"max abs err {err:.3e} > 1e-5"
    else:
        bad = np.abs(got - ref) > 2e-2 + 1e-2 * np.abs(ref)
        assert not bad.any(), f"{bad.sum()} elements beyond 2e-2 abs + 1e-2 rel; max abs err {np.abs(got - ref).max():.3e}"
        rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert rel <= 1e-2, f"relative Frobenius error {rel:.3e} > 1e-2"


def assert_keys_close(got: np.ndarray, ref: np.ndarray, dtype: str):
    if dtype == "f32":
        err = np.abs(got.astype(np.float64) - ref).max()
        assert err <= 1e-5, f"max abs err {err:.3e}"
        return 1.0
    # one bf16 ulp of the correctly rounded value, plus the float32 arithmetic bound 1e-5
    # (the latter only matters for results that nearly cancel, where an ulp is tiny)
    diff = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    bad = diff > bf16_ulp(ref) * 1.0000001 + 1e-5
    assert not bad.any(), f"{bad.sum()} keys beyond 1 bf16 ulp + 1e-5; worst excess {(diff - bf16_ulp(ref)).max():.3e}"
    return float((got.view(np.uint32) == ref.view(np.uint32)).mean())

"""Plain CPU oracle of the position-independent cache-hit path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module; only the tests, the smoke check and the benchmark's CPU-baseline leg do.
It shares no code with the GPU library: it is numpy only, written from the
paper's definitions, and deliberately slow and literal.

What it computes (SemPIC, "Learning Semantic Position-Independent KV Caches"):

* Request layout: the canonical order prefix, D_1, S_1, ..., D_m, S_m, Q
  (Sec. 2), with the link operator assigning each cached state its final
  logical position (Sec. 2) through a token-level map from physical cache
  slots to logical positions (App. C.1).  Here a physical slot index equals
  its logical position.  The plain layout has a stored prefix and empty S_i;
  the general (frontier) layout interleaves inline spans - tokens computed at
  request time, whose keys/values sit at their own logical slots and whose
  queries are prefilled - with the cached documents.
* RoPE relocation of a key compiled at position a to position b,
  k_b = R(b) R(a)^{-1} k_a (Sec. 2, Eq. 3); values are reused unchanged (Sec. 2).
* Causal attention of inline tokens over the linked cache with a frontier
  mask: a token never sees a logically later position, whatever the physical
  slot order (App. C.1); the completed cache then serves ordinary one-token
  decoding (App. C.1, Sec. 5 "Cache-hit serving").

Precision: inputs are float32 (bf16 inputs are exactly representable in it),
angles, cos/sin, rotations, dot products and softmax sums are float64, and a
stored result is rounded once to its storage type.

Readings where the paper is silent (each one is also pinned by a test):
  * rotate-half pairing of element i with element i + D/2 and inverse
    frequencies theta_i = base^(-2i/D), no frequency scaling, by default; the
    interleaved pairing (2i, 2i+1), explicit (e.g. Llama-3.1 frequency-scaled)
    frequencies and a different transform per layer ("layer-specific R_l",
    Sec. 2) are available as options;
  * one rotary transform shared by all layers unless given per layer;
  * softmax scale 1/sqrt(D); GQA query head h reads kv head h // (Hq/Hkv);
  * a token attends to every position <= its own (itself included).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# --------------------------------------------------------------------------------------
# Storage rounding
# --------------------------------------------------------------------------------------


def round_to_f32(x) -> np.ndarray:
    """Round to float32 (nearest, ties to even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def round_to_bf16(x) -> np.ndarray:
    """Round a float64 value to the nearest bfloat16 (ties to even), returned as float32.

    bfloat16 keeps 8 significant bits and float32's exponent range: split x into
    mantissa m in [0.5, 1) and exponent e, round m * 2^8 to an integer with
    ties to even (np.rint), and scale back.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8).astype(np.float32)


def store(x, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return round_to_f32(x)
    if dtype == "bf16":
        return round_to_bf16(x)
    raise ValueError(dtype)


# --------------------------------------------------------------------------------------
# Rotary transform R(p)  (Sec. 2, Eq. 3)
# --------------------------------------------------------------------------------------


def inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """theta_i = theta^(-2i/D) for i = 0 .. D/2-1, float64."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(theta), -2.0 * i / head_dim)


def llama3_inv_freq(head_dim: int, theta: float, factor: float = 8.0, low_freq_factor: float = 1.0,
                    high_freq_factor: float = 4.0, original_max_position: int = 8192) -> np.ndarray:
    """Frequency-scaled rotary frequencies of the Llama-3.1 family, float64.

    A frequency whose wavelength 2 pi / theta_i is shorter than original_max_position /
    high_freq_factor is kept; one whose wavelength exceeds original_max_position /
    low_freq_factor is divided by `factor`; in between the two are blended linearly in
    original_max_position / wavelength.
    """
    f = inv_freq(head_dim, theta)
    wavelen = 2.0 * np.pi / f
    smooth = (original_max_position / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    blended = (1.0 - smooth) * f / factor + smooth * f
    out = np.where(wavelen > original_max_position / low_freq_factor, f / factor, blended)
    return np.where(wavelen < original_max_position / high_freq_factor, f, out)


def _frequencies(head_dim: int, theta: float, freqs) -> np.ndarray:
    return inv_freq(head_dim, theta) if freqs is None else np.asarray(freqs, np.float64)


def _cos_sin(pos, head_dim: int, theta: float, freqs=None):
    ang = np.asarray(pos, dtype=np.float64)[:, None] * _frequencies(head_dim, theta, freqs)[None, :]
    return np.cos(ang), np.sin(ang)


def _split_pairs(x, pairing: str):
    """The two members of every rotated pair: (x_i, x_{i+D/2}) or (x_{2i}, x_{2i+1})."""
    if pairing == "half":
        h = x.shape[-1] // 2
        return x[..., :h], x[..., h:]
    if pairing == "interleaved":
        return x[..., 0::2], x[..., 1::2]
    raise ValueError(pairing)


def _join_pairs(a, b, pairing: str):
    if pairing == "half":
        return np.concatenate([a, b], axis=-1)
    return np.stack([a, b], axis=-1).reshape(a.shape[:-1] + (2 * a.shape[-1],))


def rope(x, pos, theta: float, pairing: str = "half", freqs=None) -> np.ndarray:
    """R(p) x for rows x[..., n, D] at positions pos[n]; float64 result.

    Pair i of a head (elements i and i + D/2 for "half", 2i and 2i + 1 for "interleaved")
    is turned by the angle p * theta_i: (x cos - y sin, x sin + y cos).  theta_i is
    theta^(-2i/D) unless `freqs` gives the D/2 frequencies explicitly.
    """
    x = np.asarray(x, dtype=np.float64)
    c, s = _cos_sin(pos, x.shape[-1], theta, freqs)
    x1, x2 = _split_pairs(x, pairing)
    return _join_pairs(x1 * c - x2 * s, x1 * s + x2 * c, pairing)


def rope_inverse(x, pos, theta: float, pairing: str = "half", freqs=None) -> np.ndarray:
    """R(p)^{-1} x = R(p)^T x (a rotation's inverse is its transpose); float64 result."""
    x = np.asarray(x, dtype=np.float64)
    c, s = _cos_sin(pos, x.shape[-1], theta, freqs)
    x1, x2 = _split_pairs(x, pairing)
    return _join_pairs(x1 * c + x2 * s, -x1 * s + x2 * c, pairing)


def rerotate_keys(k, a, b, theta: float, pairing: str = "half", freqs=None) -> np.ndarray:
    """Eq. 3 taken literally: k_b = R(b) (R(a)^{-1} k_a), two rotations in float64.

    k: [..., n, D]; a, b: [n] compile-time and request-time positions.
    """
    return rope(rope_inverse(k, a, theta, pairing, freqs), b, theta, pairing, freqs)


# --------------------------------------------------------------------------------------
# Layout: token-level map from cache slots to logical positions (Sec. 2; App. C.1)
# --------------------------------------------------------------------------------------


@dataclass
class RequestMap:
    ctx_len: int
    src_token: np.ndarray     # [ctx] pool token feeding each slot
    compile_pos: np.ndarray   # [ctx] position a the slot's key was compiled at
    logical_pos: np.ndarray   # [ctx] position b the slot holds in the request


def plan_layout(requests, doc_offset, doc_len, doc_compile_pos) -> list[RequestMap]:
    """Place each request's pool entries back to back in request order from position 0.

    Entry e of a request occupies logical positions [b_e, b_e + len_e) with
    b_e the running total of the entries before it; its token t was compiled at
    doc_compile_pos[e] + t.  Slot index = logical position.
    """
    maps = []
    for entries in requests:
        src, a, b = [], [], []
        pos = 0
        for e in entries:
            n = int(doc_len[e])
            for t in range(n):
                src.append(int(doc_offset[e]) + t)
                a.append(int(doc_compile_pos[e]) + t)
                b.append(pos + t)
            pos += n
        maps.append(RequestMap(pos, np.asarray(src, np.int64), np.asarray(a, np.int64),
                               np.asarray(b, np.int64)))
    return maps


@dataclass
class FrontierMap:
    total_len: int            # positions the request occupies (cached + inline)
    cached: RequestMap        # cached slots; cached.ctx_len = number of cached tokens
    inline_pos: np.ndarray    # [n_inline] positions of the inline tokens, increasing


def plan_frontier(items_per_request, doc_offset, doc_len, doc_compile_pos) -> list[FrontierMap]:
    """General canonical order P, D_1, S_1, ..., D_m, S_m, Q (Sec. 2) with inline spans.

    Each request is a list of items in logical order: a pool entry id (>= 0), whose
    tokens keep their compiled keys up to the relocation of Eq. 3, or -n for a span of n
    inline tokens (computed at request time).  Items occupy consecutive logical
    positions from 0; slot index = logical position (App. C.1).
    """
    maps = []
    for items in items_per_request:
        src, a, b, inl = [], [], [], []
        pos = 0
        for it in items:
            if it < 0:
                inl.extend(range(pos, pos - it))
                pos -= it
                continue
            n = int(doc_len[it])
            for t in range(n):
                src.append(int(doc_offset[it]) + t)
                a.append(int(doc_compile_pos[it]) + t)
                b.append(pos + t)
            pos += n
        cached = RequestMap(len(src), np.asarray(src, np.int64), np.asarray(a, np.int64),
                            np.asarray(b, np.int64))
        maps.append(FrontierMap(pos, cached, np.asarray(inl, np.int64)))
    return maps


# --------------------------------------------------------------------------------------
# Composition (link operator): re-rotated keys, unchanged values
# --------------------------------------------------------------------------------------


def compose_request(pool_k, pool_v, rmap: RequestMap, theta: float, dtype: str,
                    pairing: str = "half", freqs=None):
    """One request, one layer.  pool_k/pool_v: [Hkv][pool_tokens][D] (float32 values).

    Returns (K, V) of shape [Hkv][ctx][D], float32 values of the storage type.  `pairing`
    and `freqs` select the layer's rotary transform (see rope()).
    """
    k_src = np.asarray(pool_k, np.float64)[:, rmap.src_token, :]
    k = store(rerotate_keys(k_src, rmap.compile_pos, rmap.logical_pos, theta, pairing, freqs), dtype)
    v = np.asarray(pool_v, np.float32)[:, rmap.src_token, :].copy()
    return k, v


# --------------------------------------------------------------------------------------
# Attention with the frontier causal mask (App. C.1)
# --------------------------------------------------------------------------------------


def attention(q, q_pos, k, v, k_pos, scale: float | None = None) -> np.ndarray:
    """Masked softmax attention, float64.

    q: [Hq][nq][D] at positions q_pos[nq]; k, v: [Hkv][nk][D] at positions k_pos[nk].
    Query head h reads kv head h // (Hq // Hkv).  Key j is visible to query i
    iff k_pos[j] <= q_pos[i] (the mask is by position, not by slot).
    Returns o: [Hq][nq][D].
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    Hq, nq, D = q.shape
    Hkv = k.shape[0]
    n_rep = Hq // Hkv
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]          # [nq, nk]
    out = np.empty((Hq, nq, D), np.float64)
    for h in range(Hq):
        g = h // n_rep
        s = scale * (q[h] @ k[g].T)                                             # [nq, nk]
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        w = np.exp(s - m)
        out[h] = (w @ v[g]) / w.sum(axis=1, keepdims=True)
    return out


def suffix_prefill(k_ctx, v_ctx, q, k_suf, v_suf, scale: float | None = None):
    """Prefill of Ls suffix tokens after a composed context (one request, one layer).

    k_ctx, v_ctx: [Hkv][ctx][D] composed cache; q: [Ls][Hq][D]; k_suf, v_suf: [Ls][Hkv][D]
    (suffix keys already carry their own positions).  The suffix K/V are appended at
    positions [ctx, ctx + Ls) (App. C.1: inline KVs interleaved with the prepared
    states); suffix token i sits at position ctx + i.
    Returns (out [Ls][Hq][D] float64, K [Hkv][ctx+Ls][D], V [Hkv][ctx+Ls][D]).
    """
    ctx = k_ctx.shape[1]
    Ls = q.shape[0]
    K = np.concatenate([np.asarray(k_ctx, np.float32),
                        np.transpose(np.asarray(k_suf, np.float32), (1, 0, 2))], axis=1)
    V = np.concatenate([np.asarray(v_ctx, np.float32),
                        np.transpose(np.asarray(v_suf, np.float32), (1, 0, 2))], axis=1)
    pos = np.arange(ctx + Ls)
    o = attention(np.transpose(q, (1, 0, 2)), ctx + np.arange(Ls), K, V, pos, scale)
    return np.transpose(o, (1, 0, 2)), K, V


def frontier_prefill(k_cached, v_cached, fmap: FrontierMap, q, k_inl, v_inl,
                     scale: float | None = None):
    """Prefill of a request's inline tokens in the general layout (one layer).

    k_cached, v_cached: [Hkv][n_cached][D] composed cache rows in the order of
    fmap.cached (logical positions fmap.cached.logical_pos); q: [n_inline][Hq][D];
    k_inl, v_inl: [n_inline][Hkv][D] (inline keys already carry their positions).
    The inline K/V are placed at their own logical slots, interleaved with the
    cached states (App. C.1), and inline token i attends over every position
    <= fmap.inline_pos[i].
    Returns (out [n_inline][Hq][D] float64, K, V [Hkv][total_len][D] by position).
    """
    Hkv, _, D = np.shape(k_cached)
    T = fmap.total_len
    K = np.full((Hkv, T, D), np.nan, np.float32)
    V = np.full((Hkv, T, D), np.nan, np.float32)
    K[:, fmap.cached.logical_pos] = np.asarray(k_cached, np.float32)
    V[:, fmap.cached.logical_pos] = np.asarray(v_cached, np.float32)
    K[:, fmap.inline_pos] = np.transpose(np.asarray(k_inl, np.float32), (1, 0, 2))
    V[:, fmap.inline_pos] = np.transpose(np.asarray(v_inl, np.float32), (1, 0, 2))
    o = attention(np.transpose(q, (1, 0, 2)), fmap.inline_pos, K, V, np.arange(T), scale)
    return np.transpose(o, (1, 0, 2)), K, V


def decode_step(K, V, length: int, q, k_new, v_new, scale: float | None = None):
    """One decode step (one request, one layer): write k_new/v_new at position `length`,
    then attend the single query at that position over positions [0, length].

    K, V: [Hkv][>= length][D] valid up to `length`; q: [Hq][D]; k_new, v_new: [Hkv][D].
    Returns (out [Hq][D] float64, K', V' of length + 1).
    """
    K2 = np.concatenate([np.asarray(K, np.float32)[:, :length],
                         np.asarray(k_new, np.float32)[:, None, :]], axis=1)
    V2 = np.concatenate([np.asarray(V, np.float32)[:, :length],
                         np.asarray(v_new, np.float32)[:, None, :]], axis=1)
    o = attention(np.asarray(q)[:, None, :], np.asarray([length]), K2, V2,
                  np.arange(length + 1), scale)
    return o[:, 0, :], K2, V2

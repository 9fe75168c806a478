"""Seeded synthetic inputs for the cache-hit path.

Every tensor is i.i.d. N(0, 1), drawn in float32 from a counter-based stream
(numpy Philox on the host, torch's generator on a device) keyed by
(seed, workload, tensor name, layer), so any single layer can be regenerated
on its own.  bf16 tensors are the float32 draws rounded to nearest-even.

Document selection (which pool documents a request composes, and in what
order) and jittered document lengths are drawn here too; they are inputs to
the method, not part of it.  Nothing in this module rotates, composes or
attends: the method's arithmetic lives only in the oracle and in the GPU path.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

from .configs import Workload


def _key128(*parts) -> tuple[int, int]:
    h = hashlib.sha256("/".join(str(p) for p in parts).encode()).digest()
    return int.from_bytes(h[:8], "little"), int.from_bytes(h[8:16], "little")


def host_stream(w: Workload, tensor: str, layer: int = 0) -> np.random.Generator:
    """numpy Philox stream for one (workload, tensor, layer)."""
    k0, k1 = _key128(w.seed, w.name, tensor, layer)
    return np.random.Generator(np.random.Philox(key=[k0, k1]))


def device_seed(w: Workload, tensor: str, layer: int = 0) -> int:
    k0, _ = _key128(w.seed, w.name, tensor, layer, "device")
    return k0 & ((1 << 63) - 1)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------------------
# Pool and request composition
# --------------------------------------------------------------------------------------

@dataclass
class PoolLayout:
    doc_offset: np.ndarray        # int32 [n_entries]: first pool token of each entry
    doc_len: np.ndarray           # int32 [n_entries]
    doc_compile_pos: np.ndarray   # int32 [n_entries]: position the entry's first key was compiled at
    pool_tokens: int
    prefix_entry: int             # index of the instruction-prefix entry, or -1
    requests: list[list[int]]     # per request: pool entries in logical order
    items: list[list[int]] | None = None   # frontier layouts: entries (>= 0) and inline spans (-n)
    header_entry: int = -1        # boundary layouts: the shared header entry, else -1


def pool_layout(w: Workload) -> PoolLayout:
    """Pool = the workload's documents, then (if any) one shared instruction prefix, then
    (boundary layouts) one shared header.

    Documents are compiled independently starting at position 0 (boundary layouts: at
    position `header`, after the header, with their trailer tokens appended).  The prefix is
    stored already at its request-time position 0.  Each request lists the pool entries it
    composes, prefix first (boundary layouts: the header before every document).
    """
    if w.doc_len_jitter is not None:
        lo, hi = w.doc_len_jitter
        lens = host_stream(w, "doc_len").integers(lo, hi + 1, size=w.pool_docs)
    else:
        lens = np.full(w.pool_docs, w.doc_len, dtype=np.int64)
    header, trailer = w.boundary if w.boundary is not None else (0, 0)
    lens = list(int(x) + trailer for x in lens)
    cpos = [header] * len(lens)
    prefix_entry = header_entry = -1
    if w.prefix_len > 0:
        prefix_entry = len(lens)
        lens.append(w.prefix_len)
        cpos.append(0)
    if header > 0:
        header_entry = len(lens)
        lens.append(header)
        cpos.append(0)
    lens_a = np.asarray(lens, dtype=np.int32)
    offs = np.zeros_like(lens_a)
    offs[1:] = np.cumsum(lens_a[:-1])
    compile_pos = np.asarray(cpos, dtype=np.int32)

    g = host_stream(w, "doc_choice")
    requests = []
    for _ in range(w.batch):
        if w.fixed_order is not None:
            docs = list(w.fixed_order)
        elif w.all_docs_permuted:
            docs = [int(x) for x in g.permutation(w.pool_docs)]
        else:
            docs = [int(x) for x in g.choice(w.pool_docs, size=w.docs_per_request, replace=False)]
        if header_entry >= 0:
            docs = [e for d in docs for e in (header_entry, d)]
        requests.append(([prefix_entry] if prefix_entry >= 0 else []) + docs)
    items = None
    if w.frontier:
        items = []
        for entries in requests:
            it = [-w.inline_prefix] if w.inline_prefix > 0 else []
            for e in entries:
                it.append(e)
                if w.inline_span > 0 and e != prefix_entry and e != header_entry:
                    it.append(-w.inline_span)
            if w.n_suffix > 0:
                it.append(-w.n_suffix)
            items.append(it)
    return PoolLayout(offs, lens_a, compile_pos, int(lens_a.sum()), prefix_entry, requests, items,
                      header_entry)


def context_lengths(layout: PoolLayout) -> np.ndarray:
    """Tokens each request composes (prefix plus its documents)."""
    return np.asarray([int(layout.doc_len[r].sum()) for r in layout.requests], dtype=np.int32)


# --------------------------------------------------------------------------------------
# Host (numpy) tensors, float32
# --------------------------------------------------------------------------------------

def normal_f32(w: Workload, tensor: str, shape, layer: int = 0) -> np.ndarray:
    return host_stream(w, tensor, layer).standard_normal(size=shape, dtype=np.float32)


def host_layer(w: Workload, layout: PoolLayout, layer: int) -> dict[str, np.ndarray]:
    """All float32 inputs of one layer, drawn on the host.

    pool_k_raw: [Hkv][pool_tokens][D] keys before any rotation (the caller
                rotates them to their compile positions);
    pool_v:     [Hkv][pool_tokens][D];
    q, k_suf, v_suf: [B][Ls][H][D] suffix tokens (already at their positions);
    dq, dk, dv: [steps][B][H][D] decode-step tokens.
    Frontier workloads: q, k_suf, v_suf hold all n_inline inline tokens of a request in
    position order (prefix, each span, the query span), already at their positions.
    For bf16 workloads the values are already bf16-representable.
    """
    Hq, Hkv, D, B = w.n_q_heads, w.n_kv_heads, w.head_dim, w.batch
    Ls = w.n_inline if w.frontier else w.n_suffix
    out = {
        "pool_k_raw": normal_f32(w, "pool_k", (Hkv, layout.pool_tokens, D), layer),
        "pool_v": normal_f32(w, "pool_v", (Hkv, layout.pool_tokens, D), layer),
        "q": normal_f32(w, "q", (B, Ls, Hq, D), layer),
        "k_suf": normal_f32(w, "k_suf", (B, Ls, Hkv, D), layer),
        "v_suf": normal_f32(w, "v_suf", (B, Ls, Hkv, D), layer),
        "dq": normal_f32(w, "dq", (w.decode_steps, B, Hq, D), layer),
        "dk": normal_f32(w, "dk", (w.decode_steps, B, Hkv, D), layer),
        "dv": normal_f32(w, "dv", (w.decode_steps, B, Hkv, D), layer),
    }
    if w.dtype == "bf16":
        out = {k: bf16_bits_to_f32(f32_to_bf16_bits(v)) for k, v in out.items()}
    return out


# --------------------------------------------------------------------------------------
# Device (torch) tensors
# --------------------------------------------------------------------------------------

def device_normal(w: Workload, tensor: str, shape, layer: int, device, dtype):
    """N(0,1) drawn on `device` from a per-(tensor, layer) seeded generator, cast to dtype."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(device_seed(w, tensor, layer))
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return x.to(dtype)

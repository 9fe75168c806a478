"""The five synthetic workloads of the cache-hit path, and their derived sizes.

Shapes follow the model families the paper evaluates (Llama-3-8B and Qwen2.5-7B
shaped attention: GQA, head_dim 128, RoPE) and long-context retrieval settings in
the spirit of its tasks (Sec. 6.1: multi-document QA and needle retrieval).  The
paper's datasets are not used; every tensor is drawn N(0, 1) from a seed.

This module holds shapes and counts only; it performs none of the method's
arithmetic and is shared by the oracle-side tests and the GPU path.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                 # storage type of q/k/v and caches: "f32" or "bf16"
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    pool_docs: int             # documents in the shared pool
    doc_len: int               # nominal document length (tokens)
    docs_per_request: int
    prefix_len: int            # instruction prefix placed at logical position 0
    n_suffix: int              # suffix query tokens prefilled per request
    batch: int
    decode_steps: int = 0
    doc_len_jitter: tuple[int, int] | None = None   # inclusive range for jittered lengths
    fixed_order: tuple[int, ...] | None = None      # fixed document order (tiny case)
    all_docs_permuted: bool = False                 # each request is a permutation of the whole pool
    # General frontier layout (P, D_1, S_1, ..., D_m, S_m, Q with inline P and S_i): tokens of
    # an inline prefix and of the inline span after every document.  0/0 = the plain layout
    # (stored prefix entry, documents back to back, then the n_suffix query tokens).
    inline_prefix: int = 0
    inline_span: int = 0
    # Reader-side rotary variants: pairing ("half" = (i, i + D/2), "interleaved" = (2i, 2i+1)),
    # Llama-3.1 frequency scaling ("llama3": factor 8, low/high frequency factors 1/4, original
    # context 8192), and per-layer bases (local, global, period): layer l uses the global base
    # when l % period == period - 1, else the local one.
    rope_pairing: str = "half"
    rope_scaling: str | None = None
    local_global: tuple[float, float, int] | None = None
    # Learned block boundaries (KV Packet / Joint): (header, trailer) tokens.  One shared
    # header entry, compiled at positions 0 .. header-1, precedes every document in a request;
    # each document entry carries its own trailer and was compiled after the header (its first
    # token at position `header`).
    boundary: tuple[int, int] | None = None
    seed: int = 0
    notes: str = ""

    @property
    def n_rep(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def per_layer_rope(self) -> bool:
        return self.local_global is not None

    def layer_theta(self, layer: int) -> float:
        if self.local_global is None:
            return self.rope_theta
        local, glob, period = self.local_global
        return glob if layer % period == period - 1 else local

    @property
    def frontier(self) -> bool:
        return self.inline_prefix > 0 or self.inline_span > 0

    @property
    def n_inline(self) -> int:
        """Inline tokens per request (prefilled as queries): P, every S_i and Q."""
        return self.inline_prefix + self.docs_per_request * self.inline_span + self.n_suffix


WORKLOADS: dict[str, Workload] = {
    "tiny_f32": Workload(
        name="tiny_f32", dtype="f32", n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64,
        rope_theta=1e4, pool_docs=2, doc_len=128, docs_per_request=2, prefix_len=16,
        n_suffix=16, batch=1, fixed_order=(0, 1),
        notes="2 docs x 128 tokens at request offsets 16 and 144 behind a 16-token prefix"),
    "llama8b_1layer": Workload(
        name="llama8b_1layer", dtype="bf16", n_layers=1, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=16, doc_len=512, docs_per_request=8,
        prefix_len=64, n_suffix=64, batch=4,
        notes="pool 16 x 512; 8 docs per request in a random order; 64-token prefix"),
    "llama8b_32layer": Workload(
        name="llama8b_32layer", dtype="bf16", n_layers=32, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=64, doc_len=1024, docs_per_request=10,
        prefix_len=128, n_suffix=128, batch=16,
        notes="pool 64 x 1024; 10 distinct docs per request (~10K context); 128-token prefix"),
    "llama8b_decode": Workload(
        name="llama8b_decode", dtype="bf16", n_layers=32, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=256, doc_len=1024, docs_per_request=16,
        prefix_len=0, n_suffix=0, batch=64, decode_steps=256,
        notes="64 requests x 16K composed context from a 256-doc pool; 256 decode steps"),
    "qwen7b_32k": Workload(
        name="qwen7b_32k", dtype="bf16", n_layers=28, n_q_heads=28, n_kv_heads=4,
        head_dim=128, rope_theta=1e6, pool_docs=32, doc_len=1024, docs_per_request=32,
        prefix_len=0, n_suffix=256, batch=8, doc_len_jitter=(768, 1280),
        all_docs_permuted=True,
        notes="32 docs with lengths ~U{768..1280}, each request a permutation of all 32 (~32K)"),
    # General frontier layout: the prefix and a span after every document are inline tokens
    # whose queries are prefilled together with the final query span.
    "tiny_frontier_f32": Workload(
        name="tiny_frontier_f32", dtype="f32", n_layers=1, n_q_heads=4, n_kv_heads=2,
        head_dim=64, rope_theta=1e4, pool_docs=3, doc_len=96, docs_per_request=3, prefix_len=0,
        n_suffix=16, batch=2, inline_prefix=16, inline_span=8,
        notes="inline prefix 16, 3 docs x 96 each followed by an 8-token inline span, 16 query tokens"),
    "llama8b_frontier_1layer": Workload(
        name="llama8b_frontier_1layer", dtype="bf16", n_layers=1, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=16, doc_len=512, docs_per_request=8,
        prefix_len=0, n_suffix=64, batch=4, inline_prefix=48, inline_span=24,
        notes="inline prefix 48, 8 docs x 512 each followed by a 24-token inline span, 64 query tokens"),
    "llama8b_frontier": Workload(
        name="llama8b_frontier", dtype="bf16", n_layers=32, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=64, doc_len=1024, docs_per_request=10,
        prefix_len=0, n_suffix=128, batch=16, inline_prefix=128, inline_span=32,
        notes="the 32-layer Llama shape with an inline 128-token prefix and a 32-token inline span "
              "after each of the 10 documents (576 inline tokens per request)"),
    # Reader-side rotary variants on the 32-layer Llama shape.
    "llama31_32layer": Workload(
        name="llama31_32layer", dtype="bf16", n_layers=32, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=64, doc_len=1024, docs_per_request=10,
        prefix_len=128, n_suffix=128, batch=16, rope_scaling="llama3",
        notes="the 32-layer Llama shape with Llama-3.1 frequency-scaled RoPE"),
    "interleaved_localglobal_32layer": Workload(
        name="interleaved_localglobal_32layer", dtype="bf16", n_layers=32, n_q_heads=32,
        n_kv_heads=8, head_dim=128, rope_theta=1e4, pool_docs=64, doc_len=1024,
        docs_per_request=10, prefix_len=128, n_suffix=128, batch=16, rope_pairing="interleaved",
        local_global=(1e4, 1e6, 6),
        notes="the 32-layer Llama shape with interleaved pairing and per-layer bases "
              "(1e4 local, 1e6 on every 6th layer)"),
    # Learned block boundaries around every document (KV Packet / Joint serving layout).
    "llama8b_joint_1layer": Workload(
        name="llama8b_joint_1layer", dtype="bf16", n_layers=1, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=16, doc_len=512, docs_per_request=8,
        prefix_len=64, n_suffix=64, batch=4, boundary=(8, 8),
        notes="the 1-layer Llama shape with an 8-token shared header before and an 8-token trailer "
              "after every document"),
    "llama8b_joint": Workload(
        name="llama8b_joint", dtype="bf16", n_layers=32, n_q_heads=32, n_kv_heads=8,
        head_dim=128, rope_theta=5e5, pool_docs=64, doc_len=1024, docs_per_request=10,
        prefix_len=128, n_suffix=128, batch=16, boundary=(8, 8),
        notes="the 32-layer Llama shape with an 8-token shared header before and an 8-token trailer "
              "after every document (10 528-token contexts)"),
}

# Short aliases in the order the workloads are listed above.
ALIASES = {"c1": "tiny_f32", "c2": "llama8b_1layer", "c3": "llama8b_32layer",
           "c4": "llama8b_decode", "c5": "qwen7b_32k"}


def get(name: str) -> Workload:
    return WORKLOADS[ALIASES.get(name, name)]

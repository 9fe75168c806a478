"""Python binding of libpic, the MI355X (gfx950) cache-hit path of position-independent KV
caching: key re-rotation, document composition, suffix prefill and decode attention.

Argument marshalling only: every step runs in the library's HIP kernels.  Tensors are
torch device tensors (their data pointers are passed); host arrays are numpy int32 arrays.
Calls enqueue on torch's current stream unless `stream` is given.  A missing library is an
error, never a fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpic.so")

PIC_F32, PIC_BF16 = 0, 1
PIC_BLOCK_TOKENS = 64
STATUS = {0: "PIC_OK", -1: "PIC_ERR_INVALID_ARG", -2: "PIC_ERR_UNSUPPORTED", -3: "PIC_ERR_WORKSPACE",
          -4: "PIC_ERR_CAPACITY", -5: "PIC_ERR_MISALIGNED", -6: "PIC_ERR_RANGE", -7: "PIC_ERR_HIP"}

# Every symbol include/pic.h declares.
EXPORTS = ("pic_plan_layout", "pic_plan_frontier", "pic_rope_table_bytes", "pic_rope_table_init",
           "pic_rope_table_init_freq", "pic_rope_llama3_freq",
           "pic_rerotate_keys", "pic_compose", "pic_plan_shared", "pic_compose_shared",
           "pic_prefill_workspace_bytes",
           "pic_suffix_prefill_attn", "pic_suffix_prefill_attn_rope", "pic_build_slot_map",
           "pic_compose_tiles", "pic_paged_prefill_attn",
           "pic_frontier_workspace_bytes", "pic_frontier_prefill_attn",
           "pic_decode_workspace_bytes", "pic_decode_attn", "pic_decode_attn_rope", "pic_status_string",
           "pic_last_error",
           "pic_decode_auto_splits", "pic_decode_attn_noalloc")
PIC_DECODE_SCRATCH_BYTES = 8 << 20


class PicError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


PIC_ROPE_HALF, PIC_ROPE_INTERLEAVED = 0, 1


class Model(ctypes.Structure):
    """pic_model: attention shape and rotary transform of the served decoder."""
    _fields_ = [("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int), ("rope_theta", ctypes.c_double),
                ("rope_pairing", ctypes.c_int32), ("rope_tables", ctypes.c_int32)]

    @classmethod
    def of(cls, n_layers, n_q_heads, n_kv_heads, head_dim, dtype, rope_theta, pairing="half",
           per_layer_tables=False):
        dt = {"f32": PIC_F32, "bf16": PIC_BF16}.get(dtype, dtype)
        pr = {"half": PIC_ROPE_HALF, "interleaved": PIC_ROPE_INTERLEAVED}.get(pairing, pairing)
        return cls(n_layers, n_q_heads, n_kv_heads, head_dim, dt, float(rope_theta), pr,
                   n_layers if per_layer_tables else 1)

    def with_layers(self, n):
        """The same decoder restricted to n layers (per-layer tables: the first n blocks)."""
        return Model(n, self.n_q_heads, self.n_kv_heads, self.head_dim, self.dtype, self.rope_theta,
                     self.rope_pairing, n if self.rope_tables > 1 else self.rope_tables)


BLOCK_DTYPE = np.dtype([("request", np.int32), ("src_token", np.int32), ("dst_slot", np.int32),
                        ("n_tokens", np.int32), ("delta", np.int32)])

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libpic.so (built by paper_2607_28069_amd.build); raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2607_28069_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
    MP = ctypes.POINTER(Model)
    sig = {
        "pic_plan_layout": (ctypes.c_int, [I32, P, P, I32, P, P, P, I64, P, I32, P, P]),
        "pic_plan_frontier": (ctypes.c_int, [I32, P, P, I32, P, P, P, I64, P, I32, P, P, P, I32, P]),
        "pic_rope_table_bytes": (SZ, [MP, I32]),
        "pic_rope_table_init": (ctypes.c_int, [MP, I32, P, SZ, P]),
        "pic_rope_table_init_freq": (ctypes.c_int, [MP, P, I32, P, SZ, P]),
        "pic_rope_llama3_freq": (ctypes.c_int, [I32, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                                ctypes.c_double, ctypes.c_double, P]),
        "pic_rerotate_keys": (ctypes.c_int, [MP, P, P, I64, I32, P, P, I32, P]),
        "pic_compose": (ctypes.c_int, [MP, P, P, I64, P, I32, P, I32, P, P, I32, I32, P]),
        "pic_plan_shared": (ctypes.c_int, [P, I32, P, P, P]),
        "pic_compose_shared": (ctypes.c_int, [MP, P, P, I64, P, I32, P, I32, P, I32, P, P, I32, I32, P]),
        "pic_prefill_workspace_bytes": (SZ, [MP, I32, I32, I32]),
        "pic_suffix_prefill_attn": (ctypes.c_int, [MP, P, P, P, P, P, I32, I32, P, I32, I32, F, P, P, SZ, P]),
        "pic_suffix_prefill_attn_rope": (ctypes.c_int, [MP, P, P, P, P, P, I32, I32, P, I32, I32, P, I32, F, P, P,
                                                        SZ, P]),
        "pic_build_slot_map": (ctypes.c_int, [P, I32, I32, I32, P, P, P, P]),
        "pic_compose_tiles": (ctypes.c_int, [MP, P, P, I64, P, P, I32, P, P, I32, P, I32, P, P, I32, I32, P]),
        "pic_paged_prefill_attn": (ctypes.c_int, [MP, P, P, I64, P, P, I32, P, P, I32, P, P, P, P, P, I32, I32,
                                                  P, I32, I32, F, P, P, SZ, P]),
        "pic_frontier_workspace_bytes": (SZ, [MP, I32, I32, I32]),
        "pic_frontier_prefill_attn": (ctypes.c_int, [MP, P, P, P, P, P, I32, I32, P, P, I32, I32, F, P, P, SZ, P]),
        "pic_decode_workspace_bytes": (SZ, [MP, I32, I32, I32]),
        "pic_decode_attn": (ctypes.c_int, [MP, P, P, P, P, P, I32, I32, P, I32, I32, F, I32, P, P, SZ, P]),
        "pic_decode_attn_rope": (ctypes.c_int, [MP, P, P, P, P, P, I32, I32, P, I32, I32, P, I32, F, I32, P, P, SZ,
                                                P]),
        "pic_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "pic_last_error": (ctypes.c_char_p, []),
        "pic_decode_auto_splits": (I32, [MP, I32, I32]),
        "pic_decode_attn_noalloc": (ctypes.c_int, [MP, P, P, P, P, P, I32, I32, P, I32, I32, F, I32, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        raise PicError(status, load().pic_last_error().decode())


def _ptr(t):
    """Device address of a tensor argument (None -> NULL).  The library reads every buffer as a
    dense array in GPU memory, so host tensors and strided views are refused here."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("device buffer expected: got a host tensor")
    if not t.is_contiguous():
        raise ValueError("device buffer must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _host_i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.c_void_p)


# ------------------------------------------------------------------------------------------
# the C calls, same names
# ------------------------------------------------------------------------------------------

def pic_plan_layout(requests, entry_offset, entry_len, entry_compile_pos, pool_tokens):
    """requests: list of lists of pool entry ids.  Returns (blocks structured array, ctx_len)."""
    lib = load()
    n_entries, p_n = _host_i32([len(r) for r in requests])
    flat, p_flat = _host_i32([e for r in requests for e in r] or [0])
    off, p_off = _host_i32(entry_offset)
    ln, p_len = _host_i32(entry_len)
    cp, p_cp = _host_i32(entry_compile_pos)
    n_blocks = ctypes.c_int32(0)
    ctx = np.zeros(len(requests), np.int32)
    st = lib.pic_plan_layout(len(requests), p_n, p_flat, len(off), p_off, p_len, p_cp, int(pool_tokens),
                             None, 0, ctypes.byref(n_blocks), ctx.ctypes.data_as(ctypes.c_void_p))
    if st not in (0, -4):
        _check(st)
    blocks = np.zeros(max(n_blocks.value, 1), BLOCK_DTYPE)
    _check(lib.pic_plan_layout(len(requests), p_n, p_flat, len(off), p_off, p_len, p_cp,
                               int(pool_tokens), blocks.ctypes.data_as(ctypes.c_void_p),
                               len(blocks), ctypes.byref(n_blocks), ctx.ctypes.data_as(ctypes.c_void_p)))
    return blocks[: n_blocks.value], ctx


def pic_plan_shared(blocks):
    """Gather blocks -> (blocks grouped by source run, group_start [n_groups + 1])."""
    blocks = np.ascontiguousarray(blocks, BLOCK_DTYPE)
    n = len(blocks)
    out = np.zeros(max(n, 1), BLOCK_DTYPE)
    starts = np.zeros(n + 1, np.int32)
    n_groups = ctypes.c_int32(0)
    _check(load().pic_plan_shared(blocks.ctypes.data_as(ctypes.c_void_p) if n else None, n,
                                  out.ctypes.data_as(ctypes.c_void_p), starts.ctypes.data_as(ctypes.c_void_p),
                                  ctypes.byref(n_groups)))
    return out[:n], starts[: n_groups.value + 1]


def pic_plan_frontier(items, entry_offset, entry_len, entry_compile_pos, pool_tokens):
    """items: per request, a list of pool entry ids (>= 0) and inline spans (-n).

    Returns (blocks structured array, total_len [B], inline_pos [B][max inline] with -1
    padding, n_inline [B])."""
    lib = load()
    n_items, p_n = _host_i32([len(r) for r in items])
    flat, p_flat = _host_i32([e for r in items for e in r] or [0])
    off, p_off = _host_i32(entry_offset)
    ln, p_len = _host_i32(entry_len)
    cp, p_cp = _host_i32(entry_compile_pos)
    cap = max([sum(-e for e in r if e < 0) for r in items] + [1])
    n_blocks = ctypes.c_int32(0)
    total = np.zeros(len(items), np.int32)
    inl = np.zeros((len(items), cap), np.int32)
    n_inl = np.zeros(len(items), np.int32)
    args = lambda blocks, n: (len(items), p_n, p_flat, len(off), p_off, p_len, p_cp, int(pool_tokens),
                              blocks, n, ctypes.byref(n_blocks), total.ctypes.data_as(ctypes.c_void_p),
                              inl.ctypes.data_as(ctypes.c_void_p), cap,
                              n_inl.ctypes.data_as(ctypes.c_void_p))
    st = lib.pic_plan_frontier(*args(None, 0))
    if st not in (0, -4):
        _check(st)
    blocks = np.zeros(max(n_blocks.value, 1), BLOCK_DTYPE)
    _check(lib.pic_plan_frontier(*args(blocks.ctypes.data_as(ctypes.c_void_p), len(blocks))))
    return blocks[: n_blocks.value], total, inl, n_inl


def pic_rope_table_bytes(model: Model, max_abs_delta: int) -> int:
    return load().pic_rope_table_bytes(ctypes.byref(model), max_abs_delta)


def pic_rope_table_init(model: Model, max_abs_delta: int, table, stream=None):
    _check(load().pic_rope_table_init(ctypes.byref(model), max_abs_delta, _ptr(table),
                                      table.numel() * table.element_size(), _stream(stream)))


def pic_rope_table_init_freq(model: Model, inv_freq, max_abs_delta: int, table, stream=None):
    """inv_freq: host array [n_tables][D/2] (or [D/2] for one table) of rotary frequencies."""
    f = np.ascontiguousarray(inv_freq, dtype=np.float64)
    _check(load().pic_rope_table_init_freq(ctypes.byref(model), f.ctypes.data_as(ctypes.c_void_p),
                                           max_abs_delta, _ptr(table),
                                           table.numel() * table.element_size(), _stream(stream)))


def pic_rope_llama3_freq(head_dim, theta, factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0,
                         original_max_position=8192) -> np.ndarray:
    out = np.zeros(head_dim // 2, np.float64)
    _check(load().pic_rope_llama3_freq(int(head_dim), float(theta), float(factor), float(low_freq_factor),
                                       float(high_freq_factor), float(original_max_position),
                                       out.ctypes.data_as(ctypes.c_void_p)))
    return out


def pic_rerotate_keys(model: Model, k_in, k_out, n_tokens, n_heads, delta, table, max_abs_delta,
                      stream=None):
    _check(load().pic_rerotate_keys(ctypes.byref(model), _ptr(k_in), _ptr(k_out), int(n_tokens),
                                    int(n_heads), _ptr(delta), _ptr(table), max_abs_delta,
                                    _stream(stream)))


def pic_compose_shared(model: Model, pool_k, pool_v, pool_tokens, blocks, n_blocks, group_start, n_groups,
                       table, max_abs_delta, cache_k, cache_v, batch, cache_cap, stream=None):
    _check(load().pic_compose_shared(ctypes.byref(model), _ptr(pool_k), _ptr(pool_v), int(pool_tokens),
                                     _ptr(blocks), int(n_blocks), _ptr(group_start), int(n_groups),
                                     _ptr(table), max_abs_delta, _ptr(cache_k), _ptr(cache_v), int(batch),
                                     int(cache_cap), _stream(stream)))


def pic_compose(model: Model, pool_k, pool_v, pool_tokens, blocks, n_blocks, table, max_abs_delta,
                cache_k, cache_v, batch, cache_cap, stream=None):
    _check(load().pic_compose(ctypes.byref(model), _ptr(pool_k), _ptr(pool_v), int(pool_tokens),
                              _ptr(blocks), int(n_blocks), _ptr(table), max_abs_delta, _ptr(cache_k),
                              _ptr(cache_v), int(batch), int(cache_cap), _stream(stream)))


def pic_prefill_workspace_bytes(model: Model, batch, n_suffix, max_ctx) -> int:
    return load().pic_prefill_workspace_bytes(ctypes.byref(model), batch, n_suffix, max_ctx)


def pic_suffix_prefill_attn(model: Model, q, k_suf, v_suf, cache_k, cache_v, batch, cache_cap, ctx_len,
                            max_ctx, n_suffix, out, workspace=None, scale=0.0, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().pic_suffix_prefill_attn(ctypes.byref(model), _ptr(q), _ptr(k_suf), _ptr(v_suf),
                                          _ptr(cache_k), _ptr(cache_v), int(batch), int(cache_cap),
                                          _ptr(ctx_len), int(max_ctx), int(n_suffix), float(scale),
                                          _ptr(out), _ptr(workspace), ws_bytes, _stream(stream)))


def pic_suffix_prefill_attn_rope(model: Model, q, k_suf, v_suf, cache_k, cache_v, batch, cache_cap, ctx_len,
                                 max_ctx, n_suffix, table, max_abs_delta, out, workspace=None, scale=0.0,
                                 stream=None):
    """q / k_suf unrotated: turned to positions ctx_len[b] + i inside the kernel."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().pic_suffix_prefill_attn_rope(ctypes.byref(model), _ptr(q), _ptr(k_suf), _ptr(v_suf),
                                               _ptr(cache_k), _ptr(cache_v), int(batch), int(cache_cap),
                                               _ptr(ctx_len), int(max_ctx), int(n_suffix), _ptr(table),
                                               int(max_abs_delta), float(scale), _ptr(out), _ptr(workspace),
                                               ws_bytes, _stream(stream)))


def pic_slot_map_tiles(map_cap) -> int:
    """64-slot tiles per request in a tile map of `map_cap` slots."""
    return (int(map_cap) + PIC_BLOCK_TOKENS - 1) // PIC_BLOCK_TOKENS


def pic_build_slot_map(blocks, n_blocks, batch, map_cap, slot_src, slot_delta, tile_map=None, stream=None):
    """tile_map: None, or int32 [batch][pic_slot_map_tiles(map_cap)][2]."""
    _check(load().pic_build_slot_map(_ptr(blocks), int(n_blocks), int(batch), int(map_cap), _ptr(slot_src),
                                     _ptr(slot_delta), _ptr(tile_map), _stream(stream)))


def pic_compose_tiles(model: Model, pool_k, pool_v, pool_tokens, slot_src, slot_delta, map_cap, tile_map, table,
                      max_abs_delta, ctx_len, max_ctx, cache_k, cache_v, batch, cache_cap, stream=None):
    """The context tiles the tile map does not mark as whole runs, composed into the caches for
    every layer of `model` in one launch (then pic_paged_prefill_attn may take slot_src =
    slot_delta = None with the tile map)."""
    _check(load().pic_compose_tiles(ctypes.byref(model), _ptr(pool_k), _ptr(pool_v), int(pool_tokens),
                                    _ptr(slot_src), _ptr(slot_delta), int(map_cap), _ptr(tile_map), _ptr(table),
                                    int(max_abs_delta), _ptr(ctx_len), int(max_ctx), _ptr(cache_k), _ptr(cache_v),
                                    int(batch), int(cache_cap), _stream(stream)))


def pic_paged_prefill_attn(model: Model, pool_k, pool_v, pool_tokens, slot_src, slot_delta, map_cap, table,
                           max_abs_delta, q, k_suf, v_suf, cache_k, cache_v, batch, cache_cap, ctx_len, max_ctx,
                           n_suffix, out, workspace=None, scale=0.0, stream=None, tile_map=None):
    """tile_map None: keys turned one by one (bit-identical to compose + prefill); a tile map from
    pic_build_slot_map: whole-run tiles turn the queries instead (slot_src = slot_delta = None:
    the other tiles were composed beforehand by pic_compose_tiles)."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().pic_paged_prefill_attn(ctypes.byref(model), _ptr(pool_k), _ptr(pool_v), int(pool_tokens),
                                         _ptr(slot_src), _ptr(slot_delta), int(map_cap), _ptr(tile_map),
                                         _ptr(table),
                                         int(max_abs_delta), _ptr(q), _ptr(k_suf), _ptr(v_suf), _ptr(cache_k),
                                         _ptr(cache_v), int(batch), int(cache_cap), _ptr(ctx_len), int(max_ctx),
                                         int(n_suffix), float(scale), _ptr(out), _ptr(workspace), ws_bytes,
                                         _stream(stream)))


def pic_frontier_workspace_bytes(model: Model, batch, n_inline, max_len) -> int:
    return load().pic_frontier_workspace_bytes(ctypes.byref(model), batch, n_inline, max_len)


def pic_frontier_prefill_attn(model: Model, q, k_inl, v_inl, cache_k, cache_v, batch, cache_cap, pos,
                              n_valid, n_inline, max_len, out, workspace=None, scale=0.0, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().pic_frontier_prefill_attn(ctypes.byref(model), _ptr(q), _ptr(k_inl), _ptr(v_inl),
                                            _ptr(cache_k), _ptr(cache_v), int(batch), int(cache_cap),
                                            _ptr(pos), _ptr(n_valid), int(n_inline), int(max_len),
                                            float(scale), _ptr(out), _ptr(workspace), ws_bytes,
                                            _stream(stream)))


def pic_decode_workspace_bytes(model: Model, batch, max_len, n_splits=0) -> int:
    return load().pic_decode_workspace_bytes(ctypes.byref(model), batch, max_len, n_splits)


def pic_decode_auto_splits(model: Model, batch, max_len) -> int:
    return load().pic_decode_auto_splits(ctypes.byref(model), batch, max_len)


def pic_decode_attn(model: Model, q, k_new, v_new, cache_k, cache_v, batch, cache_cap, base_len, step,
                    max_base_len, out, workspace=None, n_splits=0, scale=0.0, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().pic_decode_attn(ctypes.byref(model), _ptr(q), _ptr(k_new), _ptr(v_new),
                                  _ptr(cache_k), _ptr(cache_v), int(batch), int(cache_cap),
                                  _ptr(base_len), int(step), int(max_base_len), float(scale),
                                  int(n_splits), _ptr(out), _ptr(workspace), ws_bytes,
                                  _stream(stream)))


def pic_decode_attn_rope(model: Model, q, k_new, v_new, cache_k, cache_v, batch, cache_cap, base_len, step,
                         max_base_len, table, max_abs_delta, out, workspace=None, n_splits=0, scale=0.0,
                         stream=None):
    """q / k_new unrotated: turned to position base_len[b] + step inside the kernel."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().pic_decode_attn_rope(ctypes.byref(model), _ptr(q), _ptr(k_new), _ptr(v_new),
                                       _ptr(cache_k), _ptr(cache_v), int(batch), int(cache_cap),
                                       _ptr(base_len), int(step), int(max_base_len), _ptr(table),
                                       int(max_abs_delta), float(scale), int(n_splits), _ptr(out),
                                       _ptr(workspace), ws_bytes, _stream(stream)))


def pic_decode_attn_noalloc(model: Model, q, k_new, v_new, cache_k, cache_v, batch, cache_cap, base_len, step,
                            max_base_len, out, n_splits=0, scale=0.0, stream=None):
    """pic_decode_attn with its split partials in the library's per-GPU scratch array (no workspace)."""
    _check(load().pic_decode_attn_noalloc(ctypes.byref(model), _ptr(q), _ptr(k_new), _ptr(v_new),
                                          _ptr(cache_k), _ptr(cache_v), int(batch), int(cache_cap),
                                          _ptr(base_len), int(step), int(max_base_len), float(scale),
                                          int(n_splits), _ptr(out), _stream(stream)))


def pic_status_string(status: int) -> str:
    return load().pic_status_string(status).decode()


def pic_last_error() -> str:
    return load().pic_last_error().decode()

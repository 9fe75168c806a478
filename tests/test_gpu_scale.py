"""A softmax scale other than the default 1/sqrt(head_dim), through every attention entry point
that takes one, against the oracle with the same scale: the matrix-core suffix prefill (split
over key ranges, and unsplit), the zero-copy prefill (per key and with the tile map), the frontier
prefill, split and unsplit decode, and the row path (float32 at head_dim 64, bf16 at head_dim
64).  A scale of 0.05 sits well away from the default (0.088 at head_dim 128, 0.125 at 64), so a
call that ignored it would fail the attention tolerance."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import pic_oracle as O

from gpu_path import (DEV, assert_attn_close, gpu_compose, gpu_decode, gpu_frontier, gpu_prefill, host,
                      oracle_frontier, oracle_prefill, setup, setup_frontier)
from test_gpu_paged import _paged

pytestmark = pytest.mark.gpu
SCALE = 0.05


def _workload(name):
    if name == "bf16_hd64":
        return dataclasses.replace(synth.get("c2"), name="scale_hd64", head_dim=64, n_q_heads=16, n_kv_heads=4,
                                   pool_docs=6, doc_len=300, docs_per_request=4, prefix_len=13, n_suffix=45,
                                   batch=3, decode_steps=2)
    if name == "c2_unsplit":   # enough (m-tile, kv head) units that the launch is not split
        return dataclasses.replace(synth.get("c2"), name="scale_unsplit", n_suffix=256, batch=8, decode_steps=2)
    return dataclasses.replace(synth.get(name), decode_steps=2)


@pytest.mark.parametrize("name", ["c1", "c2", "c2_unsplit", "bf16_hd64"])
def test_custom_scale_prefill_and_decode(name):
    w = _workload(name)
    r = setup(w)
    gpu_compose(r)
    out = host(gpu_prefill(r, scale=SCALE))[0]
    outs = [host(o)[0] for o in gpu_decode(r, 2, scale=SCALE)]
    for b in range(w.batch):
        ref, K, V = oracle_prefill(r, b, scale=SCALE)
        assert_attn_close(out[b], ref, w.dtype)
        length = int(r.ctx[b]) + w.n_suffix
        for t in range(2):
            ref, K, V = O.decode_step(K, V, length, r.inp["dq"][t][b], r.inp["dk"][t][b], r.inp["dv"][t][b],
                                      scale=SCALE)
            length += 1
            assert_attn_close(outs[t][b], ref, w.dtype)
    print(f"[scale] {name}: prefill and 2 decode steps ok", flush=True)


@pytest.mark.parametrize("runs", [False, True], ids=["per-key", "tile-map"])
def test_custom_scale_zero_copy_prefill(runs):
    w = synth.get("c2")
    r = setup(w)
    gpu_compose(r)
    out_m = gpu_prefill(r, scale=SCALE).clone()   # compose + prefill with the same scale
    out, _, _ = _paged(r, runs=runs, scale=SCALE)
    torch.cuda.synchronize()
    if not runs:   # keys turned on load: bit-identical to compose + prefill
        assert torch.equal(out, out_m)
    got = host(out)[0]
    for b in range(w.batch):
        ref, _, _ = oracle_prefill(r, b, scale=SCALE)
        assert_attn_close(got[b], ref, "bf16")


def test_custom_scale_frontier_prefill():
    w = synth.get("llama8b_frontier_1layer")
    r = setup_frontier(w)
    out, n_inl = gpu_frontier(r, scale=SCALE)
    got = host(out)[0]
    for b in range(w.batch):
        ref, _, _ = oracle_frontier(r, b, scale=SCALE)
        n = int(n_inl[b])
        assert_attn_close(got[b][:n], ref, w.dtype)

"""Composition overlapped with prefill (the benchmark's overlapped TTFT schedule).

Layers are composed in chunks, all but the first on a second stream, and each layer's prefill
waits only for its own chunk's compose.  The kernels and inputs are those of the sequential
order, so the caches and outputs must be bit-identical to it: eagerly and replayed from a
recorded graph (whose side-stream branch must be part of the recording), for the batch and for
a request served alone.
"""
import numpy as np
import pytest
import torch

import synth
from bench import ZERO_COPY, DeviceWorkload, single_request_ttft
from oracle import pic_oracle as O

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _host(t):
    return t.float().cpu().numpy()


@pytest.mark.parametrize("chunk", [1, 4])
def test_overlapped_batch_equals_sequential(chunk):
    w = synth.get("c3")
    wl = DeviceWorkload(w, DEV, n_dec=1, layers=6)
    print(f"[overlap batch] {w.name} x {wl.L} layers, batch {w.batch}, chunk {chunk}", flush=True)
    wl.step()
    torch.cuda.synchronize()
    # the TTFT part of the step again, sequentially: compose, then every layer's prefill
    wl.cache_k.zero_(); wl.cache_v.zero_(); wl.out.zero_()
    nb, ng = wl.plan_upload()
    wl.compose(wl.blocks_dev, wl.groups_dev, nb, ng, wl.cache_k, wl.cache_v, w.batch)
    for l in range(wl.L):
        wl.prefill_layer(l)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (wl.out, wl.cache_k, wl.cache_v)]
    side = torch.cuda.Stream()
    events = [torch.cuda.Event() for _ in range(wl.L + 1)]

    def same():
        return all(torch.equal(a, b) for a, b in zip((wl.out, wl.cache_k, wl.cache_v), ref))

    wl.cache_k.zero_(); wl.cache_v.zero_(); wl.out.zero_()
    nb, ng = wl.plan_upload()
    wl.ttft_overlapped(nb, ng, side, events, chunk)
    torch.cuda.synchronize()
    assert same(), "eager overlapped schedule differs from the sequential one"
    print("[overlap batch] eager bit-identical", flush=True)
    nb, ng = wl.plan_upload()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        wl.ttft_overlapped(nb, ng, side, events, chunk)
    for rep in range(3):
        wl.cache_k.zero_(); wl.cache_v.zero_(); wl.out.zero_()   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert same(), f"graph replay {rep} differs from the sequential schedule"
    print("[overlap batch] 3 graph replays bit-identical", flush=True)


def test_overlapped_lone_request_equals_sequential():
    # the benchmark's lone-request path, sequential and overlapped (chunks of 4 of 6 layers, so
    # the side stream composes layers 4 and 5); the last launch of each is a graph replay
    w = synth.get("c3")
    wl = DeviceWorkload(w, DEV, n_dec=1, layers=6)
    print(f"[overlap lone] {w.name} x {wl.L} layers", flush=True)
    wl.out.zero_()
    single_request_ttft(wl, n_requests=1, reps=1, chunks=[0])
    torch.cuda.synchronize()
    ref = wl.out[:, :1].clone()
    wl.out.zero_()
    single_request_ttft(wl, n_requests=1, reps=1, chunks=[4])
    torch.cuda.synchronize()
    assert torch.equal(wl.out[:, :1], ref), "overlapped lone request differs from the sequential one"
    print("[overlap lone] bit-identical to the sequential schedule", flush=True)
    # and against the oracle on a layer composed on the side stream (every suffix token)
    lay, r, Ls, l = wl.lay, 0, w.n_suffix, 5
    m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
    K, V = O.compose_request(_host(wl.pool_k[l]), _host(wl.pool_v[l]), m, w.rope_theta, w.dtype)
    ref_o, _, _ = O.suffix_prefill(K, V, _host(wl.q[l, r]), _host(wl.k_suf[l, r]), _host(wl.v_suf[l, r]))
    got = _host(wl.out[l, r])
    from gpu_path import assert_attn_close
    assert_attn_close(got, ref_o, w.dtype)
    print(f"[overlap lone] layer {l} matches the oracle", flush=True)


@pytest.mark.parametrize("name", ["c3", "c5"])
def test_zero_copy_lone_request_matches_oracle(name):
    # the benchmark's zero-copy schedule for a request served alone (slot map, the tiles that are
    # not whole pool runs composed for all layers, paged prefill without the slot map): every
    # suffix token of two layers against the oracle, eager then graph replay (the last launch).
    # The 32K Qwen shape's jittered documents leave tiles that are not whole runs.
    w = synth.get(name)
    wl = DeviceWorkload(w, DEV, n_dec=1, layers=2)
    print(f"[zero-copy lone] {w.name} x {wl.L} layers", flush=True)
    wl.out.zero_()
    res = single_request_ttft(wl, n_requests=1, reps=1, chunks=[ZERO_COPY])
    torch.cuda.synchronize()
    assert set(res) == {ZERO_COPY}
    from gpu_path import assert_attn_close
    lay, r = wl.lay, 0
    m = O.plan_layout([lay.requests[r]], lay.doc_offset, lay.doc_len, lay.doc_compile_pos)[0]
    for l in range(wl.L):
        K, V = O.compose_request(_host(wl.pool_k[l]), _host(wl.pool_v[l]), m, w.rope_theta, w.dtype)
        ref_o, _, _ = O.suffix_prefill(K, V, _host(wl.q[l, r]), _host(wl.k_suf[l, r]), _host(wl.v_suf[l, r]))
        assert_attn_close(_host(wl.out[l, r]), ref_o, w.dtype)
        print(f"[zero-copy lone] layer {l} matches the oracle", flush=True)

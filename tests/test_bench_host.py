"""Host-side pieces of bench.py (no GPU): the one-GPU guard, the algorithmic work per launch that
the roofline divides by, and the rule that counter-measured traffic is reported only for the
kernel source and path it was measured on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_work_per_launch_on_the_llama_shape():
    # 32-layer Llama shape: 16 requests x 10 368 composed tokens, 128 suffix tokens, Hq 32,
    # Hkv 8, D 128, bf16 -- the sums written out by hand
    w = synth.get("c3")
    ctx = [10368] * 16
    # compose: every K and V row read once and written once, 256 bytes each
    assert bench.compose_bytes(w, ctx, 32) == 16 * 10368 * 8 * 32 * (2 * 2 * 256)
    # prefill: suffix token i sees 10368 + i + 1 keys; 4 * Hq * D flops per visible pair
    pairs = 16 * sum(10368 + i + 1 for i in range(128))
    assert bench.prefill_flops(w, pairs) == 4 * 32 * 128 * pairs
    assert abs(bench.prefill_flops(w, pairs) * 32 / 1e12 - 11.2) < 0.05   # 11.2 TFLOP over 32 layers
    # decode: the first token sees 10368 + 128 + 1 slots, K and V read once per layer
    assert bench.decode_bytes(w, [10497] * 16) == 16 * 10497 * 8 * 2 * 256


def test_traffic_only_for_the_profiled_source_and_path(tmp_path):
    h = bench.source_hash(bench.KERNEL_SOURCES["suffix_prefill_attn"])
    good = {"llama8b_32layer": {"suffix_prefill_attn": {"source_sha256_16": h, "bytes_per_launch": 7.5e8}}}
    stale = {"llama8b_32layer": {"suffix_prefill_attn": {"source_sha256_16": "0" * 16, "bytes_per_launch": 7.5e8}}}
    f_good, f_stale = tmp_path / "good.json", tmp_path / "stale.json"
    f_good.write_text(json.dumps(good))
    f_stale.write_text(json.dumps(stale))
    assert bench.lookup_traffic("llama8b_32layer", "suffix_prefill_attn", path=str(f_good)) == 7.5e8
    assert bench.lookup_traffic("llama8b_32layer", "suffix_prefill_attn", path=str(f_stale)) is None
    assert bench.lookup_traffic("llama8b_32layer", "suffix_prefill_attn", plain_path=False,
                                path=str(f_good)) is None
    assert bench.lookup_traffic("qwen7b_32k", "suffix_prefill_attn", path=str(f_good)) is None
    assert bench.lookup_traffic("llama8b_32layer", "decode_attn", path=str(tmp_path / "none.json")) is None


def test_committed_traffic_figures_are_well_formed():
    with open(bench.TRAFFIC_FILE) as f:
        t = json.load(f)
    for wl, kernels in t.items():
        for k, v in kernels.items():
            assert k in bench.KERNEL_SOURCES
            assert v["source"] == bench.KERNEL_SOURCES[k]
            assert v["bytes_per_launch"] == pytest.approx(v["read_bytes"] + v["write_bytes"])
            assert v["read_bytes"] == pytest.approx(v["fetch_size_kib"] * 1024 * v["fetch_scale"])
            assert v["write_bytes"] == pytest.approx(v["write_size_kib"] * 1024 * v["write_scale"])
            assert all("rocprofv3 --pmc" in c for c in v["commands"])


def test_compose_moved_bytes_counts_each_shared_run_once():
    # The compose launch reads every distinct 64-token source run once per group of at most 8
    # placements and writes every placement: counted here from the layout with a Counter,
    # independently of the planner's grouping.
    import collections

    import paper_2607_28069_amd as pic
    from synth import inputs as S
    w = synth.get("c3")
    lay = S.pool_layout(w)
    runs = collections.Counter()
    rows_w = 0
    for req in lay.requests:
        for e in req:
            off, n = int(lay.doc_offset[e]), int(lay.doc_len[e])
            for t in range(0, n, 64):
                runs[(off + t, min(64, n - t))] += 1
                rows_w += min(64, n - t)
    rows_r = sum(n * -(-c // 8) for (_, n), c in runs.items())
    unit = w.n_kv_heads * w.n_layers * 2 * w.head_dim * w.elem_bytes
    blocks, _ = pic.pic_plan_layout(lay.requests, lay.doc_offset, lay.doc_len, lay.doc_compile_pos,
                                    lay.pool_tokens)
    sorted_blocks, starts = pic.pic_plan_shared(blocks)
    assert bench.compose_moved_bytes(w, sorted_blocks, starts, w.n_layers) == (rows_r + rows_w) * unit
    # per-block compose reads what it writes: the per-composed-row unit
    ctx = S.context_lengths(lay)
    assert bench.compose_moved_bytes(w, blocks, None, w.n_layers) == bench.compose_bytes(w, ctx, w.n_layers)
    assert rows_r < rows_w / 2   # 16 requests share the prefix and draw 10 of 64 documents


def test_rerotate_bytes():
    # one key row read and written per (token, head), one int32 shift per token
    assert bench.rerotate_bytes(1000, 8, 128, 2) == 1000 * (8 * 512 + 4)

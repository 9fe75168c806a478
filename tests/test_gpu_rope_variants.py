"""GPU parity of the reader-side rotary variants (a layer-specific R_l, Sec. 2; Eq. 3 for any
rotary transform): delta-angle tables built from given frequencies (one block per layer),
composition and standalone re-rotation with the interleaved pairing and with Llama-3.1
frequency-scaled or per-layer frequencies, and suffix RoPE applied through the re-rotation call.

Tolerances: tables within 6e-8 of float64 cos/sin; keys within 1e-5 (float32) or 1 bf16 ulp
(+1e-5); values bit-exact.
"""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
from oracle import pic_oracle as O

from gpu_path import DEV, assert_keys_close, host, to_dev

pytestmark = pytest.mark.gpu
rng = np.random.default_rng(2607)


def _freqs(D):
    """Three layers with three different transforms."""
    return np.stack([pic.pic_rope_llama3_freq(D, 5e5), O.inv_freq(D, 1e4),
                     pic.pic_rope_llama3_freq(D, 1e6, 16.0, 1.0, 32.0, 4096)])


def test_table_from_frequencies_one_block_per_layer():
    for D in (64, 128):
        f = _freqs(D)
        m = pic.Model.of(3, 4, 2, D, "bf16", 5e5, per_layer_tables=True)
        mad = 30000
        table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
        pic.pic_rope_table_init_freq(m, f, mad, table)
        t = host(table).reshape(3, mad + 1, D // 2, 2)
        rows = np.array([0, 1, 9, 4097, 29999, 30000])
        for l in range(3):
            ang = rows[:, None].astype(np.float64) * f[l][None, :]
            assert np.abs(t[l, rows, :, 0] - np.cos(ang)).max() <= 6e-8
            assert np.abs(t[l, rows, :, 1] - np.sin(ang)).max() <= 6e-8


@pytest.mark.parametrize("dtype,D", [("f32", 64), ("bf16", 128)])
@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_compose_with_rotary_variants(dtype, D, pairing):
    # 3 layers, each with its own frequencies; 2 requests x 3 documents behind a stored prefix
    L, Hkv, B = 3, 2, 2
    f = _freqs(D)
    lens = np.array([150, 200, 64, 97, 40], np.int32)       # entry 4 is the prefix
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int32)
    cpos = np.array([0, 0, 0, 0, 0], np.int32)
    T = int(lens.sum())
    reqs = [[4, 1, 0, 3], [4, 2, 3, 1]]
    tok_cpos = np.concatenate([np.arange(n) + c for n, c in zip(lens, cpos)])
    raw = rng.standard_normal((L, Hkv, T, D))
    pool_k = np.stack([O.store(O.rope(raw[l], tok_cpos, 0.0, pairing, f[l]), dtype) for l in range(L)])
    pool_v = O.store(rng.standard_normal((L, Hkv, T, D)), dtype)
    m = pic.Model.of(L, 4, Hkv, D, dtype, 5e5, pairing=pairing, per_layer_tables=True)
    blocks, ctx = pic.pic_plan_layout(reqs, offs, lens, cpos, T)
    cap = int(ctx.max()) + 3
    mad = cap
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init_freq(m, f, mad, table)
    ck = torch.zeros((L, B, Hkv, cap, D), dtype=dt, device=DEV)
    cv = torch.zeros_like(ck)
    bl = torch.from_numpy(blocks.view(np.int32).reshape(-1).copy()).to(DEV)
    dpk, dpv = to_dev(pool_k, dt), to_dev(pool_v, dt)
    pic.pic_compose(m, dpk, dpv, T, bl, len(blocks), table, mad, ck, cv, B, cap)
    # shared sources (the two requests place documents 1 and 3 twice): the same cache, bit for bit
    sb, gs = pic.pic_plan_shared(blocks)
    assert len(gs) - 1 < len(blocks)
    ck2, cv2 = torch.zeros_like(ck), torch.zeros_like(cv)
    pic.pic_compose_shared(m, dpk, dpv, T, torch.from_numpy(sb.view(np.int32).reshape(-1).copy()).to(DEV),
                           len(sb), torch.from_numpy(gs).to(DEV), len(gs) - 1, table, mad, ck2, cv2, B, cap)
    torch.cuda.synchronize()
    assert torch.equal(ck, ck2) and torch.equal(cv, cv2), "shared-source compose differs"
    gk, gv = host(ck), host(cv)
    maps = O.plan_layout(reqs, offs, lens, cpos)
    for l in range(L):
        for b in range(B):
            K, V = O.compose_request(pool_k[l], pool_v[l], maps[b], 0.0, dtype, pairing, f[l])
            n = maps[b].ctx_len
            assert np.array_equal(gv[l, b, :, :n].view(np.uint32), V.view(np.uint32))
            assert_keys_close(gk[l, b, :, :n], K, dtype)
    # the prefix (delta 0) stays bit-identical under every transform
    p = lens[4]
    assert np.array_equal(gk[:, :, :, :p].view(np.uint32),
                          np.broadcast_to(pool_k[:, None, :, offs[4]:offs[4] + p], gk[:, :, :, :p].shape).view(np.uint32))


def test_rerotate_interleaved_scaled_and_suffix_rope():
    D, H, n = 128, 4, 257
    f = _freqs(D)
    m3 = pic.Model.of(3, 8, 4, D, "bf16", 5e5, pairing="interleaved", per_layer_tables=True)
    mad = 40000
    table = torch.empty(pic.pic_rope_table_bytes(m3, mad) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init_freq(m3, f, mad, table)
    m = m3.with_layers(1)
    block = (mad + 1) * (D // 2) * 2                          # floats per layer block
    k = O.store(rng.standard_normal((n, H, D)), "bf16")
    a = rng.integers(0, 20000, n)
    b = rng.integers(0, 20000, n)
    kin = to_dev(k, torch.bfloat16)
    for l in range(3):                                       # layer l: its own block
        kout = torch.empty_like(kin)
        pic.pic_rerotate_keys(m, kin, kout, n, H, torch.from_numpy((b - a).astype(np.int32)).to(DEV),
                              table[l * block:], mad)
        ref = O.store(O.rerotate_keys(np.transpose(k, (1, 0, 2)), a, b, 0.0, "interleaved", f[l]), "bf16")
        assert_keys_close(np.transpose(host(kout), (1, 0, 2)), ref, "bf16")
    # suffix tokens computed at request time: raw q/k turned to their positions by the same call
    ctx = 12345
    pos = (ctx + np.arange(n)).astype(np.int32)
    raw = O.store(rng.standard_normal((n, H, D)), "bf16")
    out = to_dev(raw, torch.bfloat16)
    pic.pic_rerotate_keys(m, out, out, n, H, torch.from_numpy(pos).to(DEV), table, mad)
    ref = O.store(O.rope(np.transpose(raw, (1, 0, 2)), pos, 0.0, "interleaved", f[0]), "bf16")
    assert_keys_close(np.transpose(host(out), (1, 0, 2)), ref, "bf16")

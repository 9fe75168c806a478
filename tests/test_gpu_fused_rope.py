"""Fused RoPE of request-time tokens (Sec. 5: the Reader turns the suffix and decode tokens to
their positions; R(p) from the delta-angle table of Eq. 3).

pic_suffix_prefill_attn_rope and pic_decode_attn_rope take q and the new keys unrotated and
turn them inside the kernels.  They must equal, bit for bit, turning the same rows with
pic_rerotate_keys first and calling the plain kernels (outputs and cache), and match the oracle,
which rotates with its own float64 R(p), within the attention tolerance.  Both pairings, one
table for all layers and one table per layer, ragged contexts and a suffix that is not a
multiple of the key tile; the per-layer cases also pass a softmax scale other than 1/sqrt(D).
"""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
from oracle import pic_oracle as O

from gpu_path import DEV, assert_attn_close, assert_keys_close, host, to_dev

pytestmark = pytest.mark.gpu
rng = np.random.default_rng(77)
D, HQ, HKV, L = 128, 32, 8, 2


def _model_and_table(pairing, per_layer, mad):
    m = pic.Model.of(L, HQ, HKV, D, "bf16", 5e5, pairing=pairing, per_layer_tables=per_layer)
    table = torch.empty(pic.pic_rope_table_bytes(m, mad) // 4, dtype=torch.float32, device=DEV)
    if per_layer:
        freqs = np.stack([pic.pic_rope_llama3_freq(D, 5e5), O.inv_freq(D, 1e4)])
        pic.pic_rope_table_init_freq(m, freqs, mad, table)
    else:
        freqs = np.stack([O.inv_freq(D, 5e5)] * L)
        pic.pic_rope_table_init(m, mad, table)
    block = (mad + 1) * (D // 2) * 2 if per_layer else 0     # floats per layer block
    return m, table, block, freqs


def _rerotate_rows(m1, x, pos, table, mad):
    """x [n][H][D] bf16 device rows turned to positions pos [n] by pic_rerotate_keys."""
    y = torch.empty_like(x)
    pic.pic_rerotate_keys(m1, x, y, x.shape[0], x.shape[1], torch.from_numpy(pos.astype(np.int32)).to(DEV),
                          table, mad)
    return y


def _bf16(shape):
    return O.store(rng.standard_normal(shape), "bf16")


@pytest.mark.parametrize("per_layer", [False, True], ids=["one-table", "per-layer"])
@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_fused_rope_prefill(pairing, per_layer):
    B, Ls = 3, 37
    scale = 0.05 if per_layer else 0.0
    ctx = np.array([700, 2501, 1], np.int32)
    max_ctx, cap = int(ctx.max()), int(ctx.max()) + Ls + 3
    mad = max_ctx + Ls
    m, table, block, freqs = _model_and_table(pairing, per_layer, mad)
    m1 = m.with_layers(1)
    ck = to_dev(_bf16((L, B, HKV, cap, D)), torch.bfloat16)
    cv = to_dev(_bf16((L, B, HKV, cap, D)), torch.bfloat16)
    q_raw, k_raw, v = _bf16((L, B, Ls, HQ, D)), _bf16((L, B, Ls, HKV, D)), _bf16((L, B, Ls, HKV, D))
    dq, dk, dv = (to_dev(x, torch.bfloat16) for x in (q_raw, k_raw, v))
    ctx_d = torch.from_numpy(ctx).to(DEV)
    ws = torch.empty(max(pic.pic_prefill_workspace_bytes(m, B, Ls, max_ctx), 16), dtype=torch.uint8, device=DEV)
    print(f"[{pairing}, {'per-layer' if per_layer else 'one table'}] ctx {list(ctx)}, {Ls} suffix tokens",
          flush=True)

    # fused
    ck_a, cv_a = ck.clone(), cv.clone()
    out_a = torch.zeros((L, B, Ls, HQ, D), dtype=torch.bfloat16, device=DEV)
    pic.pic_suffix_prefill_attn_rope(m, dq, dk, dv, ck_a, cv_a, B, cap, ctx_d, max_ctx, Ls, table, mad, out_a, ws,
                                     scale=scale)
    # turned first, then the plain kernel
    pos = (ctx[:, None] + np.arange(Ls)[None, :]).reshape(-1)          # [B * Ls]
    q_rot = torch.stack([_rerotate_rows(m1, dq[l].reshape(B * Ls, HQ, D), pos, table[l * block:], mad)
                         for l in range(L)]).reshape(dq.shape)
    k_rot = torch.stack([_rerotate_rows(m1, dk[l].reshape(B * Ls, HKV, D), pos, table[l * block:], mad)
                         for l in range(L)]).reshape(dk.shape)
    ck_b, cv_b = ck.clone(), cv.clone()
    out_b = torch.zeros_like(out_a)
    pic.pic_suffix_prefill_attn(m, q_rot, k_rot, dv, ck_b, cv_b, B, cap, ctx_d, max_ctx, Ls, out_b, ws, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b), "fused-RoPE prefill differs from turn-then-prefill"
    assert torch.equal(ck_a, ck_b) and torch.equal(cv_a, cv_b), "caches differ"

    # oracle: float64 R(p) of the raw rows, attention over the cached context + turned suffix
    got = host(out_a)
    ckh, cvh = host(ck), host(cv)
    for l, b in ((0, 0), (1, 1), (L - 1, 2)):
        n = int(ctx[b])
        p = n + np.arange(Ls)
        qr = O.rope(np.transpose(q_raw[l, b], (1, 0, 2)), p, 0.0, pairing, freqs[l])
        kr = O.store(O.rope(np.transpose(k_raw[l, b], (1, 0, 2)), p, 0.0, pairing, freqs[l]), "bf16")
        Kf = np.concatenate([ckh[l, b][:, :n], kr], axis=1)
        Vf = np.concatenate([cvh[l, b][:, :n], np.transpose(v[l, b], (1, 0, 2))], axis=1)
        ref = O.attention(qr, p, Kf, Vf, np.arange(n + Ls), scale or None)
        assert_attn_close(np.transpose(got[l, b], (1, 0, 2)), ref, "bf16")
    print("fused == turned + plain (bitwise), oracle ok", flush=True)


@pytest.mark.parametrize("per_layer", [False, True], ids=["one-table", "per-layer"])
@pytest.mark.parametrize("pairing", ["half", "interleaved"])
def test_fused_rope_decode(pairing, per_layer):
    B, steps = 4, 2
    scale = 0.05 if per_layer else 0.0
    base = np.array([5000, 37, 12000, 64], np.int32)
    max_base = int(base.max())
    cap, mad = max_base + steps + 5, max_base + steps
    m, table, block, freqs = _model_and_table(pairing, per_layer, mad)
    m1 = m.with_layers(1)
    ck = to_dev(_bf16((L, B, HKV, cap, D)), torch.bfloat16)
    cv = to_dev(_bf16((L, B, HKV, cap, D)), torch.bfloat16)
    base_d = torch.from_numpy(base).to(DEV)
    ck_a, cv_a, ck_b, cv_b = ck.clone(), cv.clone(), ck.clone(), cv.clone()
    for split in (0, 3):
        ws = torch.zeros(max(pic.pic_decode_workspace_bytes(m, B, max_base + steps, split), 16), dtype=torch.uint8,
                         device=DEV)
        for t in range(steps):
            q_raw, k_raw, v = _bf16((L, B, HQ, D)), _bf16((L, B, HKV, D)), _bf16((L, B, HKV, D))
            dq, dk, dv = (to_dev(x, torch.bfloat16) for x in (q_raw, k_raw, v))
            out_a = torch.zeros((L, B, HQ, D), dtype=torch.bfloat16, device=DEV)
            pic.pic_decode_attn_rope(m, dq, dk, dv, ck_a, cv_a, B, cap, base_d, t, max_base, table, mad, out_a, ws,
                                     n_splits=split, scale=scale)
            pos = base + t
            q_rot = torch.stack([_rerotate_rows(m1, dq[l], pos, table[l * block:], mad) for l in range(L)])
            k_rot = torch.stack([_rerotate_rows(m1, dk[l], pos, table[l * block:], mad) for l in range(L)])
            out_b = torch.zeros_like(out_a)
            pic.pic_decode_attn(m, q_rot, k_rot, dv, ck_b, cv_b, B, cap, base_d, t, max_base, out_b, ws,
                                n_splits=split, scale=scale)
            torch.cuda.synchronize()
            assert torch.equal(out_a, out_b), f"split {split} step {t}: fused-RoPE decode differs"
            assert torch.equal(ck_a, ck_b) and torch.equal(cv_a, cv_b), f"split {split} step {t}: caches differ"
            # oracle on one request per layer: float64 R(p) of the raw rows
            got = host(out_a)
            ckh, cvh = host(ck_a), host(cv_a)
            for l, b in ((0, 1), (L - 1, 2)):
                p = int(pos[b])
                qr = O.rope(q_raw[l, b][:, None, :], np.array([p]), 0.0, pairing, freqs[l])[:, 0]
                kr = O.store(O.rope(k_raw[l, b][:, None, :], np.array([p]), 0.0, pairing, freqs[l]), "bf16")
                assert_keys_close(ckh[l, b][:, p:p + 1], kr, "bf16")   # the stored key, turned
                ref = O.attention(qr[:, None, :], np.array([p]), ckh[l, b][:, :p + 1], cvh[l, b][:, :p + 1],
                                  np.arange(p + 1), scale or None)[:, 0]
                assert_attn_close(got[l, b], ref, "bf16")
        print(f"[{pairing}] split {split}: fused decode == turned + plain, oracle ok", flush=True)

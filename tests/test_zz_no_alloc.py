"""pic_decode_attn_noalloc: decode whose split-K partials live in the library's per-GPU scratch
array instead of a caller workspace.  Two calls in a row (the second smaller) must give outputs
and caches bit-identical to pic_decode_attn with a workspace (same kernels, same split count),
and one sampled head is checked against the CPU oracle.  A request whose partials exceed the
scratch array is refused before anything is launched."""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
from oracle import pic_oracle as O

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda", 0)


def _case(layers, batch, hq, hkv, ctx, n_splits, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    D, cap = 128, int(max(ctx)) + 4
    model = pic.Model.of(layers, hq, hkv, D, "bf16", 5e5)
    rnd = lambda *s: torch.randn(s, generator=g, device=DEV, dtype=torch.float32).to(torch.bfloat16)
    ck, cv = rnd(layers, batch, hkv, cap, D), rnd(layers, batch, hkv, cap, D)
    q, kn, vn = rnd(layers, batch, hq, D), rnd(layers, batch, hkv, D), rnd(layers, batch, hkv, D)
    base = torch.tensor(ctx, dtype=torch.int32, device=DEV)
    return model, q, kn, vn, ck, cv, base, cap, int(max(ctx)), n_splits


def _run_both(model, q, kn, vn, ck, cv, base, cap, max_base, n_splits, step=1):
    batch = q.shape[1]
    ck2, cv2 = ck.clone(), cv.clone()
    ws = torch.empty(max(pic.pic_decode_workspace_bytes(model, batch, max_base + step + 1, n_splits), 16),
                     dtype=torch.uint8, device=DEV)
    out_ref = torch.full_like(q, float("nan"))
    out = torch.full_like(q, float("nan"))
    pic.pic_decode_attn(model, q, kn, vn, ck, cv, batch, cap, base, step, max_base, out_ref, ws, n_splits=n_splits)
    pic.pic_decode_attn_noalloc(model, q, kn, vn, ck2, cv2, batch, cap, base, step, max_base, out,
                                n_splits=n_splits)
    torch.cuda.synchronize()
    assert torch.equal(out, out_ref), "no-alloc decode differs from the workspace decode"
    assert torch.equal(ck, ck2) and torch.equal(cv, cv2), "caches differ"
    return out, ck, cv


def test_noalloc_decode_matches_workspace_decode_twice():
    # first call: 2 layers, one request, ~5K context, automatic split count (many splits)
    a = _case(2, 1, 32, 8, [5000], 0, 1)
    model = a[0]
    assert pic.pic_decode_auto_splits(model, 1, 5000 + 2) > 1
    out, ck, cv = _run_both(*a)
    # the oracle on one (layer, request): all heads of the new token at slot 5001
    l = 1
    K = ck[l, 0, :, :5002].float().cpu().numpy()
    V = cv[l, 0, :, :5002].float().cpu().numpy()
    qh = a[1][l, 0].float().cpu().numpy()
    ref = O.attention(qh[:, None, :], np.asarray([5001]), K, V, np.arange(5002))[:, 0]
    got = out[l, 0].float().cpu().numpy()
    assert np.all(np.abs(got - ref) <= 2e-2 + 1e-2 * np.abs(ref))
    assert np.linalg.norm(got - ref) / np.linalg.norm(ref) <= 1e-2
    # second call, smaller: 3 requests of ragged shorter contexts, 3 explicit splits, reusing the
    # array the first call left behind
    b = _case(1, 3, 32, 8, [700, 1200, 33], 3, 2)
    _run_both(*b)
    print("no-alloc decode == workspace decode on two calls in a row", flush=True)


def test_noalloc_decode_refuses_partials_beyond_the_scratch():
    model, q, kn, vn, ck, cv, base, cap, max_base, _ = _case(1, 64, 32, 8, [600] * 64, 0, 3)
    need = pic.pic_decode_workspace_bytes(model, 64, max_base + 2, 64)
    assert need > pic.PIC_DECODE_SCRATCH_BYTES
    out = torch.full_like(q, 7.0)
    with pytest.raises(pic.PicError) as e:
        pic.pic_decode_attn_noalloc(model, q, kn, vn, ck, cv, 64, cap, base, 1, max_base, out, n_splits=64)
    assert e.value.status == -3   # PIC_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 7.0).all()), "a refused call must launch nothing"

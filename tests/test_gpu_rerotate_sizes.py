"""Standalone re-rotation (Sec. 2, Eq. 3) at the sizes where its launch changes form.

pic_rerotate_keys covers up to 2^31 (row, pair chunk) items in one pass of its grid (one item per
thread) and loops over the rest; from 2^32 items on it switches to 64-bit index arithmetic.  Two
in-place calls on bf16 keys of 8 kv heads x 128 (8 items per row) just past each boundary: 2^31
items is a 69 GB key set, 2^32 a 137 GB one (the test skips when the GPU has less free memory).
Sampled tokens (the first, the last, those at the item boundaries and random ones) are compared
with the oracle's re-rotation of their original rows; one shift per token, constant over 64-token
runs, as in the benchmark's re-rotation leg."""
import numpy as np
import pytest
import torch

import paper_2607_28069_amd as pic
from oracle import pic_oracle as O

from gpu_path import DEV, assert_keys_close

pytestmark = pytest.mark.gpu

H, D, LPR, MAD, THETA = 8, 128, 8, 16384, 5e5


@pytest.mark.parametrize("items_log2", [31, 32])
def test_rerotate_past_one_pass_and_32_bit_indices(items_log2):
    n_tok = (1 << items_log2) // (LPR * H) + 37          # items = n_tok * H * LPR, just past 2^k
    need = n_tok * H * D * 2 + n_tok * 12
    free, _ = torch.cuda.mem_get_info()
    if free < need + (16 << 30):
        pytest.skip(f"needs {need / 2**30:.0f} GiB of free GPU memory, {free / 2**30:.0f} free")
    print(f"[rerotate sizes] 2^{items_log2}: {n_tok} tokens, {need / 1e9:.1f} GB", flush=True)
    m = pic.Model.of(1, 32, H, D, "bf16", THETA)
    table = torch.empty(pic.pic_rope_table_bytes(m, MAD) // 4, dtype=torch.float32, device=DEV)
    pic.pic_rope_table_init(m, MAD, table)
    keys = torch.empty((n_tok, H, D), dtype=torch.bfloat16, device=DEV).normal_()
    tok = torch.arange(n_tok, device=DEV)
    delta = ((tok // 64 * 1031) % (2 * MAD + 1) - MAD).to(torch.int32)
    del tok
    rng = np.random.default_rng(items_log2)
    bound = [(1 << 31) // (LPR * H), (1 << 32) // (LPR * H)]
    sample = np.unique(np.clip(np.concatenate([
        [0, 1, n_tok // 2, n_tok - 1], [b + o for b in bound for o in (-1, 0, 1)],
        rng.integers(0, n_tok, 48)]), 0, n_tok - 1))
    idx = torch.from_numpy(sample).to(DEV)
    before = keys.index_select(0, idx).float().cpu().numpy()          # [S][H][D]
    shifts = delta.index_select(0, idx).cpu().numpy().astype(np.int64)
    pic.pic_rerotate_keys(m, keys, keys, n_tok, H, delta, table, MAD)
    after = keys.index_select(0, idx).float().cpu().numpy()
    torch.cuda.synchronize()
    del keys, delta
    torch.cuda.empty_cache()
    ref = O.store(O.rerotate_keys(np.transpose(before, (1, 0, 2)), np.zeros(len(sample), np.int64), shifts,
                                  THETA), "bf16")
    frac = assert_keys_close(np.transpose(after, (1, 0, 2)), ref, "bf16")
    assert frac > 0.999
    print(f"[rerotate sizes] 2^{items_log2}: {len(sample)} sampled tokens match the oracle "
          f"({100 * frac:.3f} % bit-identical)", flush=True)

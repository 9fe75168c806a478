"""The oracle's pins against planted mistakes: each case rewrites one line of the oracle's source
(a wrong sign, a dropped term, a swapped operand, an off-by-one position, a wrong rounding), loads
the result as a separate module, points the pins of test_oracle_pins at it, and requires the named
pins to fail.  A control case loads the unmodified source the same way and requires the same pins
to pass, so a failure means the mistake was caught, not that the harness broke.

CPU only; every pin named here is a plain test function of test_oracle_pins (no parameters)."""
import os
import sys
import types

import pytest

import test_oracle_pins as P

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "pic_oracle.py")

# (mistake, original line(s), planted line(s), pins expected to catch it)
MUTANTS = [
    ("rotation: sine term with the wrong sign",
     "return _join_pairs(x1 * c - x2 * s, x1 * s + x2 * c, pairing)",
     "return _join_pairs(x1 * c + x2 * s, x1 * s + x2 * c, pairing)",
     ["test_rope_frequencies_and_pairing_match_hf_transformers"]),
    ("inverse rotation taken forward",
     "return _join_pairs(x1 * c + x2 * s, -x1 * s + x2 * c, pairing)",
     "return _join_pairs(x1 * c - x2 * s, x1 * s + x2 * c, pairing)",
     ["test_rerotation_inverse_and_norm"]),
    ("re-rotation with compile and request positions swapped",
     "return rope(rope_inverse(k, a, theta, pairing, freqs), b, theta, pairing, freqs)",
     "return rope(rope_inverse(k, b, theta, pairing, freqs), a, theta, pairing, freqs)",
     ["test_composed_cache_equals_full_recompute_single_layer"]),
    ("interleaved pairs taken as halves",
     "return x[..., 0::2], x[..., 1::2]",
     "h = x.shape[-1] // 2\n        return x[..., :h], x[..., h:]",
     ["test_interleaved_pairing_matches_complex_multiplication"]),
    ("frontier mask strict (a token does not see itself)",
     "visible = np.asarray(k_pos)[None, :] <= np.asarray(q_pos)[:, None]",
     "visible = np.asarray(k_pos)[None, :] < np.asarray(q_pos)[:, None]",
     ["test_attention_brute_force_tiny"]),
    ("softmax scale dropped",
     "s = scale * (q[h] @ k[g].T)",
     "s = (q[h] @ k[g].T)",
     ["test_attention_brute_force_tiny"]),
    ("query head mapped to the wrong kv head",
     "g = h // n_rep",
     "g = h % Hkv",
     ["test_attention_brute_force_tiny"]),
    ("softmax not normalised",
     "out[h] = (w @ v[g]) / w.sum(axis=1, keepdims=True)",
     "out[h] = (w @ v[g])",
     ["test_attention_brute_force_tiny"]),
    ("decode query one position early",
     "o = attention(np.asarray(q)[:, None, :], np.asarray([length]), K2, V2,",
     "o = attention(np.asarray(q)[:, None, :], np.asarray([length - 1]), K2, V2,",
     ["test_decode_step_equals_prefill_row"]),
    ("bf16 rounding to 7 significant bits",
     "return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8).astype(np.float32)",
     "return np.ldexp(np.rint(np.ldexp(m, 7)), e - 7).astype(np.float32)",
     ["test_round_to_bf16_matches_torch_cast"]),
    ("bf16 rounding by truncation",
     "return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8).astype(np.float32)",
     "return np.ldexp(np.trunc(np.ldexp(m, 8)), e - 8).astype(np.float32)",
     ["test_round_to_bf16_matches_torch_cast"]),
    ("rotary frequencies with exponent i/D instead of 2i/D",
     "return np.power(float(theta), -2.0 * i / head_dim)",
     "return np.power(float(theta), -1.0 * i / head_dim)",
     ["test_rope_frequencies_and_pairing_match_hf_transformers"]),
    ("Llama-3.1 scaling: blend weights reversed",
     "blended = (1.0 - smooth) * f / factor + smooth * f",
     "blended = smooth * f / factor + (1.0 - smooth) * f",
     ["test_llama3_scaled_frequencies_match_hf_transformers"]),
    ("Llama-3.1 scaling: long wavelengths not divided",
     "out = np.where(wavelen > original_max_position / low_freq_factor, f / factor, blended)",
     "out = np.where(wavelen > original_max_position / low_freq_factor, f, blended)",
     ["test_llama3_scaled_frequencies_match_hf_transformers"]),
    ("layout: compile positions ignored",
     "                a.append(int(doc_compile_pos[e]) + t)\n                b.append(pos + t)\n"
     "            pos += n\n        maps.append(RequestMap(pos,",
     "                a.append(t)\n                b.append(pos + t)\n            pos += n\n"
     "        maps.append(RequestMap(pos,",
     ["test_boundary_layout_hand_computed_and_equal_to_full_recompute"]),
    ("layout: entries overlap by one position",
     "                b.append(pos + t)\n            pos += n\n        maps.append(RequestMap(pos,",
     "                b.append(pos + t)\n            pos += n - 1\n        maps.append(RequestMap(pos,",
     ["test_layout_tiny_workload_hand_computed"]),
    ("frontier layout: inline spans take no positions",
     "                inl.extend(range(pos, pos - it))\n                pos -= it",
     "                inl.extend(range(pos, pos - it))",
     ["test_frontier_layout_hand_computed"]),
    ("composition rotates the values too",
     "    v = np.asarray(pool_v, np.float32)[:, rmap.src_token, :].copy()",
     "    v = store(rerotate_keys(np.asarray(pool_v, np.float64)[:, rmap.src_token, :], rmap.compile_pos, "
     "rmap.logical_pos, theta, pairing, freqs), dtype)",
     ["test_composed_cache_equals_full_recompute_single_layer"]),
    ("composition without re-rotation",
     "    k = store(rerotate_keys(k_src, rmap.compile_pos, rmap.logical_pos, theta, pairing, freqs), dtype)",
     "    k = store(k_src, dtype)",
     ["test_composed_cache_equals_full_recompute_single_layer"]),
    ("suffix queries placed from position 0",
     "    o = attention(np.transpose(q, (1, 0, 2)), ctx + np.arange(Ls), K, V, pos, scale)",
     "    o = attention(np.transpose(q, (1, 0, 2)), np.arange(Ls), K, V, pos, scale)",
     ["test_decode_step_equals_prefill_row"]),
    ("frontier: inline keys not placed at their positions",
     "    K[:, fmap.inline_pos] = np.transpose(np.asarray(k_inl, np.float32), (1, 0, 2))\n",
     "    K[:, fmap.inline_pos] = 0.0\n",
     ["test_frontier_prefill_equals_full_causal_recompute"]),
]


def _load(monkeypatch, source: str, name: str) -> types.ModuleType:
    mod = types.ModuleType(name)
    mod.__file__ = ORACLE
    monkeypatch.setitem(sys.modules, name, mod)   # dataclasses look their module up there
    exec(compile(source, f"<{name}>", "exec"), mod.__dict__)
    return mod


def _failures(monkeypatch, module, pins):
    """Names of the pins that fail with the oracle replaced by `module`."""
    monkeypatch.setattr(P, "O", module)
    failed = []
    for pin in pins:
        try:
            getattr(P, pin)()
        except Exception:   # an assertion, or an error the planted mistake provokes
            failed.append(pin)
    return failed


def test_unmodified_source_passes_every_pin_used_here(monkeypatch):
    src = open(ORACLE).read()
    pins = sorted({p for m in MUTANTS for p in m[3]})
    assert _failures(monkeypatch, _load(monkeypatch, src, "pic_oracle_copy"), pins) == []


@pytest.mark.parametrize("mistake,old,new,pins", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(monkeypatch, mistake, old, new, pins):
    src = open(ORACLE).read()
    assert src.count(old) == 1, "the line to change is not in the oracle (exactly once)"
    assert _failures(monkeypatch, _load(monkeypatch, src.replace(old, new), "pic_oracle_mutant"), pins), mistake

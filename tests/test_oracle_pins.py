"""The oracle against its pins, and planted mistakes against the same pins.

A plausible slip anywhere in the oracle (a dropped term, a wrong sign, an
index off by one, a swapped operand, a different pooling or tie rule) must
make at least one pin fail; otherwise the pins would not be pinning anything.
"""
import importlib.util
import os
import types

import pytest

from oracle import hs2_oracle as O
from tests import oracle_pins as pins

ORACLE_SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "hs2_oracle.py")


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(O)


# (name, text in the oracle, planted replacement)
MUTANTS = [
    ("no_scale", "s = scale * (Krows @ q)", "s = Krows @ q"),
    ("exp_sign", "e = np.exp(s - M)", "e = np.exp(M - s)"),
    ("values_from_keys", "out = p @ Vrows", "out = p @ Krows"),
    ("unnormalised", "p = e / Z", "p = e"),
    ("max_not_subtracted_consistently", "M = s.max()", "M = s.min()"),
    ("pool_mean", "P[c, :n] = pooled.astype(np.float32)", "P[c, :n] = (pooled / G).astype(np.float32)"),
    ("pool_last_head_only", "pooled += p", "pooled = p"),
    ("query_pos_off_by_one", "np.arange(C, dtype=np.int64) + (int(L) - int(C))",
     "np.arange(C, dtype=np.int64) + (int(L) - int(C)) - 1"),
    ("no_causality_in_chunk", "np.arange(C, dtype=np.int64) + (int(L) - int(C))",
     "np.zeros(C, dtype=np.int64) + (int(L) - 1)"),
    ("window_one_too_wide", "lo = max(0, int(pos) - int(window) + 1)", "lo = max(0, int(pos) - int(window))"),
    ("topk_from_all_tokens", "N = max(0, int(pos) - int(window) + 1)", "N = int(pos) + 1"),
    ("topk_candidates_short", "N = max(0, int(pos) - int(window) + 1)", "N = max(0, int(pos) - int(window))"),
    ("ties_to_higher_index", "order = np.lexsort((t, -key))", "order = np.lexsort((-t, -key))"),
    ("ascending_scores", "order = np.lexsort((t, -key))", "order = np.lexsort((t, key))"),
    ("no_denormal_rule", "return np.where(P < FLT_MIN, np.float32(0.0), P)", "return P"),
    ("strided_head_groups", "return bf16_to_f64(q[b, :, g * G:(g + 1) * G, :])",
     "return bf16_to_f64(q[b, :, g::q.shape[2] // G, :])"),
    ("sparse_ignores_selection", "sel = sel[sel >= 0].astype(np.int64)", "sel = np.arange(int(sel.max()) + 1)"),
    ("sparse_keeps_padding", "sel = sel[sel >= 0].astype(np.int64)", "sel = sel.astype(np.int64)"),
    ("decode_truncated", "return (bits.astype(np.uint32) << 16)", "return (bits.astype(np.uint32) << 15)"),
    ("sink_in_numerator", "return (e @ Vrows) / (np.exp(sink - M) + e.sum())",
     "return (e @ Vrows + np.exp(sink - M)) / (np.exp(sink - M) + e.sum())"),
    ("sink_ignored", "(np.exp(sink - M) + e.sum())", "e.sum()"),
    ("sink_scaled_again", "np.exp(sink - M)", "np.exp(scale * sink - M)"),
    ("sink_of_kv_head", "float(sink[hq])", "float(sink[g])"),
    ("gate_exp", "out[b, c, hq] *= sigmoid(bf16_to_f64(gate[b, c, hq]))",
     "out[b, c, hq] *= np.exp(bf16_to_f64(gate[b, c, hq]))"),
    ("gate_sign_flipped", "1.0 / (1.0 + ex), ex / (1.0 + ex)", "ex / (1.0 + ex), 1.0 / (1.0 + ex)"),
    ("e4m3_bias_8", "np.exp2(e - 7.0)", "np.exp2(e - 8.0)"),
    ("e4m3_no_subnormals", "np.where(e == 0, m / 8.0 * 2.0 ** -6,", "np.where(e < 0, m / 8.0 * 2.0 ** -6,"),
    ("v_with_k_scale", "Vg = cache_rows(V, b, g, slice(0, L), v_scale)", "Vg = cache_rows(V, b, g, slice(0, L), k_scale)"),
    ("scale_of_head_0", "* float(scale[g])", "* float(scale[0])"),
    ("block_score_max", "out[j] = np.float32(vals[j * block: min((j + 1) * block, N)].sum())",
     "out[j] = np.float32(vals[j * block: min((j + 1) * block, N)].max())"),
    ("block_ties_to_higher", "order = np.lexsort((j, -key))", "order = np.lexsort((-j, -key))"),
    ("block_tokens_not_cut", "parts = [np.arange(j * block, min((j + 1) * block, N), dtype=np.int64)",
     "parts = [np.arange(j * block, (j + 1) * block, dtype=np.int64)"),
    ("block_budget_in_blocks", "kb = int(k) // int(block)", "kb = int(k)"),
    ("block_scores_into_window", "key = rank_key(block_scores(P_row, N, block))",
     "key = rank_key(block_scores(P_row, N + int(window), block))"),
    ("block_denormals_counted", "vals = rank_key(P_row[:N]).astype(np.float64)",
     "vals = P_row[:N].astype(np.float64)"),
]


def _mutant(name, old, new):
    src = open(ORACLE_SRC).read()
    assert src.count(old) >= 1, f"mutant {name}: text not found in the oracle"
    mod = types.ModuleType(f"hs2_oracle_mutant_{name}")
    mod.__file__ = ORACLE_SRC
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, old, new):
    mod = _mutant(name, old, new)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except Exception as e:  # noqa: BLE001 -- any failure of a pin counts
            failed.append((pin.__name__, type(e).__name__))
    assert failed, f"planted mistake {name} passed every pin"

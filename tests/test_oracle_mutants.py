"""Plants plausible mistakes in a copy of the oracle (on the CPU) and checks that
the pins catch each one: evidence that the pins constrain every part of it."""
import os
import types

import pytest

from .pins import ALL_PINS

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "reusevit.py")

# (name, original text, mutated text)
MUTANTS = [
    ("reused_key_from_own_frame", "k_t, v_t = k_r.copy(), v_r.copy()",
     "k_t, v_t = qkv_rows(x[f], P)[1:]"),
    ("fresh_value_dropped", "k_t[C], v_t[C] = k_c, v_c", "k_t[C] = k_c"),
    ("reused_row_keeps_input", "y[f] = y[r]  ", "y[f] = x[f]  "),
    ("recomputed_rows_not_written", "y[f, C] = y_c", "pass"),
    ("strict_threshold", "return cos >= tau", "return cos > tau"),
    ("equal_rows_not_one", "c[same] = 1.0", "pass"),
    ("cls_reusable", "m = np.concatenate([[False], reuse])", "m = np.concatenate([[True], reuse])"),
    ("no_attention_scale", "/ np.sqrt(dh)", "/ 1.0"),
    ("unbiased_variance", ".mean(axis=-1, keepdims=True)   # biased",
     ".sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)   #"),
    ("cls_without_pos", 'x[:, 0] = W["cls"] + W["pos"][0]', 'x[:, 0] = W["cls"]'),
    ("patch_vector_order", ".transpose(0, 2, 4, 1, 3, 5)", ".transpose(0, 2, 4, 1, 5, 3)"),
    ("patch_grid_order", ".transpose(0, 2, 4, 1, 3, 5)", ".transpose(0, 4, 2, 1, 3, 5)"),
    ("no_attention_residual", "z = x_rows + o_rows", "z = o_rows"),
    ("tanh_gelu", "0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))",
     "0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))"),
    ("gate_on_previous_frame", "c = cosine_rows(x[f, 1:], x[r, 1:])",
     "c = cosine_rows(x[f, 1:], x[f - 1, 1:])"),
    ("embedding_wrong_token", 'emb = layer_norm(x[:, 0]', 'emb = layer_norm(x[:, 1]'),
    ("qkv_transposed_slices", "return t[:, :D], t[:, D:2 * D], t[:, 2 * D:]",
     "return t[:, :D], t[:, 2 * D:], t[:, D:2 * D]"),
    ("mlp_gelu_before_bias", '@ P["W_1"].T + P["b_1"])', '@ P["W_1"].T) + P["b_1"]'),
    ("gate_on_normalised_input", "c = cosine_rows(x[f, 1:], x[r, 1:])",
     "c = cosine_rows(layer_norm(x[f, 1:], P['ln1_g'], P['ln1_b']), "
     "layer_norm(x[r, 1:], P['ln1_g'], P['ln1_b']))"),
    ("inf_tau_reuses_nothing", "return np.ones(cos.shape, dtype=bool)",
     "return np.zeros(cos.shape, dtype=bool)"),
    ("rate_counts_references", "nonref = [f for f in range(F) if f % group_size != 0]",
     "nonref = list(range(F))"),
    ("restore_difference_flipped", "x[f, Rr] - x[r, Rr]", "x[r, Rr] - x[f, Rr]"),
    ("restore_output_bias_dropped", '@ P["W_r2"].T + P["b_r2"]', '@ P["W_r2"].T'),
    ("restore_relu", 'gelu(dx @ P["W_r1"].T + P["b_r1"])',
     'np.maximum(dx @ P["W_r1"].T + P["b_r1"], 0.0)'),
    ("restore_output_difference", "x[f, Rr] - x[r, Rr]", "y[f, Rr] - y[r, Rr]"),
    ("restore_all_rows", "Rr = np.flatnonzero(m)", "Rr = np.arange(m.size)"),
    ("decision_features_swapped", "v = np.concatenate([s[:, None], t[:, None], r], axis=1)",
     "v = np.concatenate([t[:, None], s[:, None], r], axis=1)"),
    ("decision_type_b_dist2", "r[:, ftype] = 1.0", "r[:, ftype + 1] = 1.0"),
    ("decision_relu", 'gelu(v @ P["W_d1"].T + P["b_d1"])', 'np.maximum(v @ P["W_d1"].T + P["b_d1"], 0)'),
    ("decision_output_bias_dropped", '@ P["W_d2"].T + P["b_d2"])', '@ P["W_d2"].T)'),
    ("decision_tie_reuses", "return d > tau", "return d >= tau"),
    ("decision_attention_not_advanced", "        t_cls = t_next\n", "\n"),
    ("decision_attention_summed_over_heads", "(out, p0 / heads)", "(out, p0)"),
    ("decision_attention_from_reference", "t_next[f] = p_c", "t_next[f] = p_r"),
    ("decision_attention_starts_at_zero", "np.full((F, N), 1.0 / N)", "np.zeros((F, N))"),
    ("decision_attention_of_last_query", "p0 += pr[0]", "p0 += pr[-1]"),
    ("reorder_min_similarity", "s = np.maximum(c_past, c_fut)", "s = np.minimum(c_past, c_fut)"),
    ("reorder_tie_to_future", "from_fut = c_fut > c_past", "from_fut = c_fut >= c_past"),
    ("reorder_index_order", "for f in processing_order(F, G):", "for f in range(F):"),
    ("reorder_b1_skips_b2", "t, past, fut = 3, a0, a0 + 2", "t, past, fut = 3, a0, a0 + 4"),
    ("reorder_p_from_group_start", "return 1, f - 4, None", "return 1, f - p, None"),
    ("reorder_b2_past_only", "t, past, fut = 2, a0, a0 + 4", "t, past, fut = 2, a0, None"),
    ("reorder_kv_from_past", "k_t[R], v_t[R] = k_eff[src, R], v_eff[src, R]",
     "k_t[R], v_t[R] = k_eff[past, R], v_eff[past, R]"),
    ("reorder_output_from_past", "y[f, R] = y[src, R]", "y[f, R] = y[past, R]"),
    ("reorder_type_cue_p", "dv = decision_values(s, t_cls[f, 1:], ftype, P)",
     "dv = decision_values(s, t_cls[f, 1:], 1, P)"),
    ("reorder_restore_from_past", "x[f, R] - x[src, R]", "x[f, R] - x[past, R]"),
    ("reorder_anchor_after_b", "            put(a0 + 4)\n", ""),
]


def _mutant_module(orig, new):
    src = open(SRC).read()
    assert src.count(orig) >= 1, f"mutation anchor not found: {orig!r}"
    mod = types.ModuleType("reusevit_mutant")
    exec(compile(src.replace(orig, new), SRC + " (mutant)", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name,orig,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(name, orig, new):
    mod = _mutant_module(orig, new)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception as e:   # an assertion or a crash both count as caught
            caught.append((pin.__name__, type(e).__name__))
    assert caught, f"no pin caught the planted mistake {name!r}"

"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pins catch every one of them."""
import importlib.util
import inspect
import types

import pytest

import oracle.spec_oracle as real
from tests.oracle_pins import ALL_PINS

MUTANTS = {
    "dropped_retrieval_scale": ("out[h] = (K_r[:L, h, :] @ q_r[h]) * scale", "out[h] = (K_r[:L, h, :] @ q_r[h])"),
    "softmax_not_normalised": ("return e / e.sum(axis=1, keepdims=True)", "return e"),
    "softmax_wrong_axis": ("return e / e.sum(axis=1, keepdims=True)", "return e / e.sum(axis=0, keepdims=True)"),
    "max_over_heads": ("return np.asarray(p, dtype=np.float64).sum(axis=0)", "return np.asarray(p, dtype=np.float64).max(axis=0)"),
    "ties_to_higher_index": ("order = np.lexsort((t, -score))", "order = np.lexsort((-t, -score))"),
    "smallest_k": ("order = np.lexsort((t, -score))", "order = np.lexsort((t, score))"),
    "gqa_modulo_mapping": ("        g = h // G\n        s = ", "        g = h % H_kv\n        s = "),
    "v_from_head0": ("out[h] = (w / z) @ Vs[:, g, :]", "out[h] = (w / z) @ Vs[:, 0, :]"),
    "attn_scale_over_d": ("scale = 1.0 / math.sqrt(d)\n    idx", "scale = 1.0 / d\n    idx"),
    "lse_missing_max": ("lse[h] = m + math.log(z)", "lse[h] = math.log(z)"),
    "gather_off_by_one": ("Ks = np.asarray(K[idx], dtype=np.float64)", "Ks = np.asarray(K[idx - 1], dtype=np.float64)"),
    "elastic_reverse_pairing": ("loads = list(zip(free[:len(d_in)], d_in))", "loads = list(zip(free[::-1][:len(d_in)], d_in))"),
    "elastic_keeps_stale": ("free = [i for i, t in enumerate(slot_tok.tolist()) if t < 0 or t not in now]", "free = [i for i, t in enumerate(slot_tok.tolist()) if t < 0]"),
    "group_mean_not_max": ("return np.stack([p[g * per:(g + 1) * per].max(axis=0)", "return np.stack([p[g * per:(g + 1) * per].mean(axis=0)"),
    "accept_no_band_low": ("if np.any(inset & (score < s_k - band)):", "if False:"),
    "bf16_wrong_shift": ("<< np.uint32(16)", "<< np.uint32(15)"),
    "head_level_sum_not_max": ("return group_max_scores(head_softmax(retrieval_logits(q_r, K_r, L, scale)), n_sets)",
                               "return group_max_scores(head_softmax(retrieval_logits(q_r, K_r, L, scale)), 1)[[0] * n_sets]"),
    "sets_all_use_first": ("                                     idx_sets[g], scale)", "                                     idx_sets[0], scale)"),
    "yarn_no_division": ("theta_s = (1.0 - gamma) * theta / scale + gamma * theta", "theta_s = theta"),
    "yarn_ramp_reversed": ("theta_s = (1.0 - gamma) * theta / scale + gamma * theta", "theta_s = gamma * theta / scale + (1.0 - gamma) * theta"),
    "yarn_no_magnitude": ("return theta_s, 0.1 * math.log(scale) + 1.0", "return theta_s, 1.0"),
    "rope_exponent_over_d": ("theta = base ** (-2.0 * i / d_r)", "theta = base ** (-1.0 * i / d_r)"),
    "rope_rotation_sign": ("return m * np.concatenate([x * c - y * s_, x * s_ + y * c], axis=-1)", "return m * np.concatenate([x * c + y * s_, -x * s_ + y * c], axis=-1)"),
    "qk_swapped": ("k = (np.asarray(w_k, dtype=np.float64) @ x).reshape(H_r, -1)", "k = (np.asarray(w_q, dtype=np.float64) @ x).reshape(H_r, -1)"),
    "mla_uk_not_transposed": ("k_nope = cs @ np.asarray(w_uk[h], dtype=np.float64).T",
                              "k_nope = cs @ np.asarray(w_uk[h], dtype=np.float64)"),
    "mla_no_rope_term": ("s = (k_nope @ q_nope[h] + krs @ q_rope[h]) * scale",
                         "s = (k_nope @ q_nope[h]) * scale"),
    "mla_values_are_latents": ("v = cs @ np.asarray(w_uv[h], dtype=np.float64).T", "v = cs"),
    "mla_uv_head0": ("v = cs @ np.asarray(w_uv[h], dtype=np.float64).T",
                     "v = cs @ np.asarray(w_uv[0], dtype=np.float64).T"),
    "mla_scale_over_latent": ("scale = 1.0 / math.sqrt(d_nope + d_rope)",
                              "scale = 1.0 / math.sqrt(c.shape[1])"),
    "mla_all_tokens": ("cs = np.asarray(c[idx], dtype=np.float64)",
                       "cs = np.asarray(c[:len(idx)], dtype=np.float64)"),
    "dense_one_row_too_many": ("return sparse_gqa_attention(q, K, V, np.arange(L), scale)",
                               "return sparse_gqa_attention(q, K, V, np.arange(L + 1), scale)"),
    "dense_default_scale_only": ("return sparse_gqa_attention(q, K, V, np.arange(L), scale)",
                                 "return sparse_gqa_attention(q, K, V, np.arange(L))"),
    "decode_retrieval_at_llm_scale": ("s = retrieval_scores(q_r[b], K_r[b], L, scale_r)",
                                      "s = retrieval_scores(q_r[b], K_r[b], L, scale)"),
    "decode_attention_at_retrieval_scale": ("V_layers[layer][b], idx, scale)",
                                            "V_layers[layer][b], idx, scale_r)"),
    "decode_query_of_layer0": ("o, l_ = sparse_gqa_attention(q[layer][b], K_layers[layer][b],",
                               "o, l_ = sparse_gqa_attention(q[0][b], K_layers[layer][b],"),
    "decode_kv_of_sequence0": ("o, l_ = sparse_gqa_attention(q[layer][b], K_layers[layer][b],",
                               "o, l_ = sparse_gqa_attention(q[layer][b], K_layers[layer][0],"),
    "decode_budget_of_sequence0": ("idx = topk_indices(s, int(ks[b]))",
                                   "idx = topk_indices(s, int(ks[0]))"),
    "decode_values_of_layer0": ("V_layers[layer][b], idx, scale)",
                                "V_layers[0][b], idx, scale)"),
    "sets_wrong_kv_head": ("o, l_ = sparse_gqa_attention(q[g * G:(g + 1) * G], K[:, g:g + 1], V[:, g:g + 1],",
                           "o, l_ = sparse_gqa_attention(q[g * G:(g + 1) * G], K[:, 0:1], V[:, g:g + 1],"),
}


def _mutant(old, new):
    src = inspect.getsource(real)
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    mod = _mutant(*MUTANTS[name])
    caught = []
    for pin in ALL_PINS:
        try:
            pin(mod)
        except Exception:  # AssertionError, or a crash the mistake causes
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {name}"

"""The pins would catch plausible mistakes in the oracle: each case below plants one mistake in a copy of
oracle.c (a dropped term, a wrong index, a wrong tie rule, a transposed operand, ...), builds it with gcc, and
requires at least one pin of the matching group to fail on it.  Runs on the CPU only."""
import os

import pytest

import oracle
import pins

ATTN, ACC, COM, ENT, VIS, SMP, PRE = "attn", "accept", "commit", "entropy", "visual", "sampled", "prefill"
MUTANTS = [
    ("drop_scale", ATTN, "score[s] = scale * dot;", "score[s] = dot;"),
    ("wrong_kv_head", ATTN, "const int g = h / G;", "const int g = h % Hkv;"),
    ("self_not_visible", ATTN, "for (int j = i; j >= 0; j = parent[j]) visible[j] = 1;",
     "for (int j = parent[i]; j >= 0; j = parent[j]) visible[j] = 1;"),
    ("whole_tree_visible", ATTN, "for (int j = i; j >= 0; j = parent[j]) visible[j] = 1;",
     "for (int j = 0; j < T; ++j) visible[j] = 1;"),
    ("last_slot_dropped", ATTN, "const int n = L + T;", "const int n = L + T - 1;"),
    ("values_shifted", ATTN, "out_row[d] += p * (double)vb[(size_t)s * D + d];",
     "out_row[d] += p * (double)vb[(size_t)(s + 1) * D + d];"),
    ("keys_as_values", ATTN, "out_row[d] += p * (double)vb[(size_t)s * D + d];",
     "out_row[d] += p * (double)kb[(size_t)s * D + d];"),
    ("lse_without_max", ATTN, "*lse_out = m + log(l);", "*lse_out = log(l);"),
    ("no_normalisation", ATTN, "for (int d = 0; d < D; ++d) out_row[d] /= l;", ""),
    ("mask_bit_index", ATTN, "(mask_row[j / 64] >> (j % 64))", "(mask_row[j / 64] >> (j % 63))"),
    ("query_row_of_root", ATTN, "const float* qi = q + (((size_t)b * Hq + h) * T + i) * D;",
     "const float* qi = q + (((size_t)b * Hq + h) * T) * D;"),
    ("argmax_ties_high", ACC, "if (row[x] > row[best]) best = x;", "if (row[x] >= row[best]) best = x;"),
    ("own_argmax", ACC, "ok[i] = ok[par[i]] && tok[i] == am[par[i]];", "ok[i] = ok[par[i]] && tok[i] == am[i];"),
    ("ok_ignores_parent", ACC, "ok[i] = ok[par[i]] && tok[i] == am[par[i]];", "ok[i] = tok[i] == am[par[i]];"),
    ("last_ties_high", ACC, "if (ok[i] && depth[i] > depth[last]) last = i;",
     "if (ok[i] && depth[i] >= depth[last]) last = i;"),
    ("bonus_from_parent", ACC, "next_token[b] = am[last];", "next_token[b] = am[par[last] < 0 ? 0 : par[last]];"),
    ("accept_len_counts_bonus", ACC, "accept_len[b] = a;", "accept_len[b] = a + 1;"),
    ("kv_len_without_root", COM, "kv_len_out[b] = kv_len_in[b] + accept_len[b] + 1;",
     "kv_len_out[b] = kv_len_in[b] + accept_len[b];"),
    ("commit_reversed", COM, "for (int k = 0; k <= accept_len[b]; ++k) {",
     "for (int k = accept_len[b]; k >= 0; --k) {"),
    ("commit_skips_v", COM, "memmove(vc + (size_t)(L + k) * row, vc + (size_t)(L + path[k]) * row, row);", ""),
    ("commit_drops_last", COM, "for (int k = 0; k <= accept_len[b]; ++k) {",
     "for (int k = 0; k < accept_len[b]; ++k) {"),
    ("importance_no_row_norm", VIS, "if (s < L) imp[j] += exp(score[s] - m) / l;", "if (s < L) imp[j] += exp(score[s] - m);"),
    ("importance_mean_over_heads_only", VIS, "for (int j = 0; j < vis_count; ++j) imp[j] /= (double)Hq * T;",
     "for (int j = 0; j < vis_count; ++j) imp[j] /= (double)Hq;"),
    ("importance_offset_ignored", VIS, "const int s = vis_begin + j;", "const int s = j;"),
    ("importance_past_prefix", VIS, "if (s < L) imp[j] += exp(score[s] - m) / l;",
     "if (s < n && (s < L || visible[s - L])) imp[j] += exp(score[s] - m) / l;"),
    ("topk_ties_high", VIS, "if (!taken[j] && (best < 0 || v[j] > v[best])) best = j;",
     "if (!taken[j] && (best < 0 || v[j] >= v[best])) best = j;"),
    ("topk_smallest", VIS, "if (!taken[j] && (best < 0 || v[j] > v[best])) best = j;",
     "if (!taken[j] && (best < 0 || v[j] < v[best])) best = j;"),
    ("gather_without_offset", VIS, "const size_t src = (((size_t)b * Hkv + g) * S_cap + vis_begin + keep[(size_t)b * r + m]) * row;",
     "const size_t src = (((size_t)b * Hkv + g) * S_cap + keep[(size_t)b * r + m]) * row;"),
    ("entropy_log2", ENT, "if (p > 0.0) H -= p * log(p);", "if (p > 0.0) H -= p * log2(p);"),
    ("entropy_unnormalised", ENT, "const double p = exp(score[s] - m) / l;", "const double p = exp(score[s] - m);"),
    ("entropy_sign", ENT, "if (p > 0.0) H -= p * log(p);", "if (p > 0.0) H += p * log(p);"),
    ("entropy_without_scale", ENT, "    score[s] = scale * dot;\n    if (score[s] > m) m = score[s];\n  }\n  if (m == -INFINITY) return 0.0;",
     "    score[s] = dot;\n    if (score[s] > m) m = score[s];\n  }\n  if (m == -INFINITY) return 0.0;"),
    ("entropy_self_hidden", ENT, "  visible_nodes(parent ? parent + (size_t)b * T : NULL,\n                tree_mask ? tree_mask + ((size_t)b * T + i) * W : NULL, T, i, visible);\n  const int n = L + T;\n  double m = -INFINITY;\n  for (int s = 0; s < n; ++s) {\n    if (s >= L && !visible[s - L]) continue;\n    double dot = 0.0;\n    for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)kb[(size_t)s * D + d];\n    score[s] = scale * dot;\n    if (score[s] > m) m = score[s];\n  }\n  if (m == -INFINITY) return 0.0;",
     "  visible_nodes(parent ? parent + (size_t)b * T : NULL,\n                tree_mask ? tree_mask + ((size_t)b * T + i) * W : NULL, T, i, visible);\n  visible[i] = 0;\n  const int n = L + T;\n  double m = -INFINITY;\n  for (int s = 0; s < n; ++s) {\n    if (s >= L && !visible[s - L]) continue;\n    double dot = 0.0;\n    for (int d = 0; d < D; ++d) dot += (double)qi[d] * (double)kb[(size_t)s * D + d];\n    score[s] = scale * dot;\n    if (score[s] > m) m = score[s];\n  }\n  if (m == -INFINITY) return 0.0;"),
    ("prefill_causal_strict", PRE, "  for (int s = 0; s <= i; ++s) {\n    double dot = 0.0;",
     "  for (int s = 0; s < i; ++s) {\n    double dot = 0.0;"),
    ("prefill_wrong_kv_head", PRE, "const int g = h / (Hq / Hkv);", "const int g = h % Hkv;"),
    ("prefill_query_row_zero", PRE, "const float* qi = q + (((size_t)b * Hq + h) * N + i) * D;",
     "const float* qi = q + (((size_t)b * Hq + h) * N) * D;"),
    ("prefill_lse_without_max", PRE, "if (lse) lse[row] = m + log(l);", "if (lse) lse[row] = log(l);"),
    ("prefill_entropy_unnormalised", PRE, "const double p = exp(score[s] - m) / l;   /* A[h,i,s] */",
     "const double p = exp(score[s] - m);   /* A[h,i,s] */"),
    ("prefill_norm_capacity", PRE, "imp[j] /= (double)Hq * n;", "imp[j] /= (double)Hq * N;"),
    ("prefill_norm_rows_only", PRE, "imp[j] /= (double)Hq * n;", "imp[j] /= (double)n;"),
    ("prefill_padding_rows_counted", PRE, "      for (int i = 0; i < n; ++i) {\n        const double m = prefill_scores",
     "      for (int i = 0; i < N; ++i) {\n        const double m = prefill_scores"),
    ("prefill_window_offset_ignored", PRE, "const int slot = vis_begin + j;", "const int slot = j;"),
    ("prefill_diagonal_dropped", PRE, "if (slot <= i) imp[j]", "if (slot < i) imp[j]"),
    ("sampled_ratio_inverted", SMP, "if ((double)u[c] * q[x] < r[x]) {", "if ((double)u[c] * r[x] < q[x]) {"),
    ("sampled_residual_unclamped", SMP, "r[y] = (r[y] > q[y] ? r[y] - q[y] : 0.0) / z;", "r[y] = (r[y] - q[y]) / z;"),
    ("sampled_residual_not_updated", SMP, "r[y] = (r[y] > q[y] ? r[y] - q[y] : 0.0) / z;", "r[y] = r[y];"),
    ("sampled_residual_not_renormalised", SMP, "r[y] = (r[y] > q[y] ? r[y] - q[y] : 0.0) / z;",
     "r[y] = (r[y] > q[y] ? r[y] - q[y] : 0.0);"),
    ("sampled_final_from_target", SMP, "cum += r[x];", "cum += p[x];"),
    ("sampled_final_from_draft", SMP, "cum += r[x];", "cum += q[x];"),
    ("sampled_final_ge", SMP, "if (pick < 0 && cum > thr) pick = x;", "if (pick < 0 && cum >= thr) pick = x;"),
    ("sampled_target_row_of_root", SMP, "softmax_tau(target_logits + ((size_t)b * T + node) * V, V, tau, p);",
     "softmax_tau(target_logits + ((size_t)b * T) * V, V, tau, p);"),
    ("sampled_draft_row_of_root", SMP, "softmax_tau(draft_logits + ((size_t)b * T + node) * V, V, tau, q);",
     "softmax_tau(draft_logits + ((size_t)b * T) * V, V, tau, q);"),
    ("sampled_no_temperature", SMP, "out[x] = exp(((double)logits[x] - m) / tau);",
     "out[x] = exp((double)logits[x] - m);"),
    ("sampled_shared_uniform", SMP, "if ((double)u[c] * q[x] < r[x]) {", "if ((double)u[0] * q[x] < r[x]) {"),
    ("sampled_first_child_only", SMP, "      if (accepted < 0) break;\n      node = accepted;",
     "      if (accepted < 0) break;\n      if (depth > 0) break;\n      node = accepted;"),
    ("sampled_len_counts_bonus", SMP, "    accept_len[b] = depth;\n    next_token[b] = pick",
     "    accept_len[b] = depth + 1;\n    next_token[b] = pick"),
]
GROUPS = {ATTN: pins.ATTN_PINS, ACC: pins.ACCEPT_PINS, COM: pins.COMMIT_PINS, ENT: pins.ENTROPY_PINS,
          VIS: pins.VISUAL_PINS, SMP: pins.SAMPLED_PINS, PRE: pins.PREFILL_PINS}


@pytest.mark.parametrize("name,group,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, group, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) >= 1, "mutation site not found: %s" % name
    mutated = src.replace(old, new)
    path_c = os.path.join(tmp_path, "mutant.c")
    open(path_c, "w").write(mutated)
    lib = oracle.compile_source(path_c, os.path.join(tmp_path, "libmutant.so"))
    orc = oracle.Oracle(lib)
    caught = []
    for pin in GROUPS[group]:
        try:
            pin(orc)
        except (AssertionError, oracle.OracleError, ValueError, IndexError) as e:
            caught.append((pin.__name__, type(e).__name__))
    assert caught, "no pin caught mutant %s" % name


# The LM head's oracle is plain numpy (oracle/__init__.py); its planted mistakes replace the function itself.
def _decode(bits):
    import numpy as np
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _lm_swapped_operands(h, w):
    hh, ww = _decode(h), _decode(w)
    return ww @ hh.reshape(-1, hh.shape[-1]).T


def _lm_low_half_decode(h, w):
    import numpy as np
    dec = lambda b: (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)).view(np.float32).astype(np.float64)
    return dec(h) @ dec(w).T


def _lm_drops_last_k(h, w):
    hh, ww = _decode(h), _decode(w)
    return hh[..., :-1] @ ww[:, :-1].T


def _lm_extra_term(h, w):
    hh, ww = _decode(h), _decode(w)
    return hh @ ww.T + hh[..., :1]


@pytest.mark.parametrize("mutant", [_lm_swapped_operands, _lm_low_half_decode, _lm_drops_last_k, _lm_extra_term],
                         ids=lambda f: f.__name__)
def test_lm_head_pins_catch_planted_mistake(monkeypatch, mutant):
    monkeypatch.setattr(oracle, "lm_head_logits", mutant)
    orc = oracle.default()
    caught = []
    for pin in pins.LM_HEAD_PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError, IndexError) as e:
            caught.append((pin.__name__, type(e).__name__))
    assert caught, "no pin caught %s" % mutant.__name__


# The layer mean of prompt-row entropies is plain numpy too.
def _ae_all_rows(entropy, prompt_len):
    import numpy as np
    return float(np.asarray(entropy, np.float64).mean())


def _ae_mean_of_sequence_means(entropy, prompt_len):
    import numpy as np
    e = np.asarray(entropy, np.float64)
    return float(np.mean([e[b, :, :int(n)].mean() for b, n in enumerate(prompt_len)]))


@pytest.mark.parametrize("mutant", [_ae_all_rows, _ae_mean_of_sequence_means], ids=lambda f: f.__name__)
def test_prefill_entropy_mean_pins_catch_planted_mistake(monkeypatch, mutant):
    monkeypatch.setattr(oracle, "prefill_attn_entropy_mean", mutant)
    orc = oracle.default()
    caught = []
    for pin in pins.PREFILL_PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError, IndexError) as e:
            caught.append((pin.__name__, type(e).__name__))
    assert caught, "no pin caught %s" % mutant.__name__

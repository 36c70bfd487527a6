"""Planted mistakes in the oracle must be caught by its pins.

Each case rewrites one expression of an oracle module (a flipped sign, a
transposed operand, a dropped term, a changed comparison or selection rule),
loads the mutant, and checks that the named pin tests now fail. This shows
the pins constrain the oracle beyond restating it. CPU only."""
import importlib
import inspect
import json
import os
import types

import pytest

import oracle.decoder
import oracle.search
import tests.test_oracle_attention as tattn
import tests.test_oracle_decoder as tdec
import tests.test_oracle_margins as tmargin
import tests.test_oracle_search as tsearch


def _mutant(modname, old, new):
    mod = importlib.import_module(f"oracle.{modname}")
    src = inspect.getsource(mod)
    assert src.count(old) == 1, f"mutation anchor not unique in oracle.{modname}: {old}"
    m = types.ModuleType(f"oracle.{modname}")
    m.__dict__["__package__"] = "oracle"
    exec(compile(src.replace(old, new), f"<mutant oracle.{modname}>", "exec"), m.__dict__)
    return m


def _cases():
    with open(os.path.join(os.path.dirname(__file__), "golden", "scripted_beam_cases.json")) as f:
        return {c["name"]: c for c in json.load(f)["cases"]}


PINS = {
    "zero_weights": lambda: tdec.test_zero_weights_leave_only_eos_bias(9, 5, 1.0),
    "log_softmax": tdec.test_log_softmax_closed_forms,
    "orientation": tdec.test_recurrence_orientation_and_embedding_row,
    "proj_orientation": tdec.test_output_projection_orientation,
    "exhaustive": lambda: tsearch.test_exhaustive_beam_returns_every_complete_output_sorted(3, 4, 1, False),
    "greedy": lambda: tsearch.test_k1_is_greedy(0),
    "falls_off": lambda: tsearch.test_scripted_cases(_cases()["finalized_candidate_falls_off"]),
    "threshold_ref": lambda: tsearch.test_scripted_cases(_cases()["threshold_reference_is_terminated"]),
    "max_per_node": lambda: tsearch.test_scripted_cases(_cases()["max_candidates_per_node_and_maxlen"]),
    "noop": lambda: tsearch.test_scripted_cases(_cases()["noop_keeps_terminated_rank"]),
    "ties": lambda: tsearch.test_scripted_cases(_cases()["exact_ties_follow_rank_key"]),
    "fairseq": lambda: tsearch.test_scripted_cases(_cases()["fairseq_outputs_terminated_immediately"]),
    "fairseq_exhaustive": lambda: tsearch.test_fairseq_rule_exhaustive(3, 4, 1),
    "fig1": tsearch.test_fig1_schedule,
    "cap_schedule": tsearch.test_capacity_schedule,
    "cap_replay": lambda: tsearch.test_capacity_schedule_event_replay(0.25, 12),
    "stream_vs_batch": lambda: tsearch.test_var_stream_matches_var_batch(0, 4, 0.25),
    "attn_single": lambda: tattn.test_single_position_reads_its_value_row(0),
    "attn_uniform": lambda: tattn.test_uniform_scores_average_the_value_rows(0),
    "attn_two": lambda: tattn.test_two_positions_logistic_form(1),
    "attn_recurrence": tattn.test_recurrence_reads_h_not_the_attention_input,
    "margin_kth": tmargin.test_margin_kth_versus_next,
    "margin_adjacent": tmargin.test_margin_adjacent_ranks,
    "margin_noop": tmargin.test_margin_with_noop_and_two_parents,
    "margin_delta": tmargin.test_margin_threshold_boundary,
    "margin_delta_pruned": tmargin.test_margin_threshold_boundary_of_a_pruned_member,
    "margin_tie": tmargin.test_exact_tie_is_no_margin,
    "margin_fairseq": tmargin.test_fairseq_margin_window,
    "margin_search": tmargin.test_search_keeps_the_smallest_margin_of_an_input,
}

MUTATIONS = [
    ("eos_bias_sign", "decoder",
     "self.beta * (np.asarray(t, np.float64) - np.asarray(Lx, np.float64))",
     "self.beta * (np.asarray(Lx, np.float64) - np.asarray(t, np.float64))", ["zero_weights"]),
    ("bias_on_wrong_token", "decoder", "z[:, self.eos] +=", "z[:, 1] +=", ["zero_weights"]),
    ("transposed_recurrence", "decoder", "h_prev @ self.W_h.T", "h_prev @ self.W_h", ["orientation"]),
    ("dropped_embedding", "decoder", "h_prev @ self.W_h.T + self.E[np.asarray(y)]",
     "h_prev @ self.W_h.T", ["orientation"]),
    ("dropped_normalizer", "decoder", "return z - (m + np.log(s))", "return z - m",
     ["log_softmax", "zero_weights"]),
    ("reference_is_best_active", "beam", "ref = full[0][0]",
     "ref = next((e[0] for e in full if e[2] != NOOP_TOKEN), full[0][0])", ["threshold_ref"]),
    ("terminated_not_carried", "beam", "pool.append((c.score, j, NOOP_TOKEN))", "pass",
     ["noop", "exhaustive"]),
    ("max_per_node_ignored", "beam", "if per_parent.get(j, 0) >= M:", "if False:", ["max_per_node"]),
    ("maxlen_off_by_one", "beam", "elif t == max_len:", "elif t == max_len - 1:",
     ["max_per_node", "exhaustive"]),
    ("parent_rank_tiebreak_reversed", "beam", "return (-e[0], e[1], e[2])",
     "return (-e[0], -e[1], e[2])", ["ties"]),
    ("token_tiebreak_reversed", "beam", "return (-e[0], e[1], e[2])",
     "return (-e[0], e[1], -e[2])", ["ties"]),
    ("fairseq_outputs_beyond_full_beam", "beam", "for score, j, w in pool[:k]:",
     "for score, j, w in pool[:2 * k]:", ["fairseq"]),
    ("fairseq_beam_keeps_terminated", "beam", "        if terminated(w):\n            continue\n", "",
     ["fairseq", "fairseq_exhaustive"]),
    ("attn_scale_dropped", "decoder", "s = K[l] @ h / np.sqrt(self.d)", "s = K[l] @ h", ["attn_two"]),
    ("attn_keys_as_values", "decoder", "out += (w / np.sum(w)) @ V[l]", "out += (w / np.sum(w)) @ K[l]",
     ["attn_single", "attn_uniform"]),
    ("attn_layers_summed", "decoder", "return out / self.L", "return out", ["attn_single", "attn_two"]),
    ("attn_excludes_new_row", "decoder", "K, V = self.kv(st)", "K, V = self.kv((h[r], chain))",
     ["attn_single", "attn_two"]),
    ("attn_state_carries_x", "decoder", "new.append(st)", "new.append((x[r], st[1]))",
     ["attn_recurrence"]),
    ("attn_input_not_rounded", "decoder", "x[r] = bf16_round(h[r] + self.attention(h[r], K, V))",
     "x[r] = h[r] + self.attention(h[r], K, V)", ["attn_single"]),
    ("margin_only_kth_cut", "beam", "for a, b in zip(pool[:k], pool[1:k + 1]):",
     "for a, b in zip(pool[k - 1:k], pool[k:k + 1]):", ["margin_adjacent"]),
    ("margin_misses_kth_cut", "beam", "for a, b in zip(pool[:k], pool[1:k + 1]):",
     "for a, b in zip(pool[:k - 1], pool[1:k]):", ["margin_kth", "margin_noop"]),
    ("margin_counts_exact_ties", "beam", "for a, b in zip(pool[:k], pool[1:k + 1]):\n        if a[0] != b[0]:",
     "for a, b in zip(pool[:k], pool[1:k + 1]):\n        if True:", ["margin_tie"]),
    ("margin_drops_threshold_boundary", "beam", "margin = min(margin, abs(score - (ref - delta)))", "pass",
     ["margin_delta", "margin_delta_pruned"]),
    ("margin_skips_pruned_members", "beam",
     "            margin = min(margin, abs(score - (ref - delta)))\n            if score < ref - delta:\n"
     "                continue\n",
     "            if score < ref - delta:\n                continue\n"
     "            margin = min(margin, abs(score - (ref - delta)))\n", ["margin_delta_pruned"]),
    ("margin_boundary_without_abs", "beam", "margin = min(margin, abs(score - (ref - delta)))",
     "margin = min(margin, (ref - delta) - score)", ["margin_delta"]),
    ("fairseq_margin_window_short", "beam", "head = pool[:2 * k + 1]", "head = pool[:k + 1]", ["margin_fairseq"]),
    ("min_margin_keeps_last_step", "search",
     "res.min_margin[b.input] = min(res.min_margin[b.input], margin)", "res.min_margin[b.input] = margin",
     ["margin_search"]),
    ("refill_strict", "search", "len(live) <= eps * P", "len(live) < eps * P", ["fig1", "cap_schedule"]),
    ("refill_against_n", "search", "len(live) <= eps * P", "len(live) <= eps * n", ["cap_schedule"]),
    ("refill_to_n", "search", "m = min(P - len(live), N - c)", "m = min(n - len(live), N - c)",
     ["cap_schedule"]),
    ("capacity_longest_first", "search", "key=lambda b: (b.steps, b.input)",
     "key=lambda b: (-b.steps, b.input)", ["cap_schedule"]),
    ("capacity_ties_reversed", "search", "key=lambda b: (b.steps, b.input)",
     "key=lambda b: (b.steps, -b.input)", ["cap_schedule"]),
    ("capacity_limit_of_pool", "search", "if used + width > n * k:", "if used + width > P * k:",
     ["cap_schedule"]),
    ("capacity_skips_instead_of_stopping", "search", "                    break\n                sel.append(b)",
     "                    continue\n                sel.append(b)", ["cap_replay"]),
    ("expand_all_live", "search", "sel = [b for b in live if b.steps == lmin]", "sel = list(live)", ["fig1"]),
    ("bias_uses_global_timestep", "search", "t = np.array([sel[bi].steps + 1 for bi, _ in rows])",
     "t = np.array([res.timesteps + 1 for bi, _ in rows])", ["stream_vs_batch", "greedy"]),
]


@pytest.mark.parametrize("name,modname,old,new,pins", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, modname, old, new, pins):
    mut = _mutant(modname, old, new)
    if modname == "decoder":
        for target in (oracle.decoder, tdec, tsearch, tattn):
            for attr in ("ElmanDecoder", "AttnDecoder", "log_softmax", "decoder_for_workload"):
                if hasattr(target, attr):
                    monkeypatch.setattr(target, attr, getattr(mut, attr))
    elif modname == "beam":
        for target in (oracle.search, tmargin):
            monkeypatch.setattr(target, "beam_step", mut.beam_step)
            monkeypatch.setattr(target, "beam_step_fairseq", mut.beam_step_fairseq)
    else:
        for attr in ("decode", "decode_workload"):
            monkeypatch.setattr(tsearch, attr, getattr(mut, attr))
        monkeypatch.setattr(tmargin, "decode", mut.decode)
    for pin in pins:
        with pytest.raises(Exception):
            PINS[pin]()

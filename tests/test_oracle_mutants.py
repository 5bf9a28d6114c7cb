"""Plant plausible mistakes in copies of the oracle; the pins must catch each.

Every mutant below changes one line of ``oracle/ckv_oracle.c`` (a dropped
term, a wrong sign or index, a swapped operand) and is compiled into its own
library in a temporary directory.  A mutant that passes every pin would mean
the pins cannot tell that mistake from the method, so the test fails.  The
mutations are chosen to stay in bounds (they run in this process).
"""
import os
import tempfile

import pytest

import oracle
import oracle_pins

MUTANTS = {
    "drop_scale": ("double s = sc * dot;", "double s = dot;"),
    "sum_not_max": ("if (s > best) best = s;", "best = (g == 0) ? s : best + s;"),
    "min_not_max": ("if (s > best) best = s;", "if (g == 0 || s < best) best = s;"),
    "ascending_scores": ("if (si > sj) return -1;\n  if (si < sj) return 1;",
                         "if (si < sj) return -1;\n  if (si > sj) return 1;"),
    "ties_high_first": ("double si = g_sort_scores[i], sj = g_sort_scores[j];\n"
                        "  if (si > sj) return -1;\n  if (si < sj) return 1;\n"
                        "  return (i > j) - (i < j);",
                        "double si = g_sort_scores[i], sj = g_sort_scores[j];\n"
                        "  if (si > sj) return -1;\n  if (si < sj) return 1;\n"
                        "  return (i < j) - (i > j);"),
    "no_position_order": ("qsort(order, (size_t)m, sizeof(int32_t), by_position);", ""),
    "budget_off_by_one": ("int m = n < k ? n : k;", "int m = n < k ? n : k - 1;"),
    "no_max_shift": ("logit[i] = exp(logit[i] - mx);", "logit[i] = exp(logit[i]);"),
    "unnormalised": ("double w = logit[i] / z;", "double w = logit[i];"),
    "attn_head0_query": ("dot += ckvref_bf16_to_f64(q[g * d + c]) *\n"
                         "               ckvref_bf16_to_f64(k_rows",
                         "dot += ckvref_bf16_to_f64(q[c]) *\n"
                         "               ckvref_bf16_to_f64(k_rows"),
    "attn_v_from_k": ("o[c] += w * ckvref_bf16_to_f64(v_rows[(int64_t)i * d + c]);",
                      "o[c] += w * ckvref_bf16_to_f64(k_rows[(int64_t)i * d + c]);"),
    "attn_drop_scale": ("logit[i] = sc * dot;", "logit[i] = dot;"),
    "group_offset": ("const int64_t qoff = ((int64_t)b * s->num_q_heads + (int64_t)h * G) * d;",
                     "const int64_t qoff = ((int64_t)b * s->num_q_heads + (int64_t)h) * d;"),
    "no_tail_fill": ("for (int j = n; j < nmax; ++j) S[j] = -INFINITY;", ""),
    "gather_no_unit_base": ("k_src + base + row * s->kv_row_stride, sizeof(uint16_t) * d);",
                            "k_src + row * s->kv_row_stride, sizeof(uint16_t) * d);"),
    "bf16_shift": ("uint32_t u = (uint32_t)bits << 16;", "uint32_t u = (uint32_t)bits << 15;"),
    "select_with_att_query": ("ckvref_unit_scores(G, d, n, jb->q2 + qoff,",
                              "ckvref_unit_scores(G, d, n, jb->q + qoff,"),
    "landmark_sum_not_mean": ("ckvref_f64_to_bf16(sum / (j1 - j0));",
                              "ckvref_f64_to_bf16(sum);"),
    "landmark_drop_partial_chunk": ("const int nc = (n + chunk - 1) / chunk;",
                                    "const int nc = n / chunk;"),
    "bf16_ties_away": ("ldexp(nearbyint(ldexp(a, -q)), q);", "ldexp(round(ldexp(a, -q)), q);"),
    "bf16_truncate": ("ldexp(nearbyint(ldexp(a, -q)), q);", "ldexp(trunc(ldexp(a, -q)), q);"),
    "expand_no_chunk_scale": ("const int row = chunk_idx[i] * chunk + t;",
                              "const int row = chunk_idx[i] + t;"),
    "expand_past_context": ("if (row < n && r < k) rows[r++] = row;",
                            "if (r < k) rows[r++] = row;"),
    "chunk_lens_floor": ("clens[b] = (clamp_len(ctx_lens[b], s->max_ctx) + chunk - 1) / chunk;",
                         "clens[b] = clamp_len(ctx_lens[b], s->max_ctx) / chunk;"),
    "dual_cur_sees_spec": ("ckvref_unit_attn(G, d, m + 1, jb->q + qoff, kr, vr, jb->scale, jb->out + qoff, NULL);",
                           "ckvref_unit_attn(G, d, m + 2, jb->q + qoff, kr, vr, jb->scale, jb->out + qoff, NULL);"),
    "dual_spec_blind_to_itself": ("ckvref_unit_attn(G, d, m + 2, jb->q2 + qoff,",
                                  "ckvref_unit_attn(G, d, m + 1, jb->q2 + qoff,"),
    "dual_spec_with_cur_query": ("ckvref_unit_attn(G, d, m + 2, jb->q2 + qoff,",
                                 "ckvref_unit_attn(G, d, m + 2, jb->q + qoff,"),
    "recon_transposed_w": ("ckvref_bf16_to_f64(W[(int64_t)j * d + c]);",
                           "ckvref_bf16_to_f64(W[(int64_t)c * rank + j]);"),
    "recon_drop_last_rank": ("for (int j = 0; j < rank; ++j)\n          acc +=",
                             "for (int j = 0; j < rank - 1; ++j)\n          acc +="),
    "recon_slot_not_row": ("const uint16_t* U = u_fac + ((int64_t)u * s->max_ctx + idx[(int64_t)u * k + i]) * rank;",
                           "const uint16_t* U = u_fac + ((int64_t)u * s->max_ctx + i) * rank;"),
    "scores_skip_last_channel": ("for (int c = 0; c < d; ++c)\n        dot += ckvref_bf16_to_f64(q[g * d + c]) * ckvref_bf16_to_f64(kr[c]);",
                                 "for (int c = 0; c < d - 1; ++c)\n        dot += ckvref_bf16_to_f64(q[g * d + c]) * ckvref_bf16_to_f64(kr[c]);"),
}


def _fast_pins():
    # the planted-key pin is the slow one; a subset of seeds suffices here
    out = []
    for p in oracle_pins.ALL_PINS:
        if p is oracle_pins.pin_select_planted:
            out.append(lambda orc: oracle_pins.pin_select_planted(orc, seeds=range(3)))
        else:
            out.append(p)
    return out


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/found"
    mutated = src.replace(old, new)
    csrc = tmp_path / f"m_{name}.c"
    csrc.write_text(mutated)
    lib = str(tmp_path / f"libm_{name}.so")
    oracle.build(str(csrc), lib)
    orc = oracle.Oracle(lib)
    caught = []
    for pin in _fast_pins():
        try:
            pin(orc)
        except AssertionError:
            caught.append(pin)
    assert caught, f"mutant {name} passed every pin"

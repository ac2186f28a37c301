"""Strength of the oracle pins: plant a plausible mistake in a copy of the
oracle source (on the CPU), rebuild it, and check that at least one pin in
test_oracle_pins.py fails against the planted copy."""
import ctypes
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as P

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTATIONS = {
    "offsets_shifted": ("off[v + 1] = off[v] + counts[v];",
                        "off[v + 1] = off[v] + counts[v + 1 < n ? v + 1 : v];"),
    "dedup_upper_bound": ("if (uni[mid] < ids[i]) lo = mid + 1;",
                          "if (uni[mid] <= ids[i]) lo = mid + 1;"),
    "gather_slot0_miss": ("if (slot >= 0 && slot < table_rows)",
                          "if (slot > 0 && slot < table_rows)"),
    "te_fp64_argument": ("float arg = fmaf(omega[j], dt, phi[j]);",
                         "double arg = (double)omega[j] * ((double)t_dst[v] - (double)t_e[e]) + phi[j];"),
    "te_wrong_segment": ("float dt = t_dst[v] - t_e[e];",
                         "float dt = t_dst[v > 0 ? v - 1 : 0] - t_e[e];"),
    "te_transposed_out": ("te[e * d_t + j] =", "te[(j * 0 + e) * d_t + (d_t - 1 - j)] ="),
    "occ_unstable": ("for (int64_t p = 0; p < n; ++p)\n    if (index[p] >= 0 && index[p] < num_rows) occ[cursor[",
                     "for (int64_t p = n - 1; p >= 0; --p)\n    if (index[p] >= 0 && index[p] < num_rows) occ[cursor["),
    "occ_offsets_shifted": ("occ_off[index[p] + 1] += 1;", "occ_off[index[p]] += 1;"),
    "index_add_drops_last": ("for (int64_t p = 0; p < n; ++p) {\n    if (index[p] < 0 || index[p] >= num_rows) continue;",
                             "for (int64_t p = 0; p < n - 1; ++p) {\n    if (index[p] < 0 || index[p] >= num_rows) continue;"),
    "scaled_rows_edge_row": ("scal[e * H + h] * src[v * D + h * dh + j];",
                             "scal[e * H + h] * src[(v > 0 ? v - 1 : 0) * D + h * dh + j];"),
    "scaled_rows_head_swap": ("dst[(int64_t)index[e] * D + h * dh + j] += scal[e * H + h]",
                              "dst[(int64_t)index[e] * D + h * dh + j] += scal[e * H + (H - 1 - h)]"),
    "sample_not_strict": ("if (ts[p] < root_t[i]) c += 1;", "if (ts[p] <= root_t[i]) c += 1;"),
    "sample_oldest_k": ("int64_t skip = c > k ? c - k : 0;", "int64_t skip = 0;"),
    "sample_k_minus_one": ("int64_t skip = c > k ? c - k : 0;", "int64_t skip = c > k - 1 ? c - k + 1 : 0;"),
    "sample_eid_for_nbr": ("src[e] = nbr[p];", "src[e] = eid[p];"),
    "count_repeats": ("if (i > 0 && b[i] == b[i - 1]) continue;", "if (0) continue;"),
    "count_skips_first": ("for (int64_t i = 0; i < n; ++i) {\n      if (i > 0 && b[i] == b[i - 1])",
                          "for (int64_t i = 1; i < n; ++i) {\n      if (i > 0 && b[i] == b[i - 1])"),
    "greedy_ties_to_nodes": ("else take_node = sv[i].f > se[j].f;", "else take_node = sv[i].f >= se[j].f;"),
    "greedy_ascending_rank": ("if (x->f != y->f) return x->f > y->f ? -1 : 1;",
                              "if (x->f != y->f) return x->f < y->f ? -1 : 1;"),
    "greedy_ties_desc_id": ("return (x->id > y->id) - (x->id < y->id);\n}\n\nstatic freq_id_t",
                            "return (x->id < y->id) - (x->id > y->id);\n}\n\nstatic freq_id_t"),
    "greedy_budget_off_by_one": ("while ((double)(i + j) < alpha * (double)(nv + ne)",
                                 "while ((double)(i + j) <= alpha * (double)(nv + ne)"),
    "tebwd_cos_for_sin": ("double dcos = -sin((double)arg);", "double dcos = -cos((double)arg);"),
    "tebwd_sign": ("double dcos = -sin((double)arg);", "double dcos = sin((double)arg);"),
    "tebwd_fp64_argument": ("double dcos = -sin((double)arg);",
                            "double dcos = -sin((double)omega[j] * ((double)t_dst[v] - (double)t_e[e]) + phi[j]);"),
    "tebwd_no_dt": ("domega[j] += dte[e * d_t + j] * dcos * (double)dt;",
                    "domega[j] += dte[e * d_t + j] * dcos;"),
    "tebwd_wrong_row": ("dphi[j] += dte[e * d_t + j] * dcos;",
                        "dphi[j] += dte[(e > 0 ? e - 1 : 0) * d_t + j] * dcos;"),
    "tebwd_column_swap": ("float arg = fmaf(omega[j], dt, phi[j]);\n        double dcos",
                          "float arg = fmaf(omega[d_t - 1 - j], dt, phi[j]);\n        double dcos"),
    "lrelu_swapped": ("alpha[e * H + h] = p > 0.0 ? p : slope * p;",
                      "alpha[e * H + h] = p > 0.0 ? slope * p : p;"),
    "no_max_shift": ("Z += exp(alpha[e * H + h] - m);", "Z += exp(alpha[e * H + h]);"),
    "no_normalise": ("alpha[e * H + h] = exp(alpha[e * H + h] - m) / Z;",
                     "alpha[e * H + h] = exp(alpha[e * H + h] - m);"),
    "lse_missing_log": ("m + log(Z)", "m + Z"),
    "agg_wrong_head": ("acc += alpha[e * H + h] * V[(e * H + h) * dh + i];",
                       "acc += alpha[e * H + h] * V[(e * H + (H - 1 - h)) * dh + i];"),
    "aggbwd_drop_alpha": ("dV[(e * H + h) * dh + i] = alpha[e * H + h] * dout[(v * H + h) * dh + i];",
                          "dV[(e * H + h) * dh + i] = dout[(v * H + h) * dh + i];"),
    "smbwd_drop_D": ("(dalpha[e * H + h] - D)", "(dalpha[e * H + h])"),
    "smbwd_branch_swapped": ("(p > 0.0 ? 1.0 : slope)", "(p > 0.0 ? slope : 1.0)"),
    "smbwd_drop_scale": ("* r * scale;", "* r;"),
    "smbwd_dK_uses_K": ("dK[(e * H + h) * dh + i] = g * Q[(v * H + h) * dh + i];",
                        "dK[(e * H + h) * dh + i] = g * K[(e * H + h) * dh + i];"),
}

PINS = [
    (P.test_offsets_vs_cumsum, dict(n=1000)),
    (P.test_offsets_vs_cumsum, dict(n=7)),
    (P.test_dedup_vs_numpy_unique, dict(case="random")),
    (P.test_dedup_vs_numpy_unique, dict(case="zipf")),
    (P.test_gather_identity_slots, dict(dtype=P.np.float32)),
    (P.test_gather_slot_map_and_miss_list, {}),
    (P.test_time_encode_zero_dt_and_segment_mapping, {}),
    (P.test_time_encode_closed_forms, {}),
    (P.test_time_encode_double_angle_columns, {}),
    (P.test_time_encode_fp32_difference, {}),
    (P.test_occurrence_csr_vs_numpy, {}),
    (P.test_index_add_rows_vs_numpy, {}),
    (P.test_index_add_scaled_rows_vs_numpy, {}),
    (P.test_bwd_scalars_are_the_per_edge_gradient_coefficients, {}),
    (P.test_indexed_attention_gradients_by_finite_differences, {}),
    (P.test_sample_recent_hand_example, {}),
    (P.test_sample_recent_vs_numpy, dict(k=3)),
    (P.test_access_count_hand_example, {}),
    (P.test_access_count_vs_numpy, {}),
    (P.test_greedy_hot_set_hand_example, {}),
    (P.test_greedy_hot_set_properties, dict(alpha=0.37)),
    (P.test_greedy_hot_set_properties, dict(alpha=0.1)),
    (P.test_time_encode_bwd_finite_differences, {}),
    (P.test_time_encode_bwd_pythagorean_with_the_forward, {}),
    (P.test_fwd_vs_torch_sdpa, {}),
    (P.test_fwd_vs_dense_masked_attention, dict(slope=0.2)),
    (P.test_softmax_invariants, {}),
    (P.test_huge_logits_stay_finite, {}),
    (P.test_bwd_vs_torch_autograd_sdpa, {}),
    (P.test_bwd_finite_differences_leaky, dict(slope=0.2)),
    (P.test_bwd_finite_differences_leaky, dict(slope=-0.3)),
    (P.test_softmax_bwd_vs_jacobian_matrix, {}),
    (P.test_aggregate_bwd_is_the_transpose, {}),
]


def _build_mutant(tmp_path, name):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new)
    c_path = tmp_path / f"{name}.c"
    c_path.write_text(mutated)
    so = tmp_path / f"lib{name}.so"
    hdr_dir = os.path.dirname(SRC)
    subprocess.run(["gcc", "-std=c11", "-O1", "-ffp-contract=off", "-fPIC", "-shared",
                    "-I", hdr_dir, "-o", str(so), str(c_path), "-lm"], check=True)
    L = ctypes.CDLL(str(so))
    for fn, (res, args) in oracle._SIGS.items():
        f = getattr(L, fn)
        f.restype = res
        f.argtypes = args
    return L


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(tmp_path, name):
    good = oracle.lib()
    mutant = _build_mutant(tmp_path, name)
    caught = []
    oracle._lib = mutant
    try:
        for fn, kw in PINS:
            try:
                with P.np.errstate(all="ignore"):
                    fn(**kw)
            except (AssertionError, ValueError, IndexError, FloatingPointError):
                caught.append(fn.__name__)
    finally:
        oracle._lib = good
    assert caught, f"no pin detects the planted mistake {name!r}"

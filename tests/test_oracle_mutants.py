"""The oracle's pins must be strong enough to catch plausible mistakes.

Each case plants one mistake in a copy of oracle.c (on the CPU, in a
temporary directory), builds it, points the oracle front end at the mutant
and runs the pins that should notice.  At least one must fail."""
import os
import subprocess

import numpy as np
import pytest

import oracle as O
import tests.test_oracle_pins as P

SRC = os.path.join(os.path.dirname(O.__file__), "oracle.c")

MUTANTS = {
    # GCN: self message dropped
    "gcn_no_self_term": (
        "for (int64_t j = 0; j < d_in; j++) a[j] += cs * or_load(H, h_dtype, v * d_in + j);",
        "(void)cs;",
        [lambda: P.test_gcn_matches_dense(0, True)]),
    # GCN: degree without the added self loop
    "gcn_degree_without_self_loop": (
        "double c = 1.0 / sqrt(((double)deg_out[u] + 1.0) * din_hat);",
        "double c = 1.0 / sqrt(((double)deg_out[u] + (deg_out[u] ? 0.0 : 1.0)) * din_hat);",
        [lambda: P.test_gcn_matches_dense(0, True), P.test_closed_form_gcn_degrees_only]),
    # GCN: in- and out-degree swapped in the source factor
    "gcn_degrees_swapped": (
        "double din_hat = (double)m + 1.0;",
        "double din_hat = (double)deg_out[v] + 1.0;",
        [lambda: P.test_gcn_matches_dense(1, False)]),
    # SAGE: mean over all in-neighbours instead of the propagated ones
    "sage_mean_over_full_degree": (
        "for (int64_t j = 0; j < d_in; j++) a[j] = a[j] / (double)m;",
        "for (int64_t j = 0; j < d_in; j++) a[j] = a[j] / (double)(in_off[v + 1] - in_off[v]);",
        [P.test_sampled_sage_matches_dense_on_kept_edges]),
    # SAGE: self and neighbour halves of W swapped
    "sage_halves_swapped": (
        "for (int64_t j = 0; j < d_in; j++) a[d_in + j] = or_load(H, h_dtype, v * d_in + j);",
        "for (int64_t j = 0; j < d_in; j++) { double t = a[j]; a[j] = or_load(H, h_dtype, v * d_in + j); a[d_in + j] = t; }",
        [lambda: P.test_sage_matches_dense(0, True)]),
    # bias dropped
    "no_bias": (
        "double z = bias ? bias[o] : 0.0;",
        "double z = 0.0;",
        [lambda: P.test_sage_matches_dense(1, False)]),
    # activation applied the wrong way round
    "relu_flipped": (
        "z += W[o * cols + j] * a[j];\n                if (relu && z < 0.0) z = 0.0;",
        "z += W[o * cols + j] * a[j];\n                if (relu && z > 0.0) z = 0.0;",
        [lambda: P.test_sage_matches_dense(0, True)]),
    # sampler keeps the largest keys
    "sampler_keeps_largest": (
        "int kept = j < keep;",
        "int kept = j >= d - keep;",
        [P.test_sampler_brute_force_and_invariants]),
    # sampler ignores the layer in the hash
    "sampler_ignores_layer": (
        "uint64_t args[3] = {(uint64_t)layer, (uint64_t)v, (uint64_t)u};",
        "uint64_t args[3] = {(uint64_t)1, (uint64_t)v, (uint64_t)u};",
        [P.test_sampler_brute_force_and_invariants, P.test_sampler_layers_differ]),
    # hash with the increment left out
    "hash_without_gamma": (
        "uint64_t h = or_mix64(seed + 0x9e3779b97f4a7c15ULL + tag);",
        "uint64_t h = or_mix64(seed + tag);",
        [lambda: P.test_oracle_hash_matches_published_splitmix64(P_GOLDEN)]),
    # CSR sorted by destination first
    "csr_sorted_by_destination": (
        "if (p->a != q->a) return p->a < q->a ? -1 : 1;\n    if (p->b != q->b) return p->b < q->b ? -1 : 1;",
        "if (p->b != q->b) return p->b < q->b ? -1 : 1;\n    if (p->a != q->a) return p->a < q->a ? -1 : 1;",
        [lambda: P.test_csr_brute_force(0)]),
    # BFS children appended in discovery order instead of (d_in desc, id asc)
    "bfs_children_unsorted": (
        "qsort(kids, (size_t)nk, sizeof(int32_t), or_rank_cmp);",
        "(void)0;",
        [P.test_reorder_tree_levels, lambda: P.test_reorder_random_graphs_are_valid_bfs_orders(0)]),
    # BFS over out-edges would need a different graph walk; a root-order slip instead:
    "bfs_roots_by_id": (
        "if (g_or_deg[a] != g_or_deg[b]) return g_or_deg[a] > g_or_deg[b] ? -1 : 1;",
        "if (0) return 0;",
        [P.test_reorder_star, P.test_reorder_path_and_two_components]),
    # total span without the self message
    "span_without_self": (
        "int64_t lo = pi[v], hi = pi[v];",
        "if (in_off[v + 1] == in_off[v]) continue;\n        int64_t lo = INT64_MAX, hi = INT64_MIN;",
        [P.test_total_span_hand_example, P.test_span_equals_sum_of_active_counts]),
    # Alg. 1: centre without the vertex's own position
    "ta_mu_without_self": (
        "double s = r_in[v];",
        "double s = 0.0;",
        [lambda: P.test_ta_updates_are_the_minimisers(0), P.test_ta_special_cases, lambda: P.test_ta_worked_example(P_GOLDEN)]),
    # Alg. 1: out-neighbour centres not weighted by 1/d
    "ta_r_unweighted": (
        "num += mu[v] / dv;",
        "num += mu[v] / d;",
        [lambda: P.test_ta_updates_are_the_minimisers(0)]),
    # Alg. 1: each update restarts from the ranks instead of carrying r
    "ta_resets_positions_to_ranks": (
        "rank[pos[k].v] = (double)k;\n        }",
        "rank[pos[k].v] = (double)k;\n        }\n        memcpy(r, rank, nn * sizeof(double));",
        [lambda: P.test_ta_worked_example(P_GOLDEN), lambda: P.test_ta_positions_follow_dense_operator(0)]),
    # Alg. 1: the loop runs on after the order has converged
    "ta_ignores_convergence": (
        "if (!changed) break;",
        "(void)changed;",
        [P.test_ta_special_cases, P.test_ta_stops_when_the_order_converges]),
    # Alg. 1: ArgSort breaks ties by the higher ID
    "ta_ties_by_higher_id": (
        "return (a->v > b->v) - (a->v < b->v);\n}\n\n/*\n * The dispersion",
        "return (a->v < b->v) - (a->v > b->v);\n}\n\n/*\n * The dispersion",
        [P.test_ta_special_cases]),
    # J without the 1/d(v) weight of each destination
    "dispersion_unweighted": (
        "total += q / d;",
        "total += q;",
        [lambda: P.test_dispersion_is_neighbourhood_variance(0)]),
    # J's centre without the vertex's own position
    "dispersion_centre_without_self": (
        "double s = x[v];",
        "double s = 0.0;",
        [lambda: P.test_dispersion_is_neighbourhood_variance(0), lambda: P.test_ta_worked_example(P_GOLDEN)]),
    # RCMK: Cuthill-McKee order not reversed
    "rcm_not_reversed": (
        "new_of_old[queue[i]] = (int32_t)(n - 1 - i);",
        "new_of_old[queue[i]] = (int32_t)i;",
        [P.test_rcm_matches_scipy, P.test_rcm_special_cases]),
    # RCMK: children by descending degree
    "rcm_children_by_degree_desc": (
        "if (g_or_sdeg[a] != g_or_sdeg[b]) return g_or_sdeg[a] < g_or_sdeg[b] ? -1 : 1;",
        "if (g_or_sdeg[a] != g_or_sdeg[b]) return g_or_sdeg[a] > g_or_sdeg[b] ? -1 : 1;",
        [P.test_rcm_matches_scipy, lambda: P.test_rcm_random_graphs_are_valid(0)]),
    # RCMK: a reciprocal pair counted twice in the symmetric degree
    "rcm_repeats_kept": (
        "if (a[i] != v && (m == 0 || a[i] != a[m - 1])) a[m++] = a[i];",
        "if (a[i] != v) a[m++] = a[i];",
        [P.test_rcm_special_cases, P.test_rcm_matches_scipy]),
    # residency: LRU ranked by admission instead of last use
    "residency_lru_by_admission": (
        "key = mark[v];",
        "key = adm[v];",
        [lambda: P.test_residency_hand_cases("case1")]),
    # residency: the self message not counted in pending
    "residency_no_self_message": (
        "pend[v] = (int64_t)m[v] + 1;",
        "pend[v] = (int64_t)m[v];",
        [lambda: P.test_residency_hand_cases("case1"), lambda: P.test_residency_invariants(0)]),
    # residency: FIFO keeps the first admission across reloads
    "residency_fifo_first_admission_only": (
        "adm[v] = (int32_t)k;\n            if (evicted[v])",
        "if (!evicted[v]) adm[v] = (int32_t)k;\n            if (evicted[v])",
        [P.test_residency_fifo_readmission]),
    # residency: most pending evicted first
    "residency_most_pending_first": (
        "key = pend[v];",
        "key = -pend[v];",
        [lambda: P.test_residency_hand_cases("case1"), P.test_fewest_pending_reloads_least]),
    # residency: pending counts capped at 14 bits
    "residency_pending_capped": (
        "key = pend[v];",
        "key = pend[v] < 16383 ? pend[v] : 16383;",
        [P.test_residency_fewest_pending_is_exact_above_16383]),
    # sampled GCN normalised by the full in-degree
    "gcn_sampled_full_in_degree": (
        "double din_hat = (double)m + 1.0;",
        "double din_hat = (double)(in_off[v + 1] - in_off[v]) + 1.0;",
        [P.test_sampled_gcn_matches_dense_on_kept_edges]),
    # GIN without its self term
    "gin_no_self_term": (
        "for (int64_t j = 0; j < d_in; j++) a[j] += or_load(H, h_dtype, v * d_in + j);\n            }",
        "(void)0;\n            }",
        [lambda: P.test_gin_matches_dense(False)]),
    # GIN with a perceptron: hidden ReLU dropped
    "gin_mlp_no_hidden_relu": (
        "t[h] = x > 0.0 ? x : 0.0;",
        "t[h] = x;",
        [lambda: P.test_gin_mlp_matches_dense(False)]),
    # GIN with a perceptron: the second layer's weight transposed
    "gin_mlp_w2_transposed": (
        "for (int64_t h = 0; h < d_h; h++) z += W2[o * d_h + h] * t[h];",
        "for (int64_t h = 0; h < d_h; h++) z += W2[h * d_out + o] * t[h];",
        [lambda: P.test_gin_mlp_matches_dense(False)]),
    # GAT without the self message in the softmax
    "gat_no_self_message": (
        "for (int64_t k = in_off[v] - 1; k < in_off[v + 1]; k++) {",
        "for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {",
        [lambda: P.test_gat_matches_dense(False, True), P.test_gat_special_cases]),
    # GAT: source and destination halves of a swapped
    "gat_attention_halves_swapped": (
        "s_src += attn[o] * z;\n            s_dst += attn[d_out + o] * z;",
        "s_src += attn[d_out + o] * z;\n            s_dst += attn[o] * z;",
        [lambda: P.test_gat_matches_dense(False, False)]),
    # GAT: LeakyReLU slope on the positive side
    "gat_leaky_relu_flipped": (
        "e = e > 0.0 ? e : slope * e;\n                double w = exp(e - m);",
        "e = e < 0.0 ? e : slope * e;\n                double w = exp(e - m);",
        [lambda: P.test_gat_matches_dense(False, True)]),
    # fp16 rounding truncates
    "f16_truncates": (
        "double r = nearbyint(q);\n    if (r >= 2048.0)",
        "double r = floor(q);\n    if (r >= 2048.0)",
        [P.test_round_store_matches_library_conversions]),
}

P_GOLDEN = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "tests", "golden")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, tmp_path):
    old, new, pins = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/found"
    path = tmp_path / "mutant.c"
    path.write_text(src.replace(old, new))
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-o", str(so), str(path), "-lm"])
    saved = O._lib
    O._lib = O.load(str(so))
    failures = 0
    try:
        for pin in pins:
            try:
                pin()
            except (AssertionError, ValueError, RuntimeError):
                failures += 1
    finally:
        O._lib = saved
    assert failures > 0, f"no pin noticed mutant {name}"

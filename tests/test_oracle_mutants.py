"""Plant plausible mistakes in copies of the oracle and check that the pins
catch every one (CPU only; the real oracle source is never modified)."""
import concurrent.futures as cf
import json
import os
import subprocess
import sys

import pytest

import oracle

# (name, original text, mutated text); each original must occur in oracle.c
MUTANTS = [
    ("propagate_swaps_src_dst",
     "return reduce_edges(x, N, F, src, dst, E, N, w, ea, msg, aggr, out, argmax, sabs, E);",
     "return reduce_edges(x, N, F, dst, src, E, N, w, ea, msg, aggr, out, argmax, sabs, E);"),
    ("sum_overwrites", "out[o] += m;", "out[o] = m;"),
    ("diff_wrong_sign", "m = (double)xj - (double)x[i * F + f];", "m = (double)xj + (double)x[i * F + f];"),
    ("diff_max_wrong_operand", "if (msg == ORACLE_MSG_DIFF) m = xj - x[i * F + f];",
     "if (msg == ORACLE_MSG_DIFF) m = xj - x[j * F + f];"),
    ("max_tie_takes_last", "m > best[o]", "m >= best[o]"),
    ("max_keeps_negative_zero", "if (m == 0.0f) m = 0.0f; /* -0.0 -> +0.0 */", ""),
    ("max_drops_weight", "else if (w) m = w[k] * xj;", "else if (w) m = xj;"),
    ("sum_drops_weight", "else if (w) m = (double)w[k] * (double)xj;", "else if (w) m = (double)xj;"),
    ("mean_not_divided", "out[o] = out[o] / (double)cnt[i];", ""),
    ("mean_divides_by_count_plus_one", "out[o] = out[o] / (double)cnt[i];", "out[o] = out[o] / (double)(cnt[i] + 1);"),
    ("empty_max_not_zero", "out[o] = cnt[i] > 0 ? (double)best[o] : 0.0;", "out[o] = (double)best[o] - (cnt[i] > 0 ? 0.0 : 1.0);"),
    ("sabs_signed", "if (sabs) sabs[o] += fabs(m);", "if (sabs) sabs[o] += m;"),
    ("gcn_degree_at_source", "d[dst[k]] += w ? w[k] : 1.0;", "d[src[k]] += w ? w[k] : 1.0;"),
    ("gcn_no_sqrt", "1.0 / sqrt(d[i])", "1.0 / d[i]"),
    ("gcn_drops_weight", "norm[k] = d[src[k]] * (w ? w[k] : 1.0) * d[dst[k]];", "norm[k] = d[src[k]] * d[dst[k]];"),
    ("gcn_one_sided", "norm[k] = d[src[k]] * (w ? w[k] : 1.0) * d[dst[k]];", "norm[k] = d[dst[k]] * (w ? w[k] : 1.0) * d[dst[k]];"),
    ("csr_perm_is_source", "perm[p] = k;", "perm[p] = src[k];"),
    ("csr_col_is_target", "col[p] = src[k];", "col[p] = dst[k];"),
    ("degree_counts_sources", "deg[i] = 0;\n    for (int64_t k = 0; k < E; ++k) deg[dst[k]] += 1;",
     "deg[i] = 0;\n    for (int64_t k = 0; k < E; ++k) deg[edge_index[k]] += 1;"),
    ("pool_reads_first_node", "for (int64_t n = 0; n < N; ++n) node[n] = n;", "for (int64_t n = 0; n < N; ++n) node[n] = 0;"),
    ("pool_wrong_sentinel", "aggr, out, argmax, sabs, N);", "aggr, out, argmax, sabs, B);"),
    ("bwd_grad_to_target", "                grad_x[j * F + f] += wk * g;\n                if (sabs_x) sabs_x[j * F + f] += fabs(wk * g);\n                if (grad_w) {\n                    grad_w[k] += g * (double)x[j * F + f];\n                    if (sabs_w) sabs_w[k] += fabs(g * (double)x[j * F + f]);\n                }\n            }\n        }\n    }\n    free(deg);",
     "                grad_x[i * F + f] += wk * g;\n                if (sabs_x) sabs_x[j * F + f] += fabs(wk * g);\n                if (grad_w) {\n                    grad_w[k] += g * (double)x[j * F + f];\n                    if (sabs_w) sabs_w[k] += fabs(g * (double)x[j * F + f]);\n                }\n            }\n        }\n    }\n    free(deg);"),
    ("bwd_mean_not_scaled", "const double sc = aggr == ORACLE_MEAN ? 1.0 / (double)deg[i] : 1.0;", "const double sc = 1.0;"),
    ("bwd_grad_w_uses_target_x", "                    grad_w[k] += g * (double)x[j * F + f];\n                    if (sabs_w) sabs_w[k] += fabs(g * (double)x[j * F + f]);\n                }\n            }\n        }\n    }\n    free(deg);",
     "                    grad_w[k] += g * (double)x[i * F + f];\n                    if (sabs_w) sabs_w[k] += fabs(g * (double)x[j * F + f]);\n                }\n            }\n        }\n    }\n    free(deg);"),
    ("bwd_diff_drops_self_term", "                grad_x[j * F + f] += g;\n                grad_x[i * F + f] -= g;\n                if (sabs_x) {\n                    sabs_x[j * F + f] += fabs(g);\n                    sabs_x[i * F + f] += fabs(g);\n                }\n            } else {\n                grad_x[j * F + f] += wk * g;",
     "                grad_x[j * F + f] += g;\n                if (sabs_x) {\n                    sabs_x[j * F + f] += fabs(g);\n                    sabs_x[i * F + f] += fabs(g);\n                }\n            } else {\n                grad_x[j * F + f] += wk * g;"),
    ("bwd_max_ignores_weight", "                    const double wk = w ? (double)w[k] : 1.0;\n                    grad_x[j * F + f] += wk * g;", "                    const double wk = 1.0;\n                    grad_x[j * F + f] += wk * g;"),
    ("softmax_den_without_max", "den[dst[k] * H + h] += exp(s[k * H + h] - m[dst[k] * H + h]);",
     "den[dst[k] * H + h] += exp(s[k * H + h]);"),
    ("softmax_segment_by_source", "const int64_t *dst = edge_index + E;\n    if (check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;\n    for (int64_t t = 0; t < E * H; ++t)",
     "const int64_t *dst = edge_index;\n    if (check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;\n    for (int64_t t = 0; t < E * H; ++t)"),
    ("softmax_max_of_head0", "if (s[k * H + h] > m[dst[k] * H + h]) m[dst[k] * H + h] = s[k * H + h];",
     "if (s[k * H] > m[dst[k] * H + h]) m[dst[k] * H + h] = s[k * H];"),
    ("softmax_not_normalised", "alpha[k * H + h] = exp(s[k * H + h] - m[dst[k] * H + h]) / den[dst[k] * H + h];",
     "alpha[k * H + h] = exp(s[k * H + h] - m[dst[k] * H + h]);"),
    ("gat_slope_on_positive", "e[k * H + h] = v >= 0.0 ? v : (double)slope * v;", "e[k * H + h] = v >= 0.0 ? (double)slope * v : v;"),
    ("gat_scores_swap_ends", "(double)a_src[src[k] * H + h] + (double)a_dst[dst[k] * H + h];\n            e[k * H + h]",
     "(double)a_src[dst[k] * H + h] + (double)a_dst[src[k] * H + h];\n            e[k * H + h]"),
    ("softmax_bwd_sign", "grad_s[k * H + h] = a * ((double)g[k * H + h] - t[dst[k] * H + h]);",
     "grad_s[k * H + h] = a * ((double)g[k * H + h] + t[dst[k] * H + h]);"),
    ("softmax_bwd_t_without_alpha", "const double ag = (double)alpha[k * H + h] * (double)g[k * H + h];",
     "const double ag = (double)g[k * H + h];"),
    ("heads_weight_of_head0", "const double a = alpha[k * H + h];\n            for (int64_t c = 0; c < C; ++c) {\n                const double term",
     "const double a = alpha[k * H];\n            for (int64_t c = 0; c < C; ++c) {\n                const double term"),
    ("heads_bwd_grad_to_target", "grad_x[j * F + h * C + c] += a * gi;", "grad_x[i * F + h * C + c] += a * gi;"),
    ("heads_bwd_dot_uses_target_x", "dot += gi * (double)x[j * F + h * C + c];", "dot += gi * (double)x[i * F + h * C + c];"),
    ("transform_theta_transposed", "const double t = (double)x[n * Fi + k] * (double)theta[k * Fo + o];",
     "const double t = (double)x[n * Fi + k] * (double)theta[o * Fi + k];"),
    ("edge_add_ignores_edge", "else if (msg == ORACLE_MSG_EDGE_ADD) m = (double)xj + (double)ea[k * F + f];",
     "else if (msg == ORACLE_MSG_EDGE_ADD) m = (double)xj;"),
    ("edge_attr_by_source", "else if (msg == ORACLE_MSG_EDGE_MUL) m = (double)xj * (double)ea[k * F + f];",
     "else if (msg == ORACLE_MSG_EDGE_MUL) m = (double)xj * (double)ea[(j % E) * F + f];"),
    ("edge_relu_missing", "else if (msg == ORACLE_MSG_EDGE_RELU) m = fmax((double)xj + (double)ea[k * F + f], 0.0);",
     "else if (msg == ORACLE_MSG_EDGE_RELU) m = (double)xj + (double)ea[k * F + f];"),
    ("edge_max_relu_keeps_negative", "else if (msg == ORACLE_MSG_EDGE_RELU) m = xj + ea[k * F + f] > 0.0f ? xj + ea[k * F + f] : 0.0f;",
     "else if (msg == ORACLE_MSG_EDGE_RELU) m = xj + ea[k * F + f];"),
    ("gat_bwd_slope_on_positive", "const double gv = (double)g[k * H + h] * (v >= 0.0 ? 1.0 : (double)slope);",
     "const double gv = (double)g[k * H + h] * (v >= 0.0 ? (double)slope : 1.0);"),
    ("gat_bwd_dst_to_src", "            grad_dst[dst[k] * H + h] += gv;", "            grad_dst[src[k] * H + h] += gv;"),
    ("transform_skips_last_k", "for (int64_t k = 0; k < Fi; ++k) {\n                const double t",
     "for (int64_t k = 0; k + 1 < Fi; ++k) {\n                const double t"),
    ("edge_bwd_relu_gate_ignores_edge", "const double on = xj + e > 0.0 ? 1.0 : 0.0;",
     "const double on = xj > 0.0 ? 1.0 : 0.0;"),
    ("edge_bwd_mul_swaps_factors", "                dx = d * e;\n                de = d * xj;",
     "                dx = d * xj;\n                de = d * e;"),
    ("edge_bwd_mean_unscaled", "                if (aggr == ORACLE_MEAN) d /= (double)deg[i];", ""),
    ("edge_bwd_max_routes_everywhere", "d = a == k ? (double)grad_out[i * F + f] : 0.0;",
     "d = (double)grad_out[i * F + f];"),
    ("edge_bwd_grad_to_target", "                grad_x[j * F + f] += dx;", "                grad_x[i * F + f] += dx;"),
]


@pytest.fixture(scope="module")
def outcomes(tmp_path_factory):
    """Compile every mutant and run all pins against it in a fresh process
    (a mutant that corrupts memory only kills its own process, which also
    counts as caught)."""
    with open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")) as f:
        source = f.read()
    d = tmp_path_factory.mktemp("mutants")
    runner = os.path.join(os.path.dirname(os.path.abspath(__file__)), "mutant_runner.py")

    def one(m):
        name, orig, mut = m
        if source.count(orig) != 1:
            return name, None
        src = d / f"{name}.c"
        src.write_text(source.replace(orig, mut))
        libpath = oracle.build(str(src), str(d / f"lib{name}.so"))
        try:
            r = subprocess.run([sys.executable, runner, libpath], capture_output=True, text=True, timeout=300)
        except subprocess.TimeoutExpired:
            return name, ["<timeout>"]
        if r.returncode != 0:
            return name, [f"<exit {r.returncode}>"]
        return name, json.loads(r.stdout.strip().splitlines()[-1])

    with cf.ThreadPoolExecutor(4) as ex:
        return dict(ex.map(one, MUTANTS))


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_pins_catch_mutant(outcomes, name):
    caught = outcomes[name]
    assert caught is not None, f"mutation site for {name} is not unique in oracle.c"
    assert caught, f"no pin catches mutant {name}"

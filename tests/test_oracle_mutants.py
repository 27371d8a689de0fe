"""Plant plausible mistakes in copies of the oracle and check that the pins
catch every one (CPU only; the real oracle source is never modified)."""
import multiprocessing
import os

import pytest

import oracle
from tests.oracle_pins import ALL_PINS

# (name, original text, mutated text); each original must occur in oracle.c
MUTANTS = [
    ("propagate_swaps_src_dst",
     "const int64_t *src = edge_index;\n    const int64_t *dst = edge_index + E;\n    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;\n    if (!all_finite",
     "const int64_t *dst = edge_index;\n    const int64_t *src = edge_index + E;\n    if (check_index_range(src, E, N) || check_index_range(dst, E, N)) return ORACLE_ERR_INDEX;\n    if (!all_finite"),
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
    ("degree_counts_sources", "for (int64_t k = 0; k < E; ++k) deg[dst[k]] += 1;",
     "for (int64_t k = 0; k < E; ++k) deg[edge_index[k]] += 1;"),
    ("pool_reads_first_node", "for (int64_t n = 0; n < N; ++n) node[n] = n;", "for (int64_t n = 0; n < N; ++n) node[n] = 0;"),
    ("pool_wrong_sentinel", "aggr, out, argmax, sabs, N);", "aggr, out, argmax, sabs, B);"),
]


@pytest.fixture(scope="module")
def source():
    with open(os.path.join(os.path.dirname(oracle.__file__), "oracle.c")) as f:
        return f.read()


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, source, name, orig, mut):
    assert source.count(orig) == 1, f"mutation site for {name} not unique"
    src = tmp_path / f"{name}.c"
    src.write_text(source.replace(orig, mut))
    libpath = oracle.build(str(src), str(tmp_path / f"lib{name}.so"))
    # run the pins in a forked child so a mutant that corrupts memory cannot
    # take the test process down (a crash also counts as caught)
    ctx = multiprocessing.get_context("fork")
    recv, send = ctx.Pipe(duplex=False)
    proc = ctx.Process(target=_run_pins, args=(libpath, send))
    proc.start()
    proc.join(120)
    caught = recv.recv() if proc.exitcode == 0 and recv.poll() else ["<crashed>"]
    assert caught, f"no pin catches mutant {name}"


def _run_pins(libpath, send):
    lib = oracle.load(libpath)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    send.send(caught)

"""Parity of the narrow-window propagate: when the source rows are at least
two 128-byte windows wide and total 16 MB or more, the plain messages run
one launch per window and long rows are folded once after the last window.
Graphs just above that size, against the oracle: hub rows longer than a
chunk (pieces from every window folded together), light and heavy mean
degrees, ragged window counts (rows of 384 and 640 bytes), the plain
messages with sum, mean and max, fp32 and bf16; and a graph just below the
size, which keeps whole rows, as a control."""
import numpy as np
import pytest
import torch

import synth
from tests.parity import run_propagate_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pyg():
    import paper_1903_02428_amd as m
    assert torch.cuda.is_available()
    m.library()
    return m


# (N, E, F, dtype, hub edges): x bytes N*F*s
CASES = [
    (40_000, 600_000, 128, torch.float32, 60_000),    # 20.5 MB, 4 windows, light rows + two hubs
    (40_000, 1_500_000, 128, torch.float32, 0),       # heavy rows (mean degree 37)
    (45_000, 500_000, 96, torch.float32, 30_000),     # 384-byte rows: 3 windows
    (30_000, 400_000, 160, torch.float32, 30_000),    # 640-byte rows: 5 windows
    (70_000, 600_000, 128, torch.bfloat16, 40_000),   # 17.9 MB bf16, 2 windows
    (50_000, 500_000, 192, torch.bfloat16, 20_000),   # 384-byte bf16 rows: 3 windows
    (30_000, 400_000, 128, torch.float32, 30_000),    # 15.4 MB: below the size, whole rows
]
RUNS = [("src", False, "sum"), ("src", True, "mean"), ("diff", False, "sum"), ("src", False, "max"),
        ("src", True, "max")]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_narrow_window_propagate(pyg, case):
    N, E, F, dtype, hub = CASES[case]
    rng = np.random.default_rng(900 + case)
    ei = synth.random_coo(rng, N, E)
    if hub:
        ei[1, :hub] = 0
        ei[1, hub:2 * hub] = N - 1
    x = rng.standard_normal((N, F)).astype(np.float32)
    w = rng.standard_normal(E).astype(np.float32)
    for msg, weighted, aggr in RUNS:
        run_propagate_case(pyg, ei, x, w if weighted else None, msg=msg, aggr=aggr, dtype=dtype,
                           what=f"narrow case {case} N={N} E={E} F={F}")

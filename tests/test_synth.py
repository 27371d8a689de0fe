"""Generated workloads have the stated shapes (CPU only)."""
import numpy as np

import synth


def _simple(ei, N):
    keys = ei[0] * N + ei[1]
    return np.unique(keys).size == keys.size and not (ei[0] == ei[1]).any()


def test_config1_shape():
    c = synth.make_config(1)
    assert c["x"].shape == (2708, 16) and c["x"].dtype == np.float32
    assert c["edge_index"].shape == (2, 10556) and _simple(c["edge_index"], 2708)
    assert c["edge_index_gcn"].shape == (2, 13264)
    # symmetric: every edge has its reverse
    ei = c["edge_index"]
    assert np.array_equal(np.sort(ei[0] * 2708 + ei[1]), np.sort(ei[1] * 2708 + ei[0]))


def test_config2_shape():
    c = synth.make_config(2)
    assert c["edge_index"].shape == (2, 88648) and _simple(c["edge_index"], 19717)
    assert c["edge_index_gcn"].shape == (2, 108365)
    assert c["x64"].shape == (19717, 64) and c["x500"].shape == (19717, 500)
    deg = np.bincount(c["edge_index"][1], minlength=19717)
    assert deg.max() > 50 * np.median(deg[deg > 0])  # heavy tail


def test_config3_shape():
    c = synth.make_config(3)
    assert c["B"] == 128 and c["batch"].shape == (c["N"],)
    assert (np.diff(c["batch"]) >= 0).all() and c["sizes"].min() >= 10 and c["sizes"].max() <= 40
    ei = c["edge_index"]
    assert (c["batch"][ei[0]] == c["batch"][ei[1]]).all()  # block-diagonal
    assert 1.5 < ei.shape[1] / 2 / c["N"] < 3.0


def test_config4_shape():
    c = synth.make_config(4)
    ei = c["edge_index"]
    assert ei.shape == (2, 262144) and c["x"].shape == (16384, 64)
    assert (np.bincount(ei[1], minlength=16384) == 16).all()
    assert ((ei[0] // 1024) == (ei[1] // 1024)).all() and not (ei[0] == ei[1]).any()
    es = c["edge_index_shuffled"]
    assert np.array_equal(np.sort(es[0] * 16384 + es[1]), np.sort(ei[0] * 16384 + ei[1]))


def test_config5_recipe_small():
    c = synth.config5_large_power_law(pairs=200_000, N=5000, F=8)
    ei = c["edge_index_gcn"]
    assert ei.shape == (2, 400_000 + 5000)
    assert _simple(ei[:, ~(ei[0] == ei[1])], 5000)
    assert (ei[0] == ei[1]).sum() == 5000


def test_erdos_renyi_shapes():
    rng = np.random.default_rng(0)
    for coalesced in (False, True):
        ei = synth.erdos_renyi(1000, 16, rng, coalesced)
        assert ei.shape == (2, 16000) and not (ei[0] == ei[1]).any()
        assert np.unique(ei[1] * 1000 + ei[0]).size == 16000
        if coalesced:
            assert (np.diff(ei[1] * 1000 + ei[0]) > 0).all()


def test_hashed_values_match_a_plain_python_hash():
    """The tensor generator equals a plain-integer rendering of its definition
    on sample counters (including ones above 2^32), and stays in [-1, 1)."""
    import torch

    from synth.hashed import hashed_values

    def lowbias32(x):
        x ^= x >> 16
        x = (x * 0x7FEB352D) & 0xFFFFFFFF
        x ^= x >> 15
        x = (x * 0x846CA68B) & 0xFFFFFFFF
        return x ^ (x >> 16)

    F, seed = 7, 5
    rows = [0, 1, 12345, 2**29 + 3, 114_832_964]
    got = hashed_values(torch.tensor(rows), F, seed).numpy()
    for a, r in enumerate(rows):
        for f in range(F):
            c = r * F + f
            lo, hi = c & 0xFFFFFFFF, (c >> 32) & 0xFFFFFFFF
            x = lowbias32(lo ^ lowbias32((hi + seed * 0x9E37) & 0xFFFFFFFF))
            assert got[a, f] == np.float32((x >> 8) * 2.0 ** -23 - 1.0)
    assert got.min() >= -1.0 and got.max() < 1.0

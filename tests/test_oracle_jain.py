"""Pins of Jain, MaxVio and Comm. Red. (App. H eqs. jain, maxvio, comm-red) -- CPU only."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_main.txt")


def test_jain_special_cases(oracle_mod):
    G = 8
    eq = np.full((1, 3, G), 5, dtype=np.int64)
    j, v = oracle_mod.jain(eq)
    assert j[0] == 1.0 and v[0] == 0.0
    one = np.zeros((1, 2, G), dtype=np.int64)
    one[0, :, 3] = 7
    j, v = oracle_mod.jain(one)
    assert abs(j[0] - 1.0 / G) < 1e-15 and abs(v[0] - (G - 1)) < 1e-12
    z = np.zeros((2, 2, G), dtype=np.int64)
    j, v = oracle_mod.jain(z)
    assert np.all(j == 1.0) and np.all(v == 0.0)


def test_jain_range_and_per_layer(oracle_mod):
    rng = np.random.default_rng(0)
    ld = rng.integers(0, 1000, size=(50, 4, 6))
    j, v = oracle_mod.jain(ld)
    assert np.all(j >= 1 / 6 - 1e-15) and np.all(j <= 1 + 1e-15)
    tot = ld.sum(axis=1).astype(float)
    np.testing.assert_allclose(j, tot.sum(1) ** 2 / (6 * (tot ** 2).sum(1)), rtol=1e-14)
    np.testing.assert_allclose(v, tot.max(1) / tot.mean(1) - 1, rtol=1e-13)
    jl, vl = oracle_mod.jain(ld, per_layer=True)
    assert jl.shape == (50, 4)
    np.testing.assert_allclose(jl[:, 2], ld[:, 2].sum(1) ** 2 / (6 * (ld[:, 2].astype(float) ** 2).sum(1)), rtol=1e-14)


def _table():
    rows = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        parts = line.split()
        rows[(parts[0], parts[1])] = np.array([float(x) for x in parts[2:]])
    return rows


def test_comm_reduction_reproduces_table(oracle_mod):
    """Every printed Comm. Red. of the main table equals eq. comm-red applied to the printed Comm of
    the method and of the default placement, to the printed two decimals."""
    t = _table()
    for model in ("DeepSeek-MoE-16B", "Qwen1.5-MoE-A2.7B", "Moonlight-16B-A3B"):
        comm = t[(model, "Comm")]
        red = oracle_mod.comm_reduction(comm[0], comm)
        np.testing.assert_allclose(np.round(red, 2), t[(model, "CommRed")], atol=1e-9)


def test_table_averages(oracle_mod):
    """The averaged row is the mean of the per-model rows (Comm. Red. within the printed rounding)."""
    t = _table()
    models = ("DeepSeek-MoE-16B", "Qwen1.5-MoE-A2.7B", "Moonlight-16B-A3B")
    for metric, tol in (("Comm", 1e-4), ("Jain", 1e-4), ("MaxVio", 1e-4), ("CommRed", 0.0101)):
        mean = np.mean([t[(m, metric)] for m in models], axis=0)
        np.testing.assert_allclose(mean, t[("Average", metric)], atol=tol)

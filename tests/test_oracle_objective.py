"""Pins of the oracle's grouping objective (eq. grouping-objective), CPU only."""
import numpy as np

from paper_2606_01007_amd import synth


def test_hand_worked(oracle_mod):
    # 4 experts on 2 GPUs: {0, 1} on GPU 0 and {2, 3} on GPU 1
    a = np.array([[[0, 1, 2, 3], [1, 0, 4, 5], [2, 4, 0, 6], [3, 5, 6, 0]]], dtype=np.float64)
    prim = np.array([[[0, 0, 1, 1]]], dtype=np.uint8)
    np.testing.assert_allclose(oracle_mod.grouping_objective(a, prim, 2), [[2 * 1 + 2 * 6]])
    prim = np.array([[[0, 1, 0, 1]]], dtype=np.uint8)    # {0, 2} and {1, 3}
    np.testing.assert_allclose(oracle_mod.grouping_objective(a, prim, 2), [[2 * 2 + 2 * 5]])


def test_one_gpu_is_the_total_and_singletons_are_zero(oracle_mod):
    rng = np.random.default_rng(1)
    a = rng.random((2, 6, 6))
    a = (a + a.transpose(0, 2, 1)) / 2
    for l in range(2):
        np.fill_diagonal(a[l], 0.0)
    np.testing.assert_allclose(oracle_mod.grouping_objective(a, np.zeros((1, 2, 6), np.uint8), 1)[0],
                               a.sum(axis=(1, 2)))
    single = np.arange(6, dtype=np.uint8)[None, None].repeat(2, axis=1)
    np.testing.assert_array_equal(oracle_mod.grouping_objective(a, single, 6), [[0.0, 0.0]])


def test_matches_quadratic_form(oracle_mod):
    # sum_m x_m^T A x_m with one-hot columns x_m, off the diagonal
    rng = np.random.default_rng(2)
    E, G, L, P = 24, 4, 3, 5
    a = rng.random((L, E, E))
    prim = synth.random_placements(P, L, E, G, 6, 3)
    got = oracle_mod.grouping_objective(a, prim, G)
    for p in range(P):
        for l in range(L):
            x = np.zeros((E, G))
            x[np.arange(E), prim[p, l]] = 1.0
            ref = np.trace(x.T @ a[l] @ x) - np.trace(np.diag(np.diag(a[l])) @ (x @ x.T))
            np.testing.assert_allclose(got[p, l], ref, rtol=1e-12)

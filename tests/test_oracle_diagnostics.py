"""Pins of the oracle's motivation diagnostics (App. H, auxiliary motivation metrics), CPU only."""
import numpy as np

from paper_2606_01007_amd import synth


def test_activation_distance_hand_worked(oracle_mod):
    # k = 1, one layer, E = 2: family 0 always picks expert 0 (P = (1, 0)), family 1 splits (1/2, 1/2)
    D = np.array([[[4, 0]], [[3, 3]]], dtype=np.int64)
    d = oracle_mod.activation_distance(D, 1)
    np.testing.assert_allclose(d, [[0, np.sqrt(0.5)], [np.sqrt(0.5), 0]])


def test_activation_distance_metric(oracle_mod):
    w = synth.make_workload("deepseek16b", n_tokens=8 * 800, layers=2)
    D, C, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, 64)
    d = oracle_mod.activation_distance(D, 6)
    np.testing.assert_allclose(d, d.T)
    np.testing.assert_array_equal(np.diag(d), 0.0)
    F = d.shape[0]
    for i in range(F):
        for j in range(F):
            for k in range(F):
                assert d[i, k] <= d[i, j] + d[j, k] + 1e-12


def test_top_pairs_hand_worked(oracle_mod):
    # E = 4: counts of pairs (0,1)=5, (0,2)=2, (0,3)=2, (1,2)=0, (1,3)=7, (2,3)=2
    C = np.zeros((1, 1, 4, 4), np.int64)
    for (a, b, c) in [(0, 1, 5), (0, 2, 2), (0, 3, 2), (1, 3, 7), (2, 3, 2)]:
        C[0, 0, a, b] = C[0, 0, b, a] = c
    # top 3: (1,3)=7, (0,1)=5, then the tie at 2 goes to the lowest pair index, (0,2) = 2
    np.testing.assert_array_equal(oracle_mod.top_pairs(C, 3)[0, 0], [0 * 4 + 1, 0 * 4 + 2, 1 * 4 + 3])
    # with room for all, the zero-count pair (1,2) stays out
    np.testing.assert_array_equal(oracle_mod.top_pairs(C, 8)[0, 0], [1, 2, 3, 7, 11, -1, -1, -1])


def test_pair_jaccard_properties(oracle_mod):
    w = synth.make_workload("qwen15", n_tokens=6 * 900, layers=2)
    D, C, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, 60)
    J = oracle_mod.pair_jaccard(C, 64)
    for l in range(J.shape[0]):
        np.testing.assert_allclose(J[l], J[l].T)
        np.testing.assert_array_equal(np.diag(J[l]), 1.0)
    assert ((J >= 0) & (J <= 1)).all()
    # a family compared with a copy of itself overlaps fully; with a disjoint family not at all
    C2 = np.zeros((2, 1, 6, 6), np.int64)
    C2[0, 0, 0, 1] = C2[0, 0, 1, 0] = 3
    C2[1, 0, 4, 5] = C2[1, 0, 5, 4] = 3
    np.testing.assert_array_equal(oracle_mod.pair_jaccard(C2, 64)[0], [[1, 0], [0, 1]])

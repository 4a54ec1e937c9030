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


def test_activation_distance_hand_worked_top2(oracle_mod):
    # k = 2, one layer, E = 3, four tokens per family.  Family 0 always picks {0, 1}: each of experts 0
    # and 1 is activated by every token, P_0 = (1, 1, 0) (an activation probability per expert, so the
    # row sums to k = 2).  Family 1 picks {0, 2} twice and {1, 2} twice: P_1 = (1/2, 1/2, 1).
    # dist = sqrt(1/4 + 1/4 + 1) = sqrt(3/2).  A share of dispatches (D / sum D, rows summing to 1)
    # would give sqrt(3/8) instead.
    D = np.array([[[4, 4, 0]], [[2, 2, 4]]], dtype=np.int64)
    d = oracle_mod.activation_distance(D, 2)
    np.testing.assert_allclose(d, [[0, np.sqrt(1.5)], [np.sqrt(1.5), 0]], rtol=1e-15)


def test_activation_distance_brute_force(oracle_mod):
    # The definition written out over the tokens: P_f[l][e] = (tokens of f whose layer-l selection holds
    # e) / (tokens of f), for every family, on a tiny seeded trace with top-3 and an empty family.
    rng = np.random.default_rng(7)
    L, E, k = 2, 6, 3
    counts = [5, 0, 9]
    off = np.concatenate([[0], np.cumsum(counts)])
    N = off[-1]
    trace = np.stack([[rng.permutation(E)[:k] for _ in range(N)] for _ in range(L)]).astype(np.int16)
    D, _, err = oracle_mod.coact(trace, off, E)
    assert err == 0
    F = len(counts)
    P = np.zeros((F, L, E))
    for f in range(F):
        for l in range(L):
            toks = [set(int(x) for x in trace[l, t]) for t in range(off[f], off[f + 1])]
            for e in range(E):
                P[f, l, e] = sum(e in s for s in toks) / len(toks) if toks else 0.0
    want = np.array([[np.sqrt(((P[i] - P[j]) ** 2).sum()) for j in range(F)] for i in range(F)])
    np.testing.assert_allclose(oracle_mod.activation_distance(D, k), want, rtol=1e-13, atol=1e-15)
    # each non-empty family's per-layer activation probabilities sum to k
    np.testing.assert_allclose(P[[0, 2]].sum(axis=2), k, rtol=1e-15)


def test_pair_jaccard_partial_overlap(oracle_mod):
    # Unequal, partially overlapping top sets: family 0 co-activates {(0,1), (0,2)}, family 1
    # {(0,1), (2,3), (3,4)}: |A & B| = 1 and |A | B| = 4, so the overlap is 1/4 (a max(|A|, |B|)
    # denominator would give 1/3, a min one 1/2).
    C = np.zeros((2, 1, 5, 5), np.int64)
    for f, pairs in ((0, [(0, 1), (0, 2)]), (1, [(0, 1), (2, 3), (3, 4)])):
        for a, b in pairs:
            C[f, 0, a, b] = C[f, 0, b, a] = 2
    J = oracle_mod.pair_jaccard(C, 64)[0]
    np.testing.assert_array_equal(J, [[1.0, 0.25], [0.25, 1.0]])
    # with top_n = 2 family 1 keeps its two lowest-index pairs (a tie at count 2): {(0,1), (2,3)},
    # and the overlap with {(0,1), (0,2)} is 1/3
    np.testing.assert_array_equal(oracle_mod.pair_jaccard(C, 2)[0], [[1.0, 1 / 3], [1 / 3, 1.0]])

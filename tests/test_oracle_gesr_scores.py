"""Pins of the oracle's GESR identification scores (Sec. 3.4, eq. generic-score), CPU only."""
import numpy as np
import pytest

from paper_2606_01007_amd import synth


def _counts_from_sets(tokens_per_family, E):
    """D, C of one layer from explicit token expert sets (one list per family)."""
    F = len(tokens_per_family)
    D = np.zeros((F, 1, E), np.int64)
    C = np.zeros((F, 1, E, E), np.int64)
    for f, toks in enumerate(tokens_per_family):
        for t in toks:
            for a in t:
                D[f, 0, a] += 1
                for b in t:
                    if a != b:
                        C[f, 0, a, b] += 1
        for e in range(E):
            C[f, 0, e, e] = D[f, 0, e]
    return D, C


def test_hand_worked(oracle_mod):
    # E = 3, k = 2.  Family 0: tokens {0,1}, {0,1}  -> N = 2, A_0(0,1) = 1, A_0(0,2) = 0
    #                 Family 1: tokens {0,2}, {1,2}  -> N = 2, A_1(0,2) = 1/2, A_1(1,2) = 1/2
    D, C = _counts_from_sets([[(0, 1), (0, 1)], [(0, 2), (1, 2)]], 3)
    cent, cons, spec = oracle_mod.gesr_scores(D, C, 2)
    # A-bar row 0 = (0, 1/2, 1/4): Cent = 3/4
    np.testing.assert_allclose(cent[0, 0], 0.75)
    # cos(A_0(0,:) = (0,1,0), A-bar) = (1/2) / (1 * sqrt(5/16)); cos(A_1(0,:) = (0,0,1/2), A-bar) = (1/8) / (1/2 * sqrt(5/16))
    nb = np.sqrt(5 / 16)
    np.testing.assert_allclose(cons[0, 0], ((0.5 / nb) + (0.125 / (0.5 * nb))) / 2)
    # deviations: ||(0, 1/2, -1/4)|| and ||(0, -1/2, 1/4)||, both sqrt(5/16)
    np.testing.assert_allclose(spec[0, 0], nb)


def test_identical_families_are_consistent(oracle_mod):
    w = synth.make_workload("tiny")
    D, C, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, 8)
    D2 = np.concatenate([D[:1]] * 3)
    C2 = np.concatenate([C[:1]] * 3)
    cent, cons, spec = oracle_mod.gesr_scores(D2, C2, 2)
    active = cent > 0
    np.testing.assert_allclose(cons[active], 1.0, rtol=1e-12)
    np.testing.assert_allclose(spec, 0.0, atol=1e-15)


def test_ranges_and_centrality_identity(oracle_mod):
    w = synth.make_workload("qwen15", n_tokens=6000, layers=2)
    D, C, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, 60)
    cent, cons, spec = oracle_mod.gesr_scores(D, C, 4)
    assert (cons >= -1e-12).all() and (cons <= 1 + 1e-12).all() and (spec >= 0).all()
    # exact top-k: each token with e co-selects k - 1 others, so Cent(e) = (k - 1) * mean_f u_f(e) * k
    N = D.sum(axis=2) / 4.0                                    # [F][L]
    u = D / (N[:, :, None] * 4)
    np.testing.assert_allclose(cent, 3 * 4 * u.mean(axis=0), rtol=1e-12)


def test_relabelling_permutes(oracle_mod):
    w = synth.make_workload("tiny")
    D, C, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, 8)
    perm = np.random.default_rng(0).permutation(8)
    Dp = D[:, :, perm]
    Cp = C[:, :, perm][:, :, :, perm]
    a = oracle_mod.gesr_scores(D, C, 2)
    b = oracle_mod.gesr_scores(Dp, Cp, 2)
    for x, y in zip(a, b):
        np.testing.assert_allclose(y, x[:, perm], rtol=1e-12, atol=1e-15)

"""Pins of the oracle's family preferences and task-modulated graph (CPU only).

The paper prints no worked example for these steps, so the pins are: a hand-derived example with
closed-form values, library cross-checks (scipy's z-score and logistic function, numpy products),
and exact identities that a dropped term, a wrong sign, a wrong index or a transposed operand would
break (Sec. 3.3, eqs. usage-coact-advantage .. task-modulated-graph).
"""
import numpy as np
import pytest
import scipy.special
import scipy.stats

from paper_2606_01007_amd import synth


def _counts_from_sets(fams, E):
    """D [F][1][E], C [F][1][E][E] written out by hand from lists of token sets (one layer)."""
    F = len(fams)
    D = np.zeros((F, 1, E), dtype=np.int64)
    C = np.zeros((F, 1, E, E), dtype=np.int64)
    for f, toks in enumerate(fams):
        for S in toks:
            for i in S:
                D[f, 0, i] += 1
                for j in S:
                    if i != j:
                        C[f, 0, i, j] += 1
        for i in range(E):
            C[f, 0, i, i] = D[f, 0, i]
    return D, C


def test_hand_worked_example(oracle_mod):
    """E = 3, k = 2, two families of four tokens:
       family 0: {0,1} x3, {0,2} x1      family 1: {1,2} x2, {0,2} x2
    u0 = (4,3,1)/8, u1 = (2,2,4)/8, so du0 = (1/4, 1/8, -3/8) = -du1 (mean 0, population
    variance 7/96).  c = k(k-1) u for top-k traces, so dc = 2 du and
    s0 = 2 du0 / sqrt(7/96) = -s1;  p0 = 1 / (1 + exp(-2 s0)).
    A-bar off-diagonal: (0,1) = 3/8, (0,2) = 3/8, (1,2) = 1/4 -> A-hat = (1, 1, 2/3)."""
    D, C = _counts_from_sets([[{0, 1}] * 3 + [{0, 2}], [{1, 2}] * 2 + [{0, 2}] * 2], 3)
    alpha = 0.25
    pref, at, ah = oracle_mod.reweight(D, C, 2, alpha=alpha, tau=1.0, eps=0.0)
    du0 = np.array([1 / 4, 1 / 8, -3 / 8])
    s0 = 2 * du0 / np.sqrt(7 / 96)
    p0 = 1.0 / (1.0 + np.exp(-2 * s0))
    np.testing.assert_allclose(pref[0, :, 0], p0, rtol=1e-12)
    np.testing.assert_allclose(pref[0, :, 1], 1 - p0, rtol=1e-12)
    ah_exp = np.array([[0, 1, 1], [1, 0, 2 / 3], [1, 2 / 3, 0]])
    np.testing.assert_allclose(ah[0], ah_exp, rtol=1e-12, atol=0)
    P = np.stack([p0, 1 - p0], axis=1)
    task = np.array([[P[i] @ P[j] for j in range(3)] for i in range(3)])
    np.testing.assert_allclose(at[0], (1 - alpha) * ah_exp + alpha * task * ah_exp, rtol=1e-12)


@pytest.fixture(scope="module")
def qwen_small(oracle_mod):
    w = synth.make_workload("qwen15", n_tokens=6 * 2000, layers=3)
    D, C, err = oracle_mod.coact(w.trace_group, w.fam_off_group, w.cfg.E)
    assert err == 0
    return w, D, C


def test_zscore_matches_scipy(oracle_mod, qwen_small):
    _, D, C = qwen_small
    t = oracle_mod.layer_terms(D[:, 1], C[:, 1], 4, eps=0.0)
    for f in range(D.shape[0]):
        z = scipy.stats.zscore(t["du"][f], ddof=0)
        np.testing.assert_allclose(oracle_mod._zscore(t["du"][f], 0.0), z, rtol=1e-10, atol=1e-12)


def test_advantage_identities(oracle_mod, qwen_small):
    """mean_e du = 0 (u sums to 1 per family);  c = k(k-1) u and dc = k(k-1) du for top-k traces,
    so z(dc) = z(du) and s = 2 z(du);  u sums to one;  du matches a direct recomputation."""
    w, D, C = qwen_small
    k = w.cfg.k
    for l in range(D.shape[1]):
        t = oracle_mod.layer_terms(D[:, l], C[:, l], k, eps=0.0)
        np.testing.assert_allclose(t["u"].sum(axis=1), 1.0, rtol=1e-13)
        np.testing.assert_allclose(t["du"].mean(axis=1), 0.0, atol=1e-15)
        np.testing.assert_allclose(t["c"], k * (k - 1) * t["u"], rtol=1e-12)
        np.testing.assert_allclose(t["dc"], k * (k - 1) * t["du"], rtol=1e-10, atol=1e-15)
        z = np.stack([scipy.stats.zscore(t["du"][f]) for f in range(D.shape[0])])
        np.testing.assert_allclose(t["s"], 2 * z, rtol=1e-9, atol=1e-12)
        nf = D[:, l].sum(axis=1) / k
        F = D.shape[0]
        for f in range(F):
            rest = [g for g in range(F) if g != f]
            direct = D[f, l] / (nf[f] * k) - np.mean([D[g, l] / (nf[g] * k) for g in rest], axis=0)
            np.testing.assert_allclose(t["du"][f], direct, rtol=1e-12, atol=1e-15)


def test_preferences_are_distributions(oracle_mod, qwen_small):
    w, D, C = qwen_small
    pref, at, ah = oracle_mod.reweight(D, C, w.cfg.k)
    np.testing.assert_allclose(pref.sum(axis=2), 1.0, rtol=1e-13)
    assert np.all(pref > 0) and np.all(pref < 1)


def test_softmax_matches_scipy(oracle_mod, qwen_small):
    w, D, C = qwen_small
    tau = 0.7
    pref, _, _ = oracle_mod.reweight(D, C, w.cfg.k, tau=tau)
    for l in range(D.shape[1]):
        t = oracle_mod.layer_terms(D[:, l], C[:, l], w.cfg.k, tau=tau)
        np.testing.assert_allclose(pref[l].T, scipy.special.softmax(t["s"] / tau, axis=0), rtol=1e-12)


def test_two_families_logistic(oracle_mod):
    """F = 2: du2 = -du1, so s2 = -s1 and p1 = sigmoid(2 s1 / tau), with s1 from scipy's z-score of
    the usage and co-activation differences computed directly from the counts."""
    w = synth.make_workload("deepseek16b", n_tokens=8 * 400, layers=2)
    D8, C8, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, w.cfg.E)
    D, C = D8[:2], C8[:2]
    k, tau = w.cfg.k, 1.3
    pref, _, _ = oracle_mod.reweight(D, C, k, tau=tau, eps=0.0)
    for l in range(2):
        n = D[:, l].sum(axis=1) / k
        u = D[:, l] / (n[:, None] * k)
        A = C[:, l] / n[:, None, None]
        c = A.sum(axis=2) - np.diagonal(A, axis1=1, axis2=2)
        s1 = scipy.stats.zscore(u[0] - u[1]) + scipy.stats.zscore(c[0] - c[1])
        np.testing.assert_allclose(pref[l, :, 0], scipy.special.expit(2 * s1 / tau), rtol=1e-10)


def test_identical_families(oracle_mod):
    """F identical families: du = 0 so every preference is 1/F, A_task = 1/F and
    A-tilde = (1 - alpha + alpha / F) A-hat."""
    w = synth.make_workload("tiny")
    D1, C1, _ = oracle_mod.coact(w.trace_group, w.fam_off_group, 8)
    F = 4
    D = np.repeat(D1[:1], F, axis=0)
    C = np.repeat(C1[:1], F, axis=0)
    alpha = 0.4
    pref, at, ah = oracle_mod.reweight(D, C, 2, alpha=alpha)
    np.testing.assert_allclose(pref, 1.0 / F, rtol=1e-12)
    np.testing.assert_allclose(at, (1 - alpha + alpha / F) * ah, rtol=1e-12)


def test_graph_properties(oracle_mod, qwen_small):
    """alpha = 0 gives A-hat; A-tilde symmetric with 0 <= A-tilde <= A-hat <= 1, the same zero pattern
    as A-bar, a zero diagonal, and max off-diagonal A-hat = 1;  A-hat = A-bar / max (A-bar = mean_f A)."""
    w, D, C = qwen_small
    k = w.cfg.k
    p0, at0, ah0 = oracle_mod.reweight(D, C, k, alpha=0.0)
    np.testing.assert_array_equal(at0, ah0)
    pref, at, ah = oracle_mod.reweight(D, C, k, alpha=0.25)
    np.testing.assert_array_equal(ah, ah0)
    assert np.array_equal(at, np.swapaxes(at, 1, 2))
    assert np.all(at >= 0) and np.all(at <= ah + 1e-15) and np.all(ah <= 1.0)
    E = D.shape[2]
    off = ~np.eye(E, dtype=bool)
    for l in range(D.shape[1]):
        n = D[:, l].sum(axis=1) / k
        abar = (C[:, l] / n[:, None, None]).mean(axis=0) * off
        assert np.array_equal(at[l] == 0, abar == 0)
        assert ah[l][off].max() == 1.0
        np.testing.assert_allclose(ah[l], abar / abar[off].max(), rtol=1e-13)
        np.testing.assert_allclose(at[l], 0.75 * ah[l] + 0.25 * (pref[l] @ pref[l].T) * ah[l], rtol=1e-13)


def test_empty_family_and_zero_layer(oracle_mod):
    """An empty family keeps u = 0 and still takes part in the advantages; an all-zero layer gives
    A-hat = A-tilde = 0 and uniform preferences (all advantages are zero)."""
    D, C = _counts_from_sets([[{0, 1}, {1, 2}], [], [{2, 3}, {0, 3}]], 4)
    pref, at, ah = oracle_mod.reweight(D, C, 2)
    assert np.all(np.isfinite(pref)) and np.allclose(pref.sum(axis=2), 1)
    Dz = np.zeros((3, 1, 4), dtype=np.int64)
    Cz = np.zeros((3, 1, 4, 4), dtype=np.int64)
    pref, at, ah = oracle_mod.reweight(Dz, Cz, 2)
    assert np.all(ah == 0) and np.all(at == 0)
    np.testing.assert_allclose(pref, 1 / 3)
    with pytest.raises(ValueError):
        oracle_mod.reweight(D[:1], C[:1], 2)

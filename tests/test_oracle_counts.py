"""Pins of the oracle's dispatch and co-activation counts (CPU only).

The oracle follows the set definition of the per-family statistics (Sec. 3.3, "Scoring task-family
preference").  Here it is checked against things other than itself: a pure-Python brute force over
expert pairs, the one-hot product R^T R computed by numpy, exact invariants of top-k traces, and
relabelling / reordering symmetries.
"""
import itertools

import numpy as np
import pytest

from paper_2606_01007_amd import synth


def _random_trace(L, N, k, E, seed):
    rng = np.random.default_rng(seed)
    tr = np.zeros((L, N, k), dtype=np.int16)
    for l in range(L):
        for t in range(N):
            tr[l, t] = rng.choice(E, size=k, replace=False)
    return tr


def _brute(tr, fam_off, E):
    """For every (f, l) and every pair (i, j): scan the tokens and test membership of both."""
    L, N, k = tr.shape
    F = len(fam_off) - 1
    D = np.zeros((F, L, E), dtype=np.int64)
    C = np.zeros((F, L, E, E), dtype=np.int64)
    for f in range(F):
        for l in range(L):
            sets = [set(int(x) for x in tr[l, t]) for t in range(fam_off[f], fam_off[f + 1])]
            for i in range(E):
                D[f, l, i] = sum(1 for S in sets if i in S)
                for j in range(E):
                    if i == j:
                        C[f, l, i, j] = D[f, l, i]
                    else:
                        C[f, l, i, j] = sum(1 for S in sets if i in S and j in S)
    return D, C


@pytest.mark.parametrize("E,k,L,counts,seed", [
    (5, 2, 2, [7, 0, 11], 1),
    (9, 3, 3, [30, 25], 2),
    (12, 4, 2, [40, 1, 33, 20], 3),
    (6, 6, 1, [9, 4], 4),
    (7, 1, 2, [13, 5], 5),
])
def test_counts_match_brute_force(oracle_mod, E, k, L, counts, seed):
    off = synth.fam_offsets(counts)
    tr = _random_trace(L, int(off[-1]), k, E, seed)
    D, C, err = oracle_mod.coact(tr, off, E)
    assert err == 0
    Db, Cb = _brute(tr, off, E)
    np.testing.assert_array_equal(D, Db)
    np.testing.assert_array_equal(C, Cb)


def test_tiny_config_brute_force(oracle_mod):
    w = synth.make_workload("tiny")
    D, C, err = oracle_mod.coact(w.trace_group, w.fam_off_group, 8)
    assert err == 0
    Db, Cb = _brute(w.trace_group.numpy(), w.fam_off_group, 8)
    np.testing.assert_array_equal(D, Db)
    np.testing.assert_array_equal(C, Cb)


def test_counts_equal_onehot_gram(oracle_mod):
    """C_f[l] = R^T R for the one-hot token-by-expert matrix R of the segment (numpy int64 matmul)."""
    w = synth.make_workload("deepseek16b", n_tokens=8 * 700, layers=2)
    E = w.cfg.E
    tr = w.trace_group.numpy()
    D, C, err = oracle_mod.coact(tr, w.fam_off_group, E)
    assert err == 0
    for f in range(w.cfg.F):
        for l in range(2):
            seg = tr[l, w.fam_off_group[f]:w.fam_off_group[f + 1]]
            R = np.zeros((seg.shape[0], E), dtype=np.int64)
            R[np.arange(seg.shape[0])[:, None], seg.astype(np.int64)] = 1
            np.testing.assert_array_equal(C[f, l], R.T @ R)
            np.testing.assert_array_equal(D[f, l], R.sum(axis=0))


@pytest.mark.parametrize("name", ["tiny", "deepseek16b", "qwen15", "qwen3_30b", "deepseek_v3"])
def test_count_invariants(oracle_mod, name):
    """C symmetric, C_ii = D_i, sum_{j != i} C_ij = (k - 1) D_i, sum_i D_i = N_f k,
    sum_{i<j} C_ij = N_f k (k - 1) / 2 -- on every preset shape (reduced token count)."""
    cfg = synth.CONFIGS[name]
    w = synth.make_workload(name, n_tokens=cfg.F * 97, layers=2)
    D, C, err = oracle_mod.coact(w.trace_group, w.fam_off_group, cfg.E)
    assert err == 0
    k = cfg.k
    nf = np.diff(w.fam_off_group)
    assert np.array_equal(C, np.swapaxes(C, 2, 3))
    assert np.array_equal(np.diagonal(C, axis1=2, axis2=3), D)
    off = C.sum(axis=3) - D
    assert np.array_equal(off, (k - 1) * D)
    assert np.array_equal(D.sum(axis=2), np.repeat(nf[:, None] * k, 2, axis=1))
    iu = np.triu_indices(cfg.E, 1)
    assert np.array_equal(C[:, :, iu[0], iu[1]].sum(axis=2), np.repeat(nf[:, None] * k * (k - 1) // 2, 2, axis=1))


def test_relabel_and_reorder(oracle_mod):
    """Renaming experts permutes D and C; shuffling tokens inside a family changes nothing."""
    E, k, L = 10, 3, 2
    counts = [50, 30]
    off = synth.fam_offsets(counts)
    tr = _random_trace(L, 80, k, E, 7)
    D, C, _ = oracle_mod.coact(tr, off, E)
    perm = np.random.default_rng(0).permutation(E)
    D2, C2, _ = oracle_mod.coact(perm[tr].astype(np.int16), off, E)
    np.testing.assert_array_equal(D2[:, :, perm], D)
    np.testing.assert_array_equal(C2[:, :, perm][:, :, :, perm], C)
    rng = np.random.default_rng(1)
    tr3 = tr.copy()
    for l in range(L):
        for f in range(2):
            a, b = off[f], off[f + 1]
            tr3[l, a:b] = tr3[l, a:b][rng.permutation(b - a)]
            tr3[l, a:b] = np.take_along_axis(tr3[l, a:b], rng.permutation(k)[None, :].repeat(b - a, 0), axis=1)
    D3, C3, _ = oracle_mod.coact(tr3, off, E)
    np.testing.assert_array_equal(D3, D)
    np.testing.assert_array_equal(C3, C)


def test_chunked_equals_whole(oracle_mod):
    """Counting the two halves of every family segment separately and adding gives the whole."""
    E, k = 11, 4
    off = synth.fam_offsets([60, 44])
    tr = _random_trace(2, 104, k, E, 9)
    D, C, _ = oracle_mod.coact(tr, off, E)
    Dsum = np.zeros_like(D)
    Csum = np.zeros_like(C)
    for f in range(2):
        for l in range(2):
            a, b = off[f], off[f + 1]
            mid = (a + b) // 2
            for lo, hi in ((a, mid), (mid, b)):
                sub = tr[:, lo:hi]
                Dp, Cp, _ = oracle_mod.coact_segment(sub, [0, hi - lo], E, 0, l)
                Dsum[f, l] += Dp
                Csum[f, l] += Cp
    np.testing.assert_array_equal(Dsum, D)
    np.testing.assert_array_equal(Csum, C)


def test_errors_flagged(oracle_mod):
    E, k = 6, 3
    tr = _random_trace(1, 20, k, E, 3)
    off = [0, 20]
    bad = tr.copy()
    bad[0, 5, 1] = bad[0, 5, 0]
    assert oracle_mod.coact(bad, off, E)[2] & oracle_mod.ERR_ID_DUP
    bad = tr.copy()
    bad[0, 7, 2] = E
    assert oracle_mod.coact(bad, off, E)[2] & oracle_mod.ERR_ID_RANGE
    bad = tr.copy()
    bad[0, 7, 2] = -1
    assert oracle_mod.coact(bad, off, E)[2] & oracle_mod.ERR_ID_RANGE
    assert oracle_mod.coact(tr, [0, 19], E)[2] & oracle_mod.ERR_ARG
    assert oracle_mod.coact(tr, off, E)[2] == 0


def test_all_pairs_once_small(oracle_mod):
    """Exhaustive: a trace holding every k-subset of E experts once has C_ij = C(E-2, k-2)."""
    from math import comb
    E, k = 7, 3
    subsets = list(itertools.combinations(range(E), k))
    tr = np.array(subsets, dtype=np.int16)[None]
    D, C, _ = oracle_mod.coact(tr, [0, len(subsets)], E)
    iu = ~np.eye(E, dtype=bool)
    assert np.all(C[0, 0][iu] == comb(E - 2, k - 2))
    assert np.all(D[0, 0] == comb(E - 1, k - 1))

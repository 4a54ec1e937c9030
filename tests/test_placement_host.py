"""Host-side placement inputs (CPU only): TACG grouping (Sec. 3.3 "Capacity-feasible expert
grouping", eqs. grouping-objective and greedy-insert) and GESR replica tables (Sec. 3.4, eqs.
generic-score and candidate-set)."""
import itertools

import numpy as np
import pytest

from paper_2606_01007_amd import placement as pm


def _planted(E, G, cap, seed, noise=0.05, sizes=None):
    """Block affinity: experts in the same planted block have affinity in [0.5, 1], others below
    `noise`; blocks are random expert subsets (sizes default to the capacities)."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(E)
    sizes = sizes or [cap] * G
    blocks, o = [], 0
    for s in sizes:
        blocks.append(perm[o:o + s])
        o += s
    A = rng.uniform(0, noise, (E, E))
    for b in blocks:
        A[np.ix_(b, b)] = rng.uniform(0.5, 1.0, (len(b), len(b)))
    A = (A + A.T) / 2
    np.fill_diagonal(A, 0)
    return A, blocks


@pytest.mark.parametrize("E,G,cap", [(8, 4, 2), (60, 4, 15), (60, 6, 10), (64, 8, 8), (128, 8, 16),
                                     (256, 32, 8), (10, 3, 4)])
def test_grouping_meets_capacities(E, G, cap):
    rng = np.random.default_rng(E + G)
    A = rng.uniform(0, 1, (E, E))
    A = (A + A.T) / 2
    caps = pm.capacities(E, G, cap)
    g = pm.tacg_grouping(A, caps)
    assert g.dtype == np.uint8 and g.shape == (E,)
    np.testing.assert_array_equal(np.bincount(g, minlength=G), caps)


@pytest.mark.parametrize("E,G,cap,seed", [(64, 8, 8, 1), (60, 6, 10, 2), (128, 8, 16, 3), (256, 32, 8, 4)])
def test_grouping_recovers_planted_blocks(E, G, cap, seed):
    A, blocks = _planted(E, G, cap, seed)
    g = pm.tacg_grouping(A, pm.capacities(E, G, cap))
    for b in blocks:
        assert len(set(g[b].tolist())) == 1, "a planted block was split"
    # the objective of eq. grouping-objective beats the contiguous default
    default = np.repeat(np.arange(G), cap)[:E].astype(np.uint8)
    assert pm.group_affinity(A, g, G) > pm.group_affinity(A, default, G)


def test_grouping_repairs_unequal_clusters():
    # planted blocks of sizes 12 / 4 / 8 / 8 with capacities 8: spectral clustering finds the blocks,
    # the repair keeps the 8 strongest of the 12 and inserts the rest where they fit
    E, G, cap = 32, 4, 8
    A, blocks = _planted(E, G, cap, 7, sizes=[12, 4, 8, 8])
    g = pm.tacg_grouping(A, pm.capacities(E, G, cap))
    np.testing.assert_array_equal(np.bincount(g, minlength=G), [8, 8, 8, 8])
    for b in blocks[2:]:
        assert len(set(g[b].tolist())) == 1
    # the 4-expert block stays together (it is inserted into or kept by one group)
    assert len(set(g[blocks[1]].tolist())) == 1


def test_grouping_optimal_on_tiny_by_exhaustion():
    # E = 6 into 3 GPUs of 2: compare with the best of all 15 pairings on a clear planted instance
    A, _ = _planted(6, 3, 2, 11, noise=0.01)
    g = pm.tacg_grouping(A, pm.capacities(6, 3, 2))
    best = -1.0
    for perm in itertools.permutations(range(6)):
        cand = np.empty(6, dtype=np.uint8)
        cand[list(perm)] = np.repeat(np.arange(3), 2)
        best = max(best, pm.group_affinity(A, cand, 3))
    assert pm.group_affinity(A, g, 3) == pytest.approx(best)


def test_grouping_is_deterministic_and_validates():
    A, _ = _planted(64, 8, 8, 5)
    caps = pm.capacities(64, 8, 8)
    np.testing.assert_array_equal(pm.tacg_grouping(A, caps, seed=3), pm.tacg_grouping(A, caps, seed=3))
    with pytest.raises(ValueError):
        pm.tacg_grouping(A, pm.capacities(63, 8, 8))
    with pytest.raises(ValueError):
        pm.capacities(65, 8, 8)


def test_single_gpu_and_zero_affinity():
    g = pm.tacg_grouping(np.zeros((5, 5)), np.array([5]))
    np.testing.assert_array_equal(g, np.zeros(5))
    g = pm.tacg_grouping(np.zeros((12, 12)), pm.capacities(12, 3, 4))
    np.testing.assert_array_equal(np.bincount(g, minlength=3), [4, 4, 4])


def test_tacg_placement_layers():
    A0, _ = _planted(16, 4, 4, 1)
    A1, _ = _planted(16, 4, 4, 2)
    P = pm.tacg_placement(np.stack([A0, A1]), 4, 4)
    assert P.shape == (2, 16)
    for l in range(2):
        np.testing.assert_array_equal(np.bincount(P[l], minlength=4), [4, 4, 4, 4])


def test_generic_experts_by_centrality():
    # layer 0: expert 3 most central, then 1 (tie with 5 broken to the lower id)
    a = np.zeros((1, 6, 6))
    a[0, 3, :] = 1.0
    a[0, 1, 0] = a[0, 5, 0] = 0.5
    np.testing.assert_array_equal(pm.generic_experts(a, 2), [[1, 3]])
    np.testing.assert_array_equal(pm.generic_experts(a, 1), [[3]])


def test_affinity_secondaries():
    # 6 experts on 3 GPUs: {0,1} on 0, {2,3} on 1, {4,5} on 2.  Expert 0 co-activates strongly with
    # expert 4 (GPU 2) and weakly with expert 2 (GPU 1).
    a = np.zeros((1, 6, 6))
    a[0, 0, 4] = a[0, 4, 0] = 0.9
    a[0, 0, 2] = a[0, 2, 0] = 0.1
    prim = np.array([[0, 0, 1, 1, 2, 2]], dtype=np.uint8)
    sec = pm.affinity_secondaries(a, prim, np.array([[0]]), 3, 2)
    assert sec.shape == (1, 6, 2)
    np.testing.assert_array_equal(sec[0, 0], [2, 1])
    assert (sec[0, 1:] == pm.NONE).all()
    # one secondary: the strongest; ties (all zero) go to the lower GPU number other than the primary
    np.testing.assert_array_equal(pm.affinity_secondaries(a, prim, np.array([[0]]), 3, 1)[0, 0], [2])
    np.testing.assert_array_equal(pm.affinity_secondaries(a, prim, np.array([[3]]), 3, 1)[0, 3], [0])
    with pytest.raises(ValueError):
        pm.affinity_secondaries(a, prim, np.array([[0]]), 3, 3)

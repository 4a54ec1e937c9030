"""Host-side placement inputs for the scoring pass: the TACG primary placement from the
task-modulated graph, and GESR replica tables (generic experts and their secondary GPUs).

These run once per layer on the host, before the trace passes: plain numpy over E x E matrices
(E <= 256).  They are inputs to `tacg_eval_placements`, not part of the timed path.

  tacg_grouping        Sec. 3.3 "Capacity-feasible expert grouping" (eq. grouping-objective):
                       Stage 1 normalized spectral clustering of A-tilde (symmetrised, scaled to
                       [0, 1], diagonal jitter; M smallest eigenvectors of L_sym; k-means with k = M),
                       Stage 2 capacity repair (overfull groups keep their top-C_m members by
                       intra-group affinity; the overflow is inserted by eq. greedy-insert)
  generic_experts      the top experts of each layer by centrality Cent = sum_e' A-bar(e, e')
                       (Sec. 3.4 eq. generic-score with the consistency and specificity weights at 0)
  affinity_secondaries secondary GPUs of each generic expert: the non-primary GPUs with the largest
                       co-activation affinity sum_{e' on m} A-bar(e, e') (Sec. 3.4, the candidate
                       set of eq. candidate-set)

Readings where the paper leaves details open: spectral embedding rows are normalised to unit length
before k-means (normalized spectral clustering); k-means uses k-means++ seeding from a fixed seed and
keeps the best of several starts; the overflow pool is inserted in decreasing weighted degree (ties:
lower expert id) and eq. greedy-insert breaks ties towards the lower GPU number.  Inserting only into
non-full groups fills every group to its exact capacity (the capacities sum to E), so the
donor-receiver swap loop that the paper runs afterwards has nothing left to move.
"""
from __future__ import annotations

import numpy as np

from .synth import capacities  # noqa: F401  (per-GPU capacities, shared with the input generator)

NONE = 0xFF


def _kmeans(X: np.ndarray, k: int, rng: np.random.Generator, n_init: int, iters: int) -> np.ndarray:
    """Lloyd's k-means with k-means++ seeding; the best of n_init starts by inertia."""
    n = X.shape[0]
    best, best_in = None, np.inf
    for _ in range(n_init):
        c = np.empty((k, X.shape[1]))
        c[0] = X[rng.integers(n)]
        d2 = ((X - c[0]) ** 2).sum(axis=1)
        for j in range(1, k):
            p = d2 / d2.sum() if d2.sum() > 0 else np.full(n, 1.0 / n)
            c[j] = X[rng.choice(n, p=p)]
            d2 = np.minimum(d2, ((X - c[j]) ** 2).sum(axis=1))
        lab = None
        for _ in range(iters):
            dist = ((X[:, None, :] - c[None, :, :]) ** 2).sum(axis=2)
            new = dist.argmin(axis=1)
            if lab is not None and np.array_equal(new, lab):
                break
            lab = new
            for j in range(k):
                members = X[lab == j]
                if len(members):
                    c[j] = members.mean(axis=0)
                else:                                   # empty cluster: take the farthest point
                    far = int(dist.min(axis=1).argmax())
                    c[j] = X[far]
        inertia = float(((X - c[lab]) ** 2).sum())
        if inertia < best_in:
            best, best_in = lab.copy(), inertia
    return best


def spectral_groups(aff: np.ndarray, M: int, seed: int = 0, jitter: float = 1e-6, n_init: int = 8,
                    iters: int = 100) -> np.ndarray:
    """Stage 1: normalized spectral clustering of the affinity into M (unconstrained) groups."""
    A = np.asarray(aff, dtype=np.float64)
    A = 0.5 * (A + A.T)
    mx = A.max()
    if mx > 0:
        A = A / mx
    A = A + jitter * np.eye(A.shape[0])
    dinv = 1.0 / np.sqrt(A.sum(axis=1))
    lsym = np.eye(A.shape[0]) - dinv[:, None] * A * dinv[None, :]
    _, vec = np.linalg.eigh(lsym)
    U = vec[:, :M]
    U = U / np.maximum(np.linalg.norm(U, axis=1, keepdims=True), 1e-300)
    return _kmeans(U, M, np.random.default_rng(seed), n_init, iters)


def tacg_grouping(aff: np.ndarray, caps: np.ndarray, seed: int = 0) -> np.ndarray:
    """Assign the E experts of one layer to len(caps) GPUs with exactly caps[m] experts on GPU m.

    aff: [E][E] non-negative affinity (the task-modulated graph A-tilde of the layer).
    Returns uint8 [E], the GPU of every expert (group m of the clustering goes to GPU m)."""
    aff = np.asarray(aff, dtype=np.float64)
    E = aff.shape[0]
    caps = np.asarray(caps, dtype=np.int64)
    G = caps.shape[0]
    if aff.shape != (E, E) or int(caps.sum()) != E or G > 255:
        raise ValueError("affinity must be E x E and the capacities must sum to E")
    w = 0.5 * (aff + aff.T)
    np.fill_diagonal(w, 0.0)
    lab = spectral_groups(aff, G, seed) if G > 1 else np.zeros(E, dtype=np.int64)
    gpu = np.full(E, NONE, dtype=np.uint8)
    pool = []
    for m in range(G):
        members = np.flatnonzero(lab == m)
        if len(members) > caps[m]:
            intra = w[np.ix_(members, members)].sum(axis=1)
            order = np.lexsort((members, -intra))       # strongest first, ties: lower id
            keep = members[order[:caps[m]]]
            pool.extend(members[order[caps[m]:]].tolist())
        else:
            keep = members
        gpu[keep] = m
    free = caps - np.bincount(gpu[gpu != NONE].astype(np.int64), minlength=G)
    degree = w.sum(axis=1)
    pool = sorted(pool, key=lambda e: (-degree[e], e))
    for e in pool:                                      # eq. greedy-insert
        placed = gpu != NONE
        to_gpu = np.zeros(G)
        np.add.at(to_gpu, gpu[placed].astype(np.int64), w[e, placed])
        score = np.where(free > 0, to_gpu, -np.inf)
        m = int(np.argmax(score))                       # first maximum: lowest GPU number
        gpu[e] = m
        free[m] -= 1
    return gpu


def tacg_placement(a_tilde: np.ndarray, n_gpus: int, cap: int, seed: int = 0) -> np.ndarray:
    """uint8 [L][E] placement: tacg_grouping of every layer of a_tilde [L][E][E]."""
    a_tilde = np.asarray(a_tilde)
    L, E, _ = a_tilde.shape
    caps = capacities(E, n_gpus, cap)
    return np.stack([tacg_grouping(a_tilde[l], caps, seed + l) for l in range(L)])


def group_affinity(a_bar: np.ndarray, gpu: np.ndarray, n_gpus: int) -> np.ndarray:
    """Within-group affinity sum_m sum_{e != e' on m} a(e, e') of one layer (eq. grouping-objective,
    off-diagonal)."""
    a = np.asarray(a_bar, dtype=np.float64).copy()
    np.fill_diagonal(a, 0.0)
    onehot = np.zeros((a.shape[0], n_gpus))
    onehot[np.arange(a.shape[0]), gpu.astype(np.int64)] = 1.0
    return float(np.einsum("em,ef,fm->", onehot, a, onehot))


def generic_experts(a_bar: np.ndarray, n_generic: int) -> np.ndarray:
    """int64 [L][n_generic]: per layer the experts of largest centrality sum_e' A-bar(e, e'),
    ties to the lower id, listed in increasing id."""
    a_bar = np.asarray(a_bar, dtype=np.float64)
    L, E, _ = a_bar.shape
    cent = a_bar.sum(axis=2)
    out = np.empty((L, n_generic), dtype=np.int64)
    for l in range(L):
        order = np.lexsort((np.arange(E), -cent[l]))
        out[l] = np.sort(order[:n_generic])
    return out


def affinity_secondaries(a_bar: np.ndarray, primary: np.ndarray, generic: np.ndarray, n_gpus: int,
                         n_secondary: int) -> np.ndarray:
    """uint8 [L][E][n_secondary] secondary GPUs (0xFF = none) for one placement primary [L][E].

    Expert e of generic[l] gets the n_secondary GPUs m != primary[l][e] with the largest affinity
    sum_{e' on m, e' != e} A-bar(e, e') (ties: lower GPU number); other experts get none."""
    a_bar = np.asarray(a_bar, dtype=np.float64)
    L, E, _ = a_bar.shape
    sec = np.full((L, E, n_secondary), NONE, dtype=np.uint8)
    if n_secondary == 0:
        return sec
    if n_secondary > n_gpus - 1:
        raise ValueError("more secondaries than non-primary GPUs")
    for l in range(L):
        a = a_bar[l].copy()
        np.fill_diagonal(a, 0.0)
        onehot = np.zeros((E, n_gpus))
        onehot[np.arange(E), primary[l].astype(np.int64)] = 1.0
        aff = a @ onehot                                   # [E][G]
        for e in generic[l]:
            s = aff[e].copy()
            s[int(primary[l][e])] = -np.inf
            order = np.lexsort((np.arange(n_gpus), -s))
            sec[l, e] = order[:n_secondary]
    return sec

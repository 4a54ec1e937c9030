"""CPU oracle of the TACG/GESR trace passes -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use this
package.  It is a plain, slow, obviously correct CPU implementation of the paper's definitions in
int64 and float64, written independently of the HIP library (it imports nothing from it and shares
no code with it).

Integer passes (counts, scoring) are plain C loops in ``tacg_oracle.c`` (built with gcc, OpenMP over
independent segments / placements); the float steps (preferences, reweighted graph, Jain, MaxVio)
are literal numpy transcriptions of the equations below, in float64.

Paper passages followed (Sec. = section of the paper):
  counts               Sec. 3.3 "Scoring task-family preference" (u and A from per-family traces)
  preference           Sec. 3.3 eqs. usage-coact-advantage, coact-advantage, zscore, soft-score,
                       family-pref
  reweighted graph     Sec. 3.3 "Task-modulated coactivation graph": pooled A-bar, max-normalised
                       A-hat, eqs. same-family-kernel and task-modulated-graph
  scoring              Sec. 3.4 eqs. mean-load, feasible-set (+ fallback), candidate-set; App. C
                       per-token dispatch sets; App. H "Comm"
  Jain, MaxVio         App. H eqs. jain, maxvio;  Comm. Red.: App. H eq. comm-red
  decayed-load scoring Sec. 3.4 eq. load-update (the sequential form of the serving rule)
  grouping objective   Sec. 3.3 eq. grouping-objective
  GESR scores          Sec. 3.4 eq. generic-score (Cent, Cons, Spec)
  trace statistics     App. C statistics (i)-(iii) per family (score(..., stats=True))
  diagnostics          App. H auxiliary motivation metrics (activation distance, top-pair Jaccard)

Readings where the paper is silent:
  * u = D / (N_f k) (sums to 1 over experts); A = C / N_f off the diagonal, A(e, e) = 0;
    N_f = sum_e D_f[l][e] / k (the family's token count).
  * z-score uses the population standard deviation; eps and tau are parameters.
  * An empty family (N_f = 0) has u = A = 0 and still enters the advantages and the softmax.
  * max A-bar is taken over off-diagonal entries of the layer; an all-zero layer gives A-hat = 0.
  * Jain and MaxVio are taken over the per-GPU loads summed over layers (one "global" value per
    placement), or per layer when asked; all-zero loads give Jain = 1, MaxVio = 0.
  * Serving-time candidate choice: see the header of tacg_oracle.c.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tacg_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

ERR_ID_RANGE, ERR_ID_DUP, ERR_TABLE, ERR_ARG = 0x1, 0x2, 0x4, 0x8


def build(force: bool = False) -> str:
    """Compile tacg_oracle.c with gcc into liboracle.so (next to the source)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-ffp-contract=off", "-o", tmp, _SRC,
                        "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized(path: str) -> str:
    """Compile tacg_oracle.c with AddressSanitizer and UndefinedBehaviorSanitizer into `path` (for the
    CPU sanitizer tests: load it with TACG_ORACLE_LIBRARY=path and gcc's libasan preloaded)."""
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=undefined", "-fopenmp", "-fPIC", "-shared", "-Wall", "-ffp-contract=off",
                    "-o", path, _SRC, "-lm"], check=True)
    return path


def _load():
    global _lib
    with _lock:
        if _lib is None:
            # TACG_ORACLE_LIBRARY names another build of tacg_oracle.c (a sanitized one, for instance)
            path = os.environ.get("TACG_ORACLE_LIBRARY") or build()
            lib = ctypes.CDLL(path)
            P = ctypes.c_void_p
            i32, i64 = ctypes.c_int32, ctypes.c_int64
            lib.oracle_coact_segment.argtypes = [P, i64, i32, i32, i32, i64, i64, P, P]
            lib.oracle_coact_segment.restype = ctypes.c_int
            lib.oracle_coact.argtypes = [P, i64, i32, i32, i32, P, i32, P, P]
            lib.oracle_coact.restype = ctypes.c_int
            lib.oracle_score.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, i32, i32, i32, i32,
                                         P, P, i32, P, i32, i32, P, P, P, P, P, P, P]
            lib.oracle_score.restype = ctypes.c_int
            lib.oracle_score_online.argtypes = [P, i64, i32, i32, i32, P, i32, P, P, i32, i32, i32, i32,
                                                P, P, i32, ctypes.c_double, i32, i32, P, P, P, P, P, P]
            lib.oracle_score_online.restype = ctypes.c_int
            lib.oracle_num_threads.restype = ctypes.c_int
            lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
            lib.oracle_set_num_threads.restype = None
            _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _np(x, dtype):
    """numpy view/copy of a host array or torch tensor (moved to host if needed)."""
    if hasattr(x, "detach"):
        x = x.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(x), dtype=dtype)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (timing only; results do not depend on it)."""
    _load().oracle_set_num_threads(int(n))


# ------------------------------------------------------------------------------------------------
# counts
# ------------------------------------------------------------------------------------------------
def coact(trace, fam_off, n_experts: int):
    """D [F][L][E], C [F][L][E][E] (int64) and the error bits, over the whole trace."""
    tr = _np(trace, np.int16)
    L, N, k = tr.shape
    off = _np(fam_off, np.int64)
    F = off.size - 1
    D = np.zeros((F, L, n_experts), dtype=np.int64)
    C = np.zeros((F, L, n_experts, n_experts), dtype=np.int64)
    err = _load().oracle_coact(_ptr(tr), N, L, k, n_experts, _ptr(off), F, _ptr(D), _ptr(C))
    return D, C, int(err)


def coact_segment(trace, fam_off, n_experts: int, f: int, l: int):
    """D [E], C [E][E] of one (family, layer) segment."""
    tr = _np(trace, np.int16)
    L, N, k = tr.shape
    off = _np(fam_off, np.int64)
    D = np.zeros(n_experts, dtype=np.int64)
    C = np.zeros((n_experts, n_experts), dtype=np.int64)
    err = _load().oracle_coact_segment(_ptr(tr), N, k, n_experts, l, int(off[f]), int(off[f + 1]), _ptr(D), _ptr(C))
    return D, C, int(err)


# ------------------------------------------------------------------------------------------------
# preferences and the task-modulated graph (float64, literal equations)
# ------------------------------------------------------------------------------------------------
def _zscore(x: np.ndarray, eps: float) -> np.ndarray:
    """eq. zscore: (x - mean over experts) / (std over experts + eps), population std."""
    mu = x.mean()
    sigma = np.sqrt(((x - mu) ** 2).mean())
    return (x - mu) / (sigma + eps)


def layer_terms(D_l, C_l, top_k: int, tau: float = 1.0, eps: float = 1e-8) -> dict:
    """Per-layer intermediates u, A, c, du, dc, s, p (all [F][...]) for D_l [F][E], C_l [F][E][E]."""
    D_l = np.asarray(D_l, dtype=np.float64)
    C_l = np.asarray(C_l, dtype=np.float64)
    F, E = D_l.shape
    u = np.zeros((F, E))
    A = np.zeros((F, E, E))
    for f in range(F):
        n_f = D_l[f].sum() / top_k                           # tokens of family f
        if n_f > 0:
            u[f] = D_l[f] / (n_f * top_k)                    # relative dispatch frequency
            A[f] = C_l[f] / n_f                              # pair frequency per token
            np.fill_diagonal(A[f], 0.0)
    c = np.abs(A).sum(axis=2)                                # c_e = sum_e' |A(e, e')|
    du = np.zeros((F, E))
    dc = np.zeros((F, E))
    s = np.zeros((F, E))
    for f in range(F):
        others = [g for g in range(F) if g != f]
        du[f] = u[f] - u[others].sum(axis=0) / (F - 1)       # eq. usage-coact-advantage
        dc[f] = c[f] - c[others].sum(axis=0) / (F - 1)       # eq. coact-advantage
        s[f] = _zscore(du[f], eps) + _zscore(dc[f], eps)     # eqs. zscore, soft-score
    z = s / tau                                              # eq. family-pref (max-shifted softmax)
    w = np.exp(z - z.max(axis=0, keepdims=True))
    p = w / w.sum(axis=0, keepdims=True)                     # [F][E]
    return dict(u=u, A=A, c=c, du=du, dc=dc, s=s, p=p)


def reweight(D, C, top_k: int, alpha: float = 0.25, tau: float = 1.0, eps: float = 1e-8):
    """Returns pref [L][E][F], a_tilde [L][E][E], a_hat [L][E][E] (float64)."""
    D = _np(D, np.float64)
    C = _np(C, np.float64)
    F, L, E = D.shape
    if F < 2:
        raise ValueError("the advantages of eq. usage-coact-advantage need at least two families")
    pref = np.zeros((L, E, F))
    a_hat = np.zeros((L, E, E))
    a_tilde = np.zeros((L, E, E))
    for l in range(L):
        t = layer_terms(D[:, l], C[:, l], top_k, tau, eps)
        A, p = t["A"], t["p"]
        pref[l] = p.T
        a_bar = A.sum(axis=0) / F                            # pooled co-activation
        off = ~np.eye(E, dtype=bool)
        mx = a_bar[off].max() if E > 1 else 0.0
        ah = a_bar / mx if mx > 0 else np.zeros((E, E))
        a_task = p.T @ p                                     # eq. same-family-kernel: P P^T
        a_hat[l] = ah
        a_tilde[l] = (1.0 - alpha) * ah + alpha * (a_task * ah)   # eq. task-modulated-graph
    return pref, a_tilde, a_hat


# ------------------------------------------------------------------------------------------------
# scoring
# ------------------------------------------------------------------------------------------------
def placement_load(D, primary, n_gpus: int):
    """Snapshot loads of the serving guard: load_ref[p][l][m] = number of dispatches, summed over
    families, of the experts whose primary GPU is m (every expert served by its primary)."""
    D = _np(D, np.int64)
    prim = _np(primary, np.uint8)
    F, L, E = D.shape
    P = prim.shape[0]
    out = np.zeros((P, L, n_gpus), dtype=np.int64)
    dsum = D.sum(axis=0)                                     # [L][E]
    for p in range(P):
        for l in range(L):
            for e in range(E):
                out[p, l, prim[p, l, e]] += dsum[l, e]
    return out


def score(trace, fam_off, n_experts: int, home_start, home_size, n_gpus: int, primary,
          secondary=None, load_ref=None, theta=(3, 20), p_range=None, stats=False):
    """Returns dict(cost_home [P], cost_span [P], load [P][L][G], cost_home_fam [P][F], err) (int64).
    Only placements in p_range = (p0, p1) are scored (others left zero).  stats=True adds the
    per-token statistics of App. C per family: span_fam, cross_fam, home_mass_fam ([P][F])."""
    tr = _np(trace, np.int16)
    L, N, k = tr.shape
    off = _np(fam_off, np.int64)
    F = off.size - 1
    hs = _np(home_start, np.int32)
    hz = _np(home_size, np.int32)
    prim = _np(primary, np.uint8)
    P = prim.shape[0]
    if secondary is not None and secondary.shape[-1] > 0:
        sec = _np(secondary, np.uint8)
        R = sec.shape[-1]
        ref = _np(load_ref, np.int64)
    else:
        sec, R, ref = None, 0, None
    p0, p1 = p_range if p_range is not None else (0, P)
    cost_home = np.zeros(P, dtype=np.int64)
    cost_span = np.zeros(P, dtype=np.int64)
    load = np.zeros((P, L, n_gpus), dtype=np.int64)
    fam = np.zeros((P, F), dtype=np.int64)
    st = [np.zeros((P, F), dtype=np.int64) for _ in range(3)] if stats else [None, None, None]
    tn, td = theta if theta is not None else (0, 0)
    err = _load().oracle_score(_ptr(tr), N, L, k, n_experts, _ptr(off), F, _ptr(hs), _ptr(hz), n_gpus, P, p0, p1,
                               _ptr(prim), _ptr(sec), R, _ptr(ref), int(tn), int(td),
                               _ptr(cost_home), _ptr(cost_span), _ptr(load), _ptr(fam), *[_ptr(a) for a in st])
    out = dict(cost_home=cost_home, cost_span=cost_span, load=load, cost_home_fam=fam, err=int(err))
    if stats:
        out.update(span_fam=st[0], cross_fam=st[1], home_mass_fam=st[2])
    return out


def score_online(trace, fam_off, n_experts: int, home_start, home_size, n_gpus: int, primary,
                 secondary=None, rho: float = 0.995, theta=(3, 20), state=None, p_range=None):
    """Sequential serving with decayed per-GPU loads (Sec. 3.4, eq. load-update); see
    oracle_score_online in tacg_oracle.c.  state: float64 [P][L][G] initial loads (None = zero).
    Returns dict(cost_home, cost_span, load, cost_home_fam, state (final loads), err)."""
    tr = _np(trace, np.int16)
    L, N, k = tr.shape
    off = _np(fam_off, np.int64)
    F = off.size - 1
    hs = _np(home_start, np.int32)
    hz = _np(home_size, np.int32)
    prim = _np(primary, np.uint8)
    P = prim.shape[0]
    if secondary is not None and secondary.shape[-1] > 0:
        sec = _np(secondary, np.uint8)
        R = sec.shape[-1]
    else:
        sec, R = None, 0
    p0, p1 = p_range if p_range is not None else (0, P)
    st_in = None if state is None else _np(state, np.float64)
    st_out = np.zeros((P, L, n_gpus), dtype=np.float64)
    cost_home = np.zeros(P, dtype=np.int64)
    cost_span = np.zeros(P, dtype=np.int64)
    load = np.zeros((P, L, n_gpus), dtype=np.int64)
    fam = np.zeros((P, F), dtype=np.int64)
    tn, td = theta if theta is not None else (0, 0)
    err = _load().oracle_score_online(_ptr(tr), N, L, k, n_experts, _ptr(off), F, _ptr(hs), _ptr(hz), n_gpus, P,
                                      p0, p1, _ptr(prim), _ptr(sec), R, float(rho), int(tn), int(td), _ptr(st_in),
                                      _ptr(st_out), _ptr(cost_home), _ptr(cost_span), _ptr(load), _ptr(fam))
    return dict(cost_home=cost_home, cost_span=cost_span, load=load, cost_home_fam=fam, state=st_out,
                err=int(err))


# ------------------------------------------------------------------------------------------------
# Jain, MaxVio, Comm. Red.
# ------------------------------------------------------------------------------------------------
def jain_maxvio(loads: np.ndarray):
    """eqs. jain and maxvio over the last axis (per-GPU loads).  All-zero rows: Jain 1, MaxVio 0."""
    Lm = np.asarray(loads, dtype=np.float64)
    G = Lm.shape[-1]
    tot = Lm.sum(axis=-1)
    sq = (Lm ** 2).sum(axis=-1)
    with np.errstate(invalid="ignore", divide="ignore"):
        jain = np.where(sq > 0, tot ** 2 / (G * sq), 1.0)
        mean = tot / G
        maxvio = np.where(tot > 0, (Lm.max(axis=-1) - mean) / mean, 0.0)
    return jain, maxvio


def jain(load, per_layer: bool = False):
    """Jain and MaxVio of load [P][L][G]: over sum_l (-> [P]) or per layer (-> [P][L])."""
    ld = _np(load, np.int64)
    if per_layer:
        return jain_maxvio(ld)
    return jain_maxvio(ld.sum(axis=1))


def comm_reduction(comm_base, comm_method):
    """eq. comm-red, in percent."""
    return (np.asarray(comm_base, dtype=np.float64) - np.asarray(comm_method, dtype=np.float64)) \
        / np.asarray(comm_base, dtype=np.float64) * 100.0


# ------------------------------------------------------------------------------------------------
# grouping objective
# ------------------------------------------------------------------------------------------------
def grouping_objective(a_tilde, primary, n_gpus: int):
    """Within-group affinity of eq. grouping-objective for every placement and layer:
    obj[p][l] = sum over GPUs m of sum over ordered pairs e != e' both placed on m of a_tilde[l][e][e']
    (float64; literal loops over the members of each GPU)."""
    at = np.asarray(a_tilde, dtype=np.float64)
    prim = np.asarray(primary)
    P, L, E = prim.shape
    out = np.zeros((P, L), dtype=np.float64)
    for p in range(P):
        for l in range(L):
            members = [[] for _ in range(n_gpus)]
            for e in range(E):
                members[int(prim[p, l, e])].append(e)
            total = 0.0
            for m in range(n_gpus):
                for e in members[m]:
                    for e2 in members[m]:
                        if e2 != e:
                            total += at[l, e, e2]
            out[p, l] = total
    return out


# ------------------------------------------------------------------------------------------------
# GESR identification scores
# ------------------------------------------------------------------------------------------------
def gesr_scores(D, C, top_k: int):
    """Centrality, cross-family consistency and task-specific deviation of every expert (Sec. 3.4,
    eq. generic-score), per layer, in float64:
      Cent(e) = sum_e' A-bar(e, e'),    A-bar = mean over families of A_f (zero diagonal);
      Cons(e) = mean over families of cos(A_f(e, :), A-bar(e, :))   (0 when either row is zero);
      Spec(e) = max over families of || A_f(e, :) - A-bar(e, :) ||_2.
    Returns cent, cons, spec, each [L][E]."""
    D = _np(D, np.float64)
    C = _np(C, np.float64)
    F, L, E = D.shape
    cent = np.zeros((L, E))
    cons = np.zeros((L, E))
    spec = np.zeros((L, E))
    for l in range(L):
        A = layer_terms(D[:, l], C[:, l], top_k, 1.0, 1e-8)["A"]     # [F][E][E], zero diagonal
        a_bar = A.sum(axis=0) / F
        for e in range(E):
            cent[l, e] = a_bar[e].sum()
            nb = np.sqrt((a_bar[e] ** 2).sum())
            cs = 0.0
            worst = 0.0
            for f in range(F):
                na = np.sqrt((A[f, e] ** 2).sum())
                cs += float(A[f, e] @ a_bar[e]) / (na * nb) if na > 0 and nb > 0 else 0.0
                worst = max(worst, float(np.sqrt(((A[f, e] - a_bar[e]) ** 2).sum())))
            cons[l, e] = cs / F
            spec[l, e] = worst
    return cent, cons, spec


# ------------------------------------------------------------------------------------------------
# motivation diagnostics
# ------------------------------------------------------------------------------------------------
def activation_distance(D, top_k: int):
    """Frobenius distance between the expert-activation distributions of every two families
    (App. H, auxiliary motivation metrics): P_f[l][e] = D_f[l][e] / N_{f,l} (the probability that a
    token of family f activates expert e at layer l; 0 for an empty family), dist[i][j] = ||P_i - P_j||_F
    over all layers and experts.  float64 [F][F]."""
    D = _np(D, np.float64)
    F, L, E = D.shape
    Pm = np.zeros((F, L, E))
    for f in range(F):
        for l in range(L):
            n = D[f, l].sum() / top_k
            if n > 0:
                Pm[f, l] = D[f, l] / n
    dist = np.zeros((F, F))
    for i in range(F):
        for j in range(F):
            dist[i, j] = np.sqrt(((Pm[i] - Pm[j]) ** 2).sum())
    return dist


def top_pairs(C, top_n: int = 64):
    """The top_n most frequently co-activated expert pairs of every family and layer: pairs e < e'
    with a positive count, by count (descending), ties by pair index e * E + e' (ascending); the set
    listed in increasing pair index, padded with -1.  int64 [F][L][top_n]."""
    C = _np(C, np.int64)
    F, L, E, _ = C.shape
    out = np.full((F, L, top_n), -1, dtype=np.int64)
    iu, ju = np.triu_indices(E, k=1)
    idx = iu * E + ju
    for f in range(F):
        for l in range(L):
            cnt = C[f, l][iu, ju]
            keep = cnt > 0
            order = np.lexsort((idx[keep], -cnt[keep]))[:top_n]
            sel = np.sort(idx[keep][order])
            out[f, l, :sel.size] = sel
    return out


def pair_jaccard(C, top_n: int = 64):
    """Jaccard overlap of the top_n co-activated pair sets of every two families, per layer
    (App. H): |T_i & T_j| / |T_i | T_j| (1 when both sets are empty).  float64 [L][F][F]."""
    T = top_pairs(C, top_n)
    F, L, _ = T.shape
    out = np.zeros((L, F, F))
    for l in range(L):
        for i in range(F):
            a = set(int(x) for x in T[i, l] if x >= 0)
            for j in range(F):
                b = set(int(x) for x in T[j, l] if x >= 0)
                u = len(a | b)
                out[l, i, j] = len(a & b) / u if u else 1.0
    return out

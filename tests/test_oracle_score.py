"""Pins of the oracle's placement scoring, GESR candidate choice, loads, Jain and MaxVio (CPU only).

Scoring follows the per-token dispatch sets of App. C (cards_l = GPUs serving the token's experts at
layer l; cross-group dispatch count max(0, |cards_l| - 1)) and the serving rule of Sec. 3.4 (eqs.
mean-load, feasible-set and the fallback to the full candidate set).  The exact choice among
feasible candidates is a reading of that passage (local first, then the anchor, then the least loaded),
so the GESR rule is pinned by hand-built cases and an independent brute force, not by the paper.
"""
from fractions import Fraction
from math import comb
import numpy as np
import pytest

from paper_2606_01007_amd import synth

NONE = 0xFF


def brute_score(tr, off, E, hs, hz, G, prim, sec=None, ref=None, theta=(3, 20)):
    """Independent pure-Python scorer with sets and exact fractions."""
    L, N, k = tr.shape
    P = prim.shape[0]
    F = len(off) - 1
    ch = np.zeros(P, dtype=np.int64)
    cs = np.zeros(P, dtype=np.int64)
    load = np.zeros((P, L, G), dtype=np.int64)
    fam = np.zeros((P, F), dtype=np.int64)
    for p in range(P):
        for l in range(L):
            if ref is not None and theta[1] > 0:
                lbar = Fraction(int(ref[p, l].sum()), G)
                bound = (1 + Fraction(theta[0], theta[1])) * lbar
                feas = {m for m in range(G) if ref[p, l, m] <= bound}
            else:
                feas = set(range(G))
            cands = {}
            for e in range(E):
                c = [int(prim[p, l, e])]
                if sec is not None:
                    c += [int(g) for g in sec[p, l, e] if g != NONE]
                cands[e] = c
            for f in range(F):
                for t in range(off[f], off[f + 1]):
                    h = int(hs[f] + (t - off[f]) % hz[f])
                    ids = [int(x) for x in tr[l, t]]
                    gpu = {}
                    R = set()
                    for s, e in enumerate(ids):
                        if len(cands[e]) == 1:
                            gpu[s] = cands[e][0]
                            R.add(gpu[s])
                    for s, e in enumerate(ids):
                        if s in gpu:
                            continue
                        FC = set(cands[e]) & feas or set(cands[e])
                        if FC & R:
                            pick = min(FC & R)
                        elif h in FC:
                            pick = h
                        else:
                            pick = min(FC, key=lambda m: (int(ref[p, l, m]), m))
                        gpu[s] = pick
                        R.add(pick)
                    ch[p] += len(R - {h})
                    cs[p] += len(R) - 1
                    fam[p, f] += len(R - {h})
                    for s in range(k):
                        load[p, l, gpu[s]] += 1
    return ch, cs, load, fam


def _check(oracle_mod, tr, off, E, hs, hz, G, prim, sec=None, ref=None, theta=(3, 20)):
    r = oracle_mod.score(tr, off, E, hs, hz, G, prim, sec, ref, theta)
    assert r["err"] == 0
    ch, cs, load, fam = brute_score(np.asarray(tr), off, E, hs, hz, G, prim, sec, ref, theta)
    np.testing.assert_array_equal(r["cost_home"], ch)
    np.testing.assert_array_equal(r["cost_span"], cs)
    np.testing.assert_array_equal(r["load"], load)
    np.testing.assert_array_equal(r["cost_home_fam"], fam)
    return r


def test_tiny_config_brute(oracle_mod):
    w = synth.make_workload("tiny")
    ps = w.placement_sets[0]
    _check(oracle_mod, w.trace_serve.numpy(), w.fam_off_serve, 8, ps["home_start"], ps["home_size"], 4,
           ps["primary"])


@pytest.mark.parametrize("name,setidx", [("qwen15", 0), ("qwen15", 1), ("qwen3_30b", 0), ("deepseek_v3", 0)])
def test_gesr_configs_brute(oracle_mod, name, setidx):
    """Replicated presets at small size: oracle == brute force with the guard on, off and tight."""
    cfg = synth.CONFIGS[name]
    w = synth.make_workload(name, n_tokens=cfg.F * 23, layers=2, n_place=3)
    ps = w.placement_sets[setidx]
    G = ps["n_gpus"]
    D, C, _ = oracle_mod.coact(w.trace_serve, w.fam_off_serve, cfg.E)
    ref = oracle_mod.placement_load(D, ps["primary"], G)
    for theta in [(3, 20), (0, 0), (0, 1)]:
        _check(oracle_mod, w.trace_serve.numpy(), w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G,
               ps["primary"], ps["secondary"], ref, theta)


def test_loads_without_replicas_equal_counts(oracle_mod):
    """With single candidates, load[p][l][m] = sum of D over experts whose primary is m, and every
    (p, l) row of loads sums to N k."""
    w = synth.make_workload("deepseek16b", n_tokens=8 * 300, layers=3, n_place=5)
    ps = w.placement_sets[0]
    D, _, _ = oracle_mod.coact(w.trace_serve, w.fam_off_serve, 64)
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 64, ps["home_start"], ps["home_size"], 8, ps["primary"])
    expect = oracle_mod.placement_load(D, ps["primary"], 8)
    np.testing.assert_array_equal(r["load"], expect)
    assert np.all(r["load"].sum(axis=2) == 8 * 300 * 6)
    np.testing.assert_array_equal(r["cost_home_fam"].sum(axis=1), r["cost_home"])


def test_bounds_and_replica_load_totals(oracle_mod):
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", n_tokens=16 * 40, layers=2, n_place=3)
    ps = w.placement_sets[0]
    G, k, N, L = 32, cfg.k, 16 * 40, 2
    D, _, _ = oracle_mod.coact(w.trace_serve, w.fam_off_serve, cfg.E)
    ref = oracle_mod.placement_load(D, ps["primary"], G)
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G,
                         ps["primary"], ps["secondary"], ref)
    assert np.all(r["load"].sum(axis=2) == N * k)
    assert np.all(r["cost_home"] >= 0) and np.all(r["cost_home"] <= N * L * min(k, G - 1))
    assert np.all(r["cost_span"] >= 0) and np.all(r["cost_span"] <= N * L * (min(k, G) - 1))


def test_all_experts_home_is_free(oracle_mod):
    """Family f only routes to experts placed on its own anchor GPU f (bands of one GPU):
    cost_home = cost_span = 0."""
    E, k, G, F = 8, 2, 4, 4
    prim = (np.arange(E) // 2).astype(np.uint8)[None, None].repeat(2, axis=1)    # expert e on GPU e // 2
    n = 50
    tr = np.zeros((2, F * n, k), dtype=np.int16)
    for f in range(F):
        tr[:, f * n:(f + 1) * n] = [2 * f, 2 * f + 1]
    hs, hz = synth.home_bands(F, G)
    r = _check(oracle_mod, tr, synth.fam_offsets([n] * F), E, hs, hz, G, prim)
    assert r["cost_home"][0] == 0 and r["cost_span"][0] == 0


def test_single_gpu_is_free(oracle_mod):
    w = synth.make_workload("tiny")
    prim = np.zeros((2, 2, 8), dtype=np.uint8)
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 8, [0, 0, 0], [1, 1, 1], 1, prim)
    assert np.all(r["cost_home"] == 0) and np.all(r["cost_span"] == 0)


def test_gpu_relabelling(oracle_mod):
    """Without replicas, renaming GPUs (and the anchors with them) permutes loads and keeps costs."""
    w = synth.make_workload("qwen3_30b", n_tokens=16 * 30, layers=2, n_place=3)
    ps = w.placement_sets[0]
    G = 8
    hs, hz = np.arange(16, dtype=np.int32) % G, np.ones(16, dtype=np.int32)
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 128, hs, hz, G, ps["primary"])
    perm = np.random.default_rng(3).permutation(G).astype(np.uint8)
    r2 = oracle_mod.score(w.trace_serve, w.fam_off_serve, 128, perm[hs].astype(np.int32), hz, G, perm[ps["primary"]])
    np.testing.assert_array_equal(r2["cost_home"], r["cost_home"])
    np.testing.assert_array_equal(r2["cost_span"], r["cost_span"])
    np.testing.assert_array_equal(r2["load"][:, :, perm], r["load"])


@pytest.mark.parametrize("E,k,G,cap", [(64, 6, 8, 8), (60, 4, 4, 15), (60, 4, 6, 10), (128, 8, 8, 16), (256, 8, 32, 8)])
def test_uniform_routing_closed_form(oracle_mod, E, k, G, cap):
    """Uniform k-subsets: P(GPU m is touched) = 1 - C(E - c_m, k) / C(E, k), so the mean span per
    token-layer is sum_m P_m - 1 and the mean non-anchor count is sum_{m != h} P_m.  Check the
    oracle's totals within 5 standard errors (the per-token-layer variance is at most k^2 / 4)."""
    N, L = 6000, 2
    tr = synth.uniform_trace(E, k, L, N, seed=E * 100 + G).numpy()
    caps = synth.capacities(E, G, cap)
    prim = synth.contiguous_placement(E, caps)[None, None].repeat(L, axis=1)
    pm = np.array([1 - comb(E - int(c), k) / comb(E, k) for c in caps])
    h = 0
    r = oracle_mod.score(tr, [0, N], E, [h], [1], G, prim)
    n = N * L
    se = k / 2 / np.sqrt(n)
    assert abs(r["cost_span"][0] / n - (pm.sum() - 1)) < 5 * se
    assert abs(r["cost_home"][0] / n - (pm.sum() - pm[h])) < 5 * se


# ---------------------------------------------------------------------------------------------
# hand-built GESR cases: G = 4, E = 4, k = 2, one family with a one-GPU band at anchor `h`
# ---------------------------------------------------------------------------------------------
def _gesr_case(oracle_mod, tokens, prim_row, sec_rows, ref_row, h, theta=(3, 20)):
    E, G = 4, 4
    tr = np.array(tokens, dtype=np.int16)[None]
    prim = np.array(prim_row, dtype=np.uint8)[None, None]
    sec = np.full((1, 1, E, 2), NONE, dtype=np.uint8)
    for e, rows in sec_rows.items():
        sec[0, 0, e, :len(rows)] = rows
    ref = np.array(ref_row, dtype=np.int64)[None, None]
    r = _check(oracle_mod, tr, [0, len(tokens)], E, [h], [1], G, prim, sec, ref, theta)
    return r


def test_gesr_local_replica_preferred(oracle_mod):
    # expert 0 -> GPU 0; expert 1 candidates {1, 0}; token {0, 1}: GPU 0 is already accessed
    r = _gesr_case(oracle_mod, [[0, 1]], [0, 1, 2, 3], {1: [0]}, [1, 1, 1, 1], h=2)
    assert r["cost_span"][0] == 0 and list(r["load"][0, 0]) == [2, 0, 0, 0]


def test_gesr_guard_excludes_overloaded(oracle_mod):
    # GPU 0 has 4x the mean load: infeasible, so expert 1 stays on its primary GPU 1
    r = _gesr_case(oracle_mod, [[0, 1]], [0, 1, 2, 3], {1: [0]}, [100, 0, 0, 0], h=2)
    assert r["cost_span"][0] == 1 and list(r["load"][0, 0]) == [1, 1, 0, 0]
    # guard disabled (theta_den = 0): local choice again
    r = _gesr_case(oracle_mod, [[0, 1]], [0, 1, 2, 3], {1: [0]}, [100, 0, 0, 0], h=2, theta=(0, 0))
    assert r["cost_span"][0] == 0


def test_gesr_fallback_when_nothing_feasible(oracle_mod):
    # both candidates of expert 1 ({1, 0}) overloaded: fall back to the full set -> local GPU 0
    r = _gesr_case(oracle_mod, [[0, 1]], [0, 1, 2, 3], {1: [0]}, [100, 100, 0, 0], h=2)
    assert r["cost_span"][0] == 0 and list(r["load"][0, 0]) == [2, 0, 0, 0]


def test_gesr_anchor_then_least_loaded(oracle_mod):
    # token {2, 1}: expert 2 on GPU 2, expert 1 candidates {1, 0, 3}; no candidate is local.
    # anchor 3 is a feasible candidate -> 3
    r = _gesr_case(oracle_mod, [[2, 1]], [0, 1, 2, 3], {1: [0, 3]}, [5, 5, 5, 5], h=3)
    assert list(r["load"][0, 0]) == [0, 0, 1, 1]
    # anchor 2 is not a candidate -> least loaded feasible candidate: GPU 0 (load 1) beats 1 and 3
    r = _gesr_case(oracle_mod, [[2, 1]], [0, 1, 2, 3], {1: [0, 3]}, [1, 5, 5, 5], h=2)
    assert list(r["load"][0, 0]) == [1, 0, 1, 0]
    # ties go to the lowest GPU number
    r = _gesr_case(oracle_mod, [[2, 1]], [0, 1, 2, 3], {1: [3, 0]}, [4, 4, 0, 4], h=2)
    assert list(r["load"][0, 0]) == [1, 0, 1, 0]


def test_gesr_slot_order_and_lowest_local(oracle_mod):
    # both slots replicated: expert 1 {1, 2}, expert 3 {3, 2}; anchor 0 not a candidate.
    # slot 0 (expert 3): nothing local, least loaded of {3, 2} is 2; slot 1 (expert 1) then finds 2 local.
    r = _gesr_case(oracle_mod, [[3, 1]], [0, 1, 2, 3], {1: [2], 3: [2]}, [6, 6, 5, 6], h=0)
    assert list(r["load"][0, 0]) == [0, 0, 2, 0] and r["cost_span"][0] == 0 and r["cost_home"][0] == 1
    # with two local feasible candidates (3 and 0, listed in that order) the lower GPU number wins
    r = _gesr_case(oracle_mod, [[0, 3, 1]], [0, 1, 2, 3], {1: [3, 0]}, [1, 1, 1, 1], h=2)
    assert list(r["load"][0, 0]) == [2, 0, 0, 1] and r["cost_span"][0] == 1


def test_table_errors_flagged(oracle_mod):
    w = synth.make_workload("tiny")
    ps = w.placement_sets[0]
    prim = ps["primary"].copy()
    prim[1, 0, 3] = 4
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 8, ps["home_start"], ps["home_size"], 4, prim)
    assert r["err"] & oracle_mod.ERR_TABLE


# ---------------------------------------------------------------------------------------------
# per-token trace statistics of App. C (cross-group dispatches, cross-family layers, home-family
# dispatch mass) per family
# ---------------------------------------------------------------------------------------------
def brute_stats(tr, off, E, hs, hz, G, prim, sec=None, ref=None, theta=(3, 20)):
    """Independent pure-Python statistics: resolve every slot as in brute_score, then apply the
    three definitions with Python sets."""
    L, N, k = tr.shape
    P = prim.shape[0]
    F = len(off) - 1
    span = np.zeros((P, F), dtype=np.int64)
    cross = np.zeros((P, F), dtype=np.int64)
    mass = np.zeros((P, F), dtype=np.int64)
    bands = [set(range(int(hs[f]), int(hs[f]) + int(hz[f]))) for f in range(F)]
    for p in range(P):
        for l in range(L):
            if ref is not None and theta[1] > 0:
                bound = (1 + Fraction(theta[0], theta[1])) * Fraction(int(ref[p, l].sum()), G)
                feas = {m for m in range(G) if ref[p, l, m] <= bound}
            else:
                feas = set(range(G))
            cands = {e: [int(prim[p, l, e])] + ([int(g) for g in sec[p, l, e] if g != NONE] if sec is not None
                                                 else []) for e in range(E)}
            for f in range(F):
                for t in range(off[f], off[f + 1]):
                    h = int(hs[f] + (t - off[f]) % hz[f])
                    ids = [int(x) for x in tr[l, t]]
                    gpu = {s: cands[e][0] for s, e in enumerate(ids) if len(cands[e]) == 1}
                    R = set(gpu.values())
                    for s, e in enumerate(ids):
                        if s in gpu:
                            continue
                        FC = set(cands[e]) & feas or set(cands[e])
                        pick = min(FC & R) if FC & R else (h if h in FC else
                                                            min(FC, key=lambda m: (int(ref[p, l, m]), m)))
                        gpu[s] = pick
                        R.add(pick)
                    span[p, f] += len(R) - 1
                    cross[p, f] += not any(R <= b for b in bands)
                    mass[p, f] += sum(gpu[s] in bands[f] for s in range(k))
    return span, cross, mass


def _check_stats(oracle_mod, tr, off, E, hs, hz, G, prim, sec=None, ref=None, theta=(3, 20)):
    r = oracle_mod.score(tr, off, E, hs, hz, G, prim, sec, ref, theta, stats=True)
    assert r["err"] == 0
    span, cross, mass = brute_stats(np.asarray(tr), off, E, hs, hz, G, prim, sec, ref, theta)
    np.testing.assert_array_equal(r["span_fam"], span)
    np.testing.assert_array_equal(r["cross_fam"], cross)
    np.testing.assert_array_equal(r["home_mass_fam"], mass)
    np.testing.assert_array_equal(r["span_fam"].sum(axis=1), r["cost_span"])
    return r


def test_trace_stats_hand_worked(oracle_mod):
    """G = 4 in two bands {0, 1} and {2, 3}; expert e on GPU e; k = 2, one layer.
    family 0: {0,1} (inside band 0, 2 home slots), {0,2} (spans both, 1 home slot);
    family 1: {2,3} (inside, 2), {1,3} (spans, 1), {3,2} (inside, 2)."""
    tr = np.array([[[0, 1], [0, 2], [2, 3], [1, 3], [3, 2]]], dtype=np.int16)
    prim = np.arange(4, dtype=np.uint8)[None, None]
    r = oracle_mod.score(tr, [0, 2, 5], 4, [0, 2], [2, 2], 4, prim, stats=True)
    assert r["err"] == 0
    np.testing.assert_array_equal(r["span_fam"], [[2, 3]])
    np.testing.assert_array_equal(r["cross_fam"], [[1, 1]])
    np.testing.assert_array_equal(r["home_mass_fam"], [[3, 5]])


@pytest.mark.parametrize("name,setidx", [("tiny", 0), ("qwen15", 0), ("qwen15", 1), ("deepseek_v3", 0)])
def test_trace_stats_brute(oracle_mod, name, setidx):
    cfg = synth.CONFIGS[name]
    w = synth.make_workload(name, n_tokens=cfg.F * 19, layers=2, n_place=3)
    ps = w.placement_sets[setidx]
    G = ps["n_gpus"]
    ref = None
    if ps["secondary"] is not None:
        D, _, _ = oracle_mod.coact(w.trace_serve, w.fam_off_serve, cfg.E)
        ref = oracle_mod.placement_load(D, ps["primary"], G)
    _check_stats(oracle_mod, w.trace_serve.numpy(), w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G,
                 ps["primary"], ps["secondary"], ref)


def test_trace_stats_mass_from_counts(oracle_mod):
    """Without replicas every slot of expert e goes to its primary, so the home-family mass is the
    family's dispatch count of the experts placed in its band: sum_l sum_{e: prim(e) in band f} D_f[l][e]
    (D from the independent counting pass)."""
    w = synth.make_workload("qwen3_30b", n_tokens=16 * 40, layers=3, n_place=4)
    ps = w.placement_sets[0]
    G = ps["n_gpus"]
    D, _, _ = oracle_mod.coact(w.trace_serve, w.fam_off_serve, 128)
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 128, ps["home_start"], ps["home_size"], G, ps["primary"],
                         stats=True)
    hs, hz = ps["home_start"], ps["home_size"]
    for p in range(ps["primary"].shape[0]):
        inb = [(ps["primary"][p] >= hs[f]) & (ps["primary"][p] < hs[f] + hz[f]) for f in range(len(hs))]
        expect = [int((D[f] * inb[f]).sum()) for f in range(len(hs))]
        np.testing.assert_array_equal(r["home_mass_fam"][p], expect)


def test_trace_stats_degenerate_bands(oracle_mod):
    """One band holding every GPU: no layer spans two families and every slot is home mass.
    One GPU per band (G = F): a layer is cross-family exactly when it touches two or more GPUs."""
    w = synth.make_workload("deepseek16b", n_tokens=8 * 50, layers=2, n_place=3)
    ps = w.placement_sets[0]
    N, L, k, G, F = 8 * 50, 2, 6, 8, 8
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 64, [0] * F, [G] * F, G, ps["primary"], stats=True)
    assert np.all(r["cross_fam"] == 0)
    np.testing.assert_array_equal(r["home_mass_fam"].sum(axis=1), [N * L * k] * 3)
    r = oracle_mod.score(w.trace_serve, w.fam_off_serve, 64, np.arange(F), [1] * F, G, ps["primary"], stats=True)
    tr = w.trace_serve.numpy()
    for p in range(3):
        n_multi = sum(len({int(ps["primary"][p, l, e]) for e in tr[l, t]}) >= 2 for l in range(L) for t in range(N))
        assert int(r["cross_fam"][p].sum()) == n_multi

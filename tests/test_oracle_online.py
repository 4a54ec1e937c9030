"""Pins of the oracle's sequential serving rule with decayed loads (Sec. 3.4, eqs. mean-load,
feasible-set, load-update), CPU only.

The choice among feasible candidates follows the same reading as the snapshot rule (local, then
the anchor, then the least loaded); only the loads differ: they are the decayed per-GPU dispatch
loads of the tokens already served, in trace order.  The pins are a hand-worked sequence, the
reduction to the snapshot rule when nothing is replicated, an exact rational brute force, and the
carry of the load state across trace chunks.
"""
from fractions import Fraction

import numpy as np
import pytest

from paper_2606_01007_amd import synth


def _one_replicated_expert(n_tok):
    """G = 3; expert 0 has candidates {0, 1}, expert 1 sits on GPU 2; every token picks expert 0;
    one family whose anchor band is GPU 2 (not a candidate)."""
    tr = np.zeros((1, n_tok, 1), dtype=np.int16)
    prim = np.array([[[0, 2]]], dtype=np.uint8)
    sec = np.array([[[[1], [0xFF]]]], dtype=np.uint8)
    return tr, prim, sec


def test_hand_worked_alternation(oracle_mod):
    # rho = 1/2, theta = 3/20, so the guard is 60 L_m <= 23 S:
    #   t0: L = (0, 0, 0): both feasible, nothing reached, anchor 2 not a candidate -> least loaded,
    #       tie -> GPU 0;                              L = (1, 0, 0)
    #   t1: S = 1: 60 > 23 excludes GPU 0 -> 1;         L = (1/2, 1, 0)
    #   t2: S = 3/2: 30 <= 34.5 keeps 0, 60 > 34.5 drops 1 -> 0;   L = (5/4, 1/2, 0)
    #   t3: S = 7/4: 75 > 40.25 drops 0 -> 1;           L = (5/8, 5/4, 0)
    #   t4: S = 15/8: 37.5 <= 43.125 keeps 0, 75 drops 1 -> 0;    L = (21/16, 5/8, 0)
    tr, prim, sec = _one_replicated_expert(5)
    r = oracle_mod.score_online(tr, [0, 5], 2, [2], [1], 3, prim, sec, rho=0.5, theta=(3, 20))
    assert r["err"] == 0
    np.testing.assert_array_equal(r["load"][0, 0], [3, 2, 0])
    np.testing.assert_array_equal(r["state"][0, 0], [21 / 16, 5 / 8, 0.0])
    assert r["cost_span"][0] == 0 and r["cost_home"][0] == 5


def test_decay_zero_uses_last_token_only(oracle_mod):
    # rho = 0: the loads are the previous token's dispatches, so the choice alternates 0, 1, 0, ...
    # even with the guard off (the least-loaded fallback decides)
    tr, prim, sec = _one_replicated_expert(6)
    r = oracle_mod.score_online(tr, [0, 6], 2, [2], [1], 3, prim, sec, rho=0.0, theta=(0, 0))
    np.testing.assert_array_equal(r["load"][0, 0], [3, 3, 0])
    np.testing.assert_array_equal(r["state"][0, 0], [0.0, 1.0, 0.0])


def test_initial_state_steers_first_choice(oracle_mod):
    tr, prim, sec = _one_replicated_expert(1)
    st = np.array([[[5.0, 1.0, 0.0]]])
    r = oracle_mod.score_online(tr, [0, 1], 2, [2], [1], 3, prim, sec, rho=0.5, theta=(3, 20), state=st)
    np.testing.assert_array_equal(r["load"][0, 0], [0, 1, 0])
    np.testing.assert_array_equal(r["state"][0, 0], [2.5, 1.5, 0.0])


def test_guard_boundary_is_inclusive(oracle_mod):
    # eq. feasible-set keeps a GPU whose load equals (1 + theta) times the mean.  G = 3, theta = 0,
    # loads (2, 1, 0): mean 1, so GPU 1 sits on the boundary (feasible), GPU 2 below it, GPU 0 above.
    # One token picks expert 0 (only on GPU 1, so GPU 1 is reached) and expert 1 (candidates GPU 2 and
    # GPU 1): the lowest reached feasible candidate is GPU 1, and the token stays on one GPU.  Were
    # the boundary excluded, expert 1 would go to GPU 2 and the token would span two GPUs.
    tr = np.array([[[0, 1]]], dtype=np.int16)
    prim = np.array([[[1, 2, 0, 0]]], dtype=np.uint8)
    sec = np.array([[[[0xFF], [1], [0xFF], [0xFF]]]], dtype=np.uint8)
    st = np.array([[[2.0, 1.0, 0.0]]])
    r = oracle_mod.score_online(tr, [0, 1], 4, [0], [1], 3, prim, sec, rho=0.5, theta=(0, 1), state=st)
    assert r["err"] == 0
    np.testing.assert_array_equal(r["load"][0, 0], [0, 2, 0])
    assert r["cost_span"][0] == 0 and r["cost_home"][0] == 1
    np.testing.assert_array_equal(r["state"][0, 0], [1.0, 2.5, 0.0])


def test_without_replicas_equals_snapshot_rule(oracle_mod):
    w = synth.make_workload("qwen15", n_tokens=3000, n_place=5, layers=2)
    ps = w.placement_sets[0]
    a = oracle_mod.score(w.trace_serve, w.fam_off_serve, 60, ps["home_start"], ps["home_size"], 4, ps["primary"])
    b = oracle_mod.score_online(w.trace_serve, w.fam_off_serve, 60, ps["home_start"], ps["home_size"], 4,
                                ps["primary"], rho=0.995)
    for key in ("cost_home", "cost_span", "load", "cost_home_fam"):
        np.testing.assert_array_equal(a[key], b[key])
    # the final loads are the decayed dispatch counts: each GPU's state is at most k / (1 - rho)
    assert (b["state"] >= 0).all() and (b["state"].sum(axis=2) <= 4 / 0.005 + 1e-9).all()


def _brute(trace, fam_off, E, hs, hz, G, prim, sec, rho, theta):
    """Independent exact evaluation with rational loads (for dyadic rho the float64 arithmetic of the
    oracle is exact on these short traces, so the two must agree bit for bit)."""
    L, N, k = trace.shape
    P = prim.shape[0]
    R = sec.shape[-1]
    tn, td = theta
    rho = Fraction(rho)
    cost_home = np.zeros(P, np.int64)
    cost_span = np.zeros(P, np.int64)
    load = np.zeros((P, L, G), np.int64)
    state = np.zeros((P, L, G))
    for p in range(P):
        for l in range(L):
            Lm = [Fraction(0)] * G
            cands = []
            for e in range(E):
                c = [int(prim[p, l, e])] + [int(g) for g in sec[p, l, e] if g != 0xFF]
                cands.append(c)
            for f in range(len(fam_off) - 1):
                for t in range(fam_off[f], fam_off[f + 1]):
                    h = hs[f] + (t - fam_off[f]) % hz[f]
                    ids = [int(x) for x in trace[l, t]]
                    S = sum(Lm)
                    feas = [True] * G if td == 0 else [td * G * Lm[m] <= (td + tn) * S for m in range(G)]
                    gpu = {}
                    for s, e in enumerate(ids):
                        if len(cands[e]) == 1:
                            gpu[s] = cands[e][0]
                    reached = set(gpu.values())
                    for s, e in enumerate(ids):
                        if s in gpu:
                            continue
                        fc = sorted(m for m in cands[e] if feas[m]) or sorted(cands[e])
                        local = [m for m in fc if m in reached]
                        if local:
                            pick = local[0]
                        elif h in fc:
                            pick = h
                        else:
                            pick = min(fc, key=lambda m: (Lm[m], m))
                        gpu[s] = pick
                        reached.add(pick)
                    cost_span[p] += len(reached) - 1
                    cost_home[p] += len(reached - {h})
                    delta = [0] * G
                    for s in range(k):
                        load[p, l, gpu[s]] += 1
                        delta[gpu[s]] += 1
                    Lm = [rho * Lm[m] + delta[m] for m in range(G)]
            state[p, l] = [float(x) for x in Lm]
    return cost_home, cost_span, load, state


@pytest.mark.parametrize("E,k,G,R,n_rep,counts,rho,theta,seed", [
    (8, 2, 4, 2, 3, [9, 7, 11], 0.5, (3, 20), 1),
    (12, 3, 6, 3, 6, [13, 0, 12], 0.75, (3, 20), 2),
    (16, 4, 8, 2, 16, [10, 10], 0.5, (1, 10), 3),
    (10, 5, 5, 1, 4, [6, 5], 0.875, (0, 0), 4),        # short: 7/8 grows 3 bits a token
])
def test_matches_rational_brute_force(oracle_mod, E, k, G, R, n_rep, counts, rho, theta, seed):
    rng = np.random.default_rng(seed)
    L, P = 2, 4
    off = synth.fam_offsets(counts)
    N = int(off[-1])
    tr = np.stack([np.stack([rng.choice(E, k, replace=False) for _ in range(N)]) for _ in range(L)]).astype(np.int16)
    tr = tr.reshape(L, N, k)
    cap = -(-E // G)
    prim = synth.random_placements(P, L, E, G, cap, seed)
    rep = np.stack([np.sort(rng.choice(E, n_rep, replace=False)) for _ in range(L)])
    sec = synth.random_secondaries(prim, G, rep, R, seed + 7)
    hs, hz = synth.home_bands(len(counts), G)
    r = oracle_mod.score_online(tr, off, E, hs, hz, G, prim, sec, rho=rho, theta=theta)
    assert r["err"] == 0
    ch, cs, ld, st = _brute(tr, off, E, hs, hz, G, prim, sec, rho, theta)
    np.testing.assert_array_equal(r["cost_home"], ch)
    np.testing.assert_array_equal(r["cost_span"], cs)
    np.testing.assert_array_equal(r["load"], ld)
    np.testing.assert_array_equal(r["state"], st)
    assert (r["load"].sum(axis=2) == N * k).all()


def test_chunks_carry_the_state(oracle_mod):
    # one family: scoring the first 700 tokens and then the rest from the carried loads equals scoring
    # the whole trace in one call
    w = synth.make_workload("deepseek_v3", n_tokens=1600, n_place=3, layers=2)
    ps = w.placement_sets[0]
    tr = w.trace_serve.numpy()[:, :1600]
    args = (256, [16], [2], 32, ps["primary"], ps["secondary"])
    whole = oracle_mod.score_online(tr, [0, 1600], *args, rho=0.995)
    a = oracle_mod.score_online(np.ascontiguousarray(tr[:, :700]), [0, 700], *args, rho=0.995)
    b = oracle_mod.score_online(np.ascontiguousarray(tr[:, 700:]), [0, 900], *args, rho=0.995, state=a["state"])
    np.testing.assert_array_equal(a["load"] + b["load"], whole["load"])
    np.testing.assert_array_equal(b["state"], whole["state"])

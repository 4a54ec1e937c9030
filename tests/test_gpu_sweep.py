"""A seeded sweep over random shapes: every entry point of the hot path (co-activation counts,
reweighting, snapshot scoring with its App. C statistics, decayed-load scoring, Jain / MaxVio and the
grouping objective) against the oracle on the same inputs.

The shapes are drawn to reach the kernels' branches in combination: expert counts on both sides of
the 64 / 128 launch thresholds, every top-k width from 1 to 16 (packed ids of one to four words, the
matrix-core paths at E <= 64 from k = 4 and at E <= 128 for k = 8 to 12), one to five small families
with empty ones, 1 to 32 GPUs with narrow and wide bands, zero to four secondaries with up to 16
replicated experts, the guard on and off, and decay factors 0, 0.5 and 0.995.  A large-shape variant draws up to eight families of up
to 60,000 tokens (some nearly empty), so that several co-activation workgroups meet at segment
boundaries and the scoring kernel runs many pieces.  Counts, costs, loads and the final float64
loads are compared exactly; float outputs within the tolerances of the other parity tests.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2606_01007_amd as tacg
from paper_2606_01007_amd import synth

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build()


def _err(e):
    torch.cuda.synchronize()
    return int(e.item()) & 0xFFFFFFFF


def _u32(t):
    return tacg.as_u32(t).cpu().numpy()


def _draw(seed):
    rng = np.random.default_rng(7000 + seed)
    E = int(rng.choice([2, 5, 8, 13, 33, 60, 64, 65, 100, 128, 129, 200, 256]))
    k = int(rng.integers(1, min(E, 16) + 1))
    L = int(rng.integers(1, 4))
    F = int(rng.integers(1, 6))
    counts = [int(rng.integers(0, 700)) if rng.random() > 0.15 else 0 for _ in range(F)]
    if sum(counts) == 0:
        counts[0] = 257
    G = int(rng.choice([1, 2, 3, 4, 7, 8, 9, 16, 31, 32]))
    cap = -(-E // G) + int(rng.integers(0, 3))
    P = int(rng.integers(1, 300))
    R = int(rng.integers(0, min(4, G - 1) + 1))
    n_rep = min(int(rng.integers(1, 17)), E) if R > 0 else 0
    theta = [(3, 20), (0, 0), (1, 10)][int(rng.integers(0, 3))]
    rho = [0.0, 0.5, 0.995][int(rng.integers(0, 3))]
    return dict(E=E, k=k, L=L, counts=counts, G=G, cap=cap, P=P, R=R, n_rep=n_rep, theta=theta, rho=rho)


def _draw_large(seed):
    """Larger families (5,000 to 60,000 tokens, some nearly empty): several co-activation workgroups
    per segment boundary and many scoring pieces."""
    rng = np.random.default_rng(9000 + seed)
    E = int(rng.choice([60, 64, 100, 128, 129, 200, 256]))
    k = int(rng.integers(2, min(E, 16) + 1))
    L = int(rng.integers(1, 4))
    F = int(rng.integers(1, 9))
    counts = [int(rng.integers(5000, 60000)) if rng.random() > 0.15 else int(rng.integers(0, 50)) for _ in range(F)]
    G = int(rng.choice([2, 4, 8, 16, 32]))
    cap = -(-E // G) + int(rng.integers(0, 3))
    P = int(rng.integers(1, 300))
    R = int(rng.integers(0, min(4, G - 1) + 1))
    n_rep = min(int(rng.integers(1, 17)), E) if R > 0 else 0
    theta = [(3, 20), (0, 0), (1, 10)][int(rng.integers(0, 3))]
    rho = [0.0, 0.5, 0.995][int(rng.integers(0, 3))]
    return dict(E=E, k=k, L=L, counts=counts, G=G, cap=cap, P=P, R=R, n_rep=n_rep, theta=theta, rho=rho)


# seeds drawn: 256 and 16 by default; TACG_SWEEP_SMALL / TACG_SWEEP_LARGE widen the sweep
N_SMALL = int(os.environ.get("TACG_SWEEP_SMALL", "256"))
N_LARGE = int(os.environ.get("TACG_SWEEP_LARGE", "16"))


@pytest.mark.parametrize("seed", range(N_SMALL))
def test_random_shape_sweep(seed):
    _check(_draw(seed), seed)


@pytest.mark.parametrize("seed", range(N_LARGE))
def test_random_large_shape_sweep(seed):
    _check(_draw_large(seed), seed)


def _check(c, seed):
    E, k, L, G, P, R = c["E"], c["k"], c["L"], c["G"], c["P"], c["R"]
    _say(f"sweep seed={seed} {c}")
    off = synth.fam_offsets(c["counts"])
    F = len(c["counts"])
    g = torch.Generator(device="cpu").manual_seed(900 + seed)
    tr = torch.topk(torch.rand((L, int(off[-1]), E), generator=g), k, dim=2).indices.to(torch.int16)
    tr_g = tr.cuda()

    # co-activation counts
    Do, Co, eo = oracle.coact(tr, off, E)
    assert eo == 0
    D, C, err = tacg.coact_build(tr_g, off, E)
    assert _err(err) == 0
    np.testing.assert_array_equal(_u32(D), Do)
    np.testing.assert_array_equal(_u32(C), Co)

    # reweighting (two or more families) and the grouping objective of the placements on its graph
    prim = synth.random_placements(P, L, E, G, c["cap"], 300 + seed)
    prim_t = torch.as_tensor(prim).cuda()
    if F >= 2:
        po, ato, _ = oracle.reweight(Do, Co, k, alpha=0.25)
        pref, at, _ = tacg.reweight(D, C, k, alpha=0.25)
        np.testing.assert_allclose(pref.cpu().double().numpy(), po, rtol=1e-5, atol=1e-30)
        np.testing.assert_allclose(at.cpu().double().numpy(), ato, rtol=1e-5, atol=1e-30)
        at32 = ato.astype(np.float32)
        got = tacg.group_objective(torch.as_tensor(at32).cuda(), prim_t, G)
        ref = oracle.grouping_objective(at32.astype(np.float64), prim, G)
        np.testing.assert_allclose(got.cpu().numpy(), ref, rtol=1e-12, atol=1e-300)

    # snapshot scoring with GESR replicas and its App. C statistics
    rng = np.random.default_rng(500 + seed)
    rep = np.stack([np.sort(rng.choice(E, c["n_rep"], replace=False)) for _ in range(L)]) if R > 0 else None
    sec = synth.random_secondaries(prim, G, rep, R, 600 + seed) if R > 0 else None
    sec_t = torch.as_tensor(sec).cuda() if sec is not None else None
    hs, hz = synth.home_bands(F, G)
    ref_o = oracle.placement_load(Do, prim, G) if R > 0 else None
    ref_g = tacg.placement_load(D, prim_t, G, err=err) if R > 0 else None
    ro = oracle.score(tr, off, E, hs, hz, G, prim, sec, ref_o, c["theta"], stats=True)
    assert ro["err"] == 0
    out = tacg.eval_placements(tr_g, off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=c["theta"])
    assert _err(out["err"]) == 0
    if R > 0:
        np.testing.assert_array_equal(ref_g.cpu().numpy(), ref_o)
    for key in ("cost_home", "cost_span", "cost_home_fam"):
        np.testing.assert_array_equal(out[key].cpu().numpy(), ro[key], err_msg=key)
    np.testing.assert_array_equal(_u32(out["load"]), ro["load"])
    if F <= G:  # distinct family bands tile the GPUs
        st = tacg.eval_trace_stats(tr_g, off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=c["theta"])
        assert _err(st["err"]) == 0
        for key in ("span_fam", "cross_fam", "home_mass_fam", "cost_span"):
            np.testing.assert_array_equal(st[key].cpu().numpy(), ro[key], err_msg=key)

    # Jain / MaxVio of the loads
    jn, mv = tacg.jain_index(out["load"])
    jo, vo = oracle.jain(ro["load"])
    np.testing.assert_allclose(jn.cpu().double().numpy(), jo, rtol=1e-5)
    np.testing.assert_allclose(mv.cpu().double().numpy(), vo, rtol=1e-5, atol=1e-30)

    # decayed-load scoring
    oo = oracle.score_online(tr, off, E, hs, hz, G, prim, sec, rho=c["rho"], theta=c["theta"])
    assert oo["err"] == 0
    on = tacg.eval_online(tr_g, off, E, hs, hz, G, prim_t, sec_t, rho=c["rho"], theta=c["theta"])
    assert _err(on["err"]) == 0
    for key in ("cost_home", "cost_span", "cost_home_fam", "state"):
        np.testing.assert_array_equal(on[key].cpu().numpy(), oo[key], err_msg=key)
    np.testing.assert_array_equal(_u32(on["load"]), oo["load"])

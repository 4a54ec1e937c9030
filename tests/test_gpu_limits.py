"""GPU parity at the documented limits of the C ABI, every entry point on one input: 64 families (some
empty, others of one token), 256 experts, top-16, 32 simulated GPUs, 4 secondaries per replicated
expert, 16 replicated experts per layer, a ragged placement count, and the top-4096 pair sets."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2606_01007_amd as tacg
from paper_2606_01007_amd import synth

pytestmark = pytest.mark.gpu

E, K, L, G, CAP, R, NREP, P, F = 256, 16, 2, 32, 8, 4, 16, 130, 64


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def case():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build()
    rng = np.random.default_rng(64)
    counts = rng.integers(0, 120, size=F)
    counts[[3, 17, 40]] = 0
    counts[[5, 63]] = 1
    off = synth.fam_offsets(counts)
    N = int(off[-1])
    g = torch.Generator(device="cpu").manual_seed(64)
    tr = torch.topk(torch.rand((L, N, E), generator=g), K, dim=2).indices.to(torch.int16)
    prim = synth.random_placements(P, L, E, G, CAP, 164)
    rep = np.stack([np.sort(rng.choice(E, NREP, replace=False)) for _ in range(L)])
    sec = synth.random_secondaries(prim, G, rep, R, 264)
    hs, hz = synth.home_bands(F, G)
    _say(f"limits case: F={F} N={N} E={E} k={K} G={G} R={R} P={P}")
    return dict(off=off, tr=tr, prim=prim, sec=sec, hs=hs, hz=hz)


def _err(e):
    torch.cuda.synchronize()
    return int(e.item()) & 0xFFFFFFFF


def test_limits_counts_and_reweight(case):
    tr, off = case["tr"], case["off"]
    D, C, err = tacg.coact_build(tr.cuda(), off, E)
    assert _err(err) == 0
    Do, Co, e = oracle.coact(tr, off, E)
    assert e == 0
    np.testing.assert_array_equal(tacg.as_u32(D).cpu().numpy(), Do)
    np.testing.assert_array_equal(tacg.as_u32(C).cpu().numpy(), Co)
    pref, at, ah = tacg.reweight(D, C, K, want_hat=True)
    po, ato, aho = oracle.reweight(Do, Co, K)
    for got, ref in ((pref, po), (at, ato), (ah, aho)):
        np.testing.assert_allclose(got.cpu().double().numpy(), ref, rtol=1e-5, atol=1e-30)
    cent, cons, spec = tacg.gesr_scores(D, C, K)
    for got, ref in zip((cent, cons, spec), oracle.gesr_scores(Do, Co, K)):
        np.testing.assert_allclose(got.cpu().numpy(), ref, rtol=1e-12, atol=1e-15)
    dist = tacg.activation_distance(D, K)
    np.testing.assert_allclose(dist.cpu().numpy(), oracle.activation_distance(Do, K), rtol=1e-12, atol=1e-15)
    pairs, jac = tacg.pair_jaccard(C, 4096)
    np.testing.assert_array_equal(pairs.cpu().numpy(), oracle.top_pairs(Co, 4096))
    np.testing.assert_array_equal(jac.cpu().numpy(), oracle.pair_jaccard(Co, 4096))


def test_limits_scoring(case):
    tr, off, prim, sec, hs, hz = (case[k] for k in ("tr", "off", "prim", "sec", "hs", "hz"))
    Do, _, _ = oracle.coact(tr, off, E)
    ref_o = oracle.placement_load(Do, prim, G)
    ro = oracle.score(tr, off, E, hs, hz, G, prim, sec, ref_o, (3, 20), stats=True)
    assert ro["err"] == 0
    prim_t, sec_t = torch.as_tensor(prim).cuda(), torch.as_tensor(sec).cuda()
    D, _, e1 = tacg.coact_build(tr.cuda(), off, E)
    ref_g = tacg.placement_load(D, prim_t, G, err=e1)
    out = tacg.eval_placements(tr.cuda(), off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=(3, 20))
    st = tacg.eval_trace_stats(tr.cuda(), off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=(3, 20))
    assert _err(out["err"]) == 0 and _err(st["err"]) == 0 and _err(e1) == 0
    np.testing.assert_array_equal(ref_g.cpu().numpy(), ref_o)
    for key in ("cost_home", "cost_span", "cost_home_fam"):
        np.testing.assert_array_equal(out[key].cpu().numpy(), ro[key], err_msg=key)
    np.testing.assert_array_equal(tacg.as_u32(out["load"]).cpu().numpy(), ro["load"])
    for key in ("span_fam", "cross_fam", "home_mass_fam", "cost_span"):
        np.testing.assert_array_equal(st[key].cpu().numpy(), ro[key], err_msg=key)
    jn, mv = tacg.jain_index(out["load"])
    jo, vo = oracle.jain(ro["load"])
    np.testing.assert_allclose(jn.cpu().double().numpy(), jo, rtol=1e-5)
    np.testing.assert_allclose(mv.cpu().double().numpy(), vo, rtol=1e-5, atol=1e-30)


def test_limits_online_and_objective(case):
    tr, off, prim, sec, hs, hz = (case[k] for k in ("tr", "off", "prim", "sec", "hs", "hz"))
    oo = oracle.score_online(tr, off, E, hs, hz, G, prim, sec, rho=0.995, theta=(3, 20))
    assert oo["err"] == 0
    on = tacg.eval_online(tr.cuda(), off, E, hs, hz, G, torch.as_tensor(prim).cuda(), torch.as_tensor(sec).cuda(),
                          rho=0.995, theta=(3, 20))
    assert _err(on["err"]) == 0
    for key in ("cost_home", "cost_span", "cost_home_fam", "state"):
        np.testing.assert_array_equal(on[key].cpu().numpy(), oo[key], err_msg=key)
    np.testing.assert_array_equal(tacg.as_u32(on["load"]).cpu().numpy(), oo["load"])
    Do, Co, _ = oracle.coact(tr, off, E)
    _, ato, _ = oracle.reweight(Do, Co, K)
    at32 = ato.astype(np.float32)
    got = tacg.group_objective(torch.as_tensor(at32).cuda(), torch.as_tensor(prim).cuda(), G)
    ref = oracle.grouping_objective(at32.astype(np.float64), prim, G)
    np.testing.assert_allclose(got.cpu().numpy(), ref, rtol=1e-12, atol=1e-300)

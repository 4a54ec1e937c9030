"""GPU parity at the full workload sizes (the preset shapes at their full token, layer and placement
counts, in the launch configuration the benchmark times; the decayed-load scoring on the benchmark's
sample of the serving trace, its first 2^19 tokens).

The oracle computes the whole of D and C (every family/layer segment, compared bit for bit) and the
activation distance; the reweighted graph, GESR scores, top pairs, Jaccard overlaps and grouping
objective of sampled layers; and fifteen scored placements per placement set over the whole trace
(first and last lanes of placement blocks, interior lanes, every placement position within a lane,
several blocks), two of them with the per-token statistics of App. C, eight with the decayed-load
scoring.  Every other output is checked through
properties that hold at any size (symmetry, diagonal, row sums and totals of the counts; per-layer
load totals and cost bounds of the scores).
"""
import os
import sys
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2606_01007_amd as tacg
from paper_2606_01007_amd import synth

pytestmark = pytest.mark.gpu


_T0 = time.time()
_CAPMAN = None


def _say(msg):
    """Progress line, written past pytest's output capture: each full-size case runs for minutes and
    a run that prints nothing for that long looks hung."""
    line = f"{time.time() - _T0:7.1f}s {msg}"
    if _CAPMAN is not None:
        with _CAPMAN.global_and_fixture_disabled():
            print(line, flush=True)
    else:
        print(line, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu(request):
    global _CAPMAN
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _CAPMAN = request.config.pluginmanager.getplugin("capturemanager")
    oracle.build()


def _u32(t):
    return tacg.as_u32(t)


def sampled_placements(P: int, n_experts: int):
    """Placements compared with the oracle one by one.  The scoring kernel gives each lane two
    placements (four when E <= 64) and each workgroup 64 lanes' worth, so the sample covers the first
    and last lanes of blocks, interior lanes, every position within a lane's group and several blocks."""
    ppl = 4 if n_experts <= 64 else 2
    pb = 64 * ppl
    want = {0, 1, 2, 3, 37, 2 * 37 + 1, pb - 2, pb - 1, pb, pb + 1, P // 2 + 5, P // 2 + 70, (3 * P) // 4 + 43,
            P - 2, P - 1}
    if os.environ.get("TACG_FULLSIZE_BLOCKS"):
        # opt-in (minutes of oracle time per preset): the whole first placement block, every lane and
        # every position within a lane, and the last 64 placements
        want |= set(range(pb)) | set(range(P - 64, P))
    return sorted(p for p in want if 0 <= p < P)


def _runs(ps):
    """Contiguous runs [p0, p1) of a sorted list of placements (one oracle call each)."""
    out = []
    for p in ps:
        if out and out[-1][1] == p:
            out[-1][1] = p + 1
        else:
            out.append([p, p + 1])
    return [tuple(r) for r in out]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["deepseek16b", "qwen15", "qwen3_30b", "deepseek_v3"])
def test_full_size(name):
    cfg = synth.CONFIGS[name]
    _say(f"[{name}] generating full workload")
    w = synth.make_workload(name, device="cuda")
    E, k, L, F = cfg.E, cfg.k, cfg.L, cfg.F
    Ng = w.trace_group.shape[1]

    # ---- co-activation counts: properties and the oracle on every segment ----
    D, C, err = tacg.coact_build(w.trace_group, w.fam_off_group, E)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    Dl, Cl = _u32(D), _u32(C)
    nf = torch.as_tensor(np.diff(w.fam_off_group), device="cuda")
    assert torch.equal(Cl, Cl.transpose(2, 3))
    assert torch.equal(torch.diagonal(Cl, dim1=2, dim2=3), Dl)
    assert torch.equal(Cl.sum(dim=3) - Dl, (k - 1) * Dl)
    assert torch.equal(Dl.sum(dim=2), (nf[:, None] * k).expand(F, L))
    tg = w.trace_group.cpu().numpy()
    _say(f"[{name}] oracle counts of the whole grouping trace")
    Do_all, Co_all, e = oracle.coact(tg, w.fam_off_group, E)
    assert e == 0
    # every (family, layer) segment of D and C, bit for bit
    np.testing.assert_array_equal(Dl.cpu().numpy(), Do_all)
    np.testing.assert_array_equal(Cl.cpu().numpy(), Co_all)
    del Dl, Cl
    _say(f"[{name}] counts ok")

    # ---- reweighting: sampled layers against the oracle (on the oracle's counts) ----
    pref, at, _ = tacg.reweight(D, C, k)
    per_layer = {}
    for l in [0, L - 1]:
        Dol = np.ascontiguousarray(Do_all[:, l:l + 1])
        Col = np.ascontiguousarray(Co_all[:, l:l + 1])
        po, ato, _ = oracle.reweight(Dol, Col, k)
        np.testing.assert_allclose(pref[l].cpu().double().numpy(), po[0], rtol=1e-5, atol=1e-30)
        np.testing.assert_allclose(at[l].cpu().double().numpy(), ato[0], rtol=1e-5, atol=1e-30)
        per_layer[l] = (Dol, Col, ato[0])
    _say(f"[{name}] reweight ok")

    # ---- the auxiliary calls of the benchmark on the full counts: sampled layers against the oracle ----
    cent, cons, spec = tacg.gesr_scores(D, C, k)
    pairs, jac = tacg.pair_jaccard(C, 64)
    dist = tacg.activation_distance(D, k)
    for l, (Dol, Col, ato_l) in per_layer.items():
        co, so, sp = oracle.gesr_scores(Dol, Col, k)
        np.testing.assert_allclose(cent[l].cpu().numpy(), co[0], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(cons[l].cpu().numpy(), so[0], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(spec[l].cpu().numpy(), sp[0], rtol=1e-12, atol=1e-15)
        np.testing.assert_array_equal(pairs[:, l].cpu().numpy(), oracle.top_pairs(Col, 64)[:, 0])
        np.testing.assert_array_equal(jac[l].cpu().numpy(), oracle.pair_jaccard(Col, 64)[0])
    np.testing.assert_allclose(dist.cpu().numpy(), oracle.activation_distance(Do_all, k), rtol=1e-12, atol=1e-15)
    del tg, Do_all, Co_all
    ps = w.placement_sets[0]
    prim0 = torch.as_tensor(ps["primary"]).cuda()
    obj = tacg.group_objective(at, prim0, ps["n_gpus"])           # all placements x layers, as benchmarked
    torch.cuda.synchronize()
    assert bool(torch.isfinite(obj).all()) and bool((obj >= 0).all())
    for l, (_, _, ato_l) in per_layer.items():                    # the oracle's graph on both sides
        a32 = ato_l.astype(np.float32)[None]
        got = tacg.group_objective(torch.as_tensor(a32).cuda(), prim0[:, l:l + 1].contiguous(), ps["n_gpus"])
        ref = oracle.grouping_objective(a32.astype(np.float64), ps["primary"][:, l:l + 1], ps["n_gpus"])
        np.testing.assert_allclose(got.cpu().numpy(), ref, rtol=1e-12, atol=1e-300)
    _say(f"[{name}] auxiliary calls ok")

    # ---- placement scoring at full size: every placement set of the preset ----
    ts = w.trace_serve.cpu().numpy()
    Dso = None
    for ps in w.placement_sets:
        G, P = ps["n_gpus"], ps["primary"].shape[0]
        prim = torch.as_tensor(ps["primary"]).cuda()
        sec = torch.as_tensor(ps["secondary"]).cuda() if ps["secondary"] is not None else None
        ref_g = ref_o = None
        if sec is not None:
            Ds, _, e1 = tacg.coact_build(w.trace_serve, w.fam_off_serve, E)
            ref_g = tacg.placement_load(Ds, prim, G, err=e1)
            if Dso is None:
                Dso, _, _ = oracle.coact(ts, w.fam_off_serve, E)
            ref_o = oracle.placement_load(Dso, ps["primary"], G)
        out = tacg.eval_placements(w.trace_serve, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, prim,
                                   sec, ref_g, theta=(3, 20))
        jn, mv = tacg.jain_index(out["load"])
        torch.cuda.synchronize()
        assert int(out["err"].item()) == 0
        if ref_g is not None:
            np.testing.assert_array_equal(ref_g.cpu().numpy(), ref_o)
        load = _u32(out["load"])
        Ns = w.trace_serve.shape[1]
        assert bool((load.sum(dim=2) == Ns * k).all())
        ch, cs = out["cost_home"], out["cost_span"]
        assert bool((ch >= 0).all()) and bool((ch <= Ns * L * min(k, G - 1)).all())
        assert bool((cs >= 0).all()) and bool((cs <= Ns * L * (min(k, G) - 1)).all())
        assert torch.equal(out["cost_home_fam"].sum(dim=1), ch)
        # the per-token statistics of App. C (their own kernel variant) in the same launch configuration
        st = tacg.eval_trace_stats(w.trace_serve, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, prim,
                                   sec, ref_g, theta=(3, 20))
        torch.cuda.synchronize()
        assert int(st["err"].item()) == 0
        for key in ("cost_home", "cost_span", "load"):
            assert torch.equal(st[key], out[key]), key
        assert torch.equal(st["span_fam"].sum(dim=1), cs)
        sample = sampled_placements(P, n_experts=E)
        with_stats = {sample[0], sample[len(sample) // 2]}  # App. C statistics: ~8x the oracle's scoring time
        for p0, p1 in _runs(sample):
            _say(f"[{name}] oracle scoring placements {p0}..{p1 - 1} of {P} (G={G})")
            ro = oracle.score(ts, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, ps["primary"],
                              ps["secondary"], ref_o, (3, 20), p_range=(p0, p1))
            assert ro["err"] == 0
            for p in range(p0, p1):
                assert int(ch[p]) == int(ro["cost_home"][p])
                assert int(cs[p]) == int(ro["cost_span"][p])
                np.testing.assert_array_equal(load[p].cpu().numpy(), ro["load"][p])
                np.testing.assert_array_equal(out["cost_home_fam"][p].cpu().numpy(), ro["cost_home_fam"][p])
                jo, vo = oracle.jain(ro["load"][p:p + 1])
                np.testing.assert_allclose(float(jn[p]), jo[0], rtol=1e-5)
                np.testing.assert_allclose(float(mv[p]), vo[0], rtol=1e-5, atol=1e-30)
        for p in sorted(with_stats):
            _say(f"[{name}] oracle App. C statistics of placement {p} of {P} (G={G})")
            ro = oracle.score(ts, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, ps["primary"],
                              ps["secondary"], ref_o, (3, 20), p_range=(p, p + 1), stats=True)
            assert ro["err"] == 0
            for key in ("span_fam", "cross_fam", "home_mass_fam"):
                np.testing.assert_array_equal(st[key][p].cpu().numpy(), ro[key][p], err_msg=key)
    _say(f"[{name}] scoring ok")

    # ---- decayed-load scoring on the benchmark's sample: all placements, sampled ones vs the oracle ----
    ps = w.placement_sets[0]
    G, P = ps["n_gpus"], ps["primary"].shape[0]
    n = min(1 << 19, w.trace_serve.shape[1])
    tr = w.trace_serve[:, :n].contiguous()
    off = np.minimum(np.asarray(w.fam_off_serve, dtype=np.int64), n)
    prim = torch.as_tensor(ps["primary"]).cuda()
    sec = torch.as_tensor(ps["secondary"]).cuda() if ps["secondary"] is not None else None
    on = tacg.eval_online(tr, off, E, ps["home_start"], ps["home_size"], G, prim, sec, rho=0.995, theta=(3, 20))
    torch.cuda.synchronize()
    assert int(on["err"].item()) == 0
    load = _u32(on["load"])
    assert bool((load.sum(dim=2) == n * k).all())
    assert torch.equal(on["cost_home_fam"].sum(dim=1), on["cost_home"])
    tsn = np.ascontiguousarray(ts[:, :n])
    for p in sampled_placements(P, n_experts=E)[::2]:
        _say(f"[{name}] oracle decayed-load scoring placement {p} of {P} (G={G}, {n} tokens)")
        ro = oracle.score_online(tsn, off, E, ps["home_start"], ps["home_size"], G, ps["primary"], ps["secondary"],
                                 rho=0.995, theta=(3, 20), p_range=(p, p + 1))
        assert ro["err"] == 0
        assert int(on["cost_home"][p]) == int(ro["cost_home"][p])
        assert int(on["cost_span"][p]) == int(ro["cost_span"][p])
        np.testing.assert_array_equal(load[p].cpu().numpy(), ro["load"][p])
        np.testing.assert_array_equal(on["cost_home_fam"][p].cpu().numpy(), ro["cost_home_fam"][p])
        np.testing.assert_array_equal(on["state"][p].cpu().numpy(), ro["state"][p])
    _say(f"[{name}] decayed-load scoring ok")

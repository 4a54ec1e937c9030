"""GPU parity of the per-token trace statistics of App. C (tacg_eval_trace_stats) against the oracle:
per family, the cross-group dispatch count, the layers whose cards span more than one family band
and the home-family dispatch mass, all bit-exact, together with the costs and loads of the same call
(which must also equal tacg_eval_placements)."""
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


def _rand_trace(L, N, k, E, seed):
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.rand((L, N, E), generator=g)
    return torch.topk(x, k, dim=2).indices.to(torch.int16)


def _both(tr, off, E, hs, hz, G, prim, sec=None, theta=(3, 20), expect_err=0):
    """Device statistics vs the oracle's on the same trace and tables (loads for the guard from each
    side's own counting pass)."""
    tr_c = torch.as_tensor(tr).cpu()
    ref_o = None
    if sec is not None:
        Do, _, _ = oracle.coact(tr_c, off, E)
        ref_o = oracle.placement_load(Do, prim, G)
    ro = oracle.score(tr_c, off, E, hs, hz, G, prim, sec, ref_o, theta, stats=True)
    assert ro["err"] == expect_err
    tr_g = tr_c.cuda()
    prim_t = torch.as_tensor(prim).cuda()
    sec_t = torch.as_tensor(sec).cuda() if sec is not None else None
    ref_g = None
    if sec is not None:
        D, _, e1 = tacg.coact_build(tr_g, off, E)
        ref_g = tacg.placement_load(D, prim_t, G, err=e1)
        assert _err(e1) == expect_err
    out = tacg.eval_trace_stats(tr_g, off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=theta)
    assert _err(out["err"]) == expect_err
    for key in ("span_fam", "cross_fam", "home_mass_fam", "cost_home", "cost_span"):
        np.testing.assert_array_equal(out[key].cpu().numpy(), ro[key], err_msg=key)
    np.testing.assert_array_equal(tacg.as_u32(out["load"]).cpu().numpy(), ro["load"])
    plain = tacg.eval_placements(tr_g, off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=theta)
    np.testing.assert_array_equal(plain["cost_span"].cpu().numpy(), out["cost_span"].cpu().numpy())
    np.testing.assert_array_equal(tacg.as_u32(plain["load"]).cpu().numpy(), tacg.as_u32(out["load"]).cpu().numpy())
    return out, ro


def test_trace_stats_hand_worked():
    tr = np.array([[[0, 1], [0, 2], [2, 3], [1, 3], [3, 2]]], dtype=np.int16)
    prim = np.arange(4, dtype=np.uint8)[None, None]
    out, _ = _both(tr, [0, 2, 5], 4, [0, 2], [2, 2], 4, prim)
    np.testing.assert_array_equal(out["span_fam"].cpu().numpy(), [[2, 3]])
    np.testing.assert_array_equal(out["cross_fam"].cpu().numpy(), [[1, 1]])
    np.testing.assert_array_equal(out["home_mass_fam"].cpu().numpy(), [[3, 5]])


@pytest.mark.parametrize("name,setidx,n_place", [
    ("tiny", 0, 16),
    ("deepseek16b", 0, 130),      # E = 64 (the statistics variant scores two placements per lane)
    ("qwen15", 0, 70),            # F = 6 > G = 4: families share one-GPU bands
    ("qwen15", 1, 70),
    ("qwen3_30b", 0, 129),
    ("deepseek_v3", 0, 65),
])
def test_trace_stats_presets(name, setidx, n_place):
    cfg = synth.CONFIGS[name]
    n = cfg.tokens_group if name == "tiny" else cfg.F * 900 + 37
    w = synth.make_workload(name, n_tokens=n, layers=min(cfg.L, 3), n_place=n_place)
    ps = w.placement_sets[setidx]
    _say(f"trace stats {name} set{setidx} P={n_place}")
    _both(w.trace_serve, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], ps["n_gpus"], ps["primary"],
          ps["secondary"])


@pytest.mark.parametrize("name,n_place,dense", [("deepseek16b", 130, False), ("deepseek_v3", 65, False),
                                                ("deepseek_v3", 65, True)])
def test_trace_stats_invalid_ids_not_counted(name, n_place, dense):
    """Token-layers with an id out of range or a repeated id are flagged and left out of every
    statistic, cost and load, as in the oracle: scattered ones, and (dense) a whole layer, a whole
    family and a run of 200 token-layers."""
    cfg = synth.CONFIGS[name]
    w = synth.make_workload(name, n_tokens=cfg.F * 900 + 37, layers=2, n_place=n_place)
    ps = w.placement_sets[0]
    tr = w.trace_serve.clone()
    L, N, k = tr.shape
    rng = np.random.default_rng(23)
    for i in range(30):
        l, t, s = int(rng.integers(L)), int(rng.integers(N)), int(rng.integers(k))
        tr[l, t, s] = [cfg.E, -7, int(tr[l, t, (s + 1) % k])][i % 3]
    tr[:, 64:68, 0] = cfg.E   # a whole group of four
    if dense:
        tr[1, :, 0] = cfg.E
        f0, f1 = int(w.fam_off_serve[1]), int(w.fam_off_serve[2])
        tr[:, f0:f1, k - 1] = tr[:, f0:f1, 0]
        tr[0, 200:400, k // 2] = -5
    _say(f"trace stats invalid ids {name} dense={dense}")
    _both(tr, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], ps["n_gpus"], ps["primary"],
          ps["secondary"], expect_err=tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP)


@pytest.mark.parametrize("band", [2, 4, 8, 32])
def test_trace_stats_band_widths(band):
    """Bands of 2, 4 and 8 GPUs that tile the 32 GPUs (families share a band when there are fewer
    bands than families), and one band holding all 32 (no layer can span two families)."""
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", n_tokens=16 * 700 + 5, layers=2, n_place=65)
    ps = w.placement_sets[0]
    hs = ((np.arange(16) % (32 // band)) * band).astype(np.int32)
    hz = np.full(16, band, np.int32)
    _say(f"trace stats bands of {band}")
    out, _ = _both(w.trace_serve, w.fam_off_serve, cfg.E, hs, hz, 32, ps["primary"], ps["secondary"])
    if band == 32:
        assert int(out["cross_fam"].abs().sum()) == 0


@pytest.mark.parametrize("E,k,L,counts,G,cap,n_rep,R,P,seed", [
    (16, 8, 2, [700, 0, 513], 4, 4, 16, 2, 20, 1),       # every expert replicated
    (16, 16, 1, [300, 301], 8, 2, 16, 3, 9, 2),         # k = 16
    (60, 5, 2, [800, 801], 6, 10, 4, 2, 257, 7),        # E <= 64, odd k, a ragged placement block
    (256, 8, 1, [900, 77], 32, 8, 16, 4, 70, 4),        # G = 32, the most replicated experts
    (40, 1, 2, [500, 500, 1], 5, 8, 6, 2, 33, 5),       # k = 1
    (30, 4, 2, [400, 400], 1, 30, 0, 0, 10, 8),         # G = 1
])
def test_trace_stats_random(E, k, L, counts, G, cap, n_rep, R, P, seed):
    _say(f"trace stats random E={E} k={k} counts={counts} G={G} R={R} P={P}")
    off = synth.fam_offsets(counts)
    tr = _rand_trace(L, int(off[-1]), k, E, seed)
    prim = synth.random_placements(P, L, E, G, cap, seed + 100)
    sec = None
    if R > 0:
        rng = np.random.default_rng(seed)
        rep = np.stack([np.sort(rng.choice(E, n_rep, replace=False)) for _ in range(L)])
        sec = synth.random_secondaries(prim, G, rep, R, seed + 200)
    hs, hz = synth.home_bands(len(counts), G)
    _both(tr, off, E, hs, hz, G, prim, sec)


def test_trace_stats_empty_trace():
    E, k, L, G, F = 32, 4, 2, 4, 3
    tr = torch.zeros((L, 0, k), dtype=torch.int16, device="cuda")
    prim = torch.as_tensor(synth.random_placements(5, L, E, G, 8, 1)).cuda()
    hs, hz = synth.home_bands(F, G)
    out = tacg.eval_trace_stats(tr, synth.fam_offsets([0] * F), E, hs, hz, G, prim)
    assert _err(out["err"]) == 0
    for key in ("span_fam", "cross_fam", "home_mass_fam"):
        assert int(out[key].abs().sum()) == 0


def test_trace_stats_bands_must_tile():
    w = synth.make_workload("tiny", device="cuda")
    prim = torch.as_tensor(w.placement_sets[0]["primary"]).cuda()
    with pytest.raises(tacg.TacgError) as e:
        tacg.eval_trace_stats(w.trace_serve, w.fam_off_serve, 8, [0, 1, 2], [2, 2, 2], 4, prim)
    assert e.value.status == tacg.E_UNSUPPORTED

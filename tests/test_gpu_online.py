"""GPU parity of the scoring with decayed per-GPU loads (tacg_eval_online) against the oracle.

Every output is compared exactly: costs and loads bit for bit, and the final float64 loads bit for
bit too (both sides evaluate the same fused multiply-adds and the same summation order).
"""
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


def _both(tr, off, E, hs, hz, G, prim, sec, rho, theta, state=None, expect_err=0):
    ro = oracle.score_online(tr, off, E, hs, hz, G, prim, sec, rho=rho, theta=theta, state=state)
    assert ro["err"] == expect_err
    st = torch.as_tensor(state).cuda() if state is not None else None
    out = tacg.eval_online(tr.cuda() if isinstance(tr, torch.Tensor) else torch.as_tensor(tr).cuda(), off, E, hs, hz,
                           G, torch.as_tensor(prim).cuda(),
                           torch.as_tensor(sec).cuda() if sec is not None else None, rho=rho, theta=theta, state=st)
    assert _err(out["err"]) == expect_err
    np.testing.assert_array_equal(out["cost_home"].cpu().numpy(), ro["cost_home"])
    np.testing.assert_array_equal(out["cost_span"].cpu().numpy(), ro["cost_span"])
    np.testing.assert_array_equal(tacg.as_u32(out["load"]).cpu().numpy(), ro["load"])
    np.testing.assert_array_equal(out["cost_home_fam"].cpu().numpy(), ro["cost_home_fam"])
    np.testing.assert_array_equal(out["state"].cpu().numpy(), ro["state"])
    return out, ro


def test_hand_worked_alternation():
    tr = np.zeros((1, 5, 1), dtype=np.int16)
    prim = np.array([[[0, 2]]], dtype=np.uint8)
    sec = np.array([[[[1], [0xFF]]]], dtype=np.uint8)
    out, _ = _both(tr, [0, 5], 2, [2], [1], 3, prim, sec, 0.5, (3, 20))
    np.testing.assert_array_equal(tacg.as_u32(out["load"]).cpu().numpy()[0, 0], [3, 2, 0])
    np.testing.assert_array_equal(out["state"].cpu().numpy()[0, 0], [21 / 16, 5 / 8, 0.0])


def test_guard_boundary_is_inclusive():
    """A GPU whose decayed load equals (1 + theta) times the mean stays feasible (loads (2, 1, 0),
    theta = 0): the token's replicated expert joins the GPU it already reaches."""
    tr = np.array([[[0, 1]]], dtype=np.int16)
    prim = np.array([[[1, 2, 0, 0]]], dtype=np.uint8)
    sec = np.array([[[[0xFF], [1], [0xFF], [0xFF]]]], dtype=np.uint8)
    st = np.array([[[2.0, 1.0, 0.0]]])
    out, _ = _both(tr, [0, 1], 4, [0], [1], 3, prim, sec, 0.5, (0, 1), state=st)
    np.testing.assert_array_equal(tacg.as_u32(out["load"]).cpu().numpy()[0, 0], [0, 2, 0])


@pytest.mark.parametrize("E,k,L,counts,G,cap,n_rep,R,P,rho,theta,seed", [
    (16, 8, 2, [700, 0, 513], 4, 4, 16, 2, 20, 0.995, (3, 20), 1),     # every expert replicated
    (16, 16, 1, [300, 301], 8, 2, 16, 3, 9, 0.9, (3, 20), 2),          # k = 16 (8-bit dispatch counts)
    (64, 6, 2, [1000, 999], 8, 8, 12, 2, 131, 0.995, (1, 10), 3),
    (256, 8, 1, [900, 77], 32, 8, 40, 4, 70, 0.995, (3, 20), 4),       # G = 32, more than 16 replicated
    (40, 1, 2, [500, 500, 1], 5, 8, 6, 2, 33, 0.0, (3, 20), 5),        # k = 1, rho = 0
    (200, 3, 2, [1200, 3], 25, 8, 10, 2, 65, 0.5, (0, 0), 6),          # guard off
    (60, 5, 2, [800, 801], 6, 10, 4, 2, 64, 0.999, (3, 20), 7),
    (30, 4, 2, [400, 400], 1, 30, 0, 0, 10, 0.995, (3, 20), 8),        # G = 1, no replicas
    (256, 8, 1, [600, 300], 32, 8, 100, 2, 64, 0.995, (3, 20), 9),     # more replicated experts than LDS rows
])
def test_online_parity(E, k, L, counts, G, cap, n_rep, R, P, rho, theta, seed):
    _say(f"online E={E} k={k} L={L} counts={counts} G={G} R={R} P={P} rho={rho} theta={theta}")
    off = synth.fam_offsets(counts)
    tr = _rand_trace(L, int(off[-1]), k, E, seed)
    prim = synth.random_placements(P, L, E, G, cap, seed + 100)
    sec = None
    if R > 0:
        rng = np.random.default_rng(seed)
        rep = np.stack([np.sort(rng.choice(E, n_rep, replace=False)) for _ in range(L)])
        sec = synth.random_secondaries(prim, G, rep, R, seed + 200)
    hs, hz = synth.home_bands(len(counts), G)
    _both(tr, off, E, hs, hz, G, prim, sec, rho, theta)


@pytest.mark.parametrize("name,setidx", [("qwen15", 0), ("qwen15", 1), ("qwen3_30b", 0), ("deepseek_v3", 0)])
def test_online_presets(name, setidx):
    cfg = synth.CONFIGS[name]
    _say(f"online preset {name} set {setidx}")
    w = synth.make_workload(name, n_tokens=cfg.F * 700 + 13, layers=2, n_place=70)
    ps = w.placement_sets[setidx]
    _both(w.trace_serve, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], ps["n_gpus"], ps["primary"],
          ps["secondary"], 0.995, (3, 20))


def test_online_state_carry_and_initial_state():
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", n_tokens=4000, layers=2, n_place=64)
    ps = w.placement_sets[0]
    tr = w.trace_serve[:, :4000].contiguous()
    args = (256, [16], [2], 32, ps["primary"], ps["secondary"], 0.995, (3, 20))
    whole, _ = _both(tr, [0, 4000], *args)
    a, _ = _both(tr[:, :1500].contiguous(), [0, 1500], *args)
    b, _ = _both(tr[:, 1500:].contiguous(), [0, 2500], *args, state=a["state"].cpu().numpy())
    np.testing.assert_array_equal(b["state"].cpu().numpy(), whole["state"].cpu().numpy())
    np.testing.assert_array_equal((tacg.as_u32(a["load"]) + tacg.as_u32(b["load"])).cpu().numpy(),
                                  tacg.as_u32(whole["load"]).cpu().numpy())
    # the state buffer may be passed as both input and output
    st = a["state"].clone()
    out = tacg.eval_online(tr[:, 1500:].contiguous().cuda(), [0, 2500], 256, [16], [2], 32,
                           torch.as_tensor(ps["primary"]).cuda(), torch.as_tensor(ps["secondary"]).cuda(),
                           rho=0.995, theta=(3, 20), state=st,
                           out=dict(cost_home=torch.empty(64, dtype=torch.int64, device="cuda"),
                                    cost_span=torch.empty(64, dtype=torch.int64, device="cuda"),
                                    load=torch.empty((64, 2, 32), dtype=torch.int32, device="cuda"),
                                    cost_home_fam=None, state=st))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.cpu().numpy(), whole["state"].cpu().numpy())


@pytest.mark.parametrize("dense", [False, True])
def test_online_invalid_ids_not_served(dense):
    """Token-layers with an id out of range or a repeated id are flagged, not served and leave the
    decayed loads untouched, as in the oracle: every output, the final loads included, is equal.
    Dense: also a whole layer, a whole family and a run of 200 token-layers."""
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", n_tokens=16 * 300 + 11, layers=2, n_place=70)
    ps = w.placement_sets[0]
    tr = w.trace_serve.clone()
    L, N, k = tr.shape
    rng = np.random.default_rng(31)
    for i in range(24):
        l, t, s = int(rng.integers(L)), int(rng.integers(N)), int(rng.integers(k))
        tr[l, t, s] = [cfg.E, -2, int(tr[l, t, (s + 1) % k])][i % 3]
    if dense:
        tr[1, :, 0] = cfg.E
        f0, f1 = int(w.fam_off_serve[1]), int(w.fam_off_serve[2])
        tr[:, f0:f1, k - 1] = tr[:, f0:f1, 0]
        tr[0, 200:400, k // 2] = -5
    _say(f"online invalid ids dense={dense}")
    _both(tr, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], ps["n_gpus"], ps["primary"],
          ps["secondary"], 0.995, (3, 20), expect_err=tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP)


def test_online_errors_flagged():
    w = synth.make_workload("tiny")
    ps = w.placement_sets[0]
    tr = w.trace_serve.clone()
    tr[1, 7, 0] = 99
    out = tacg.eval_online(tr.cuda(), w.fam_off_serve, 8, ps["home_start"], ps["home_size"], 4,
                           torch.as_tensor(ps["primary"]).cuda())
    assert _err(out["err"]) & tacg.ERR_ID_RANGE
    prim = ps["primary"].copy()
    prim[2, 0, 3] = 9
    out = tacg.eval_online(w.trace_serve.cuda(), w.fam_off_serve, 8, ps["home_start"], ps["home_size"], 4,
                           torch.as_tensor(prim).cuda())
    assert _err(out["err"]) & tacg.ERR_TABLE

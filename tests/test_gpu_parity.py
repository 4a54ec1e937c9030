"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same seeded inputs.

Integer outputs (counts, costs, loads) must match bit for bit; preferences, reweighted edges and
Jain / MaxVio (float32 from float64 device arithmetic) within 1e-5 relative of the float64 oracle.
The oracle always computes from the trace itself (its inputs never come from the HIP path).
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

RTOL = 1e-5
ATOL = 1e-30


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(tacg.LIB_PATH):
        pytest.fail("libtacg.so is not built")
    oracle.build()


def _u32(t):
    return tacg.as_u32(t).cpu().numpy()


def _err(e):
    torch.cuda.synchronize()
    return int(e.item()) & 0xFFFFFFFF


def _rand_trace(L, N, k, E, seed, device="cuda"):
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.rand((L, N, E), generator=g)
    return torch.topk(x, k, dim=2).indices.to(torch.int16).to(device)


# ------------------------------------------------------------------------------------------------
# co-activation counts
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("E,k,L,counts,seed", [
    (8, 2, 2, [2048, 2048, 2048], 1),
    (60, 4, 3, [5000, 0, 3001, 777], 2),
    (64, 6, 2, [4096, 9000], 3),
    (13, 1, 2, [300, 200], 4),
    (37, 5, 2, [1000, 1], 5),
    (128, 8, 2, [3333, 4444], 6),
    (256, 8, 2, [5000, 7000, 11], 7),
    (256, 16, 1, [2000], 8),
    (200, 3, 3, [4000, 4000], 9),
    (32, 12, 2, [1500, 500], 10),
    (100, 6, 2, [2500, 1700], 11),
    (129, 7, 3, [999, 3001], 12),
    # several histogram workgroups (one per 32768 token-layers) whose ranges cross segment boundaries
    (256, 8, 3, [30000, 17, 25000], 13),
    (128, 8, 2, [40000, 33000], 14),
    (60, 4, 2, [50000, 20000, 1], 15),
    # on both sides of the matrix-core threshold (E <= 64, k >= 4)
    (65, 6, 2, [3000, 1, 2500], 16),
    (127, 9, 2, [4100, 0, 900], 17),
    (128, 10, 1, [6000, 70], 18),
    (100, 7, 3, [20000, 9000], 19),
    (64, 5, 2, [3000, 3000], 20),
    (33, 16, 1, [2000], 21),
    (64, 3, 2, [4000, 900], 22),
    (64, 4, 2, [4000, 900, 3], 23),
    (32, 4, 3, [2500, 0, 1200], 24),
    (20, 4, 2, [3100, 77], 25),
    # the four-block matrix path (64 < E <= 128, 8 <= k <= 12) and the histogram around it
    (100, 8, 2, [3000, 1, 2200], 26),
    (65, 12, 1, [2600, 900], 27),
    (128, 7, 2, [3000, 2000], 28),
    (128, 13, 1, [2500], 29),
    (97, 6, 2, [3500, 1500], 30),
    # top-6 and top-7 histograms (the lane orders through constant lane masks) at E > 128
    (256, 6, 2, [20000, 30000], 31),
    (160, 7, 2, [15000, 1, 9000], 32),
])
def test_coact_parity(E, k, L, counts, seed):
    _say(f"coact E={E} k={k} L={L} counts={counts}")
    off = synth.fam_offsets(counts)
    tr = _rand_trace(L, int(off[-1]), k, E, seed)
    D, C, err = tacg.coact_build(tr, off, E)
    assert _err(err) == 0
    Do, Co, eo = oracle.coact(tr.cpu(), off, E)
    assert eo == 0
    np.testing.assert_array_equal(_u32(D), Do)
    np.testing.assert_array_equal(_u32(C), Co)


def test_coact_tiny_config():
    w = synth.make_workload("tiny", device="cuda")
    D, C, err = tacg.coact_build(w.trace_group, w.fam_off_group, 8)
    assert _err(err) == 0
    Do, Co, _ = oracle.coact(w.trace_group.cpu(), w.fam_off_group, 8)
    np.testing.assert_array_equal(_u32(D), Do)
    np.testing.assert_array_equal(_u32(C), Co)


@pytest.mark.parametrize("E,k", [(64, 6), (128, 8), (256, 8), (100, 5)])  # both matrix paths, histograms
def test_coact_accumulate_chunks(E, k):
    """Streaming: counting a trace in two token chunks with TACG_ACCUMULATE equals one call."""
    counts = [6000, 4000]
    off = synth.fam_offsets(counts)
    tr = _rand_trace(2, 10000, k, E, 11)
    D, C, _ = tacg.coact_build(tr, off, E)
    # chunk 1: first half of each family; chunk 2: second half (each chunk family-contiguous)
    halves = []
    for part in (0, 1):
        idx, sub_counts = [], []
        for f in range(2):
            a, b = int(off[f]), int(off[f + 1])
            mid = (a + b) // 2
            lo, hi = (a, mid) if part == 0 else (mid, b)
            idx.append(torch.arange(lo, hi))
            sub_counts.append(hi - lo)
        halves.append((tr[:, torch.cat(idx).cuda()].contiguous(), synth.fam_offsets(sub_counts)))
    D2, C2, err = tacg.coact_build(halves[0][0], halves[0][1], E)
    tacg.coact_build(halves[1][0], halves[1][1], E, D=D2, C=C2, accumulate=True, err=err)
    assert _err(err) == 0
    assert torch.equal(D, D2) and torch.equal(C, C2)


def test_coact_repeat_is_deterministic():
    E, k = 256, 8
    tr = _rand_trace(3, 20000, k, E, 12)
    off = [0, 12000, 20000]
    D1, C1, _ = tacg.coact_build(tr, off, E)
    D2, C2, _ = tacg.coact_build(tr, off, E)
    assert torch.equal(D1, D2) and torch.equal(C1, C2)


@pytest.mark.parametrize("E,k,counts,L", [(8, 2, [2048, 2048, 2048], 2), (100, 4, [300, 0, 513, 7], 3),
                                           (256, 8, [600, 1, 900], 2), (13, 1, [700, 300], 2),
                                           (48, 7, [900, 0, 1500, 65], 2), (90, 6, [800, 77, 1200], 2),
                                           (128, 8, [700, 0, 1900, 3], 2)])
def test_coact_repeated_builds_exact(E, k, counts, L):
    """Many short segments flush the workgroup triangles often; every one of repeated builds into the
    same outputs must equal the oracle (a lost or late increment at a flush would show here)."""
    _say(f"coact repeated E={E} k={k} counts={counts} L={L}")
    off = synth.fam_offsets(counts)
    tr = _rand_trace(L, int(off[-1]), k, E, 77)
    Do, Co, _ = oracle.coact(tr.cpu(), off, E)
    D, C, err = tacg.coact_build(tr, off, E)
    for _ in range(12):
        tacg.coact_build(tr, off, E, D=D, C=C, err=err)
        np.testing.assert_array_equal(_u32(C), Co)
        np.testing.assert_array_equal(_u32(D), Do)
    assert _err(err) == 0


@pytest.mark.parametrize("E,k", [(16, 4), (16, 6), (200, 8), (64, 8), (32, 5), (100, 7), (128, 12), (96, 9),
                                 (256, 6), (200, 7)])   # histogram / matrix-core paths
def test_coact_data_errors_flagged(E, k):
    """Repeated and out-of-range ids are flagged; the offending token-layer is skipped, as the oracle
    skips it."""
    tr = _rand_trace(1, 3000, k, E, 13)
    for t, s, v, bit in [(100, 1, None, tacg.ERR_ID_DUP), (7, 3, E, tacg.ERR_ID_RANGE), (9, 2, -3, tacg.ERR_ID_RANGE)]:
        bad = tr.clone()
        bad[0, t, s] = bad[0, t, 0] if v is None else v
        D, C, err = tacg.coact_build(bad, [0, 3000], E)
        assert _err(err) & bit
        Do, Co, eo = oracle.coact(bad.cpu(), [0, 3000], E)
        assert eo & bit
        np.testing.assert_array_equal(_u32(C), Co)
        np.testing.assert_array_equal(_u32(D), Do)


@pytest.mark.parametrize("E,k", [(16, 3), (64, 6), (60, 4), (128, 8), (100, 10), (96, 6), (256, 8), (200, 6)])
def test_coact_dense_invalid(E, k):
    """Invalid token-layers as the rule in places (histogram and matrix-core paths): a whole segment
    out of range, a whole segment with repeated ids, and a run of 300 token-layers across several
    batches of 64; the valid rest is counted exactly as the oracle counts it."""
    off = [0, 1500, 2900, 4100]
    tr = _rand_trace(2, off[-1], k, E, 29)
    tr[1, off[0]:off[1], 0] = E
    tr[0, off[1]:off[2], k - 1] = tr[0, off[1]:off[2], 0]
    tr[1, 2950:3250, k // 2] = -1
    _say(f"coact dense invalid E={E} k={k} matrix={tacg.coact_uses_matrix_cores(E, k)}")
    D, C, err = tacg.coact_build(tr, off, E)
    assert _err(err) == tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP
    Do, Co, eo = oracle.coact(tr.cpu(), off, E)
    assert eo == tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP
    np.testing.assert_array_equal(_u32(D), Do)
    np.testing.assert_array_equal(_u32(C), Co)
    assert int(Do[0, 1].sum()) == 0 and int(Do[1, 0].sum()) == 0


@pytest.mark.parametrize("E,k", [(16, 4), (16, 6), (64, 8), (100, 8), (256, 8)])
def test_coact_empty_trace(E, k):
    tr = torch.zeros((2, 0, k), dtype=torch.int16, device="cuda")
    D, C, err = tacg.coact_build(tr, [0, 0, 0], E)
    assert _err(err) == 0
    assert int(D.abs().sum()) == 0 and int(C.abs().sum()) == 0


# ------------------------------------------------------------------------------------------------
# preferences and graph
# ------------------------------------------------------------------------------------------------
def _close(gpu, ref):
    g = gpu.detach().cpu().double().numpy()
    np.testing.assert_allclose(g, ref, rtol=RTOL, atol=ATOL)


@pytest.mark.parametrize("name,alpha,tau", [("tiny", 0.25, 1.0), ("deepseek16b", 0.25, 1.0),
                                            ("qwen15", 0.0, 0.5), ("qwen3_30b", 0.6, 2.0),
                                            ("deepseek_v3", 0.25, 1.0)])
def test_reweight_parity(name, alpha, tau):
    cfg = synth.CONFIGS[name]
    n = cfg.tokens_group if name == "tiny" else cfg.F * 3000
    w = synth.make_workload(name, device="cuda", n_tokens=n, layers=min(cfg.L, 3))
    _say(f"reweight {name}")
    D, C, err = tacg.coact_build(w.trace_group, w.fam_off_group, cfg.E)
    pref, at, ah = tacg.reweight(D, C, cfg.k, alpha=alpha, tau=tau, want_hat=True)
    assert _err(err) == 0
    Do, Co, _ = oracle.coact(w.trace_group.cpu(), w.fam_off_group, cfg.E)
    po, ato, aho = oracle.reweight(Do, Co, cfg.k, alpha=alpha, tau=tau)
    _close(pref, po)
    _close(at, ato)
    _close(ah, aho)


def test_reweight_empty_family_and_zero_layer():
    E, k = 12, 3
    tr = _rand_trace(2, 900, k, E, 21)
    off = [0, 500, 500, 900]                    # family 1 is empty
    D, C, _ = tacg.coact_build(tr, off, E)
    pref, at, ah = tacg.reweight(D, C, k, want_hat=True)
    Do, Co, _ = oracle.coact(tr.cpu(), off, E)
    po, ato, aho = oracle.reweight(Do, Co, k)
    _close(pref, po)
    _close(at, ato)
    Dz = torch.zeros((3, 1, E), dtype=torch.int32, device="cuda")
    Cz = torch.zeros((3, 1, E, E), dtype=torch.int32, device="cuda")
    pref, at, ah = tacg.reweight(Dz, Cz, k, want_hat=True)
    assert float(at.abs().max()) == 0.0 and float(ah.abs().max()) == 0.0
    _close(pref, np.full((1, E, 3), 1 / 3))


# ------------------------------------------------------------------------------------------------
# placement scoring
# ------------------------------------------------------------------------------------------------
def _score_both(w, ps, E, theta=(3, 20), use_oracle_ref=False, tr=None, expect_err=0):
    G = ps["n_gpus"]
    prim = torch.as_tensor(ps["primary"]).cuda()
    sec = torch.as_tensor(ps["secondary"]).cuda() if ps["secondary"] is not None else None
    tr = w.trace_serve if tr is None else tr
    Do, _, _ = oracle.coact(tr.cpu(), w.fam_off_serve, E)
    ref_o = oracle.placement_load(Do, ps["primary"], G) if sec is not None else None
    ref_g = None
    if sec is not None:
        if use_oracle_ref:
            ref_g = torch.as_tensor(ref_o).cuda()
        else:
            D, _, e1 = tacg.coact_build(tr, w.fam_off_serve, E)
            ref_g = tacg.placement_load(D, prim, G, err=e1)
            assert _err(e1) == expect_err
    out = tacg.eval_placements(tr, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, prim, sec, ref_g,
                               theta=theta)
    assert _err(out["err"]) == expect_err
    ro = oracle.score(tr.cpu(), w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, ps["primary"],
                      ps["secondary"], ref_o, theta)
    assert ro["err"] == expect_err
    if ref_g is not None:
        np.testing.assert_array_equal(ref_g.cpu().numpy(), ref_o)
    np.testing.assert_array_equal(out["cost_home"].cpu().numpy(), ro["cost_home"])
    np.testing.assert_array_equal(out["cost_span"].cpu().numpy(), ro["cost_span"])
    np.testing.assert_array_equal(_u32(out["load"]), ro["load"])
    np.testing.assert_array_equal(out["cost_home_fam"].cpu().numpy(), ro["cost_home_fam"])
    return out, ro


@pytest.mark.parametrize("name,setidx,n_place,theta", [
    ("tiny", 0, 16, (3, 20)),
    ("deepseek16b", 0, 130, (3, 20)),
    ("qwen15", 0, 70, (3, 20)),
    ("qwen15", 1, 70, (0, 0)),
    ("qwen3_30b", 0, 129, (3, 20)),
    ("deepseek_v3", 0, 65, (3, 20)),
    ("deepseek_v3", 0, 3, (0, 1)),
])
def test_eval_parity(name, setidx, n_place, theta):
    cfg = synth.CONFIGS[name]
    n = cfg.tokens_group if name == "tiny" else cfg.F * 1500 + 37
    w = synth.make_workload(name, device="cuda", n_tokens=n, layers=min(cfg.L, 3), n_place=n_place)
    _say(f"eval {name} set{setidx} P={n_place} theta={theta}")
    _score_both(w, w.placement_sets[setidx], cfg.E, theta)


def _plant_invalid(tr, E, seed):
    """A copy of trace tr with invalid token-layers: ids out of range (E, negative), repeated ids, a
    run of four invalid token-layers (one scoring group), one invalid token-layer among three valid
    ones, and the trace's last token-layer."""
    tr = tr.clone()
    L, N, k = tr.shape
    rng = np.random.default_rng(seed)
    spots = [(int(rng.integers(L)), int(rng.integers(N))) for _ in range(40)]
    spots += [(0, t) for t in range(64, 68)] + [(L - 1, 130), (L - 1, N - 1)]
    for i, (l, t) in enumerate(spots):
        s = int(rng.integers(k))
        kind = i % 3
        if kind == 0:
            tr[l, t, s] = E
        elif kind == 1:
            tr[l, t, s] = -1 - int(rng.integers(100))
        else:
            tr[l, t, s] = tr[l, t, (s + 1) % k]
    return tr


@pytest.mark.parametrize("name,setidx,n_place", [("tiny", 0, 16), ("deepseek16b", 0, 130), ("qwen15", 0, 70),
                                                 ("deepseek_v3", 0, 65)])
def test_eval_invalid_ids_not_scored(name, setidx, n_place):
    """A token-layer with an id out of range or a repeated id is flagged and not scored, as in the
    oracle: every cost, load and per-family cost equals the oracle's on a trace with such token-layers
    (the replicated-slot choices and the snapshot loads of the guard skip them too)."""
    cfg = synth.CONFIGS[name]
    n = cfg.tokens_group if name == "tiny" else cfg.F * 1500 + 37
    w = synth.make_workload(name, device="cuda", n_tokens=n, layers=min(cfg.L, 3), n_place=n_place)
    _say(f"eval invalid ids {name} P={n_place}")
    tr = _plant_invalid(w.trace_serve, cfg.E, 17)
    _score_both(w, w.placement_sets[setidx], cfg.E, tr=tr, expect_err=tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP)


def _plant_dense_invalid(tr, E, fam_off):
    """A copy of trace tr where invalid token-layers are the rule in places: every token-layer of
    layer 1 out of range, every token-layer of the second family repeats an id, and a run of 200
    token-layers of layer 0 across several groups of 64 with a negative id."""
    tr = tr.clone()
    L, N, k = tr.shape
    tr[1 % L, :, 0] = E
    f0, f1 = int(fam_off[1]), int(fam_off[2])
    tr[:, f0:f1, k - 1] = tr[:, f0:f1, 0]
    tr[0, 200:400, k // 2] = -5
    return tr


@pytest.mark.parametrize("name,n_place", [("tiny", 16), ("deepseek16b", 130), ("deepseek_v3", 65)])
def test_eval_dense_invalid_ids_not_scored(name, n_place):
    """Whole layers, whole families and long runs of invalid token-layers: every tile of some layers
    is skipped, and costs, loads and per-family costs still equal the oracle's."""
    cfg = synth.CONFIGS[name]
    n = cfg.tokens_group if name == "tiny" else cfg.F * 700 + 37
    w = synth.make_workload(name, device="cuda", n_tokens=n, layers=min(cfg.L, 3), n_place=n_place)
    _say(f"eval dense invalid ids {name} P={n_place}")
    tr = _plant_dense_invalid(w.trace_serve, cfg.E, w.fam_off_serve)
    _score_both(w, w.placement_sets[0], cfg.E, tr=tr, expect_err=tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP)


def test_eval_every_id_invalid():
    """A trace with no valid token-layer: nothing is scored (zero costs and loads), and both error
    bits are raised."""
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", device="cuda", n_tokens=16 * 300 + 5, layers=2, n_place=65)
    tr = w.trace_serve.clone()
    tr[0, :, 0] = cfg.E
    tr[1, :, 1] = tr[1, :, 0]
    _say("eval every id invalid")
    out, _ = _score_both(w, w.placement_sets[0], cfg.E, tr=tr, expect_err=tacg.ERR_ID_RANGE | tacg.ERR_ID_DUP)
    assert int(out["cost_span"].abs().sum()) == 0 and int(out["load"].abs().sum()) == 0


def test_eval_guard_boundary_is_inclusive():
    """Snapshot guard: a GPU whose load equals (1 + theta) times the mean stays feasible (loads
    (2, 1, 0), theta = 0), so the replicated expert joins the GPU the token already reaches."""
    tr = torch.tensor([[[0, 1]]], dtype=torch.int16, device="cuda")
    prim = np.array([[[1, 2, 0, 0]]], dtype=np.uint8)
    sec = np.array([[[[0xFF], [1], [0xFF], [0xFF]]]], dtype=np.uint8)
    ref = np.array([[[2, 1, 0]]], dtype=np.int64)
    out = tacg.eval_placements(tr, [0, 1], 4, [0], [1], 3, torch.as_tensor(prim).cuda(), torch.as_tensor(sec).cuda(),
                               torch.as_tensor(ref).cuda(), theta=(0, 1))
    assert _err(out["err"]) == 0
    ro = oracle.score(tr.cpu(), [0, 1], 4, [0], [1], 3, prim, sec, ref, (0, 1))
    assert ro["err"] == 0
    np.testing.assert_array_equal(_u32(out["load"]), ro["load"])
    np.testing.assert_array_equal(ro["load"][0, 0], [0, 2, 0])
    assert int(out["cost_span"][0]) == int(ro["cost_span"][0]) == 0
    assert int(out["cost_home"][0]) == int(ro["cost_home"][0]) == 1


@pytest.mark.parametrize("band", [1, 2, 4, 8])
def test_eval_band_widths(band):
    """Anchor bands of 1, 2, 4 (fallbacks packed per band position) and 8 GPUs (tested per token),
    with 16 families whose offsets are odd and even."""
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", device="cuda", n_tokens=16 * 1500 + 37, layers=2, n_place=65)
    ps = dict(w.placement_sets[0])
    ps["home_start"] = ((np.arange(16) * band) % 32 // band * band).astype(np.int32)
    ps["home_size"] = np.full(16, band, np.int32)
    _score_both(w, ps, cfg.E)


def test_eval_partial_replication():
    """An expert with secondaries in some placements only: where it has a single candidate it is
    served by its primary before the multi-candidate slots are resolved."""
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", device="cuda", n_tokens=16 * 1200 + 5, layers=2, n_place=70)
    ps = dict(w.placement_sets[0])
    sec = ps["secondary"].copy()
    rng = np.random.default_rng(3)
    drop = rng.random(sec.shape[:3]) < 0.5
    sec[drop] = 0xFF
    sec[:, :, :, 2][rng.random(sec.shape[:3]) < 0.3] = 0xFF       # some experts with fewer secondaries
    ps["secondary"] = sec
    _score_both(w, ps, cfg.E)


def test_eval_with_oracle_snapshot():
    cfg = synth.CONFIGS["deepseek_v3"]
    w = synth.make_workload("deepseek_v3", device="cuda", n_tokens=16 * 800, layers=2, n_place=70)
    _score_both(w, w.placement_sets[0], cfg.E, use_oracle_ref=True)


def test_eval_home_only_and_single_gpu():
    E, k, G, F = 8, 2, 4, 4
    n = 300
    tr = torch.zeros((2, F * n, k), dtype=torch.int16)
    for f in range(F):
        tr[:, f * n:(f + 1) * n, 0] = 2 * f
        tr[:, f * n:(f + 1) * n, 1] = 2 * f + 1
    tr = tr.cuda()
    prim = torch.as_tensor((np.arange(E) // 2).astype(np.uint8)[None, None].repeat(2, axis=1)).cuda()
    hs, hz = synth.home_bands(F, G)
    out = tacg.eval_placements(tr, synth.fam_offsets([n] * F), E, hs, hz, G, prim)
    assert _err(out["err"]) == 0
    assert int(out["cost_home"][0]) == 0 and int(out["cost_span"][0]) == 0
    prim1 = torch.zeros((3, 2, E), dtype=torch.uint8, device="cuda")
    out = tacg.eval_placements(tr, synth.fam_offsets([n] * F), E, [0] * F, [1] * F, 1, prim1)
    assert int(out["cost_home"].abs().sum()) == 0 and int(out["cost_span"].abs().sum()) == 0
    assert np.all(_u32(out["load"]).sum(axis=2) == F * n * k)


def test_eval_table_errors_flagged():
    w = synth.make_workload("tiny", device="cuda")
    ps = w.placement_sets[0]
    prim = ps["primary"].copy()
    prim[3, 1, 2] = 9
    out = tacg.eval_placements(w.trace_serve, w.fam_off_serve, 8, ps["home_start"], ps["home_size"], 4,
                               torch.as_tensor(prim).cuda())
    assert _err(out["err"]) & tacg.ERR_TABLE


def test_jain_parity():
    rng = np.random.default_rng(5)
    ld = rng.integers(0, 1 << 20, size=(37, 5, 32)).astype(np.int64)
    ld[3] = 0
    ld[4, :, 1:] = 0
    t = torch.as_tensor(ld.astype(np.int32)).cuda()
    j, v = tacg.jain_index(t)
    jo, vo = oracle.jain(ld)
    _close(j, jo)
    _close(v, vo)
    j, v = tacg.jain_index(t, per_layer=True)
    jo, vo = oracle.jain(ld, per_layer=True)
    _close(j, jo)
    _close(v, vo)


# ------------------------------------------------------------------------------------------------
# host placement inputs (TACG grouping, GESR tables) built from the oracle's graph, scored by both
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("name,setidx", [("qwen15", 0), ("qwen3_30b", 0)])
def test_tacg_placement_scored(name, setidx):
    from paper_2606_01007_amd import placement as pm
    _say(f"tacg placement {name} set {setidx}")
    cfg = synth.CONFIGS[name]
    w = synth.make_workload(name, device="cuda", n_tokens=24000, n_place=2, layers=3)
    ps = w.placement_sets[setidx]
    G, cap = ps["n_gpus"], ps["capacity"]
    spec = cfg.placements[setidx]
    tg = w.trace_group.cpu().numpy()
    Do, Co, _ = oracle.coact(tg, w.fam_off_group, cfg.E)
    _, at_o, ah_o = oracle.reweight(Do, Co, cfg.k, alpha=0.25)
    L = tg.shape[0]
    default = np.repeat(np.arange(G, dtype=np.uint8), pm.capacities(cfg.E, G, cap))[None].repeat(L, axis=0)
    prim = np.stack([default, pm.tacg_placement(at_o, G, cap)])
    gen = pm.generic_experts(ah_o, spec.n_generic_rep)
    sec = np.stack([pm.affinity_secondaries(ah_o, prim[i], gen, G, spec.n_secondary) for i in range(2)])
    ts = w.trace_serve.cpu().numpy()
    Dso, _, _ = oracle.coact(ts, w.fam_off_serve, cfg.E)
    ref_o = oracle.placement_load(Dso, prim, G)
    ro = oracle.score(ts, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G, prim, sec, ref_o, (3, 20))
    prim_t, sec_t = torch.as_tensor(prim).cuda(), torch.as_tensor(sec).cuda()
    Ds, _, e1 = tacg.coact_build(w.trace_serve, w.fam_off_serve, cfg.E)
    ref_g = tacg.placement_load(Ds, prim_t, G, err=e1)
    out = tacg.eval_placements(w.trace_serve, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G, prim_t,
                               sec_t, ref_g, theta=(3, 20))
    assert _err(out["err"]) == 0 and _err(e1) == 0
    np.testing.assert_array_equal(ref_g.cpu().numpy(), ref_o)
    np.testing.assert_array_equal(out["cost_span"].cpu().numpy(), ro["cost_span"])
    np.testing.assert_array_equal(out["cost_home"].cpu().numpy(), ro["cost_home"])
    np.testing.assert_array_equal(_u32(out["load"]), ro["load"])
    # the grouped placement co-locates the planted clusters: fewer GPUs spanned than the default
    assert ro["cost_span"][1] < ro["cost_span"][0]


# ------------------------------------------------------------------------------------------------
# scoring on uniformly random traces: top-k widths with packed ids of 1-4 words, every replicated
# slot of a token resolved (tokens with more replicated slots than the per-token word holds), empty
# families, empty traces
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("E,k,L,counts,G,cap,n_rep,R,P,seed", [
    (16, 8, 2, [700, 0, 513], 4, 4, 16, 2, 20, 1),       # every expert replicated: all slots resolved
    (16, 16, 1, [300, 301], 8, 2, 16, 3, 9, 2),         # k = 16: two replica indices per token word
    (64, 16, 2, [1000, 999], 8, 8, 12, 1, 131, 3),
    (256, 16, 1, [900, 77], 32, 8, 16, 4, 130, 4),      # maximum k, G, R and replicated experts
    (40, 1, 2, [500, 500, 1], 5, 8, 6, 2, 33, 5),       # k = 1
    (200, 3, 2, [1200, 3], 25, 8, 10, 2, 129, 6),       # odd k, E > 64
    (60, 5, 2, [800, 801], 6, 10, 4, 2, 257, 7),        # odd k, E <= 64 (four placements per lane)
])
def test_eval_random_shapes(E, k, L, counts, G, cap, n_rep, R, P, seed):
    _say(f"eval random E={E} k={k} L={L} counts={counts} G={G} R={R} P={P}")
    off = synth.fam_offsets(counts)
    F = len(counts)
    tr = _rand_trace(L, int(off[-1]), k, E, seed)
    prim = synth.random_placements(P, L, E, G, cap, seed + 100)
    rng = np.random.default_rng(seed)
    rep = np.stack([np.sort(rng.choice(E, n_rep, replace=False)) for _ in range(L)])
    sec = synth.random_secondaries(prim, G, rep, R, seed + 200)
    hs, hz = synth.home_bands(F, G)
    Do, _, _ = oracle.coact(tr.cpu(), off, E)
    ref_o = oracle.placement_load(Do, prim, G)
    ro = oracle.score(tr.cpu(), off, E, hs, hz, G, prim, sec, ref_o, (3, 20))
    assert ro["err"] == 0
    prim_t, sec_t = torch.as_tensor(prim).cuda(), torch.as_tensor(sec).cuda()
    D, _, e1 = tacg.coact_build(tr, off, E)
    ref_g = tacg.placement_load(D, prim_t, G, err=e1)
    out = tacg.eval_placements(tr, off, E, hs, hz, G, prim_t, sec_t, ref_g, theta=(3, 20))
    assert _err(out["err"]) == 0 and _err(e1) == 0
    np.testing.assert_array_equal(ref_g.cpu().numpy(), ref_o)
    np.testing.assert_array_equal(out["cost_home"].cpu().numpy(), ro["cost_home"])
    np.testing.assert_array_equal(out["cost_span"].cpu().numpy(), ro["cost_span"])
    np.testing.assert_array_equal(_u32(out["load"]), ro["load"])
    np.testing.assert_array_equal(out["cost_home_fam"].cpu().numpy(), ro["cost_home_fam"])


def test_eval_empty_trace():
    E, k, L, G, F = 32, 4, 2, 4, 3
    tr = torch.zeros((L, 0, k), dtype=torch.int16, device="cuda")
    prim = torch.as_tensor(synth.random_placements(5, L, E, G, 8, 1)).cuda()
    hs, hz = synth.home_bands(F, G)
    out = tacg.eval_placements(tr, synth.fam_offsets([0] * F), E, hs, hz, G, prim)
    assert _err(out["err"]) == 0
    assert int(out["cost_home"].abs().sum()) == 0 and int(out["cost_span"].abs().sum()) == 0
    assert int(out["load"].abs().sum()) == 0


# ------------------------------------------------------------------------------------------------
# grouping objective over many placements
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("name,setidx,n_place", [("qwen15", 0, 300), ("qwen15", 1, 70), ("deepseek16b", 0, 130),
                                                 ("deepseek_v3", 0, 65)])
def test_group_objective_parity(name, setidx, n_place):
    cfg = synth.CONFIGS[name]
    _say(f"group objective {name} set {setidx} P={n_place}")
    w = synth.make_workload(name, n_tokens=cfg.F * 500, layers=3, n_place=n_place)
    ps = w.placement_sets[setidx]
    Do, Co, _ = oracle.coact(w.trace_group, w.fam_off_group, cfg.E)
    _, ato, _ = oracle.reweight(Do, Co, cfg.k)
    at32 = ato.astype(np.float32)                      # the device input precision, used by both sides
    got = tacg.group_objective(torch.as_tensor(at32).cuda(), torch.as_tensor(ps["primary"]).cuda(), ps["n_gpus"])
    ref = oracle.grouping_objective(at32.astype(np.float64), ps["primary"], ps["n_gpus"])
    np.testing.assert_allclose(got.cpu().numpy(), ref, rtol=1e-12, atol=1e-300)


def test_group_objective_table_error():
    at = torch.zeros((1, 8, 8), dtype=torch.float32, device="cuda")
    prim = torch.zeros((2, 1, 8), dtype=torch.uint8, device="cuda")
    prim[1, 0, 3] = 7
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    tacg.group_objective(at, prim, 4, err=err)
    assert _err(err) & tacg.ERR_TABLE


# ------------------------------------------------------------------------------------------------
# GESR identification scores
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny", "deepseek16b", "qwen15", "qwen3_30b", "deepseek_v3"])
def test_gesr_scores_parity(name):
    cfg = synth.CONFIGS[name]
    _say(f"gesr scores {name}")
    n = cfg.tokens_group if name == "tiny" else cfg.F * 700 + 3
    w = synth.make_workload(name, n_tokens=n, layers=min(cfg.L, 2), n_place=2)
    D, C, err = tacg.coact_build(w.trace_group.cuda(), w.fam_off_group, cfg.E)
    cent, cons, spec = tacg.gesr_scores(D, C, cfg.k)
    assert _err(err) == 0
    Do, Co, _ = oracle.coact(w.trace_group, w.fam_off_group, cfg.E)
    co, so, po = oracle.gesr_scores(Do, Co, cfg.k)
    np.testing.assert_allclose(cent.cpu().numpy(), co, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(cons.cpu().numpy(), so, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(spec.cpu().numpy(), po, rtol=1e-12, atol=1e-15)


def test_gesr_scores_empty_family():
    off = [0, 500, 500, 900]
    tr = _rand_trace(1, 900, 3, 20, 11)
    D, C, _ = tacg.coact_build(tr, off, 20)
    cent, cons, spec = tacg.gesr_scores(D, C, 3)
    Do, Co, _ = oracle.coact(tr.cpu(), off, 20)
    co, so, po = oracle.gesr_scores(Do, Co, 3)
    np.testing.assert_allclose(cons.cpu().numpy(), so, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(spec.cpu().numpy(), po, rtol=1e-12, atol=1e-15)


# ------------------------------------------------------------------------------------------------
# motivation diagnostics
# ------------------------------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny", "deepseek16b", "qwen15", "qwen3_30b", "deepseek_v3"])
def test_diagnostics_parity(name):
    cfg = synth.CONFIGS[name]
    _say(f"diagnostics {name}")
    n = cfg.tokens_group if name == "tiny" else cfg.F * 900 + 7
    w = synth.make_workload(name, n_tokens=n, layers=min(cfg.L, 3), n_place=2)
    D, C, err = tacg.coact_build(w.trace_group.cuda(), w.fam_off_group, cfg.E)
    dist = tacg.activation_distance(D, cfg.k)
    pairs, jac = tacg.pair_jaccard(C, 64)
    assert _err(err) == 0
    Do, Co, _ = oracle.coact(w.trace_group, w.fam_off_group, cfg.E)
    np.testing.assert_allclose(dist.cpu().numpy(), oracle.activation_distance(Do, cfg.k), rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(pairs.cpu().numpy(), oracle.top_pairs(Co, 64))
    np.testing.assert_array_equal(jac.cpu().numpy(), oracle.pair_jaccard(Co, 64))


@pytest.mark.parametrize("E,top_n,vmax,seed", [(2, 1, 3, 1), (9, 5, 2, 2), (60, 64, 3, 3), (256, 4096, 100000, 4),
                                              (128, 200, 1, 5), (256, 64, 0, 6)])
def test_top_pairs_ties_and_edges(E, top_n, vmax, seed):
    """Dense symmetric counts with many ties (vmax small), all-zero counts and top_n above the number
    of pairs."""
    rng = np.random.default_rng(seed)
    F, L = 3, 2
    C = rng.integers(0, vmax + 1, size=(F, L, E, E)).astype(np.int64)
    C = np.triu(C, 1)
    C = C + C.transpose(0, 1, 3, 2)
    pairs, jac = tacg.pair_jaccard(torch.as_tensor(C.astype(np.int32)).cuda(), top_n)
    np.testing.assert_array_equal(pairs.cpu().numpy(), oracle.top_pairs(C, top_n))
    np.testing.assert_array_equal(jac.cpu().numpy(), oracle.pair_jaccard(C, top_n))

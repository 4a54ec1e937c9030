"""The no-allocation scoring entry point, tacg_eval_placements_noalloc, against tacg_eval_placements
(the same kernels with a caller-owned workspace): bit-exact costs, loads and error bits on two calls in
a row, the second with a smaller input, so that the second call runs on the scratch contents the
first one left behind."""
import sys

import numpy as np
import pytest
import torch

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


def _inputs(name, n_tokens, n_place, layers):
    cfg = synth.CONFIGS[name]
    w = synth.make_workload(name, device="cuda", n_tokens=n_tokens, n_place=n_place, layers=layers)
    ps = w.placement_sets[0]
    G = ps["n_gpus"]
    prim = torch.as_tensor(ps["primary"]).cuda()
    sec = torch.as_tensor(ps["secondary"]).cuda() if ps["secondary"] is not None else None
    ref = None
    if sec is not None:
        Ds, _, e = tacg.coact_build(w.trace_serve, w.fam_off_serve, cfg.E)
        ref = tacg.placement_load(Ds, prim, G, err=e)
        torch.cuda.synchronize()
        assert int(e.item()) == 0
    return dict(trace=w.trace_serve, fam_off=w.fam_off_serve, n_experts=cfg.E, home_start=ps["home_start"],
                home_size=ps["home_size"], n_gpus=G, primary=prim, secondary=sec, load_ref=ref, theta=(3, 20))


def _same(got, want):
    for key in ("cost_home", "cost_span", "load", "cost_home_fam", "err"):
        assert torch.equal(got[key], want[key]), key


@pytest.mark.parametrize("name, big, small", [
    # (tokens, placements, layers) of the first and the second call
    ("deepseek_v3", (16 * 3000 + 17, 300, 3), (16 * 700 + 5, 130, 2)),
    ("qwen15", (6 * 4000 + 3, 520, 4), (6 * 1000, 64, 2)),
    ("deepseek16b", (8 * 5000 + 11, 256, 3), (8 * 900 + 1, 100, 1)),
])
def test_noalloc_matches_workspace_entry_point(name, big, small):
    a = _inputs(name, *big)
    b = _inputs(name, *small)
    _say(f"[no-alloc {name}] first call {big}, second call {small}")
    got_a = tacg.eval_placements_noalloc(**a)
    got_b = tacg.eval_placements_noalloc(**b)        # right after, on the scratch the first call left
    torch.cuda.synchronize()
    want_a = tacg.eval_placements(**a)
    want_b = tacg.eval_placements(**b)
    torch.cuda.synchronize()
    assert int(want_a["err"].item()) == 0 and int(want_b["err"].item()) == 0
    _same(got_a, want_a)
    _same(got_b, want_b)
    # and once more on the first input, after the smaller call
    again = tacg.eval_placements_noalloc(**a)
    torch.cuda.synchronize()
    _same(again, want_a)
    _say(f"[no-alloc {name}] ok")


def test_noalloc_rejects_oversized_scratch():
    a = _inputs("deepseek_v3", 16 * 64, 2, 1)
    P = 1
    while tacg.lib().tacg_eval_workspace_bytes(1 << 10, 58, 256, 32, P, 16) <= tacg.NOALLOC_SCRATCH_BYTES:
        P *= 2
    # the size check comes from the arguments alone: 58 layers x P placements need more than the scratch
    L, N, k = 58, a["trace"].shape[1], a["trace"].shape[2]
    trace = torch.zeros((L, N, k), dtype=torch.int16, device="cuda")
    prim = torch.zeros((P, L, 256), dtype=torch.uint8, device="cuda")
    with pytest.raises(tacg.TacgError) as ei:
        tacg.eval_placements_noalloc(trace, a["fam_off"], 256, a["home_start"], a["home_size"], 32, prim)
    assert ei.value.status == tacg.E_SCRATCH

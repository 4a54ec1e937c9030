#!/usr/bin/env python3
"""Benchmark of the TACG/GESR trace passes on one MI355X.

One step = one pass of the whole hot path over the resident synthetic input:
  tacg_coact_build (grouping trace) -> tacg_reweight -> tacg_eval_placements (serving trace,
  P placements with GESR replicas) -> tacg_jain.
The placement tables and the snapshot loads that feed the guard are host inputs built before the
timed region (the snapshot loads come from the serving trace's dispatch counts, computed with the
same library before timing).

Prints one JSON line.  Default workload: DeepSeek-V3-like shape (E=256, top-8, 58 MoE layers,
16 families, 2^23 tokens per trace, 1024 placements on 32 simulated GPUs, 16 generic experts with 3
secondaries each).  --config selects another preset; --config all prints one line per preset.
Every line records the seeds of its workload, the SHA-256 of its traces and the host's core counts.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "routed token·layers/sec (coact build) + placements×tokens/sec scored; % HBM BW"
HBM_PEAK_GBS = 8000.0                 # MI355X HBM3E, GB/s
N_CU, CLOCK_HZ = 256, 2.4e9
VALU_PEAK_TOPS = N_CU * 64 * CLOCK_HZ / 1e12   # T int32 lane-ops per second (64 lanes / CU / clock)
SINGLE_THREAD_PRESETS = ("tiny", "deepseek16b")  # presets with a one-thread oracle figure
CALIB_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def code_text(src: str) -> str:
    """The code of a C/C++/HIP source without its comments and layout (comments become one space,
    runs of white space one space)."""
    import re
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def source_digest(files) -> str:
    """SHA-256 over the code of the HIP sources that hold one kernel (and the shared internal header),
    comments and layout left out: HBM traffic figures are only reported for the kernel code they
    were measured on."""
    import hashlib
    h = hashlib.sha256()
    for f in sorted(set(files) | {"tacg_internal.h"}):
        h.update(f.encode())
        h.update(code_text(open(os.path.join(ROOT, "paper_2606_01007_amd", "csrc", f)).read()).encode())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str):
    """Per-launch HBM bytes of `kernel` from profiles/hbm_traffic.json, if measured on its current
    sources and on this workload."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    k = rec.get("kernels", {}).get(kernel)
    if not k or k.get("workload") != workload:
        return None
    if k.get("source_sha256") != source_digest(TRAFFIC_KERNELS[kernel][1]):
        return None
    return k.get("bytes_per_launch")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="deepseek_v3", help="a preset name, or 'all' (one JSON line per preset)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-quality", action="store_true", help="skip the untimed placement-quality context")
    ap.add_argument("--no-online", action="store_true", help="skip the decayed-load scoring measurement")
    ap.add_argument("--online-tokens", type=int, default=1 << 19,
                    help="serving-trace tokens of the decayed-load scoring sample")
    ap.add_argument("--tokens", type=int, default=0, help="tokens per trace (0 = the preset's; for profiling runs)")
    ap.add_argument("--layers", type=int, default=0, help="MoE layers (0 = the preset's; for profiling runs)")
    ap.add_argument("--cpu-layers", type=int, default=0, help="layers of the oracle's scoring sample (0 = all)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/hbm_traffic.json from the counter_collection.csv files of two "
                         "rocprofv3 --pmc runs of this script (FETCH_SIZE, then WRITE_SIZE) and exit")
    return ap.parse_args()


# kernels whose HBM bytes are reported: the device kernels each one is made of, and their sources
TRAFFIC_KERNELS = {"ev_main": (("ev_main",), ("eval.hip",)),
                   "coact_build": (("coact_hist_kernel", "coact_reduce_kernel"), ("coact.hip",))}


def write_traffic(fetch_csv: str, write_csv: str, workload: str) -> dict:
    """Per-launch HBM bytes from rocprofv3 FETCH_SIZE / WRITE_SIZE counters (KiB per dispatch).

    Each counter is scaled by what it reads for the 1 GiB device copy this script makes before the
    timed region (the largest copy kernel of the run): bytes = KiB * 1024 * (2^30 / copy bytes)."""
    import csv
    import re
    out = {"kernels": {}, "scale": {}}
    per = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        if not copies:
            raise SystemExit(f"no copy kernel in {path}")
        scale = CALIB_BYTES / (max(copies) * 1024.0)
        out["scale"][counter] = scale
        sums = {}
        for r in rows:
            m = re.search(r"tacg::\(anonymous namespace\)::(\w+)", r["Kernel_Name"])
            if m:
                sums.setdefault(m.group(1), []).append(float(r["Counter_Value"]) * 1024.0 * scale)
        per[counter] = {k: sum(v) / len(v) for k, v in sums.items()}
    for name, (parts, files) in TRAFFIC_KERNELS.items():
        if all(p in per["FETCH_SIZE"] and p in per["WRITE_SIZE"] for p in parts):
            f = sum(per["FETCH_SIZE"][p] for p in parts)
            w = sum(per["WRITE_SIZE"][p] for p in parts)
            out["kernels"][name] = {"workload": workload, "fetch_bytes": f, "write_bytes": w,
                                    "bytes_per_launch": f + w, "source_sha256": source_digest(files)}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    return out


def main():
    args = parse()
    if args.traffic_from:
        print(json.dumps(write_traffic(args.traffic_from[0], args.traffic_from[1], args.config)))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; multi-GPU runs are not supported "
                                   "(the simulated GPU count G is a parameter of the workload, not of the launch)"}))
        sys.exit(2)

    import torch

    from paper_2606_01007_amd import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    names = list(synth.CONFIGS) if args.config == "all" else [args.config]
    for name in names:
        result = run_config(name, args, all_mode=args.config == "all")
        print(json.dumps(result), flush=True)
        torch.cuda.empty_cache()


def host_info() -> dict:
    import oracle
    oracle.build()
    aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None
    return {"nproc": os.cpu_count(), "cpus_usable": aff, "oracle_threads": oracle.num_threads()}


def run_config(name: str, args, all_mode: bool = False) -> dict:
    import numpy as np
    import torch

    import paper_2606_01007_amd as tacg
    from paper_2606_01007_amd import synth

    dev = "cuda"
    cfg = synth.CONFIGS[name]
    t0 = time.time()
    w = synth.make_workload(name, device=dev, n_tokens=args.tokens or None, layers=args.layers or None)
    torch.cuda.synchronize()
    gen_s = time.time() - t0
    log(f"generated {name} in {gen_s:.1f} s")
    ps = w.placement_sets[0]
    E, k, F = cfg.E, cfg.k, cfg.F
    L = w.trace_group.shape[0]
    G, P = ps["n_gpus"], ps["primary"].shape[0]
    Ng, Ns = w.trace_group.shape[1], w.trace_serve.shape[1]
    prim = torch.as_tensor(ps["primary"]).to(dev)
    sec = torch.as_tensor(ps["secondary"]).to(dev) if ps["secondary"] is not None else None
    theta = (3, 20)

    # ---- host inputs, untimed: snapshot loads from the serving trace's dispatch counts ----
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ref = None
    if sec is not None:
        Ds, _, _ = tacg.coact_build(w.trace_serve, w.fam_off_serve, E, err=err)
        ref = tacg.placement_load(Ds, prim, G, err=err)
        del Ds

    # ---- preallocated outputs and workspaces ----
    D = torch.empty((F, L, E), dtype=torch.int32, device=dev)
    C = torch.empty((F, L, E, E), dtype=torch.int32, device=dev)
    ws_c = tacg.workspace(tacg.lib().tacg_coact_workspace_bytes(Ng, L, k, E, F), dev)
    ws_r = tacg.workspace(tacg.lib().tacg_reweight_workspace_bytes(F, L, E), dev)
    ws_e = tacg.workspace(tacg.lib().tacg_eval_workspace_bytes(Ns, L, E, G, P, F), dev)
    out = dict(cost_home=torch.empty(P, dtype=torch.int64, device=dev),
               cost_span=torch.empty(P, dtype=torch.int64, device=dev),
               load=torch.empty((P, L, G), dtype=torch.int32, device=dev),
               cost_home_fam=torch.empty((P, F), dtype=torch.int64, device=dev))

    # a plain copy of known size, untimed: the reference that scales the HBM byte counters of a
    # rocprofv3 --pmc run of this script (FETCH_SIZE / WRITE_SIZE of the copy kernel vs 1 GiB)
    calib_src = torch.ones(CALIB_BYTES // 4, dtype=torch.int32, device=dev)
    calib_dst = calib_src.clone()
    del calib_src, calib_dst

    # one set of stage events per timed step, read after the closing synchronize: no host sync
    # inside the timed region
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(max(1, args.steps))]
    reduced = bool(args.tokens or args.layers)

    def step(timed, ev=evs[0]):
        if timed:
            ev[0].record()
        tacg.coact_build(w.trace_group, w.fam_off_group, E, D=D, C=C, ws=ws_c, err=err)
        if timed:
            ev[1].record()
        pref, at, _ = tacg.reweight(D, C, k, alpha=0.25, tau=1.0, eps=1e-8, ws=ws_r)
        if timed:
            ev[2].record()
        tacg.eval_placements(w.trace_serve, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, prim, sec, ref,
                             theta=theta, ws=ws_e, err=err, out=out)
        if timed:
            ev[3].record()
        j, v = tacg.jain_index(out["load"])
        if timed:
            ev[4].record()
        return j, v

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    log("warm-up done")
    stage = np.zeros((args.steps, 4))
    t_start = time.perf_counter()
    for s in range(args.steps):
        step(True, evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    for s in range(args.steps):
        for i in range(4):
            stage[s, i] = evs[s][i].elapsed_time(evs[s][i + 1]) * 1e-3
    assert int(err.item()) == 0, f"device data error bits {int(err.item()):#x}"

    t_coact, t_rw, t_eval, t_jain = stage.mean(axis=0)
    tl = Ng * L                                        # routed token-layers per coact build
    ptl = P * Ns * L                                   # placement-token-layers per scoring call
    coact_rate = tl / t_coact
    score_rate = P * Ns / t_eval                       # placements x tokens / s
    trace_bytes_g = Ng * L * k * 2
    trace_bytes_s = Ns * L * k * 2
    c_bytes = F * L * E * E * 4 + F * L * E * 4
    coact_gbs = (trace_bytes_g + c_bytes) / t_coact / 1e9
    # algorithmic integer work per placement-token-layer: k table lookups, k-1 ORs of one-hot GPU
    # masks, two popcounts and the replica resolution, about 2k + 6 lane-ops; the lookups run on the
    # LDS here, one read serving every placement of a lane, so at four placements per lane this count
    # can pass the VALU peak.  k + 2 (the ORs, the and-not with the anchor bit and the two popcounts) is
    # a lower bound for any scoring on GPU masks in 32-bit lanes.
    eval_tops = ptl * (2 * k + 6) / t_eval / 1e12
    eval_tops_strict = ptl * (k + 2) / t_eval / 1e12
    result = {
        "metric": METRIC,
        "value": coact_rate,
        "unit": "routed token·layers/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}{' (reduced for profiling)' if args.tokens or args.layers else ''}: "
                        f"E={E} top-{k} L={L} F={F}, grouping trace {Ng} tokens (uniform mix), "
                        f"serving trace {Ns} tokens ({cfg.serve_mix} mix), {P} placements on G={G} cap "
                        f"{ps['capacity']}, replicas {cfg.placements[0].n_generic_rep}x{cfg.placements[0].n_secondary}"
                        f", theta=3/20",
            "E": E, "top_k": k, "layers": L, "families": F, "tokens": Ng, "placements": P, "sim_gpus": G,
        },
        "coact_build": {"value": coact_rate, "unit": "routed token·layers/s", "ms": t_coact * 1e3,
                        "hbm_GBps": coact_gbs, "hbm_frac": coact_gbs / HBM_PEAK_GBS},
        "scoring": {"value": score_rate, "unit": "placements×tokens/s", "ms": t_eval * 1e3,
                    "placement_token_layers_per_s": ptl / t_eval,
                    "trace_equivalent_GBps": P * trace_bytes_s / t_eval / 1e9,
                    "trace_equivalent_frac": P * trace_bytes_s / t_eval / 1e9 / HBM_PEAK_GBS},
        "reweight_ms": t_rw * 1e3,
        "jain_ms": t_jain * 1e3,
        "roofline": {"kernel": "ev_main (tacg_eval_placements)", "bound": "alu",
                     "achieved": eval_tops, "peak": VALU_PEAK_TOPS, "unit": "T int32 lane-ops/s",
                     "frac": eval_tops / VALU_PEAK_TOPS,
                     "achieved_k_plus_2": eval_tops_strict, "frac_k_plus_2": eval_tops_strict / VALU_PEAK_TOPS,
                     "traffic": None if reduced else measured_traffic("ev_main", cfg.name),
                     "note": "achieved/frac: 2k + 6 int32 lane-ops per placement-token-layer (k table "
                             "lookups, k-1 ORs of one-hot GPU masks, two popcounts, replica resolution); "
                             "the lookups run on the LDS, one read serving all placements of a lane, so "
                             "at four placements per lane (E <= 64) frac can exceed 1; *_k_plus_2: only "
                             "the ORs, the and-not with the anchor bit and the two popcounts, a lower "
                             "bound for any mask-based scoring; peak = 256 CUs x 64 lanes x 2.4 GHz"},
        "roofline_coact": {"kernel": ("coact_mfma" if tacg.coact_uses_matrix_cores(E, k) else "coact_hist")
                                     + " + coact_reduce (tacg_coact_build)", "bound": "hbm",
                           "achieved": coact_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                           "frac": coact_gbs / HBM_PEAK_GBS,
                           "traffic": None if reduced else measured_traffic("coact_build", cfg.name),
                           "note": "algorithmic bytes: the int16 trace once + dense C and D written"},
        "gen_s": gen_s,
        "seeds": synth.workload_seeds(cfg),
    }

    log(f"timed {args.steps} steps: {wall / args.steps * 1e3:.1f} ms/step")
    result["aux_ms"] = aux_timings(D, C, prim, cfg, G)
    if not args.no_quality:
        result["placement_quality"] = placement_quality(w, ps, cfg, D, C, err)
    if not args.no_online:
        result["online_scoring"] = online_scoring(w, ps, cfg, prim, sec, err, args.online_tokens)
    del D, C, ws_c, ws_r, ws_e, out
    torch.cuda.empty_cache()
    # host copies of the traces: their SHA-256 and the oracle's input
    t0 = time.time()
    tg = w.trace_group.cpu().numpy()
    ts = tg if w.trace_serve is w.trace_group else w.trace_serve.cpu().numpy()
    result["trace_sha256"] = {"grouping": synth.trace_digest(tg),
                              "serving": synth.trace_digest(ts) if ts is not tg else "same as grouping"}
    result["host"] = host_info()
    log(f"trace digests in {time.time() - t0:.1f} s")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, tg, ts, ps, cfg, args.cpu_layers)
        st = {}
        for sname in SINGLE_THREAD_PRESETS:
            if all_mode and sname != name:
                continue  # with --config all each of these presets reports its own
            st[sname] = single_thread_oracle(sname, w if sname == name else None)
        if st:
            result["cpu_baseline"]["single_thread"] = st
    return result


def aux_timings(D, C, prim, cfg, G, reps=5):
    """Untimed by the step: the host-input helpers on the grouping trace's counts (GESR
    identification scores) and on the timed placements (grouping objective of every placement)."""
    import torch

    import paper_2606_01007_amd as tacg

    _, at, _ = tacg.reweight(D, C, cfg.k)

    def timed(fn):
        fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    return {"gesr_scores": timed(lambda: tacg.gesr_scores(D, C, cfg.k)),
            "group_objective": timed(lambda: tacg.group_objective(at, prim, G)),
            "activation_distance": timed(lambda: tacg.activation_distance(D, cfg.k)),
            "pair_jaccard_top64": timed(lambda: tacg.pair_jaccard(C, 64)),
            "note": "gesr_scores, activation_distance and pair_jaccard over the grouping counts; "
                    "group_objective of all placements x layers"}


def online_scoring(w, ps, cfg, prim, sec, err, n_tokens, reps=3):
    """Untimed by the step: tacg_eval_online (decayed per-GPU loads, rho = 0.995, theta = 3/20) over
    the first tokens of the serving trace (one family mix prefix), every placement and layer."""
    import numpy as np
    import torch

    import paper_2606_01007_amd as tacg

    n = min(n_tokens, w.trace_serve.shape[1])
    tr = w.trace_serve[:, :n].contiguous()
    off = np.minimum(np.asarray(w.fam_off_serve, dtype=np.int64), n)
    out = None
    t = []
    for _ in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        out = tacg.eval_online(tr, off, cfg.E, ps["home_start"], ps["home_size"], ps["n_gpus"], prim, sec,
                               rho=0.995, theta=(3, 20), err=err, out=out)
        b.record()
        torch.cuda.synchronize()
        t.append(a.elapsed_time(b) * 1e-3)
    sec_per = float(np.mean(t[1:]))
    P, L = prim.shape[0], tr.shape[0]
    return {"value": P * n / sec_per, "unit": "placements×tokens/s", "ms": sec_per * 1e3,
            "placement_token_layers_per_s": P * n * L / sec_per,
            "sample": f"first {n} tokens of the serving trace, {P} placements x {L} layers, rho=0.995, theta=3/20"}


def placement_quality(w, ps, cfg, D, C, err):
    """Untimed context: the paper's communication metric (App. H "Comm": mean over tokens of
    sum_l (|cards_l| - 1)) on the serving trace, for the contiguous default placement and for the
    TACG placement grouped on the host from this run's A-tilde (grouping trace) with GESR replicas
    (generic experts by centrality, secondaries by affinity), plus Jain and MaxVio and the per-token
    statistics of App. C (layers spanning more than one family band, home-family dispatch mass)."""
    import numpy as np
    import torch

    import paper_2606_01007_amd as tacg
    from paper_2606_01007_amd import placement as pm

    t0 = time.time()
    E, k = cfg.E, cfg.k
    L = w.trace_group.shape[0]
    G, cap = ps["n_gpus"], ps["capacity"]
    n_rep, n_sec = cfg.placements[0].n_generic_rep, cfg.placements[0].n_secondary
    _, at, ah = tacg.reweight(D, C, k, alpha=0.25, tau=1.0, eps=1e-8, want_hat=True)
    at, ah = at.cpu().double().numpy(), ah.cpu().double().numpy()
    default = np.repeat(np.arange(G, dtype=np.uint8), pm.capacities(E, G, cap))[None].repeat(L, axis=0)
    grouped = pm.tacg_placement(at, G, cap)
    prim = np.stack([default, grouped])                                    # [2][L][E]
    sec = None
    if n_sec > 0:
        gen = pm.generic_experts(ah, n_rep)
        sec = np.stack([pm.affinity_secondaries(ah, prim[i], gen, G, n_sec) for i in range(2)])
    dev = "cuda"
    prim_t = torch.as_tensor(prim).to(dev)
    sec_t = torch.as_tensor(sec).to(dev) if sec is not None else None
    ref = None
    if sec_t is not None:
        Ds, _, _ = tacg.coact_build(w.trace_serve, w.fam_off_serve, E, err=err)
        ref = tacg.placement_load(Ds, prim_t, G, err=err)
    out = tacg.eval_trace_stats(w.trace_serve, w.fam_off_serve, E, ps["home_start"], ps["home_size"], G, prim_t,
                                sec_t, ref, theta=(3, 20), err=err)
    jn, mv = tacg.jain_index(out["load"])
    torch.cuda.synchronize()
    Ns = w.trace_serve.shape[1]
    span = out["cost_span"].cpu().numpy().astype(np.float64) / Ns
    home = out["cost_home"].cpu().numpy().astype(np.float64) / Ns
    # App. C per-token statistics, averaged over the families that have tokens
    nf = np.diff(np.asarray(w.fam_off_serve, dtype=np.int64)).astype(np.float64)
    has = nf > 0
    cross = out["cross_fam"].cpu().numpy()[:, has] / nf[has]
    mass = out["home_mass_fam"].cpu().numpy()[:, has] / (nf[has] * L * k)
    return {"placements": "contiguous default vs TACG (host spectral grouping of this run's A-tilde, alpha=0.25)"
                          f" with GESR ({n_rep} generic experts by centrality x {n_sec} secondaries by affinity)",
            "trace": "serving trace (synthetic)",
            "comm_default": span[0], "comm_tacg": span[1],
            "comm_reduction_pct": 100.0 * (span[0] - span[1]) / span[0] if span[0] > 0 else None,
            "home_cost_default": home[0], "home_cost_tacg": home[1],
            "cross_family_layers_per_token": [float(cross[0].mean()), float(cross[1].mean())],
            "home_family_mass_pct": [float(100 * mass[0].mean()), float(100 * mass[1].mean())],
            "home_family_mass_uniform_pct": float(100 * np.mean(np.asarray(ps["home_size"])[has] / G)),
            "jain": [float(jn[0]), float(jn[1])], "maxvio": [float(mv[0]), float(mv[1])],
            "host_s": time.time() - t0}


def cpu_baseline(w, tg, ts, ps, cfg, cpu_layers):
    """The oracle as it stands, on this host's cores: the whole co-activation build of the grouping
    trace, and the first three placements scored over the serving trace (scaled to placements x
    tokens / s); about 15 s of CPU work at the full DeepSeek-V3-like workload.  tg, ts: host copies
    of the two traces."""
    import numpy as np
    import oracle

    oracle.build()
    log("cpu baseline: oracle co-activation build")
    t0 = time.perf_counter()
    _, _, e1 = oracle.coact(tg, w.fam_off_group, cfg.E)
    t_coact = time.perf_counter() - t0
    Ls = ts.shape[0] if cpu_layers <= 0 else min(cpu_layers, ts.shape[0])
    ts = np.ascontiguousarray(ts[:Ls])
    G = ps["n_gpus"]
    n_p = min(3, ps["primary"].shape[0])
    sec = ps["secondary"][:n_p, :Ls] if ps["secondary"] is not None else None
    prim = ps["primary"][:n_p, :Ls]
    ref = None
    if sec is not None:
        Ds, _, _ = oracle.coact(ts, w.fam_off_serve, cfg.E)
        ref = oracle.placement_load(Ds, prim, G)
    log(f"cpu baseline: oracle scoring of {n_p} placements")
    t0 = time.perf_counter()
    r = oracle.score(ts, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G, prim, sec, ref, (3, 20),
                     p_range=(0, n_p))
    t_score = time.perf_counter() - t0
    Ns = ts.shape[1]
    coact_rate = w.trace_group.shape[1] * w.trace_group.shape[0] / t_coact
    return {"value": coact_rate, "unit": "routed token·layers/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"co-activation build of the whole grouping trace ({w.trace_group.shape[1]} tokens x "
                      f"{w.trace_group.shape[0]} layers, {t_coact:.1f} s); scoring of placements 0..{n_p - 1} on "
                      f"the serving trace over {Ls} layers ({t_score:.1f} s)",
            "scoring_value": n_p * Ns * Ls / w.trace_serve.shape[0] / t_score if Ls else None,
            "scoring_unit": "placements×tokens/s (over all layers, scaled from the sample)",
            "err": int(e1) | int(r["err"])}


def single_thread_oracle(name: str, w=None, device: str = "cuda") -> dict:
    """The oracle on one thread, on a preset's full grouping trace (co-activation build) and one
    placement scored over its serving trace: the per-core figure beside the all-cores baseline."""
    import numpy as np
    import oracle

    from paper_2606_01007_amd import synth

    cfg = synth.CONFIGS[name]
    if w is None:
        w = synth.make_workload(name, device=device)
    tg = w.trace_group.cpu().numpy()
    ts = w.trace_serve.cpu().numpy()
    ps = w.placement_sets[0]
    G = ps["n_gpus"]
    prim = ps["primary"][:1]
    sec = ps["secondary"][:1] if ps["secondary"] is not None else None
    oracle.build()
    threads = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        log(f"cpu baseline: one-thread oracle on {name}")
        t0 = time.perf_counter()
        _, _, e1 = oracle.coact(tg, w.fam_off_group, cfg.E)
        t_coact = time.perf_counter() - t0
        ref = None
        if sec is not None:
            Ds, _, _ = oracle.coact(ts, w.fam_off_serve, cfg.E)
            ref = oracle.placement_load(Ds, prim, G)
        t0 = time.perf_counter()
        r = oracle.score(ts, w.fam_off_serve, cfg.E, ps["home_start"], ps["home_size"], G, prim, sec, ref,
                         (3, 20))
        t_score = time.perf_counter() - t0
    finally:
        oracle.set_num_threads(threads)
    L, Ng, Ns = tg.shape[0], tg.shape[1], ts.shape[1]
    return {"cores": 1, "coact_value": Ng * L / t_coact, "coact_unit": "routed token·layers/s",
            "scoring_value": Ns / t_score, "scoring_unit": "placements×tokens/s",
            "sample": f"co-activation build of the whole grouping trace ({Ng} tokens x {L} layers, "
                      f"{t_coact:.2f} s); placement 0 scored over the serving trace ({Ns} tokens x {L} layers, "
                      f"{t_score:.2f} s)",
            "trace_sha256": synth.trace_digest(tg), "err": int(e1) | int(r["err"])}


if __name__ == "__main__":
    main()

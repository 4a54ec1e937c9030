"""Seeded synthetic inputs: routing traces, family mixes, placements, replica tables, home bands.

This module only *builds inputs*.  It holds none of the method's arithmetic (no counts, no
preferences, no graph, no scoring); both the HIP path and the CPU oracle consume what it makes.

Trace law (stands in for the calibration and serving traces of Sec. 4.1, which are not available):
every (family f, layer l) has fixed logits mu[f, l, e] ~ N(0, 1); planted "cluster" experts of f get
+bias_cluster and globally "generic" experts of layer l get +bias_generic in every family.  Each
token draws its top-k experts without replacement by Gumbel-top-k on mu + Gumbel(0, 1) noise, i.e.
the k largest of mu - log(X) with X ~ Exp(1).  Slot 0 holds the highest-scoring expert (router rank
order).  Shared experts are excluded (Table moe-backbones lists them separately).

Layouts (all C-contiguous):
  trace      int16  [L][N][k]   tokens contiguous per family, family f owns [fam_off[f], fam_off[f+1])
  fam_off    int64  [F+1]
  primary    uint8  [P][L][E]   GPU of each expert
  secondary  uint8  [P][L][E][R] extra candidate GPUs, 0xFF = none
  home_start int32  [F], home_size int32 [F]
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional, Sequence

import numpy as np
import torch

NONE = 0xFF


# --------------------------------------------------------------------------------------------
# configuration presets (shapes of the MoE backbones of Table moe-backbones and two larger shapes)
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class PlacementSet:
    n_gpus: int
    capacity: int            # experts per GPU; n_gpus * capacity >= E ("exact capacity" when ==)
    n_place: int
    n_generic_rep: int = 0   # experts given secondary GPUs (the planted generic experts)
    n_secondary: int = 0     # secondary GPUs per replicated expert


@dataclasses.dataclass(frozen=True)
class TraceConfig:
    name: str
    E: int
    k: int
    L: int
    F: int
    tokens_group: int                 # total tokens of the grouping (calibration) trace
    cluster_size: int
    clusters_per_family: int
    bias_cluster: float
    n_generic: int
    bias_generic: float
    placements: Sequence[PlacementSet]
    seed: int
    serve_mix: str = "same"           # "same" (score the grouping trace), "zipf", "dirichlet"
    serve_param: float = 0.0          # Zipf exponent or Dirichlet concentration
    drift: float = 0.0                # fraction of each cluster re-randomised in the serving trace
    seed_serve: int = 0


CONFIGS = {
    # E=8 experts, top-2, 2 layers, 3 families x 2048 tokens; +2.0 on a 3-expert block per family.
    "tiny": TraceConfig("tiny", E=8, k=2, L=2, F=3, tokens_group=3 * 2048, cluster_size=3,
                        clusters_per_family=1, bias_cluster=2.0, n_generic=0, bias_generic=0.0,
                        placements=(PlacementSet(4, 2, 16),), seed=101),
    # DeepSeekMoE-16B-like: 64 routed experts, top-6, 27 MoE layers, 8 families x 262144 tokens.
    "deepseek16b": TraceConfig("deepseek16b", E=64, k=6, L=27, F=8, tokens_group=8 * 262144,
                               cluster_size=8, clusters_per_family=2, bias_cluster=1.5, n_generic=6,
                               bias_generic=1.0, placements=(PlacementSet(8, 8, 256),), seed=102),
    # Qwen1.5-MoE-A2.7B-like: 60 experts, top-4, 24 layers, 6 families x 524288 tokens.
    "qwen15": TraceConfig("qwen15", E=60, k=4, L=24, F=6, tokens_group=6 * 524288, cluster_size=6,
                          clusters_per_family=2, bias_cluster=1.5, n_generic=4, bias_generic=1.0,
                          placements=(PlacementSet(4, 15, 512, 4, 2), PlacementSet(6, 10, 512, 4, 2)),
                          seed=103),
    # Qwen3-30B-A3B-like: 128 experts, top-8, 48 layers, 16 families, 4M tokens; Zipf(1.1) serving mix.
    "qwen3_30b": TraceConfig("qwen3_30b", E=128, k=8, L=48, F=16, tokens_group=1 << 22, cluster_size=10,
                             clusters_per_family=2, bias_cluster=1.5, n_generic=8, bias_generic=1.0,
                             placements=(PlacementSet(8, 16, 1024, 8, 2),), seed=104,
                             serve_mix="zipf", serve_param=1.1, seed_serve=204),
    # DeepSeek-V3-like: 256 experts, top-8, 58 layers, 16 families, 8M tokens; Dirichlet(0.3) serving
    # mix and 20% of every cluster re-randomised between grouping and serving traces.
    "deepseek_v3": TraceConfig("deepseek_v3", E=256, k=8, L=58, F=16, tokens_group=1 << 23, cluster_size=10,
                               clusters_per_family=2, bias_cluster=1.5, n_generic=16, bias_generic=1.0,
                               placements=(PlacementSet(32, 8, 1024, 16, 3),), seed=105,
                               serve_mix="dirichlet", serve_param=0.3, drift=0.2, seed_serve=205),
}


# --------------------------------------------------------------------------------------------
# family mixes
# --------------------------------------------------------------------------------------------
def largest_remainder(n_total: int, shares: Sequence[float]) -> np.ndarray:
    """Integer token counts per family summing to n_total, proportional to `shares`."""
    s = np.asarray(shares, dtype=np.float64)
    s = s / s.sum()
    raw = s * n_total
    base = np.floor(raw).astype(np.int64)
    rest = int(n_total - base.sum())
    order = np.argsort(-(raw - base), kind="stable")
    base[order[:rest]] += 1
    return base


def fam_offsets(counts: Sequence[int]) -> np.ndarray:
    off = np.zeros(len(counts) + 1, dtype=np.int64)
    off[1:] = np.cumsum(np.asarray(counts, dtype=np.int64))
    return off


def mix_shares(kind: str, F: int, param: float, seed: int) -> np.ndarray:
    if kind in ("same", "uniform"):
        return np.full(F, 1.0 / F)
    if kind == "zipf":
        w = (np.arange(F, dtype=np.float64) + 1.0) ** (-param)
        return w / w.sum()
    if kind == "dirichlet":
        return np.random.default_rng(seed).dirichlet(np.full(F, param))
    raise ValueError(kind)


# --------------------------------------------------------------------------------------------
# logits with planted structure
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass
class Planted:
    raw: np.ndarray           # float64 [F][L][E], the N(0, 1) part
    clusters: np.ndarray      # int64 [F][L][clusters_per_family * cluster_size]
    generic: np.ndarray       # int64 [L][n_generic]
    bias_cluster: float
    bias_generic: float

    @property
    def mu(self) -> np.ndarray:
        """Logits with the planted biases added."""
        mu = self.raw.copy()
        F, L, _ = mu.shape
        for l in range(L):
            mu[:, l, self.generic[l]] += self.bias_generic
        if self.clusters.shape[2]:
            for f in range(F):
                for l in range(L):
                    mu[f, l, self.clusters[f, l]] += self.bias_cluster
        return mu


def planted_logits(E: int, L: int, F: int, cluster_size: int, clusters_per_family: int,
                   bias_cluster: float, n_generic: int, bias_generic: float, seed: int) -> Planted:
    """Per-(family, layer) logits with planted family clusters and shared generic experts."""
    rng = np.random.default_rng(seed)
    raw = rng.standard_normal((F, L, E))
    n_cl = clusters_per_family * cluster_size
    generic = np.zeros((L, n_generic), dtype=np.int64)
    clusters = np.zeros((F, L, n_cl), dtype=np.int64)
    for l in range(L):
        perm = rng.permutation(E)
        generic[l] = np.sort(perm[:n_generic])
        others = perm[n_generic:]
        for f in range(F):
            clusters[f, l] = rng.choice(others, size=n_cl, replace=False)
    return Planted(raw, clusters, generic, bias_cluster, bias_generic)


def drifted(base: Planted, cluster_size: int, clusters_per_family: int, drift: float, seed: int) -> Planted:
    """Distribution shift: swap round(drift * cluster_size) members of every cluster for random
    experts outside the family's clusters and the generic set; logits otherwise unchanged."""
    F, L, E = base.raw.shape
    clusters = base.clusters.copy()
    rng = np.random.default_rng(seed)
    n_swap = int(round(drift * cluster_size))
    if n_swap > 0:
        for f in range(F):
            for l in range(L):
                for c in range(clusters_per_family):
                    outside = np.setdiff1d(np.arange(E), np.concatenate([clusters[f, l], base.generic[l]]))
                    who = rng.choice(cluster_size, size=n_swap, replace=False) + c * cluster_size
                    clusters[f, l, who] = rng.choice(outside, size=n_swap, replace=False)
    return Planted(base.raw, clusters, base.generic, base.bias_cluster, base.bias_generic)


# --------------------------------------------------------------------------------------------
# trace sampling
# --------------------------------------------------------------------------------------------
def sample_trace(mu: np.ndarray, counts: Sequence[int], k: int, seed: int,
                 device: str | torch.device = "cpu", chunk_rows: int = 1 << 20) -> torch.Tensor:
    """Gumbel-top-k without replacement; returns int16 [L][N][k] on `device`."""
    F, L, E = mu.shape
    counts = [int(c) for c in counts]
    N = sum(counts)
    dev = torch.device(device)
    out = torch.empty((L, N, k), dtype=torch.int16, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(int(seed))
    mu_t = torch.as_tensor(mu, dtype=torch.float32, device=dev)
    rows = max(1, min(chunk_rows, (1 << 28) // max(E, 1)))
    for l in range(L):
        t0 = 0
        for f in range(F):
            n_f = counts[f]
            done = 0
            while done < n_f:
                r = min(rows, n_f - done)
                x = torch.empty((r, E), dtype=torch.float32, device=dev).exponential_(generator=gen)
                score = mu_t[f, l].unsqueeze(0) - torch.log(x.clamp_min_(1e-30))
                idx = torch.topk(score, k, dim=1, largest=True, sorted=True).indices
                out[l, t0 + done:t0 + done + r] = idx.to(torch.int16)
                done += r
            t0 += n_f
    return out


def uniform_trace(E: int, k: int, L: int, N: int, seed: int, device="cpu") -> torch.Tensor:
    """Uniformly random k-subsets (no planted structure)."""
    mu = np.zeros((1, L, E))
    return sample_trace(mu, [N], k, seed, device)


# --------------------------------------------------------------------------------------------
# placements, replica tables, home bands
# --------------------------------------------------------------------------------------------
def capacities(E: int, G: int, cap: int) -> np.ndarray:
    """Per-GPU capacities: `cap` each, the last GPUs trimmed so that they sum to E."""
    c = np.full(G, cap, dtype=np.int64)
    excess = int(c.sum()) - E
    if excess < 0:
        raise ValueError(f"{G} GPUs x capacity {cap} cannot hold {E} experts")
    g = G - 1
    while excess > 0:
        d = min(excess, int(c[g]))
        c[g] -= d
        excess -= d
        g -= 1
    return c


def contiguous_placement(E: int, caps: np.ndarray) -> np.ndarray:
    """The default placement: experts 0..E-1 filled GPU by GPU in order."""
    return np.repeat(np.arange(len(caps), dtype=np.uint8), caps)[:E]


def random_placements(P: int, L: int, E: int, G: int, cap: int, seed: int,
                      first_contiguous: bool = True) -> np.ndarray:
    caps = capacities(E, G, cap)
    base = contiguous_placement(E, caps)
    rng = np.random.default_rng(seed)
    out = np.empty((P, L, E), dtype=np.uint8)
    for p in range(P):
        for l in range(L):
            out[p, l] = base if (p == 0 and first_contiguous) else rng.permutation(base)
    return out


def random_secondaries(primary: np.ndarray, G: int, rep_experts: np.ndarray, n_sec: int,
                       seed: int) -> np.ndarray:
    """For each (p, l) and each expert of rep_experts[l], n_sec distinct random GPUs other than its
    primary.  Other experts get 0xFF (no secondary)."""
    P, L, E = primary.shape
    if n_sec == 0:
        return np.full((P, L, E, 0), NONE, dtype=np.uint8)
    sec = np.full((P, L, E, n_sec), NONE, dtype=np.uint8)
    rng = np.random.default_rng(seed)
    R = rep_experts.shape[1]
    lidx = np.arange(L)[:, None]
    prim_rep = primary[:, lidx, rep_experts]                     # [P][L][R]
    keys = rng.random((P, L, R, G))
    np.put_along_axis(keys, prim_rep[..., None].astype(np.int64), np.inf, axis=3)
    pick = np.argsort(keys, axis=3, kind="stable")[..., :n_sec].astype(np.uint8)
    sec[:, lidx, rep_experts] = pick
    return sec


def home_bands(F: int, G: int):
    """Family GPU bands: f owns [floor(fG/F), floor((f+1)G/F)), at least one GPU (shared if F > G)."""
    start = np.zeros(F, dtype=np.int32)
    size = np.zeros(F, dtype=np.int32)
    for f in range(F):
        a = (f * G) // F
        b = ((f + 1) * G) // F
        if b <= a:
            b = a + 1
        start[f] = min(a, G - 1)
        size[f] = b - start[f]
    return start, size


# --------------------------------------------------------------------------------------------
# whole workloads
# --------------------------------------------------------------------------------------------
@dataclasses.dataclass
class Workload:
    cfg: TraceConfig
    trace_group: torch.Tensor
    fam_off_group: np.ndarray
    trace_serve: torch.Tensor
    fam_off_serve: np.ndarray
    planted: Planted
    placement_sets: list        # list of dicts: n_gpus, primary, secondary, home_start, home_size


def make_workload(name: str, device="cpu", n_tokens: Optional[int] = None, n_place: Optional[int] = None,
                  layers: Optional[int] = None, placement_seed_offset: int = 0) -> Workload:
    """Build a preset workload.  n_tokens / n_place / layers shrink it (same law) for tests."""
    cfg = CONFIGS[name]
    L = layers or cfg.L
    N = n_tokens or cfg.tokens_group
    pl = planted_logits(cfg.E, L, cfg.F, cfg.cluster_size, cfg.clusters_per_family, cfg.bias_cluster,
                        cfg.n_generic, cfg.bias_generic, cfg.seed)
    counts_g = largest_remainder(N, np.full(cfg.F, 1.0 / cfg.F))
    tr_g = sample_trace(pl.mu, counts_g, cfg.k, cfg.seed, device)
    off_g = fam_offsets(counts_g)
    if cfg.serve_mix == "same":
        tr_s, off_s, pl_s = tr_g, off_g, pl
    else:
        shares = mix_shares(cfg.serve_mix, cfg.F, cfg.serve_param, cfg.seed_serve)
        counts_s = largest_remainder(N, shares)
        pl_s = drifted(pl, cfg.cluster_size, cfg.clusters_per_family, cfg.drift, cfg.seed_serve) \
            if cfg.drift > 0 else pl
        tr_s = sample_trace(pl_s.mu, counts_s, cfg.k, cfg.seed_serve, device)
        off_s = fam_offsets(counts_s)
    sets = []
    for i, ps in enumerate(cfg.placements):
        P = n_place or ps.n_place
        prim = random_placements(P, L, cfg.E, ps.n_gpus, ps.capacity, cfg.seed + 1000 * (i + 1) + placement_seed_offset)
        if ps.n_secondary > 0:
            rep = pl.generic[:, :ps.n_generic_rep]
            sec = random_secondaries(prim, ps.n_gpus, rep, ps.n_secondary, cfg.seed + 2000 * (i + 1) + placement_seed_offset)
        else:
            sec = None
        hs, hz = home_bands(cfg.F, ps.n_gpus)
        sets.append(dict(n_gpus=ps.n_gpus, capacity=ps.capacity, primary=prim, secondary=sec,
                         home_start=hs, home_size=hz))
    return Workload(cfg, tr_g, off_g, tr_s, off_s, pl, sets)


def trace_digest(trace) -> str:
    """SHA-256 of the trace bytes (recorded with results); a torch tensor or a host numpy array."""
    h = hashlib.sha256()
    if isinstance(trace, torch.Tensor):
        t = trace.detach().to("cpu").contiguous().view(torch.uint8).numpy()
    else:
        t = np.ascontiguousarray(trace).view(np.uint8)
    step = 1 << 28
    flat = t.reshape(-1)
    for i in range(0, flat.size, step):
        h.update(flat[i:i + step].tobytes())
    return h.hexdigest()


def workload_seeds(cfg: TraceConfig, placement_seed_offset: int = 0) -> dict:
    """The seeds make_workload draws a preset from (recorded with results)."""
    out = {"logits_and_grouping_trace": cfg.seed,
           "serving_trace": cfg.seed_serve if cfg.serve_mix != "same" else cfg.seed}
    for i, _ in enumerate(cfg.placements):
        out[f"placements_{i}"] = cfg.seed + 1000 * (i + 1) + placement_seed_offset
        out[f"secondaries_{i}"] = cfg.seed + 2000 * (i + 1) + placement_seed_offset
    return out

"""Do the oracle's pins see plausible mistakes?

Each mutant below plants one plausible mistake in a copy of the oracle, on the CPU. Mistakes are
dropped terms, wrong bounds or indices, a wrong tie rule, or a rule step left out. The CPU pin tests
that cover that part of the oracle then run against the copy, in a fresh interpreter, and must fail.
The pins come from the paper and the mathematics: brute force, closed forms, invariants and
hand-worked cases. A surviving mutant would be a mistake those pins cannot see.

An unmutated copy must pass the same pins. That shows the harness itself does not cause the failures.
"""
import os
import shutil
import subprocess
import sys
import textwrap
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.timeout(900)

C, PY = "tacg_oracle.c", "__init__.py"

# (name, file, text, replacement, occurrence of the text to replace, pin modules that must fail)
MUTANTS = [
    # ---- co-activation counts (Sec. 3.3) ----
    ("pairs counted in one order only", C, "if (a != b) C[", "if (a < b) C[", 0, ["counts"]),
    ("diagonal left at zero", C, "C[(int64_t)i * E + i] = D[i];", "C[(int64_t)i * E + i] = 0;", 0, ["counts"]),
    ("repeated ids accepted", C, "if (ids[s] == ids[s2]) err |= ORC_ERR_ID_DUP;", "if (0) err |= ORC_ERR_ID_DUP;", 0,
     ["counts"]),
    ("last token of every family dropped", C, "l, fam_off[f], fam_off[f + 1],",
     "l, fam_off[f], fam_off[f + 1] - (fam_off[f + 1] > fam_off[f]),", 0, ["counts"]),
    # ---- snapshot scoring (Sec. 3.4, App. C, App. H) ----
    ("loads of the first slot only", C, "for (int32_t s = 0; s < k; ++s) ld[slot_gpu[s]] += 1;",
     "for (int32_t s = 0; s < k; ++s) ld[slot_gpu[0]] += 1;", 0, ["score"]),
    ("single-candidate GPUs not reached first", C,
     "if (n_cand[e] == 1) { slot_gpu[s] = cand[e][0]; in_r[cand[e][0]] = 1; }",
     "if (n_cand[e] == 1) { slot_gpu[s] = cand[e][0]; }", 0, ["score"]),
    ("band test off by one", C, "if (in_r[m] && (m < home_start[f2] || m >= home_start[f2] + home_size[f2]))",
     "if (in_r[m] && (m < home_start[f2] || m > home_start[f2] + home_size[f2]))", 0, ["score"]),
    ("guard strict", C, "feas[m] = lhs <= rhs;", "feas[m] = lhs < rhs;", 0, ["score"]),
    ("guard without theta", C, "__int128 rhs = (__int128)(theta_den + theta_num) * total;",
     "__int128 rhs = (__int128)theta_den * total;", 0, ["score"]),
    ("highest reached candidate", C,
     "for (int32_t m = 0; m < G && pick < 0; ++m)\n                        if (fc[e][m] && in_r[m]) pick = m;",
     "for (int32_t m = G - 1; m >= 0 && pick < 0; --m)\n                        if (fc[e][m] && in_r[m]) pick = m;",
     0, ["score"]),
    ("anchor step left out", C, "if (pick < 0 && fc[e][h]) pick = h;", "if (pick < 0 && 0) pick = h;", 0,
     ["score"]),
    ("least-loaded ties to the highest GPU", C, "(pick < 0 || ref[m] < ref[pick])",
     "(pick < 0 || ref[m] <= ref[pick])", 0, ["score"]),
    ("fallback to the primary only", C,
     "if (!any)\n                for (int c = 0; c < n_cand[e]; ++c) fc[e][cand[e][c]] = 1;",
     "if (!any)\n                for (int c = 0; c < n_cand[e]; ++c) fc[e][cand[e][0]] = 1;", 0, ["score"]),
    ("anchor always the band start", C, "(int32_t)((t - fam_off[f]) % home_size[f])", "(int32_t)0", 0,
     ["score"]),
    ("span counts every card", C, "span_acc += n_cards - 1;", "span_acc += n_cards;", 0, ["score"]),
    ("home cost counts the anchor", C, "int64_t home_cost = n_cards - in_r[h];", "int64_t home_cost = n_cards;",
     0, ["score"]),
    ("every layer cross-family", C, "within_one = inside;", "within_one = 0;", 0, ["score"]),
    ("home mass counts every slot", C,
     "st_mass[f] += slot_gpu[s] >= home_start[f] && slot_gpu[s] < home_start[f] + home_size[f];",
     "st_mass[f] += 1;", 0, ["score"]),
    # ---- decayed-load scoring (Sec. 3.4, eq. load-update) ----
    ("no decay", C, "Lm[m] = fma(rho, Lm[m], (double)delta[m]);", "Lm[m] = Lm[m] + (double)delta[m];", 0,
     ["online"]),
    ("loads never updated", C, "Lm[m] = fma(rho, Lm[m], (double)delta[m]);",
     "Lm[m] = fma(rho, Lm[m], 0.0);", 0, ["online"]),
    ("decayed guard strict", C, "feas[m] = gden * Lm[m] <= rhs;", "feas[m] = gden * Lm[m] < rhs;", 0,
     ["online"]),
    ("decayed least-loaded ties to the highest GPU", C, "(pick < 0 || Lm[m] < Lm[pick])",
     "(pick < 0 || Lm[m] <= Lm[pick])", 0, ["online"]),
    ("decayed anchor step left out", C, "if (pick < 0 && fc[h]) pick = h;", "if (pick < 0 && 0) pick = h;", 0,
     ["online"]),
    ("decayed: anchor always the band start", C, "(int32_t)((t - fam_off[f]) % home_size[f])", "(int32_t)0", 1,
     ["online"]),
    ("decayed: span counts every card", C, "span_acc += n_cards - 1;", "span_acc += n_cards;", 1, ["online"]),
    ("decayed: home cost counts the anchor", C, "int64_t home_cost = n_cards - in_r[h];",
     "int64_t home_cost = n_cards;", 1, ["online"]),
    ("guard sum misses the last GPU", C, "for (int32_t m = 0; m < G; ++m) S += Lm[m];",
     "for (int32_t m = 0; m < G - 1; ++m) S += Lm[m];", 0, ["online"]),
    # ---- preferences and graph (Sec. 3.3) ----
    ("self pairs kept in A", PY, "np.fill_diagonal(A[f], 0.0)", "pass", 0, ["reweight"]),
    ("softmax over experts", PY, "w = np.exp(z - z.max(axis=0, keepdims=True))\n    p = w / w.sum(axis=0, keepdims=True)",
     "w = np.exp(z - z.max(axis=1, keepdims=True))\n    p = w / w.sum(axis=1, keepdims=True)", 0, ["reweight"]),
    ("graph normalised by its sum", PY, "ah = a_bar / mx if mx > 0 else np.zeros((E, E))",
     "ah = a_bar / a_bar.sum() if mx > 0 else np.zeros((E, E))", 0, ["reweight"]),
    ("sample standard deviation", PY, "sigma = np.sqrt(((x - mu) ** 2).mean())",
     "sigma = np.sqrt(((x - mu) ** 2).sum() / max(x.size - 1, 1))", 0, ["reweight"]),
    ("usage without the factor k", PY, "u[f] = D_l[f] / (n_f * top_k)", "u[f] = D_l[f] / n_f", 0,
     ["reweight"]),
    ("advantage over F families", PY, "dc[f] = c[f] - c[others].sum(axis=0) / (F - 1)",
     "dc[f] = c[f] - c[others].sum(axis=0) / F", 0, ["reweight"]),
    ("temperature multiplies", PY, "z = s / tau", "z = s * tau", 0, ["reweight"]),
    ("task kernel without the graph", PY, "alpha * (a_task * ah)", "alpha * a_task", 0, ["reweight"]),
    # ---- snapshot loads, Jain and MaxVio (App. H) ----
    ("snapshot loads of one family", PY, "out[p, l, prim[p, l, e]] += dsum[l, e]",
     "out[p, l, prim[p, l, e]] += D[0, l, e]", 0, ["score"]),
    ("Jain of the first layer only", PY, "return jain_maxvio(ld.sum(axis=1))", "return jain_maxvio(ld[:, 0])", 0,
     ["jain"]),
    ("Jain without G", PY, "tot ** 2 / (G * sq)", "tot ** 2 / sq", 0, ["jain"]),
    ("MaxVio over the total", PY, "(Lm.max(axis=-1) - mean) / mean", "(Lm.max(axis=-1) - mean) / tot", 0,
     ["jain"]),
    # ---- GESR scores (Sec. 3.4, eq. generic-score) and grouping objective (Sec. 3.3) ----
    ("consistency without normalisation", PY, "cs += float(A[f, e] @ a_bar[e]) / (na * nb)",
     "cs += float(A[f, e] @ a_bar[e])", 0, ["gesr_scores"]),
    ("specificity summed", PY, "worst = max(worst, float(np.sqrt(((A[f, e] - a_bar[e]) ** 2).sum())))",
     "worst = worst + float(np.sqrt(((A[f, e] - a_bar[e]) ** 2).sum()))", 0, ["gesr_scores"]),
    ("centrality of one family", PY, "cent[l, e] = a_bar[e].sum()", "cent[l, e] = A[0, e].sum()", 0,
     ["gesr_scores"]),
    ("objective over unordered pairs", PY, "if e2 != e:", "if e2 > e:", 0, ["objective"]),
    # ---- motivation diagnostics (App. H) ----
    ("activation probability without k", PY, "n = D[f, l].sum() / top_k", "n = D[f, l].sum()", 0,
     ["diagnostics"]),
    ("Jaccard over the larger set", PY, "out[l, i, j] = len(a & b) / u if u else 1.0",
     "out[l, i, j] = len(a & b) / max(len(a), len(b)) if u else 1.0", 0, ["diagnostics"]),
    ("activation distance in L1", PY, "dist[i, j] = np.sqrt(((Pm[i] - Pm[j]) ** 2).sum())",
     "dist[i, j] = np.abs(Pm[i] - Pm[j]).sum()", 0, ["diagnostics"]),
    ("zero-count pairs ranked", PY, "keep = cnt > 0", "keep = cnt >= 0", 0, ["diagnostics"]),
    ("top pairs ties to the higher index", PY, "np.lexsort((idx[keep], -cnt[keep]))",
     "np.lexsort((-idx[keep], -cnt[keep]))", 0, ["diagnostics"]),
]

# Runs the pin modules with the copy at `pkg` imported as the package `oracle`.
DRIVER = textwrap.dedent("""
    import importlib.util, os, sys
    pkg, root, files = sys.argv[1], sys.argv[2], sys.argv[3:]
    spec = importlib.util.spec_from_file_location("oracle", os.path.join(pkg, "__init__.py"),
                                                  submodule_search_locations=[pkg])
    mod = importlib.util.module_from_spec(spec)
    sys.modules["oracle"] = mod
    spec.loader.exec_module(mod)
    sys.path.insert(0, root)
    import pytest
    sys.exit(pytest.main(["-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu", "--rootdir", root, *files]))
""")


def _replace(text: str, old: str, new: str, occurrence: int) -> str:
    starts, i = [], text.find(old)
    while i >= 0:
        starts.append(i)
        i = text.find(old, i + 1)
    assert occurrence < len(starts), f"text to mutate not found: {old!r}"
    at = starts[occurrence]
    return text[:at] + new + text[at + len(old):]


def _run(workdir: str, mutant):
    name, fname, old, new, occ, pins = mutant
    pkg = os.path.join(workdir, "oracle")
    os.makedirs(pkg)
    for f in (C, PY):
        shutil.copy(os.path.join(ROOT, "oracle", f), os.path.join(pkg, f))
    if fname is not None:
        path = os.path.join(pkg, fname)
        with open(path) as fh:
            text = fh.read()
        with open(path, "w") as fh:
            fh.write(_replace(text, old, new, occ))
    driver = os.path.join(workdir, "driver.py")
    with open(driver, "w") as fh:
        fh.write(DRIVER)
    env = dict(os.environ)
    env.pop("TACG_ORACLE_LIBRARY", None)
    env.update(OMP_NUM_THREADS="2", PYTHONDONTWRITEBYTECODE="1")
    files = [os.path.join(ROOT, "tests", f"test_oracle_{p}.py") for p in pins]
    r = subprocess.run([sys.executable, driver, pkg, ROOT, *files], cwd=workdir, env=env, capture_output=True,
                       text=True, timeout=600)
    return r.returncode, (r.stdout + r.stderr)[-1500:]


def test_mutated_oracle_fails_its_pins(tmp_path):
    pins_all = sorted({p for m in MUTANTS for p in m[5]})
    control = ("unmutated copy", None, None, None, 0, pins_all)
    jobs = [control] + MUTANTS
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda im: _run(str(tmp_path / f"m{im[0]}"), im[1]), enumerate(jobs)))
    rc0, out0 = results[0]
    assert rc0 == 0, f"the unmutated copy fails its pins:\n{out0}"
    survivors = [(m[0], out) for m, (rc, out) in zip(MUTANTS, results[1:]) if rc == 0]
    broken = [(m[0], rc, out) for m, (rc, out) in zip(MUTANTS, results[1:]) if rc not in (0, 1)]
    assert not broken, f"mutants that did not run to a test verdict: {broken}"
    assert not survivors, "mutants no pin detects: " + ", ".join(s[0] for s in survivors)

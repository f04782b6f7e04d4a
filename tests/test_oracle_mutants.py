"""Planted mistakes: every variant of the oracle below carries one plausible
error (a dropped term, a wrong sign, index or table entry, a transposed
operand, a broken tie-break), and the oracle pins must reject each of them.

Each variant is a textual edit of a copy of the oracle source, built with the
same flags in a temporary directory; the pin suites then run against it in a
subprocess.  The unedited copy must pass.
"""

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_pins.py", "tests/test_oracle_terms.py", "tests/test_oracle_reduce.py",
        "tests/test_oracle_alpha.py", "tests/test_oracle_pareto.py", "tests/test_oracle_calib.py",
        "tests/test_oracle_flops.py"]

MUTANTS = {
    "forward peak drops the optimizer-step unit": (
        "const R BF = (base + Obuf) + Xd;", "const R BF = base + Xd;"),
    "backward peak drops the recomputed layer": (
        "const R BB = ((base + Gbuf) + Rc) + Xd;", "const R BB = (base + Gbuf) + Xd;"),
    "delta with the wrong sign": ("const R d = T1 - t;", "const R d = t - T1;"),
    "gradients sharded from ZeRO-1": (
        "const R sg = (z >= 2) ? iD : R(1.0);", "const R sg = (z >= 1) ? iD : R(1.0);"),
    "ZeRO-3 per-microbatch traffic 2 instead of 3": ("{0.0, 0.0, 1.0, 3.0}", "{0.0, 0.0, 1.0, 2.0}"),
    "first microbatch uses the stable ZeRO traffic": (
        "const R G2Gf = fma3(R(mf_tab[z]), r_, p2p);", "const R G2Gf = fma3(R(ms_tab[z]), r_, p2p);"),
    "interference divides by a neighbour's factor": (
        "alone[j] = (corun[j] - len) * R(psi[set * 4 + j]);",
        "alone[j] = (corun[j] - len) * R(psi[set * 4 + (j ^ 1)]);"),
    "interference phase lasts until the last stream ends": (
        "len = first ? corun[j] : min2(len, corun[j]);", "len = first ? corun[j] : max2(len, corun[j]);"),
    "interference keeps the all-stream factors after a stream ends": (
        "corun[j] = alone[j] * R(phi[set][j]);", "corun[j] = alone[j] * R(phi[15][j]);"),
    "activation swap-in uses the kept fraction": (
        "const R H2Ds = fma3(ra, A, HW) * iP;", "const R H2Ds = fma3(qa, A, HW) * iP;"),
    "recomputation counted twice": ("R(exact(3 * l + c))", "R(exact(3 * l + 2 * c))"),
    "stash ignores the accumulation steps": ("const R KA = R(exact(ke * Amb));", "const R KA = R(exact(k * Amb));"),
    "host and device streams transposed": (
        "const R Xs[4] = {C, G2Gs, H2Ds, D2Hs};", "const R Xs[4] = {C, G2Gs, D2Hs, H2Ds};"),
    "objective weights the first microbatch": ("const R obj = fma3(Gd, t, d);", "const R obj = fma3(Gd, T1, d);"),
    "frontier keeps equal objectives": ("if (bobj[j] < below)", "if (bobj[j] <= below)"),
    "ties broken by the highest id": ("(o1 == o2 && i1 < i2)", "(o1 == o2 && i1 > i2)"),
    "bucket edges shifted by one": ("(h.mem_bytes * (double)(j + 1))", "(h.mem_bytes * (double)(j + 2))"),
    "norm parameters split over TP": (
        "const int64_t Psi = (Pq + Pm) / TP + 2 * h * hkvr + Prep;",
        "const int64_t Psi = (Pq + Pm + Prep) / TP + 2 * h * hkvr;"),
    "one KV projection forgotten in the activations": ("+ 2 * hkvr + (m.flash", "+ hkvr + (m.flash"),
    "optimizer-step fetch takes the weight bytes": (
        "const R HX = fma3(ro, So, DG);", "const R HX = fma3(ro, So, DW);"),
    "weights fetched once per microbatch": ("const R HWz = R(2.0) * Sw;", "const R HWz = Sw;"),
    "logits missing from the backward peak": (
        "const R BB = ((base + Gbuf) + Rc) + Xd;", "const R BB = ((base + Gbuf) + Rc);"),
    "efficiency of the wrong microbatch": (
        "R(X.inv_eta[g.hw][pr.mb_index])", "R(X.inv_eta[g.hw][0])"),
    "weight sample applied to the delta instead of the time": (
        "for (int32_t a = 0; a < n_alpha; ++a) beta[a] = 1.0 - alphas[a];",
        "for (int32_t a = 0; a < n_alpha; ++a) beta[a] = alphas[a];"),
    "weight-sampled argmin ignores the memory budget": (
        "      if (bucket_of(X, g.hw, mem) < 0) return;  // Eq. 4 constraint: mem <= budget\n      const uint64_t id = g.base + (uint64_t)local;\n      for (int32_t a",
        "      const uint64_t id = g.base + (uint64_t)local;\n      for (int32_t a"),
    "weight-sampled argmin keeps the last of equal values": (
        "        if (lex_less(v, id, out_obj[o * n_alpha + a], out_id[o * n_alpha + a])) {",
        "        if (!(out_obj[o * n_alpha + a] < v)) {"),
    "exact frontier keeps equal objectives": (
        "    if (p.obj < run) {\n      if (n < cap)", "    if (p.obj <= run) {\n      if (n < cap)"),
    "exact frontier ordered by objective first": (
        "    if (a.mem != b.mem) return a.mem < b.mem;\n    if (a.obj != b.obj) return a.obj < b.obj;",
        "    if (a.obj != b.obj) return a.obj < b.obj;\n    if (a.mem != b.mem) return a.mem < b.mem;"),
    "pipeline sends counted once for middle stages": (
        "(int64_t)((k > 1) + (k < PP))", "(int64_t)((k > 1) || (k < PP))"),
    "measured efficiency multiplied instead of divided": (
        "ie.push_back(1.0 / h.eta_tab[i]);", "ie.push_back(h.eta_tab[i]);"),
    "operation counter scores a fused multiply-add as one operation": (
        "inline Counted fma3(Counted a, Counted b, Counted c) { g_flops += 2;",
        "inline Counted fma3(Counted a, Counted b, Counted c) { g_flops += 1;"),
    "operation counter scores a comparison (min/max) as an operation": (
        "inline bool operator<(Counted a, Counted b) { return a.v < b.v; }",
        "inline bool operator<(Counted a, Counted b) { ++g_flops; return a.v < b.v; }"),
    "operation counter skips subtractions": (
        "inline Counted operator-(Counted a, Counted b) { ++g_flops; return",
        "inline Counted operator-(Counted a, Counted b) { return"),
    "measured efficiency of the next microbatch size": (
        "ie.push_back(1.0 / h.eta_tab[i]);", "ie.push_back(1.0 / h.eta_tab[(i + 1) % X.mb.size()]);"),
}

# Planted mistakes in the plain-Python calibration reference (co-run window and fit).
CALIB_MUTANTS = {
    "fit takes the ratio of sums": ("        num[mask][j] += c * s\n        den[mask][j] += s * s",
                                    "        num[mask][j] += c\n        den[mask][j] += s"),
    "fit keeps speed-ups below 1": ("phi[mask][j] = max(1.0, num[mask][j] / den[mask][j])",
                                    "phi[mask][j] = num[mask][j] / den[mask][j]"),
    "window opens at the earliest start": ("lo = max(t[j][0] for j in members)", "lo = min(t[j][0] for j in members)"),
    "window keeps units that start before it": ("if t[j][i] >= lo and t[j][i + 1] <= hi:",
                                                "if t[j][i + 1] >= lo and t[j][i + 1] <= hi:"),
    "window mean over all units": ("            mean[j] = total / n", "            mean[j] = total / (len(t[j]) - 1)"),
}


def _build(tmp, name, src):
    path = os.path.join(tmp, name + ".cpp")
    with open(path, "w") as f:
        f.write(src)
    lib = os.path.join(tmp, name + ".so")
    subprocess.run(["g++", *O.CXXFLAGS, path, "-o", lib], check=True, capture_output=True)
    return lib


def _pins_pass(lib):
    env = dict(os.environ, MIST_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PINS],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode == 0, r.stdout[-2000:]


def test_planted_mistakes_are_caught():
    with open(O.SRC) as f:
        src = f.read()
    jobs = {"unchanged": src}
    for i, (what, (old, new)) in enumerate(MUTANTS.items()):
        assert src.count(old) == 1, what
        jobs["m%02d" % i] = src.replace(old, new)
    names = {"m%02d" % i: what for i, what in enumerate(MUTANTS)}
    with tempfile.TemporaryDirectory() as tmp:
        def run(item):
            key, text = item
            return key, _pins_pass(_build(tmp, key, text))
        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
            results = dict(ex.map(run, jobs.items()))
    ok, out = results.pop("unchanged")
    assert ok, out
    survivors = [names[k] for k, (passed, _) in sorted(results.items()) if passed]
    assert not survivors, "pins did not catch: %s" % survivors


# Planted mistakes in the plain-Python inter-stage planner (Eq. 1-3).
PLAN_MUTANTS = {
    "inner sum includes the stage itself": ("        v = d - t_sum\n        m = v if m is None else max(m, v)\n        t_sum = t_sum + t",
                                            "        t_sum = t_sum + t\n        v = d - t_sum\n        m = v if m is None else max(m, v)"),
    "G microbatches behind the bottleneck": ("return (float(G - 1) * t_max + t_sum) + m", "return (float(G) * t_max + t_sum) + m"),
    "stage i draws from the wrong in-flight count": ("cand.get((G, PP, PP - i, parts[i]), [])", "cand.get((G, PP, i + 1, parts[i]), [])"),
    "delta ignored": ("return (float(G - 1) * t_max + t_sum) + m", "return float(G - 1) * t_max + t_sum"),
}


@pytest.mark.parametrize("module,mutants,pins", [
    ("calib_oracle", "CALIB_MUTANTS", ["tests/test_oracle_calib.py"]),
    ("plan_oracle", "PLAN_MUTANTS", ["tests/test_oracle_plan.py", "tests/test_plan.py"]),
])
def test_planted_mistakes_in_the_python_references_are_caught(module, mutants, pins):
    """Each variant of a plain-Python reference (the calibration's window and fit, the planner)
    shadows the real one in a copy of the oracle package; its pins must fail on every variant and
    pass on the unedited copy."""
    import shutil
    src_path = os.path.join(ROOT, "oracle", module + ".py")
    with open(src_path) as f:
        src = f.read()
    lib = O.build(force=False)
    table = globals()[mutants]
    variants = {"unchanged": src}
    for i, (what, (old, new)) in enumerate(table.items()):
        assert src.count(old) == 1, what
        variants["c%02d" % i] = src.replace(old, new)
    names = {"c%02d" % i: what for i, what in enumerate(table)}
    with tempfile.TemporaryDirectory() as tmp:
        def run(item):
            key, text = item
            pkg = os.path.join(tmp, key, "oracle")
            os.makedirs(pkg)
            for fn in os.listdir(os.path.join(ROOT, "oracle")):
                if fn.endswith(".py"):
                    shutil.copy(os.path.join(ROOT, "oracle", fn), pkg)
            with open(os.path.join(pkg, module + ".py"), "w") as f:
                f.write(text)
            env = dict(os.environ, MIST_ORACLE_LIB=lib,
                       PYTHONPATH=os.pathsep.join([os.path.join(tmp, key), ROOT]))
            r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                                "-p", "no:randomly", "--rootdir", os.path.join(tmp, key),
                                *[os.path.join(ROOT, p) for p in pins]],
                               cwd=os.path.join(tmp, key), env=env, capture_output=True, text=True, timeout=300)
            return key, (r.returncode == 0, r.stdout[-1500:])
        with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
            results = dict(ex.map(run, variants.items()))
    ok, out = results.pop("unchanged")
    assert ok, out
    survivors = [names[k] for k, (passed, _) in sorted(results.items()) if passed]
    assert not survivors, "pins did not catch: %s" % survivors

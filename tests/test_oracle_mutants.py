"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of oracle/moe_oracle.cpp
(a sign, a dropped term, swapped operands, a wrong index, the tie order,
the router chain's start value or fusion), rebuilds the copy with g++ and
runs tests/test_oracle_pins.py against it.  Every mutant must fail at least
one pin; the unmutated copy must pass, so a failure means the pins caught
the mistake and not that the harness broke.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name -> (text in moe_oracle.cpp, replacement); each text occurs once
MUTANTS = {
    "silu_grad_sign": ("return s + z * s * (R(1) - s);", "return s - z * s * (R(1) - s);"),
    "dx_drops_dhu_term": ("    for (int n = 0; n < f; ++n) s += dhu[n] * widen<R>(u[n]);\n", ""),
    "silu_operands_swapped": ("a[n] = silu(hg[n]) * hu[n];", "a[n] = silu(hu[n]) * hg[n];"),
    "gate_up_weights_swapped": (
        "      hg[n] += xj * widen<R>(g[n]);\n      hu[n] += xj * widen<R>(u[n]);",
        "      hg[n] += xj * widen<R>(u[n]);\n      hu[n] += xj * widen<R>(g[n]);"),
    "ties_prefer_higher_index": ("return key(a) > key(b); });",
                                 "return key(a) > key(b) || (key(a) == key(b) && a > b); });"),
    "nan_ranks_first": ("return std::isnan(l[e]) ? -std::numeric_limits<L>::infinity() : l[e];",
                        "return std::isnan(l[e]) ? std::numeric_limits<L>::infinity() : l[e];"),
    "bias_sign": ("if (bias) acc = acc + bias[e];", "if (bias) acc = acc - bias[e];"),
    "dw_down_wrong_operand": ("const R am = a[p * f + m];", "const R am = dhg[p * f + m];"),
    "dy_perm_without_gate": ("dy_perm[p * d + c] = g * dv;", "dy_perm[p * d + c] = dv;"),
    "rank_reversed": ("const int64_t p = offsets[el] + run[el]++;",
                      "const int64_t p = offsets[el + 1] - 1 - run[el]++;"),
    "chain_starts_at_minus_zero": ("float acc = +0.0f;", "float acc = -0.0f;"),
    "chain_unfused": ("acc = std::fma(widen<float>(x[t * d + j]), w_r[(int64_t)j * E + e], acc);",
                      "acc = widen<float>(x[t * d + j]) * w_r[(int64_t)j * E + e] + acc;"),
    "router_bwd_renorm_sign": (
        "g[idx[t * k + i]] = gate[t * k + i] * (dgate[t * k + i] - s);",
        "g[idx[t * k + i]] = gate[t * k + i] * (dgate[t * k + i] + s);"),
}

_IGNORE = shutil.ignore_patterns("*.so", "*.so.tmp*", "__pycache__", "test_gpu_*", "test_oracle_mutants.py")


def _run(base, name, old, new):
    d = os.path.join(base, name)
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"), ignore=_IGNORE)
    shutil.copytree(os.path.join(ROOT, "tests"), os.path.join(d, "tests"), ignore=_IGNORE)
    shutil.copy(os.path.join(ROOT, "workloads.py"), d)
    src = os.path.join(d, "oracle", "moe_oracle.cpp")
    text = open(src).read()
    if old is not None:
        assert text.count(old) == 1, (name, text.count(old))
        text = text.replace(old, new)
        open(src, "w").write(text)
    env = dict(os.environ, OMP_NUM_THREADS="2", PYTHONDONTWRITEBYTECODE="1")
    # the mutant must compile: a failing pin then means a caught mistake
    build = subprocess.run([sys.executable, "-c", "import oracle; oracle.build(force=True)"],
                           cwd=d, env=env, capture_output=True, text=True, timeout=300)
    assert build.returncode == 0, (name, build.stderr[-2000:])
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_oracle_pins.py", "-x", "-q",
                        "-p", "no:cacheprovider"],
                       cwd=d, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-600:]


def test_every_planted_oracle_mistake_fails_a_pin(tmp_path):
    cases = [("control", None, None)] + [(n, o, w) for n, (o, w) in MUTANTS.items()]
    with ThreadPoolExecutor(max_workers=4) as ex:
        res = dict(zip([c[0] for c in cases],
                       ex.map(lambda c: _run(str(tmp_path), *c), cases)))
    rc, out = res.pop("control")
    assert rc == 0, "the unmutated copy must pass its pins:\n" + out
    survivors = {n: out for n, (rc, out) in res.items() if rc == 0}
    assert not survivors, "mutants no pin caught: " + ", ".join(survivors)
    # pytest exit code 1: tests ran and failed (not a collection or usage error)
    assert all(rc == 1 for rc, _ in res.values()), {n: rc for n, (rc, _) in res.items()}

"""Mutation check of the least-loaded plan's pins (CPU only).

Each case plants one plausible mistake in a copy of oracle/llep.py (a
dropped clamp, the capacity rounded the wrong way, a tie broken the other
way, the spill handed out in the wrong order, the load measured in rows
instead of units, the first spilled row counted in units) and runs
tests/test_oracle_llep.py against it.  Every mutant must fail at least one
pin; the unmutated copy must pass.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name -> (text in oracle/llep.py, replacement); each text occurs once
MUTANTS = {
    "keep_not_clamped": ("hi[r, e] = min(n[e], keep * g)", "hi[r, e] = keep * g"),
    "capacity_floor": ("-(-sum(u) // E_p))", "sum(u) // E_p)"),
    "least_loaded_ties_to_higher_rank": ("key=lambda q: (load_u[q], q))", "key=lambda q: (load_u[q], -q))"),
    "spill_smallest_first": ("key=lambda e: (-spill[e], e))", "key=lambda e: (spill[e], e))"),
    "piece_not_clamped": ("rows = min(n[e] - start, take * g)", "rows = take * g"),
    "least_loaded_by_rows": ("key=lambda q: (load_u[q], q))", "key=lambda q: (load_rows[q], q))"),
    "first_spilled_row_in_units": ("start = (u[e] - spill[e]) * g", "start = n[e] - spill[e]"),
    "units_rounded_down": ("u = [-(-c // g) for c in n]", "u = [c // g for c in n]"),
}


def _run(base, name, old, new):
    d = os.path.join(base, name)
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"),
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    os.makedirs(os.path.join(d, "tests"))
    for f in ("__init__.py", "conftest.py", "test_oracle_llep.py"):
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(d, "tests", f))
    src = os.path.join(d, "oracle", "llep.py")
    text = open(src).read()
    if old is not None:
        assert text.count(old) == 1, (name, text.count(old))
        open(src, "w").write(text.replace(old, new))
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1", MOE_ORACLE_LIB=os.devnull)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_llep.py"], cwd=d, env=env, capture_output=True, text=True,
                       timeout=600)
    return name, r.returncode, r.stdout[-1500:] + r.stderr[-1500:]


def test_every_planted_llep_mistake_fails_a_pin(tmp_path):
    cases = [("unmutated", None, None)] + [(k, a, b) for k, (a, b) in MUTANTS.items()]
    with ThreadPoolExecutor(4) as ex:
        res = list(ex.map(lambda c: _run(str(tmp_path), *c), cases))
    base = res[0]
    assert base[1] == 0, f"the unmutated copy fails its pins:\n{base[2]}"
    survivors = [(n, out) for n, rc, out in res[1:] if rc == 0]
    assert not survivors, "mutants no pin caught: " + ", ".join(n for n, _ in survivors)

"""Every plausible mistake planted in the oracle must fail at least one pin.

Each mutant is a copy of the oracle source with one textual change (a
dropped term, a wrong sign, a wrong index or bound, a skipped sort, a broken
mask test), compiled with gcc into a temporary library on the CPU.  The pin
suite of ``oracle_pins.py`` is then run against it and has to fail.
"""
import json
import os
import subprocess
import sys

import pytest

import oracle
import oracle_pins as pins

MUTANTS = {
    "sign": ("acc[i] += prod;", "acc[i] -= prod;"),
    "drop_x": ("double prod = cvals[p] * xj;", "double prod = cvals[p];"),
    "wrong_row": ("            int32_t i = row_idx[p];\n            if (!row_allowed(mask, complement, i)) continue;\n            double prod",
                  "            int32_t i = row_idx[p] % (j + 1);\n            if (!row_allowed(mask, complement, i)) continue;\n            double prod"),
    "drop_last_entry": ("        double xj = x_val[t];\n        for (int64_t p = col_ptr[j]; p < col_ptr[j + 1]; ++p)",
                        "        double xj = x_val[t];\n        for (int64_t p = col_ptr[j]; p < col_ptr[j + 1] - 1; ++p)"),
    "abs_scale": ("sabs[i] += prod < 0 ? -prod : prod;", "sabs[i] += prod;"),
    "unsorted_y": ("    qsort(touched, (size_t)nt, sizeof(int32_t), cmp_i32);\n", ""),
    "mask_inverted": ("return complement ? !bit : bit;", "return complement ? bit : !bit;"),
    "mask_bit_order": ("(mask[i >> 5] >> (i & 31)) & 1u", "(mask[i >> 5] >> (31 - (i & 31))) & 1u"),
    "bool_dupes": ("            if (!seen[i]) { seen[i] = 1; y_idx[nt++] = i; }",
                   "            if (!seen[i]) { seen[i] = 1; y_idx[nt++] = i; } else if (nt < m) { y_idx[nt++] = i; }"),
    "csc_shifted": ("            row_idx[q] = i;", "            row_idx[q] = i > 0 ? i - 1 : i;"),
    "bfs_no_sort": ("        qsort(frontier, (size_t)nf, sizeof(int32_t), cmp_i32);\n", ""),
    "bfs_parent_self": ("                    parent[v] = u;", "                    parent[v] = v;"),
    "bfs_level_off": ("                    level[v] = L + 1;", "                    level[v] = L;"),
    "bfs_last_parent": ("                if (level[v] == -1) {",
                        "                if (level[v] == L + 1) parent[v] = u;\n                if (level[v] == -1) {"),
}


# The pins run against a mutant in a child process: a mutant may write out of
# bounds, and its damage must not reach the test process.  A child that dies
# (a mutant that crashes) has failed the pins as well.
_CHILD = """
import json, sys
sys.path[:0] = [{tests!r}, {root!r}]
import oracle_pins as pins
caught = []
for check in pins.ALL_CHECKS:
    try:
        check(lib_path={lib!r})
    except (AssertionError, ValueError, IndexError) as e:
        caught.append([check.__name__, type(e).__name__])
print(json.dumps(caught), flush=True)
"""


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(oracle._SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    mutated = src.replace(old, new, 1)
    msrc = tmp_path / "oracle_mut.c"
    msrc.write_text(mutated)
    lib = str(tmp_path / f"liboracle_{name}.so")
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-o", lib, str(msrc)], check=True)
    here = os.path.dirname(os.path.abspath(__file__))
    code = _CHILD.format(tests=here, root=os.path.dirname(here), lib=lib)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    if r.returncode == 0:
        caught = json.loads(r.stdout.strip().splitlines()[-1])
    else:
        caught = [["child", f"exit status {r.returncode}"]]
    assert caught, f"mutant {name} survived every pin"
    os.remove(lib)


# Plausible slips in the acceptance rule every value comparison uses; each
# must fail the rule's own pin (check_within_tol).
TOL_MUTANTS = {
    "tol_rel_plus_S": ("rel * s", "rel + s"),
    "tol_no_abs": ("np.abs(g - r)", "(g - r)"),
    "tol_strict": ("<= rel * s", "< rel * s"),
    "tol_ref_scaled": ("rel * s", "rel * np.abs(r)"),
    "tol_nan_either": ("np.isnan(g) & np.isnan(r)", "np.isnan(g) | np.isnan(r)"),
    "tol_no_nan_rule": ("return close | same | both_nan", "return close | same"),
    "tol_infinite_ref": ("np.isfinite(r) & ", ""),
    "tol_reduced": ("return close | same | both_nan", "return bool(np.all(close | same | both_nan))"),
    "tol_broadcast": ("if g.shape != r.shape or g.shape != s.shape:", "if False:"),
    "tol_rel_ignored": ("rel * s", "1e-5 * s"),
}


@pytest.mark.parametrize("name", sorted(TOL_MUTANTS))
def test_tolerance_mutant_is_caught(name):
    import inspect
    import textwrap

    import numpy as np

    old, new = TOL_MUTANTS[name]
    src = textwrap.dedent(inspect.getsource(oracle.within_tol))
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    ns = {"np": np}
    exec(compile(src.replace(old, new, 1), f"<within_tol:{name}>", "exec"), ns)
    with pytest.raises((AssertionError, ValueError, TypeError)):
        pins.check_within_tol(fn=ns["within_tol"])

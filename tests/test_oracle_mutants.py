"""Plant plausible mistakes in copies of the oracle source and check that the pins catch each.

Each mutant is a text edit of ``oracle/eqref.c`` compiled into a temporary
library and exercised in a child process (a mutant may index out of bounds).
A mutant is caught when any pin fails or the child crashes.  CPU only.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "eqref.c")

# (name, old text, new text, occurrence index among matches)
MUTANTS = [
    ("fwd_lag_sign", "const int s = wrap(t - j, T);\n          for (int c", "const int s = wrap(t + j, T);\n          for (int c", 0),
    ("fwd_lag_offset", "const int s = wrap(t - j, T);\n          for (int c", "const int s = wrap(t - j + 1, T);\n          for (int c", 0),
    ("fwd_drop_bias", "if (b) acc += b[o];", "(void)b;", 0),
    ("fwd_drop_last_channel", "for (int c = 0; c < Cin; ++c)\n            acc += w", "for (int c = 0; c < Cin - 1; ++c)\n            acc += w", 0),
    ("fwd_transposed_weight", "acc += w[IDX3(j, o, c, Cout, Cin)] * x", "acc += w[IDX3(j, c % Cout, o % Cin, Cout, Cin)] * x", 0),
    ("fwd_x_index_swap", "x[IDX3(n, c, s, Cin, T)];\n        }", "x[IDX3(n, s % Cin, c % T, Cin, T)];\n        }", 0),
    ("dx_gather_sign", "const int t = wrap(s + j, T);", "const int t = wrap(s - j, T);", 0),
    ("dx_weight_lag", "acc += w[IDX3(j, o, c, Cout, Cin)] * dy", "acc += w[IDX3((T - j) % T, o, c, Cout, Cin)] * dy", 0),
    ("dw_lag_sign", "const int s = wrap(t - j, T);\n        for (int c", "const int s = wrap(t + j, T);\n        for (int c", 0),
    ("dw_skip_first_row", "for (int64_t n = 0; n < N; ++n) {\n      for (int t = 0; t < T; ++t) {\n        const double g", "for (int64_t n = 1; n < N; ++n) {\n      for (int t = 0; t < T; ++t) {\n        const double g", 0),
    ("db_drop_group_term", "for (int t = 0; t < T; ++t) acc += dy", "for (int t = 1; t < T; ++t) acc += dy", 0),
    ("entries_lag_sign", "const int s = wrap(t - j[e], T);", "const int s = wrap(t + j[e], T);", 0),
]

CHILD = r"""
import sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import oracle
from oracle_pins import ALL_PINS
orc = oracle.Oracle(oracle.load({lib!r}))
failed = []
for pin in ALL_PINS:
    try:
        pin(orc)
    except AssertionError:
        failed.append(pin.__name__)
print("FAILED:" + ",".join(failed))
"""


def _mutate(text, old, new, occ):
    start = -1
    for _ in range(occ + 1):
        start = text.find(old, start + 1)
        assert start >= 0, "mutation anchor not found: %r" % old
    return text[:start] + new + text[start + len(old):]


@pytest.mark.parametrize("name,old,new,occ", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, old, new, occ):
    import oracle
    with open(SRC) as f:
        text = f.read()
    mutated = _mutate(text, old, new, occ)
    assert mutated != text
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "eqref_mut.c")
        lib = os.path.join(d, "libeqref_mut.so")
        with open(src, "w") as f:
            f.write(mutated)
        oracle.build(src, lib)
        code = CHILD.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
        env = dict(os.environ, OMP_NUM_THREADS="2")
        r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                           timeout=600, env=env)
        if r.returncode != 0:
            return  # crashed: caught
        line = [l for l in r.stdout.splitlines() if l.startswith("FAILED:")][-1]
        caught = [p for p in line[len("FAILED:"):].split(",") if p]
        assert caught, "mutant %s passed every pin" % name

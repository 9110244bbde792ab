"""Plant plausible mistakes into copies of the oracle source (on the CPU) and
check that the pins reject every one of them."""
import os
import tempfile

import pytest

from oracle import oracle
from tests import oracle_pins as pins

# (name, text to replace, replacement): each is a mistake someone could make
# while writing Eq. 1-4 as loops.
MUTANTS = [
    ("window_edge_le", "(i - j < w)", "(i - j <= w)"),
    ("distant_scale_sqrt_ddown", "s[j] = acc * scale;",
     "s[j] = acc * ((i - j < w) ? scale : 2.0 * scale);"),
    ("scale_dropped", "s[j] = acc * scale;", "s[j] = acc;"),
    ("value_uses_lifted_key", "v + (size_t)j * d : vl + (size_t)j * d",
     "v + (size_t)j * d : kl + (size_t)j * d"),
    ("tied_up_not_transposed", "wd[(size_t)e * dd + c];", "wd[(size_t)c * d + e];"),
    ("untied_up_transposed", "wu[(size_t)c * d + e]", "wu[(size_t)e * dd + c]"),
    ("self_excluded", "for (int j = 0; j <= i; ++j) {\n        const double* key",
     "for (int j = 0; j < i; ++j) {\n        const double* key"),
    ("sum_drops_first_term", "sum += s[j]; }", "if (j > 0) sum += s[j]; }"),
    ("gqa_interleaved", "const int g = h / group;", "const int g = h % Hkv;"),
    ("down_wrong_operand", "acc += x[(size_t)t * d + e] * wd[(size_t)e * dd + c];",
     "acc += x[(size_t)t * d + e] * wd[(size_t)c * d + e % dd];"),
    ("lift_only_keys", "double* vl = lift_all(T, d, dd, v, wd, wu);",
     "double* vl = lift_all(T, d, dd, k, wd, wu);"),
    ("max_not_subtracted_sign", "s[j] = exp(s[j] - m);", "s[j] = exp(m - s[j]);"),
]


def _cheap_checks():
    # everything except the pure-Python brute force (slow); it is covered
    # by the unmutated pin run
    return [c for c in pins.ALL_CHECKS if c is not pins.check_brute_force]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, old, new):
    with open(oracle.SRC) as f:
        src = f.read()
    assert src.count(old) >= 1, "mutation site not found: " + name
    with tempfile.TemporaryDirectory() as td:
        cpath = os.path.join(td, "mutant.c")
        with open(cpath, "w") as f:
            f.write(src.replace(old, new))
        lib = oracle.compile_source(cpath, os.path.join(td, "libmutant.so"))
        orc = oracle.Oracle(lib)
        caught = []
        for check in _cheap_checks():
            try:
                check(orc)
            except (AssertionError, ValueError):
                caught.append(check.__name__)
        assert caught, "no pin rejects mutant " + name

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
    ("lse_drops_max", "if (lse) *lse = m + log(sum);", "if (lse) *lse = log(sum);"),
    # backward
    ("bwd_softmax_jacobian_drops_delta", "const double ds = p[j] * (dp[j] - delta);",
     "const double ds = p[j] * dp[j];"),
    ("bwd_dq_unscaled", "dqi[e] += ds * key[e] * scale;", "dqi[e] += ds * key[e];"),
    ("bwd_dv_uses_ds", "dval[e] += p[j] * doi[e];", "dval[e] += ds * doi[e];"),
    ("bwd_window_edge_le", "const int local = i - j < w;", "const int local = i - j <= w;"),
    ("bwd_tied_misses_up_term", "else dwdg[(size_t)e * dd + c] += u[(size_t)c * d + e];",
     "else (void)0;"),
    ("bwd_lift_skips_input_gradient", "dxb[(size_t)j * d + e] += u * wdg[(size_t)e * dd + c];",
     "(void)dxb;"),
    ("bwd_dwd_uses_latent", "pwdg[(size_t)e * dd + c] += xj[e] * u;",
     "pwdg[(size_t)e * dd + c] += xj[e] * hc;"),
    ("bwd_delta_from_key", "delta += p[j] * acc;", "delta += p[j] * acc * (j > 0);"),
    ("bwd_dwu_from_gradient_of_key_only", "const double* dxl = which ? dvl : dkl;",
     "const double* dxl = dkl;"),
    # RoPE inside Eq. 3
    ("rope_sin_sign", "yr[m] = xr[m] * c - xr[m + half] * s;", "yr[m] = xr[m] * c + xr[m + half] * s;"),
    ("rope_pairs_adjacent",
     "yr[m] = xr[m] * c - xr[m + half] * s;\n            yr[m + half] = xr[m + half] * c + xr[m] * s;",
     "yr[2 * m] = xr[2 * m] * c - xr[2 * m + 1] * s;\n            yr[2 * m + 1] = xr[2 * m + 1] * c + xr[2 * m] * s;"),
    ("rope_frequency_over_d", "(double)pos[t] * pow(base, -2.0 * m / r)",
     "(double)pos[t] * pow(base, -2.0 * m / d)"),
    ("rope_distant_key_unrotated", "qrr + (size_t)i * d, kr, v, klr, vl,", "qrr + (size_t)i * d, kr, v, kl, vl,"),
    ("rope_window_key_unrotated", "qrr + (size_t)i * d, kr, v, klr, vl,", "qrr + (size_t)i * d, k, v, klr, vl,"),
    ("rope_query_unrotated", "qrr + (size_t)i * d, kr, v, klr, vl,", "qr + (size_t)i * d, kr, v, klr, vl,"),
    ("rope_query_position_shifted", "qpos[i] = pos0 + pos[i];", "qpos[i] = pos0 + pos[i] + 1;"),
    # single shared latent
    ("shared_value_lifted_with_key_matrix", "av += c[(size_t)j * dd + cc] * uv[(size_t)cc * d + e];",
     "av += c[(size_t)j * dd + cc] * uk[(size_t)cc * d + e];"),
    ("shared_key_lifted_with_value_matrix", "ak += c[(size_t)j * dd + cc] * uk[(size_t)cc * d + e];",
     "ak += c[(size_t)j * dd + cc] * uv[(size_t)cc * d + e];"),
    ("shared_matrix_transposed", "uk[(size_t)cc * d + e]", "uk[(size_t)e * dd + cc % dd]"),
    ("shared_distant_uses_full_value", "one_row(d, w, pos[i], qr + (size_t)i * d, k, v, kl, vl, s, o + (size_t)i * d,\n                            NULL, lse ? lse + i : NULL);",
     "one_row(d, w, pos[i], qr + (size_t)i * d, k, v, kl, v, s, o + (size_t)i * d,\n                            NULL, lse ? lse + i : NULL);"),
    # RoPE in the backward
    ("bwd_rope_dq_rotated_forward", "dar_oracle_rope(T, d, r, base, npos, dqr, dq",
     "dar_oracle_rope(T, d, r, base, tpos, dqr, dq"),
    ("bwd_rope_window_key_grad_rotated_forward", "dar_oracle_rope(T, d, r, base, npos, dkr, dkb);",
     "dar_oracle_rope(T, d, r, base, tpos, dkr, dkb);"),
    ("bwd_rope_distant_key_grad_not_rotated_back", "dar_oracle_rope(T, d, r, base, npos, dkd, dkl);",
     "memcpy(dkl, dkd, sizeof(double) * td);"),
    ("bwd_rope_distant_pairs_use_window_key",
     "const double* key = local ? kr + (size_t)j * d : kdr + (size_t)j * d;",
     "const double* key = kr + (size_t)j * d;"),
    ("bwd_rope_distant_keys_unrotated", "dar_oracle_rope(T, d, r, base, tpos, kl, kdr);",
     "memcpy(kdr, kl, sizeof(double) * td);"),
    ("rope_before_lift", "dar_oracle_rope(T, d, r, base, tpos, kl, klr);",
     "{ double* t_ = lift_all(T, d, dd, kr, wd, wu); memcpy(klr, t_, sizeof(double) * (size_t)T * d); free(t_); }"),
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

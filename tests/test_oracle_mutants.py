"""Planted mistakes in a copy of the oracle must each fail at least one pin.

Each mutant is a one-line edit of ``oracle/bdlm_oracle.c`` of the kind a slip in
reading the paper would produce (a dropped term, a wrong sign, an index off by
one, a swapped operand).  The copy is compiled with gcc into a temporary
directory and swapped in for the real oracle only inside this test; the real
source is never touched.
"""
import ctypes
import os
import subprocess

import pytest

import oracle
import tests.test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "bdlm_oracle.c")

# (name, text in the source, replacement)
MUTANTS = [
    ("decay-sign", "const double a = exp(dtv * A_h);", "const double a = exp(-dtv * A_h);"),
    ("no-dt-on-input", "a * S[p * N + n] + dtv * xv * bv", "a * S[p * N + n] + xv * bv"),
    ("zoh-style-input", "a * S[p * N + n] + dtv * xv * bv",
     "a * S[p * N + n] + (a - 1.0) / A_h * xv * bv"),
    ("readout-before-update",
     "S[p * N + n] = a * S[p * N + n] + dtv * xv * bv;\n            acc += S[p * N + n] *",
     "acc += S[p * N + n] *"),
    ("B-C-swapped", "const double bv = rd(Bm,", "const double bv = rd(Cm,"),
    ("skip-dropped", "if (out) out[p] = acc + skip * xv;", "if (out) out[p] = acc;"),
    ("reverse-skip-uses-D", "(double)D_rev[h],\n                             yr + t * P",
     "(double)D[h],\n                             yr + t * P"),
    ("reverse-starts-from-cache", "memset(R, 0, sizeof(double) * P * N);",
     "memcpy(R, h_pool + (slot * H + h) * P * N, sizeof(double) * P * N);"),
    ("decay-includes-own-input", "a * S[p * N + n] + dtv * xv * bv",
     "a * (S[p * N + n] + dtv * xv * bv)"),
    ("reverse-skips-last-token", "for (int64_t t = L - 1; t >= 0; --t)",
     "for (int64_t t = L - 2; t >= 0; --t)"),
    ("forward-only-output", "y[o] = yf[t * P + p] + yr[t * P + p];", "y[o] = yf[t * P + p];"),
    ("wrong-group", "const int64_t g = h / hpg;", "const int64_t g = h % s->ngroups;"),
    ("commit-offset-unchecked", "n_blocks[slot] != expected_block_index", "0"),
    ("commit-counts-blocks-as-tokens", "n_committed[slot] += s->len;", "n_committed[slot] += 1;"),
    ("bf16-decode-shift", "(uint32_t)((const uint16_t *)base)[i] << 16",
     "(uint32_t)((const uint16_t *)base)[i] << 15"),
]

PIN_TESTS = [
    lambda: pins.test_hand_example(),
    lambda: pins.test_closed_form_constant_inputs(-1.5, 0.25, 7),
    lambda: pins.test_closed_form_constant_inputs(-3.0, 0.125, 1),
    lambda: pins.test_single_token_block(),
    lambda: pins.test_zero_B_and_zero_C(),
    lambda: pins.test_scans_as_bidiagonal_linear_systems(False),
    lambda: pins.test_scans_as_bidiagonal_linear_systems(True),
    lambda: pins.test_dual_form(True, 7),
    lambda: pins.test_reverse_is_flip_of_forward_on_flipped_block(),
    lambda: pins.test_reverse_ignores_cache_and_palindrome_symmetry(),
    lambda: pins.test_commits_equal_one_pass_bitwise(),
    lambda: pins.test_commit_offset_and_slot_checks_leave_state_untouched(),
    lambda: pins.test_bf16_encoding(),
]


def _load_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutant {name}: pattern not found in the oracle source"
    msrc = tmp_path / f"{name}.c"
    msrc.write_text(src.replace(old, new, 1))
    so = tmp_path / f"{name}.so"
    subprocess.run(["gcc", "-O1", "-shared", "-fPIC", "-std=c11", "-o", str(so), str(msrc),
                    "-lm"], check=True, capture_output=True)
    return ctypes.CDLL(str(so))


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new, monkeypatch):
    real = oracle.lib()
    mut = _load_mutant(tmp_path, name, old, new)
    for f in ("bdlm_oracle_block_step", "bdlm_oracle_commit", "bdlm_oracle_scan_forward",
              "bdlm_oracle_full_window", "bdlm_oracle_num_threads"):
        getattr(mut, f).argtypes = getattr(real, f).argtypes
        getattr(mut, f).restype = getattr(real, f).restype
    monkeypatch.setattr(oracle, "_lib", mut)
    caught = []
    for i, pin in enumerate(PIN_TESTS):
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(i)
    assert caught, f"no pin catches mutant {name}"


# Mutants of the convolution part (oracle.conv), caught by the convolution pins.
import tests.test_oracle_conv as cpins  # noqa: E402

CONV_MUTANTS = [
    ("conv-kernel-reversed", "vf += (double)w[c * 4 + k] * u[3 + t - 3 + k];",
     "vf += (double)w[c * 4 + 3 - k] * u[3 + t - 3 + k];"),
    ("conv-no-silu", "if (of) of[oi + t * ts] = silu(vf);", "if (of) of[oi + t * ts] = vf;"),
    ("conv-bias-dropped", "double vf = bias[c], vr = bias[c];", "double vf = 0.0, vr = bias[c];"),
    ("conv-reverse-reads-cache", "for (int k = 0; k < 3; ++k) u[L + 3 + k] = 0.0;",
     "for (int k = 0; k < 3; ++k) u[L + 3 + k] = u[k];"),
    ("conv-reverse-window-shifted", "vr += (double)w[c * 4 + k] * u[3 + t + 3 - k];",
     "vr += (double)w[c * 4 + k] * u[3 + t + 2 - k];"),
    ("conv-cache-rows-reversed", "for (int k = 0; k < 3; ++k) u[k] = crow[k * ch + c];",
     "for (int k = 0; k < 3; ++k) u[k] = crow[(2 - k) * ch + c];"),
    ("conv-commit-keeps-first-rows", "for (int k = 0; k < 3; ++k) crow[k * ch + c] = u[L + k];",
     "for (int k = 0; k < 3; ++k) crow[k * ch + c] = u[3 + k];"),
]

CONV_PINS = [
    lambda: cpins.test_identity_kernel_gives_silu_of_the_input(),
    lambda: cpins.test_against_numpy_correlate(5),
    lambda: cpins.test_against_numpy_correlate(1),
    lambda: cpins.test_reverse_is_flip_of_forward_from_zero(),
    lambda: cpins.test_cache_continuation_equals_one_pass(),
    lambda: cpins.test_commit_keeps_last_three_rows(1),
    lambda: cpins.test_commit_keeps_last_three_rows(6),
]


@pytest.mark.parametrize("name,old,new", CONV_MUTANTS, ids=[m[0] for m in CONV_MUTANTS])
def test_conv_mutant_is_caught(tmp_path, name, old, new, monkeypatch):
    mut = _load_mutant(tmp_path, name, old, new)
    monkeypatch.setattr(oracle, "_lib", mut)
    caught = []
    for i, pin in enumerate(CONV_PINS):
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(i)
    assert caught, f"no pin catches mutant {name}"


# Mutants of the gated RMS normalisation (oracle.gated_rmsnorm), caught by its pins.
import tests.test_oracle_norm as npins  # noqa: E402

NORM_MUTANTS = [
    ("norm-no-gate", "g[c] = y[t * nch + c] * silu(rd(z, t * nch + c, zdtype));",
     "g[c] = y[t * nch + c];"),
    ("norm-gate-is-sigmoid", "g[c] = y[t * nch + c] * silu(rd(z, t * nch + c, zdtype));",
     "g[c] = y[t * nch + c] / (1.0 + exp(-rd(z, t * nch + c, zdtype)));"),
    ("norm-mean-over-all-channels", "sqrt(ss / (double)gs + eps)", "sqrt(ss / (double)nch + eps)"),
    ("norm-eps-outside-sqrt", "1.0 / sqrt(ss / (double)gs + eps)", "1.0 / (sqrt(ss / (double)gs) + eps)"),
    ("norm-eps-on-sum", "sqrt(ss / (double)gs + eps)", "sqrt((ss + eps) / (double)gs)"),
    ("norm-weight-dropped", "out[t * nch + c] = (double)w[c] * g[c] * r;", "out[t * nch + c] = g[c] * r;"),
    ("norm-sums-first-group", "for (int64_t c = k * gs; c < (k + 1) * gs; ++c) ss += g[c] * g[c];",
     "for (int64_t c = 0; c < gs; ++c) ss += g[c] * g[c];"),
]

NORM_PINS = [
    lambda: npins.test_hand_example_and_gate_sign(),
    lambda: npins.test_gate_is_silu_against_scipy_expit(),
    lambda: npins.test_unit_mean_square_per_group(2),
    lambda: npins.test_weight_scales_each_channel(),
    lambda: npins.test_eps_closed_form(),
    lambda: npins.test_groups_are_independent_and_consecutive(),
]


@pytest.mark.parametrize("name,old,new", NORM_MUTANTS, ids=[m[0] for m in NORM_MUTANTS])
def test_norm_mutant_is_caught(tmp_path, name, old, new, monkeypatch):
    mut = _load_mutant(tmp_path, name, old, new)
    monkeypatch.setattr(oracle, "_lib", mut)
    caught = []
    for i, pin in enumerate(NORM_PINS):
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(i)
    assert caught, f"no pin catches mutant {name}"

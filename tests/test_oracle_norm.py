"""Pins of the oracle's gated RMS normalisation (the Mamba-2 mixer's output path after
the scan, App. C): out = w * g / sqrt(mean_group(g^2) + eps), g = y * silu(z), checked
against hand values, closed forms, invariants and scipy's logistic function.  CPU only."""
import numpy as np
import pytest
from scipy.special import expit

import oracle


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def test_hand_example_and_gate_sign():
    """y = (3, 4), one z for both channels, w = 1, eps = 0: g = silu(z) * (3, 4), so
    out = sign(silu(z)) * (3, 4) / sqrt(12.5) = sign * (0.848528..., 1.131370...)."""
    y = np.array([[3.0, 4.0], [3.0, 4.0]])
    z = np.array([[1.0, 1.0], [-1.0, -1.0]], np.float32)     # silu(-1) < 0
    out = oracle.gated_rmsnorm(y, z, np.ones(2, np.float32), 0.0)
    want = np.array([3.0, 4.0]) / np.sqrt(12.5)
    np.testing.assert_allclose(out[0], want, rtol=1e-14)
    np.testing.assert_allclose(out[1], -want, rtol=1e-14)


def test_gate_is_silu_against_scipy_expit():
    """y = 1, w = 1, eps = 0: out[c] = s_c / sqrt(mean(s^2)), s = z * logistic(z)."""
    z = (rng(1).standard_normal((3, 128)) * 3).astype(np.float32)
    out = oracle.gated_rmsnorm(np.ones((3, 128)), z, np.ones(128, np.float32), 0.0)
    s = z.astype(np.float64) * expit(z.astype(np.float64))
    want = s / np.sqrt(np.mean(s * s, axis=-1, keepdims=True))
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("ngroups", [1, 2, 4])
def test_unit_mean_square_per_group(ngroups):
    """w = 1, eps = 0: every group of every token has mean(out^2) = 1 exactly."""
    r = rng(2 + ngroups)
    y = r.standard_normal((5, 256))
    z = r.standard_normal((5, 256)).astype(np.float32)
    out = oracle.gated_rmsnorm(y, z, np.ones(256, np.float32), 0.0, ngroups)
    ms = np.mean(out.reshape(5, ngroups, -1) ** 2, axis=-1)
    np.testing.assert_allclose(ms, 1.0, rtol=1e-12)


def test_weight_scales_each_channel():
    r = rng(7)
    y = r.standard_normal((4, 128))
    z = r.standard_normal((4, 128)).astype(np.float32)
    w = r.standard_normal(128).astype(np.float32)
    one = oracle.gated_rmsnorm(y, z, np.ones(128, np.float32), 1e-5, 2)
    np.testing.assert_allclose(oracle.gated_rmsnorm(y, z, w, 1e-5, 2), one * w, rtol=1e-13)


def test_eps_closed_form():
    """z = 30 (silu(30) = 30 up to 1e-13), y = (3, 4) * a, eps = 11250 a^2:
    out = 30 a (3, 4) / sqrt(900 a^2 * 12.5 + 11250 a^2) = (3, 4) / 5."""
    for a in (1.0, 0.01):
        y = np.array([[3.0, 4.0]]) * a
        out = oracle.gated_rmsnorm(y, np.full((1, 2), 30.0, np.float32), np.ones(2, np.float32),
                                   11250.0 * a * a)
        np.testing.assert_allclose(out[0], [0.6, 0.8], rtol=1e-12)


def test_scale_and_sign_invariance():
    r = rng(9)
    y = r.standard_normal((3, 64))
    z = r.standard_normal((3, 64)).astype(np.float32)
    w = np.ones(64, np.float32)
    base = oracle.gated_rmsnorm(y, z, w, 0.0)
    np.testing.assert_allclose(oracle.gated_rmsnorm(7.5 * y, z, w, 0.0), base, rtol=1e-12)
    np.testing.assert_allclose(oracle.gated_rmsnorm(-y, z, w, 0.0), -base, rtol=1e-14)


def test_groups_are_independent_and_consecutive():
    """Changing one group's inputs leaves the other groups alone, and each group of 64
    consecutive channels is normalised as if it were a token of its own."""
    r = rng(11)
    y = r.standard_normal((2, 192))
    z = r.standard_normal((2, 192)).astype(np.float32)
    w = r.standard_normal(192).astype(np.float32)
    out = oracle.gated_rmsnorm(y, z, w, 1e-3, 3)
    y2 = y.copy()
    y2[:, 64:128] *= 10.0
    y2[:, 70] = -3.0
    out2 = oracle.gated_rmsnorm(y2, z, w, 1e-3, 3)
    np.testing.assert_array_equal(out2[:, :64], out[:, :64])
    np.testing.assert_array_equal(out2[:, 128:], out[:, 128:])
    for k in range(3):
        sl = slice(64 * k, 64 * (k + 1))
        np.testing.assert_allclose(oracle.gated_rmsnorm(y[:, sl], z[:, sl], w[sl], 1e-3),
                                   out[:, sl], rtol=1e-14)


def test_bf16_gate_decodes_exactly():
    """z given as bf16 bit patterns equals z given as the decoded fp32 values."""
    r = rng(13)
    zf = r.standard_normal((2, 64)).astype(np.float32)
    zb = (zf.view(np.uint32) >> 16).astype(np.uint16)
    zd = (zb.astype(np.uint32) << 16).view(np.float32)
    y = r.standard_normal((2, 64))
    w = np.ones(64, np.float32)
    np.testing.assert_array_equal(oracle.gated_rmsnorm(y, zb, w, 1e-5),
                                  oracle.gated_rmsnorm(y, zd, w, 1e-5))

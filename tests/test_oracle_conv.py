"""Pins of the oracle's convolution part of the Mamba boundary state (width-4 depthwise
causal convolution + SiLU over x, B, C; forward continued from the cached last three
input rows, reverse zero-padded inside the block; App. C, Sec. 2, Sec. 4), checked
against independent computations: numpy's correlate, closed forms, the flip identity
and cache continuation.  CPU only."""
import math

import numpy as np
import pytest

import bdlm_inputs as bi
import oracle


def silu(v):
    return v / (1.0 + np.exp(-v))


def setup(batch=2, H=2, N=16, G=1, L=7, nslots=3, seed=3, bf16=True):
    w = bi.Workload("t", batch, H, 64, N, G, L, 0, bf16, 1, seed)
    d = bi.block_inputs(w, 0)
    ch = H * 64 + 2 * G * N
    r = np.random.Generator(np.random.PCG64(seed + 100))
    wts = (r.standard_normal((ch, 4)) * 0.5).astype(np.float32)
    bias = (r.standard_normal(ch) * 0.1).astype(np.float32)
    cache = r.standard_normal((nslots, 3, ch))
    return w, d, wts, bias, cache


def channels(d):
    """The block's pre-convolution inputs as float64 [batch, L, channels]."""
    x, Bm, Cm = (oracle.decode(d[k]) for k in ("x", "B", "C"))
    b, L = x.shape[:2]
    return np.concatenate([x.reshape(b, L, -1), Bm.reshape(b, L, -1), Cm.reshape(b, L, -1)], -1)


def as_channels(o):
    b, L = o["x"].shape[:2]
    return np.concatenate([o["x"].reshape(b, L, -1), o["B"].reshape(b, L, -1),
                           o["C"].reshape(b, L, -1)], -1)


def test_silu_value():
    # silu(1) = 1 / (1 + e^-1); silu(0) = 0; silu(-v) = silu(v) - v
    assert math.isclose(silu(1.0), 0.7310585786300049, rel_tol=1e-15)
    assert silu(0.0) == 0.0
    assert math.isclose(silu(-2.5), silu(2.5) - 2.5, rel_tol=1e-14)


def test_identity_kernel_gives_silu_of_the_input():
    w, d, wts, bias, cache = setup()
    wts[:] = 0.0
    wts[:, 3] = 1.0
    bias[:] = 0.0
    f, r = oracle.conv(d, wts, bias, cache)
    u = channels(d)
    np.testing.assert_allclose(as_channels(f), silu(u), rtol=1e-15, atol=0)
    np.testing.assert_allclose(as_channels(r), silu(u), rtol=1e-15, atol=0)


@pytest.mark.parametrize("L", [1, 2, 5, 16])
def test_against_numpy_correlate(L):
    w, d, wts, bias, cache = setup(L=L, seed=10 + L)
    slots = [2, 0]
    f, r = oracle.conv(d, wts, bias, cache, slot_idx=slots)
    u = channels(d)
    F, R = as_channels(f), as_channels(r)
    for b in range(2):
        for c in range(u.shape[2]):
            seq = np.concatenate([cache[slots[b], :, c], u[b, :, c]])
            ref_f = silu(bias[c] + np.correlate(seq, wts[c].astype(np.float64), "valid"))
            seqr = np.concatenate([u[b, :, c], np.zeros(3)])
            ref_r = silu(bias[c] + np.correlate(seqr, wts[c, ::-1].astype(np.float64), "valid"))
            np.testing.assert_allclose(F[b, :, c], ref_f, rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(R[b, :, c], ref_r, rtol=1e-13, atol=1e-15)


def test_reverse_is_flip_of_forward_from_zero():
    w, d, wts, bias, cache = setup(L=9)
    _, r = oracle.conv(d, wts, bias, cache)
    flipped = {k: np.ascontiguousarray(d[k][:, ::-1]) for k in ("x", "B", "C")}
    f_of_flip, _ = oracle.conv(flipped, wts, bias, np.zeros_like(cache))
    for k in ("x", "B", "C"):
        np.testing.assert_array_equal(r[k], f_of_flip[k][:, ::-1])


def test_cache_continuation_equals_one_pass():
    """Forward output of a block from the cache holding the prefix's last three rows
    equals the one-pass convolution of prefix ++ block (bitwise: same operations)."""
    w, d, wts, bias, cache = setup(L=12, nslots=2)
    zero = np.zeros_like(cache)
    f_all, _ = oracle.conv(d, wts, bias, zero)
    first = {k: np.ascontiguousarray(d[k][:, :5]) for k in ("x", "B", "C")}
    rest = {k: np.ascontiguousarray(d[k][:, 5:]) for k in ("x", "B", "C")}
    c = zero.copy()
    oracle.conv(first, wts, bias, c, commit=True)
    f_rest, _ = oracle.conv(rest, wts, bias, c)
    for k in ("x", "B", "C"):
        np.testing.assert_array_equal(f_rest[k], f_all[k][:, 5:])


@pytest.mark.parametrize("L", [1, 2, 3, 6])
def test_commit_keeps_last_three_rows(L):
    w, d, wts, bias, cache = setup(L=L)
    slots = [1, 2]
    before = cache.copy()
    oracle.conv(d, wts, bias, cache, slot_idx=slots, commit=True)
    u = channels(d)
    for b, s in enumerate(slots):
        seq = np.concatenate([before[s], u[b]], axis=0)
        np.testing.assert_array_equal(cache[s], seq[-3:])
    np.testing.assert_array_equal(cache[0], before[0])          # unused slot untouched


def test_commit_rejects_repeated_slots():
    w, d, wts, bias, cache = setup()
    before = cache.copy()
    with pytest.raises(ValueError):
        oracle.conv(d, wts, bias, cache, slot_idx=[1, 1], commit=True)
    np.testing.assert_array_equal(cache, before)


def test_f64_inputs_equal_f32_storage_of_the_same_values():
    """The block step on already-decoded (float64) inputs equals the step on the same
    values stored as float32 (exactly representable), bitwise."""
    w = bi.Workload("t", 2, 3, 64, 16, 1, 8, 0, False, 1, 77)
    d = bi.block_inputs(w, 0)
    d64 = dict(d)
    for k in ("x", "dt", "B", "C"):
        d64[k] = d[k].astype(np.float64)
    h = bi.random_state(w, 2, 5).astype(np.float64)
    np.testing.assert_array_equal(oracle.block_step(d, h), oracle.block_step(d64, h))

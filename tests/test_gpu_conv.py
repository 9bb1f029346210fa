"""GPU parity of the block step and commit with the convolution part of the Mamba
boundary state (width-4 depthwise causal convolution + SiLU over x, B, C; forward
continued from the cached input rows, reverse zero-padded inside the block; App. C,
Sec. 2, Sec. 4) against the oracle composed from its pinned parts: oracle.conv, then
the oracle's block step on the convolved (float64) inputs -- forward part from the
cached state, reverse part from zero.

Bar: max relative error 2e-3 (tests/gpu_util.py); cached convolution rows bit-exact
(they are copies of the stored inputs); bookkeeping bit-exact.
"""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import DEV, REL_TOL, from_pool, pool_dev, rel_err, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-conv]", *a, flush=True)
    sys.stdout.flush()


def conv_params(w, seed):
    ch = w.nheads * 64 + 2 * w.ngroups * w.dstate
    r = np.random.Generator(np.random.PCG64(seed))
    cw = (r.standard_normal((ch, 4)) * 0.5).astype(np.float32)
    cb = (r.standard_normal(ch) * 0.1).astype(np.float32)
    return cw, cb


def oracle_step(d, cw, cb, cache, pool, slots):
    """y of the conv step and the forward branch's inputs (float64)."""
    f, r = oracle.conv(d, cw, cb, cache, slot_idx=slots)
    dt = oracle.decode(d["dt"])
    fin = dict(f, dt=dt, A=d["A"], D=d["D"], D_rev=d["D_rev"])
    rin = dict(r, dt=dt, A=d["A"], D=d["D"], D_rev=d["D_rev"])
    _, yf, _ = oracle.block_step(fin, pool, slot_idx=slots, parts=True)
    _, _, yr = oracle.block_step(rin, np.zeros_like(pool), slot_idx=slots, parts=True)
    return yf + yr, fin


@pytest.mark.parametrize("H,N,L,bf16,G", [(4, 16, 1, True, 1), (4, 64, 2, True, 1), (32, 128, 32, True, 1),
                                          (8, 128, 64, False, 1), (4, 32, 256, True, 1),
                                          (3, 64, 17, False, 1),
                                          # convolution inside the block kernel's staging
                                          # (bf16, L <= 32): ragged tiles, two groups
                                          (6, 32, 27, True, 1), (5, 128, 9, True, 1),
                                          (8, 64, 24, True, 2)])
def test_conv_step(H, N, L, bf16, G):
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 3, H, 64, N, G, L, 0, bf16, 1, 11000 + H + N + L)
    d = bi.block_inputs(w, 0)
    d["D_rev"] = (d["D"] * 0.5).astype(np.float32)
    cw, cb = conv_params(w, 11100 + L)
    ch = cw.shape[0]
    cache = np.random.Generator(np.random.PCG64(7)).standard_normal((4, 3, ch)).astype(np.float32)
    pool = bi.random_state(w, 4, 3, 0.5).astype(np.float64)
    slots = [3, 0, 3]
    y_ref, _ = oracle_step(d, cw, cb, cache.astype(np.float64), pool, slots)
    v = to_dev(d)
    say("conv step", dict(H=H, N=N, L=L, bf16=bf16, G=G))
    y = bd.conv_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                           torch.from_numpy(cw).to(DEV), torch.from_numpy(cb).to(DEV),
                           torch.from_numpy(cache).to(DEV), pool_dev(pool), slot_idx=slots)
    torch.cuda.synchronize()
    e = rel_err(y, y_ref)
    say("  rel err", e)
    assert e <= REL_TOL


def test_conv_step_full_size():
    """The convolution-state step at the size the bench times it (350M layer shape: batch
    16, 32 heads, dstate 128, 32-token bf16 blocks; the convolution inside the block
    kernel's staging, 512 workgroups per launch), every element against the oracle."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 16, 32, 64, 128, 1, 32, 0, True, 1, 11500)
    d = bi.block_inputs(w, 0)
    cw, cb = conv_params(w, 11501)
    ch = cw.shape[0]
    cache = np.random.Generator(np.random.PCG64(11502)).standard_normal((16, 3, ch)).astype(np.float32)
    pool = bi.random_state(w, 16, 3, 0.5).astype(np.float64)
    y_ref, _ = oracle_step(d, cw, cb, cache.astype(np.float64), pool, list(range(16)))
    v = to_dev(d)
    say("conv step, full size", w)
    y = bd.conv_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                           torch.from_numpy(cw).to(DEV), torch.from_numpy(cb).to(DEV),
                           torch.from_numpy(cache).to(DEV), pool_dev(pool))
    torch.cuda.synchronize()
    e = rel_err(y, y_ref)
    say("  rel err", e)
    assert e <= REL_TOL


@pytest.mark.parametrize("L,want_y", [(32, True), (2, True), (64, False)])
def test_conv_commit(L, want_y):
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, 8, 64, 128, 1, L, 0, True, 1, 11200 + L)
    d = bi.commit_inputs(w)
    cw, cb = conv_params(w, 11300 + L)
    ch = cw.shape[0]
    cache = np.random.Generator(np.random.PCG64(9)).standard_normal((3, 3, ch)).astype(np.float32)
    pool = bi.random_state(w, 3, 4, 0.5).astype(np.float64)
    slots = [2, 0]
    y_ref, fin = oracle_step(d, cw, cb, cache.astype(np.float64), pool, slots)
    *_, s_ref = oracle.block_step(fin, pool, slot_idx=slots, parts=True, final_state=True)
    cache_ref = cache.astype(np.float64)
    oracle.conv(d, cw, cb, cache_ref, slot_idx=slots, commit=True)
    nb = np.array([5, 9, 5], np.int64)
    nc = nb * L
    v = to_dev(d)
    h = pool_dev(pool)
    cp = torch.from_numpy(cache).to(DEV)
    out = bd.conv_commit_boundary(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                                  torch.from_numpy(cw).to(DEV), torch.from_numpy(cb).to(DEV), cp, h,
                                  nc, nb, 5, slot_idx=slots, y_clean=True if want_y else None)
    torch.cuda.synchronize()
    assert nb.tolist() == [6, 9, 6] and nc.tolist() == [6 * L, 9 * L, 6 * L]
    got = from_pool(h)
    assert rel_err(got[slots], s_ref) <= REL_TOL
    np.testing.assert_array_equal(got[1], pool[1].astype(np.float32))
    np.testing.assert_array_equal(cp.cpu().numpy(), cache_ref.astype(np.float32))
    if want_y:
        assert rel_err(out, y_ref) <= REL_TOL


def test_conv_commit_full_size():
    """The convolution-state commit at the size the bench times it (350M layer shape:
    batch 16, 32 heads, dstate 128, a 32-token bf16 block, identity slots): the new
    states, the kept convolution rows and the clean-block outputs against the oracle."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 16, 32, 64, 128, 1, 32, 0, True, 1, 11600)
    d = bi.commit_inputs(w)
    cw, cb = conv_params(w, 11601)
    ch = cw.shape[0]
    cache = np.random.Generator(np.random.PCG64(11602)).standard_normal((16, 3, ch)).astype(np.float32)
    pool = bi.random_state(w, 16, 4, 0.5).astype(np.float64)
    slots = list(range(16))
    y_ref, fin = oracle_step(d, cw, cb, cache.astype(np.float64), pool, slots)
    *_, s_ref = oracle.block_step(fin, pool, slot_idx=slots, parts=True, final_state=True)
    cache_ref = cache.astype(np.float64)
    oracle.conv(d, cw, cb, cache_ref, slot_idx=slots, commit=True)
    nb = np.zeros(16, np.int64)
    nc = np.zeros(16, np.int64)
    v = to_dev(d)
    h = pool_dev(pool)
    cp = torch.from_numpy(cache).to(DEV)
    say("conv commit, full size", w)
    out = bd.conv_commit_boundary(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                                  torch.from_numpy(cw).to(DEV), torch.from_numpy(cb).to(DEV), cp, h,
                                  nc, nb, 0, y_clean=True)
    torch.cuda.synchronize()
    assert nb.tolist() == [1] * 16 and nc.tolist() == [32] * 16
    e = (rel_err(from_pool(h), s_ref), rel_err(out, y_ref))
    say("  state, clean y rel err", e)
    assert max(e) <= REL_TOL
    np.testing.assert_array_equal(cp.cpu().numpy(), cache_ref.astype(np.float32))


def test_conv_commits_then_step_equal_oracle_history():
    """Three conv commits, then a conv step: the cached convolution rows and SSM states
    carry the history exactly as the oracle's composition does."""
    import paper_2607_02805_amd as bd
    L, K = 32, 3
    w = bi.Workload("t", 2, 4, 64, 64, 1, L, K * L, True, 1, 11400)
    pre = bi.prefix_inputs(w)
    blk = bi.block_inputs(w, 0)
    cw, cb = conv_params(w, 11500)
    ch = cw.shape[0]
    cache_ref = np.zeros((2, 3, ch))
    pool_ref = np.zeros((2, 4, 64, 64))
    cache = bd.Cache(2, 4, 64, ngroups=1)
    cwd, cbd = torch.from_numpy(cw).to(DEV), torch.from_numpy(cb).to(DEV)
    for k in range(K):
        part = bi.slice_tokens(pre, k * L, (k + 1) * L)
        _, fin = oracle_step(part, cw, cb, cache_ref, pool_ref, None)
        *_, pool_ref = oracle.block_step(fin, pool_ref, parts=True, final_state=True)
        oracle.conv(part, cw, cb, cache_ref, commit=True)
        v = to_dev(part)
        cache.conv_commit(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], cwd, cbd, k)
    y_ref, _ = oracle_step(blk, cw, cb, cache_ref, pool_ref, None)
    v = to_dev(blk)
    y = cache.conv_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], cwd, cbd)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(cache.conv.cpu().numpy(), cache_ref.astype(np.float32))
    assert rel_err(cache.states(), pool_ref) <= REL_TOL
    assert rel_err(y, y_ref) <= REL_TOL
    assert cache.n_blocks.tolist() == [K, K]

"""GPU parity of slot-mapped calls whose slot table spans several launches (more than
256 batch rows; the per-sequence cache of Sec. 4 remapped over a larger pool): the
block step and commit at batch 1024 over a 2048-slot pool, and the other slot-mapped
entry points (long blocks, separate reverse inputs, the convolution state, the
prefill) at batch 300.

Bar: max relative error 2e-3 (tests/gpu_util.py); bookkeeping bit-exact; slots no
row maps to are bit-identical before and after.
"""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import DEV, REL_TOL, commit, from_pool, pool_dev, rel_err, step, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-slots]", *a, flush=True)
    sys.stdout.flush()


def wl(batch, H, N, L, bf16=True, seed=15000):
    return bi.Workload("t", batch, H, 64, N, 1, L, 0, bf16, 1, seed)


def test_step_and_commit_batch_1024_over_2048_slots():
    """Batch 1024 (four launches of 256 rows) over a 2048-slot pool: a step with rows
    sharing slots, then a commit of distinct slots with the clean-block outputs."""
    import paper_2607_02805_amd as bd
    B, S = 1024, 2048
    w = wl(B, 8, 64, 32, seed=15100)
    rng = np.random.default_rng(15101)
    pool = bi.random_state(w, S, 15102, 0.5)
    hp = pool_dev(pool)
    # step: rows drawn with repeats from the whole pool
    sl = rng.integers(0, S, size=B).astype(np.int32)
    d = bi.block_inputs(w, 0)
    say("step batch 1024 over 2048 slots")
    y = step(to_dev(d), hp, slot_idx=sl)
    torch.cuda.synchronize()
    e = rel_err(y, oracle.block_step(d, pool.astype(np.float64), slot_idx=sl))
    say("  rel err", e)
    assert e <= REL_TOL
    # commit: distinct slots, a random subset of the pool
    sc = rng.permutation(S)[:B].astype(np.int32)
    c = bi.commit_inputs(w)
    nb = rng.integers(3, 6, size=S).astype(np.int64)
    nb[sc] = 4
    nc = nb * 32
    onb, onc = nb.copy(), nc.copy()
    say("commit batch 1024 over 2048 slots")
    yc = commit(to_dev(c), hp, nc, nb, expected=4, slot_idx=sc, y_clean=True)
    torch.cuda.synchronize()
    ref = pool.astype(np.float64)
    rc, ycr = oracle.commit(c, ref, onc, onb, slot_idx=sc, expected_block_index=4)
    assert rc == 0
    got = from_pool(hp)
    eh, ey = rel_err(got[sc], ref[sc]), rel_err(yc, ycr)
    say("  state rel err", eh, "y_clean rel err", ey)
    assert eh <= REL_TOL and ey <= REL_TOL
    assert nb.tolist() == onb.tolist() and nc.tolist() == onc.tolist()
    untouched = np.setdiff1d(np.arange(S), sc)
    np.testing.assert_array_equal(got[untouched], pool[untouched])


def test_long_block_and_separate_inputs_over_256_rows():
    """Batch 300 slot-mapped: an 80-token bf16 block (the masked long-block kernel, one
    launch per 256 rows) step and commit, and a separate-reverse-input step of 32 tokens
    (one fused launch per 256 rows)."""
    import paper_2607_02805_amd as bd
    B, S = 300, 400
    rng = np.random.default_rng(15200)
    w = wl(B, 4, 32, 80, seed=15201)
    pool = bi.random_state(w, S, 15202, 0.5)
    sl = rng.permutation(S)[:B].astype(np.int32)
    d = bi.block_inputs(w, 0)
    hp = pool_dev(pool)
    say("long block step, batch 300")
    y = step(to_dev(d), hp, slot_idx=sl)
    torch.cuda.synchronize()
    assert rel_err(y, oracle.block_step(d, pool.astype(np.float64), slot_idx=sl)) <= REL_TOL
    c = bi.commit_inputs(w)
    nc, nb = np.zeros(S, np.int64), np.zeros(S, np.int64)
    say("long block commit, batch 300")
    commit(to_dev(c), hp, nc, nb, expected=0, slot_idx=sl)
    torch.cuda.synchronize()
    ref = pool.astype(np.float64)
    onc, onb = np.zeros(S, np.int64), np.zeros(S, np.int64)
    assert oracle.commit(c, ref, onc, onb, slot_idx=sl, expected_block_index=0)[0] == 0
    assert rel_err(from_pool(hp)[sl], ref[sl]) <= REL_TOL
    assert nb.tolist() == onb.tolist() and nc.tolist() == onc.tolist()

    w2 = wl(B, 4, 64, 32, seed=15203)
    f = bi.block_inputs(w2, 0)
    r = bi.block_inputs(w2, 1)
    r["A"] = (r["A"] * 0.5).astype(np.float32)
    pool2 = bi.random_state(w2, S, 15204, 0.5)
    fv, rv = to_dev(f), to_dev(r)
    say("separate-input step, batch 300")
    y2 = bd.scan_block_step_sep((fv["x"], fv["dt"], fv["A"], fv["B"], fv["C"], fv["D"]),
                                (rv["x"], rv["dt"], rv["A"], rv["B"], rv["C"], rv["D_rev"]),
                                pool_dev(pool2), slot_idx=sl)
    torch.cuda.synchronize()
    _, yf, _ = oracle.block_step(f, pool2.astype(np.float64), slot_idx=sl, parts=True)
    _, _, yr = oracle.block_step(r, np.zeros((S, 4, 64, 64)), slot_idx=sl, parts=True)
    assert rel_err(y2, yf + yr) <= REL_TOL


def test_prefill_over_256_rows():
    """A slot-mapped prefill of batch 300 (two launches' worth of rows, one workspace
    reused in order) over a 500-slot pool: states and forward outputs."""
    import paper_2607_02805_amd as bd
    B, S, T = 300, 500, 320
    w = bi.Workload("t", B, 2, 64, 32, 1, 32, T, True, 1, 15300)
    pre = bi.prefix_inputs(w)
    s0 = bi.random_state(w, S, 15301, 0.5)
    sl = np.random.default_rng(15302).permutation(S)[:B].astype(np.int32)
    cache = bd.Cache(S, 2, 32)
    cache.h.copy_(pool_dev(s0))
    v = to_dev(pre)
    say("prefill batch 300")
    yf = cache.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], expected_block_index=0,
                       blocks_in_prefix=T // 32, slot_idx=sl, y_fwd=True)
    torch.cuda.synchronize()
    s_ref, y_ref = oracle.scan_forward(pre, s0[sl].astype(np.float64), want_y=True)
    got = from_pool(cache.h)
    assert rel_err(got[sl], s_ref) <= REL_TOL
    assert rel_err(yf, y_ref) <= REL_TOL
    other = np.setdiff1d(np.arange(S), sl)
    np.testing.assert_array_equal(got[other], s0[other])
    assert cache.n_blocks[sl].tolist() == [T // 32] * B
    assert cache.n_committed[other].tolist() == [0] * len(other)


@pytest.mark.parametrize("L,bf16", [(32, True), (16, False)])
def test_conv_commit_over_256_rows(L, bf16):
    """Convolution-state commit of batch 300 over a 320-slot pool: the fused staging path
    (bf16, 32 tokens) and the convolution kernel with its workspace (fp32)."""
    import paper_2607_02805_amd as bd
    B, S = 300, 320
    w = bi.Workload("t", B, 2, 64, 32, 1, L, 0, bf16, 1, 15400 + L)
    d = bi.commit_inputs(w)
    ch = 2 * 64 + 2 * 32
    r = np.random.Generator(np.random.PCG64(15401))
    cw = (r.standard_normal((ch, 4)) * 0.5).astype(np.float32)
    cb = (r.standard_normal(ch) * 0.1).astype(np.float32)
    cache = r.standard_normal((S, 3, ch)).astype(np.float32)
    pool = bi.random_state(w, S, 15402, 0.5).astype(np.float64)
    sl = np.random.default_rng(15403).permutation(S)[:B].astype(np.int32)
    f, _ = oracle.conv(d, cw, cb, cache.astype(np.float64), slot_idx=sl)
    fin = dict(f, dt=oracle.decode(d["dt"]), A=d["A"], D=d["D"], D_rev=d["D_rev"])
    *_, s_ref = oracle.block_step(fin, pool, slot_idx=sl, parts=True, final_state=True)
    cache_ref = cache.astype(np.float64)
    oracle.conv(d, cw, cb, cache_ref, slot_idx=sl, commit=True)
    nc, nb = np.zeros(S, np.int64), np.zeros(S, np.int64)
    v = to_dev(d)
    h = pool_dev(pool)
    cp = torch.from_numpy(cache).to(DEV)
    say("conv commit batch 300", dict(L=L, bf16=bf16))
    bd.conv_commit_boundary(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                            torch.from_numpy(cw).to(DEV), torch.from_numpy(cb).to(DEV), cp, h,
                            nc, nb, 0, slot_idx=sl)
    torch.cuda.synchronize()
    got = from_pool(h)
    assert rel_err(got[sl], s_ref) <= REL_TOL
    np.testing.assert_array_equal(cp.cpu().numpy(), cache_ref.astype(np.float32))
    assert nb[sl].tolist() == [1] * B

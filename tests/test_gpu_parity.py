"""GPU parity: the HIP path, called through the C ABI, against the fp64 oracle on the
same seeded bytes.  Bar: max relative error 2e-3 on y and on committed states (the
error measure is in tests/gpu_util.py); bookkeeping (tokens and blocks committed
per slot) bit-exact; outputs deterministic bit for bit.
"""
import dataclasses
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import (DEV, REL_TOL, commit, from_pool, pool_dev, rel_err, step,
                            to_dev, to_pool)

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-parity]", *a, flush=True)
    sys.stdout.flush()


def wl(batch, H, N, L, G=1, bf16=True, seed=7000):
    return bi.Workload("t", batch, H, 64, N, G, L, 0, bf16, 1, seed)


def check_step(w: bi.Workload, nslots=None, slot_idx=None, seed_state=1, scale=1.0, step_no=0):
    d = bi.block_inputs(w, step_no)
    nslots = w.batch if nslots is None else nslots
    pool = bi.random_state(w, nslots, seed_state, scale)
    say("step", w, "slots", slot_idx)
    y = step(to_dev(d), pool_dev(pool), slot_idx=slot_idx)
    torch.cuda.synchronize()
    ref = oracle.block_step(d, pool.astype(np.float64), slot_idx=slot_idx)
    e = rel_err(y, ref)
    say("  rel err", e)
    assert e <= REL_TOL
    return y, ref


# ------------------------------------------------------------------ workloads
def test_tiny_fp32_workload_with_oracle_prefix():
    """Batch 1, 4 heads x 64, N = 16, L = 16, fp32; the cached state is the oracle's
    forward scan over a seeded 1024-token prefix."""
    w = bi.WORKLOADS[0]
    pre = bi.prefix_inputs(w)
    s = oracle.scan_forward(pre).astype(np.float32)          # [1, H, P, N]
    d = bi.block_inputs(w, 0)
    say("tiny fp32", w)
    y = step(to_dev(d), pool_dev(s))
    ref = oracle.block_step(d, s.astype(np.float64))
    assert rel_err(y, ref) <= REL_TOL
    # commit of the clean block
    c = bi.commit_inputs(w)
    hp = pool_dev(s)
    nc, nb = np.array([1024], np.int64), np.array([64], np.int64)
    yc = commit(to_dev(c), hp, nc, nb, expected=64, y_clean=True)
    torch.cuda.synchronize()
    hr = s.astype(np.float64)
    onc, onb = np.array([1024], np.int64), np.array([64], np.int64)
    rc, ycr = oracle.commit(c, hr, onc, onb, expected_block_index=64)
    assert rc == 0
    assert rel_err(from_pool(hp), hr) <= REL_TOL
    assert rel_err(yc, ycr) <= REL_TOL
    assert nc.tolist() == onc.tolist() == [1040] and nb.tolist() == onb.tolist() == [65]


@pytest.mark.parametrize("k", [1, 2, 3])
def test_layer_workloads_full_size(k):
    """87M layer (B 8, 24 heads, N 64, L 32) and 350M layer (B 16, 32 heads, N 128,
    L 32), every element against the oracle, plus the commit."""
    w = bi.WORKLOADS[k]
    check_step(w, step_no=k)
    c = bi.commit_inputs(w)
    pool = bi.random_state(w, w.batch, 5)
    hp = pool_dev(pool)
    k0 = 4096 // w.block_len
    nc, nb = np.full(w.batch, 4096, np.int64), np.full(w.batch, k0, np.int64)
    onc, onb = nc.copy(), nb.copy()
    say("commit", w)
    yc = commit(to_dev(c), hp, nc, nb, expected=k0, y_clean=True)
    torch.cuda.synchronize()
    hr = pool.astype(np.float64)
    rc, ycr = oracle.commit(c, hr, onc, onb, expected_block_index=k0)
    assert rc == 0
    eh, ey = rel_err(from_pool(hp), hr), rel_err(yc, ycr)
    say("  state rel err", eh, "y_clean rel err", ey)
    assert eh <= REL_TOL and ey <= REL_TOL
    assert nc.tolist() == onc.tolist() and nb.tolist() == onb.tolist()


@pytest.mark.parametrize("L", [16, 64])
def test_350m_layer_other_block_lengths(L):
    w = bi.WORKLOADS[3].with_block_len(L)
    check_step(w)


def test_350m_layer_batch_128():
    """The 350M layer shape at batch 128: 4,096 workgroups over the remapped grid (the
    largest launch the bench's batch sweep times), every element against the oracle."""
    check_step(dataclasses.replace(bi.WORKLOADS[3], batch=128))


# ------------------------------------------------------------- shapes and edges
@pytest.mark.parametrize("N", [16, 32, 64, 128])
@pytest.mark.parametrize("L", [1, 5, 16, 17, 31, 33, 47, 64])
def test_ragged_block_lengths(N, L):
    check_step(wl(3, 5, N, L, seed=7100 + L))


@pytest.mark.parametrize("N,L", [(16, 16), (64, 20), (128, 33)])
def test_fp32_storage(N, L):
    check_step(wl(2, 3, N, L, bf16=False, seed=7200 + L))


def test_groups():
    check_step(wl(4, 8, 64, 24, G=4, seed=7300))
    check_step(wl(2, 6, 128, 32, G=2, seed=7301))


def test_slot_mapping_with_repeats():
    w = wl(5, 8, 64, 32, seed=7400)
    check_step(w, nslots=9, slot_idx=[8, 0, 3, 3, 7])


def test_slot_mapping_at_max_rows():
    """A slot map over the largest batch it accepts, rows drawn with repeats from a
    larger pool."""
    w = wl(256, 4, 16, 16, seed=7410)
    slots = np.random.default_rng(7411).integers(0, 300, size=256).tolist()
    check_step(w, nslots=300, slot_idx=slots)


def test_strided_views():
    """x, dt, B, C as slices of one fused projection output [B, L, width]."""
    w = wl(3, 4, 64, 24, seed=7500)
    d = bi.block_inputs(w, 0)
    Bsz, L, H, P, N = 3, 24, 4, 64, 64
    width = H * P + 2 * N + H + 12                      # x | B | C | dt | pad (16-byte rows)
    fused = np.zeros((Bsz, L, width), np.uint16)
    fused[:, :, :H * P] = d["x"].reshape(Bsz, L, H * P)
    fused[:, :, H * P:H * P + N] = d["B"][:, :, 0]
    fused[:, :, H * P + N:H * P + 2 * N] = d["C"][:, :, 0]
    fused[:, :, H * P + 2 * N:H * P + 2 * N + H] = d["dt"]
    f = to_dev({"f": fused})["f"]
    dv = to_dev({k: d[k] for k in ("A", "D", "D_rev")})
    dv["x"] = f[:, :, :H * P].unflatten(2, (H, P))
    dv["B"] = f[:, :, H * P:H * P + N].unsqueeze(2)
    dv["C"] = f[:, :, H * P + N:H * P + 2 * N].unsqueeze(2)
    dv["dt"] = f[:, :, H * P + 2 * N:H * P + 2 * N + H]
    assert not dv["x"].is_contiguous()
    pool = bi.random_state(w, Bsz, 3)
    y = step(dv, pool_dev(pool))
    torch.cuda.synchronize()
    assert rel_err(y, oracle.block_step(d, pool.astype(np.float64))) <= REL_TOL


def test_empty_inputs():
    w = wl(2, 4, 64, 0, seed=7600)
    d = to_dev(bi.block_inputs(w, 0))
    pool = torch.zeros((2, 4, 16, 64, 4), device=DEV)
    y = step(d, pool)
    assert tuple(y.shape) == (2, 0, 4, 64)
    w0 = wl(0, 4, 64, 16, seed=7601)
    d0 = to_dev(bi.block_inputs(w0, 0))
    y0 = step(d0, pool)
    assert tuple(y0.shape) == (0, 16, 4, 64)
    nc, nb = np.zeros(2, np.int64), np.zeros(2, np.int64)
    keep = pool.clone()
    commit(d, pool, nc, nb, expected=0)
    torch.cuda.synchronize()
    assert torch.equal(pool, keep) and nc.tolist() == [0, 0] and nb.tolist() == [1, 1]


def test_large_state_magnitudes():
    """States far larger than the block's own contribution (long, slowly decaying prefix)."""
    check_step(wl(2, 4, 128, 32, seed=7700), scale=300.0)


# ------------------------------------------------------------ cache behaviour
def test_cache_equivalence_4k_prefix_by_commits():
    """128 commits of L = 32 over a seeded 4096-token prefix (350M layer shape, 2 rows),
    then a step, against one oracle pass over the prefix."""
    w = bi.Workload("replay", 2, 32, 64, 128, 1, 32, 4096, True, 1, 7800)
    pre = bi.prefix_inputs(w)
    pool = torch.zeros((2, 32, 32, 64, 4), device=DEV)
    nc, nb = np.zeros(2, np.int64), np.zeros(2, np.int64)
    say("4K replay: 128 commits")
    for k in range(128):
        blk = to_dev(bi.slice_tokens(pre, 32 * k, 32 * (k + 1)))
        commit(blk, pool, nc, nb, expected=k)
    d = bi.block_inputs(w, 0)
    y = step(to_dev(d), pool)
    torch.cuda.synchronize()
    assert nc.tolist() == [4096, 4096] and nb.tolist() == [128, 128]
    s_ref = oracle.scan_forward(pre)
    es = rel_err(from_pool(pool), s_ref)
    ey = rel_err(y, oracle.block_step(d, s_ref))
    say("  state rel err", es, "step rel err", ey)
    assert es <= REL_TOL and ey <= REL_TOL


def test_step_never_writes_cache_and_is_deterministic():
    w = bi.WORKLOADS[2]
    d = to_dev(bi.block_inputs(w, 1))
    pool = pool_dev(bi.random_state(w, w.batch, 9))
    keep = pool.clone()
    y1 = step(d, pool)
    y2 = step(d, pool)
    torch.cuda.synchronize()
    assert torch.equal(pool, keep)
    assert torch.equal(y1, y2)


def test_output_fully_written_and_guard_bands_intact():
    w = wl(3, 8, 128, 29, seed=7900)
    d = bi.block_inputs(w, 0)
    pool = bi.random_state(w, 3, 4)
    n = 3 * 29 * 8 * 64
    buf = torch.full((n + 2048,), float("nan"), device=DEV)
    buf[:1024] = 7.0
    buf[-1024:] = 7.0
    y = buf[1024:1024 + n].view(3, 29, 8, 64)
    step(to_dev(d), pool_dev(pool), y=y)
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    assert (buf[:1024] == 7.0).all() and (buf[-1024:] == 7.0).all()
    assert rel_err(y, oracle.block_step(d, pool.astype(np.float64))) <= REL_TOL


def test_commit_with_slots_and_reset():
    import paper_2607_02805_amd as bd
    w = wl(3, 4, 64, 32, seed=8000)
    c = bi.commit_inputs(w)
    pool_np = bi.random_state(w, 5, 6)
    cache = bd.Cache(5, 4, 64)
    cache.h.copy_(pool_dev(pool_np))
    cache.n_blocks[:] = [2, 7, 2, 1, 2]
    cache.n_committed[:] = cache.n_blocks * 32
    slots = [4, 0, 2]
    dv = to_dev(c)
    cache.commit(dv["x"], dv["dt"], dv["A"], dv["B"], dv["C"], dv["D"], dv["D_rev"],
                 expected_block_index=2, slot_idx=slots)
    torch.cuda.synchronize()
    ref = pool_np.astype(np.float64)
    onb = np.array([2, 7, 2, 1, 2], np.int64)
    onc = onb * 32
    assert oracle.commit(c, ref, onc, onb, slot_idx=slots, expected_block_index=2)[0] == 0
    assert rel_err(from_pool(cache.h), ref) <= REL_TOL
    assert cache.n_blocks.tolist() == onb.tolist() and cache.n_committed.tolist() == onc.tolist()
    # untouched slots are bit-identical
    assert torch.equal(cache.h[[1, 3]], pool_dev(pool_np[[1, 3]]))
    # a wrong block index is refused and changes nothing
    before = cache.h.clone()
    with pytest.raises(bd.BdlmError) as ei:
        cache.commit(dv["x"], dv["dt"], dv["A"], dv["B"], dv["C"], dv["D"], dv["D_rev"],
                     expected_block_index=2, slot_idx=slots)
    assert ei.value.code == bd.E_OFFSET
    torch.cuda.synchronize()
    assert torch.equal(cache.h, before)
    # reset two slots
    cache.reset([0, 4])
    torch.cuda.synchronize()
    assert (cache.h[[0, 4]] == 0).all() and torch.equal(cache.h[[1, 2, 3]], before[[1, 2, 3]])
    assert cache.n_blocks.tolist() == [0, 7, 3, 1, 0]


def test_checkpoint_resume_bitwise():
    import paper_2607_02805_amd as bd
    w = wl(2, 4, 64, 32, seed=8100, )
    pre = bi.prefix_inputs(w, 32 * 6)
    a = bd.Cache(2, 4, 64)
    for k in range(3):
        dv = to_dev(bi.slice_tokens(pre, 32 * k, 32 * (k + 1)))
        a.commit(dv["x"], dv["dt"], dv["A"], dv["B"], dv["C"], dv["D"], dv["D_rev"], k)
    sd = a.state_dict()
    b = bd.Cache(2, 4, 64)
    b.load_state_dict(sd)
    for k in range(3, 6):
        dv = to_dev(bi.slice_tokens(pre, 32 * k, 32 * (k + 1)))
        for c in (a, b):
            c.commit(dv["x"], dv["dt"], dv["A"], dv["B"], dv["C"], dv["D"], dv["D_rev"], k)
    torch.cuda.synchronize()
    assert torch.equal(a.h, b.h) and a.n_blocks.tolist() == b.n_blocks.tolist() == [6, 6]


def test_side_stream():
    w = wl(4, 8, 128, 32, seed=8200)
    d = bi.block_inputs(w, 0)
    pool = bi.random_state(w, 4, 8)
    s = torch.cuda.Stream()
    dv = to_dev(d)
    hp = pool_dev(pool)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        y = step(dv, hp, stream=s)
    s.synchronize()
    assert rel_err(y, oracle.block_step(d, pool.astype(np.float64))) <= REL_TOL


def test_state_pack_unpack_match_documented_layout():
    import paper_2607_02805_amd as bd
    for N in (16, 32, 64, 128):
        rm = np.random.default_rng(N).standard_normal((3, 5, 64, N)).astype(np.float32)
        t = torch.from_numpy(rm).to(DEV)
        pool = bd.state_pack(t)
        back = bd.state_unpack(pool)
        torch.cuda.synchronize()
        assert tuple(pool.shape) == (3, 5, N // 4, 64, 4)
        assert np.array_equal(pool.cpu().numpy(), to_pool(rm))
        assert torch.equal(back, t)
    with pytest.raises(bd.BdlmError):
        bd.state_pack(t, pool=t.view(-1)[: t.numel()].view(3, 5, 32, 64, 4))   # overlap

"""GPU parity of the sequence entry points against the fp64 oracle:

* bdlm_scan_full_window -- forward over the whole window from zero plus reverse over the
  whole window from zero (the full-sequence contrast);
* bdlm_prefill -- a clean prefix summarised into the cached states, which must equal
  committing it block by block.

Both cut the sequence into segments of >= 256 tokens (one workgroup per row, head and
segment; the states entering each segment come from a combine pass over the segments'
local states), so cases span one segment, several segments and a ragged last segment.

Bar: max relative error 2e-3 (tests/gpu_util.py); bookkeeping bit-exact.
"""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import (DEV, REL_TOL, edge_cover, from_pool, host_slice, pick,
                            pool_dev, rel_err, to_dev, to_host)

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-chain]", *a, flush=True)
    sys.stdout.flush()


def wl(batch, H, N, W, G=1, bf16=True, seed=9000):
    return bi.Workload("t", batch, H, 64, N, G, W, 0, bf16, 1, seed)


def full_window(d):
    import paper_2607_02805_amd as bd
    v = to_dev(d)
    return bd.scan_full_window(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"])


@pytest.mark.parametrize("N", [16, 32, 64, 128])
@pytest.mark.parametrize("W", [1, 63, 64, 65, 200])
def test_full_window_small(N, W):
    w = wl(2, 3, N, W, seed=9100 + W)
    d = bi.block_inputs(w, 0)
    d["D_rev"] = (d["D"] * 0.5).astype(np.float32)      # distinct skips per direction
    say("full window", w)
    y = full_window(d)
    torch.cuda.synchronize()
    e = rel_err(y, oracle.full_window(d))
    say("  rel err", e)
    assert e <= REL_TOL


@pytest.mark.parametrize("N,W", [(16, 130), (128, 300)])
def test_full_window_fp32_storage(N, W):
    w = wl(2, 2, N, W, bf16=False, seed=9200 + W)
    d = bi.block_inputs(w, 0)
    y = full_window(d)
    torch.cuda.synchronize()
    assert rel_err(y, oracle.full_window(d)) <= REL_TOL


@pytest.mark.parametrize("N", [16, 32, 64, 128])
@pytest.mark.parametrize("bf16", [True, False])
def test_full_window_segments(N, bf16):
    """1 row x 2 heads over 1000 tokens: four segments of 256, the last one ragged."""
    import paper_2607_02805_amd as bd
    assert bd.full_window_workspace_bytes(1, 2, N, 1000) > 0
    w = wl(1, 2, N, 1000, bf16=bf16, seed=9250 + N)
    d = bi.block_inputs(w, 0)
    d["D_rev"] = (d["D"] * 0.5).astype(np.float32)
    say("full window segments", w)
    y = full_window(d)
    torch.cuda.synchronize()
    e = rel_err(y, oracle.full_window(d))
    say("  rel err", e)
    assert e <= REL_TOL


def test_full_window_caller_workspace_and_determinism():
    import paper_2607_02805_amd as bd
    w = wl(2, 3, 64, 1500, seed=9270)
    d = bi.block_inputs(w, 0)
    v = to_dev(d)
    need = bd.full_window_workspace_bytes(2, 3, 64, 1500)
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    args = (v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"])
    y1 = bd.scan_full_window(*args, workspace=ws)
    y2 = bd.scan_full_window(*args)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)                       # bitwise, run to run
    assert rel_err(y1, oracle.full_window(d)) <= REL_TOL
    with pytest.raises(bd.BdlmError) as ei:
        bd.scan_full_window(*args, workspace=ws[:need - 256])
    assert ei.value.code == bd.E_WORKSPACE


@pytest.mark.parametrize("B,H,N,W", [(2, 256, 16, 64), (8, 256, 128, 64), (4, 64, 64, 3000)])
def test_full_window_many_workgroups(B, H, N, W):
    """More workgroups than CUs, so CUs run several in turn: the result must not depend
    on that (bitwise equal across calls, y pre-filled differently) and must match the
    oracle on sampled heads."""
    import paper_2607_02805_amd as bd
    w = wl(B, H, N, W, seed=9280 + H + W)
    d = bi.block_inputs(w, 0)
    v = to_dev(d)
    args = (v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"])
    y1 = torch.zeros((B, W, H, 64), device=DEV)
    y2 = torch.full((B, W, H, 64), float("nan"), device=DEV)
    bd.scan_full_window(*args, y=y1)
    bd.scan_full_window(*args, y=y2)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    for b, h in ((0, 0), (B - 1, H - 1), (B // 2, H // 3)):
        sub = {"x": d["x"][b:b + 1, :, h:h + 1], "dt": d["dt"][b:b + 1, :, h:h + 1],
               "B": d["B"][b:b + 1], "C": d["C"][b:b + 1],
               "A": d["A"][h:h + 1], "D": d["D"][h:h + 1], "D_rev": d["D_rev"][h:h + 1]}
        e = rel_err(y1[b:b + 1, :, h:h + 1], oracle.full_window(sub))
        say("  (b, h) =", (b, h), "rel err", e)
        assert e <= REL_TOL


def test_full_window_groups_and_long():
    w = wl(2, 4, 64, 2000, G=2, seed=9300)
    d = bi.block_inputs(w, 0)
    y = full_window(d)
    torch.cuda.synchronize()
    assert rel_err(y, oracle.full_window(d)) <= REL_TOL


def test_full_window_contrast_shape_sampled():
    """The contrast workload: 350M layer shape, batch 4, 65,536-token window (inputs drawn
    on the GPU).  Every output of every head of batch rows 0 and 3 and of every row of
    heads 0 and 31 (68 of the 128 (row, head) pairs) against the oracle run on just those
    rows and heads."""
    import paper_2607_02805_amd as bd
    w = bi.WORKLOADS[4]
    v = bi.tokens_device(w, w.block_len, w.base_seed + 10)
    hp = {k: torch.from_numpy(a).to(DEV) for k, a in bi.head_params(w).items()}
    say("contrast shape", w)
    y = bd.scan_full_window(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], hp["D_rev"])
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    for rows, heads in edge_cover(w.batch, w.nheads):
        ref = oracle.full_window(host_slice(v, rows, heads, hp))
        e = rel_err(pick(y, rows, heads), ref)
        say("  rows", rows, "heads", heads, "rel err", e)
        assert e <= REL_TOL
        del ref


def test_full_window_equals_block_step_from_zero():
    """With a window that fits one block, the two kernels compute the same thing."""
    import paper_2607_02805_amd as bd
    w = wl(3, 4, 128, 48, seed=9400)
    d = bi.block_inputs(w, 0)
    v = to_dev(d)
    pool = torch.zeros((3, 4, 32, 64, 4), device=DEV)
    y1 = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], pool)
    y2 = full_window(d)
    torch.cuda.synchronize()
    ref = oracle.full_window(d)
    assert rel_err(y1, ref) <= REL_TOL and rel_err(y2, ref) <= REL_TOL


# ------------------------------------------------------------------------ prefill
@pytest.mark.parametrize("N,T", [(16, 100), (64, 1000), (128, 4096)])
def test_prefill_matches_oracle_prefix_scan(N, T):
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 3, 4, 64, N, 1, 32, T, True, 1, 9500 + T)
    pre = bi.prefix_inputs(w)
    s0 = bi.random_state(w, 5, 3, 0.5)
    slots = [4, 0, 2]
    cache = bd.Cache(5, 4, N)
    cache.h.copy_(pool_dev(s0))
    cache.n_blocks[:] = [1, 2, 1, 9, 1]
    cache.n_committed[:] = cache.n_blocks * 32
    v = to_dev(pre)
    say("prefill", w)
    yf = cache.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], expected_block_index=1,
                       blocks_in_prefix=T // 32, slot_idx=slots, y_fwd=True)
    torch.cuda.synchronize()
    s_ref, y_ref = oracle.scan_forward(pre, s0[slots].astype(np.float64), want_y=True)
    got = from_pool(cache.h)
    e = rel_err(got[slots], s_ref)
    say("  state rel err", e)
    assert e <= REL_TOL
    assert rel_err(yf, y_ref) <= REL_TOL
    np.testing.assert_array_equal(got[[1, 3]], s0[[1, 3]])          # other slots untouched
    k = T // 32
    assert cache.n_blocks.tolist() == [1 + k, 2, 1 + k, 9, 1 + k]
    assert cache.n_committed.tolist() == [32 + T, 64, 32 + T, 288, 32 + T]


def test_prefill_equals_commits():
    """One prefill launch over 64 blocks equals 64 commits of the same blocks."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, 8, 64, 128, 1, 32, 2048, True, 1, 9600)
    pre = bi.prefix_inputs(w)
    a, b = bd.Cache(2, 8, 128), bd.Cache(2, 8, 128)
    v = to_dev(pre)
    a.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], 0, 64)
    for k in range(64):
        blk = to_dev(bi.slice_tokens(pre, 32 * k, 32 * (k + 1)))
        b.commit(blk["x"], blk["dt"], blk["A"], blk["B"], blk["C"], blk["D"], blk["D_rev"], k)
    torch.cuda.synchronize()
    assert a.n_blocks.tolist() == b.n_blocks.tolist() == [64, 64]
    assert a.n_committed.tolist() == b.n_committed.tolist() == [2048, 2048]
    ref = oracle.scan_forward(pre)
    assert rel_err(a.states(), ref) <= REL_TOL and rel_err(b.states(), ref) <= REL_TOL


def test_prefill_fp32_storage_segments():
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, 3, 64, 32, 1, 32, 1300, False, 1, 9650)
    pre = bi.prefix_inputs(w)
    s0 = bi.random_state(w, 2, 4, 0.5)
    cache = bd.Cache(2, 3, 32)
    cache.h.copy_(pool_dev(s0))
    v = to_dev(pre)
    yf = cache.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], y_fwd=True)
    torch.cuda.synchronize()
    s_ref, y_ref = oracle.scan_forward(pre, s0.astype(np.float64), want_y=True)
    assert rel_err(from_pool(cache.h), s_ref) <= REL_TOL
    assert rel_err(yf, y_ref) <= REL_TOL


def test_prefill_rejects_wrong_block_index():
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 1, 2, 64, 32, 1, 32, 64, True, 1, 9700)
    v = to_dev(bi.prefix_inputs(w))
    cache = bd.Cache(1, 2, 32)
    with pytest.raises(bd.BdlmError) as ei:
        cache.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], 3, 2)
    assert ei.value.code == bd.E_OFFSET
    assert cache.n_blocks.tolist() == [0]


def test_prefill_bench_shape_sampled():
    """The prefill the bench times: 350M layer shape, batch 16, a 16,384-token clean
    prefix drawn on the GPU, states only.  The committed states of every head of batch
    rows 0 and 15 and of every row of heads 0 and 31 against the oracle's prefix scan of
    those slices."""
    import paper_2607_02805_amd as bd
    w = bi.WORKLOADS[3]
    T = 16384
    v = bi.tokens_device(w, T, w.base_seed + 1)
    hp = bi.head_params(w)
    dhp = {k: torch.from_numpy(a).to(DEV) for k, a in hp.items()}
    cache = bd.Cache(w.batch, w.nheads, w.dstate)
    say("prefill, bench shape", w)
    cache.prefill(v["x"], v["dt"], dhp["A"], v["B"], v["C"], dhp["D"])
    torch.cuda.synchronize()
    got = from_pool(cache.h)
    for rows, heads in edge_cover(w.batch, w.nheads):
        ref = oracle.scan_forward(host_slice(v, rows, heads, hp))
        e = rel_err(got[rows][:, heads], ref)
        say("  rows", rows, "heads", heads, "state rel err", e)
        assert e <= REL_TOL
    assert cache.n_committed.tolist() == [T] * w.batch


def test_prefill_states_bitwise_repeatable_many_workgroups():
    """Batch 8 x 256 heads x 1024 tokens (more workgroups than CUs): the committed states
    are bitwise equal across calls, and sampled heads match the oracle's prefix scan."""
    import paper_2607_02805_amd as bd
    B, H, N, T = 8, 256, 128, 1024
    w = wl(B, H, N, T, seed=9500)
    d = bi.block_inputs(w, 0)
    v = to_dev(d)
    states = []
    for _ in range(3):
        c = bd.Cache(B, H, N)
        c.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"])
        torch.cuda.synchronize()
        states.append(c.h.clone())
    assert torch.equal(states[0], states[1]) and torch.equal(states[0], states[2])
    got = from_pool(states[0])
    for b, h in ((0, 0), (B - 1, H - 1), (3, 101)):
        sub = {"x": d["x"][b:b + 1, :, h:h + 1], "dt": d["dt"][b:b + 1, :, h:h + 1],
               "B": d["B"][b:b + 1], "C": d["C"][b:b + 1],
               "A": d["A"][h:h + 1], "D": d["D"][h:h + 1], "D_rev": d["D_rev"][h:h + 1]}
        ref = oracle.scan_forward(sub)
        assert rel_err(got[b:b + 1, h:h + 1], ref) <= REL_TOL

"""GPU parity of bdlm_commit_step (the clean block's commit followed by the next block's
first denoising step from the committed state, Eq. boundary-state then Eq.
partial-reverse) against the oracle's commit then block step, and against the two calls
it replaces (bdlm_commit_boundary, then bdlm_scan_block_step): bitwise equal, since the
fused launch runs the same arithmetic in the same order.

Bar: max relative error 2e-3 (tests/gpu_util.py); bookkeeping bit-exact.
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
    print("[gpu-commit-step]", *a, flush=True)
    sys.stdout.flush()


def run(w, nslots, slots, want_clean=True, seed_state=21):
    import paper_2607_02805_amd as bd
    c = bi.commit_inputs(w)
    n = bi.block_inputs(w, 3)
    pool = bi.random_state(w, nslots, seed_state, 0.5)
    rows = slots if slots is not None else list(range(w.batch))
    nb = np.arange(nslots, dtype=np.int64) + 1
    nb[rows] = 7
    nc = nb * w.block_len
    cv, nv = to_dev(c), to_dev(n)
    h = pool_dev(pool)
    say("commit_step", w, "slots", slots)
    y_next, y_clean = bd.commit_step((cv["x"], cv["dt"], cv["B"], cv["C"]),
                                     (nv["x"], nv["dt"], nv["B"], nv["C"]), cv["A"], cv["D"],
                                     cv["D_rev"], h, nc, nb, 7, slot_idx=slots,
                                     y_clean=True if want_clean else None)
    torch.cuda.synchronize()
    ref = pool.astype(np.float64)
    onc, onb = (np.arange(nslots, dtype=np.int64) + 1) * w.block_len, np.arange(nslots, dtype=np.int64) + 1
    onb[rows] = 7
    onc[rows] = 7 * w.block_len
    rc, yc_ref = oracle.commit(c, ref, onc, onb, slot_idx=slots, expected_block_index=7)
    assert rc == 0
    y_ref = oracle.block_step(n, ref, slot_idx=slots)
    e = [rel_err(from_pool(h)[rows], ref[rows]), rel_err(y_next, y_ref)]
    if want_clean:
        e.append(rel_err(y_clean, yc_ref))
    say("  rel err state, next y, clean y", e)
    assert max(e) <= REL_TOL
    assert nc.tolist() == onc.tolist() and nb.tolist() == onb.tolist()
    other = np.setdiff1d(np.arange(nslots), rows)
    np.testing.assert_array_equal(from_pool(h)[other], pool[other])


@pytest.mark.parametrize("N", [16, 32, 64, 128])
@pytest.mark.parametrize("L", [1, 16, 17, 32])
def test_commit_step_fused(N, L):
    """bf16 blocks of up to 32 tokens: one launch."""
    run(bi.Workload("t", 5, 8, 64, N, 1, L, 0, True, 1, 18000 + N + L), 9, [8, 0, 3, 5, 1])


@pytest.mark.parametrize("N,L,bf16", [(128, 48, True), (64, 64, True), (32, 20, False)])
def test_commit_step_two_launches(N, L, bf16):
    """Longer blocks and fp32 storage: a commit launch and a step launch."""
    run(bi.Workload("t", 3, 4, 64, N, 1, L, 0, bf16, 1, 18100 + N + L), 3, None)


def test_commit_step_without_clean_outputs_and_groups():
    run(bi.Workload("t", 4, 8, 64, 64, 2, 32, 0, True, 1, 18200), 4, None, want_clean=False)


def test_commit_step_full_size_equals_commit_then_step():
    """The 350M layer shape at batch 16 (the bench's block cycle): every element against the
    oracle, and bit for bit equal to bdlm_commit_boundary followed by bdlm_scan_block_step."""
    import paper_2607_02805_amd as bd
    w = bi.WORKLOADS[3]
    run(w, 16, None)
    c, n = to_dev(bi.commit_inputs(w)), to_dev(bi.block_inputs(w, 2))
    pool = pool_dev(bi.random_state(w, 16, 22, 0.5))
    h1, h2 = pool.clone(), pool.clone()
    z = np.zeros(16, np.int64)
    y1, yc1 = bd.commit_step((c["x"], c["dt"], c["B"], c["C"]), (n["x"], n["dt"], n["B"], n["C"]),
                             c["A"], c["D"], c["D_rev"], h1, z.copy(), z.copy(), y_clean=True)
    yc2 = bd.commit_boundary(c["x"], c["dt"], c["A"], c["B"], c["C"], c["D"], c["D_rev"], h2,
                             z.copy(), z.copy(), y_clean=True)
    y2 = bd.scan_block_step(n["x"], n["dt"], n["A"], n["B"], n["C"], n["D"], n["D_rev"], h2)
    torch.cuda.synchronize()
    assert torch.equal(h1, h2) and torch.equal(yc1, yc2) and torch.equal(y1, y2)


def test_commit_step_refuses_wrong_block_index():
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, 4, 64, 32, 1, 32, 0, True, 1, 18300)
    c, n = to_dev(bi.commit_inputs(w)), to_dev(bi.block_inputs(w, 0))
    h = torch.zeros(bd.pool_shape(2, 4, 32), device=DEV)
    nc, nb = np.zeros(2, np.int64), np.array([1, 2], np.int64)
    with pytest.raises(bd.BdlmError) as ei:
        bd.commit_step((c["x"], c["dt"], c["B"], c["C"]), (n["x"], n["dt"], n["B"], n["C"]),
                       c["A"], c["D"], c["D_rev"], h, nc, nb, 1)
    assert ei.value.code == bd.E_OFFSET
    torch.cuda.synchronize()
    assert (h == 0).all() and nb.tolist() == [1, 2]

"""Bitwise run-to-run repeatability of every shipped kernel family on grids larger than
the chip (so CUs run several workgroups in turn, in an order that varies between calls):
ten calls each, outputs pre-filled differently before every call.  The kernels are
deterministic by construction (no atomics: the reverse sequence pass reads and rewrites
each output it adds onto, one reader and writer per element; LDS traffic modelled
race-free in tests/test_lds_model.py; no MFMA accumulator handed between MFMA shapes,
checked on the generated code by tests/test_mfma_chains.py); these repeats are the
measurement that backs it."""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
from tests.gpu_util import DEV, pool_dev, to_dev

pytestmark = pytest.mark.gpu
REPEATS = 10


def say(*a):
    print("[gpu-determinism]", *a, flush=True)
    sys.stdout.flush()


def repeats(fn):
    outs = []
    for r in range(REPEATS):
        outs.append(fn(r))
    torch.cuda.synchronize()
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert torch.equal(a, b)


def filled(shape, r):
    return torch.full(shape, float(r) if r % 2 else float("nan"), device=DEV)


def test_block_step_and_commit_repeat():
    import dataclasses

    import paper_2607_02805_amd as bd
    w = dataclasses.replace(bi.WORKLOADS[3], batch=128)       # 4,096 workgroups
    d = to_dev(bi.block_inputs(w, 0))
    pool = pool_dev(bi.random_state(w, 128, 3, 0.5))
    say("block step / commit, batch 128")

    def step(r):
        y = filled((128, 32, 32, 64), r)
        bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], pool, y=y)
        return (y,)
    repeats(step)

    def commit(r):
        h = pool.clone()
        yc = filled((128, 32, 32, 64), r)
        bd.commit_boundary(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], h,
                           np.zeros(128, np.int64), np.zeros(128, np.int64), y_clean=yc)
        return (h, yc)
    repeats(commit)


def test_sequence_kernels_repeat():
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 4, 64, 64, 128, 1, 3000, 0, True, 1, 17000)
    v = bi.tokens_device(w, 3000, 17001)
    hp = {k: torch.from_numpy(a).to(DEV) for k, a in bi.head_params(w).items()}
    say("full window, prefill, boundary states")

    def full(r):
        y = filled((4, 3000, 64, 64), r)
        bd.scan_full_window(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], hp["D_rev"], y=y)
        return (y,)
    repeats(full)

    def pre(r):
        c = bd.Cache(4, 64, 128)
        yf = filled((4, 3000, 64, 64), r)
        c.prefill(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], y_fwd=yf)
        return (c.h, yf)
    repeats(pre)

    x, dt, B, C = (v[k][:, :2048].contiguous() for k in ("x", "dt", "B", "C"))

    def states(r):
        s, yf = bd.block_boundary_states(x, dt, hp["A"], B, C, hp["D"], 32,
                                         y_fwd=filled((4, 2048, 64, 64), r))
        return (s, yf)
    repeats(states)


@pytest.mark.parametrize("N", [16, 64, 128])
def test_single_chunk_windows_repeat(N):
    """2,048 workgroups of one 64-token chunk each (batch 8, 256 heads): the shape on which
    an MFMA accumulator handed from a 32-deep to a 16-deep MFMA showed up (outputs at
    tokens 32 + {0, 1, 4, 5, 8, 9, 12, 13} of a chunk changed from call to call).  The full
    window and the forward outputs of a prefill, ten calls each."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 8, 256, 64, N, 1, 64, 0, True, 1, 17500 + N)
    v = to_dev(bi.block_inputs(w, 0))
    say("single-chunk windows", dict(N=N))

    def full(r):
        y = filled((8, 64, 256, 64), r)
        bd.scan_full_window(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], y=y)
        return (y,)
    repeats(full)

    def pre(r):
        c = bd.Cache(8, 256, N)
        yf = filled((8, 64, 256, 64), r)
        c.prefill(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], y_fwd=yf)
        return (c.h, yf)
    repeats(pre)


def test_long_block_and_variants_repeat():
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 16, 26, 64, 128, 1, 256, 0, True, 1, 17100)
    d = to_dev(bi.block_inputs(w, 0))
    pool = pool_dev(bi.random_state(w, 16, 4, 0.5))
    say("256-token block step")

    def step(r):
        y = filled((16, 256, 26, 64), r)
        bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], pool, y=y)
        return (y,)
    repeats(step)
    say("256-token block commit, with and without its outputs")

    def commit(r):
        h, h2 = pool.clone(), pool.clone()
        yc = filled((16, 256, 26, 64), r)
        bd.commit_boundary(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], h,
                           np.zeros(16, np.int64), np.zeros(16, np.int64), y_clean=yc)
        bd.commit_boundary(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], h2,
                           np.zeros(16, np.int64), np.zeros(16, np.int64))
        assert torch.equal(h, h2)   # the outputs do not change the committed state
        return (h, yc, h2)
    repeats(commit)

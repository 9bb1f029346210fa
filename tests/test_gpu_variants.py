"""GPU parity of the block-step variants against the fp64 oracle:

* blocks longer than 64 tokens (the paper's block length 256, ragged lengths), at the
  paper's layer widths (d_inner 896 and 1664: 14 and 26 heads of 64): step and commit;
* separate reverse-direction inputs (the reverse branch with its own projections and
  A, D): the oracle's forward part on the forward inputs plus its reverse part on the
  reverse inputs.

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
    print("[gpu-variants]", *a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("H,N,L", [(14, 128, 256), (26, 128, 256), (4, 64, 65), (3, 16, 300),
                                   (8, 128, 128)])
def test_long_block_step(H, N, L):
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 3, H, 64, N, 1, L, 0, True, 1, 10000 + H + L)
    d = bi.block_inputs(w, 0)
    d["D_rev"] = (d["D"] * 0.75).astype(np.float32)
    pool = bi.random_state(w, 5, 3, 0.5).astype(np.float64)
    slots = [4, 1, 4]
    v = to_dev(d)
    say("long step", dict(H=H, N=N, L=L))
    y = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                           pool_dev(pool), slot_idx=slots)
    torch.cuda.synchronize()
    e = rel_err(y, oracle.block_step(d, pool, slot_idx=slots))
    say("  rel err", e)
    assert e <= REL_TOL


@pytest.mark.parametrize("H,N,L,want_y", [(26, 128, 256, True), (14, 64, 256, False),
                                          (4, 32, 100, True)])
def test_long_block_commit(H, N, L, want_y):
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, H, 64, N, 1, L, 0, True, 1, 10100 + H + L)
    d = bi.commit_inputs(w)
    pool = bi.random_state(w, 3, 5, 0.5).astype(np.float64)
    slots = [2, 0]
    nb = np.array([3, 1, 3], np.int64)
    nc = nb * L
    ref_pool, ref_nc, ref_nb = pool.copy(), nc.copy(), nb.copy()
    rc, y_ref = oracle.commit(d, ref_pool, ref_nc, ref_nb, slot_idx=slots, expected_block_index=3,
                              want_y=True)
    assert rc == 0
    v = to_dev(d)
    h = pool_dev(pool)
    yc = True if want_y else None
    out = bd.commit_boundary(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], h, nc, nb,
                             3, slot_idx=slots, y_clean=yc)
    torch.cuda.synchronize()
    assert nc.tolist() == ref_nc.tolist() and nb.tolist() == ref_nb.tolist()
    got = from_pool(h)
    assert rel_err(got[slots], ref_pool[slots]) <= REL_TOL
    np.testing.assert_array_equal(got[1], pool[1].astype(np.float32))     # untouched slot
    if want_y:
        assert rel_err(out, y_ref) <= REL_TOL


@pytest.mark.parametrize("H,N,L,G", [(4, 16, 256, 1), (4, 32, 129, 2), (6, 64, 191, 1),
                                   (2, 128, 200, 2), (5, 128, 255, 1), (3, 64, 66, 1),
                                   (8, 32, 192, 4), (3, 16, 130, 1), (1, 64, 193, 1)])
def test_long_block_chunked_shapes(H, N, L, G):
    """Blocks of 65 to 256 tokens with bf16 inputs run as one masked-matrix launch (8 or
    16 token tiles; ragged last tiles from 1 to 15 tokens; every dstate, the lone quad
    of dstate 16 paired with zeros; several groups): the step and then the commit with
    its clean-block outputs, against the oracle."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 3, H, 64, N, G, L, 0, True, 1, 10200 + H + N + L)
    d, c = bi.block_inputs(w, 0), bi.commit_inputs(w)
    d["D_rev"] = (d["D"] * 0.5).astype(np.float32)
    c["D_rev"] = d["D_rev"]
    pool = bi.random_state(w, 4, 9, 0.5).astype(np.float64)
    slots = [3, 0, 2]
    h = pool_dev(pool)
    v = to_dev(d)
    say("long step", dict(H=H, N=N, L=L, G=G))
    y = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], h,
                           slot_idx=slots)
    torch.cuda.synchronize()
    e = rel_err(y, oracle.block_step(d, pool, slot_idx=slots))
    say("  step rel err", e)
    assert e <= REL_TOL
    nb = np.array([2, 5, 2, 2], np.int64)
    nc = nb * L
    ref_pool, ref_nc, ref_nb = pool.copy(), nc.copy(), nb.copy()
    rc, y_ref = oracle.commit(c, ref_pool, ref_nc, ref_nb, slot_idx=slots, expected_block_index=2,
                              want_y=True)
    assert rc == 0
    vc = to_dev(c)
    out = bd.commit_boundary(vc["x"], vc["dt"], vc["A"], vc["B"], vc["C"], vc["D"], vc["D_rev"], h,
                             nc, nb, 2, slot_idx=slots, y_clean=True)
    torch.cuda.synchronize()
    got = from_pool(h)
    eh, ey = rel_err(got[slots], ref_pool[slots]), rel_err(out, y_ref)
    say("  commit state rel err", eh, "y_clean rel err", ey)
    assert eh <= REL_TOL and ey <= REL_TOL
    assert nc.tolist() == ref_nc.tolist() and nb.tolist() == ref_nb.tolist()
    np.testing.assert_array_equal(got[1], pool[1].astype(np.float32))     # untouched slot


def _decay_regime(d, regime):
    """Inputs with extreme decays: "fast" (dt x 300: a token's decay reaches 2^-60, and
    most products of decay factors underflow to zero) or "slow" (A x 1e-4: decays within
    1e-3 of one, so whole blocks add up undamped)."""
    if regime == "fast":
        dt = bi.bf16_bits_to_f32(d["dt"]) * np.float32(300.0)
        d["dt"] = bi.to_bf16_bits(dt)
    else:
        d["A"] = (d["A"] * np.float32(1e-4)).astype(np.float32)
    return d


@pytest.mark.parametrize("regime", ["fast", "slow"])
@pytest.mark.parametrize("L", [32, 256, 150])
def test_extreme_decays(regime, L):
    """The block kernel (L 32) and the long-block kernel (L 150, 256) under extreme decays:
    no overflow, NaN or lost precision in the decay factors; step and commit against the
    oracle."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, 4, 64, 128, 1, L, 0, True, 1, 10400 + L + (regime == "fast"))
    d = _decay_regime(bi.block_inputs(w, 0), regime)
    c = _decay_regime(bi.commit_inputs(w), regime)
    pool = bi.random_state(w, 2, 11, 0.5).astype(np.float64)
    h = pool_dev(pool)
    v = to_dev(d)
    say("extreme decays", regime, "L", L)
    y = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], h)
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    e = rel_err(y, oracle.block_step(d, pool))
    nc, nb = np.zeros(2, np.int64), np.zeros(2, np.int64)
    ref_pool = pool.copy()
    rc, y_ref = oracle.commit(c, ref_pool, nc.copy(), nb.copy(), expected_block_index=0, want_y=True)
    assert rc == 0
    vc = to_dev(c)
    out = bd.commit_boundary(vc["x"], vc["dt"], vc["A"], vc["B"], vc["C"], vc["D"], vc["D_rev"], h,
                             nc, nb, 0, y_clean=True)
    torch.cuda.synchronize()
    eh, ey = rel_err(from_pool(h), ref_pool), rel_err(out, y_ref)
    say("  rel err step", e, "state", eh, "clean y", ey)
    assert max(e, eh, ey) <= REL_TOL


def test_long_block_fp32_sequence_path():
    """fp32 activations in blocks longer than 64 tokens keep the sequence kernels' path."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, 3, 64, 64, 1, 256, 0, False, 1, 10300)
    d = bi.block_inputs(w, 0)
    pool = bi.random_state(w, 2, 4, 0.5).astype(np.float64)
    v = to_dev(d)
    say("fp32 long step", w)
    y = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"],
                           pool_dev(pool))
    torch.cuda.synchronize()
    e = rel_err(y, oracle.block_step(d, pool))
    say("  rel err", e)
    assert e <= REL_TOL


def test_paper_geometry_full_size():
    """The paper's 350M geometry at the size the bench times it (batch 16, 26 heads,
    dstate 128, 256-token blocks, identity slots: 416 workgroups per launch): the step,
    then the commit with the clean-block outputs, every element against the oracle."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("350m-paper-geometry", 16, 26, 64, 128, 1, 256, 0, True, 1, 6000)
    d, c = bi.block_inputs(w, 0), bi.commit_inputs(w)
    pool = bi.random_state(w, 16, 7, 0.5).astype(np.float64)
    h = pool_dev(pool)
    v = to_dev(d)
    say("paper geometry step", w)
    y = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], h)
    torch.cuda.synchronize()
    e = rel_err(y, oracle.block_step(d, pool))
    say("  rel err", e)
    assert e <= REL_TOL
    nc, nb = np.zeros(16, np.int64), np.zeros(16, np.int64)
    ref_pool, ref_nc, ref_nb = pool.copy(), nc.copy(), nb.copy()
    rc, y_ref = oracle.commit(c, ref_pool, ref_nc, ref_nb, expected_block_index=0, want_y=True)
    assert rc == 0
    vc = to_dev(c)
    say("paper geometry commit", w)
    out = bd.commit_boundary(vc["x"], vc["dt"], vc["A"], vc["B"], vc["C"], vc["D"], vc["D_rev"], h,
                             nc, nb, 0, y_clean=True)
    torch.cuda.synchronize()
    eh, ey = rel_err(from_pool(h), ref_pool), rel_err(out, y_ref)
    say("  state rel err", eh, "y_clean rel err", ey)
    assert eh <= REL_TOL and ey <= REL_TOL
    assert nc.tolist() == ref_nc.tolist() and nb.tolist() == ref_nb.tolist()


def sep_inputs(w, seed):
    """Forward inputs and independent reverse inputs (own x, dt, B, C, A, D)."""
    fwd = bi.block_inputs(w, 0)
    rev = bi.tokens(w, w.block_len, seed)
    rp = bi.head_params(w, seed + 1)
    rev.update({"A": rp["A"], "D": rp["D"], "D_rev": rp["D"]})
    return fwd, rev


@pytest.mark.parametrize("H,N,L,bf16", [(32, 128, 32, True), (4, 64, 256, True), (3, 16, 50, False),
                                        (8, 128, 64, True),
                                        # one fused launch (bf16, L <= 32): 16-token tile,
                                        # ragged lengths, every dstate
                                        (8, 64, 13, True), (6, 16, 27, True), (4, 32, 16, True),
                                        (5, 128, 1, True)])
def test_step_separate_reverse_inputs(H, N, L, bf16):
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 2, H, 64, N, 1, L, 0, bf16, 1, 10200 + H + L)
    fwd, rev = sep_inputs(w, 10300 + L)
    pool = bi.random_state(w, 2, 7, 0.5).astype(np.float64)
    vf, vr = to_dev(fwd), to_dev(rev)
    say("separate reverse inputs", dict(H=H, N=N, L=L, bf16=bf16))
    y = bd.scan_block_step_sep((vf["x"], vf["dt"], vf["A"], vf["B"], vf["C"], vf["D"]),
                               (vr["x"], vr["dt"], vr["A"], vr["B"], vr["C"], vr["D_rev"]),
                               pool_dev(pool))
    torch.cuda.synchronize()
    _, yf, _ = oracle.block_step(fwd, pool, parts=True)
    _, _, yr = oracle.block_step(rev, np.zeros_like(pool), parts=True)
    e = rel_err(y, yf + yr)
    say("  rel err", e)
    assert e <= REL_TOL


def test_step_separate_reverse_inputs_full_size():
    """Separate reverse inputs at the size the bench times them (350M layer shape: batch
    16, 32 heads, dstate 128, 32-token bf16 blocks; one launch of 512 workgroups staging
    both input sets), every element against the oracle."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 16, 32, 64, 128, 1, 32, 0, True, 1, 10400)
    fwd, rev = sep_inputs(w, 10401)
    pool = bi.random_state(w, 16, 7, 0.5).astype(np.float64)
    vf, vr = to_dev(fwd), to_dev(rev)
    say("separate reverse inputs, full size", w)
    y = bd.scan_block_step_sep((vf["x"], vf["dt"], vf["A"], vf["B"], vf["C"], vf["D"]),
                               (vr["x"], vr["dt"], vr["A"], vr["B"], vr["C"], vr["D_rev"]),
                               pool_dev(pool))
    torch.cuda.synchronize()
    _, yf, _ = oracle.block_step(fwd, pool, parts=True)
    _, _, yr = oracle.block_step(rev, np.zeros_like(pool), parts=True)
    e = rel_err(y, yf + yr)
    say("  rel err", e)
    assert e <= REL_TOL


def test_step_separate_reverse_inputs_groups_and_slots():
    """The fused separate-input launch with two groups and a slot map: rows read the
    states of their slots, the pool is not written."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 3, 8, 64, 64, 2, 24, 0, True, 1, 10500)
    fwd, rev = sep_inputs(w, 10510)
    pool = bi.random_state(w, 5, 11, 0.5).astype(np.float64)
    slots = np.array([4, 0, 2], dtype=np.int32)
    vf, vr = to_dev(fwd), to_dev(rev)
    h = pool_dev(pool)
    before = from_pool(h).copy()
    say("separate reverse inputs, groups and slots", dict(H=8, N=64, G=2, L=24))
    y = bd.scan_block_step_sep((vf["x"], vf["dt"], vf["A"], vf["B"], vf["C"], vf["D"]),
                               (vr["x"], vr["dt"], vr["A"], vr["B"], vr["C"], vr["D_rev"]),
                               h, slot_idx=slots)
    torch.cuda.synchronize()
    _, yf, _ = oracle.block_step(fwd, pool[slots], parts=True)
    _, _, yr = oracle.block_step(rev, np.zeros_like(pool[slots]), parts=True)
    assert rel_err(y, yf + yr) <= REL_TOL
    np.testing.assert_array_equal(from_pool(h), before)


def test_step_separate_with_shared_inputs_equals_step():
    """With the same inputs in both branches the variant is the ordinary step."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 4, 32, 64, 128, 1, 32, 0, True, 1, 10400)
    d = bi.block_inputs(w, 0)
    pool = pool_dev(bi.random_state(w, 4, 9, 0.5))
    v = to_dev(d)
    y1 = bd.scan_block_step(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"], pool)
    y2 = bd.scan_block_step_sep((v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"]),
                                (v["x"], v["dt"], v["A"], v["B"], v["C"], v["D_rev"]), pool)
    torch.cuda.synchronize()
    ref = oracle.block_step(d, from_pool(pool).astype(np.float64))
    assert rel_err(y1, ref) <= REL_TOL and rel_err(y2, ref) <= REL_TOL

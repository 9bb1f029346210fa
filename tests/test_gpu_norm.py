"""GPU parity of the gated RMS normalisation of the scan output (bdlm_gated_rmsnorm; the
Mamba-2 mixer's output path, App. C) against the fp64 oracle on the same seeded inputs:
alone, after a block step (the step's y gated and normalised), in place, with a strided
gate, in channel groups, at the 350M layer width and the paper's widths (14 and 26 heads),
and over more tokens than one launch grid holds.

Bar: max relative error 2e-3 (tests/gpu_util.py).
"""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import DEV, REL_TOL, pool_dev, rel_err, step, to_dev

pytestmark = pytest.mark.gpu
EPS = 1e-5


def say(*a):
    print("[gpu-norm]", *a, flush=True)
    sys.stdout.flush()


def draw(batch, L, H, bf16=True, seed=7100):
    w = bi.Workload("t", batch, H, 64, 16, 1, L, 0, bf16, 1, seed)
    r = np.random.Generator(np.random.PCG64(seed + 1))
    y = (r.standard_normal((batch, L, H, 64)) * 2.0).astype(np.float32)
    g = bi.gate_inputs(w, L, seed + 2)
    return y, g["z"], g["norm_w"]


def dev_z(z):
    return to_dev({"z": z})["z"]


@pytest.mark.parametrize("batch,L,H,G,bf16", [(2, 5, 3, 1, True), (2, 7, 6, 3, False),
                                              (16, 32, 32, 1, True), (3, 9, 14, 2, True),
                                              (2, 4, 26, 13, True), (1, 3, 1, 1, False),
                                              (2, 3, 256, 4, True), (4, 16, 24, 1, False)])
def test_gated_rmsnorm_matches_oracle(batch, L, H, G, bf16):
    import paper_2607_02805_amd as bd
    y, z, w = draw(batch, L, H, bf16, seed=7100 + H + G)
    say("norm", dict(batch=batch, L=L, H=H, G=G, bf16=bf16))
    out = bd.gated_rmsnorm(torch.from_numpy(y).to(DEV), dev_z(z),
                           torch.from_numpy(w).to(DEV), EPS, G)
    torch.cuda.synchronize()
    ref = oracle.gated_rmsnorm(y.reshape(batch, L, -1), z, w, EPS, G)
    e = rel_err(out.reshape(batch, L, -1), ref)
    say("  rel err", e)
    assert e <= REL_TOL


def test_in_place_strided_gate_and_deterministic():
    """z as a slice of a wider projection output (row stride 2 * channels + 128) and as a
    token slice of a longer sequence; out = y (in place); repeated calls agree bitwise."""
    import paper_2607_02805_amd as bd
    batch, L, H = 4, 12, 8
    y, z, w = draw(batch, L, H, True, seed=7200)
    nch = H * 64
    proj = torch.zeros((batch, L, 2 * nch + 128), dtype=torch.bfloat16, device=DEV)
    zt = dev_z(z)
    proj[:, :, nch:2 * nch] = zt
    zview = proj[:, :, nch:2 * nch]
    yt = torch.from_numpy(y).to(DEV)
    wt = torch.from_numpy(w).to(DEV)
    a = bd.gated_rmsnorm(yt, zview, wt, EPS)
    b = bd.gated_rmsnorm(yt, zt, wt, EPS)
    yt2 = yt.clone()
    c = bd.gated_rmsnorm(yt2, zview, wt, EPS, out=yt2)
    # the block's tokens as a slice of a longer sequence: batch stride != len * token stride
    longer = torch.zeros((batch, L + 5, nch), dtype=torch.bfloat16, device=DEV)
    longer[:, 3:3 + L] = zt
    e = bd.gated_rmsnorm(yt, longer[:, 3:3 + L], wt, EPS)
    torch.cuda.synchronize()
    assert c.data_ptr() == yt2.data_ptr()
    assert torch.equal(a, b) and torch.equal(a, c) and torch.equal(a, e)
    ref = oracle.gated_rmsnorm(y.reshape(batch, L, -1), z, w, EPS)
    assert rel_err(a.reshape(batch, L, -1), ref) <= REL_TOL


def test_step_then_norm_equals_oracle():
    """The block step's y, gated and normalised, against the oracle's step then norm."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("t", 4, 8, 64, 64, 1, 32, 0, True, 1, 7300)
    d = bi.block_inputs(w, 0)
    d.update(bi.head_params(w))
    s0 = bi.random_state(w, 4, 7301, 0.5)
    g = bi.gate_inputs(w, 32, 7302)
    v = to_dev(d)
    y = step(v, pool_dev(s0))
    out = bd.gated_rmsnorm(y, dev_z(g["z"]), torch.from_numpy(g["norm_w"]).to(DEV), EPS)
    torch.cuda.synchronize()
    y_ref = oracle.block_step(d, s0.astype(np.float64))
    ref = oracle.gated_rmsnorm(y_ref.reshape(4, 32, -1), g["z"], g["norm_w"], EPS)
    assert rel_err(out.reshape(4, 32, -1), ref) <= REL_TOL


def test_more_tokens_than_the_grid():
    """2^20 + 37 tokens of one head: workgroups take several tokens in turn; sampled tokens
    (first, last and random) against the oracle, all finite."""
    import paper_2607_02805_amd as bd
    ntok = (1 << 20) + 37
    gen = torch.Generator(device=DEV)
    gen.manual_seed(7400)
    y = torch.randn((1, ntok, 1, 64), generator=gen, device=DEV)
    z = torch.randn((1, ntok, 64), generator=gen, device=DEV).to(torch.bfloat16)
    wt = 1.0 + 0.1 * torch.randn(64, generator=gen, device=DEV)
    say("grid-stride", ntok)
    out = bd.gated_rmsnorm(y, z, wt, EPS)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all())
    rows = np.concatenate([[0, 1, ntok - 1, (1 << 20) - 1, 1 << 20],
                           np.random.Generator(np.random.PCG64(7401)).integers(0, ntok, 64)])
    idx = torch.from_numpy(rows).to(DEV)
    ys = y[0, idx].reshape(len(rows), 64).cpu().numpy()
    zs = z[0, idx].cpu().view(torch.int16).numpy().view(np.uint16)
    ref = oracle.gated_rmsnorm(ys, zs, wt.cpu().numpy(), EPS)
    assert rel_err(out[0, idx].reshape(len(rows), 64), ref) <= REL_TOL


def test_empty_batch():
    import paper_2607_02805_amd as bd
    y = torch.empty((0, 4, 2, 64), device=DEV)
    z = torch.empty((0, 4, 128), dtype=torch.bfloat16, device=DEV)
    out = bd.gated_rmsnorm(y, z, torch.ones(128, device=DEV), EPS)
    assert out.shape == y.shape

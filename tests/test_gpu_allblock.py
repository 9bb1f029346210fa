"""GPU parity of the all-block training forward (Fig. 1, Eq. prefix-cache-loss): the
states entering every block of a clean window (bdlm_block_boundary_states) and every
noised block stepped from its clean prefix's state in one batched block step
(paper_2607_02805_amd.all_block_forward), against the fp64 oracle composed block by
block: s_{k+1} = forward scan of clean block k from s_k, y_k = block step of noised
block k from s_k.

Bar: max relative error 2e-3 (tests/gpu_util.py).
"""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import (DEV, REL_TOL, edge_cover, from_pool, host_slice, pick, pool_dev,
                            rel_err, to_dev, to_host)

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-allblock]", *a, flush=True)
    sys.stdout.flush()


def window(batch, H, N, L, K, bf16=True, seed=9800, G=1):
    """A clean window and its noised counterpart (independent seeded draws)."""
    w = bi.Workload("t", batch, H, 64, N, G, L, K * L, bf16, 1, seed)
    clean = bi.prefix_inputs(w)
    noised = bi.tokens(w, K * L, seed + 5)
    noised.update(bi.head_params(w))
    return w, clean, noised


def oracle_states(clean, K, L, s0):
    """States entering each block (float64 [K, B, H, P, N]) and the forward outputs."""
    states = [s0]
    for k in range(K - 1):
        blk = bi.slice_tokens(clean, k * L, (k + 1) * L)
        states.append(oracle.scan_forward(blk, states[-1]))
    _, y = oracle.scan_forward(clean, s0, want_y=True)
    return np.stack(states), y


# K * L above 256 tokens splits the window into segments of whole blocks (with a short
# last segment where K is not a multiple of the segment's blocks)
@pytest.mark.parametrize("N,L,K", [(16, 16, 5), (64, 32, 4), (128, 32, 6), (128, 64, 3),
                                   (32, 24, 3), (128, 32, 1), (64, 32, 21), (32, 24, 25),
                                   (16, 16, 40), (128, 64, 9)])
def test_boundary_states_and_clean_outputs(N, L, K):
    import paper_2607_02805_amd as bd
    w, clean, _ = window(2, 3, N, L, K, seed=9800 + N + L + K)
    s0 = bi.random_state(w, 2, 11, 0.5).astype(np.float64)
    v = to_dev(clean)
    say("boundary states", dict(N=N, L=L, K=K))
    s_out, yf = bd.block_boundary_states(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], L,
                                         s_init=pool_dev(s0), y_fwd=True)
    torch.cuda.synchronize()
    ref, y_ref = oracle_states(clean, K, L, s0)
    got = from_pool(s_out).reshape(2, K, 3, 64, N)
    e = rel_err(got, ref.transpose(1, 0, 2, 3, 4))
    say("  states rel err", e)
    assert e <= REL_TOL
    assert np.array_equal(got[:, 0], s0.astype(np.float32))      # block 0 enters with s_init
    assert rel_err(yf, y_ref) <= REL_TOL


@pytest.mark.parametrize("N,L,K,bf16", [(64, 32, 4, True), (128, 32, 5, True), (16, 16, 3, False),
                                        (128, 64, 2, True), (64, 32, 20, True), (32, 16, 35, False)])
def test_all_block_forward(N, L, K, bf16):
    import paper_2607_02805_amd as bd
    w, clean, noised = window(2, 4, N, L, K, bf16=bf16, seed=9900 + N + L + K)
    noised["D_rev"] = (noised["D"] * 0.5).astype(np.float32)
    vc, vn = to_dev(clean), to_dev(noised)
    say("all-block forward", dict(N=N, L=L, K=K, bf16=bf16))
    y, s_out = bd.all_block_forward((vc["x"], vc["dt"], vc["B"], vc["C"]),
                                    (vn["x"], vn["dt"], vn["B"], vn["C"]),
                                    vn["A"], vn["D"], vn["D_rev"], L)
    torch.cuda.synchronize()
    states, _ = oracle_states(clean, K, L, np.zeros((2, 4, 64, N)))
    for k in range(K):
        blk = bi.slice_tokens(noised, k * L, (k + 1) * L)
        y_ref = oracle.block_step(blk, states[k])
        e = rel_err(y[:, k * L:(k + 1) * L], y_ref)
        assert e <= REL_TOL, (k, e)


def test_all_block_forward_equals_sampler():
    """Each noised block's output equals the sampler's step after committing the clean
    blocks before it (the cache the training computation shares with inference)."""
    import paper_2607_02805_amd as bd
    L, K = 32, 4
    w, clean, noised = window(2, 8, 128, L, K, seed=9950)
    vc, vn = to_dev(clean), to_dev(noised)
    y, _ = bd.all_block_forward((vc["x"], vc["dt"], vc["B"], vc["C"]),
                                (vn["x"], vn["dt"], vn["B"], vn["C"]), vn["A"], vn["D"],
                                vn["D_rev"], L)
    cache = bd.Cache(2, 8, 128)
    for k in range(K):
        sl = slice(k * L, (k + 1) * L)
        ys = cache.step(vn["x"][:, sl].contiguous(), vn["dt"][:, sl].contiguous(), vn["A"],
                        vn["B"][:, sl].contiguous(), vn["C"][:, sl].contiguous(), vn["D"], vn["D_rev"])
        torch.cuda.synchronize()
        assert rel_err(y[:, sl], ys.cpu().double().numpy()) <= REL_TOL
        cache.commit(vc["x"][:, sl].contiguous(), vc["dt"][:, sl].contiguous(), vc["A"],
                     vc["B"][:, sl].contiguous(), vc["C"][:, sl].contiguous(), vc["D"], vc["D_rev"], k)


def test_all_block_forward_full_size_sampled():
    """The all-block forward at the size the bench times it (350M layer shape, batch 8, an
    8,192-token window of 256 blocks of 32 tokens, inputs drawn on the GPU): for every head
    of batch rows 0 and 7 and every row of heads 0 and 31, the states entering all 256
    blocks, the clean stream's forward outputs and the noised stream's outputs against the
    oracle run on those slices."""
    import paper_2607_02805_amd as bd
    w = bi.Workload("350m-train-window", 8, 32, 64, 128, 1, 32, 8192, True, 1, 5000)
    T, L, K = 8192, 32, 256
    c = bi.tokens_device(w, T, w.base_seed + 1)
    n = bi.tokens_device(w, T, w.base_seed + 10)
    hp = bi.head_params(w)
    dhp = {k: torch.from_numpy(a).to(DEV) for k, a in hp.items()}
    say("all-block forward, full size", w)
    y, s_out, yc = bd.all_block_forward((c["x"], c["dt"], c["B"], c["C"]),
                                        (n["x"], n["dt"], n["B"], n["C"]),
                                        dhp["A"], dhp["D"], dhp["D_rev"], L, want_clean_y=True)
    torch.cuda.synchronize()
    states = from_pool(s_out).reshape(8, K, 32, 64, 128)
    for rows, heads in edge_cover(w.batch, w.nheads):
        cs, ns = host_slice(c, rows, heads, hp), host_slice(n, rows, heads, hp)
        R, Hs = len(rows), len(heads)
        ref_states, ref_yc = oracle_states(cs, K, L, np.zeros((R, Hs, 64, 128)))   # [K, R, Hs, ..]
        # the noised blocks as R * K rows of one block each, stepped from their entering states
        blk = {k: (ns[k].reshape(R * K, L, *ns[k].shape[2:]) if k in ("x", "dt", "B", "C") else ns[k])
               for k in ns}
        ref_y = oracle.block_step(blk, np.ascontiguousarray(ref_states.swapaxes(0, 1)).reshape(
            R * K, Hs, 64, 128))
        got_states = states[rows][:, :, heads]                                        # [R, K, Hs, ..]
        e = (rel_err(got_states, ref_states.swapaxes(0, 1)), rel_err(pick(yc, rows, heads), ref_yc),
             rel_err(pick(y, rows, heads).reshape(R * K, L, Hs, 64), ref_y))
        say("  rows", rows, "heads", heads, "rel err states, clean y, noised y", e)
        assert max(e) <= REL_TOL


def test_boundary_states_many_workgroups_deterministic():
    """Batch 4 x 32 heads x 64 blocks: far more workgroups than CUs; bitwise repeatable."""
    import paper_2607_02805_amd as bd
    w, clean, _ = window(4, 32, 128, 32, 64, seed=9970)
    v = to_dev(clean)
    a = bd.block_boundary_states(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], 32)
    b = bd.block_boundary_states(v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], 32)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    # spot-check two (row, head) pairs against the oracle
    for bb, h in ((0, 0), (3, 17)):
        sub = {k: (clean[k][bb:bb + 1, :, h:h + 1] if k in ("x", "dt") else
                   clean[k][bb:bb + 1] if k in ("B", "C") else clean[k][h:h + 1]) for k in clean}
        ref, _ = oracle_states(sub, 64, 32, np.zeros((1, 1, 64, 128)))
        got = from_pool(a).reshape(4, 64, 32, 64, 128)[bb, :, h]
        assert rel_err(got, ref[:, 0, 0]) <= REL_TOL

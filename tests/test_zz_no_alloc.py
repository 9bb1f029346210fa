"""GPU test of the no-allocation prefill (bdlm_prefill_noalloc), called through the C ABI:
two calls in a row on one device -- the second with a smaller input -- each against
bdlm_prefill with a caller workspace on the same inputs and the same starting cache
(states and forward outputs within the parity bar, bookkeeping bit-exact), the small
case also against the oracle; and a request too large for the library's scratch is
refused before anything is enqueued."""
import sys

import numpy as np
import pytest
import torch

import bdlm_inputs as bi
import oracle
from tests.gpu_util import DEV, REL_TOL, from_pool, pool_dev, rel_err, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-noalloc]", *a, flush=True)
    sys.stdout.flush()


def both(v, hp, s0_dev, nslots, slots, T, blocks, want_y):
    """The same prefill through bdlm_prefill (caller workspace) and bdlm_prefill_noalloc."""
    import paper_2607_02805_amd as bd
    bsz, H, N = v["x"].shape[0], v["x"].shape[2], v["B"].shape[3]
    out = []
    for noalloc in (False, True):
        h = s0_dev.clone()
        nc = np.arange(nslots, dtype=np.int64) * 32
        nb = np.arange(nslots, dtype=np.int64)
        nb[slots if slots is not None else np.arange(bsz)] = 2
        y = torch.full((bsz, T, H, 64), float("nan"), device=DEV) if want_y else None
        args = (v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], h, nc, nb)
        if noalloc:
            bd.prefill_noalloc(*args, expected_block_index=2, blocks_in_prefix=blocks,
                               slot_idx=slots, y_fwd=y)
        else:
            bd.prefill(*args, expected_block_index=2, blocks_in_prefix=blocks, slot_idx=slots,
                       y_fwd=y)
        torch.cuda.synchronize()
        out.append((h, y, nc, nb))
    return out


def test_noalloc_prefill_two_calls_then_smaller():
    import paper_2607_02805_amd as bd
    # call 1: the bench's prefill shape (350M layer, batch 16, 16,384 tokens): its standard
    # segment plan needs 64 MiB + 8 KiB, so the scratch plan uses fewer, longer segments
    w = bi.WORKLOADS[3]
    T = 16384
    v = bi.tokens_device(w, T, w.base_seed + 1)
    hp = {k: torch.from_numpy(a).to(DEV) for k, a in bi.head_params(w).items()}
    assert bd.prefill_workspace_bytes(16, 32, 128, T) > bd.SCRATCH_BYTES
    s0 = torch.randn(bd.pool_shape(16, 32, 128), device=DEV) * 0.1
    say("call 1: batch 16, 32 heads, dstate 128, 16384 tokens")
    (h1, _, nc1, nb1), (h2, _, nc2, nb2) = both(v, hp, s0, 16, None, T, 512, False)
    e = rel_err(h2, h1.cpu().double().numpy())
    say("  state rel err vs bdlm_prefill", e)
    assert e <= REL_TOL
    assert nc1.tolist() == nc2.tolist() and nb1.tolist() == nb2.tolist()
    del v
    # call 2, smaller: batch 3 of a 5-slot pool through a slot map, with forward outputs
    w2 = bi.Workload("t", 3, 4, 64, 64, 1, 32, 1000, True, 1, 16000)
    pre = bi.prefix_inputs(w2)
    v2 = to_dev(pre)
    hp2 = {k: v2[k] for k in ("A", "D", "D_rev")}
    s0n = bi.random_state(w2, 5, 16001, 0.5)
    slots = [4, 0, 2]
    say("call 2: batch 3, 4 heads, dstate 64, 1000 tokens, slot map")
    (h1, y1, nc1, nb1), (h2, y2, nc2, nb2) = both(v2, hp2, pool_dev(s0n), 5, slots, 1000, 31, True)
    assert rel_err(h2, h1.cpu().double().numpy()) <= REL_TOL
    assert rel_err(y2, y1.cpu().double().numpy()) <= REL_TOL
    assert nc1.tolist() == nc2.tolist() and nb1.tolist() == nb2.tolist()
    s_ref, y_ref = oracle.scan_forward(pre, s0n[slots].astype(np.float64), want_y=True)
    got = from_pool(h2)
    assert rel_err(got[slots], s_ref) <= REL_TOL and rel_err(y2, y_ref) <= REL_TOL
    np.testing.assert_array_equal(got[[1, 3]], s0n[[1, 3]])     # slots outside the map untouched


def test_noalloc_prefill_refuses_what_the_scratch_cannot_hold():
    import paper_2607_02805_amd as bd
    # 512 row-heads x 64 x 128 fp32 states need 16 MiB per segment: fine; 2,560 row-heads
    # need 80 MiB even as one segment: refused before anything is enqueued
    w = bi.Workload("t", 80, 32, 64, 128, 1, 32, 256, True, 1, 16100)
    v = bi.tokens_device(w, 256, 16101)
    hp = {k: torch.from_numpy(a).to(DEV) for k, a in bi.head_params(w).items()}
    h = torch.zeros(bd.pool_shape(80, 32, 128), device=DEV)
    nc, nb = np.zeros(80, np.int64), np.zeros(80, np.int64)
    with pytest.raises(bd.BdlmError) as ei:
        bd.prefill_noalloc(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], h, nc, nb)
    assert ei.value.code == bd.E_WORKSPACE
    torch.cuda.synchronize()
    assert (h == 0).all() and nc.tolist() == [0] * 80
    with pytest.raises(ValueError):
        bd.prefill_noalloc(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], h, nc, nb, y_fwd=True)

"""Pins for the fp64 CPU oracle: each test checks it against something other than itself.

* a two-token example worked by hand (tests/golden/hand_example_L2.json);
* closed forms (geometric series) for constant inputs, including the A = 0 limit;
* special cases L = 1, B = 0, C = 0;
* each scan direction as a bidiagonal linear system solved by LAPACK;
* the masked-matrix (state-space dual) form of the same operator;
* the paper's definition of the reverse branch, rev(F(rev(block))), rebuilt from
  the forward scan of the flipped block (Sec. 4, Eq. partial-reverse);
* structural claims of Sec. 4: the cache is a function of the clean prefix only
  (committing block by block equals one pass), the reverse branch is local to the
  block and never sees the cache, causality / anti-causality inside the block;
* linearity in (x, h) and the palindrome symmetry of the two branches;
* the bookkeeping of a commit (offsets, block indices, slot checks).
"""
import json
import math
import os

import numpy as np
import pytest

import bdlm_inputs as bi
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def mk(x, dt, Bm, Cm, A, D, D_rev=None):
    return {"x": f32(x), "dt": f32(dt), "B": f32(Bm), "C": f32(Cm), "A": f32(A), "D": f32(D),
            "D_rev": f32(D if D_rev is None else D_rev)}


def rand_inputs(batch=2, L=6, H=4, P=3, N=5, G=2, seed=0, bf16=False, prefix=0):
    w = bi.Workload("t", batch, H, P, N, G, L, prefix, bf16, 1, seed)
    d = bi.tokens(w, L, seed + 7)
    d.update(bi.head_params(w, seed + 3))
    # give D_rev its own values so a swapped skip term is visible
    d["D_rev"] = f32(np.random.default_rng(seed + 5).standard_normal(H))
    return w, d


def dec(d):
    return {k: oracle.decode(v) if k in ("x", "dt", "B", "C") else v.astype(np.float64)
            for k, v in d.items()}


# --------------------------------------------------------------------- worked example
def test_hand_example():
    g = json.load(open(os.path.join(GOLDEN, "hand_example_L2.json")))
    d = mk(np.array(g["x"]).reshape(1, 2, 1, 1), np.full((1, 2, 1), g["dt"]),
           np.array(g["B"]).reshape(1, 2, 1, 1), np.array(g["C"]).reshape(1, 2, 1, 1),
           [g["A"]], [g["D"]], [g["D_rev"]])
    h = np.full((1, 1, 1, 1), g["h"])
    y, yf, yr = oracle.block_step(d, h, parts=True)
    rt = g["rtol"]
    np.testing.assert_allclose(y.ravel(), g["y"], rtol=rt)
    np.testing.assert_allclose(yf.ravel(), g["y_fwd"], rtol=rt)
    np.testing.assert_allclose(yr.ravel(), g["y_rev"], rtol=rt)
    nc, nb = np.zeros(1, np.int64), np.zeros(1, np.int64)
    rc, yc = oracle.commit(d, h, nc, nb, expected_block_index=0)
    assert rc == 0
    np.testing.assert_allclose(h.ravel(), [g["h_new"]], rtol=rt)
    np.testing.assert_allclose(yc.ravel(), g["y"], rtol=rt)
    assert nc.tolist() == [2] and nb.tolist() == [1]


# ------------------------------------------------------------------------ closed forms
def geo(a, m):
    """1 + a + ... + a^(m-1), with the a -> 1 limit."""
    return float(m) if a == 1.0 else (1.0 - a ** m) / (1.0 - a)


@pytest.mark.parametrize("A,dtv,L", [(-1.5, 0.25, 7), (-0.2, 0.0625, 12), (0.0, 0.5, 5),
                                     (-3.0, 0.125, 1)])
def test_closed_form_constant_inputs(A, dtv, L):
    P, N = 3, 4
    rng = np.random.default_rng(11)
    xr = f32(rng.standard_normal(P))
    Br, Cr = f32(rng.standard_normal(N)), f32(rng.standard_normal(N))
    h0 = rng.standard_normal((P, N))
    D, Dr = 0.75, -0.5
    d = mk(np.broadcast_to(xr, (1, L, 1, P)), np.full((1, L, 1), dtv),
           np.broadcast_to(Br, (1, L, 1, N)), np.broadcast_to(Cr, (1, L, 1, N)), [A], [D], [Dr])
    hp = h0.reshape(1, 1, P, N).copy()
    y, yf, yr = oracle.block_step(d, hp, parts=True)
    x, Bv, Cv = xr.astype(np.float64), Br.astype(np.float64), Cr.astype(np.float64)
    A, dtv = float(np.float32(A)), float(np.float32(dtv))     # the stored fp32 values
    a = math.exp(dtv * A)
    hC = h0 @ Cv
    CB = float(Cv @ Bv)
    for t in range(L):
        ef = a ** (t + 1) * hC + dtv * CB * x * geo(a, t + 1) + D * x
        er = dtv * CB * x * geo(a, L - t) + Dr * x
        np.testing.assert_allclose(yf[0, t, 0], ef, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(yr[0, t, 0], er, rtol=1e-12, atol=1e-13)
    nc, nb = np.zeros(1, np.int64), np.zeros(1, np.int64)
    assert oracle.commit(d, hp, nc, nb)[0] == 0
    eh = a ** L * h0 + dtv * np.outer(x, Bv) * geo(a, L)
    np.testing.assert_allclose(hp[0, 0], eh, rtol=1e-12, atol=1e-13)


def test_single_token_block():
    """L = 1: both branches see only the token itself; the diagonal counts twice."""
    _, d = rand_inputs(L=1, seed=3)
    D = dec(d)
    h = np.random.default_rng(4).standard_normal((2, 4, 3, 5))
    y = oracle.block_step(d, h)
    for b in range(2):
        for hh in range(4):
            g = hh // 2
            dt = D["dt"][b, 0, hh]
            a = math.exp(dt * D["A"][hh])
            x, Bv, Cv = D["x"][b, 0, hh], D["B"][b, 0, g], D["C"][b, 0, g]
            e = 2 * dt * (Cv @ Bv) * x + a * (h[b, hh] @ Cv) + (D["D"][hh] + D["D_rev"][hh]) * x
            np.testing.assert_allclose(y[b, 0, hh], e, rtol=1e-12, atol=1e-14)


def test_zero_B_and_zero_C():
    _, d = rand_inputs(seed=5)
    h = np.random.default_rng(6).standard_normal((2, 4, 3, 5))
    D = dec(d)
    # B = 0: nothing enters either state; reverse branch is only its skip term
    dB = dict(d, B=np.zeros_like(d["B"]))
    y, yf, yr = oracle.block_step(dB, h, parts=True)
    np.testing.assert_array_equal(yr, D["D_rev"][None, None, :, None] * D["x"])
    cs = np.cumsum(D["dt"] * D["A"][None, None, :], axis=1)
    Cg = np.repeat(D["C"], 2, axis=2)
    ef = np.exp(cs)[..., None] * np.einsum("bhpn,bthn->bthp", h, Cg) \
        + D["D"][None, None, :, None] * D["x"]
    np.testing.assert_allclose(yf, ef, rtol=1e-12, atol=1e-14)
    # C = 0: only the two skip terms survive
    dC = dict(d, C=np.zeros_like(d["C"]))
    y = oracle.block_step(dC, h)
    np.testing.assert_allclose(y, (D["D"] + D["D_rev"])[None, None, :, None] * D["x"],
                               rtol=1e-15, atol=0)


# ----------------------------------------------------------- library linear-solve pin
@pytest.mark.parametrize("bf16", [False, True])
def test_scans_as_bidiagonal_linear_systems(bf16):
    """Forward: S_t - a_t S_{t-1} = dt_t x_t B_t^T, S_{-1} = h.  Reverse: R_t - a_t R_{t+1} =
    dt_t x_t B_t^T, R_L = 0.  Solved with numpy.linalg.solve, read out with C_t."""
    batch, L, H, P, N, G = 2, 6, 4, 3, 5, 2
    _, d = rand_inputs(batch, L, H, P, N, G, seed=21, bf16=bf16)
    h = np.random.default_rng(22).standard_normal((batch, H, P, N))
    y, yf, yr = oracle.block_step(d, h, parts=True)
    D = dec(d)
    for b in range(batch):
        for hh in range(H):
            g = hh // (H // G)
            dt, x = D["dt"][b, :, hh], D["x"][b, :, hh]
            Bm, Cm = D["B"][b, :, g], D["C"][b, :, g]
            a = np.exp(dt * D["A"][hh])
            u = (dt[:, None, None] * x[:, :, None] * Bm[:, None, :]).reshape(L, P * N)
            Mf = np.eye(L) - np.diag(a[1:], k=-1)
            rf = u.copy()
            rf[0] += a[0] * h[b, hh].reshape(-1)
            S = np.linalg.solve(Mf, rf).reshape(L, P, N)
            Mr = np.eye(L) - np.diag(a[:-1], k=1)
            R = np.linalg.solve(Mr, u).reshape(L, P, N)
            ef = np.einsum("tpn,tn->tp", S, Cm) + D["D"][hh] * x
            er = np.einsum("tpn,tn->tp", R, Cm) + D["D_rev"][hh] * x
            np.testing.assert_allclose(yf[b, :, hh], ef, rtol=1e-11, atol=1e-13)
            np.testing.assert_allclose(yr[b, :, hh], er, rtol=1e-11, atol=1e-13)
    np.testing.assert_array_equal(y, yf + yr)


# ------------------------------------------------------------------- dual (SSD) form
def dual_form(D, h):
    """Masked-matrix form: y = exp(cs) (C h^T) + (M_f + M_r) (dt x) + (D + D_rev) x with
    M_f[t,j] = exp(cs_t - cs_j) C_t.B_j for j <= t and M_r[t,j] = exp(cs_{j-1} - cs_{t-1})
    C_t.B_j for j >= t (cs inclusive cumulative sum of dt * A)."""
    batch, L, H, P = D["x"].shape
    G = D["B"].shape[2]
    y = np.zeros((batch, L, H, P))
    tt, jj = np.meshgrid(np.arange(L), np.arange(L), indexing="ij")
    for b in range(batch):
        for hh in range(H):
            g = hh // (H // G)
            dt, x = D["dt"][b, :, hh], D["x"][b, :, hh]
            Bm, Cm = D["B"][b, :, g], D["C"][b, :, g]
            l = dt * D["A"][hh]
            cs = np.cumsum(l)
            ex = cs - l                      # exclusive sum
            Gm = Cm @ Bm.T
            wf = np.where(jj <= tt, np.exp(np.minimum(cs[tt] - cs[jj], 0)), 0.0)
            wr = np.where(jj >= tt, np.exp(np.minimum(ex[jj] - ex[tt], 0)), 0.0)
            y[b, :, hh] = (np.exp(cs)[:, None] * (Cm @ h[b, hh].T)
                           + ((wf + wr) * Gm) @ (dt[:, None] * x)
                           + (D["D"][hh] + D["D_rev"][hh]) * x)
    return y


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("L", [1, 2, 7, 16])
def test_dual_form(bf16, L):
    _, d = rand_inputs(3, L, 4, 5, 6, 1, seed=31 + L, bf16=bf16)
    h = np.random.default_rng(32).standard_normal((3, 4, 5, 6))
    y = oracle.block_step(d, h)
    np.testing.assert_allclose(y, dual_form(dec(d), h), rtol=1e-11, atol=1e-12)


# --------------------------------------------- the paper's definition of the reverse
def test_reverse_is_flip_of_forward_on_flipped_block():
    """y_rev = rev(F(rev(block))) with F the forward scan from a zero state."""
    _, d = rand_inputs(2, 9, 4, 3, 5, 2, seed=41)
    h = np.random.default_rng(42).standard_normal((2, 4, 3, 5))
    _, _, yr = oracle.block_step(d, h, parts=True)
    flipped = {k: (np.ascontiguousarray(v[:, ::-1]) if k in ("x", "dt", "B", "C") else v)
               for k, v in d.items()}
    flipped["D"] = d["D_rev"]
    _, yfl = oracle.scan_forward(flipped, None, want_y=True)
    np.testing.assert_array_equal(yr, yfl[:, ::-1])


def test_reverse_ignores_cache_and_palindrome_symmetry():
    _, d = rand_inputs(2, 8, 4, 3, 5, 2, seed=51)
    r = np.random.default_rng(52)
    _, _, yr1 = oracle.block_step(d, r.standard_normal((2, 4, 3, 5)), parts=True)
    _, _, yr2 = oracle.block_step(d, r.standard_normal((2, 4, 3, 5)), parts=True)
    np.testing.assert_array_equal(yr1, yr2)
    # palindromic block, zero cache, D = D_rev: the forward branch is the mirrored reverse
    pal = {k: (np.ascontiguousarray(np.concatenate([v[:, :4], v[:, :4][:, ::-1]], axis=1))
               if k in ("x", "dt", "B", "C") else v) for k, v in d.items()}
    pal["D_rev"] = pal["D"]
    _, yf, yr = oracle.block_step(pal, np.zeros((2, 4, 3, 5)), parts=True)
    np.testing.assert_array_equal(yf, yr[:, ::-1])


def test_causality_inside_block():
    """Perturbing token j leaves y_fwd before j and y_rev after j bit-identical."""
    _, d = rand_inputs(1, 8, 2, 3, 4, 1, seed=61)
    h = np.random.default_rng(62).standard_normal((1, 2, 3, 4))
    _, yf0, yr0 = oracle.block_step(d, h, parts=True)
    for j in (0, 3, 7):
        e = {k: v.copy() for k, v in d.items()}
        e["x"][:, j] += 1.0
        e["B"][:, j] *= -2.0
        e["dt"][:, j] *= 1.5
        _, yf, yr = oracle.block_step(e, h, parts=True)
        np.testing.assert_array_equal(yf[:, :j], yf0[:, :j])
        np.testing.assert_array_equal(yr[:, j + 1:], yr0[:, j + 1:])
        assert not np.array_equal(yf[:, j:], yf0[:, j:])
        assert not np.array_equal(yr[:, :j + 1], yr0[:, :j + 1])


def test_linearity_in_x_and_h():
    _, d = rand_inputs(2, 6, 4, 3, 5, 2, seed=71)
    h = np.random.default_rng(72).standard_normal((2, 4, 3, 5))
    y = oracle.block_step(d, h)
    y2 = oracle.block_step(dict(d, x=f32(d["x"] * 2.0)), 2.0 * h)
    np.testing.assert_allclose(y2, 2.0 * y, rtol=1e-13, atol=1e-14)
    y_x = oracle.block_step(d, np.zeros_like(h))
    y_h = oracle.block_step(dict(d, x=np.zeros_like(d["x"])), h)
    np.testing.assert_allclose(y_x + y_h, y, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ cache equivalence
def test_commits_equal_one_pass_bitwise():
    """Eq. boundary-state: the cache depends on the clean prefix only.  Committing K blocks
    one by one and then stepping the active block equals one forward pass over
    prefix ++ block, bit for bit (same fp64 operation order)."""
    L, K = 4, 3
    w = bi.Workload("t", 2, 4, 3, 5, 2, L, K * L, True, 1, 81)
    pre = bi.prefix_inputs(w)
    blk = bi.block_inputs(w, 0)
    # one pass
    full = {k: (np.concatenate([pre[k], blk[k]], axis=1) if k in ("x", "dt", "B", "C")
                else pre[k]) for k in pre}
    s_end, y_full = oracle.scan_forward(full, None, want_y=True)
    # block by block, through a pool with non-identity slots
    slots = np.array([2, 0], np.int32)
    pool = np.zeros((3, 4, 3, 5))
    nc, nb = np.zeros(3, np.int64), np.zeros(3, np.int64)
    for k in range(K):
        rc, _ = oracle.commit(bi.slice_tokens(pre, k * L, (k + 1) * L), pool, nc, nb,
                              slot_idx=slots, expected_block_index=k)
        assert rc == 0
    assert nc.tolist() == [K * L, 0, K * L] and nb.tolist() == [K, 0, K]
    s_k = oracle.scan_forward(pre, None)
    np.testing.assert_array_equal(pool[slots], s_k)
    _, yf, _, hfin = oracle.block_step(blk, pool, slot_idx=slots, parts=True, final_state=True)
    np.testing.assert_array_equal(yf, y_full[:, K * L:])
    np.testing.assert_array_equal(hfin, s_end)


def test_full_window_is_block_step_from_zero():
    _, d = rand_inputs(2, 11, 4, 3, 5, 2, seed=91)
    z = np.zeros((2, 4, 3, 5))
    y, yf, _ = oracle.block_step(d, z, parts=True)
    np.testing.assert_array_equal(oracle.full_window(d), y)
    _, yfw = oracle.scan_forward(d, None, want_y=True)
    np.testing.assert_array_equal(yf, yfw)


# ------------------------------------------------------------------------ bookkeeping
def test_commit_offset_and_slot_checks_leave_state_untouched():
    _, d = rand_inputs(2, 4, 4, 3, 5, 2, seed=95)
    pool = np.random.default_rng(96).standard_normal((3, 4, 3, 5))
    nc, nb = np.array([8, 4, 8], np.int64), np.array([2, 1, 2], np.int64)
    before = (pool.copy(), nc.copy(), nb.copy())
    rc, _ = oracle.commit(d, pool, nc, nb, slot_idx=[0, 1], expected_block_index=2)
    assert rc == oracle.ERR_OFFSET
    rc, _ = oracle.commit(d, pool, nc, nb, slot_idx=[2, 2], expected_block_index=-1)
    assert rc == oracle.ERR_SLOT
    rc, _ = oracle.commit(d, pool, nc, nb, slot_idx=[0, 3], expected_block_index=-1)
    assert rc == oracle.ERR_SLOT
    np.testing.assert_array_equal(pool, before[0])
    assert nc.tolist() == before[1].tolist() and nb.tolist() == before[2].tolist()
    rc, _ = oracle.commit(d, pool, nc, nb, slot_idx=[2, 0], expected_block_index=2)
    assert rc == 0
    assert nc.tolist() == [12, 4, 12] and nb.tolist() == [3, 1, 3]


def test_empty_batch_and_empty_block():
    _, d = rand_inputs(2, 0, 4, 3, 5, 2, seed=97)
    pool = np.random.default_rng(98).standard_normal((2, 4, 3, 5))
    y = oracle.block_step(d, pool)
    assert y.shape == (2, 0, 4, 3)
    keep = pool.copy()
    nc, nb = np.zeros(2, np.int64), np.zeros(2, np.int64)
    assert oracle.commit(d, pool, nc, nb)[0] == 0
    np.testing.assert_array_equal(pool, keep)      # zero tokens: state unchanged
    assert nc.tolist() == [0, 0] and nb.tolist() == [1, 1]


# ----------------------------------------------------------------- input encoding pins
def test_bf16_encoding():
    v = np.array([1.0, -2.0, 1.0078125, 1.00390625, 1.01171875, 3.0e-39, 65504.0], np.float32)
    bits = bi.to_bf16_bits(v)
    # 1.00390625 is halfway between 0x3F80 and 0x3F81 -> even (0x3F80); 1.01171875 is
    # halfway between 0x3F81 and 0x3F82 -> even (0x3F82)
    assert bits[:5].tolist() == [0x3F80, 0xC000, 0x3F81, 0x3F80, 0x3F82]
    np.testing.assert_array_equal(oracle.decode(bits), bi.bf16_bits_to_f32(bits))
    assert oracle.decode(np.array([0x3F80, 0x4049], np.uint16)).tolist() == [1.0, 3.140625]

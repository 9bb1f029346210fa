"""C ABI checks that need no GPU: the library loads, exports every function the
header declares, and every argument check returns its documented code before
anything is enqueued.  Device pointers here are fake (aligned integers): the
checks never dereference them, and no call in this file reaches a kernel launch.
"""
import ctypes

import numpy as np
import pytest

import paper_2607_02805_amd as bd

FAKE = 0x7F0000000000          # a 256-byte aligned fake device address
H, N, P = 4, 32, 64


@pytest.fixture(scope="module")
def L():
    return bd.lib()


def desc(batch=2, H=H, N=N, G=1, L=16, dtype=bd.DTYPE_BF16):
    d = bd.Desc()
    assert bd.lib().bdlm_desc_init(ctypes.byref(d), batch, H, P, N, G, L, dtype) == 0
    return d


def ptrs(**over):
    p = dict(x=FAKE, dt=FAKE + 0x1000, A=FAKE + 0x2000, B=FAKE + 0x3000, C=FAKE + 0x4000,
             D=FAKE + 0x5000, Drev=FAKE + 0x6000, h=FAKE + 0x7000, y=FAKE + 0x8000)
    p.update(over)
    return p


def i32p(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def i64p(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def check_step(L, d, p, nslots=4, slots=None):
    return L.bdlm_check_block_step(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                   p["D"], p["Drev"], p["h"], nslots, i32p(slots), p["y"])


def check_commit(L, d, p, nslots=4, slots=None, nc=None, nb=None, expect=-1):
    nc = np.zeros(nslots, np.int64) if nc is None else nc
    nb = np.zeros(nslots, np.int64) if nb is None else nb
    return L.bdlm_check_commit(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                               p["Drev"], p["h"], nslots, i32p(slots), i64p(nc), i64p(nb), expect)


def test_exports_every_declared_function(L):
    names = bd.header_functions()
    assert "bdlm_scan_block_step" in names and "bdlm_commit_boundary" in names
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/bdlm.h but not exported"
    assert L.bdlm_abi_version() == 1


def test_strerror(L):
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert bd.strerror(code) and bd.strerror(code) != "unknown status"
    assert bd.strerror(12345) == "unknown status"


def test_desc_init_contiguous_strides(L):
    d = desc(batch=3, H=8, N=64, G=2, L=32)
    assert list(d.x_stride) == [32 * 8 * 64, 8 * 64, 64]
    assert list(d.dt_stride) == [32 * 8, 8]
    assert list(d.bc_stride) == [32 * 2 * 64, 2 * 64, 64]
    assert L.bdlm_desc_init(None, 1, 1, 64, 16, 1, 1, 0) == bd.E_NULL


def test_valid_arguments_pass(L):
    assert check_step(L, desc(), ptrs()) == bd.OK
    assert check_step(L, desc(dtype=bd.DTYPE_F32), ptrs()) == bd.OK
    assert check_commit(L, desc(), ptrs()) == bd.OK
    for N_ in (16, 32, 64, 128):
        for L_ in (0, 1, 17, 32, 64):
            assert check_step(L, desc(N=N_, L=L_), ptrs()) == bd.OK


@pytest.mark.parametrize("field", ["x", "dt", "A", "B", "C", "D", "Drev", "h", "y"])
def test_null_pointers(L, field):
    assert check_step(L, desc(), ptrs(**{field: None})) == bd.E_NULL


def test_null_desc_and_meta(L):
    p = ptrs()
    assert L.bdlm_check_block_step(None, p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                                   p["Drev"], p["h"], 4, None, p["y"]) == bd.E_NULL
    d = desc()
    assert L.bdlm_check_commit(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                               p["Drev"], p["h"], 4, None, None, None, -1) == bd.E_NULL


@pytest.mark.parametrize("mut,code", [
    (dict(headdim=32), bd.E_SHAPE), (dict(dstate=48), bd.E_SHAPE), (dict(dstate=256), bd.E_SHAPE),
    (dict(block_len=2 ** 31), bd.E_SHAPE), (dict(block_len=-1), bd.E_SHAPE),
    (dict(nheads=6, ngroups=4), bd.E_SHAPE), (dict(ngroups=0), bd.E_SHAPE),
    (dict(nheads=0), bd.E_SHAPE), (dict(batch=-1), bd.E_SHAPE),
    (dict(in_dtype=7), bd.E_DTYPE), (dict(reserved=1), bd.E_DTYPE),
])
def test_bad_shapes_and_dtypes(L, mut, code):
    d = desc()
    for k, v in mut.items():
        setattr(d, k, v)
    assert check_step(L, d, ptrs()) == code


def test_negative_stride(L):
    d = desc()
    d.x_stride[1] = -64
    assert check_step(L, d, ptrs()) == bd.E_SHAPE


@pytest.mark.parametrize("over,dtype", [
    (dict(x=FAKE + 1), bd.DTYPE_BF16), (dict(x=FAKE + 8), bd.DTYPE_F32),
    (dict(B=FAKE + 0x3004), bd.DTYPE_BF16), (dict(C=FAKE + 0x4008), bd.DTYPE_F32),
    (dict(dt=FAKE + 0x1002), bd.DTYPE_F32), (dict(dt=FAKE + 0x1001), bd.DTYPE_BF16),
    (dict(h=FAKE + 0x7008), bd.DTYPE_BF16), (dict(A=FAKE + 0x2002), bd.DTYPE_BF16),
    (dict(y=FAKE + 0x8002), bd.DTYPE_BF16),
])
def test_misaligned(L, over, dtype):
    assert check_step(L, desc(dtype=dtype), ptrs(**over)) == bd.E_ALIGN


@pytest.mark.parametrize("which,i,v,dtype", [
    ("bc", 1, 36, bd.DTYPE_BF16), ("bc", 0, 1028, bd.DTYPE_BF16), ("bc", 2, 6, bd.DTYPE_F32),
    ("x", 1, 260, bd.DTYPE_BF16), ("x", 2, 66, bd.DTYPE_F32), ("x", 0, 2052, bd.DTYPE_BF16)])
def test_stride_alignment(L, which, i, v, dtype):
    d = desc(dtype=dtype)
    getattr(d, f"{which}_stride")[i] = v     # not a whole number of 16-byte units
    assert check_step(L, d, ptrs()) == bd.E_ALIGN
    getattr(d, f"{which}_stride")[i] = v + (16 // (2 if dtype == bd.DTYPE_BF16 else 4)) - \
        v % (16 // (2 if dtype == bd.DTYPE_BF16 else 4))
    assert check_step(L, d, ptrs()) == bd.OK


def test_slots(L):
    d = desc(batch=3)
    assert check_step(L, d, ptrs(), nslots=4, slots=np.array([3, 0, 3], np.int32)) == bd.OK
    assert check_step(L, d, ptrs(), nslots=4, slots=np.array([4, 0, 1], np.int32)) == bd.E_SLOT
    assert check_step(L, d, ptrs(), nslots=4, slots=np.array([-1, 0, 1], np.int32)) == bd.E_SLOT
    assert check_step(L, d, ptrs(), nslots=2) == bd.E_SLOT        # identity needs batch <= nslots
    assert check_step(L, d, ptrs(), nslots=0) == bd.E_SHAPE
    # slot tables longer than one launch's table are accepted (the call is split into
    # launches of MAX_SLOT_ROWS rows); duplicates anywhere in a commit's table are refused
    big = desc(batch=4 * bd.MAX_SLOT_ROWS + 7)
    slots = np.arange(4 * bd.MAX_SLOT_ROWS + 7, dtype=np.int32)[::-1].copy()
    assert check_step(L, big, ptrs(), nslots=len(slots), slots=slots) == bd.OK
    assert check_commit(L, big, ptrs(), nslots=len(slots), slots=slots) == bd.OK
    dup = slots.copy()
    dup[-1] = dup[3]
    assert check_step(L, big, ptrs(), nslots=len(slots), slots=dup) == bd.OK
    assert check_commit(L, big, ptrs(), nslots=len(slots), slots=dup) == bd.E_SLOT
    slots[600] = len(slots)
    assert check_step(L, big, ptrs(), nslots=len(slots), slots=slots) == bd.E_SLOT
    # repeated slots are fine for a step, not for a commit
    assert check_commit(L, d, ptrs(), slots=np.array([3, 0, 3], np.int32)) == bd.E_SLOT
    assert check_commit(L, d, ptrs(), slots=np.array([3, 0, 1], np.int32)) == bd.OK


def test_commit_offsets(L):
    d = desc(batch=2)
    nb = np.array([5, 5, 4, 5], np.int64)
    nc = nb * 16
    assert check_commit(L, d, ptrs(), nc=nc, nb=nb, expect=5) == bd.OK
    assert check_commit(L, d, ptrs(), nc=nc, nb=nb, expect=4) == bd.E_OFFSET
    assert check_commit(L, d, ptrs(), slots=np.array([2, 3], np.int32), nc=nc, nb=nb,
                        expect=5) == bd.E_OFFSET
    assert check_commit(L, d, ptrs(), slots=np.array([2, 3], np.int32), nc=nc, nb=nb,
                        expect=-1) == bd.OK


def test_entry_points_reject_before_launch(L):
    """The enqueueing entry points run the same checks first (no GPU is touched)."""
    d = desc()
    p = ptrs(x=None)
    assert L.bdlm_scan_block_step(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                  p["D"], p["Drev"], p["h"], 4, None, p["y"], None) == bd.E_NULL
    nc, nb = np.zeros(4, np.int64), np.array([1, 1, 1, 1], np.int64)
    p = ptrs()
    rc = L.bdlm_commit_boundary(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                                p["Drev"], p["h"], 4, None, i64p(nc), i64p(nb), 0, None, None)
    assert rc == bd.E_OFFSET
    assert nb.tolist() == [1, 1, 1, 1] and nc.tolist() == [0, 0, 0, 0]   # untouched
    rc = L.bdlm_commit_boundary(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                                p["Drev"], p["h"], 4, None, i64p(nc), i64p(nb), 1, FAKE + 1, None)
    assert rc == bd.E_ALIGN
    assert L.bdlm_cache_reset(None, 4, 1024, None, 0, None, None, None) == bd.E_NULL
    assert L.bdlm_cache_reset(FAKE, 4, 1022, None, 0, None, None, None) == bd.E_SHAPE
    assert L.bdlm_cache_reset(FAKE + 8, 4, 1024, None, 0, None, None, None) == bd.E_ALIGN
    bad = np.array([4], np.int32)
    assert L.bdlm_cache_reset(FAKE, 4, 1024, i32p(bad), 1, None, None, None) == bd.E_SLOT


WS = FAKE + 0x100000           # a 256-byte aligned fake workspace
BIG = 1 << 40                  # "large enough" workspace size


def ws_bytes(L, fn, d):
    n = ctypes.c_int64(-1)
    assert getattr(L, fn)(ctypes.byref(d), ctypes.byref(n)) == bd.OK
    return n.value


def check_window(L, d, p, ws=WS, wsb=BIG):
    return L.bdlm_check_full_window(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                    p["D"], p["Drev"], p["y"], ws, wsb)


def check_prefill(L, d, p, nslots=4, slots=None, nc=None, nb=None, expect=-1, blocks=0,
                  yf=None, ws=WS, wsb=BIG):
    nc = np.zeros(nslots, np.int64) if nc is None else nc
    nb = np.zeros(nslots, np.int64) if nb is None else nb
    return L.bdlm_check_prefill(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                                p["h"], nslots, i32p(slots), i64p(nc), i64p(nb), expect, blocks,
                                yf, ws, wsb)


def test_sequence_entry_points_accept_long_sequences(L):
    """The full window and the prefill take any length up to BDLM_MAX_SEQ_LEN; the
    block entry points stop at 64 tokens."""
    for T in (0, 1, 65, 4096, 65536, 2 ** 31 - 1):
        assert check_window(L, desc(L=T), ptrs()) == bd.OK
        assert check_prefill(L, desc(L=T), ptrs(), blocks=T // 32) == bd.OK
    assert check_window(L, desc(L=2 ** 31), ptrs()) == bd.E_SHAPE
    assert check_prefill(L, desc(L=2 ** 31), ptrs()) == bd.E_SHAPE
    # blocks longer than 64 run on the sequence kernels (the paper's block length 256)
    assert check_step(L, desc(L=65), ptrs()) == bd.OK
    assert check_step(L, desc(L=256), ptrs()) == bd.OK
    assert check_commit(L, desc(L=256), ptrs()) == bd.OK
    d = desc(L=256)
    d.x_stride[1] = (1 << 23) + 8                # too large a token stride for that path
    d.x_stride[0] = d.x_stride[1] * 256
    assert check_step(L, d, ptrs()) == bd.E_SHAPE
    d = desc(L=64)
    d.x_stride[1] = (1 << 23) + 8                # the fused block kernel has no such limit
    d.x_stride[0] = d.x_stride[1] * 64
    assert check_step(L, d, ptrs()) == bd.OK


def test_full_window_checks(L):
    assert check_window(L, desc(), ptrs(h=None)) == bd.OK          # no pool involved
    for field in ("x", "dt", "A", "B", "C", "D", "Drev", "y"):
        assert check_window(L, desc(), ptrs(**{field: None})) == bd.E_NULL
    assert check_window(L, desc(batch=0), ptrs(x=None, dt=None, B=None, C=None, y=None)) == bd.OK
    assert check_window(L, desc(), ptrs(y=FAKE + 0x8004)) == bd.OK   # y only 4-byte aligned
    assert check_window(L, desc(), ptrs(y=FAKE + 0x8002)) == bd.E_ALIGN
    assert check_window(L, desc(), ptrs(x=FAKE + 8)) == bd.E_ALIGN
    assert check_window(L, desc(N=48), ptrs()) == bd.E_SHAPE
    assert L.bdlm_check_full_window(None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                    FAKE, WS, BIG) == bd.E_NULL


def test_prefill_checks(L):
    d = desc(batch=3)
    slots = np.array([3, 0, 1], np.int32)
    nb = np.array([2, 2, 1, 2], np.int64)
    nc = nb * 32
    assert check_prefill(L, d, ptrs(Drev=None), slots=slots, nc=nc, nb=nb, expect=2) == bd.OK
    assert check_prefill(L, d, ptrs(), slots=slots, nc=nc, nb=nb, expect=1) == bd.E_OFFSET
    assert check_prefill(L, d, ptrs(), slots=np.array([3, 0, 3], np.int32)) == bd.E_SLOT
    assert check_prefill(L, d, ptrs(), slots=np.array([4, 0, 1], np.int32)) == bd.E_SLOT
    assert check_prefill(L, d, ptrs(), blocks=-1) == bd.E_SHAPE
    assert check_prefill(L, d, ptrs(h=None)) == bd.E_NULL
    assert check_prefill(L, d, ptrs(h=FAKE + 0x7008)) == bd.E_ALIGN
    assert L.bdlm_check_prefill(ctypes.byref(d), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4,
                                None, None, None, -1, 0, None, WS, BIG) == bd.E_NULL
    assert check_prefill(L, d, ptrs(), yf=FAKE + 0x9004) == bd.OK
    assert check_prefill(L, d, ptrs(), yf=FAKE + 0x9002) == bd.E_ALIGN


def test_row_limit(L):
    """batch * nheads is capped so that every launch grid fits 32 bits."""
    assert check_step(L, desc(batch=2 ** 20, H=4), ptrs(), nslots=2 ** 20) == bd.OK
    assert check_step(L, desc(batch=2 ** 20 + 1, H=4), ptrs(), nslots=2 ** 21) == bd.E_SHAPE
    assert check_window(L, desc(batch=2 ** 21, H=4), ptrs()) == bd.E_SHAPE
    assert check_window(L, desc(batch=2 ** 62, H=4), ptrs()) == bd.E_SHAPE   # no overflow


def test_sequence_entry_points_reject_before_launch(L):
    d = desc(batch=2, L=1000)
    p = ptrs(x=None)
    assert L.bdlm_scan_full_window(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                   p["D"], p["Drev"], p["y"], WS, BIG, None) == bd.E_NULL
    nc, nb = np.array([64, 64, 0, 0], np.int64), np.array([2, 2, 0, 0], np.int64)
    p = ptrs()
    rc = L.bdlm_prefill(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"], p["h"],
                        4, None, i64p(nc), i64p(nb), 3, 31, None, WS, BIG, None)
    assert rc == bd.E_OFFSET
    assert nc.tolist() == [64, 64, 0, 0] and nb.tolist() == [2, 2, 0, 0]   # untouched
    rc = L.bdlm_prefill(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"], p["h"],
                        4, None, i64p(nc), i64p(nb), 2, 31, FAKE + 2, WS, BIG, None)
    assert rc == bd.E_ALIGN
    rc = L.bdlm_prefill(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"], p["h"],
                        4, None, i64p(nc), i64p(nb), 2, 31, None, None, 0, None)
    assert rc == bd.E_WORKSPACE
    assert nc.tolist() == [64, 64, 0, 0] and nb.tolist() == [2, 2, 0, 0]


def test_workspace_sizes(L):
    """Segments of >= 256 tokens sized for ~2048 workgroups; per (row, head, segment)
    one state per direction plus one float, rounded up to 256 bytes."""
    d = desc(batch=4, H=32, N=128, L=65536)
    nseg = 16                                  # 128 (row, head) pairs -> 16 segments of 4096
    states = 4 * 32 * nseg * 64 * 128 * 4
    assert ws_bytes(L, "bdlm_full_window_workspace", d) == 2 * states + (4 * 32 * nseg * 4 + 255) // 256 * 256
    assert ws_bytes(L, "bdlm_prefill_workspace", d) == states + (4 * 32 * nseg * 4 + 255) // 256 * 256
    # a window that is one segment needs no workspace; a prefill always does
    d1 = desc(batch=2, H=3, N=16, L=200)
    assert ws_bytes(L, "bdlm_full_window_workspace", d1) == 0
    assert ws_bytes(L, "bdlm_prefill_workspace", d1) == 2 * 3 * 64 * 16 * 4 + 256
    assert ws_bytes(L, "bdlm_prefill_workspace", desc(batch=0, L=100)) == 0
    n = ctypes.c_int64(0)
    assert L.bdlm_full_window_workspace(ctypes.byref(desc(N=48)), ctypes.byref(n)) == bd.E_SHAPE
    assert L.bdlm_prefill_workspace(ctypes.byref(desc()), None) == bd.E_NULL


def test_workspace_checks(L):
    d = desc(batch=1, H=2, N=32, L=1000)        # several segments
    need = ws_bytes(L, "bdlm_full_window_workspace", d)
    assert need > 0
    assert check_window(L, d, ptrs(), WS, need) == bd.OK
    assert check_window(L, d, ptrs(), WS, need - 1) == bd.E_WORKSPACE
    assert check_window(L, d, ptrs(), None, need) == bd.E_WORKSPACE
    assert check_window(L, d, ptrs(), WS + 16, need) == bd.E_ALIGN
    assert check_window(L, d, ptrs(), WS, -1) == bd.E_SHAPE
    d1 = desc(batch=2, H=3, N=16, L=200)        # one segment: no workspace needed
    assert check_window(L, d1, ptrs(), None, 0) == bd.OK
    needp = ws_bytes(L, "bdlm_prefill_workspace", d)
    assert check_prefill(L, d, ptrs(), ws=WS, wsb=needp) == bd.OK
    assert check_prefill(L, d, ptrs(), ws=WS, wsb=needp - 4) == bd.E_WORKSPACE
    assert bd.strerror(bd.E_WORKSPACE) != "unknown status"


def test_sequence_stride_limit(L):
    """Chunks are addressed with 32-bit offsets: per-token strides up to 16 MiB."""
    d = desc(batch=1, H=4, L=1000)
    d.x_stride[1] = (1 << 23)                   # bf16: 16 MiB per token
    d.x_stride[0] = d.x_stride[1] * 1000
    assert check_window(L, d, ptrs()) == bd.OK
    d.x_stride[1] = (1 << 23) + 8
    assert check_window(L, d, ptrs()) == bd.E_SHAPE
    assert check_prefill(L, d, ptrs()) == bd.E_SHAPE
    assert check_step(L, desc(), ptrs()) == bd.OK   # the block entry points are not limited


def check_bstates(L, d, K=4, p=None, s_init=FAKE + 0xA000, s_out=FAKE + 0xB000, yf=None,
                  ws=WS, wsb=BIG):
    p = ptrs() if p is None else p
    return L.bdlm_check_block_boundary_states(ctypes.byref(d), K, p["x"], p["dt"], p["A"], p["B"],
                                              p["C"], p["D"], s_init, s_out, yf, ws, wsb)


def test_boundary_states_checks(L):
    d = desc(batch=2, H=4, N=32, L=32)
    assert check_bstates(L, d) == bd.OK
    assert check_bstates(L, d, s_init=None) == bd.OK                  # zero initial states
    assert check_bstates(L, d, p=ptrs(C=None)) == bd.OK               # C only for y_fwd
    assert check_bstates(L, d, p=ptrs(C=None), yf=FAKE + 0xC000) == bd.E_NULL
    assert check_bstates(L, d, K=-1) == bd.E_SHAPE
    assert check_bstates(L, d, s_out=None) == bd.E_NULL
    assert check_bstates(L, d, s_out=FAKE + 0xB008) == bd.E_ALIGN
    assert check_bstates(L, d, s_init=FAKE + 0xA004) == bd.E_ALIGN
    assert check_bstates(L, desc(L=65)) == bd.E_SHAPE                 # blocks of at most 64
    assert check_bstates(L, d, K=(2 ** 31) // 32 + 1) == bd.E_SHAPE   # sequence too long
    assert check_bstates(L, desc(batch=1 << 10, H=1 << 10), K=2 ** 11) == bd.E_SHAPE   # grid
    assert ws_bytes_b(L, d, 4) == 0                                   # one segment
    assert check_bstates(L, d, ws=None, wsb=0) == bd.OK
    # 4096 blocks of 32 tokens over 8 (row, head) units: 512 segments of 8 blocks, each
    # with a 64 x 32 fp32 state and a log-decay
    need = ws_bytes_b(L, d, 4096)
    assert need == 8 * 512 * 64 * 32 * 4 + (8 * 512 * 4 + 255) // 256 * 256
    d = desc(batch=2, H=4, N=32, L=32)
    assert check_bstates(L, d, K=4096, ws=WS, wsb=need) == bd.OK
    assert check_bstates(L, d, K=4096, ws=WS, wsb=need - 4) == bd.E_WORKSPACE
    assert check_bstates(L, d, K=4096, ws=None, wsb=need) == bd.E_WORKSPACE
    assert check_bstates(L, d, K=0, ws=None, wsb=0) == bd.OK          # empty: nothing to do
    assert L.bdlm_block_boundary_states(None, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                        FAKE, None, WS, BIG, None) == bd.E_NULL


def ws_bytes_b(L, d, K):
    n = ctypes.c_int64(-1)
    assert L.bdlm_boundary_states_workspace(ctypes.byref(d), K, ctypes.byref(n)) == bd.OK
    return n.value


def check_sep(L, d, p=None, q=None, slots=None, nslots=4):
    p = ptrs() if p is None else p
    q = ptrs(x=FAKE + 0x20000, dt=FAKE + 0x21000, A=FAKE + 0x22000, B=FAKE + 0x23000,
             C=FAKE + 0x24000, D=FAKE + 0x25000) if q is None else q
    return L.bdlm_check_block_step_sep(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                       p["D"], q["x"], q["dt"], q["A"], q["B"], q["C"], q["D"],
                                       p["h"], nslots, i32p(slots), p["y"])


def test_block_step_sep_checks(L):
    d = desc(batch=2, L=32)
    assert check_sep(L, d) == bd.OK
    assert check_sep(L, desc(batch=2, L=256)) == bd.OK
    for field in ("x", "dt", "A", "B", "C", "D"):
        q = ptrs(x=FAKE + 0x20000, dt=FAKE + 0x21000, A=FAKE + 0x22000, B=FAKE + 0x23000,
                 C=FAKE + 0x24000, D=FAKE + 0x25000)
        q[field] = None
        assert check_sep(L, d, q=q) == bd.E_NULL, field
    q = ptrs(x=FAKE + 0x20008)
    assert check_sep(L, d, q=q) == bd.E_ALIGN
    assert check_sep(L, d, p=ptrs(h=None)) == bd.E_NULL
    assert check_sep(L, d, slots=np.array([5, 0], np.int32)) == bd.E_SLOT


def test_conv_entry_point_checks(L):
    d = desc(batch=2, H=4, N=32, L=32)
    ch = 4 * 64 + 2 * 32
    n = ctypes.c_int64(-1)
    assert L.bdlm_conv_workspace(ctypes.byref(d), ctypes.byref(n)) == bd.OK
    assert n.value == (2 * 32 * (2 * 256 + 4 * 32 + 4) * 4 + 255) // 256 * 256
    p = ptrs()
    cw, cb, cp = FAKE + 0x30000, FAKE + 0x31000, FAKE + 0x32000

    def step(cw=cw, cb=cb, cp=cp, ws=WS, wsb=BIG):
        return L.bdlm_check_conv_block_step(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"],
                                            p["C"], p["D"], p["Drev"], cw, cb, cp, p["h"], 4,
                                            None, p["y"], ws, wsb)
    assert step() == bd.OK
    assert step(cw=None) == bd.E_NULL and step(cb=None) == bd.E_NULL and step(cp=None) == bd.E_NULL
    assert step(cw=cw + 8) == bd.E_ALIGN
    # biases and cached rows are read as 16-byte vectors too
    assert step(cb=cb + 4) == bd.E_ALIGN and step(cb=cb + 8) == bd.E_ALIGN
    assert step(cp=cp + 4) == bd.E_ALIGN and step(cp=cp + 8) == bd.E_ALIGN
    assert step(wsb=n.value - 4) == bd.E_WORKSPACE
    nc, nb = np.zeros(4, np.int64), np.array([1, 1, 2, 2], np.int64)
    rc = L.bdlm_check_conv_commit(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                                  p["Drev"], cw, cb, cp, p["h"], 4, None, i64p(nc), i64p(nb), 1,
                                  None, WS, BIG)
    assert rc == bd.OK
    rc = L.bdlm_check_conv_commit(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"], p["D"],
                                  p["Drev"], cw, cb, cp, p["h"], 4, i32p(np.array([1, 1], np.int32)),
                                  i64p(nc), i64p(nb), -1, None, WS, BIG)
    assert rc == bd.E_SLOT


def check_norm(L, batch=2, ln=8, H=4, G=1, zdt=bd.DTYPE_BF16, y=FAKE, z=FAKE + 0x100000,
               zsb=None, zst=None, w=FAKE + 0x200000, eps=1e-5, out=FAKE + 0x300000):
    zst = H * 64 if zst is None else zst
    zsb = ln * zst if zsb is None else zsb
    return L.bdlm_check_gated_rmsnorm(batch, ln, H, G, zdt, y, z, zsb, zst, w, eps, out)


def test_gated_rmsnorm_checks(L):
    assert check_norm(L) == bd.OK
    assert check_norm(L, zdt=bd.DTYPE_F32) == bd.OK
    assert check_norm(L, out=FAKE) == bd.OK                          # in place
    assert check_norm(L, H=6, G=3) == bd.OK
    assert check_norm(L, H=256) == bd.OK
    assert check_norm(L, H=257) == bd.E_SHAPE                        # too many channels
    assert check_norm(L, H=0) == bd.E_SHAPE
    assert check_norm(L, H=6, G=4) == bd.E_SHAPE                     # groups of whole heads
    assert check_norm(L, zdt=7) == bd.E_DTYPE
    assert check_norm(L, eps=-1.0) == bd.E_SHAPE
    assert check_norm(L, eps=float("nan")) == bd.E_SHAPE
    assert check_norm(L, eps=float("inf")) == bd.E_SHAPE
    assert check_norm(L, batch=-1) == bd.E_SHAPE
    assert check_norm(L, zst=-256) == bd.E_SHAPE
    assert check_norm(L, y=None) == bd.E_NULL
    assert check_norm(L, z=None) == bd.E_NULL
    assert check_norm(L, w=None) == bd.E_NULL
    assert check_norm(L, out=None) == bd.E_NULL
    assert check_norm(L, batch=0, y=None, z=None, out=None) == bd.OK  # empty: nothing read
    assert check_norm(L, y=FAKE + 8) == bd.E_ALIGN
    assert check_norm(L, out=FAKE + 0x300008) == bd.E_ALIGN
    assert check_norm(L, w=FAKE + 0x200004) == bd.E_ALIGN
    assert check_norm(L, z=FAKE + 0x100008) == bd.OK                 # bf16: 8-byte quads
    assert check_norm(L, zdt=bd.DTYPE_F32, z=FAKE + 0x100008) == bd.E_ALIGN
    assert check_norm(L, zst=258) == bd.E_ALIGN                      # strides in quads
    # y spans 2 * 8 * 256 * 4 = 16 KiB: out partly over y, or over z / w
    assert check_norm(L, out=FAKE + 0x1000) == bd.E_SHAPE
    assert check_norm(L, out=FAKE + 0x100000 - 0x1000) == bd.E_SHAPE
    assert check_norm(L, out=FAKE + 0x200000) == bd.E_SHAPE
    assert check_norm(L, out=FAKE + 0x100000 - 0x4000) == bd.OK      # ends where z starts


# ----------------------------------------------------------------- binding checks
# The binding refuses mis-shaped tensors and slot lists before it takes any device
# pointer, so CPU tensors reach these checks (a well-formed CPU call would instead be
# refused for not being on the GPU).
def _blk(batch=2, Lb=16, H=H, N=N, dtype=None):
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    f32 = torch.float32
    return dict(x=torch.zeros(batch, Lb, H, 64, dtype=dtype), dt=torch.zeros(batch, Lb, H, dtype=dtype),
                A=torch.zeros(H, dtype=f32), B=torch.zeros(batch, Lb, 1, N, dtype=dtype),
                C=torch.zeros(batch, Lb, 1, N, dtype=dtype), D=torch.zeros(H, dtype=f32),
                D_rev=torch.zeros(H, dtype=f32))


def _args(v):
    return v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"], v["D_rev"]


@pytest.mark.parametrize("shape", [(2, 16, H, 32), (1, 16, H, 64), (2, 15, H, 64), (2, 16, H * 64)])
def test_binding_rejects_misshaped_outputs(shape):
    import torch
    v = _blk()
    pool = torch.zeros(bd.pool_shape(4, H, N))
    bad = torch.zeros(shape)
    nc, nb = np.zeros(4, np.int64), np.zeros(4, np.int64)
    cw, cb = torch.zeros(bd.conv_channels(H, 1, N), 4), torch.zeros(bd.conv_channels(H, 1, N))
    cpool = torch.zeros(4, 3, bd.conv_channels(H, 1, N))
    calls = {
        "step": lambda: bd.scan_block_step(*_args(v), pool, y=bad),
        "sep": lambda: bd.scan_block_step_sep(_args(v)[:6], _args(v)[:5] + (v["D_rev"],), pool,
                                              y=bad),
        "commit": lambda: bd.commit_boundary(*_args(v), pool, nc, nb, y_clean=bad),
        "conv_step": lambda: bd.conv_block_step(*_args(v), cw, cb, cpool, pool, y=bad),
        "conv_commit": lambda: bd.conv_commit_boundary(*_args(v), cw, cb, cpool, pool, nc, nb,
                                                       y_clean=bad),
        "full_window": lambda: bd.scan_full_window(*_args(v), y=bad),
        "prefill": lambda: bd.prefill(*_args(v)[:6], pool, nc, nb, y_fwd=bad),
        "boundary": lambda: bd.block_boundary_states(*_args(v)[:6], 16, y_fwd=bad),
    }
    for name, fn in calls.items():
        with pytest.raises(ValueError, match="float32 tensor of shape"):
            fn()
    # wrong dtype or a non-contiguous view of the right shape are refused too
    with pytest.raises(ValueError, match="float32 tensor of shape"):
        bd.scan_block_step(*_args(v), pool, y=torch.zeros(2, 16, H, 64, dtype=torch.float64))
    with pytest.raises(ValueError, match="float32 tensor of shape"):
        bd.scan_block_step(*_args(v), pool, y=torch.zeros(2, 16, 64, H).transpose(2, 3))


@pytest.mark.parametrize("field", ["x", "dt", "A", "B", "C", "D"])
def test_binding_sep_rejects_reverse_shape_mismatch(field):
    import torch
    v = _blk(batch=2)
    small = _blk(batch=1)
    fwd = (v["x"], v["dt"], v["A"], v["B"], v["C"], v["D"])
    rev = dict(zip(("x", "dt", "A", "B", "C", "D"), fwd))
    if field in ("A", "D"):
        rev[field] = torch.zeros(H + 1)
    else:
        rev[field] = small[field]
    pool = torch.zeros(bd.pool_shape(4, H, N))
    with pytest.raises(ValueError, match="same shape"):
        bd.scan_block_step_sep(fwd, tuple(rev[k] for k in ("x", "dt", "A", "B", "C", "D")), pool)


@pytest.mark.parametrize("slots", [[0], [0, 1, 2], [[0, 1]], np.zeros((2, 1), np.int32)])
def test_binding_rejects_slot_list_of_wrong_length(slots):
    import torch
    v = _blk(batch=2)
    pool = torch.zeros(bd.pool_shape(4, H, N))
    nc, nb = np.zeros(4, np.int64), np.zeros(4, np.int64)
    with pytest.raises(ValueError, match="exactly 2 slot indices"):
        bd.scan_block_step(*_args(v), pool, slot_idx=slots)
    with pytest.raises(ValueError, match="exactly 2 slot indices"):
        bd.commit_boundary(*_args(v), pool, nc, nb, slot_idx=slots)
    with pytest.raises(ValueError, match="exactly 2 slot indices"):
        bd.prefill(*_args(v)[:6], pool, nc, nb, slot_idx=slots)


def test_noalloc_prefill_host_refusals(L):
    """bdlm_prefill_noalloc's checks run before it touches the device: argument errors and
    a request its scratch cannot hold are refused without a GPU, bookkeeping untouched."""
    i64 = ctypes.POINTER(ctypes.c_int64)
    nc, nb = np.zeros(4, np.int64), np.zeros(4, np.int64)

    def call(d, p, nslots=4, expect=-1):
        return L.bdlm_prefill_noalloc(ctypes.byref(d), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                      p["D"], p["h"], nslots, None, nc.ctypes.data_as(i64),
                                      nb.ctypes.data_as(i64), expect, 0, None, None)
    assert call(desc(batch=2, L=300), ptrs(x=None)) == bd.E_NULL
    assert call(desc(batch=2, L=300), ptrs(B=FAKE + 0x3008)) == bd.E_ALIGN
    nb[:] = 1
    assert call(desc(batch=2, L=300), ptrs(), expect=0) == bd.E_OFFSET
    # 80 rows x 32 heads x 64 x 128 fp32 = 80 MiB of segment states even as one segment
    big = desc(batch=80, H=32, N=128, L=256)
    assert call(big, ptrs(), nslots=80) == bd.E_WORKSPACE
    assert nb.tolist() == [1, 1, 1, 1] and nc.tolist() == [0] * 4
    # nothing to do: succeeds without a device
    assert call(desc(batch=0, L=300), ptrs(x=None, dt=None, B=None, C=None)) == bd.OK


def test_commit_step_checks(L):
    d = desc(batch=2, L=32)
    p = ptrs()
    q = dict(x=FAKE + 0x40000, dt=FAKE + 0x41000, B=FAKE + 0x42000, C=FAKE + 0x43000)
    yn = FAKE + 0x50000

    def chk(p=p, q=q, yn=yn, yc=None, slots=None, nb=None, expect=-1, dd=d):
        nc = np.zeros(4, np.int64)
        nb = np.zeros(4, np.int64) if nb is None else nb
        return L.bdlm_check_commit_step(ctypes.byref(dd), p["x"], p["dt"], p["A"], p["B"], p["C"],
                                        p["D"], p["Drev"], q["x"], q["dt"], q["B"], q["C"], p["h"],
                                        4, i32p(slots), i64p(nc), i64p(nb), expect, yc, yn)
    assert chk() == bd.OK
    assert chk(yc=FAKE + 0x60000) == bd.OK
    for f in ("x", "dt", "B", "C"):
        assert chk(q=dict(q, **{f: None})) == bd.E_NULL, f
    assert chk(yn=None) == bd.E_NULL
    assert chk(yn=FAKE + 0x50008) == bd.E_ALIGN
    assert chk(yc=FAKE + 0x60004) == bd.E_ALIGN
    assert chk(q=dict(q, B=FAKE + 0x42008)) == bd.E_ALIGN
    assert chk(slots=np.array([1, 1], np.int32)) == bd.E_SLOT          # a commit: distinct
    assert chk(nb=np.array([3, 3, 0, 0], np.int64), expect=3) == bd.OK
    assert chk(nb=np.array([3, 2, 0, 0], np.int64), expect=3) == bd.E_OFFSET
    assert chk(dd=desc(batch=2, L=65)) == bd.E_SHAPE                   # up to 64 tokens


def test_binding_fails_loudly_without_the_library(monkeypatch, tmp_path):
    """With the HIP library absent the binding raises instead of computing anything (there
    is no CPU path)."""
    import paper_2607_02805_amd as bd
    monkeypatch.setattr(bd, "_lib", None)
    monkeypatch.setattr(bd, "LIB_PATH", str(tmp_path / "libbdlm.so"))
    with pytest.raises(RuntimeError, match="missing"):
        bd.lib()

"""fp64 CPU oracle for the block-restricted bidirectional Mamba scan.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The HIP library in
``paper_2607_02805_amd`` never imports it, and it imports nothing from there.

The arithmetic lives in ``bdlm_oracle.c`` (plain loops, fp64); this module only
builds it with gcc and marshals numpy arrays through ctypes.  The passages each
C function follows are cited in that file:

* ``block_step``   -- Sec. 4, Eq. partial-reverse (forward scan continued from the
  cached boundary state, block-local reverse scan from zero, summed), built on the
  selective update of Sec. 3, Eq. mamba-scan-background.
* ``commit``       -- Sec. 4, Eq. boundary-state, and the cache-append step of the
  BDLM sampler (Sec. 3; Sec. 4.1): the clean block's forward state becomes the cache.
* ``scan_forward`` -- Eq. boundary-state: a clean prefix summarised by the forward scan.
* ``full_window``  -- the full-sequence bidirectional (DiffuMamba-style) scan the paper
  contrasts against (Sec. 4; Sec. 5.1).
* ``conv``         -- the convolution part of the Mamba boundary state (Sec. 2, Sec. 4;
  App. C: width 4): forward continued from the cached last three input rows, reverse
  zero-padded inside the block, SiLU; a commit keeps the last three rows.
* ``gated_rmsnorm`` -- the gated RMS normalisation after the scan in the Mamba-2 mixers
  the paper uses (App. C): y * silu(z), normalised over channel groups, scaled by w.

Inputs are the exact stored bytes the GPU reads: activations as fp32 or bf16
(numpy ``uint16`` holding the bf16 bit pattern), ``A``/``D``/``D_rev`` fp32.
States and outputs are float64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bdlm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_bdlm.so")

DTYPE_F32 = 0
DTYPE_BF16 = 1
DTYPE_F64 = 2      # already-decoded values (e.g. convolution outputs)

OK = 0
ERR_ARG = -1
ERR_OFFSET = -2
ERR_SLOT = -3


class _Shape(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int64),
        ("nheads", ctypes.c_int64),
        ("headdim", ctypes.c_int64),
        ("dstate", ctypes.c_int64),
        ("ngroups", ctypes.c_int64),
        ("len", ctypes.c_int64),
        ("in_dtype", ctypes.c_int32),
    ]


def build() -> str:
    """Compile the oracle with gcc (always recompiles)."""
    tmp = _LIB + ".tmp"
    cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-Wall", "-Wextra",
           "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    """Load the compiled oracle, building it only if nothing is built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        vp, dp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)
        fp = ctypes.POINTER(ctypes.c_float)
        i32p, i64p = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64)
        sp = ctypes.POINTER(_Shape)
        L.bdlm_oracle_block_step.argtypes = [sp, vp, vp, fp, vp, vp, fp, fp, dp, ctypes.c_int64,
                                             i32p, dp, dp, dp, dp]
        L.bdlm_oracle_commit.argtypes = [sp, vp, vp, fp, vp, vp, fp, fp, dp, ctypes.c_int64, i32p,
                                         i64p, i64p, ctypes.c_int64, dp]
        L.bdlm_oracle_scan_forward.argtypes = [sp, vp, vp, fp, vp, vp, fp, dp, dp]
        L.bdlm_oracle_full_window.argtypes = [sp, vp, vp, fp, vp, vp, fp, fp, dp]
        for f in ("bdlm_oracle_block_step", "bdlm_oracle_commit", "bdlm_oracle_scan_forward",
                  "bdlm_oracle_full_window", "bdlm_oracle_num_threads"):
            getattr(L, f).restype = ctypes.c_int
        L.bdlm_oracle_set_num_threads.argtypes = [ctypes.c_int]
        L.bdlm_oracle_set_num_threads.restype = None
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().bdlm_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Thread count of the oracle's loops over (batch, head) (timing only)."""
    lib().bdlm_oracle_set_num_threads(ctypes.c_int(int(n)))


# ---------------------------------------------------------------- marshalling
def _act(a: np.ndarray) -> tuple[np.ndarray, int]:
    if a.dtype == np.uint16:
        return np.ascontiguousarray(a), DTYPE_BF16
    if a.dtype == np.float32:
        return np.ascontiguousarray(a), DTYPE_F32
    if a.dtype == np.float64:
        return np.ascontiguousarray(a), DTYPE_F64
    raise TypeError(f"activation dtype must be float32, float64 or uint16 (bf16 bits), got {a.dtype}")


def _shape(inp: dict) -> tuple[_Shape, dict]:
    x, dty = _act(inp["x"])
    dt, d2 = _act(inp["dt"])
    Bm, d3 = _act(inp["B"])
    Cm, d4 = _act(inp["C"])
    if len({dty, d2, d3, d4}) != 1:
        raise TypeError("x, dt, B and C must share one storage dtype")
    bsz, L, H, P = x.shape
    _, _, G, N = Bm.shape
    if dt.shape != (bsz, L, H) or Bm.shape != (bsz, L, G, N) or Cm.shape != Bm.shape:
        raise ValueError("inconsistent activation shapes")
    arrs = dict(
        x=x, dt=dt, B=Bm, C=Cm,
        A=np.ascontiguousarray(inp["A"], dtype=np.float32),
        D=np.ascontiguousarray(inp["D"], dtype=np.float32),
        D_rev=np.ascontiguousarray(inp.get("D_rev", inp["D"]), dtype=np.float32),
    )
    return _Shape(bsz, H, P, N, G, L, dty), arrs


def _p(a, ct):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ct))


def _v(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def block_step(inp: dict, h_pool: np.ndarray, slot_idx=None, parts: bool = False,
               final_state: bool = False):
    """Active-block step.  ``h_pool`` is float64 [nslots, H, P, N] (read only).

    Returns ``y`` float64 [B, L, H, P]; with ``parts`` also ``(y_fwd, y_rev)``;
    with ``final_state`` also the forward state after the block, [B, H, P, N].
    """
    s, a = _shape(inp)
    h_pool = np.ascontiguousarray(h_pool, dtype=np.float64)
    y = np.zeros(a["x"].shape, np.float64)
    yf = np.zeros_like(y) if parts else None
    yr = np.zeros_like(y) if parts else None
    hout = np.zeros((s.batch, s.nheads, s.headdim, s.dstate)) if final_state else None
    si = None if slot_idx is None else np.ascontiguousarray(slot_idx, dtype=np.int32)
    rc = lib().bdlm_oracle_block_step(
        ctypes.byref(s), _v(a["x"]), _v(a["dt"]), _p(a["A"], ctypes.c_float), _v(a["B"]),
        _v(a["C"]), _p(a["D"], ctypes.c_float), _p(a["D_rev"], ctypes.c_float),
        _p(h_pool, ctypes.c_double), h_pool.shape[0], _p(si, ctypes.c_int32),
        _p(y, ctypes.c_double), _p(yf, ctypes.c_double), _p(yr, ctypes.c_double),
        _p(hout, ctypes.c_double))
    if rc != OK:
        raise ValueError(f"oracle block_step failed: {rc}")
    out = [y]
    if parts:
        out += [yf, yr]
    if final_state:
        out.append(hout)
    return out[0] if len(out) == 1 else tuple(out)


def commit(inp: dict, h_pool: np.ndarray, n_committed: np.ndarray, n_blocks: np.ndarray,
           slot_idx=None, expected_block_index: int = -1, want_y: bool = True):
    """Block finalisation, in place on ``h_pool`` (float64) and the int64 bookkeeping.

    Returns ``(rc, y_clean)``; ``rc`` is 0 or a negative oracle error code and on
    error nothing is modified.
    """
    s, a = _shape(inp)
    for arr, dt in ((h_pool, np.float64), (n_committed, np.int64), (n_blocks, np.int64)):
        if arr.dtype != dt or not arr.flags.c_contiguous:
            raise TypeError("h_pool / n_committed / n_blocks must be contiguous float64/int64")
    yc = np.zeros(a["x"].shape, np.float64) if want_y else None
    si = None if slot_idx is None else np.ascontiguousarray(slot_idx, dtype=np.int32)
    rc = lib().bdlm_oracle_commit(
        ctypes.byref(s), _v(a["x"]), _v(a["dt"]), _p(a["A"], ctypes.c_float), _v(a["B"]),
        _v(a["C"]), _p(a["D"], ctypes.c_float), _p(a["D_rev"], ctypes.c_float),
        _p(h_pool, ctypes.c_double), h_pool.shape[0], _p(si, ctypes.c_int32),
        _p(n_committed, ctypes.c_int64), _p(n_blocks, ctypes.c_int64),
        int(expected_block_index), _p(yc, ctypes.c_double))
    return rc, yc


def scan_forward(inp: dict, h: np.ndarray | None = None, want_y: bool = False):
    """Forward scan over the whole sequence in ``inp`` from state ``h`` (zero if None).

    Returns the final state float64 [B, H, P, N] (and the forward outputs if asked).
    """
    s, a = _shape(inp)
    if h is None:
        h = np.zeros((s.batch, s.nheads, s.headdim, s.dstate))
    h = np.array(h, dtype=np.float64, copy=True, order="C")
    y = np.zeros(a["x"].shape, np.float64) if want_y else None
    rc = lib().bdlm_oracle_scan_forward(
        ctypes.byref(s), _v(a["x"]), _v(a["dt"]), _p(a["A"], ctypes.c_float), _v(a["B"]),
        _v(a["C"]), _p(a["D"], ctypes.c_float), _p(h, ctypes.c_double), _p(y, ctypes.c_double))
    if rc != OK:
        raise ValueError(f"oracle scan_forward failed: {rc}")
    return (h, y) if want_y else h


def full_window(inp: dict) -> np.ndarray:
    """Full-window forward + reverse scan, both from zero (no cache)."""
    s, a = _shape(inp)
    y = np.zeros(a["x"].shape, np.float64)
    rc = lib().bdlm_oracle_full_window(
        ctypes.byref(s), _v(a["x"]), _v(a["dt"]), _p(a["A"], ctypes.c_float), _v(a["B"]),
        _v(a["C"]), _p(a["D"], ctypes.c_float), _p(a["D_rev"], ctypes.c_float),
        _p(y, ctypes.c_double))
    if rc != OK:
        raise ValueError(f"oracle full_window failed: {rc}")
    return y


def decode(a: np.ndarray) -> np.ndarray:
    """Stored activation bytes -> float64 (bf16 bit patterns widened exactly)."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def conv(inp: dict, w: np.ndarray, bias: np.ndarray, cache: np.ndarray, slot_idx=None,
         commit: bool = False):
    """Width-4 depthwise causal convolution + SiLU over the x, B, C channels of a block
    (``inp`` holds the pre-convolution x, B, C; channels x head-major, then B, then C).

    ``w`` fp32 [channels, 4] (``w[:, 3]`` multiplies the current token), ``bias`` fp32
    [channels], ``cache`` float64 [nslots, 3, channels] (row 0 the oldest input).
    Returns ``(fwd, rev)``: dicts of float64 x, B, C -- the forward branch continues from
    the cached rows, the reverse branch is zero-padded past the block end.  With
    ``commit`` the cache rows become the last three rows of (cache rows ++ block).
    """
    x, dty = _act(inp["x"])
    Bm, d2 = _act(inp["B"])
    Cm, d3 = _act(inp["C"])
    if len({dty, d2, d3}) != 1:
        raise TypeError("x, B and C must share one storage dtype")
    bsz, L, H, P = x.shape
    _, _, G, N = Bm.shape
    s = _Shape(bsz, H, P, N, G, L, dty)
    ch = H * P + 2 * G * N
    w = np.ascontiguousarray(w, dtype=np.float32)
    bias = np.ascontiguousarray(bias, dtype=np.float32)
    if w.shape != (ch, 4) or bias.shape != (ch,) or cache.dtype != np.float64 \
            or not cache.flags.c_contiguous or cache.shape[1:] != (3, ch):
        raise ValueError("conv weights [channels, 4], bias [channels], cache float64 [n, 3, channels]")
    out = [np.zeros(a.shape, np.float64) for a in (x, Bm, Cm, x, Bm, Cm)]
    si = None if slot_idx is None else np.ascontiguousarray(slot_idx, dtype=np.int32)
    L_ = lib()
    L_.bdlm_oracle_conv.restype = ctypes.c_int
    rc = L_.bdlm_oracle_conv(ctypes.byref(s), _v(x), _v(Bm), _v(Cm), _p(w, ctypes.c_float),
                             _p(bias, ctypes.c_float), _p(cache, ctypes.c_double),
                             ctypes.c_int64(cache.shape[0]), _p(si, ctypes.c_int32),
                             ctypes.c_int(1 if commit else 0),
                             *[_p(o, ctypes.c_double) for o in out])
    if rc != OK:
        raise ValueError(f"oracle conv failed: {rc}")
    return dict(x=out[0], B=out[1], C=out[2]), dict(x=out[3], B=out[4], C=out[5])



def gated_rmsnorm(y: np.ndarray, z: np.ndarray, w: np.ndarray, eps: float,
                  ngroups: int = 1) -> np.ndarray:
    """Gated RMS normalisation over the channels of each token.

    ``y`` float [..., nch] (any float dtype; taken as float64), ``z`` stored bytes
    [..., nch] (fp32, or bf16 bits as uint16), ``w`` fp32 [nch]; the channels split into
    ``ngroups`` groups of consecutive channels.  Returns float64 of ``y``'s shape.
    """
    y = np.ascontiguousarray(y, dtype=np.float64)
    z, zdt = _act(z)
    w = np.ascontiguousarray(w, dtype=np.float32)
    nch = y.shape[-1]
    if z.shape != y.shape or w.shape != (nch,):
        raise ValueError("y and z share a shape; w is [channels]")
    ntok = y.size // nch if nch else 0
    out = np.zeros(y.shape, np.float64)
    L_ = lib()
    L_.bdlm_oracle_gated_rmsnorm.restype = ctypes.c_int
    rc = L_.bdlm_oracle_gated_rmsnorm(ctypes.c_int64(ntok), ctypes.c_int64(nch),
                                      ctypes.c_int64(ngroups), _p(y, ctypes.c_double), _v(z),
                                      ctypes.c_int(zdt), _p(w, ctypes.c_float),
                                      ctypes.c_double(eps), _p(out, ctypes.c_double))
    if rc != OK:
        raise ValueError(f"oracle gated_rmsnorm failed: {rc}")
    return out

"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This module draws random numbers and encodes them; it holds none of the scan's
arithmetic.  Both the CPU oracle and the HIP library consume the exact bytes it
returns (fp32, or bf16 bit patterns stored as ``uint16``).

Value distributions (per the workload recipe; the paper's own throughput runs
use random-initialised models and synthetic batches, Sec. 5.3):

* ``x  ~ N(0, 1)``                              [batch, len, nheads, headdim]
* ``dt = softplus(0.5 * N(0, 1) - 4.6)``        [batch, len, nheads]
* ``A_h = -exp(U(0, ln 16))``                   [nheads]   (fp32, always)
* ``B, C ~ N(0, 1) / sqrt(dstate)``             [batch, len, ngroups, dstate]
* ``D ~ N(0, 1)``, ``D_rev = D``                [nheads]   (fp32, always)
* gate ``z ~ N(0, 1)``                          [batch, len, nheads * headdim]
* normalisation weight ``1 + 0.1 * N(0, 1)``    [nheads * headdim]  (fp32, always)

Everything is drawn in fp32 from numpy's PCG64 and, for bf16 workloads, rounded
to bf16 with round-to-nearest-even.  Seeds: workload ``c`` uses ``base = 1000*c``;
per-head parameters from ``base``, prefix tokens from ``base + 1``, the clean block
to commit from ``base + 9`` and the noised active block at denoising step ``s``
from ``base + 10 + s``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    nheads: int
    headdim: int
    dstate: int
    ngroups: int
    block_len: int
    prefix: int
    bf16: bool
    steps: int = 1          # denoising steps per block before the commit
    base_seed: int = 0

    @property
    def d_inner(self) -> int:
        return self.nheads * self.headdim

    def with_block_len(self, L: int) -> "Workload":
        return replace(self, block_len=L)


# The five workloads: a tiny fp32 correctness case, the 87M- and 350M-model Mamba
# layer shapes, the long-context 350M case and the full-window contrast.
WORKLOADS = {
    0: Workload("tiny-fp32", 1, 4, 64, 16, 1, 16, 1024, False, 1, 0),
    1: Workload("87m-layer-b8-prefix8k", 8, 24, 64, 64, 1, 32, 8192, True, 1, 1000),
    2: Workload("350m-layer-b16-prefix65k", 16, 32, 64, 128, 1, 32, 65536, True, 8, 2000),
    3: Workload("350m-layer-b16-prefix262k", 16, 32, 64, 128, 1, 32, 262144, True, 8, 3000),
    4: Workload("350m-layer-b4-fullwindow65k", 4, 32, 64, 128, 1, 65536, 0, True, 1, 4000),
}


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even.  Finite inputs
    only (the largest finite pattern plus the rounding increment still fits 32 bits)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp32, exact."""
    return (np.ascontiguousarray(a, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def head_params(w: Workload, seed: int | None = None) -> dict:
    """Per-head A (negative), D and D_rev (= D), fp32."""
    r = _rng(w.base_seed if seed is None else seed)
    A = -np.exp(r.uniform(0.0, math.log(16.0), size=w.nheads)).astype(np.float32)
    D = r.standard_normal(w.nheads, dtype=np.float32)
    return {"A": A, "D": D, "D_rev": D.copy()}


def tokens(w: Workload, ntok: int, seed: int, batch: int | None = None) -> dict:
    """x, dt, B, C for ``ntok`` tokens of every batch row, in the workload's storage dtype."""
    bsz = w.batch if batch is None else batch
    r = _rng(seed)
    x = r.standard_normal((bsz, ntok, w.nheads, w.headdim), dtype=np.float32)
    z = r.standard_normal((bsz, ntok, w.nheads), dtype=np.float32).astype(np.float64)
    dt = np.log1p(np.exp(0.5 * z - 4.6)).astype(np.float32)
    scale = np.float32(1.0 / math.sqrt(w.dstate))
    Bm = r.standard_normal((bsz, ntok, w.ngroups, w.dstate), dtype=np.float32) * scale
    Cm = r.standard_normal((bsz, ntok, w.ngroups, w.dstate), dtype=np.float32) * scale
    out = {"x": x, "dt": dt, "B": Bm, "C": Cm}
    if w.bf16:
        out = {k: to_bf16_bits(v) for k, v in out.items()}
    return out


def tokens_device(w: Workload, ntok: int, seed: int, device="cuda:0",
                  batch: int | None = None) -> dict:
    """Like :func:`tokens`, drawn on the GPU with torch's seeded generator (for sizes too
    large to draw on the host in reasonable time, e.g. a 65,536-token window).  Same
    distributions; a different generator, so not the same numbers as :func:`tokens`.
    Returns torch tensors (bfloat16 or float32) on ``device``."""
    import torch
    bsz = w.batch if batch is None else batch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    f32 = torch.float32
    x = torch.randn((bsz, ntok, w.nheads, w.headdim), generator=g, device=device, dtype=f32)
    z = torch.randn((bsz, ntok, w.nheads), generator=g, device=device, dtype=f32).double()
    dt = torch.log1p(torch.exp(0.5 * z - 4.6)).float()
    scale = 1.0 / math.sqrt(w.dstate)
    Bm = torch.randn((bsz, ntok, w.ngroups, w.dstate), generator=g, device=device, dtype=f32)
    Cm = torch.randn((bsz, ntok, w.ngroups, w.dstate), generator=g, device=device, dtype=f32)
    Bm, Cm = Bm * scale, Cm * scale
    out = {"x": x, "dt": dt, "B": Bm, "C": Cm}
    if w.bf16:
        out = {k: v.to(torch.bfloat16) for k, v in out.items()}   # round to nearest even
    return out


def block_inputs(w: Workload, step: int = 0, batch: int | None = None) -> dict:
    """The noised active block at denoising step ``step`` plus the head parameters."""
    d = tokens(w, w.block_len, w.base_seed + 10 + step, batch)
    d.update(head_params(w))
    return d


def commit_inputs(w: Workload, batch: int | None = None) -> dict:
    """The clean (finalised) block that is committed to the cache."""
    d = tokens(w, w.block_len, w.base_seed + 9, batch)
    d.update(head_params(w))
    return d


def prefix_inputs(w: Workload, ntok: int | None = None, batch: int | None = None) -> dict:
    """A clean prefix of ``ntok`` tokens (default: the workload's prefix length)."""
    d = tokens(w, w.prefix if ntok is None else ntok, w.base_seed + 1, batch)
    d.update(head_params(w))
    return d


def slice_tokens(d: dict, t0: int, t1: int) -> dict:
    """Tokens [t0, t1) of an input dict (per-head parameters are kept)."""
    out = dict(d)
    for k in ("x", "dt", "B", "C"):
        out[k] = np.ascontiguousarray(d[k][:, t0:t1])
    return out


def random_state(w: Workload, nslots: int, seed: int, scale: float = 1.0) -> np.ndarray:
    """A seeded fp32 state pool [nslots, H, P, N] (for tests that need an arbitrary cache)."""
    r = _rng(seed)
    return (r.standard_normal((nslots, w.nheads, w.headdim, w.dstate), dtype=np.float32)
            * np.float32(scale))


def gate_inputs(w: Workload, ntok: int, seed: int, batch: int | None = None) -> dict:
    """The gate ``z`` (workload storage dtype, [batch, ntok, nheads * headdim]) and the
    normalisation weight ``norm_w`` (fp32 [nheads * headdim]) of the mixer's output path."""
    bsz = w.batch if batch is None else batch
    r = _rng(seed)
    z = r.standard_normal((bsz, ntok, w.nheads * w.headdim), dtype=np.float32)
    norm_w = (1.0 + 0.1 * r.standard_normal(w.nheads * w.headdim, dtype=np.float32)).astype(
        np.float32)
    return {"z": to_bf16_bits(z) if w.bf16 else z, "norm_w": norm_w}

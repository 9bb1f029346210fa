"""Helpers shared by the GPU tests: host <-> device transfer of seeded inputs and the
error measure of the parity bar.  No arithmetic of the scan lives here."""
import numpy as np
import torch

DEV = "cuda:0"
REL_TOL = 2e-3     # max relative error, bf16 or fp32 inputs, fp32 accumulation


def to_dev(d: dict) -> dict:
    """numpy inputs (bf16 bit patterns as uint16, or fp32) -> GPU tensors."""
    out = {}
    for k, v in d.items():
        if v.dtype == np.uint16:
            out[k] = torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).to(DEV)
        else:
            out[k] = torch.from_numpy(np.ascontiguousarray(v)).to(DEV)
    return out


def to_pool(a: np.ndarray) -> np.ndarray:
    """Row-major states [..., 64, N] -> the pool layout [..., N/4, 64, 4] (index permutation
    as documented in include/bdlm.h)."""
    *lead, P, N = a.shape
    return np.ascontiguousarray(a.reshape(*lead, P, N // 4, 4).swapaxes(-3, -2))


def from_pool(a) -> np.ndarray:
    """Pool layout [..., N/4, 64, 4] (numpy or GPU tensor) -> row-major [..., 64, N]."""
    if torch.is_tensor(a):
        a = a.detach().cpu().numpy()
    *lead, N4, P, _ = a.shape
    return np.ascontiguousarray(a.swapaxes(-3, -2).reshape(*lead, P, N4 * 4))


def pool_dev(a: np.ndarray):
    """Row-major fp32 states -> a GPU pool tensor."""
    return torch.from_numpy(to_pool(np.asarray(a, np.float32))).to(DEV)


def rel_err(gpu, ref) -> float:
    """max_i |gpu_i - ref_i| / max(|ref_i|, 1e-2 * rms(ref))."""
    g = gpu.detach().double().cpu().numpy() if torch.is_tensor(gpu) else np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (g.shape, r.shape)
    if r.size == 0:
        return 0.0
    assert np.all(np.isfinite(g)), "non-finite GPU output"
    floor = 1e-2 * np.sqrt(np.mean(r * r))
    den = np.maximum(np.abs(r), max(floor, 1e-30))
    return float(np.max(np.abs(g - r) / den))


def step(d: dict, h_pool, slot_idx=None, y=None, stream=None):
    import paper_2607_02805_amd as bd
    return bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                              h_pool, y=y, slot_idx=slot_idx, stream=stream)


def commit(d: dict, h_pool, nc, nb, expected=-1, slot_idx=None, y_clean=None, stream=None):
    import paper_2607_02805_amd as bd
    return bd.commit_boundary(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                              h_pool, nc, nb, expected, slot_idx, y_clean, stream)


def to_host(t):
    """GPU tensor -> the stored bytes as numpy (bf16 bit patterns as uint16)."""
    t = t.contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def edge_cover(batch: int, nheads: int) -> list:
    """(rows, heads) index sets covering every head of the first and last batch rows and
    every batch row of the first and last heads (each pair once): a full-size parity
    check on them meets every XCD's share of the remapped grid at its ends."""
    rows = sorted({0, batch - 1})
    mid = [b for b in range(batch) if b not in rows]
    cover = [(rows, list(range(nheads)))]
    if mid:
        cover.append((mid, sorted({0, nheads - 1})))
    return cover


def host_slice(v: dict, rows: list, heads: list, hp: dict) -> dict:
    """Stored bytes of batch rows ``rows`` and heads ``heads`` of device inputs ``v`` (x, dt,
    B, C; one group), with the per-head parameters ``hp`` of those heads."""
    r = torch.as_tensor(rows, device=v["x"].device)
    h = torch.as_tensor(heads, device=v["x"].device)
    out = {"x": to_host(v["x"].index_select(0, r).index_select(2, h)),
           "dt": to_host(v["dt"].index_select(0, r).index_select(2, h)),
           "B": to_host(v["B"].index_select(0, r)), "C": to_host(v["C"].index_select(0, r))}
    for k in ("A", "D", "D_rev"):
        a = hp[k]
        out[k] = (a.cpu().numpy() if torch.is_tensor(a) else np.asarray(a))[heads].copy()
    return out


def pick(t, rows: list, heads: list, head_dim: int = 2):
    """Rows ``rows`` and heads ``heads`` (on axis ``head_dim``) of a device tensor."""
    r = torch.as_tensor(rows, device=t.device)
    h = torch.as_tensor(heads, device=t.device)
    return t.index_select(0, r).index_select(head_dim, h)

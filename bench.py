"""Benchmark: active-block tokens/s per Mamba layer of BDLM Mamba-H's block-restricted
bidirectional scan on one MI355X, with the HBM roofline of the block-step kernel and
the CPU oracle timed beside it.

Workload (defaults): the 350M-model Mamba layer shape -- batch 16, 32 heads x 64,
dstate 128, one group -- with block length 32 and a 262,144-token committed prefix.
One benchmark step is one block cycle of the sampler: 8 denoising steps of the
active block (Sec. 4, Eq. partial-reverse) followed by the commit of the clean
block (Eq. boundary-state), with the commit also producing the layer output on the
clean block.  Inputs are seeded synthetic data already resident in HBM.

Cold-cache protocol: a real model runs many Mamba layers between two steps of the
same layer, so a layer's state is never found in the 256 MB Infinity Cache.  The
benchmark keeps a ring of ``--layers`` independent layers (default 32: 537 MB of
state, more than twice the Infinity Cache), each with its own state pool, inputs
and outputs, and runs every step over the whole ring.  Per-layer figures divide by
the ring size.

Launches are captured once into two HIP graphs (the ring's denoising steps, the
ring's commits) and replayed; HIP events recorded on the replay stream between the
two graphs time each part.  ``value`` = 8 * batch * block_len / (time of one block
cycle of one layer).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0     # MI355X HBM3E, GB/s
CSRC = os.path.join(ROOT, "paper_2607_02805_amd", "csrc")
# the sources each profiled kernel family is compiled from (a summary under profiles/
# records their hash; a figure is read back only while the hash still matches)
SOURCE_SETS = {
    "block": ("bdlm_scan.hip", "bdlm_device.h"),
    "seq": ("bdlm_seq.hip", "bdlm_device.h"),
    "all": ("bdlm_scan.hip", "bdlm_seq.hip", "bdlm_mask.hip", "bdlm_conv.hip", "bdlm_norm.hip",
            "bdlm_device.h", "bdlm_launch.h"),
}
KERNEL_SRCS = [os.path.join(CSRC, f) for f in SOURCE_SETS["block"]]
PROFILES = os.path.join(ROOT, "profiles")
TRAFFIC_SUMMARY = os.path.join(PROFILES, "hbm_traffic_block_step_350m_b16_L32.md")
TRACE_SUMMARY = os.path.join(PROFILES, "block_step_350m_b16_L32_kernel_trace.md")
SQ_SUMMARY = os.path.join(PROFILES, "sq_counters_block_step_350m_b16_L32.md")
PROBE_LIB = os.path.join(ROOT, "paper_2607_02805_amd", "libbdlm_probe.so")
STEP_KERNEL = "bdlm_block_kernel<32, 128, false, false, 2, 0, false>"
COMMIT_KERNEL = "bdlm_block_kernel<32, 128, false, true, 2, 0, false>"


def step_bytes(batch, H, P, N, G, L, in_bytes=2):
    """Algorithmic HBM bytes of one active-block step: the fp32 state read once, the
    block inputs (x, dt, B, C) read once, y (fp32) written once, per-head params."""
    state = batch * H * P * N * 4
    x = batch * L * H * P * in_bytes
    dt = batch * L * H * in_bytes
    bc = 2 * batch * L * G * N * in_bytes
    y = batch * L * H * P * 4
    return state + x + dt + bc + y + 3 * H * 4


def commit_bytes(batch, H, P, N, G, L, in_bytes=2):
    """A commit reads what a step reads, writes the clean-block output and the new state."""
    return step_bytes(batch, H, P, N, G, L, in_bytes) + batch * H * P * N * 4


def to_dev(d, dev):
    import torch
    out = {}
    for k, v in d.items():
        if v.dtype == np.uint16:
            out[k] = torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).to(dev)
        else:
            out[k] = torch.from_numpy(np.ascontiguousarray(v)).to(dev)
    return out


class Ring:
    """A ring of ``nl`` independent Mamba layers at one shape: per layer the ``p`` noised
    blocks, the clean block, the outputs and a cache.  The prefix is committed into one
    staging cache and copied into every layer's cache, so all layers sit at the same
    prefix length."""

    def __init__(self, w, nl, p, dev):
        import torch

        import bdlm_inputs as bi
        import paper_2607_02805_amd as bd
        self.w, self.nl, self.p, self.dev = w, nl, p, dev
        Bsz, H, P, N, L = w.batch, w.nheads, w.headdim, w.dstate, w.block_len
        base_steps = [to_dev(bi.block_inputs(w, s), dev) for s in range(p)]
        base_clean = to_dev(bi.commit_inputs(w), dev)
        self.layers = []
        for _ in range(nl):
            self.layers.append({
                "steps": [{k: v.clone() for k, v in d.items()} for d in base_steps],
                "clean": {k: v.clone() for k, v in base_clean.items()},
                "y": torch.empty((Bsz, L, H, P), dtype=torch.float32, device=dev),
                "y_clean": torch.empty((Bsz, L, H, P), dtype=torch.float32, device=dev)})
        self.caches = [bd.Cache(Bsz, H, N, device=dev) for _ in range(nl)]
        self.stage = bd.Cache(Bsz, H, N, device=dev)
        pre = bi.prefix_inputs(w, 16 * L)
        self.pre_blocks = [to_dev(bi.slice_tokens(pre, L * i, L * (i + 1)), dev)
                           for i in range(16)]
        self.graphs = None

    def extend_prefix(self, tokens: int) -> float:
        """Commit blocks (16 seeded clean blocks, cycled) until the prefix holds ``tokens``
        tokens; returns the seconds taken."""
        import torch
        t0 = time.time()
        L = self.w.block_len
        k = int(self.stage.n_blocks[0])
        while (k + 1) * L <= tokens:
            d = self.pre_blocks[k % 16]
            self.stage.commit(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                              expected_block_index=k)
            k += 1
        for c in self.caches:
            c.h.copy_(self.stage.h)
            c.n_committed[:] = self.stage.n_committed
            c.n_blocks[:] = self.stage.n_blocks
        torch.cuda.synchronize()
        return time.time() - t0

    def enqueue_steps(self):
        import paper_2607_02805_amd as bd
        for s in range(self.p):
            for lay, c in zip(self.layers, self.caches):
                d = lay["steps"][s]
                bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                                   c.h, y=lay["y"])

    def enqueue_commits(self):
        import paper_2607_02805_amd as bd
        for lay, c in zip(self.layers, self.caches):
            d = lay["clean"]
            # bookkeeping is advanced by the host after each replay (advance_books)
            bd.commit_boundary(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], c.h,
                               c.n_committed.copy(), c.n_blocks.copy(), -1, y_clean=lay["y_clean"])

    def capture(self, stream):
        """Capture the ring's denoising steps and the ring's commits as two HIP graphs."""
        import torch
        g_steps, g_commit = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            self.enqueue_steps()          # eager warm-up of both kernels before capture
            self.enqueue_commits()
        stream.synchronize()
        with torch.cuda.graph(g_steps, stream=stream):
            self.enqueue_steps()
        with torch.cuda.graph(g_commit, stream=stream):
            self.enqueue_commits()
        torch.cuda.synchronize()
        self.graphs = (g_steps, g_commit)

    def parity_sample(self, stream) -> dict:
        """One eager step and one eager commit of layer 0 on its step-0 and clean inputs,
        from the layer's current cached state (the one the timed steps read), into fresh
        buffers: the GPU side of the bench's parity check against the oracle."""
        import torch

        import paper_2607_02805_amd as bd
        c, lay = self.caches[0], self.layers[0]
        d, cl = lay["steps"][0], lay["clean"]
        with torch.cuda.stream(stream):
            before = bd.state_unpack(c.h, stream=stream)
            y = bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                                   c.h, stream=stream)
            h = c.h.clone()
            nb = c.n_blocks.copy()
            yc = bd.commit_boundary(cl["x"], cl["dt"], cl["A"], cl["B"], cl["C"], cl["D"],
                                    cl["D_rev"], h, c.n_committed.copy(), nb, int(nb[0]),
                                    y_clean=True, stream=stream)
            after = bd.state_unpack(h, stream=stream)
        stream.synchronize()
        return {"state": before.cpu().numpy(), "y": y.cpu().numpy(),
                "y_clean": yc.cpu().numpy(), "state_after": after.cpu().numpy(),
                "prefix_tokens": int(c.n_committed[0])}

    def advance_books(self):
        for c in self.caches:
            c.n_committed += self.w.block_len
            c.n_blocks += 1

    def time_cycles(self, stream, steps: int, warmup: int) -> dict:
        """Replay ``warmup`` then exactly ``steps`` block cycles (p steps + commit of every
        layer); HIP events on the replay stream around each graph."""
        import torch
        g_steps, g_commit = self.graphs
        with torch.cuda.stream(stream):
            for _ in range(warmup):
                g_steps.replay()
                g_commit.replay()
                self.advance_books()
        torch.cuda.synchronize()
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        torch.cuda.synchronize()
        t_wall = time.perf_counter()
        with torch.cuda.stream(stream):
            for k in range(steps):
                ev[k][0].record(stream)
                g_steps.replay()
                ev[k][1].record(stream)
                g_commit.replay()
                ev[k][2].record(stream)
                self.advance_books()
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t_wall
        nl, p = self.nl, self.p
        step_us = np.array([e[0].elapsed_time(e[1]) for e in ev]) * 1e3 / (p * nl)
        commit_us = np.array([e[1].elapsed_time(e[2]) for e in ev]) * 1e3 / nl
        t_total = ev[0][0].elapsed_time(ev[-1][2]) * 1e-3
        return {"step_us": step_us, "commit_us": commit_us, "t_total": t_total,
                "wall_s": wall_s, "prefix_tokens": int(self.caches[0].n_committed[0])}


def ring_layers(w, min_bytes: int = 512 << 20, least: int = 32) -> int:
    """Layers in a cold ring: enough that their states alone exceed twice the 256 MB
    Infinity Cache, so no step finds its state there."""
    per = w.batch * w.nheads * w.headdim * w.dstate * 4
    return max(least, -(-min_bytes // per))


def run_config(w, p: int, nl: int, prefix: int, steps: int, warmup: int,
               parity: bool = False) -> dict:
    """Block cycles (``p`` denoising steps + the commit) of a ring of ``nl`` layers at
    workload ``w`` with a ``prefix``-token committed prefix, replayed from HIP graphs."""
    import torch
    dev = "cuda:0"
    torch.cuda.set_device(0)
    Bsz, H, P, N, G, L = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups, w.block_len
    ring = Ring(w, nl, p, dev)
    prefill_s = ring.extend_prefix(prefix)
    print(f"[bench] {w.name}: prefix of {prefix} tokens committed ({prefix // L} commits) in "
          f"{prefill_s:.2f}s; ring of {nl} layers, state {nl * Bsz * H * P * N * 4 / 2**20:.0f} MiB",
          file=sys.stderr, flush=True)
    stream = torch.cuda.Stream()
    ring.capture(stream)
    t = ring.time_cycles(stream, steps, warmup)
    sample = ring.parity_sample(stream) if parity else None
    avg_step_s = float(t["step_us"].mean()) * 1e-6
    avg_commit_s = float(t["commit_us"].mean()) * 1e-6
    per_layer_cycle_s = t["t_total"] / (steps * nl)
    sb = step_bytes(Bsz, H, P, N, G, L)
    cb = commit_bytes(Bsz, H, P, N, G, L)
    del ring
    torch.cuda.empty_cache()
    return {
        "value": p * Bsz * L / per_layer_cycle_s,
        "finalised_tokens_per_s": Bsz * L / per_layer_cycle_s,
        "ms_per_step": t["t_total"] / steps * 1e3,
        "wall_s": t["wall_s"],
        "avg_step_us": avg_step_s * 1e6,
        "median_step_us": float(np.median(t["step_us"])),
        "min_step_us": float(t["step_us"].min()),
        "step_us_per_replay": [float(v) for v in t["step_us"]],
        "commit_us_per_replay": [float(v) for v in t["commit_us"]],
        "avg_commit_us": avg_commit_s * 1e6,
        "step_bytes": sb,
        "commit_bytes": cb,
        "achieved_gbs": sb / avg_step_s / 1e9,
        "commit_gbs": cb / avg_commit_s / 1e9,
        "prefix_tokens": t["prefix_tokens"],
        "layers": nl,
        "denoise_steps": p,
        "shape": dict(batch=Bsz, nheads=H, headdim=P, dstate=N, ngroups=G, block_len=L),
        "sample": sample,
    }


def run_gpu(args):
    import bdlm_inputs as bi
    w = bi.WORKLOADS[3].with_block_len(args.block_len)
    return run_config(w, args.denoise, args.layers, args.prefix, args.steps, args.warmup,
                      parity=not args.no_cpu_baseline)


def step_unit_bytes(r: dict):
    """Per-unit byte shape of a benched step for the streaming probe: ((row, head) units,
    (state, inputs, output) bytes per unit, the inputs rounded down to 64 bytes)."""
    s = r["shape"]
    st, out = s["headdim"] * s["dstate"] * 4, s["block_len"] * s["headdim"] * 4
    units = s["batch"] * s["nheads"]
    return units, (st, (r["step_bytes"] - units * (st + out)) // units // 64 * 64, out)


def config_line(r: dict, name: str) -> dict:
    """A benched configuration in the headline's format, with the streaming probe at its
    step's byte shape beside it."""
    s = r["shape"]
    units, unit = step_unit_bytes(r)
    ceiling = run_stream_ceiling(unit, units)
    return {
        "workload": name,
        "value": round(r["value"], 1), "unit": "tokens/s",
        "finalised_tokens_per_s": round(r["finalised_tokens_per_s"], 1),
        "ms_per_step": round(r["ms_per_step"], 4),
        "batch": s["batch"], "nheads": s["nheads"], "dstate": s["dstate"],
        "block_len": s["block_len"], "prefix_tokens": r["prefix_tokens"],
        "denoise_steps": r["denoise_steps"], "layer_ring": r["layers"],
        "step_us": round(r["avg_step_us"], 3), "commit_us": round(r["avg_commit_us"], 3),
        "step_bytes": r["step_bytes"], "step_gbs": round(r["achieved_gbs"], 1),
        "frac": round(r["achieved_gbs"] / HBM_PEAK_GBS, 4),
        "commit_gbs": round(r["commit_gbs"], 1),
        "stream_ceiling_gbs": None if ceiling is None else ceiling["gbs"],
        "frac_of_stream_ceiling": None if ceiling is None
        else round(r["achieved_gbs"] / ceiling["gbs"], 4),
    }


def run_other_configs(args) -> dict:
    """The 87M layer (batch 8, 24 heads, dstate 64, L 32, 8,192-token prefix, one
    denoising step + commit per block) and the 350M layer at a 65,536-token prefix
    (batch 16, 8 steps + commit), each over its own cold ring."""
    import bdlm_inputs as bi
    out = {}
    w1 = bi.WORKLOADS[1]
    r1 = run_config(w1, 1, ring_layers(w1), w1.prefix, args.steps, args.warmup)
    out["87m_b8_prefix8192"] = config_line(
        r1, f"87m-mamba-layer-b{w1.batch}-L{w1.block_len}-prefix{w1.prefix}-1step+commit")
    w2 = bi.WORKLOADS[2]
    r2 = run_config(w2, w2.steps, ring_layers(w2), w2.prefix, args.steps, args.warmup)
    out["350m_b16_prefix65536"] = config_line(
        r2, f"350m-mamba-layer-b{w2.batch}-L{w2.block_len}-prefix{w2.prefix}"
            f"-{w2.steps}steps+commit")
    for k, v in out.items():
        print(f"[bench] {k}: {v['value']:.4g} tokens/s, step {v['step_us']} us "
              f"({v['step_gbs']} GB/s), commit {v['commit_us']} us", file=sys.stderr, flush=True)
    return out


def parity_vs_oracle(w, sample: dict) -> dict:
    """The benched step and commit of one layer (the GPU outputs of ``sample``) against the
    oracle on the same inputs and the same cached state: max relative error per output,
    max_i |gpu_i - ref_i| / max(|ref_i|, 1e-2 rms(ref))."""
    import bdlm_inputs as bi
    import oracle

    def rel(g, r):
        floor = 1e-2 * np.sqrt(np.mean(r * r))
        return float(np.max(np.abs(g.astype(np.float64) - r) / np.maximum(np.abs(r), floor)))
    d, c = bi.block_inputs(w, 0), bi.commit_inputs(w)
    h = sample["state"].astype(np.float64)
    y_ref = oracle.block_step(d, h)
    nc, nb = np.zeros(w.batch, np.int64), np.zeros(w.batch, np.int64)
    rc, yc_ref = oracle.commit(c, h, nc, nb, want_y=True)
    if rc != 0:
        raise RuntimeError(f"oracle commit failed: {rc}")
    return {"y": rel(sample["y"], y_ref), "state": rel(sample["state_after"], h),
            "y_clean": rel(sample["y_clean"], yc_ref), "tol": 2e-3,
            "sample": f"layer 0 of the ring at prefix {sample['prefix_tokens']}: one step (step-0 "
                      "inputs) and one commit (clean block, with its outputs) from the cached "
                      "state the timed steps read, against the fp64 oracle on the same bytes"}


def run_flatness(args, prefixes=(4096, 65536, 262144), block_lens=(16, 32, 64)) -> dict:
    """Per-launch block-step and commit times at each prefix length and block length: the
    state is O(1) in the prefix, so the times must not move with it."""
    import torch

    import bdlm_inputs as bi
    dev = "cuda:0"
    stream = torch.cuda.Stream()
    out = {"prefix_tokens": list(prefixes), "cycles": args.sweep_steps}
    spreads = []
    for L in block_lens:
        w = bi.WORKLOADS[3].with_block_len(L)
        ring = Ring(w, args.layers, args.denoise, dev)
        ring.capture(stream)
        st, cm = [], []
        for pre in prefixes:
            ring.extend_prefix(pre)
            t = ring.time_cycles(stream, args.sweep_steps, 2)
            st.append(round(float(np.median(t["step_us"])), 3))
            cm.append(round(float(np.median(t["commit_us"])), 3))
        out[f"L{L}"] = {"step_us": st, "commit_us": cm,
                        "step_gbs": [round(step_bytes(16, 32, 64, 128, 1, L) / (u * 1e3), 1)
                                     for u in st]}
        spreads.append((max(st) - min(st)) / min(st))
        print(f"[bench] flatness L={L}: step us {st}, commit us {cm}", file=sys.stderr, flush=True)
        del ring
        torch.cuda.empty_cache()
    out["max_step_spread"] = round(max(spreads), 4)
    return out


def full_window_bytes(batch, H, P, N, G, W, in_bytes=2):
    """Algorithmic HBM bytes of the full-window scan: the window's inputs read once and y
    (fp32) written once; no state."""
    return step_bytes(batch, H, P, N, G, W, in_bytes) - batch * H * P * N * 4


def run_contrast(args, block: dict) -> dict:
    """The full-window bidirectional scan at batch 4 over a 65,536-token window (inputs
    drawn on the GPU), timed with HIP events after warm-up calls (the paper's protocol:
    5 warm-up, then the timed calls; the median is reported), and the ratio of
    per-sequence rates against the block-restricted cycle at an equal number of denoising
    steps per block."""
    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd
    dev = "cuda:0"
    w = bi.WORKLOADS[4]
    v = bi.tokens_device(w, w.block_len, w.base_seed + 10, dev)
    hp = {k: torch.from_numpy(a).to(dev) for k, a in bi.head_params(w).items()}
    y = torch.empty((w.batch, w.block_len, w.nheads, w.headdim), dtype=torch.float32, device=dev)
    stream = torch.cuda.Stream()
    reps = args.contrast_reps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(args.contrast_warmup):                  # warm-up
            bd.scan_full_window(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], hp["D_rev"], y,
                                stream=stream)
        ev[0].record(stream)
        for r in range(reps):
            bd.scan_full_window(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], hp["D_rev"],
                                y, stream=stream)
            ev[r + 1].record(stream)
    torch.cuda.synchronize()
    ms = [ev[r].elapsed_time(ev[r + 1]) for r in range(reps)]
    t_full = float(np.median(ms)) * 1e-3
    fb = full_window_bytes(w.batch, w.nheads, w.headdim, w.dstate, w.ngroups, w.block_len)
    # per-sequence time of one denoising step: the full window serves w.batch sequences per
    # call; the block step serves 16 per launch, plus the commit once every p steps
    t_seq_full = t_full / w.batch
    t_seq_block = None
    if block is not None:
        t_seq_block = (block["avg_step_us"] + block["avg_commit_us"] / args.denoise) * 1e-6 \
            / block["shape"]["batch"]
    del v, y
    torch.cuda.empty_cache()
    return {
        "workload": f"350m-mamba-layer-b{w.batch}-fullwindow{w.block_len}",
        "full_window_ms": round(t_full * 1e3, 3),
        "full_window_ms_all": [round(m, 3) for m in ms],
        "alg_bytes": fb,
        "achieved_gbs": round(fb / t_full / 1e9, 1),
        "frac": round(fb / t_full / 1e9 / HBM_PEAK_GBS, 4),
        "per_sequence_step_us": {"full_window": round(t_seq_full * 1e6, 3),
                                 "block_restricted": None if t_seq_block is None
                                 else round(t_seq_block * 1e6, 4)},
        "ratio": None if t_seq_block is None else round(t_seq_full / t_seq_block, 1),
        # the same ratio against a full window that moved only its algorithmic bytes at the
        # HBM peak: a lower bound on the contrast that no full-window kernel can beat
        "ratio_vs_full_window_hbm_floor": None if t_seq_block is None
        else round(fb / (HBM_PEAK_GBS * 1e9) / w.batch / t_seq_block, 1),
    }


def run_prefill(args) -> dict:
    """Chunked prefill of a clean prefix into the cached states at the 350M layer shape,
    batch 16 (inputs drawn on the GPU)."""
    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd
    dev = "cuda:0"
    w = bi.WORKLOADS[3]
    T = args.prefill_tokens
    v = bi.tokens_device(w, T, w.base_seed + 1, dev)
    hp = {k: torch.from_numpy(a).to(dev) for k, a in bi.head_params(w).items()}
    cache = bd.Cache(w.batch, w.nheads, w.dstate, device=dev)
    stream = torch.cuda.Stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        cache.prefill(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], stream=stream)
        e0.record(stream)
        cache.prefill(v["x"], v["dt"], hp["A"], v["B"], v["C"], hp["D"], stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) * 1e-3
    nbytes = full_window_bytes(w.batch, w.nheads, w.headdim, w.dstate, w.ngroups, T) \
        - w.batch * T * w.nheads * w.headdim * 4 + 2 * w.batch * w.nheads * w.headdim * w.dstate * 4
    del v, cache
    torch.cuda.empty_cache()
    return {"tokens": T, "batch": w.batch, "ms": round(t * 1e3, 3),
            "tokens_per_s": round(w.batch * T / t, 1), "alg_bytes": nbytes,
            "achieved_gbs": round(nbytes / t / 1e9, 1)}


def run_all_block(args) -> dict:
    """The all-block training forward of one Mamba layer (Fig. 1): an 8,192-token window
    at the 350M layer shape, batch 8 (a 64-sequence global batch over 8 GPUs), blocks of
    32 tokens.  Clean stream: the states entering all 256 blocks and its forward outputs;
    noised stream: every block stepped from its clean prefix's state (one batched block
    step over 2,048 block rows).  Inputs drawn on the GPU."""
    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd
    dev = "cuda:0"
    w = bi.Workload("350m-train-window", 8, 32, 64, 128, 1, 32, 8192, True, 1, 5000)
    T, L, K = w.prefix, w.block_len, w.prefix // w.block_len
    c = bi.tokens_device(w, T, w.base_seed + 1, dev)
    n = bi.tokens_device(w, T, w.base_seed + 10, dev)
    hp = {k: torch.from_numpy(a).to(dev) for k, a in bi.head_params(w).items()}
    stream = torch.cuda.Stream()
    reps = 3
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]

    def once():
        return bd.all_block_forward((c["x"], c["dt"], c["B"], c["C"]), (n["x"], n["dt"], n["B"], n["C"]),
                                    hp["A"], hp["D"], hp["D_rev"], L, want_clean_y=True,
                                    stream=stream)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        out = once()                                 # warm-up (and the allocations)
        del out
        ev[0].record(stream)
        for r in range(reps):
            out = once()
            ev[r + 1].record(stream)
            del out
    torch.cuda.synchronize()
    ms = [ev[r].elapsed_time(ev[r + 1]) for r in range(reps)]
    t = float(np.median(ms)) * 1e-3
    Bsz, H, P, N = w.batch, w.nheads, w.headdim, w.dstate
    inputs = Bsz * T * (H * P + H + 2 * N) * 2      # x, dt, B, C of one stream (bf16)
    y = Bsz * T * H * P * 4
    states = Bsz * K * H * P * N * 4
    nbytes = 2 * inputs + 2 * y + 2 * states        # both streams; states written, read
    del c, n
    torch.cuda.empty_cache()
    return {"workload": "350m-mamba-layer-b8-window8192-L32-allblock", "blocks": K,
            "ms": round(t * 1e3, 3), "ms_all": [round(m, 3) for m in ms],
            "tokens_per_s": round(2 * Bsz * T / t, 1), "alg_bytes": nbytes,
            "achieved_gbs": round(nbytes / t / 1e9, 1),
            "frac": round(nbytes / t / 1e9 / HBM_PEAK_GBS, 4)}


def _graph_time(fn, nlayers, reps=10):
    """Per-call time of fn(layer) over a ring of layers captured in one HIP graph."""
    import torch
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for li in range(nlayers):
            fn(li)
    stream.synchronize()
    with torch.cuda.graph(g, stream=stream):
        for li in range(nlayers):
            fn(li)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        g.replay()
        e0.record(stream)
        for _ in range(reps):
            g.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / (reps * nlayers)


def run_variants(args) -> dict:
    """Block-step variants, each over a ring of 24 layers' states (cold reads):
    the paper's 350M geometry (d_inner 1664: 26 heads of 64, dstate 128) with its block
    length 256 at batch 16 (step and commit, on the masked long-block kernel), and the step with
    separate reverse-direction inputs at the 350M layer shape (32 heads, L 32)."""
    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd
    dev = "cuda:0"
    nl = 24
    out = {}
    # paper geometry, L = 256
    w = bi.Workload("350m-paper-geometry", 16, 26, 64, 128, 1, 256, 0, True, 1, 6000)
    d = to_dev(bi.block_inputs(w, 0), dev)
    c = to_dev(bi.commit_inputs(w), dev)
    pools = [torch.zeros(bd.pool_shape(16, 26, 128), device=dev) for _ in range(nl)]
    y = torch.empty((16, 256, 26, 64), device=dev)
    yc = torch.empty_like(y)
    nc, nb = np.zeros(16, np.int64), np.zeros(16, np.int64)
    t_step = _graph_time(lambda li: bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"],
                                                       d["D"], d["D_rev"], pools[li], y=y), nl)
    t_commit = _graph_time(lambda li: bd.commit_boundary(c["x"], c["dt"], c["A"], c["B"], c["C"],
                                                         c["D"], c["D_rev"], pools[li], nc.copy(),
                                                         nb.copy(), -1, y_clean=yc), nl)
    sb = step_bytes(16, 26, 64, 128, 1, 256)
    out["paper_geometry_L256"] = {
        "workload": "350m-paper-geometry-b16-h26-L256", "step_us": round(t_step * 1e6, 2),
        "commit_us": round(t_commit * 1e6, 2), "step_bytes": sb,
        "step_gbs": round(sb / t_step / 1e9, 1),
        "active_tokens_per_s": round(16 * 256 / t_step, 1)}
    del pools, y, yc
    # commit of the clean block + the next block's first step in one launch (the state read
    # once), against the commit launch followed by the step launch (350M layer, L 32)
    w = bi.WORKLOADS[3]
    cl = to_dev(bi.commit_inputs(w), dev)
    nx = to_dev(bi.block_inputs(w, 1), dev)
    pools = [torch.randn(bd.pool_shape(16, 32, 128), device=dev) * 0.01 for _ in range(nl)]
    y = torch.empty((16, 32, 32, 64), device=dev)
    yc = torch.empty_like(y)
    z = np.zeros(16, np.int64)
    t_cs = _graph_time(lambda li: bd.commit_step(
        (cl["x"], cl["dt"], cl["B"], cl["C"]), (nx["x"], nx["dt"], nx["B"], nx["C"]), cl["A"],
        cl["D"], cl["D_rev"], pools[li], z.copy(), z.copy(), y_clean=yc, y_next=y), nl)

    def two(li):
        bd.commit_boundary(cl["x"], cl["dt"], cl["A"], cl["B"], cl["C"], cl["D"], cl["D_rev"],
                           pools[li], z.copy(), z.copy(), y_clean=yc)
        bd.scan_block_step(nx["x"], nx["dt"], nx["A"], nx["B"], nx["C"], nx["D"], nx["D_rev"],
                           pools[li], y=y)
    t_two = _graph_time(two, nl)
    sb = step_bytes(16, 32, 64, 128, 1, 32)
    cb = commit_bytes(16, 32, 64, 128, 1, 32)
    fused_bytes = cb + sb - 16 * 32 * 64 * 128 * 4      # one state read fewer
    out["commit_step_L32"] = {
        "workload": "350m-mamba-layer-b16-L32-commit+next-step",
        "fused_us": round(t_cs * 1e6, 2), "commit_then_step_us": round(t_two * 1e6, 2),
        "fused_bytes": fused_bytes, "fused_gbs": round(fused_bytes / t_cs / 1e9, 1)}
    del pools, y, yc
    # separate reverse-direction inputs, L = 32
    f = to_dev(bi.block_inputs(w, 0), dev)
    r = to_dev(bi.block_inputs(w, 1), dev)
    pools = [torch.zeros(bd.pool_shape(16, 32, 128), device=dev) for _ in range(nl)]
    y = torch.empty((16, 32, 32, 64), device=dev)
    t_sep = _graph_time(lambda li: bd.scan_block_step_sep(
        (f["x"], f["dt"], f["A"], f["B"], f["C"], f["D"]),
        (r["x"], r["dt"], r["A"], r["B"], r["C"], r["D_rev"]), pools[li], y=y), nl)
    sb = step_bytes(16, 32, 64, 128, 1, 32) + (step_bytes(16, 32, 64, 128, 1, 32)
                                               - 16 * 32 * 64 * 128 * 4 - 16 * 32 * 32 * 64 * 4)
    out["separate_reverse_L32"] = {
        "workload": "350m-mamba-layer-b16-L32-separate-reverse-inputs",
        "step_us": round(t_sep * 1e6, 2), "step_bytes": sb,
        "step_gbs": round(sb / t_sep / 1e9, 1)}
    del pools, y
    # with the mixer's convolution (pre-convolution inputs, cached convolution rows)
    ch = bd.conv_channels(32, 1, 128)
    rng = np.random.Generator(np.random.PCG64(7000))
    cw = torch.from_numpy((rng.standard_normal((ch, 4)) * 0.5).astype(np.float32)).to(dev)
    cb = torch.from_numpy((rng.standard_normal(ch) * 0.1).astype(np.float32)).to(dev)
    pools = [torch.zeros(bd.pool_shape(16, 32, 128), device=dev) for _ in range(nl)]
    convs = [torch.zeros((16, 3, ch), device=dev) for _ in range(nl)]
    y = torch.empty((16, 32, 32, 64), device=dev)
    ws = torch.empty(bd._workspace_bytes(bd.lib().bdlm_conv_workspace,
                                         bd._desc(f["x"], f["dt"], f["B"], f["C"])),
                     dtype=torch.uint8, device=dev)
    nc, nb = np.zeros(16, np.int64), np.zeros(16, np.int64)
    t_cs = _graph_time(lambda li: bd.conv_block_step(f["x"], f["dt"], f["A"], f["B"], f["C"], f["D"],
                                                     f["D_rev"], cw, cb, convs[li], pools[li], y=y,
                                                     workspace=ws), nl)
    t_cc = _graph_time(lambda li: bd.conv_commit_boundary(f["x"], f["dt"], f["A"], f["B"], f["C"],
                                                          f["D"], f["D_rev"], cw, cb, convs[li],
                                                          pools[li], nc.copy(), nb.copy(), -1,
                                                          y_clean=y, workspace=ws), nl)
    sb = step_bytes(16, 32, 64, 128, 1, 32) + 16 * 3 * ch * 4 + ch * 5 * 4
    out["conv_L32"] = {
        "workload": "350m-mamba-layer-b16-L32-with-conv-state",
        "step_us": round(t_cs * 1e6, 2), "commit_us": round(t_cc * 1e6, 2), "step_bytes": sb,
        "step_gbs": round(sb / t_cs / 1e9, 1)}
    del pools, convs, y, ws
    # the gated RMS normalisation of the step's output (the mixer's output path), alone
    # (y, gate and output over a ring of 48 layers: cold) and after the step, in place
    nl2 = 48
    gi = bi.gate_inputs(w, 32, 7500)
    zt = to_dev({"z": gi["z"]}, dev)["z"]
    ys = [torch.randn((16, 32, 32, 64), device=dev) for _ in range(nl2)]
    zs = [zt.clone() for _ in range(nl2)]
    outs = [torch.empty_like(ys[0]) for _ in range(nl2)]
    nw = torch.from_numpy(gi["norm_w"]).to(dev)
    t_norm = _graph_time(lambda li: bd.gated_rmsnorm(ys[li], zs[li], nw, 1e-5, out=outs[li]), nl2)
    pools = [torch.zeros(bd.pool_shape(16, 32, 128), device=dev) for _ in range(nl)]

    def step_norm(li):
        bd.scan_block_step(f["x"], f["dt"], f["A"], f["B"], f["C"], f["D"], f["D_rev"], pools[li],
                           y=ys[li])
        bd.gated_rmsnorm(ys[li], zs[li], nw, 1e-5, out=ys[li])
    t_sn = _graph_time(step_norm, nl)
    nbytes = 16 * 32 * 2048 * (4 + 2 + 4) + 2048 * 4
    out["gated_norm_L32"] = {
        "workload": "350m-mamba-layer-b16-L32-gated-rmsnorm", "norm_us": round(t_norm * 1e6, 2),
        "norm_bytes": nbytes, "norm_gbs": round(nbytes / t_norm / 1e9, 1),
        "step_plus_norm_us": round(t_sn * 1e6, 2)}
    del ys, zs, outs, pools
    torch.cuda.empty_cache()
    return out


def run_warm(args, nodes: int = 32, reps: int = 20) -> dict:
    """The block step of one layer replayed back to back: its 16.8 MB state and its
    inputs stay resident in the Infinity Cache between launches.  Context for the cold
    figure (every read from HBM), which is the one reported."""
    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd
    dev = "cuda:0"
    w = bi.WORKLOADS[3]
    d = to_dev(bi.block_inputs(w, 0), dev)
    pool = torch.randn(bd.pool_shape(w.batch, w.nheads, w.dstate), device=dev)
    y = torch.empty((w.batch, w.block_len, w.nheads, w.headdim), device=dev)
    # one graph of `nodes` steps of the same layer (a graph of one node would time the
    # graph launch, not the step)
    t = _graph_time(lambda li: bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"],
                                                  d["D_rev"], pool, y=y), nodes, reps=reps)
    del d, pool, y
    torch.cuda.empty_cache()
    sb = step_bytes(w.batch, w.nheads, w.headdim, w.dstate, w.ngroups, w.block_len)
    return {"workload": "350m-mamba-layer-b16-L32-one-layer-back-to-back",
            "step_us": round(t * 1e6, 3), "bytes_per_step": sb,
            "effective_gbs": round(sb / t / 1e9, 1)}


def run_batch_sweep(args, batches=(16, 32, 64, 128), nl=24) -> dict:
    """The block step at the 350M layer shape (L 32) at several batch sizes, each layer of
    a ring with its own state, inputs and outputs (cold reads), beside a plain device copy
    of the same byte count: how far the step's bandwidth is set by its launch size."""
    import dataclasses

    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd
    dev = "cuda:0"
    out = {"batch": list(batches), "step_us": [], "step_gbs": [], "frac": [], "copy_us": [],
           "copy_gbs": []}
    for b in batches:
        w = dataclasses.replace(bi.WORKLOADS[3], batch=b)
        base = to_dev(bi.block_inputs(w, 0), dev)
        lay = [{k: v.clone() for k, v in base.items()} for _ in range(nl)]
        pools = [torch.randn(bd.pool_shape(b, 32, 128), device=dev) for _ in range(nl)]
        ys = [torch.empty((b, 32, 32, 64), device=dev) for _ in range(nl)]
        t = _graph_time(lambda li: bd.scan_block_step(
            lay[li]["x"], lay[li]["dt"], lay[li]["A"], lay[li]["B"], lay[li]["C"], lay[li]["D"],
            lay[li]["D_rev"], pools[li], y=ys[li]), nl, reps=20)
        del base, lay, pools, ys
        torch.cuda.empty_cache()
        sb = step_bytes(b, 32, 64, 128, 1, 32)
        cp = run_copy_reference(sb)
        out["step_us"].append(round(t * 1e6, 3))
        out["step_gbs"].append(round(sb / t / 1e9, 1))
        out["frac"].append(round(sb / t / 1e9 / HBM_PEAK_GBS, 4))
        out["copy_us"].append(cp["us_per_launch"])
        out["copy_gbs"].append(cp["gbs"])
        print(f"[bench] batch {b}: step {t * 1e6:.2f} us ({sb / t / 1e9:.0f} GB/s), "
              f"copy of the same bytes {cp['us_per_launch']:.2f} us", file=sys.stderr, flush=True)
    return out


def run_copy_reference(nbytes: int, nbuf: int = 32, reps: int = 20) -> dict:
    """A plain device copy moving ``nbytes`` in total (half read, half written) per launch,
    over a ring of ``nbuf`` buffers so that every launch misses the Infinity Cache,
    replayed from a HIP graph: what a streaming kernel of the block step's size achieves."""
    import torch
    dev = "cuda:0"
    n = nbytes // 2 // 4
    src = [torch.empty(n, dtype=torch.float32, device=dev).uniform_() for _ in range(nbuf)]
    dst = [torch.empty(n, dtype=torch.float32, device=dev) for _ in range(nbuf)]
    stream = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for a, b in zip(src, dst):
            b.copy_(a)
    stream.synchronize()
    with torch.cuda.graph(g, stream=stream):
        for a, b in zip(src, dst):
            b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        g.replay()
        e0.record(stream)
        for _ in range(reps):
            g.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * nbuf)
    del src, dst, g
    torch.cuda.empty_cache()
    return {"bytes_per_launch": 2 * n * 4, "us_per_launch": round(us, 3),
            "gbs": round(2 * n * 4 / us / 1e3, 1)}


def cpu_baseline(args, budget_s: float):
    """The oracle, as it stands, on the host cores: whole block cycles (8 steps + commit) of
    one layer at the full workload shape, repeated until the time budget is spent."""
    import bdlm_inputs as bi
    import oracle

    w = bi.WORKLOADS[3].with_block_len(args.block_len)
    steps = [bi.block_inputs(w, s) for s in range(args.denoise)]
    clean = bi.commit_inputs(w)
    pool = bi.random_state(w, w.batch, 1).astype(np.float64)
    nc, nb = np.zeros(w.batch, np.int64), np.zeros(w.batch, np.int64)
    cycles, t0 = 0, time.perf_counter()
    while True:
        for d in steps:
            oracle.block_step(d, pool)
        oracle.commit(clean, pool, nc, nb, want_y=True)
        cycles += 1
        el = time.perf_counter() - t0
        if el >= budget_s or cycles >= 50:
            break
    tokens = cycles * args.denoise * w.batch * w.block_len
    cores = oracle.num_threads()
    # the same cycle on one thread (one cycle, or three when they are short)
    oracle.set_num_threads(1)
    one, t1 = 0, time.perf_counter()
    try:
        while one < 3:
            for d in steps:
                oracle.block_step(d, pool)
            oracle.commit(clean, pool, nc, nb, want_y=True)
            one += 1
            if time.perf_counter() - t1 >= 0.25 * budget_s:
                break
    finally:
        oracle.set_num_threads(cores)
    el1 = time.perf_counter() - t1
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")),
                         None)
    except OSError:
        pass
    return {"value": tokens / el, "unit": "tokens/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{cycles} full block cycles ({args.denoise} steps + commit) of one layer "
                      f"at batch {w.batch}, 32 heads, dstate 128, L {w.block_len}; "
                      f"{el:.1f} s, fp64",
            "value_1thread": one * args.denoise * w.batch * w.block_len / el1,
            "sample_1thread": f"{one} block cycle(s) on one thread; {el1:.1f} s",
            "cpu_model": model}


def kernel_source_sha(which: str = "block") -> str:
    """Hash of the sources a kernel family is compiled from (SOURCE_SETS)."""
    import hashlib
    h = hashlib.sha256()
    for f in SOURCE_SETS[which]:
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()[:16]


def profile_fields(path: str, which: str = "block") -> dict:
    """The ``- key: value`` lines of a committed profile summary, or {} when it is missing
    or was taken on other kernel sources (its kernel_source_sha256_16 no longer matches)."""
    if not os.path.exists(path):
        return {}
    kv = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            kv[k.strip()] = v.strip().strip("`")
    return kv if kv.get("kernel_source_sha256_16") == kernel_source_sha(which) else {}


def _num(kv: dict, key: str, cast=float):
    try:
        return cast(kv[key])
    except (KeyError, ValueError):
        return None


def measured_traffic():
    """HBM bytes per step launch from the committed counter summary, or None when the
    kernel source changed since the counters were taken."""
    return _num(profile_fields(TRAFFIC_SUMMARY), "step_hbm_bytes_per_launch", int)


def run_stream_ceiling(unit_bytes: tuple, units: int, nbuf: int = 32, reps: int = 20) -> dict:
    """A plain streaming kernel (libbdlm_probe.so) with the block step's byte shape: per
    unit a state slab read, an input slab read and an output slab written, over a ring of
    ``nbuf`` buffer sets (every launch misses the Infinity Cache), replayed from a HIP
    graph like the step; the fastest of its launch shapes.  What a launch of this size
    reaches here with no arithmetic at all."""
    import ctypes

    import torch
    if not os.path.exists(PROBE_LIB):
        return None
    lib = ctypes.CDLL(PROBE_LIB)
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    lib.bdlm_probe_stream.argtypes = [vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp]
    lib.bdlm_probe_stream.restype = ctypes.c_int
    dev = "cuda:0"
    st_b, in_b, out_b = unit_bytes
    bufs = [(torch.rand(units * st_b // 4, device=dev), torch.rand(units * in_b // 4, device=dev),
             torch.empty(units * out_b // 4, device=dev)) for _ in range(nbuf)]
    stream = torch.cuda.Stream()
    best = None
    for cfg in range(lib.bdlm_probe_configs()):
        def launch(b):
            rc = lib.bdlm_probe_stream(b[0].data_ptr(), b[1].data_ptr(), b[2].data_ptr(), units,
                                       st_b, in_b, out_b, cfg, stream.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"probe launch failed: {rc}")
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            for b in bufs:
                launch(b)
        stream.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for b in bufs:
                launch(b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            g.replay()
            e0.record(stream)
            for _ in range(reps):
                g.replay()
            e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / (reps * nbuf)
        if best is None or us < best[0]:
            best = (us, cfg)
        del g
    del bufs
    torch.cuda.empty_cache()
    nbytes = units * (st_b + in_b + out_b)
    return {"bytes_per_launch": nbytes, "unit_bytes": list(unit_bytes), "units": units,
            "us_per_launch": round(best[0], 3), "gbs": round(nbytes / best[0] / 1e3, 1),
            "config": best[1]}


def _csv_rows(path):
    import csv
    return list(csv.DictReader(open(path)))


def summarize_trace(stats_csv: str) -> str:
    """Markdown table of a rocprofv3 --kernel-trace --stats kernel_stats.csv."""
    out = ["| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for r in _csv_rows(stats_csv):
        name = r["Name"].replace("bdlm::(anonymous namespace)::", "").split("(")[0]
        out.append(f"| `{name[:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.3f} | "
                   f"{float(r['MinNs']) / 1e3:.3f} | {float(r['MaxNs']) / 1e3:.3f} | "
                   f"{float(r['Percentage']):.1f} |")
    return "\n".join(out)


def summarize_dispatches(trace_csv: str) -> str:
    """Markdown table of a rocprofv3 --kernel-trace kernel_trace.csv grouped by kernel and
    launch shape (grid threads, workgroup size): separates the workloads that launch one
    kernel template at different shapes."""
    import statistics as st
    groups = {}
    for r in _csv_rows(trace_csv):
        name = r["Kernel_Name"].replace("bdlm::(anonymous namespace)::", "").split("(")[0]
        if "bdlm" not in name:
            continue
        key = (name, int(r["Grid_Size_X"]), int(r["Workgroup_Size_X"]))
        groups.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    out = ["| kernel | workgroups x threads | calls | median us | mean us | min us |",
           "|---|---|---|---|---|---|"]
    for (name, grid, wg), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{name[:70]}` | {grid // wg} x {wg} | {len(d)} | {st.median(d):.2f} | "
                   f"{st.fmean(d):.2f} | {min(d):.2f} |")
    return "\n".join(out)


def summarize_counters(counter_csv: str) -> str:
    """Markdown table of the per-dispatch medians of each counter in a rocprofv3 --pmc
    counter_collection.csv, per bdlm kernel and launch shape."""
    import statistics as st
    groups, names = {}, []
    for r in _csv_rows(counter_csv):
        name = r["Kernel_Name"].replace("bdlm::(anonymous namespace)::", "").split("(")[0]
        if "bdlm" not in name:
            continue
        key = (name, int(r["Grid_Size"]) // int(r["Workgroup_Size"]), int(r["Workgroup_Size"]))
        c = r["Counter_Name"]
        if c not in names:
            names.append(c)
        groups.setdefault(key, {}).setdefault(c, {})[r["Dispatch_Id"]] = float(r["Counter_Value"])
    out = ["| kernel | workgroups x threads | dispatches | " + " | ".join(names) + " |",
           "|---|---|---|" + "---|" * len(names)]
    for (name, wgs, wg), d in groups.items():
        n = max(len(v) for v in d.values())
        vals = [f"{st.median(d[c].values()):.0f}" if c in d else "" for c in names]
        out.append(f"| `{name[:60]}` | {wgs} x {wg} | {n} | " + " | ".join(vals) + " |")
    return "\n".join(out)


def summarize_traffic_shapes(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv,
                             copy_bytes=256 << 20) -> str:
    """Markdown table of per-dispatch HBM bytes (medians of FETCH_SIZE / WRITE_SIZE, each
    scaled by the same counter's reading for a plain copy of known size) per bdlm kernel
    and launch shape."""
    import statistics as st

    def groups(path, counter):
        d = {}
        for r in _csv_rows(path):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"].replace("bdlm::(anonymous namespace)::", "").split("(")[0]
            key = (name, int(r["Grid_Size"]) // int(r["Workgroup_Size"]), int(r["Workgroup_Size"]))
            d.setdefault(key, []).append(float(r["Counter_Value"]))
        return d

    def copy_kib(path, counter):
        return st.median(v for (n, _, _), vs in groups(path, counter).items()
                         if "copyBuffer" in n for v in vs)

    f_scale = copy_bytes / 1024 / copy_kib(copy_fetch_csv, "FETCH_SIZE")
    w_scale = copy_bytes / 1024 / copy_kib(copy_write_csv, "WRITE_SIZE")
    fetch, write = groups(fetch_csv, "FETCH_SIZE"), groups(write_csv, "WRITE_SIZE")
    out = [f"FETCH_SIZE x {f_scale:.4f} KiB, WRITE_SIZE x {w_scale:.4f} KiB (copy calibration)",
           "", "| kernel | workgroups x threads | dispatches | fetch bytes | write bytes |",
           "|---|---|---|---|---|"]
    for key in sorted(set(fetch) | set(write), key=lambda k: -st.median(fetch.get(k, [0]))):
        if "bdlm" not in key[0]:
            continue
        fb = st.median(fetch[key]) * 1024 * f_scale if key in fetch else float("nan")
        wb = st.median(write[key]) * 1024 * w_scale if key in write else float("nan")
        n = max(len(fetch.get(key, [])), len(write.get(key, [])))
        out.append(f"| `{key[0][:60]}` | {key[1]} x {key[2]} | {n} | {fb:,.0f} | {wb:,.0f} |")
    return "\n".join(out)


def summarize_traffic(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv,
                      copy_bytes=256 << 20, kernels=None) -> dict:
    """Per-launch HBM bytes of kernels (default: the block step and the commit; else a
    {tag: name substring} map) from FETCH_SIZE / WRITE_SIZE (KiB per dispatch), each
    scaled by the same counter's reading for a plain copy of known size."""
    import statistics as st

    def per_kernel(path, counter):
        d = {}
        for r in _csv_rows(path):
            if r["Counter_Name"] == counter:
                d.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return d

    def copy_kib(path, counter):
        vals = [v for k, vs in per_kernel(path, counter).items() if "copyBuffer" in k for v in vs]
        return st.median(vals)

    f_scale = copy_bytes / 1024 / copy_kib(copy_fetch_csv, "FETCH_SIZE")
    w_scale = copy_bytes / 1024 / copy_kib(copy_write_csv, "WRITE_SIZE")
    res = {"fetch_scale": f_scale, "write_scale": w_scale}
    kernels = kernels or {"step": STEP_KERNEL, "commit": COMMIT_KERNEL}
    for tag, key in kernels.items():
        fk = [v for k, vs in per_kernel(fetch_csv, "FETCH_SIZE").items() if key in k for v in vs]
        wk = [v for k, vs in per_kernel(write_csv, "WRITE_SIZE").items() if key in k for v in vs]
        res[tag] = {"fetch_kib_median": st.median(fk), "write_kib_median": st.median(wk),
                    "dispatches": len(fk),
                    "fetch_bytes": int(st.median(fk) * 1024 * f_scale),
                    "write_bytes": int(st.median(wk) * 1024 * w_scale)}
    return res


def _step_dispatches(trace_csv: str, kernel: str, grid_threads: int):
    """(start, end) ns of the dispatches of one kernel at one launch shape."""
    out = []
    for r in _csv_rows(trace_csv):
        name = r["Kernel_Name"].replace("bdlm::(anonymous namespace)::", "")
        if kernel in name and int(r["Grid_Size_X"]) == grid_threads:
            out.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    return sorted(out)


def span_per_node(disp, run_len: int) -> float | None:
    """Median over graph replays of (last end - first start) / nodes for runs of exactly
    ``run_len`` back-to-back dispatches (one replay of the ring's steps): the trace's
    counterpart of the HIP-event time per step node."""
    import statistics as st
    runs, cur = [], [disp[0]] if disp else []
    for d in disp[1:]:
        if d[0] - cur[-1][1] < 100_000:     # within 100 us of the previous dispatch's end
            cur.append(d)
        else:
            runs.append(cur)
            cur = [d]
    if cur:
        runs.append(cur)
    runs = [r for r in runs if len(r) == run_len]
    if not runs and disp and len(disp) % run_len == 0:
        # replays closer together than the gap test separates: consecutive groups of
        # run_len dispatches (every step dispatch of the run belongs to a replay)
        runs = [disp[i:i + run_len] for i in range(0, len(disp), run_len)]
    spans = [(r[-1][1] - r[0][0]) / 1e3 / len(r) for r in runs]
    return st.median(spans) if spans else None


def profiled_sha(src: str, which: str) -> str:
    """The kernel-source hash recorded next to a rocprofv3 output directory when it was
    taken (source_sha_<which>.txt, written by the profiling commands), so a summary is
    stamped with the sources that produced its numbers; refuses to stamp a directory
    taken on other sources than the current ones."""
    f = os.path.join(src, f"source_sha_{which}.txt")
    if not os.path.exists(f):
        raise SystemExit(f"{f} missing: record `bench.py --source-sha {which}` with the profile")
    sha = open(f).read().strip()
    if sha != kernel_source_sha(which):
        raise SystemExit(f"{src} was profiled on sources {sha}, the tree holds "
                         f"{kernel_source_sha(which)}: profile again")
    return sha


def write_block_profiles(src: str, out_dir: str, nl: int = 32, p: int = 8) -> None:
    """Write the three block-step summaries under ``out_dir`` from a rocprofv3 output
    directory ``src`` holding trace_kernel_stats.csv / trace_kernel_trace.csv (kernel
    trace), fetch/write/copyfetch/copywrite_counter_collection.csv (HBM traffic) and
    mfma_counter_collection.csv (MfmaUtil), taken with the commands listed in them."""
    import statistics as st
    sha = profiled_sha(src, "block")
    hdr = f"- kernel_source_sha256_16: `{sha}`\n"
    R = "python3 $R/bench.py --steps 20 --warmup 5 --no-extras --no-cpu-baseline"
    pre = "cd /tmp && export TMPDIR=/tmp && "
    cmd_trace = (f"{pre}rocprofv3 --kernel-trace --stats --output-format csv -d $OUT -o trace -- {R}")
    # trace
    stats = os.path.join(src, "trace_kernel_stats.csv")
    trace = os.path.join(src, "trace_kernel_trace.csv")
    disp = _step_dispatches(trace, STEP_KERNEL, 512 * 512)
    durs = [(e - b) / 1e3 for b, e in disp]
    cdisp = _step_dispatches(trace, COMMIT_KERNEL, 512 * 512)
    cdur = [(e - b) / 1e3 for b, e in cdisp]
    span = span_per_node(disp, nl * p)
    # the bench's own HIP-event figure in the traced run (stdout saved as trace.log)
    ev = None
    log = os.path.join(src, "trace.log")
    if os.path.exists(log):
        for ln in open(log):
            if ln.startswith("{") and '"roofline"' in ln:
                ev = json.loads(ln)["config"]["step_us"]
    text = (f"# Block step kernel trace: 350M layer shape, batch 16, L 32, 262K prefix\n\n"
            f"The headline workload of `bench.py` (8 denoising steps + commit per block cycle, "
            f"ring of {nl} layers, graph replay), under the kernel tracer.\n\n{hdr}"
            f"- step_kernel: `{STEP_KERNEL}` (512 workgroups x 512 threads)\n"
            f"- step_kernel_dispatches: {len(durs)}\n"
            f"- step_kernel_mean_us: {st.fmean(durs):.3f}\n"
            f"- step_kernel_median_us: {st.median(durs):.3f}\n"
            f"- step_span_per_node_us: {'' if span is None else f'{span:.3f}'}\n"
            f"- commit_kernel_mean_us: {st.fmean(cdur):.3f}\n"
            f"- bench_events_step_us_under_tracer: {'' if ev is None else ev}\n\n"
            "`step_kernel_mean_us` is the mean dispatch duration the tracer records (start to end "
            "of each dispatch); `step_span_per_node_us` is, for each replay of the ring's "
            f"{nl * p} step nodes, the time from the first node's start to the last node's end "
            "divided by the node count, the quantity the bench's HIP events measure "
            "(`bench_events_step_us_under_tracer`, the bench's own figure in this traced run).  "
            "The tracer serialises dispatches: under it a node no longer starts while its "
            "predecessor drains, so the traced span per node exceeds the untraced HIP-event "
            "figure the bench reports, and each dispatch runs its ramp-up and drain alone.  The "
            "traced dispatch duration is therefore an upper bound on the pipelined per-node time "
            "the roofline fraction uses, not an equal of it.  The commit kernel's mean covers the "
            "prefix commits (no clean-block outputs) and the cycle commits (with them).\n\n"
            f"Command (R = repository root, OUT = an output directory; MI355X, ROCm 7.2):\n\n"
            f"    python3 $R/bench.py --source-sha block > $OUT/source_sha_block.txt\n"
            f"    {cmd_trace}\n    python3 bench.py --write-block-profiles $OUT profiles\n\n"
            "## Kernel statistics (whole run)\n\n" + summarize_trace(stats) + "\n")
    open(os.path.join(out_dir, "block_step_350m_b16_L32_kernel_trace.md"), "w").write(text)
    # traffic
    f = [os.path.join(src, f"{k}_counter_collection.csv") for k in ("fetch", "write", "copyfetch", "copywrite")]
    t = summarize_traffic(*f)
    sb, cb = step_bytes(16, 32, 64, 128, 1, 32), commit_bytes(16, 32, 64, 128, 1, 32)
    step_hbm = t["step"]["fetch_bytes"] + t["step"]["write_bytes"]
    commit_hbm = t["commit"]["fetch_bytes"] + t["commit"]["write_bytes"]
    cmds = "\n".join(f"    {pre}rocprofv3 --pmc {c} --output-format csv -d $OUT -o {o} -- {a}"
                     for c, o, a in (("FETCH_SIZE", "fetch", R), ("WRITE_SIZE", "write", R),
                                     ("FETCH_SIZE", "copyfetch", "python3 $R/bench.py --copy-calibration"),
                                     ("WRITE_SIZE", "copywrite", "python3 $R/bench.py --copy-calibration")))
    text = (f"# HBM traffic of the block step and the commit: 350M layer shape, batch 16, L 32\n\n"
            f"{hdr}- step_hbm_bytes_per_launch: {step_hbm}\n- step_alg_bytes: {sb}\n"
            f"- step_traffic_over_alg: {step_hbm / sb:.4f}\n"
            f"- commit_hbm_bytes_per_launch: {commit_hbm}\n- commit_alg_bytes: {cb}\n"
            f"- fetch_scale: {t['fetch_scale']:.4f}\n- write_scale: {t['write_scale']:.4f}\n\n"
            "FETCH_SIZE and WRITE_SIZE (KiB per dispatch, median over dispatches) scaled by what "
            "the same counter reads for a plain 256 MiB device copy (bytes = KiB x 1024 x scale).\n\n"
            f"Commands (R = repository root, OUT = an output directory):\n\n"
            f"    python3 $R/bench.py --source-sha block > $OUT/source_sha_block.txt\n{cmds}\n"
            f"    python3 bench.py --write-block-profiles $OUT profiles\n\n"
            f"| kernel | dispatches | fetch bytes | write bytes |\n|---|---|---|---|\n"
            f"| step `{STEP_KERNEL}` | {t['step']['dispatches']} | {t['step']['fetch_bytes']:,} | "
            f"{t['step']['write_bytes']:,} |\n"
            f"| commit `{COMMIT_KERNEL}` | {t['commit']['dispatches']} | {t['commit']['fetch_bytes']:,} | "
            f"{t['commit']['write_bytes']:,} |\n")
    open(os.path.join(out_dir, "hbm_traffic_block_step_350m_b16_L32.md"), "w").write(text)
    # MFMA utilisation
    mf = os.path.join(src, "mfma_counter_collection.csv")
    vals = {}
    for r in _csv_rows(mf):
        name = r["Kernel_Name"]
        if STEP_KERNEL in name.replace("bdlm::(anonymous namespace)::", "") \
                and int(r["Grid_Size"]) == 512 * 512:
            vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    util = st.median(vals["MfmaUtil"])
    text = (f"# MFMA utilisation of the block step: 350M layer shape, batch 16, L 32\n\n{hdr}"
            f"- step_mfma_busy_pct: {util:.2f}\n- step_dispatches: {len(vals['MfmaUtil'])}\n\n"
            "rocprofv3's derived counter MfmaUtil = 100 x SQ_VALU_MFMA_BUSY_CYCLES (summed over "
            "SIMDs) / (GRBM_GUI_ACTIVE x SIMD count), median over the step dispatches: the share "
            "of the launch's active cycles in which a SIMD's matrix unit is busy.  The step is "
            "bound by HBM, so this is evidence of where the Gram and split-bf16 products sit, "
            "not a roof.\n\nCommand (R = repository root, OUT = an output directory):\n\n"
            "    python3 $R/bench.py --source-sha block > $OUT/source_sha_block.txt\n"
            f"    {pre}rocprofv3 --pmc MfmaUtil --output-format csv -d $OUT -o mfma -- {R}\n"
            f"    python3 bench.py --write-block-profiles $OUT profiles\n")
    open(os.path.join(out_dir, "sq_counters_block_step_350m_b16_L32.md"), "w").write(text)


SEQ_WORKLOADS = """All workloads of `bench.py --sequence-only` (350M layer shape: 32 heads x 64, or the
paper's 26, dstate 128, one group, bf16 activations unless stated):

* full window: batch 4, 65,536 tokens, forward + reverse from zero; 16 segments of
  4,096 tokens per row and head -- `seg_state` (both directions' local states, 2048
  workgroups), `seg_combine` (1024 workgroups), `seg_out` forward and reverse (2048);
* prefill: batch 16, 16,384 tokens -- `seg_state` (2048), `seg_combine` (2048);
* all-block forward: batch 8, 8,192-token window, L = 32 (256 blocks; segments of 16
  blocks) -- `seg_state` (4096), `seg_combine` (4096), `seg_out` with SUB = 32 carrying
  the state block by block and writing the block states and the clean outputs (4096),
  then the block step over 2,048 rows (65536 x 512);
* paper geometry: batch 16, 26 heads, L = 256 -- `bdlm_mask_block_kernel`, the block in
  masked-matrix form, one workgroup of eight waves per (row, head), each wave owning 32
  output tokens (416 workgroups of 512 threads);
* separate reverse inputs: batch 16, L = 32 -- one block-kernel launch with both input
  sets (direction 3), 512 x 512;
* convolution state: batch 16, L = 32 -- the fp32 block kernel with the convolution in
  its staging (last template flag true), forward (direction 1; the commit instantiation
  on commits) then reverse (direction 2), and `bdlm_conv_keep_kernel` on commits;
* gated RMS normalisation: 512 tokens x 2,048 channels -- `bdlm_gated_rmsnorm_kernel`
  alone and after the block step;
* fused commit + next step: batch 16, L = 32 -- the block kernel's direction 4.
"""


def write_seq_profiles(src: str, out_dir: str) -> None:
    """Write the sequence/all-block/variant summaries under ``out_dir`` from a rocprofv3
    output directory ``src`` holding trace_kernel_trace.csv, fetch/write/copyfetch/
    copywrite_counter_collection.csv and p1/p2/mfma_counter_collection.csv, taken with the
    commands listed in them."""
    hdr = f"- kernel_source_sha256_16: `{profiled_sha(src, 'all')}`\n"
    pre = "cd /tmp && export TMPDIR=/tmp && "
    R = "python3 $R/bench.py --sequence-only"
    cal = "python3 $R/bench.py --copy-calibration"
    tail = "    python3 bench.py --write-seq-profiles $OUT profiles\n"
    f = [os.path.join(src, f"{k}_counter_collection.csv") for k in ("fetch", "write", "copyfetch", "copywrite")]
    cmds = ("    python3 $R/bench.py --source-sha all > $OUT/source_sha_all.txt\n"
            f"    {pre}rocprofv3 --kernel-trace --stats --output-format csv -d $OUT -o trace -- {R} --contrast-reps 5\n"
            + "".join(f"    {pre}rocprofv3 --pmc {c} --output-format csv -d $OUT -o {o} -- {a}\n"
                      for c, o, a in (("FETCH_SIZE", "fetch", R + " --contrast-reps 1"),
                                      ("WRITE_SIZE", "write", R + " --contrast-reps 1"),
                                      ("FETCH_SIZE", "copyfetch", cal), ("WRITE_SIZE", "copywrite", cal)))
            + tail)
    text = ("# Sequence kernels, all-block forward and block variants: kernel trace and HBM traffic\n\n"
            + hdr + "\n" + SEQ_WORKLOADS
            + "\nCommands (R = repository root, OUT = an output directory; MI355X, ROCm 7.2):\n\n"
            + cmds + "\n## Kernel trace\n\nPer kernel and launch shape (traced durations of the "
            "short launches include the dispatch start-up that untraced graph replay overlaps with "
            "the previous node):\n\n"
            + summarize_dispatches(os.path.join(src, "trace_kernel_trace.csv"))
            + "\n\n## HBM traffic per dispatch\n\nFETCH_SIZE / WRITE_SIZE medians per dispatch, "
            "each scaled by the same counter's reading for a 256 MiB device copy.\n\n"
            + summarize_traffic_shapes(*f) + "\n")
    open(os.path.join(out_dir, "sequence_allblock_variants_350m_trace_and_traffic.md"), "w").write(text)
    passes = [("p1", "SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_WAIT_INST_LDS "
                     "SQ_ACTIVE_INST_VALU SQ_ACTIVE_INST_LDS SQ_LDS_BANK_CONFLICT"),
              ("p2", "SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_LDS "
                     "SQ_LDS_IDX_ACTIVE SQ_ACTIVE_INST_VMEM SQ_WAIT_ANY"),
              ("mfma", "MfmaUtil")]
    cmds = ("    python3 $R/bench.py --source-sha all > $OUT/source_sha_all.txt\n" +
            "".join(f"    {pre}rocprofv3 --pmc {c} --output-format csv -d $OUT -o {o} -- {R} --contrast-reps 1\n"
                    for o, c in passes) + tail)
    text = ("# SQ counters per dispatch (median): sequence kernels and block variants, 350M layer shape\n\n"
            + hdr + "\nThe workloads of the sequence trace summary, one timed repetition of the "
            "contrast; one pass per counter set (at most 8 SQ counters each).  MfmaUtil is "
            "rocprofv3's derived 100 x SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x SIMD count): "
            "the share of active cycles in which a SIMD's matrix unit is busy.\n\n"
            "Commands (R = repository root, OUT = an output directory; MI355X, ROCm 7.2):\n\n"
            + cmds
            + "".join(f"\n## Pass {o}\n\n" + summarize_counters(os.path.join(src, f"{o}_counter_collection.csv")) + "\n"
                      for o, _ in passes))
    open(os.path.join(out_dir, "sq_counters_sequence_kernels_350m.md"), "w").write(text)


def write_timing_profile(path: str, r: dict, roof: dict, argv: list) -> None:
    """The HIP-event timing behind roofline.frac, written by the run that measured it: per
    timed replay of the ring's step graph, the time per step node, and the figures
    derived from them (the rocprofv3 trace of the same command serialises dispatches, so
    its durations are reported beside these, not in their place)."""
    sb = r["step_bytes"]
    st = r["step_us_per_replay"]
    lines = [
        "# Block step timing by HIP events: 350M layer shape, batch 16, L 32, 262K prefix", "",
        f"- kernel_source_sha256_16: `{kernel_source_sha('block')}`",
        f"- step_nodes_per_replay: {r['layers'] * r['denoise_steps']}",
        f"- timed_replays: {len(st)}",
        f"- step_us_mean: {np.mean(st):.4f}",
        f"- step_us_median: {np.median(st):.4f}",
        f"- step_bytes_per_launch: {sb}",
        f"- achieved_gbs: {sb / np.mean(st) / 1e3:.1f}",
        f"- frac_of_8tbs: {sb / np.mean(st) / 1e3 / HBM_PEAK_GBS:.4f}",
        f"- commit_us_mean: {np.mean(r['commit_us_per_replay']):.4f}",
        f"- stream_ceiling_gbs: {roof.get('stream_ceiling_gbs')}",
        "",
        "Each timed replay runs the ring's step graph (every layer's denoising steps, one "
        "launch per node) between two HIP events on the replay stream; the time per node is "
        "the events' interval divided by the node count.  `achieved_gbs` = algorithmic bytes "
        "per launch / `step_us_mean`, the figure `roofline.frac` is computed from.", "",
        f"Command (R = repository root; MI355X, ROCm 7.2):", "",
        f"    python3 $R/bench.py {' '.join(argv)}", "",
        "| replay | step us per node | commit us per node |", "|---|---|---|"]
    lines += [f"| {i} | {a:.4f} | {b:.4f} |" for i, (a, b) in
              enumerate(zip(st, r["commit_us_per_replay"]))]
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def copy_calibration(nbytes: int = 256 << 20, reps: int = 5):
    """A plain device-to-device copy of known size, for scaling HBM counters (FETCH_SIZE,
    WRITE_SIZE) of profiled kernels to bytes."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").uniform_()
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "reps": reps}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50, help="timed block cycles")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layers", type=int, default=32, help="layers in the cold-cache ring")
    ap.add_argument("--block-len", type=int, default=32)
    ap.add_argument("--denoise", type=int, default=8, help="denoising steps per block")
    ap.add_argument("--prefix", type=int, default=262144, help="committed prefix tokens")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds for the oracle leg")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the flatness sweep, the full-window contrast, the prefill and "
                         "the copy reference")
    ap.add_argument("--sweep-steps", type=int, default=10,
                    help="timed block cycles per point of the flatness sweep")
    ap.add_argument("--contrast-reps", type=int, default=15)
    ap.add_argument("--contrast-warmup", type=int, default=5)
    ap.add_argument("--prefill-tokens", type=int, default=16384)
    ap.add_argument("--sequence-only", action="store_true",
                    help="only time the full-window contrast and the prefill (one JSON line)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 256 MiB device copy (counter calibration) and exit")
    ap.add_argument("--summarize-trace", metavar="KERNEL_STATS_CSV",
                    help="print a markdown summary of a rocprofv3 kernel_stats.csv and exit")
    ap.add_argument("--summarize-dispatches", metavar="KERNEL_TRACE_CSV",
                    help="print per-shape kernel durations from a rocprofv3 kernel_trace.csv")
    ap.add_argument("--summarize-counters", metavar="COUNTER_COLLECTION_CSV",
                    help="print per-kernel medians of a rocprofv3 --pmc counter_collection.csv")
    ap.add_argument("--summarize-traffic-shapes", nargs=4,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="print per-dispatch HBM bytes per kernel and launch shape and exit")
    ap.add_argument("--summarize-traffic", nargs=4,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="print per-launch HBM bytes from rocprofv3 counter CSVs and exit")
    ap.add_argument("--traffic-kernels", metavar="TAG=NAME,...",
                    help="with --summarize-traffic: kernels to report (name substrings)")
    ap.add_argument("--write-block-profiles", nargs=2, metavar=("ROCPROF_DIR", "OUT_DIR"),
                    help="write the block-step profile summaries from a rocprofv3 output "
                         "directory and exit")
    ap.add_argument("--write-seq-profiles", nargs=2, metavar=("ROCPROF_DIR", "OUT_DIR"),
                    help="write the sequence/variant profile summaries from a rocprofv3 output "
                         "directory and exit")
    ap.add_argument("--timing-profile", metavar="PATH",
                    help="also write the HIP-event timing behind roofline.frac to PATH")
    ap.add_argument("--source-sha", choices=sorted(SOURCE_SETS),
                    help="print the hash of a kernel family's sources and exit")
    args = ap.parse_args()
    if args.source_sha:
        print(kernel_source_sha(args.source_sha))
        return
    if args.write_block_profiles:
        write_block_profiles(*args.write_block_profiles)
        return
    if args.write_seq_profiles:
        write_seq_profiles(*args.write_seq_profiles)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.summarize_traffic_shapes:
        print(summarize_traffic_shapes(*args.summarize_traffic_shapes))
        return
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters))
        return
    if args.summarize_dispatches:
        print(summarize_dispatches(args.summarize_dispatches))
        return
    if args.summarize_traffic:
        kern = None
        if args.traffic_kernels:
            kern = dict(kv.split("=", 1) for kv in args.traffic_kernels.split(";"))
        r = summarize_traffic(*args.summarize_traffic, kernels=kern)
        r["kernel_source_sha256_16"] = kernel_source_sha()
        r["step_alg_bytes"] = step_bytes(16, 32, 64, 128, 1, 32)
        r["commit_alg_bytes"] = commit_bytes(16, 32, 64, 128, 1, 32)
        print(json.dumps(r, indent=1))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the block step and the commit shard over "
              "(batch, head) with no exchange, so there is no multi-GPU path to time.",
              file=sys.stderr)
        sys.exit(2)

    if args.sequence_only:
        import torch
        torch.cuda.set_device(0)
        print(json.dumps({"contrast": run_contrast(args, None), "prefill": run_prefill(args),
                          "all_block": run_all_block(args), "variants": run_variants(args)}),
              flush=True)
        return

    r = run_gpu(args)
    extras = {}
    s = r["shape"]
    units, unit = step_unit_bytes(r)
    ceiling = run_stream_ceiling(unit, units)
    if not args.no_extras:
        extras["configs"] = run_other_configs(args)
        extras["copy_reference"] = run_copy_reference(r["step_bytes"])
        extras["warm"] = run_warm(args)
        extras["flatness"] = run_flatness(args)
        extras["contrast"] = run_contrast(args, r)
        extras["prefill"] = run_prefill(args)
        extras["all_block"] = run_all_block(args)
        extras["variants"] = run_variants(args)
        extras["batch_sweep"] = run_batch_sweep(args)
    cpu = None if args.no_cpu_baseline else cpu_baseline(args, args.cpu_budget)
    parity = None
    if r["sample"] is not None:
        import bdlm_inputs as bi
        parity = parity_vs_oracle(bi.WORKLOADS[3].with_block_len(args.block_len), r["sample"])
        print(f"[bench] parity vs oracle: {parity}", file=sys.stderr, flush=True)
    trace = profile_fields(TRACE_SUMMARY)
    sq = profile_fields(SQ_SUMMARY)
    rocprof_us = _num(trace, "step_kernel_mean_us")
    line = {
        "metric": "active-block tokens/s per Mamba layer (350M layer shape, batch 16, 262K "
                  "prefix); % of HBM roofline of the block step",
        "value": round(r["value"], 1),
        "unit": "tokens/s",
        # every token of the active block counts once per denoising step (the metric); a
        # block of L tokens is finalised once per cycle of p steps: value / p
        "finalised_tokens_per_s": round(r["finalised_tokens_per_s"], 1),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"350m-mamba-layer-b{s['batch']}-L{s['block_len']}-prefix{args.prefix}"
                        f"-{args.denoise}steps+commit",
            "batch": s["batch"], "nheads": s["nheads"], "headdim": s["headdim"],
            "dstate": s["dstate"], "ngroups": s["ngroups"], "block_len": s["block_len"],
            "prefix_tokens": r["prefix_tokens"], "denoise_steps": args.denoise,
            "activations": "bf16", "state": "f32", "y": "f32",
            "layer_ring": args.layers, "launch": "hip-graph replay",
            "step_us": round(r["avg_step_us"], 3),
            "step_us_median": round(r["median_step_us"], 3),
            "step_us_min": round(r["min_step_us"], 3),
            "commit_us": round(r["avg_commit_us"], 3),
            "commit_gbs": round(r["commit_gbs"], 1),
        },
        "roofline": {
            "kernel": "bdlm_block_kernel<32,128,bf16,step>",
            "bound": "hbm",
            "achieved": round(r["achieved_gbs"], 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(r["achieved_gbs"] / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic() if args.block_len == 32 else None,
            "bytes_per_launch": r["step_bytes"],
            "frac_source": "hip events on the replay stream: algorithmic bytes / mean time per "
                           "step node over the timed graph replays",
            # the same kernel's mean dispatch duration in the committed rocprofv3 kernel trace
            # of this command (null once the kernel sources differ from the traced ones)
            "kernel_us_rocprof": rocprof_us,
            "frac_rocprof": None if rocprof_us is None
            else round(r["step_bytes"] / (rocprof_us * 1e3) / HBM_PEAK_GBS, 4),
            "mfma_busy_pct": _num(sq, "step_mfma_busy_pct"),
            "stream_ceiling_gbs": None if ceiling is None else ceiling["gbs"],
            "frac_of_stream_ceiling": None if ceiling is None
            else round(r["achieved_gbs"] / ceiling["gbs"], 4),
        },
        "max_rel_err": parity,
        "cpu_baseline": cpu,
    }
    if ceiling is not None:
        line["stream_ceiling"] = ceiling
    cs = extras.get("variants", {}).get("commit_step_L32")
    if cs is not None and args.block_len == 32:
        # the same block cycle with the commit fused into the next block's first step (one
        # state read fewer per cycle; same results): p - 1 steps + the fused launch
        t = (args.denoise - 1) * r["avg_step_us"] + cs["fused_us"]
        line["fused_order"] = {
            "cycle_us_per_layer": round(t, 3),
            "value": round(args.denoise * s["batch"] * s["block_len"] / (t * 1e-6), 1),
            "note": "p - 1 steps + one commit+next-step launch per block cycle (bdlm_commit_step)"}
    if "copy_reference" in extras:
        cr = extras["copy_reference"]
        line["roofline"]["copy_same_bytes_gbs"] = cr["gbs"]
        line["roofline"]["frac_of_copy"] = round(r["achieved_gbs"] / cr["gbs"], 4)
    line.update(extras)
    if args.timing_profile:
        write_timing_profile(args.timing_profile, r, line["roofline"], sys.argv[1:])
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

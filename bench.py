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
KERNEL_SRCS = [os.path.join(ROOT, "paper_2607_02805_amd", "csrc", f)
               for f in ("bdlm_scan.hip", "bdlm_device.h")]
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "hbm_traffic_block_step_350m_b16_L32.md")
STEP_KERNEL = "bdlm_block_kernel<32, 128, false, false"
COMMIT_KERNEL = "bdlm_block_kernel<32, 128, false, true"


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


def run_gpu(args):
    import torch

    import bdlm_inputs as bi
    import paper_2607_02805_amd as bd

    dev = "cuda:0"
    torch.cuda.set_device(0)
    w = bi.WORKLOADS[3].with_block_len(args.block_len)
    Bsz, H, P, N, G, L = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups, w.block_len
    nl, p = args.layers, args.denoise

    # ---- inputs: p noised blocks + 1 clean block, copied into every layer of the ring
    steps_h = [bi.block_inputs(w, s) for s in range(p)]
    clean_h = bi.commit_inputs(w)
    base_steps = [to_dev(d, dev) for d in steps_h]
    base_clean = to_dev(clean_h, dev)
    layers = []
    for _ in range(nl):
        lay = {"steps": [{k: v.clone() for k, v in d.items()} for d in base_steps],
               "clean": {k: v.clone() for k, v in base_clean.items()},
               "y": torch.empty((Bsz, L, H, P), dtype=torch.float32, device=dev),
               "y_clean": torch.empty((Bsz, L, H, P), dtype=torch.float32, device=dev)}
        layers.append(lay)

    # ---- prefix: commit args.prefix tokens into layer 0's cache (16 seeded clean blocks
    #      cycled), then give every layer of the ring that state and bookkeeping
    t0 = time.time()
    cache0 = bd.Cache(Bsz, H, N, device=dev)
    pre = bi.prefix_inputs(w, 16 * L)
    pre_blocks = [to_dev(bi.slice_tokens(pre, L * i, L * (i + 1)), dev) for i in range(16)]
    nblk = args.prefix // L
    for k in range(nblk):
        d = pre_blocks[k % 16]
        cache0.commit(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                      expected_block_index=k)
    torch.cuda.synchronize()
    caches = []
    for _ in range(nl):
        c = bd.Cache(Bsz, H, N, device=dev)
        c.h.copy_(cache0.h)
        c.n_committed[:] = cache0.n_committed
        c.n_blocks[:] = cache0.n_blocks
        caches.append(c)
    del cache0
    torch.cuda.synchronize()
    prefill_s = time.time() - t0
    print(f"[bench] prefix of {args.prefix} tokens committed ({nblk} commits) in {prefill_s:.2f}s; "
          f"ring of {nl} layers, state {nl * Bsz * H * P * N * 4 / 2**20:.0f} MiB", flush=True)

    # ---- capture the ring's denoising steps and the ring's commits as two graphs
    stream = torch.cuda.Stream()
    g_steps, g_commit = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()

    def enqueue_steps():
        for s in range(p):
            for li in range(nl):
                d, c = layers[li]["steps"][s], caches[li]
                bd.scan_block_step(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"],
                                   c.h, y=layers[li]["y"])

    def enqueue_commits():
        for li in range(nl):
            d, c = layers[li]["clean"], caches[li]
            # bookkeeping is advanced by the host after each replay (below)
            bd.commit_boundary(d["x"], d["dt"], d["A"], d["B"], d["C"], d["D"], d["D_rev"], c.h,
                               c.n_committed.copy(), c.n_blocks.copy(), -1,
                               y_clean=layers[li]["y_clean"])

    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        enqueue_steps()          # eager warm-up of both kernels before capture
        enqueue_commits()
    stream.synchronize()
    with torch.cuda.graph(g_steps, stream=stream):
        enqueue_steps()
    with torch.cuda.graph(g_commit, stream=stream):
        enqueue_commits()
    torch.cuda.synchronize()

    def advance_books():
        for c in caches:
            c.n_committed += L
            c.n_blocks += 1

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            g_steps.replay()
            g_commit.replay()
            advance_books()
    torch.cuda.synchronize()

    # ---- timed region: exactly K block cycles
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    with torch.cuda.stream(stream):
        for k in range(args.steps):
            ev[k][0].record(stream)
            g_steps.replay()
            ev[k][1].record(stream)
            g_commit.replay()
            ev[k][2].record(stream)
            advance_books()
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall
    t_steps = sum(e[0].elapsed_time(e[1]) for e in ev) * 1e-3        # seconds
    t_commit = sum(e[1].elapsed_time(e[2]) for e in ev) * 1e-3
    t_total = ev[0][0].elapsed_time(ev[-1][2]) * 1e-3

    n_step_launch = args.steps * p * nl
    n_commit_launch = args.steps * nl
    avg_step_s = t_steps / n_step_launch
    avg_commit_s = t_commit / n_commit_launch
    per_layer_cycle_s = t_total / (args.steps * nl)
    tokens = p * Bsz * L
    value = tokens / per_layer_cycle_s
    sb = step_bytes(Bsz, H, P, N, G, L)
    cb = commit_bytes(Bsz, H, P, N, G, L)
    achieved = sb / avg_step_s / 1e9
    res = {
        "value": value,
        "ms_per_step": t_total / args.steps * 1e3,
        "wall_s": wall_s,
        "avg_step_us": avg_step_s * 1e6,
        "avg_commit_us": avg_commit_s * 1e6,
        "step_bytes": sb,
        "commit_bytes": cb,
        "achieved_gbs": achieved,
        "commit_gbs": cb / avg_commit_s / 1e9,
        "prefix_tokens": int(caches[0].n_committed[0]),
        "shape": dict(batch=Bsz, nheads=H, headdim=P, dstate=N, ngroups=G, block_len=L),
    }
    return res


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
    return {"value": tokens / el, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{cycles} full block cycles ({args.denoise} steps + commit) of one layer "
                      f"at batch {w.batch}, 32 heads, dstate 128, L {w.block_len}; "
                      f"{el:.1f} s, fp64"}


def kernel_source_sha() -> str:
    """Hash of the sources the block-step kernel is compiled from."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per step launch from the committed counter summary, or None when the
    kernel source changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    kv = {}
    for line in open(TRAFFIC_SUMMARY):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            kv[k.strip()] = v.strip().strip("`")
    if kv.get("kernel_source_sha256_16") != kernel_source_sha():
        return None
    try:
        return int(kv["step_hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


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


def summarize_traffic(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv,
                      copy_bytes=256 << 20) -> dict:
    """Per-launch HBM bytes of the step and commit kernels from FETCH_SIZE / WRITE_SIZE
    (KiB per dispatch), each scaled by the same counter's reading for a plain copy of
    known size."""
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
    for tag, key in (("step", STEP_KERNEL), ("commit", COMMIT_KERNEL)):
        fk = [v for k, vs in per_kernel(fetch_csv, "FETCH_SIZE").items() if key in k for v in vs]
        wk = [v for k, vs in per_kernel(write_csv, "WRITE_SIZE").items() if key in k for v in vs]
        res[tag] = {"fetch_kib_median": st.median(fk), "write_kib_median": st.median(wk),
                    "dispatches": len(fk),
                    "fetch_bytes": int(st.median(fk) * 1024 * f_scale),
                    "write_bytes": int(st.median(wk) * 1024 * w_scale)}
    return res


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
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 256 MiB device copy (counter calibration) and exit")
    ap.add_argument("--summarize-trace", metavar="KERNEL_STATS_CSV",
                    help="print a markdown summary of a rocprofv3 kernel_stats.csv and exit")
    ap.add_argument("--summarize-traffic", nargs=4,
                    metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="print per-launch HBM bytes from rocprofv3 counter CSVs and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.summarize_traffic:
        r = summarize_traffic(*args.summarize_traffic)
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

    r = run_gpu(args)
    cpu = None if args.no_cpu_baseline else cpu_baseline(args, args.cpu_budget)
    s = r["shape"]
    line = {
        "metric": "active-block tokens/s per Mamba layer (350M layer shape, batch 16, 262K "
                  "prefix); % of HBM roofline of the block step",
        "value": round(r["value"], 1),
        "unit": "tokens/s",
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
            "workload": f"350m-mamba-layer-b{s['batch']}-L{s['block_len']}-prefix{r['prefix_tokens']}"
                        f"-{args.denoise}steps+commit",
            "batch": s["batch"], "nheads": s["nheads"], "headdim": s["headdim"],
            "dstate": s["dstate"], "ngroups": s["ngroups"], "block_len": s["block_len"],
            "prefix_tokens": r["prefix_tokens"], "denoise_steps": args.denoise,
            "activations": "bf16", "state": "f32", "y": "f32",
            "layer_ring": args.layers, "launch": "hip-graph replay",
            "step_us": round(r["avg_step_us"], 3), "commit_us": round(r["avg_commit_us"], 3),
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
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()

"""Host-side parts of bench.py: the one-GPU contract, the algorithmic byte counts the
roofline divides by, and the profile summaries (no GPU needed)."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_algorithmic_bytes_at_the_350m_layer_shape():
    # state 16 x 32 x 64 x 128 fp32, x 16 x 32 x 32 x 64 bf16, dt 16 x 32 x 32 bf16,
    # B and C 2 x 16 x 32 x 128 bf16, y 16 x 32 x 32 x 64 fp32, A / D / D_rev 3 x 32 fp32
    state, x, dt, bc, y, par = 16777216, 2097152, 32768, 262144, 4194304, 384
    assert bench.step_bytes(16, 32, 64, 128, 1, 32) == state + x + dt + bc + y + par == 23363968
    assert bench.commit_bytes(16, 32, 64, 128, 1, 32) == 23363968 + state == 40141184
    # the full window reads its inputs and writes y once, and has no state
    assert bench.full_window_bytes(4, 32, 64, 128, 1, 65536) == 3372220800
    # bytes grow with the block's tokens only, never with the prefix
    assert (bench.step_bytes(16, 32, 64, 128, 1, 64) - bench.step_bytes(16, 32, 64, 128, 1, 32)
            == x + dt + bc + y)


def test_dispatch_summary_groups_by_kernel_and_shape(tmp_path):
    p = tmp_path / "trace.csv"
    rows = ["Kernel_Name,Grid_Size_X,Workgroup_Size_X,Start_Timestamp,End_Timestamp"]
    for i, (grid, dur) in enumerate([(262144, 6000), (262144, 7000), (262144, 8000),
                                     (2097152, 40000)]):
        rows.append(f"\"void bdlm::(anonymous namespace)::bdlm_k<32, 128>(x)\",{grid},512,"
                    f"{1000 * i},{1000 * i + dur}")
    rows.append("\"elementwise_other\",1024,256,0,5000")
    p.write_text("\n".join(rows) + "\n")
    table = bench.summarize_dispatches(str(p)).splitlines()
    assert len(table) == 4                       # header, rule, one row per launch shape
    assert "| 4096 x 512 | 1 | 40.00 | 40.00 | 40.00 |" in table[2]
    assert "| 512 x 512 | 3 | 7.00 | 7.00 | 6.00 |" in table[3]
    assert not any("elementwise_other" in t for t in table)


def test_traffic_is_dropped_once_the_kernel_source_changes(monkeypatch):
    good = bench.kernel_source_sha()
    value = bench.measured_traffic()
    if value is not None:                          # summary taken on the current source
        assert value > bench.step_bytes(16, 32, 64, 128, 1, 32) * 0.9
    monkeypatch.setattr(bench, "kernel_source_sha",
                        lambda which="block": "0" * 16 if good != "0" * 16 else "1" * 16)
    assert bench.measured_traffic() is None


def test_profile_fields_need_a_matching_source_hash(tmp_path, monkeypatch):
    p = tmp_path / "summary.md"
    p.write_text(f"# x\n\n- kernel_source_sha256_16: `{bench.kernel_source_sha()}`\n"
                 "- step_kernel_mean_us: 6.25\n- note: a: b\n")
    kv = bench.profile_fields(str(p))
    assert bench._num(kv, "step_kernel_mean_us") == 6.25 and kv["note"] == "a: b"
    assert bench._num(kv, "missing") is None
    monkeypatch.setattr(bench, "kernel_source_sha", lambda which="block": "f" * 16)
    assert bench.profile_fields(str(p)) == {}
    assert bench.profile_fields(str(tmp_path / "absent.md")) == {}


def test_source_sets_name_existing_files():
    for which, files in bench.SOURCE_SETS.items():
        for f in files:
            assert os.path.exists(os.path.join(bench.CSRC, f)), (which, f)
        assert len(bench.kernel_source_sha(which)) == 16


def test_timing_profile_recomputes_the_fraction(tmp_path):
    """The timing summary the bench writes holds what roofline.frac is computed from: the
    mean time per step node over the timed replays and the algorithmic bytes."""
    sb = bench.step_bytes(16, 32, 64, 128, 1, 32)
    r = {"step_bytes": sb, "step_us_per_replay": [6.2, 6.3, 6.25],
         "commit_us_per_replay": [9.1, 9.2, 9.3], "layers": 32, "denoise_steps": 8}
    p = tmp_path / "timing.md"
    bench.write_timing_profile(str(p), r, {"stream_ceiling_gbs": 4000.0}, ["--steps", "3"])
    kv = bench.profile_fields(str(p))
    mean = bench._num(kv, "step_us_mean")
    assert abs(mean - 6.25) < 1e-9
    frac = sb / (mean * 1e3) / bench.HBM_PEAK_GBS
    assert abs(bench._num(kv, "frac_of_8tbs") - frac) < 1e-4
    assert bench._num(kv, "timed_replays", int) == 3

"""Host-side logic of bench.py (no GPU): the algorithmic byte counts, the guard against
several GPUs, and the rule that a committed counter summary is used only for the kernel
sources it was taken on."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import workloads as W  # noqa: E402


def test_bytes_per_nts():
    f32 = bench.bytes_per_nts(W.WORKLOADS["conv"])
    assert f32["lif_forward"] == 5 and f32["lif_backward"] == 12
    assert f32["gain_forward"] == 5 and f32["gain_backward"] == 8
    assert f32["lif_forward_gain"] == 2 and f32["lif_backward_gain"] == 9
    bf = bench.bytes_per_nts(W.WORKLOADS["large"])
    assert bf["lif_forward"] == 2.125 and bf["lif_backward"] == 6
    assert bf["lif_forward_gain"] == 0.25 and bf["lif_backward_gain"] == 4.125
    # a 3-layer stack moves 77 B per position layer by layer, 39 B fused across the gain,
    # 17 B fused across depth
    unfused = 3 * (f32["lif_forward"] + f32["lif_backward"]) + 2 * (f32["gain_forward"] + f32["gain_backward"])
    fused = f32["lif_forward"] + f32["lif_backward"] + 2 * (f32["lif_forward_gain"] + f32["lif_backward_gain"])
    depth = f32["lif_stack_forward"] + f32["lif_stack_backward"]
    assert (unfused, fused, depth) == (77, 39, 17)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_traffic_only_for_current_sources(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    tag = "conv_T16_N8388608"
    assert bench.measured_traffic("lif_backward", tag) is None          # no summary
    path = tmp_path / f"lif_backward_{tag}_pmc.md"
    path.write_text(f"source_sha256_16: {bench.source_hash()}\n\ntraffic_bytes_per_launch: 1.5e+09\n")
    assert bench.measured_traffic("lif_backward", tag) == pytest.approx(1.5e9)
    path.write_text("source_sha256_16: 0000000000000000\n\ntraffic_bytes_per_launch: 1.5e+09\n")
    assert bench.measured_traffic("lif_backward", tag) is None          # taken on other sources


def test_committed_summaries_parse():
    """Every committed PMC summary names its source hash and a traffic figure."""
    names = [n for n in os.listdir(bench.PROFILES) if n.endswith("_pmc.md")]
    assert names
    for n in names:
        text = open(os.path.join(bench.PROFILES, n)).read()
        assert "source_sha256_16:" in text and "traffic_bytes_per_launch:" in text, n
        assert "rocprofv3 --pmc FETCH_SIZE" in text and "rocprofv3 --pmc WRITE_SIZE" in text, n


def test_source_hash_ignores_comments_only(tmp_path):
    """The hash that ties profiles to kernel code changes with the code, not with comments."""
    src = tmp_path / "k.hip"
    src.write_text("// leading note\nint f(int a) {  /* old */ return a + 1; }  // tail\n")
    before = bench.source_hash(str(tmp_path))
    src.write_text("// a reworded note\n/* a new block\n   comment */\nint f(int a) {\n    return a + 1;\n}\n")
    assert bench.source_hash(str(tmp_path)) == before
    src.write_text("int f(int a) { return a + 2; }\n")
    assert bench.source_hash(str(tmp_path)) != before


def test_host_info_and_sampling():
    info = bench.host_info()
    assert info["oracle_cflags"] and "-ffp-contract=off" in info["oracle_cflags"]
    assert info["threads_allowed"] >= 1
    cols = bench.sample_columns(1 << 20)
    assert cols.size == 4096 and cols[0] == 0 and cols[-1] == (1 << 20) - 1
    assert list(cols[:1024]) == list(range(1024)) and (cols[1:] > cols[:-1]).all()
    assert list(bench.sample_columns(100)) == list(range(100))


def test_pinned_single_core_oracle_timing():
    """The pinned single-core leg times forward and backward separately and restores the
    thread's core mask afterwards."""
    import oracle
    w = W.custom("tiny", 6, 300, W.HARD_05)
    before = os.sched_getaffinity(0)
    one = bench._pinned_single_core(oracle.Params.of(w.params), W.x_full(w), W.gs_full(w), None, w.F)
    assert os.sched_getaffinity(0) == before
    assert one["reps"] == 3 and len(one["forward_s"]) == 3 and one["backward_s_median"] > 0


def test_other_configs_are_workloads():
    """The default run's extra configurations name real workloads and schedules."""
    names = [n for n, _ in bench.OTHER_CONFIGS]
    assert len(set(names)) == len(names)
    for _, over in bench.OTHER_CONFIGS:
        w = W.WORKLOADS[over["workload"]]
        if "T" in over:
            assert w.name == "large" and over["T"] in W.LARGE_T
        if over.get("fused_stack") or over.get("depth_stack"):
            assert w.layers > 1
    assert {o.get("T") for _, o in bench.OTHER_CONFIGS if o["workload"] == "large"} == set(W.LARGE_T)

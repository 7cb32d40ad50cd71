"""The benchmark harness: its one-line JSON contract (GPU, in this process, on
the tiny workload) and its refusal of several GPUs (CPU)."""

import contextlib
import io
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_bench_warmup_defaults_by_op(monkeypatch):
    """Attention's default warmup covers the ~25 ms its step needs to reach
    steady clocks after the GPU idled; an explicit --warmup is kept as given."""
    import bench

    for argv, want in ((["--op", "attention"], 200), ([], 10), (["--op", "table3"], 10),
                       (["--op", "attention", "--warmup", "3"], 3),
                       (["--warmup", "0"], 0)):
        monkeypatch.setattr(sys, "argv", ["bench.py", *argv])
        assert bench.parse().warmup == want, argv


def test_attention_row_reports_a_failure_instead_of_raising():
    """The transfer line's decode-attention row never costs the line: where
    the attention step cannot run (here: no GPU) the row holds the error."""
    import torch

    import bench

    if torch.cuda.is_available():
        pytest.skip("a GPU is present: the row would run")
    row = bench.attention_context(3)
    assert set(row) <= {"error", "allocated_gib"} and row["error"]


def run_bench(*args):
    import bench

    out = io.StringIO()
    argv = sys.argv
    sys.argv = ["bench.py", *args]
    try:
        with contextlib.redirect_stdout(out):
            bench.main()
    finally:
        sys.argv = argv
    lines = [l for l in out.getvalue().splitlines() if l.strip()]
    assert len(lines) == 1, lines
    return json.loads(lines[0])


@pytest.mark.gpu
@pytest.mark.parametrize("layout", ["block", "layer"])
def test_bench_line_contract_on_tiny(layout):
    j = run_bench("--workload", "tiny", "--layout", layout, "--steps", "3", "--warmup", "1",
                  "--no-context")
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in j, key
    assert j["n_gpus"] == 1 and j["steps"] == 3 and j["warmup"] == 1
    assert j["value"] > 0 and j["ms_per_step"] > 0
    assert j["config"]["workload"].startswith("tiny") and j["config"]["blocks"] == 16
    rf = j["roofline"]
    assert rf["bound"] == "hbm" and rf["peak"] == 8000.0 and rf["unit"] == "GB/s"
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    cb = j["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0


def test_receiver_pool_shrinks_to_fit():
    """Where the device cannot hold both 65,536-block pools of the 13k
    request, the receiver's pool shrinks to the largest multiple of 4,096
    blocks that fits beside the sender's (and the request still fits)."""
    import bench
    from paper_2504_03775_amd import flowkv as fk
    from workloads import recipes

    BB, GiB = 2 << 20, 1 << 30
    r = bench.RESERVE_BYTES
    assert bench.fit_receiver_blocks(300 * GiB, 65536, 65536, BB) == 65536
    assert bench.fit_receiver_blocks(256 * GiB + r, 65536, 65536, BB) == 65536
    assert bench.fit_receiver_blocks(256 * GiB + r - 1, 65536, 65536, BB) == 61440
    assert bench.fit_receiver_blocks(200 * GiB + r, 65536, 65536, BB) == 36864
    assert bench.fit_receiver_blocks(128 * GiB + r + 4095 * BB, 65536, 65536, BB) == 0
    wl = recipes.llama8b_13k(lambda P, pol, seed: fk.Allocator(P, pol, seed), "segment",
                             dst_pool_blocks=36864)
    (S, D), = wl.tables
    assert wl.src_pool_blocks == 65536 and wl.dst_pool_blocks == 36864
    assert len(D) == 813 and D.max() < 36864 and len(set(D.tolist())) == 813


def test_traffic_is_reported_only_for_the_profiled_kernel_and_plan(tmp_path):
    """roofline.traffic comes from a committed counter summary only while the
    kernel source hash, the plan's run count and (attention) the split length
    match what the counters were taken on."""
    import bench

    src = tmp_path / "k.hip"
    src.write_text("kernel v1")
    h = bench.kernel_hash(str(src))
    summ = tmp_path / "pmc.txt"
    summ.write_text(f"algorithmic bytes: ... (payload 1, 255 runs x 16 B plan)\n"
                    f"split_tokens: 1024\nhbm_bytes_per_launch: 3410881152\n"
                    f"kernel_source_sha256_16: {h}\n")
    f = bench.traffic_from_profile
    assert f(str(summ), str(src)) == 3410881152.0
    assert f(str(summ), str(src), runs=255, split=1024) == 3410881152.0
    assert f(str(summ), str(src), runs=43) is None
    assert f(str(summ), str(src), split=256) is None
    assert f(str(tmp_path / "absent.txt"), str(src)) is None
    src.write_text("kernel v2")
    assert f(str(summ), str(src)) is None


def test_schedule_line_contract_on_cpu():
    """bench.py --op schedule runs on the host alone: one JSON line with the
    scheduler's rate, the oracle beside it and the cluster model's mixes."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--op", "schedule",
                        "--steps", "20", "--warmup", "2"],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    j = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline", "context"):
        assert key in j, key
    assert j["value"] > 0 and j["roofline"] is None and j["dtype"] == "f64"
    assert j["cpu_baseline"]["kind"] == "oracle" and j["cpu_baseline"]["value"] > 0
    sim = j["context"]["cluster_model_2p2d"]
    assert set(sim) == {"balanced", "prefill-heavy", "decode-heavy", "busy-then-quiet"}
    dh = sim["decode-heavy"]
    assert dh["load_aware"]["requests_per_s"] > dh["fixed"]["requests_per_s"]
    bq = sim["busy-then-quiet"]
    assert bq["scaling_with_spares"]["node_seconds"] < bq["four_fixed_nodes"]["node_seconds"]
    assert bq["scaling_with_spares"]["scale_downs"][0] >= 1


@pytest.mark.gpu
def test_timing_events_bracket_the_same_work_as_torch_events():
    """bench.py's timing events (no system fence) measure what torch's
    events measure: a pair nested inside a torch pair around five 1 GiB
    copies reads at most the outer interval and at least 90% of it."""
    import torch

    import bench

    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    outer = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    inner = bench.timing_pairs(1)[0]
    assert bench.TIMING["events"].startswith("hip"), bench.TIMING
    outer[0].record()
    inner[0].record()
    for _ in range(5):
        b.copy_(a)
    inner[1].record()
    outer[1].record()
    torch.cuda.synchronize()
    mi, mo = inner[0].elapsed_time(inner[1]), outer[0].elapsed_time(outer[1])
    assert 0.9 * mo <= mi <= mo * 1.01 + 0.01, (mi, mo)


@pytest.mark.gpu
def test_attention_line_contract():
    j = run_bench("--op", "attention", "--attn-workload", "70b", "--steps", "3", "--warmup", "1",
                  "--no-context", "--no-cpu-baseline")
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline"):
        assert key in j, key
    assert j["config"]["kv_heads"] == 1 and j["config"]["q_heads"] == 8
    assert j["config"]["split_tokens"] == 1024 and j["value"] > 0
    assert j["roofline"]["bound"] == "hbm"


@pytest.mark.gpu
def test_overlap_line_contract():
    """bench.py --op overlap: the prefill stand-in alone and with the three
    transfer forms, each timed; one JSON line in the same contract."""
    j = run_bench("--op", "overlap", "--steps", "2", "--warmup", "1")
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in j, key
    assert j["unit"] == "ms" and j["higher_is_better"] is False
    assert set(j["median_ms"]) == {"prefill", "one_launch_after", "layerwise_overlap",
                                   "layerwise_after"}
    assert all(v > 0 for v in j["median_ms"].values())
    assert j["value"] == j["exposed_ms"]["layerwise_overlap"]
    assert j["config"]["tokens"] == 13000 and j["config"]["layers"] == 32


@pytest.mark.gpu
def test_table3_line_contract():
    """bench.py --op table3: one launch and 32 per-layer launches at each
    length asked for, each timed three ways, the ratio per length, and the
    paper's two columns beside them as context."""
    j = run_bench("--op", "table3", "--lengths", "500,4000", "--steps", "3", "--warmup", "1")
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline", "rows"):
        assert key in j, key
    assert j["unit"] == "ms" and j["higher_is_better"] is False and j["vs_baseline"] is None
    assert [r["tokens"] for r in j["rows"]] == [500, 4000]
    for r in j["rows"]:
        assert r["blocks"] == -(-r["tokens"] // 16)
        assert r["one_launch"]["launches"] == 1 and r["layerwise"]["launches"] == 32
        assert r["layerwise_graph"]["launches"] == 32 and r["layerwise_graph"]["kernel_ms_median"] > 0
        for form in ("one_launch", "layerwise"):
            assert all(r[form][k] > 0 for k in ("kernel_ms_median", "ms_per_step",
                                                 "latency_ms_median"))
        assert set(r["paper_s_single_l20"]) == {"flowkv", "flowkv_layerwise"}
    assert j["value"] == pytest.approx(
        sum(r["one_launch"]["latency_ms_median"] for r in j["rows"]) / 2, abs=1e-3)

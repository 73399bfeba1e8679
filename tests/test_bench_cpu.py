"""Host-side pieces of bench.py: the one-GPU guard, the GEMM launch-grid
labelling used by the profile summaries, and the traffic record check."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2402_15627_amd.inputs import WORKLOADS  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_gemm_grid_matches_the_split_plan():
    s = WORKLOADS["175b_tp8_share"]
    steps = bench.gemm_steps(s)
    # dw_in: 42 x 48 = 2016 tiles, tail of 224 is too large to split
    assert bench.gemm_grid_threads(*steps["dw_in"]) == 2016 * 512
    # out_proj: 8 x 48 = 384 tiles -> 256 whole + 128 tail tiles split 2 ways
    assert bench.gemm_grid_threads(*steps["out_proj"]) == (256 + 128 * 2) * 512
    # in_proj: 8 x 42 = 336 tiles -> 256 + 80 tail tiles split 3 ways
    assert bench.gemm_grid_threads(*steps["in_proj"]) == (256 + 80 * 3) * 512
    # fewer tiles than CUs: 4 tiles, 64 K-steps -> 16 slices of 4 K-steps
    assert bench.gemm_grid_threads(512, 512, 4096) == 4 * 16 * 512
    # one tile, four K-steps: a reduction would cost more than it saves
    assert bench.gemm_grid_threads(128, 256, 256) == 512
    # K not a multiple of 64: unsplit
    assert bench.gemm_grid_threads(2048, 12288 + 256, 1000) == 8 * 49 * 512


def test_gemm_steps_are_told_apart():
    s = WORKLOADS["175b_tp8_share"]
    name = "void pb::(anonymous namespace)::gemm_bf16_dma_kernel<true, true, (pb::Epi)2, true>()"
    g = bench.gemm_grid_threads(*bench.gemm_steps(s)["out_proj"])
    assert bench.gemm_step_of(name, g, s) == "out_proj"
    dh = name.replace("<true, true, (pb::Epi)2", "<true, false, (pb::Epi)4")
    assert bench.gemm_step_of(dh, g, s) == "dh"   # same grid, other template
    assert bench.gemm_step_of(name, g + 512, s) == ""


def test_traffic_is_reported_only_for_unchanged_sources(tmp_path, monkeypatch):
    rec = {"traffic_bytes": 123, "source_fingerprint": bench.source_fingerprint("dw_in")}
    path = tmp_path / "dw_in_x_traffic.md"
    path.write_text(f"# t\n\n```json\n{json.dumps(rec)}\n```\n")
    monkeypatch.setattr(bench, "traffic_path", lambda step, wl: str(path))
    assert bench.read_traffic("dw_in", "x") == 123
    rec["source_fingerprint"] = "0" * 16
    path.write_text(f"# t\n\n```json\n{json.dumps(rec)}\n```\n")
    assert bench.read_traffic("dw_in", "x") is None
    monkeypatch.setattr(bench, "traffic_path", lambda step, wl: str(tmp_path / "missing.md"))
    assert bench.read_traffic("dw_in", "x") is None


def test_committed_traffic_profile_parses():
    p = bench.traffic_path("dh+dw_in", "175b_tp8_share")
    if not os.path.exists(p):
        pytest.skip("no traffic profile committed")
    text = open(p).read()
    assert "rocprofv3 --pmc FETCH_SIZE" in text and "rocprofv3 --pmc WRITE_SIZE" in text
    rec = json.loads(text.split("```json\n")[1].split("\n```")[0])
    assert rec["traffic_bytes"] > 0 and rec["algorithmic_bytes"] > 0


def test_serial_gemm_steps_are_labelled():
    """Every GEMM of the serial block is found by kernel template and grid;
    dW_down and dW_up (1152 tiles each, same template) share a label."""
    s = WORKLOADS["175b_tp8_share"]
    steps = bench.gemm_steps(s, "serial")
    assert len(steps) == 12
    sig = {k: bench.GEMM_SIGNATURE[k] for k in steps}
    labels = set()
    for st, mnk in steps.items():
        name = f"void pb::(anonymous namespace)::gemm_bf16_dma_kernel{sig[st]}, true>()"
        lab = bench.gemm_step_of(name, bench.gemm_grid_threads(*mnk), s, "serial")
        assert st in lab.split("/"), (st, lab)
        labels.add(lab)
    assert "dw_down/dw_up" in labels
    # paired launches of the serial backward: dG + dW_down, 8 x 24 + 48 x 24 tiles
    pair = ("void pb::(anonymous namespace)::gemm_bf16_dma_pair<true, false, (pb::Epi)3, "
            "false, false, (pb::Epi)0, true>()")
    assert bench.gemm_step_of(pair, (192 + 1152) * 512, s, "serial") == "dg+dw_down"
    # 48 tiles of the dO GEMM, K = 12288: 5 slices each
    assert bench.gemm_grid_threads(*steps["d_o"]) == 48 * 5 * 512


def test_paired_gemm_launches_are_labelled_and_counted():
    """The backward's dC + dW_out and dh + dW_in share one launch each: the
    pair kernel is found by its first GEMM's template and the two tile
    counts, and the pair's step carries both GEMMs' FLOPs."""
    s = WORKLOADS["175b_tp8_share"]
    assert bench.paired_steps(s) == {"dc": "dw_out", "dh": "dw_in"}
    assert bench.paired_steps(s, "serial") == bench.SERIAL_GEMM_PAIRS
    assert bench.paired_steps(WORKLOADS["tiny_f32"]) == {}
    name = ("void pb::(anonymous namespace)::gemm_bf16_dma_pair<true, false, (pb::Epi)4, "
            "false, false, (pb::Epi)0, true>()")
    # dh: 8 x 48 tiles, dW_in: 42 x 48 tiles, unsplit
    assert bench.gemm_step_of(name, (384 + 2016) * 512, s) == "dh+dw_in"
    assert bench.gemm_step_of(name, 384 * 512, s) == ""
    dc = name.replace("(pb::Epi)4", "(pb::Epi)3")
    # dC: 8 x 30 tiles, dW_out: 48 x 30 tiles
    assert bench.gemm_step_of(dc, (240 + 1440) * 512, s) == "dc+dw_out"
    # the persistent form: one workgroup per CU
    pers = name.replace("gemm_bf16_dma_pair<", "gemm_bf16_dma_pair_persistent<")
    assert bench.gemm_step_of(pers, 256 * 512, s) == "dh+dw_in"
    assert bench.gemm_step_of(pers, (384 + 2016) * 512, s) == ""
    # serial block: dG + dW_down and dO + dW_o share the template and the grid
    pers_dc = pers.replace("(pb::Epi)4", "(pb::Epi)3")
    assert bench.gemm_step_of(pers_dc, 256 * 512, s, "serial") == "dg+dw_down/d_o+dw_o"
    work, plain = bench.step_work(s), bench._step_work(s)
    assert work["dh"][1] == plain["dh"][1] + plain["dw_in"][1] and work["dw_in"][1] == 0
    assert work["dc"][1] == plain["dc"][1] + plain["dw_out"][1] and work["dw_out"][1] == 0
    assert sum(v for k, v in work.values() if k == "mfma") == \
        sum(v for k, v in plain.values() if k == "mfma")
    assert bench.launch_key("dh", s) == "dh+dw_in" and bench.launch_key("in_proj", s) == "in_proj"
    assert bench.traffic_path("dh+dw_in", "w").endswith("dh_dw_in_w_traffic.md")

"""Host logic of bench.py (CPU): the one-GPU contract, the attribution of
rocprofv3 kernel names to the timed classes, and the HBM traffic summary
(FETCH_SIZE / WRITE_SIZE scaled by what the same counters read for a device
copy of known size) with its source-hash check."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, timeout=120, cwd=ROOT)


@pytest.mark.parametrize("extra", [(), ("--ablation",)])
def test_more_than_one_gpu_is_refused(extra):
    r = _run_bench("--gpus", "2", *extra)
    assert r.returncode == 2
    assert r.stdout.strip() == ""
    if not extra:
        assert "one GPU" in r.stderr


@pytest.mark.parametrize("name,cls", [
    ("void wam::gemm::gemm_bf16_kernel<256, 256, 2, 4, 2, 64, 3, 0, false>(wam::GemmArgs)", "gemm_qkv"),
    ("void wam::gemm::gemm_bf16_kernel<256, 256, 2, 4, 2, 64, 2, 1, false>(wam::GemmArgs)", "gemm_proj"),
    ("void wam::gemm::gemm_bf16_kernel<320, 256, 2, 4, 2, 64, 1, 2, false>(wam::GemmArgs)", "gemm_fc1"),
    ("void wam::gemm::gemm_bf16_kernel<64, 64, 2, 2, 4, 64, 2, 3, true>(wam::GemmArgs)", "gemm_fc2"),
    ("void wam::gemm::gemm_splitk_reduce_kernel<2, 3>(wam::GemmArgs, int)", "gemm_fc2"),
    ("void wam::(anonymous namespace)::attn_bf16_kernel<4, 8, 2, true, 1>(wam::AttnArgs)", "attention"),
    ("void wam::(anonymous namespace)::rr_gate_partials_kernel<8>(wam::RRGateArgs)", "rr_gate"),
    ("wam::(anonymous namespace)::rr_gate_finish_kernel(wam::RRGateArgs)", "rr_gate"),
    ("wam::(anonymous namespace)::rr_inject_kernel(float*, float const*, double const*, int)", "rr_inject"),
    ("wam::(anonymous namespace)::rr_refresh_kernel(float const*, float const*, float*, long, int const*)",
     "rr_refresh"),
    ("void wam::(anonymous namespace)::final_kernel<4, 4, 6, 8>(wam::FinalArgs)", None),
    ("__amd_rocclr_copyBuffer", None),
])
def test_kernel_class(name, cls):
    assert bench.kernel_class(name) == cls


_FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _pmc_csv(path, counter, rows):
    with open(path, "w") as f:
        f.write(",".join(_FIELDS) + "\n")
        for i, (name, value) in enumerate(rows):
            f.write(f'{i},"{name}",{counter},{value},0,1000\n')


def test_traffic_summary_scales_by_the_copy_and_checks_the_source_hash(tmp_path, monkeypatch):
    attn = "void wam::(anonymous namespace)::attn_bf16_kernel<4, 8, 2, true, 1>(wam::AttnArgs)"
    gate = ("void wam::(anonymous namespace)::rr_gate_partials_kernel<8>(wam::RRGateArgs)",
            "wam::(anonymous namespace)::rr_gate_finish_kernel(wam::RRGateArgs)")
    # a 1 GiB copy reads as 524288 FETCH units (2048 bytes each) and 1048576
    # WRITE units (1024 bytes each); attention's two dispatches average 2000
    # and 400 units, the gate's two kernels add up per launch
    fetch, write = tmp_path / "fetch.csv", tmp_path / "write.csv"
    _pmc_csv(fetch, "FETCH_SIZE", [("__amd_rocclr_copyBuffer", 524288), (attn, 1000), (attn, 3000),
                                   (gate[0], 90000), (gate[1], 10)])
    _pmc_csv(write, "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 1048576), (attn, 300), (attn, 500),
                                   (gate[0], 100), (gate[1], 20)])
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "traffic_path", lambda w: str(out))
    bench.summarize_pmc(str(fetch), str(write), 1024, "large", ["fetch cmd", "write cmd"])
    t = json.loads(out.read_text())
    assert t["scale"] == {"read": 2048.0, "write": 1024.0}
    assert t["classes"]["attention"]["traffic_bytes"] == 2000 * 2048.0 + 400 * 1024.0
    assert t["classes"]["rr_gate"]["traffic_bytes"] == (90000 + 10) * 2048.0 + (100 + 20) * 1024.0
    assert t["commands"] == ["fetch cmd", "write cmd"]
    assert bench.lookup_traffic("large", "attention") == 2000 * 2048.0 + 400 * 1024.0
    assert bench.lookup_traffic("large", "gemm_qkv") is None
    # a summary taken for other kernel sources is not used
    t["source_hash"] = "0" * 16
    out.write_text(json.dumps(t))
    assert bench.lookup_traffic("large", "attention") is None


def test_committed_traffic_summaries_are_complete():
    """Each committed summary carries the hash of the HIP sources it was
    measured with (the bench reports no traffic for other sources), the two
    commands that produced it and a traffic figure per timed class."""
    for w in ("large", "mid", "replay"):
        with open(os.path.join(ROOT, "profiles", f"pmc_traffic_{w}.json")) as f:
            t = json.load(f)
        assert len(t["source_hash"]) == 16, w
        assert set(t["classes"]) == set(bench.CLASS_NAMES), w
        assert len(t["commands"]) == 2 and "FETCH_SIZE" in t["commands"][0] and "WRITE_SIZE" in t["commands"][1]
        assert t["classes"]["attention"]["traffic_bytes"] > 0


@pytest.mark.parametrize("name", ["small", "mid", "large"])
def test_class_flops_follow_the_layer_formula(name):
    """The four projections of a layer add up to 24 B T D^2 (F = 4 D) and
    attention is 4 B T^2 D; at the large model 576.2 and 636.2 GFLOP."""
    from synth import get_workload
    spec = get_workload(name)
    gemm = sum(bench.class_flops(spec, c) for c in ("gemm_qkv", "gemm_proj", "gemm_fc1", "gemm_fc2"))
    assert spec.F == 4 * spec.D
    assert gemm == 24.0 * spec.B * spec.T * spec.D ** 2
    assert bench.class_flops(spec, "attention") == 4.0 * spec.B * spec.T ** 2 * spec.D
    if name == "large":
        assert round(gemm / 1e9, 1) == 576.2
        assert round(bench.class_flops(spec, "attention") / 1e9, 1) == 636.2


def test_mfma_summary_formulas(tmp_path, monkeypatch):
    """Hardware FLOP = MOPS x 512; MFMA busy = busy cycles over one XCD's
    active cycles (GRBM_GUI_ACTIVE / 8) x 1024 SIMDs; clock = those cycles
    over the dispatch time."""
    from synth import get_workload
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    spec = get_workload("large")
    name = "void wam::gemm::gemm_bf16_kernel<256, 256, 2, 4, 2, 64, 3, 0, false>(wam::GemmArgs)"
    ns = 130_000.0  # one dispatch of 130 us
    active = 2.4 * ns  # cycles of one XCD at 2.4 GHz
    mops = bench.class_flops(spec, "gemm_qkv") / 512.0
    busy = 0.5 * active * 1024
    csv_path = tmp_path / "mfma.csv"
    with open(csv_path, "w") as f:
        f.write(",".join(_FIELDS) + "\n")
        for counter, value in (("SQ_INSTS_VALU_MFMA_MOPS_BF16", mops), ("SQ_VALU_MFMA_BUSY_CYCLES", busy),
                               ("GRBM_GUI_ACTIVE", 8 * active), ("SQ_BUSY_CU_CYCLES", 1.0)):
            f.write(f'7,"{name}",{counter},{value},0,{int(ns)}\n')
    bench.summarize_mfma(str(csv_path), "large", ["pmc cmd"])
    text = (tmp_path / "profiles" / "mfma_counters_large.md").read_text()
    row = [r for r in text.splitlines() if r.startswith("| gemm_qkv")][0].split("|")
    cells = [c.strip() for c in row[1:-1]]
    # class, dispatches, avg us, alg GFLOP, hw GFLOP, hw/alg, TFLOP/s, % of peak, busy, clock, issue
    assert cells[1] == "1" and cells[2] == "130.00"
    assert cells[3] == cells[4] == "144.05" and cells[5] == "1.0000"
    assert cells[8] == "50.0%" and cells[9] == "2.400"
    assert cells[6] == f"{bench.class_flops(spec, 'gemm_qkv') / ns / 1e3:.1f}"
    assert "pmc cmd" in text

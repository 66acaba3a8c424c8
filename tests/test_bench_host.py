"""Host-side logic of bench.py (no GPU): trace-name parsing, the stored-counter
gate, the algorithmic byte and FLOP counts against hand-counted So400m figures,
and the refusal of more than one GPU."""
import os
import subprocess
import sys

import pytest

import bench
from paper_2607_12287_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name,kind", [
    ("void incvit::gemm_kernel<unsigned short, 0, 1, 5>(incvit::GemmArgs)", "qkv"),
    ("void incvit::gemm_kernel<unsigned short, 1, 2, 5>(incvit::GemmArgs)", "fc1"),
    ("void incvit::gemm_kernel<unsigned short, 2, 1, 6>(incvit::GemmArgs)", "fc2"),
    ("void incvit::gemm_kernel<unsigned short, 3, 1, 5>(incvit::GemmArgs)", "oproj"),
    ("void incvit::gemm_kernel<unsigned short, 4, 1, 5>(incvit::GemmArgs)", "oproj"),
    ("void incvit::gemm_kernel<unsigned short, 5, 2, 8>(incvit::GemmArgs)", "fc2"),
    ("void incvit::gemm_kernel<float, 0, 1, 2>(incvit::GemmArgs)", "qkv"),
    ("void incvit::gemm_tiled_kernel<0, 128, 4>(incvit::GemmArgs)", "qkv"),
    ("void incvit::gemm_tiled_kernel<5, 64, 6>(incvit::GemmArgs)", "fc2"),
    ("void incvit::gemm_tiled_kernel<3, 64, 6>(incvit::GemmArgs)", "oproj"),
    ("void incvit::res_kernel<unsigned short, 3, 2>(incvit::ResArgs)", "res_ln1"),
    ("void incvit::embed_kernel<unsigned short, 0, 3, 2>(incvit::EmbedArgs)", "embed"),
    ("void incvit::keyproj_kernel<unsigned short, 0, 3, 2>(incvit::EmbedArgs)", "key_proj"),
    ("void incvit::keyln_kernel<unsigned short>(incvit::KeyLnArgs)", "key_ln"),
    ("incvit::sim_kernel(incvit::SimArgs)", "sim"),
    ("incvit::select_kernel(incvit::SelectArgs)", "select"),
    ("void incvit::attn_kernel<unsigned short, 3, 6, 2, 1, 4>(incvit::AttnArgs)", "attn"),
    ("void incvit::attn_kernel<unsigned short, 3, 6, 5, 2, 1, 4>(incvit::AttnArgs)", "attn"),
    ("__amd_rocclr_copyBuffer", None),
    ("void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<unsigned char>>", None),
])
def test_kernel_kind(name, kind):
    assert bench.kernel_kind(name) == kind


def test_so400m_bytes_and_flops():
    # hand-counted for So400m (D 1152, F 4304, bf16) at 23 refreshed rows
    m = synth.workload("so400m").model
    assert (m.dim, m.mlp_dim, m.dtype) == (1152, 4304, "bf16")
    assert bench.ksplit(m) == 3  # 72 column blocks: 256 // 72 = 3 splits of the 135 K chunks
    M = 23
    weights = {"qkv": 1152 * 3456 * 2, "oproj": 1152 * 1152 * 2, "fc1": 1152 * 4304 * 2, "fc2": 4304 * 1152 * 2}
    rows_in = {"qkv": M * 1152 * 2, "oproj": M * 1152 * 2, "fc1": M * 1152 * 2, "fc2": M * 4304 * 2}
    rows_out = {"qkv": M * 3456 * 2, "oproj": 2 * M * 1152 * 2, "fc1": M * 4304 * 2, "fc2": 3 * M * 1152 * 4}
    for kind in weights:
        assert bench.kernel_bytes(m, M, kind) == weights[kind] + rows_in[kind] + rows_out[kind], kind
        assert bench.gemm_flops(m, M, kind) == 2 * M * weights[kind] // 2, kind
    # the whole step's weights: 27 layers of 30.45 MB
    per_layer = sum(weights.values())
    assert abs(27 * per_layer / 1e6 - 822) < 1
    assert bench.kernel_bytes(m, M, "embed") is None


def test_stored_traffic_gate(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    f = tmp_path / "step_hbm_traffic_so400m.txt"
    assert bench.stored_traffic("so400m", "fc1") is None  # no file
    f.write_text(f"source_hash {bench.source_hash()}\ntraffic_bytes_per_launch fc1 10900000\n")
    assert bench.stored_traffic("so400m", "fc1") == 10900000.0
    assert bench.stored_traffic("so400m", "qkv") is None
    f.write_text("source_hash 0000000000000000\ntraffic_bytes_per_launch fc1 10900000\n")
    assert bench.stored_traffic("so400m", "fc1") is None  # kernels changed since


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_counter_summary(tmp_path):
    # two kinds, the last n dispatches of each kind are averaged (n from the run's launch counts)
    d = tmp_path / "pmc"
    d.mkdir()
    rows = ["Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value"]
    names = ["incvit::sim_kernel(incvit::SimArgs)", "void incvit::gemm_kernel<unsigned short, 1, 2, 5>(incvit::GemmArgs)"]
    vals = {0: [1.0, 10.0], 1: [3.0, 30.0], 2: [5.0, 50.0]}  # dispatch round -> (sim, fc1) values
    i = 0
    for rnd in range(3):
        for k, name in enumerate(names):
            for se in range(2):  # per shader engine: summed per dispatch
                rows.append(f'{i},"{name}",SQ_INSTS_VALU,{vals[rnd][k] / 2}')
            i += 1
    (d / "run_counter_collection.csv").write_text("\n".join(rows) + "\n")
    log = tmp_path / "drive.log"
    log.write_text('{"config": {"workload": "w", "rows_mean": 1.0}, "kernel_launches": {"sim": 2, "fc1": 1}}\n')
    out = tmp_path / "out.txt"
    bench.summarize_counters(str(d), str(log), str(out), "cmd")
    lines = {ln.split()[0]: ln.split()[1:] for ln in out.read_text().splitlines() if not ln.startswith("#")}
    assert float(lines["sim"][0]) == 4.0    # mean of rounds 1, 2
    assert float(lines["fc1"][0]) == 50.0   # the last round only
    assert lines["source_hash"] == [bench.source_hash()]


def test_quantile_and_rows_distribution():
    """The p90 and the refreshed-row distribution the bench line reports."""
    import numpy as np
    assert bench.quantile([1.0], 0.9) == 1.0
    assert bench.quantile([0.0, 10.0], 0.9) == pytest.approx(9.0)
    xs = sorted(float(i) for i in range(11))  # 0..10
    assert bench.quantile(xs, 0.5) == 5.0 and bench.quantile(xs, 0.9) == pytest.approx(9.0)
    k = np.array([[3, 1], [5, 2], [0, 0], [10, 4]])  # steps x streams
    d = bench.rows_dist(k)
    assert d["per_step"] == {"min": 0.0, "median": 5.5, "p90": pytest.approx(11.9), "max": 14.0}
    assert d["per_stream_mean"] == [4.5, 1.75]

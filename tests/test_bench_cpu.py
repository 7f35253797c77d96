"""Host-side accounting of bench.py (no GPU): the refresh roofline counts the flops of the
iteration as described (per precision), the step accounting prices the moments by their
storage, the measured traffic is used only while it fits the sources, and the --gpus guard
refuses more than one GPU."""
import dataclasses
import subprocess
import sys
import os

import pytest

import bench
import workloads as WL

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _one_matrix(rows, cols, rank):
    wl = WL.WORKLOADS["layer_d256"]
    spec = dataclasses.replace(wl.matrices[0], rows=rows, cols=cols, module=WL.Q)
    table = tuple(rank if k == WL.Q else 0 for k in range(len(wl.rank_table)))
    return dataclasses.replace(wl, matrices=(spec,), rank_table=table)


@pytest.mark.parametrize("bf16", [True, False])
def test_refresh_cost_counts_each_part(bf16):
    # s = 32, L = 64, r = 8, p = r -> w = 16, q = 5
    wl = _one_matrix(64, 32, 8)
    s, L, r, w, q = 32, 64, 8, 16, 5
    c = bench.refresh_cost(wl, -1, q, bf16)
    it = 4 * L * s * w                      # Y = X Z and Z2 = X^T Y
    n16 = q - 3 if bf16 else 0
    rows = q * s + L                        # q iterates of s rows and the L-row one
    assert c["bf16_flops"] == n16 * it
    assert c["f64_flops"] == pytest.approx(rows * w * w + (q + 1) * 2 * w ** 3 / 3)
    assert c["f32_flops"] == pytest.approx((q - n16) * it + rows * w * w + 2 * s * w * r)
    t = c["bf16_flops"] / bench.PEAK_BF16 + c["f32_flops"] / bench.PEAK_F32 + c["f64_flops"] / bench.PEAK_F64
    assert c["roofline_ms"] == pytest.approx(t * 1e3)


def test_refresh_cost_width_is_capped_by_the_short_side():
    # r + p > s: the subspace is the whole short side (w = s)
    wl = _one_matrix(40, 24, 16)
    c = bench.refresh_cost(wl, -1, 4, False)
    s, L, w = 24, 40, 24
    assert c["f32_flops"] == pytest.approx(4 * 4 * L * s * w + (4 * s + L) * w * w + 2 * s * w * 16)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stdout


@pytest.mark.parametrize("operand", ["bf16", "f32"])
def test_step_accounting_prices_the_direction_moments_by_their_storage(operand):
    # Optimizer_V reads and writes two L x r moments: 16 L r bytes in fp32, 8 L r in bf16;
    # nothing else in the projection's or the method's bytes depends on the moment dtype
    wl = _one_matrix(64, 160, 32)
    L, r = 160, 32
    c4 = bench.algorithmic_cost(wl, operand, 2, moment_bytes=4)
    c2 = bench.algorithmic_cost(wl, operand, 2, moment_bytes=2)
    assert c4["project"][0] - c2["project"][0] == 8 * L * r
    assert c4["project"][1] == c2["project"][1]
    assert c4["decompose"] == c2["decompose"] and c4["backproject"] == c2["backproject"]
    ob = 2 if operand == "bf16" else 4
    m4, f4 = bench.method_cost(wl, ob, 2, moment_bytes=4)
    m2, f2 = bench.method_cost(wl, ob, 2, moment_bytes=2)
    assert m4 - m2 == 8 * r * L and f4 == f2


def test_measured_traffic_only_for_the_profiled_sources_and_workload(tmp_path, monkeypatch):
    """The roofline's measured HBM traffic comes from the committed counter summary only
    while the kernel sources hash to the value recorded there and the workload is the
    profiled one; otherwise it is reported as null."""
    import hashlib
    h = hashlib.sha256()
    for src in bench.TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    prof = tmp_path / "traffic.txt"
    prof.write_text(f"sources-sha256 {h.hexdigest()}\ntraffic-bytes-per-launch backproject 123.0\n")
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(prof))
    assert bench.measured_traffic("backproject", "llama2_7b") == 123.0
    assert bench.measured_traffic("project", "llama2_7b") is None          # kernel not in the summary
    assert bench.measured_traffic("backproject", "qwen2_7b") is None       # another workload
    prof.write_text("sources-sha256 " + "0" * 64 + "\ntraffic-bytes-per-launch backproject 123.0\n")
    assert bench.measured_traffic("backproject", "llama2_7b") is None      # sources changed since


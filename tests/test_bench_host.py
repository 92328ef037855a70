"""Host-side logic of bench.py (CPU): the FLOP counts behind the roofline
point, the guard on the stored HBM-traffic figure, the counter summary used
for the profiles, and the one-GPU contract."""
import os
import subprocess
import sys

import pytest

import bench
from paper_2606_07878_amd import configs

W2 = configs.get_workload(2)
W4 = configs.get_workload(4)


def test_cross_attention_flops_per_launch():
    """QK^T (t x N x dc) and P X (t x N x 2d) for every (KV head, cross head)
    pair of a layer: 1.374e12 FLOP at the 8k -> 1024 Qwen-shaped layer."""
    c = W2.cfg
    qk = 2.0 * W2.t * W2.n_tokens * c.dc
    px = 2.0 * W2.t * W2.n_tokens * 2 * c.head_dim
    assert bench.ca_flops_per_launch(W2) == pytest.approx(c.n_kv_heads * c.n_cross_heads * (qk + px), rel=0)
    assert bench.ca_flops_per_launch(W2) == pytest.approx(1.374e12, rel=1e-3)
    assert bench.ca_flops_per_launch(W4) == pytest.approx(1.407e13, rel=1e-3)


def test_layer_flops_sum_of_products():
    """The layer's algorithmic FLOPs as the sum of its products (sizes of the
    8k -> 1024 layer): projections, attention, FFN and output heads."""
    G = 1e9
    H, t, N, D, d, nc, dc, ns, ds, F = 8, 1024, 8192, 1024, 128, 8, 1024, 8, 1024, 4096
    Ht = H * t
    products = [
        2 * Ht * D * nc * dc,                 # cross q
        2 * H * N * 2 * d * nc * dc,          # cross k
        2 * H * nc * t * N * (dc + 2 * d),    # QK^T and P X
        2 * Ht * 2 * d * nc * dc,             # (P X) W_V
        2 * Ht * nc * dc * D,                 # W_O
        3 * 2 * Ht * D * ns * ds,             # self q, k, v
        2 * 2 * H * ns * t * t * ds,          # self logits and P v
        2 * Ht * ns * ds * D,                 # self output
        3 * 2 * Ht * D * F,                   # SwiGLU gate, up, down
        2 * Ht * D * 2 * d,                   # output heads
    ]
    assert W2.cfg.ffn_kind == configs.FFN_SWIGLU
    assert bench.layer_flops(W2) / G == pytest.approx(sum(products) / G, rel=1e-12)
    assert bench.layer_flops(W2) == pytest.approx(2.99e12, rel=2e-3)


def test_stored_traffic_matches_kernel_sources():
    """The HBM traffic figure in bench.py belongs to the current cross-attention
    sources (re-measure and update it whenever they change)."""
    assert bench.measured_traffic(2) == bench.MEASURED_TRAFFIC["bytes_per_launch"]
    assert bench.measured_traffic(4) is None


def test_summarize_counters(tmp_path, capsys):
    """Per-kernel means and derived figures from a rocprofv3 counter CSV."""
    rows = ["Dispatch_Id,Kernel_Name,Grid_Size,Counter_Name,Counter_Value,Start_Timestamp,End_Timestamp"]
    for disp in (1, 2):
        for name, val in (("SQ_VALU_MFMA_BUSY_CYCLES", 1024 * 500.0), ("GRBM_GUI_ACTIVE", 8 * 1000.0),
                          ("SQ_INSTS_VALU_MFMA_MOPS_F16", 2e9), ("TCC_EA0_RDREQ_DRAM_32B", 1e8),
                          ("TCC_EA0_WRREQ_DRAM", 1e6), ("FETCH_SIZE", 123456.5)):
            rows.append(f"{disp},void k(int),4096,{name},{val},0,1000000")
    p = tmp_path / "c.csv"
    p.write_text("\n".join(rows) + "\n")
    bench.summarize_counters(str(p))
    out = capsys.readouterr().out.strip()
    assert out.startswith("void k grid=4096 | n=2 avg_us=1000.0")
    assert "mfma_busy=0.500" in out                 # 512000 / (8000 / 8 x 1024)
    assert "f16_TFLOPs=1024.0" in out               # 2e9 x 512 FLOP / 1 ms
    assert "dram_read_MB=3200.0 (3.20 TB/s)" in out  # 1e8 x 32 B
    assert "dram_write_MB=64.0 (0.06 TB/s)" in out   # 1e6 x 64 B
    assert "FETCH_SIZE_KiB=123456.5" in out


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(os.path.dirname(bench.__file__), "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr

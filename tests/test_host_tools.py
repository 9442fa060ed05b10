"""Host-side logic of the benchmark and of the rocprofv3 summarisers (CPU only).

* bench.py refuses any GPU count but one, before touching the GPU;
* the unit count behind every roofline (valid (batch, head, query chunk, slot)
  tuples) against a direct enumeration of the grouped cross attention's terms
  (Eq. 2-3: chunk c attends to the chunks listed in retrieval row c - 1; in decode
  the one query chunk uses row 0);
* the counter arithmetic of profiling.py (traffic scaled by a copy of known size,
  matrix-core busy fraction, SIMD issue breakdown) on small synthetic CSV files.
"""

import csv
import json
import os
import subprocess
import sys
import types

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (imports nothing that needs a GPU at module level)
import profiling  # noqa: E402


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "--gpus must be 1" in r.stderr
    assert r.stdout == ""


def _enumerate_units(idx, mode, H, Hr):
    """Count (b, h, query chunk, slot) terms of Eq. 2 one by one."""
    B, _, nQ, K = idx.shape
    n = 0
    for b in range(B):
        for h in range(H):
            hr = h if Hr == H else 0
            chunks = range(1, nQ) if mode == "causal" else [0]
            for c in chunks:
                row = c - 1 if mode == "causal" else 0
                for s in range(K):
                    if idx[b, hr, row, s] >= 0:
                        n += 1
    return n


@pytest.mark.parametrize("mode,H,Hr", [("causal", 4, 1), ("causal", 3, 3), ("decode", 4, 1), ("decode", 2, 2)])
def test_valid_units_matches_enumeration(mode, H, Hr):
    rng = np.random.default_rng(5)
    B, nQ, K = 2, 7 if mode == "causal" else 1, 4
    idx = rng.integers(0, 9, size=(B, Hr, nQ, K)).astype(np.int32)
    idx[rng.random(idx.shape) < 0.3] = -1  # pad slots
    if mode == "causal":
        idx[:, :, 0, :] = -1                   # row 0 has no earlier chunk
    w = types.SimpleNamespace(mode=mode, H=H, Hr=Hr)
    assert bench.valid_units(idx, w) == _enumerate_units(idx, mode, H, Hr)


def test_flops_per_unit():
    f = bench.flops_per_unit()
    # per (query token, slot, head): each S x d product is 2 S d flops
    assert f["xattn_fwd_kernel"] == 4 * 64 * 64
    assert f["bwd_dq_kernel"] == 6 * 64 * 64
    assert f["bwd_dkdv_kernel"] == 4 * 64 * 64


def _write_counters(path, rows):
    """rows: (kernel name, counter, value) as rocprofv3 writes them, one dispatch each."""
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (k, c, v) in enumerate(rows):
            wr.writerow([i, k, c, v])
    agent = path.replace("counter_collection", "agent_info")
    with open(agent, "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(["Name", "Simd_Count", "Num_Xcc"])
        wr.writerow(["AMD EPYC", 0, 0])
        wr.writerow(["gfx950", 1024, 8])


COPY = "void at::native::elementwise_kernel_copy(...)"
FWD = "void gca::(anonymous namespace)::xattn_fwd_kernel<__bf16, false, false>(gca::FwdParams)"


def test_traffic_scaled_by_copy(tmp_path):
    # the copy of 1 MiB reads it (FETCH_SIZE reports half: 512 KiB) and writes it (1024 KiB)
    fetch = str(tmp_path / "f" / "run_counter_collection.csv")
    write = str(tmp_path / "w" / "run_counter_collection.csv")
    _write_counters(fetch, [(COPY, "FETCH_SIZE", 512.0), (FWD, "FETCH_SIZE", 100.0), (FWD, "FETCH_SIZE", 300.0),
                            (FWD, "FETCH_SIZE", 200.0)])
    _write_counters(write, [(COPY, "WRITE_SIZE", 1024.0), (FWD, "WRITE_SIZE", 10.0)])
    t = profiling.traffic(fetch, write, 1 << 20, "cmd")
    assert t["fetch_scale"] == pytest.approx(2.0)
    assert t["write_scale"] == pytest.approx(1.0)
    k = t["kernels"]["xattn_fwd_kernel"]
    assert k["fetch_bytes_per_launch"] == pytest.approx(200.0 * 1024 * 2.0)  # median of 100, 300, 200
    assert k["write_bytes_per_launch"] == pytest.approx(10.0 * 1024)
    assert "copy" not in t["kernels"]


def test_counters_busy_fraction(tmp_path):
    m = str(tmp_path / "m" / "run_counter_collection.csv")
    l2 = str(tmp_path / "l" / "run_counter_collection.csv")
    # GRBM_GUI_ACTIVE summed over 8 XCCs: 8e6 -> 1e6 cycles; 1024 SIMDs busy 0.25 of them
    _write_counters(m, [(FWD, "GRBM_GUI_ACTIVE", 8e6), (FWD, "SQ_VALU_MFMA_BUSY_CYCLES", 0.25 * 1e6 * 1024),
                        (FWD, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1000.0)])
    _write_counters(l2, [(FWD, "TCC_HIT_sum", 30.0), (FWD, "TCC_MISS_sum", 70.0)])
    c = profiling.counters(m, l2, "cmd")
    k = c["kernels"]["xattn_fwd_kernel"]
    assert k["mfma_busy_frac"] == pytest.approx(0.25)
    assert k["mfma_bf16_flops_per_launch"] == pytest.approx(512_000.0)
    assert k["l2_hit_frac"] == pytest.approx(0.3)
    assert c["simds"] == 1024 and c["xccs"] == 8


def test_issue_breakdown(tmp_path):
    gui = 8e6          # 1e6 cycles per XCC
    simd_cycles = 1e6 * 1024
    p1 = str(tmp_path / "p1" / "run_counter_collection.csv")
    p2 = str(tmp_path / "p2" / "run_counter_collection.csv")
    _write_counters(p1, [(FWD, "GRBM_GUI_ACTIVE", gui),
                         (FWD, "SQ_ACTIVE_INST_VALU", 0.5 * simd_cycles / 4),   # quad-cycles
                         (FWD, "SQ_VALU_MFMA_BUSY_CYCLES", 0.3 * simd_cycles),
                         (FWD, "SQ_VALU_MFMA_COEXEC_CYCLES", 0.1 * simd_cycles),
                         (FWD, "SQ_WAVE_CYCLES", 1000.0), (FWD, "SQ_WAIT_ANY", 250.0),
                         (FWD, "SQ_WAIT_INST_ANY", 300.0), (FWD, "SQ_ACTIVE_INST_ANY", 450.0)])
    # the second run's counters are normalised by its own clock
    _write_counters(p2, [(FWD, "GRBM_GUI_ACTIVE", 2 * gui), (FWD, "SQ_WAVES", 100.0),
                         (FWD, "SQ_INSTS_VALU", 5000.0), (FWD, "SQ_INSTS_MFMA", 400.0)])
    d = profiling.issue([p1, p2], "cmd")
    k = d["kernels"]["xattn_fwd_kernel"]
    assert k["simd_valu_issue_frac"] == pytest.approx(0.5)
    assert k["simd_mfma_busy_frac"] == pytest.approx(0.3)
    assert k["simd_valu_and_mfma_frac"] == pytest.approx(0.1)
    assert k["simd_neither_frac"] == pytest.approx(0.3)
    assert k["wave_waitcnt_or_barrier_frac"] == pytest.approx(0.25)
    assert k["wave_ready_not_issued_frac"] == pytest.approx(0.3)
    assert k["wave_issuing_frac"] == pytest.approx(0.45)
    assert k["instructions_per_wave"] == {"valu": 50.0, "mfma": 4.0}
    json.dumps(d)  # serialisable as committed

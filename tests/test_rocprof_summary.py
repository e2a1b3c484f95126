"""The profile summaries behind bench.py's roofline.traffic and profiles/:
counter scaling by the calibration copy, per-step sums over the grouped
SwiGLU kernels, the operand-byte formulas, and the kernel-time table, on small
synthetic rocprofv3 CSV files (no GPU)."""
import csv

import pytest

from paper_2508_19078_amd import rocprof_summary as R


def write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


K = "void fm::(anonymous namespace)::{}(int, float*)"


def counter_rows(counter, per_kernel):
    """per_kernel: {kernel: [[values of dispatch 1], [values of dispatch 2], ...]}:
    several values of one dispatch (counter instances) are summed."""
    rows, did = [], 0
    for kern, dispatches in per_kernel.items():
        for vals in dispatches:
            did += 1
            for v in vals:
                rows.append({"Dispatch_Id": did, "Kernel_Name": K.format(kern), "Counter_Name": counter,
                             "Counter_Value": v})
    return rows


def test_traffic_scales_by_the_copy_and_sums_per_step(tmp_path):
    calib = 256 << 20
    fetch = counter_rows("FETCH_SIZE", {
        "__amd_rocclr_copyBuffer": [[calib / 1024 / 2]],        # the copy reads half its bytes
        "kb_gate_up": [[100, 28], [128]],                        # two steps, instances summed
        "kb_down<true>": [[64], [64]],
        "kb_dw_gu<false>": [[10], [30]],
        "k_combine<fm::bf16, 8>": [[7], [9]],
    })
    write = counter_rows("WRITE_SIZE", {
        "__amd_rocclr_copyBuffer": [[calib / 1024]],             # ... and writes them exactly
        "kb_gate_up": [[50], [50]],
        "kb_down<true>": [[20], [20]],
    })
    write_counters(tmp_path / "f.csv", fetch)
    write_counters(tmp_path / "w.csv", write)
    t = R.traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), calib)
    f, w = t["FETCH_SIZE"], t["WRITE_SIZE"]
    assert f["factor"] == pytest.approx(2.0) and w["factor"] == pytest.approx(1.0)
    assert f["steps"] == 2 and w["steps"] == 2
    assert f["per_kernel_kib"]["kb_gate_up"] == pytest.approx(128.0)
    assert f["per_kernel_kib"]["kb_down"] == pytest.approx(64.0)          # template arguments dropped
    assert f["per_kernel_kib"]["kb_dw_gu"] == pytest.approx(20.0)
    assert f["kib_per_step"] == pytest.approx(128 + 64 + 20)
    assert f["bytes_per_step"] == pytest.approx((128 + 64 + 20) * 1024 * 2.0)
    assert w["bytes_per_step"] == pytest.approx((50 + 20) * 1024 * 1.0)
    # other library kernels: scaled bytes per dispatch
    assert f["other_bytes"]["k_combine"] == pytest.approx(8 * 1024 * 2.0)


def test_traffic_needs_the_calibration_copy(tmp_path):
    write_counters(tmp_path / "f.csv", counter_rows("FETCH_SIZE", {"kb_gate_up": [[1]]}))
    write_counters(tmp_path / "w.csv", counter_rows("WRITE_SIZE", {"kb_gate_up": [[1]]}))
    with pytest.raises(SystemExit):
        R.traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 1 << 20)


def test_operand_bytes_by_hand():
    # 10 rows over 3 slots, 6 of them in 2 tuning slots; d = 4, I = 2, bf16
    ob = R.operand_bytes({"total": 10, "tuning": 6, "slots": 3, "tuning_slots": 2, "d": 4, "I": 2, "bytes": 2})
    w = 4 * 2 * 2                                     # one 4 x 2 bf16 matrix
    assert ob["kb_gate_up"] == (10 * 4 * 2 + 2 * 3 * w, 3 * 10 * 2 * 2)     # X rows + W_g, W_u; A_g, A_u, H
    assert ob["kb_down"] == (10 * 2 * 2 + 3 * w, 10 * 4 * 2)                # H + W_d; O
    assert ob["kb_dh"] == (10 * 4 * 2 + 3 * w + 2 * 10 * 2 * 2, 2 * 10 * 2 * 2)   # dO, W_d, A_g, A_u; dA_g, dA_u
    assert ob["kb_dx"] == (2 * 10 * 2 * 2 + 2 * 3 * w, 10 * 4 * 2)          # dA_g, dA_u, W_g, W_u; dX rows
    assert ob["kb_dw_gu"] == (2 * 6 * 2 * 2 + 6 * 4 * 2, 2 * 2 * 4 * 2 * 4)  # tuning rows; fp32 dW_g, dW_u
    assert ob["kb_dw_d"] == (6 * (4 + 2) * 2, 2 * 4 * 2 * 4)                # dO and H rows; fp32 dW_d


def test_stats_table_leaves_out_torch_kernels_and_sums_a_step(tmp_path):
    path = tmp_path / "s.csv"
    names = [("at::native::elementwise_kernel<...>", 5, 9e6), (K.format("kb_gate_up"), 4, 4e6),
             (K.format("kb_dw_gu<false>"), 4, 2e6), (K.format("k_combine<fm::bf16, 8>"), 4, 1e6)]
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"])
        w.writeheader()
        for n, c, tot in names:
            w.writerow({"Name": n, "Calls": c, "TotalDurationNs": tot, "AverageNs": tot / c, "Percentage": 10.0})
    out = R.stats_table(str(path), 10)
    assert "elementwise" not in out
    assert "| kb_gate_up | 4 | 1000.0 | 4.000 |" in out
    assert "k_combine<fm::bf16, 8>" in out
    # (4 + 2) ms over 4 steps of the FFN kernels
    assert "over 4 steps): 1500.0 µs" in out

"""Host logic of bench.py on the CPU: the one-GPU guard, the step's FLOP
count derived from the layer shapes, the HBM traffic report built from two
counter runs (calibration scaling, medians, the main and merge dispatches),
and the source-hash gate on the recorded traffic."""
import csv
import io
import os
from contextlib import redirect_stdout

import pytest

import bench
from seeded_inputs import configs


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


@pytest.mark.parametrize("name", ["dit_xl2_1024", "dit_xl2_2048", "tiny"])
def test_step_flops_from_layer_shapes(name):
    """Every product of a band step, counted from its operand shapes (2 M N K
    for a product, 4 M N_kv H for attention's two), per guidance branch
    (patch embedding, per block QKV, attention, out-projection, MLP and the
    adaLN vectors, the final adaLN vectors and linear); the timestep
    embedding once."""
    cfg = configs.get(name)
    H, L, B, N = cfg.hidden, cfg.n_blocks, cfg.cfg_batch, cfg.n_kv
    n_q = 3 * cfg.R
    mm = lambda m, n, k: 2 * m * n * k
    per_block = (mm(n_q, 3 * H, H) + 4 * n_q * N * H + mm(n_q, H, H) + mm(n_q, 4 * H, H)
                 + mm(n_q, H, 4 * H) + mm(1, 6 * H, H))
    in_dim, out_dim = cfg.in_ch * cfg.patch ** 2, cfg.out_ch * cfg.patch ** 2
    embed = mm(n_q, H, in_dim)
    final = mm(1, 2 * H, H) + mm(n_q, out_dim, H)
    temb = mm(1, H, cfg.freq_dim) + mm(1, H, H)
    assert bench.step_flops(cfg, n_q) == float(B * (embed + L * per_block + final) + temb)


def _counters(path, counter, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "pmc_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, grid, kib) in enumerate(rows):
            # each dispatch's value split over two instances (rocprofv3 lists one row per
            # instance of a counter); the report adds them
            for part in (0.25, 0.75):
                w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Grid_Size": grid,
                            "Counter_Name": counter, "Counter_Value": kib * part})


def test_pmc_report_scales_by_the_calibration(tmp_path):
    elems = bench.CALIB_ELEMS
    read_kib, write_kib = 8 * elems / 1024, 4 * elems / 1024
    # the counter reads half the fetched bytes and all the written ones; the
    # small-grid update dispatches (the step's own) are not the calibration
    fetch_rows = [("update_vec4_kernel", 1 << 24, read_kib / 2)] * 3 + [("update_vec4_kernel", 256, 7.0)] * 5
    write_rows = [("update_vec4_kernel", 1 << 24, write_kib)] * 3 + [("update_vec4_kernel", 256, 3.0)] * 5
    fetch_rows += [("orch::attn_bf16_mfma_kernel<72>", 512, v) for v in (1000.0, 1010.0, 990.0)]
    fetch_rows += [("orch::attn_merge_kernel<72>", 1248, v) for v in (200.0, 201.0, 199.0)]
    write_rows += [("orch::attn_bf16_mfma_kernel<72>", 512, v) for v in (500.0, 505.0, 495.0)]
    write_rows += [("orch::attn_merge_kernel<72>", 1248, v) for v in (100.0, 99.0, 101.0)]
    _counters(str(tmp_path / "f"), "FETCH_SIZE", fetch_rows)
    _counters(str(tmp_path / "w"), "WRITE_SIZE", write_rows)
    buf = io.StringIO()
    with redirect_stdout(buf):
        assert bench.pmc_report(str(tmp_path / "f"), str(tmp_path / "w")) == 0
    kv = dict(l[2:].split(": ", 1) for l in buf.getvalue().splitlines() if l.startswith("- "))
    assert int(kv["fetch_bytes_per_launch"]) == 2 * (1000 + 200) * 1024
    assert int(kv["write_bytes_per_launch"]) == (500 + 100) * 1024
    assert int(kv["hbm_bytes_per_launch"]) == (2 * 1200 + 600) * 1024
    assert kv["source_sha256"] == bench.kernel_source_hash("attention")


def test_recorded_traffic_needs_the_current_sources(tmp_path, monkeypatch):
    report = tmp_path / "traffic.md"
    monkeypatch.setattr(bench, "TRAFFIC_REPORT", str(report))
    assert bench.recorded_traffic("attention") is None                  # no report
    good = bench.kernel_source_hash("attention")
    report.write_text(f"- kernel: attention\n- source_sha256: {good}\n- hbm_bytes_per_launch: 1234\n")
    assert bench.recorded_traffic("attention") == 1234.0
    report.write_text(f"- kernel: attention\n- source_sha256: {'0' * 64}\n- hbm_bytes_per_launch: 1234\n")
    assert bench.recorded_traffic("attention") is None                  # sources changed

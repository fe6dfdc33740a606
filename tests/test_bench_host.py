"""Host logic of the measurement (CPU): the algorithmic byte counts the
roofline divides by, and the HBM-traffic record built from rocprofv3
counters (scaling by a copy of known size, the unique kernel pick, and the
record being refused once the decode sources change)."""

import csv
import json

import pytest
import torch

import bench
import gva_inputs
from paper_2609_13285_amd import traffic


def test_decode_bytes_at_the_bench_shape():
    # B32 T8192 H32 G8 d 128/128/16 bf16: 262,144 rows of (8 * 128 + 16)
    # elements, M [32][128][128] and q [32][32][144], two bytes each
    w = gva_inputs.WORKLOADS["b32_t8k"]
    lens = torch.full((w.batch,), w.t_max, dtype=torch.int32)
    rows = 32 * 8192
    expect = rows * (8 * 128 + 16) * 2 + 32 * 128 * 128 * 2 + 32 * 32 * 144 * 2
    assert expect == 546_603_008
    assert traffic.decode_bytes(lens, 32, 32, 8, 128, 128, 16, 2) == expect
    # the step adds the appended rows (read and written once) and the fp32 output
    step = traffic.step_bytes(lens, 32, 32, 8, 128, 128, 16, 2, appended_rows=32)
    assert step == expect + 2 * 32 * (8 * 128 + 16) * 2 + 32 * 32 * 128 * 4
    # matched GQA streams a key and a value row per group, no positional key
    assert traffic.gqa_decode_bytes(lens, 32, 32, 8, 128, 2) == rows * 2 * 8 * 128 * 2 + 32 * 32 * 128 * 2


def test_lengths_are_clamped_at_zero_in_the_byte_count():
    lens = torch.tensor([5, 0, -3, 2], dtype=torch.int32)
    assert traffic.stream_bytes(lens, 2, 4, 2, 2) == 7 * (2 * 4 + 2) * 2
    assert traffic.stream_bytes([5, 0, -3, 2], 2, 4, 2, 2) == 7 * (2 * 4 + 2) * 2


def _counter_csv(path, rows):
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        wr.writeheader()
        for name, counter, value in rows:
            wr.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value})


DEC = "void (anonymous namespace)::decode_bf16_kernel<4, 128, 1, false, true, false>(DecodeParams)"
COPY = "__amd_rocclr_copyBuffer"


def test_traffic_record_scales_by_the_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    f, w_, cf, cw = (str(tmp_path / n) for n in ("f.csv", "w.csv", "cf.csv", "cw.csv"))
    # two launches of the decode kernel, FETCH 1000 and 1200 units; a 1 MiB
    # copy reading 512 FETCH units and writing 1024 WRITE units
    _counter_csv(f, [(DEC, "FETCH_SIZE", 1000), (DEC, "FETCH_SIZE", 1200), ("other", "FETCH_SIZE", 9)])
    _counter_csv(w_, [(DEC, "WRITE_SIZE", 10), (DEC, "WRITE_SIZE", 14)])
    _counter_csv(cf, [(COPY, "FETCH_SIZE", 512)])
    _counter_csv(cw, [(COPY, "WRITE_SIZE", 1024)])
    bench.write_traffic(f, w_, cf, cw, "b32_t8k", 1, copy_mb=1)
    rec = json.load(open(bench.TRAFFIC_FILE))
    assert rec["fetch_scale_bytes_per_unit"] == 2048.0
    assert rec["write_scale_bytes_per_unit"] == 1024.0
    assert rec["fetch_bytes_per_launch"] == 1100 * 2048.0
    assert rec["write_bytes_per_launch"] == 12 * 1024.0
    assert rec["hbm_bytes_per_launch"] == 1100 * 2048 + 12 * 1024
    assert rec["kernel_sha"] == bench.kernel_sha()
    # the bench reports it only for the same sources, workload and splits
    assert bench.measured_traffic("b32_t8k", 1) == rec["hbm_bytes_per_launch"]
    assert bench.measured_traffic("b32_t8k", 2) is None
    assert bench.measured_traffic("ragged_b64", 1) is None
    rec["kernel_sha"] = "0" * 16
    json.dump(rec, open(bench.TRAFFIC_FILE, "w"))
    assert bench.measured_traffic("b32_t8k", 1) is None


def test_traffic_record_needs_one_decode_kernel(tmp_path, monkeypatch):
    # two template instances that both match "decode_bf16_kernel" (e.g. a
    # comparison run in the same process) make the record ambiguous
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    f, w_, cf, cw = (str(tmp_path / n) for n in ("f.csv", "w.csv", "cf.csv", "cw.csv"))
    other = DEC.replace("<4, 128, 1,", "<4, 128, 0,")
    _counter_csv(f, [(DEC, "FETCH_SIZE", 1000), (other, "FETCH_SIZE", 900)])
    _counter_csv(w_, [(DEC, "WRITE_SIZE", 10)])
    _counter_csv(cf, [(COPY, "FETCH_SIZE", 512)])
    _counter_csv(cw, [(COPY, "WRITE_SIZE", 1024)])
    with pytest.raises(SystemExit):
        bench.write_traffic(f, w_, cf, cw, "b32_t8k", 1, copy_mb=1)


def test_gqa_keys_recipe():
    # the matched-GQA key cache drawn for workloads without one: N(0, 1) in
    # the storage dtype, deterministic, and independent of make_inputs' draws
    w = gva_inputs.Workload("k", 2, 64, 4, 2, 64, 64, 16)
    a, b = gva_inputs.gqa_keys(w, 3), gva_inputs.gqa_keys(w, 3)
    assert a.shape == (2, 2, 64, 64) and a.dtype == torch.bfloat16
    assert torch.equal(a, b)
    assert not torch.equal(a, gva_inputs.gqa_keys(w, 4))
    x = a.float()
    assert abs(float(x.mean())) < 0.1 and abs(float(x.std()) - 1.0) < 0.1


def test_metric_label_names_the_workload():
    # the bench workload's label is the headline metric verbatim
    w = gva_inputs.WORKLOADS["b32_t8k"]
    assert bench.metric_label(w) == "decode attention GB/s (fraction of HBM peak) and tokens/s, B=32 T=8K bf16"
    assert bench.metric_label(gva_inputs.WORKLOADS["ragged_b64"]).endswith("B=64 T=128..32K bf16")
    assert bench.metric_label(gva_inputs.WORKLOADS["long_b4_t128k"]).endswith("B=4 T=64K..128K bf16")
    assert bench.metric_label(gva_inputs.WORKLOADS["tiny_f32"]).endswith("B=1 T=256 f32")


def test_launch_bytes_of_the_single_launch_step():
    # one split, the current rows appended in the launch: the launch moves
    # exactly the step's algorithmic bytes (append and fp32 output included)
    w = gva_inputs.WORKLOADS["b32_t8k"]
    lens = torch.full((w.batch,), w.t_max, dtype=torch.int32)
    args = (lens, 32, 32, 8, 128, 128, 16, 2)
    step = traffic.step_bytes(*args, appended_rows=32)
    assert traffic.launch_bytes(*args, appended_rows=32, writes_output=True) == step == 547_260_416
    # several splits: the combine writes the output, not the attention launch
    assert traffic.launch_bytes(*args, appended_rows=32) == step - 32 * 32 * 128 * 4
    assert traffic.launch_bytes(*args) == traffic.decode_bytes(*args)

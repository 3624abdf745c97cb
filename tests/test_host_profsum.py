"""Host-side profile summaries: counter calibration, traffic table and the
lookup bench.py uses (synthetic counter files; no profiler needed)."""
import csv
import json
import os

import pytest

from paper_2008_03602_amd import profsum

KNAME = "void ct::igemm_f32_kernel<16, 1, 1, 1, 3>(float const*, float const*, float*, ct::IgF32Args)"


def _pmc(dirpath, counter, rows):
    os.makedirs(dirpath, exist_ok=True)
    with open(os.path.join(dirpath, "x_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (name, v) in enumerate(rows):
            w.writerow([i + 1, name, counter, v])


def _replay(knobs, nbytes=1 << 30):
    return {"layer": "r18.2", "kernel": "igemm_f32_kernel<16, 1, 1, 1, 3>",
            "schedule": {"threads": 512, "blocks": 224, "lds_bytes": 25856, "knobs": knobs},
            "latency_us": 9.0, "copy_bytes_each_way": nbytes}


def test_traffic_is_scaled_by_the_copy_kernel(tmp_path):
    # the copy kernel of 1 GiB reads as 524288 KiB FETCH (scale 2) and 1048576 KiB WRITE (scale 1)
    f, w = str(tmp_path / "f"), str(tmp_path / "w")
    _pmc(f, "FETCH_SIZE", [(KNAME, 3000.0), (KNAME, 3100.0), (KNAME, 3050.0), ("ct::copy_kernel(...)", 524288.0)])
    _pmc(w, "WRITE_SIZE", [(KNAME, 784.0)] * 3 + [("ct::copy_kernel(...)", 1048576.0)])
    t = profsum.traffic_block(_replay({"mfma": 16}), f, w)
    assert t["scale_f"] == pytest.approx(2.0) and t["scale_w"] == pytest.approx(1.0)
    assert t["block"]["fetch_bytes"] == pytest.approx(3050.0 * 1024 * 2)   # median of the three
    assert t["block"]["write_bytes"] == pytest.approx(784.0 * 1024)
    assert t["block"]["traffic_bytes"] == pytest.approx(3050.0 * 2048 + 784.0 * 1024)


def test_incomplete_counter_runs_give_no_traffic(tmp_path):
    f, w = str(tmp_path / "f"), str(tmp_path / "w")
    _pmc(f, "FETCH_SIZE", [(KNAME, 3000.0)])  # no copy kernel in the run
    _pmc(w, "WRITE_SIZE", [(KNAME, 784.0), ("ct::copy_kernel(...)", 1048576.0)])
    assert profsum.traffic_block(_replay({"mfma": 16}), f, w) is None


def test_table_lookup_matches_kernel_shape_knobs_and_source_hash(tmp_path):
    entries = []
    for i, knobs in enumerate(({"mfma": 16, "cpc": 16}, {"mfma": 16, "cpc": 32})):
        f, w = str(tmp_path / ("f%d" % i)), str(tmp_path / ("w%d" % i))
        _pmc(f, "FETCH_SIZE", [(KNAME, 1000.0 * (i + 1)), ("ct::copy_kernel(...)", 524288.0)])
        _pmc(w, "WRITE_SIZE", [(KNAME, 784.0), ("ct::copy_kernel(...)", 1048576.0)])
        entries.append((_replay(knobs), f, w))
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "table.md").write_text(profsum.traffic_table(entries, ["cmd"]))
    shape = {"threads": 512, "blocks": 224, "knobs": {"mfma": 16, "cpc": 32}}
    blk = profsum.find_traffic(str(prof), "igemm_f32_kernel<16, 1, 1, 1, 3>", shape)
    assert blk is not None and blk["fetch_bytes"] == pytest.approx(2000.0 * 2048)
    # another shape, other knobs or another kernel: no figure
    assert profsum.find_traffic(str(prof), "igemm_f32_kernel<16, 1, 1, 1, 3>",
                                dict(shape, blocks=448)) is None
    assert profsum.find_traffic(str(prof), "igemm_f32_kernel<16, 1, 1, 1, 3>",
                                dict(shape, knobs={"mfma": 16, "cpc": 8})) is None
    assert profsum.find_traffic(str(prof), "igemm_f32_kernel<16, 1, 2, 1, 3>", shape) is None
    # a block whose source hash differs from the current sources is stale
    text = (prof / "table.md").read_text()
    h = profsum.kernel_source_hash("igemm_f32_kernel<16, 1, 1, 1, 3>")
    (prof / "table.md").write_text(text.replace(h, "0" * 16))
    assert profsum.find_traffic(str(prof), "igemm_f32_kernel<16, 1, 1, 1, 3>", shape) is None


def test_sq_summary_converts_quad_cycles_to_clocks(tmp_path):
    # 100 waves per dispatch: SQ_WAVE_CYCLES 2500 quad-cycles per wave = 10000
    # clocks; 2304 MFMA-busy clocks (72 MFMAs of 32) = 23.0 % of them; 144
    # bank-conflict clocks = 1.4 %; 2200 quad-cycles waiting on LDS = 88 clocks
    per = {"SQ_WAVES": 100, "SQ_WAVE_CYCLES": 250000, "SQ_INSTS_LDS": 6700, "SQ_LDS_BANK_CONFLICT": 14400,
           "SQ_WAIT_INST_LDS": 2200, "SQ_VALU_MFMA_BUSY_CYCLES": 230400, "SQ_INSTS_VALU_MFMA_F32": 7200}
    d = tmp_path / "sq"
    d.mkdir()
    with open(d / "sq_counter_collection.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for disp in range(3):
            for c, v in per.items():
                w.writerow([disp + 1, KNAME, c, v])
    rep = dict(_replay({"mfma": 16}), fraction=1.0, flops=7200 * 2048)
    text = profsum.sq_summary(rep, str(d))
    assert "| SQ_WAVE_CYCLES | quad-cycles | 250000 | 2500.0 | 34.72 | 10000 |" in text
    assert "| SQ_WAIT_INST_LDS | quad-cycles | 2200 | 22.0 | 0.31 | 88 |" in text
    assert "| SQ_VALU_MFMA_BUSY_CYCLES | cycles | 230400 | 2304.0 | 32.00 | 2304 |" in text
    assert "A wave lives 10000 clocks (4.17 us at 2.4 GHz)" in text
    assert "busy for 2304 of them (23.0 %)" in text and "stall LDS for 144 (1.4 %)" in text
    assert "the kernel issues 7200 (+0.0 %: tile padding)" in text


def test_sq_summary_merges_passes_and_splits_a_wave_s_life(tmp_path):
    # pass 1 as above; pass 2 adds the wave-time partition: of 2500
    # quad-cycles per wave, 600 issuing, 1400 waiting on a dependency and 500
    # waiting to issue (24 %, 56 %, 20 %)
    def write(d, per):
        d.mkdir()
        with open(d / "sq_counter_collection.csv", "w", newline="") as fh:
            w = csv.writer(fh)
            w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
            for disp in range(3):
                for c, v in per.items():
                    w.writerow([disp + 1, KNAME, c, v])
    write(tmp_path / "p1", {"SQ_WAVES": 100, "SQ_WAVE_CYCLES": 250000, "SQ_VALU_MFMA_BUSY_CYCLES": 230400,
                            "SQ_INSTS_VALU_MFMA_F32": 7200})
    write(tmp_path / "p2", {"SQ_WAVES": 100, "SQ_ACTIVE_INST_ANY": 60000, "SQ_WAIT_ANY": 140000,
                            "SQ_WAIT_INST_ANY": 50000})
    rep = dict(_replay({"mfma": 16}), fraction=0.25, flops=7200 * 2048)
    text = profsum.sq_summary(rep, [str(tmp_path / "p1"), str(tmp_path / "p2")])
    assert "7 SQ counters in 2 passes" in text
    assert "| SQ_WAIT_ANY | quad-cycles | 140000 | 1400.0 | 19.44 | 5600 |" in text
    assert "24 % goes to issuing instructions" in text and "56 % to waiting for a dependency" in text
    assert "20 % to waiting for its turn to issue" in text

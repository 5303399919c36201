"""The profile summary tool on synthetic rocprofv3 counter tables (CPU)."""
import csv

from paper_2607_12121_amd import rocprof_summary as rs

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(FIELDS, r)))


def test_mfma_summary_figures(tmp_path):
    k = "void (anonymous namespace)::attn_fwd_kernel<128>(int)"
    rows = []
    for d in ("1", "2"):   # two launches of 1 us; counters split over two dimension rows
        rows += [(d, k, "SQ_INSTS_MFMA", 600, 0, 1000), (d, k, "SQ_INSTS_MFMA", 400, 0, 1000),
                 (d, k, "SQ_VALU_MFMA_BUSY_CYCLES", 32000, 0, 1000), (d, k, "GRBM_GUI_ACTIVE", 16000, 0, 1000)]
    rows.append(("3", "void other_kernel(int)", "SQ_INSTS_MFMA", 0, 0, 500))
    p = tmp_path / "c.csv"
    _write(p, rows)
    ap = rs.argparse.ArgumentParser()
    a = ap.parse_args([])
    a.csv, a.title, a.cmd = str(p), "t", ["c"]
    a.alg = ["attention@attn_fwd=3.2e7", "other@attn_fwd=1e9"]
    a.flops_per_mfma, a.simds, a.xcds, a.peak_tflops, a.max_clock_ghz = 32768, 1024, 8, 2500.0, 2.4
    out = rs.mfma(a)
    row = [l for l in out.splitlines() if l.startswith("| attn_fwd_kernel<128>")]
    assert len(row) == 1 and "other_kernel" not in out
    cells = [c.strip() for c in row[0].strip("|").split("|")]
    # kernel, step, launches, avg us, instructions, flops, alg/MFMA, clock, busy %, % of peak
    assert cells[1] == "attention" and cells[2] == "2" and cells[3] == "1.0" and cells[4] == "1,000"
    assert cells[5] == "3.277e+07" and cells[6] == "0.977"
    assert cells[7] == "2.00"     # 16000 / 8 cycles in 1 us
    assert cells[8] == "1.6"      # 32000 / (1024 * 2000)
    assert cells[9] == "1.3"      # 3.2e7 flops in 1 us against 2.5e15
    a.max_clock_ghz = 1.5           # an implausible clock is not shown
    cells = [c.strip() for c in [l for l in rs.mfma(a).splitlines() if l.startswith("| attn_fwd")][0].strip("|").split("|")]
    assert cells[7] == cells[8] == "—" and cells[9] == "1.3"


def test_traffic_digest_ignores_comments(tmp_path):
    a = tmp_path / "k.hip"
    a.write_text("int f() { return 1; }  // one\n")
    d1 = rs.source_digest([str(a)])
    a.write_text("/* two */ int f()   { return 1; }\n")
    assert rs.source_digest([str(a)]) == d1
    a.write_text("int f() { return 2; }\n")
    assert rs.source_digest([str(a)]) != d1


def test_traffic_per_launch_shape(tmp_path):
    """FETCH/WRITE per dispatch scaled by the copy's readings, only launches of
    the given grid size, and the counted / algorithmic ratio."""
    hdr = FIELDS + ["Grid_Size"]

    def write(path, counter, rows):
        with open(path, "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=hdr)
            w.writeheader()
            for d, k, v, g in rows:
                w.writerow(dict(zip(hdr, (d, k, counter, v, 0, 2000, g))))
    # copy of 1 MiB: FETCH reads 512 KiB (scale 2), WRITE 1024 KiB (scale 1)
    fetch, wr = tmp_path / "f.csv", tmp_path / "w.csv"
    write(fetch, "FETCH_SIZE", [("1", "neg_kernel", 512, 1), ("2", "gather_kernel<4>", 100, 64),
                                ("3", "gather_kernel<4>", 100, 64), ("4", "gather_kernel<4>", 7, 8)])
    write(wr, "WRITE_SIZE", [("1", "neg_kernel", 1024, 1), ("2", "gather_kernel<4>", 50, 64),
                             ("3", "gather_kernel<4>", 50, 64), ("4", "gather_kernel<4>", 9, 8)])
    src = tmp_path / "k.hip"
    src.write_text("int f();\n")
    ap = rs.argparse.ArgumentParser()
    a = ap.parse_args([])
    a.fetch, a.write, a.kernel, a.copy_kernel, a.copy_bytes = str(fetch), str(wr), ["gather_kernel"], "neg_kernel", 1 << 20
    a.grid, a.alg_bytes, a.source, a.title, a.cmd = 64, 250 * 1024, [str(src)], "t", ["c"]
    out = rs.traffic(a)
    assert "bytes_per_launch: 256000" in out            # (100 * 2 + 50) KiB
    assert "counted / algorithmic = 1.000" in out
    assert "with 64 work-items (fetch pass / write pass) | 2 / 2" in out

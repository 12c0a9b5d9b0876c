"""The rocprofv3 summarizers behind profiles/ (host code, synthetic counter files)."""
import csv

from paper_2412_18934_amd import profiling

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def _row(did, name, counter, value, t0=0, t1=1000):
    return {"Dispatch_Id": did, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value,
            "Start_Timestamp": t0, "End_Timestamp": t1}


def test_hbm_scale_comes_from_the_packing_copy(tmp_path):
    # two packing dispatches that copy 3 MiB in total each way; FETCH reads
    # half of it and WRITE all of it, so the scales are 2 and 1
    ref = 3 << 20
    fetch = [_row(1, "k_pack_blocks(GemmArgs)", "FETCH_SIZE", 512),
             _row(2, "k_pack_blocks(GemmArgs)", "FETCH_SIZE", 1024),
             _row(3, "void k_proj<1, 0>(GemmArgs)", "FETCH_SIZE", 100),
             _row(4, "void k_proj<1, 0>(GemmArgs)", "FETCH_SIZE", 300)]
    write = [_row(1, "k_pack_blocks(GemmArgs)", "WRITE_SIZE", 1024),
             _row(2, "k_pack_blocks(GemmArgs)", "WRITE_SIZE", 2048),
             _row(3, "void k_proj<1, 0>(GemmArgs)", "WRITE_SIZE", 10),
             _row(4, "void k_proj<1, 0>(GemmArgs)", "WRITE_SIZE", 30)]
    f, w, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "hbm.txt"
    _write(f, fetch)
    _write(w, write)
    profiling.summarize_hbm(str(f), str(w), str(out), "cmd", ref)
    sh, per = profiling.read_hbm_summary(str(out))
    assert sh == profiling.source_hash()
    n, fb, wb = per["k_proj<1, 0>"]
    assert n == 2
    assert abs(fb - 2 * 200 * 1024) < 1e-6      # mean 200 KiB fetched, scale 2
    assert abs(wb - 1 * 20 * 1024) < 1e-6       # mean 20 KiB written, scale 1
    assert profiling.gemm_traffic_per_launch(str(out)) == fb + wb


def test_mfma_busy_and_rate(tmp_path):
    # one dispatch of 10 us: a quarter of all SIMD cycles busy and 1e6 MOPs
    dur_ns = 10_000
    busy = 0.25 * dur_ns * 1e-9 * profiling.CLOCK_HZ * profiling.N_SIMD
    rows = [_row(1, "void k_proj<1, 2>(GemmArgs)", "SQ_VALU_MFMA_BUSY_CYCLES", busy, 0, dur_ns),
            _row(1, "void k_proj<1, 2>(GemmArgs)", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e6, 0, dur_ns),
            _row(2, "void k_embed(NormArgs)", "SQ_VALU_MFMA_BUSY_CYCLES", 0, 0, dur_ns),
            _row(2, "void k_embed(NormArgs)", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 0, 0, dur_ns)]
    src, out = tmp_path / "c.csv", tmp_path / "mfma.txt"
    _write(src, rows)
    profiling.summarize_mfma(str(src), str(out), "cmd")
    lines = [ln for ln in open(out) if ln.startswith("| `")]
    assert len(lines) == 1 and "k_proj<1, 2>" in lines[0]   # kernels without MFMA are left out
    cells = [c.strip() for c in lines[0].split("|")[1:-1]]
    assert cells[1] == "1" and cells[3] == "25.0%"
    rate = 512 * 1e6 / (dur_ns * 1e-9) / 1e12
    assert abs(float(cells[4]) - rate) < 0.05

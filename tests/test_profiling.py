"""Host logic of the counter summary (no GPU)."""
import csv
import json

from paper_2607_28418_amd import profiling

FIELDS = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]


def _dump(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for name, v, *grid in rows:
            w.writerow({"Kernel_Name": name, "Grid_Size": grid[0] if grid else 256,
                        "Counter_Name": counter, "Counter_Value": v})


def test_summary_scales_by_copy_and_guards_sources(tmp_path):
    k = "void wide::wide_mn256<true, 64>(wide::MN256Args)"
    _dump(tmp_path / "f.csv", "FETCH_SIZE", [(k, 100.0), (k, 300.0), (profiling.COPY_KERNEL, 3.0, 512),
                                  (profiling.COPY_KERNEL, 512.0, 131072)])
    _dump(tmp_path / "w.csv", "WRITE_SIZE", [(k, 50.0), (k, 50.0), (profiling.COPY_KERNEL, 1024.0, 131072)])
    s = profiling.summarize(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 1024 * 1024, "cmd")
    e = s["kernels"]["wide_mn256<true, 64>"]
    assert s["fetch_scale"] == 2.0 and s["write_scale"] == 1.0
    assert e["fetch_bytes"] == 200 * 1024 * 2 and e["write_bytes"] == 50 * 1024
    p = tmp_path / "s.json"
    p.write_text(json.dumps(s))
    assert profiling.traffic_for(str(p), "wide_mn256<true>/bk64") == 200 * 1024 * 2 + 50 * 1024
    s["source_sha256"] = "0" * 64
    p.write_text(json.dumps(s))
    assert profiling.traffic_for(str(p), "wide_mn256<true>") is None


def test_calibration_is_the_last_two_copies(tmp_path):
    """Earlier copies of the program run the copy kernel with the same grid;
    only the last two dispatches (the calibration copies) set the scale."""
    k = "void wide::wide_attn_fwd<4, 1>(wide::AttnArgs)"
    c = profiling.COPY_KERNEL
    _dump(tmp_path / "f.csv", "FETCH_SIZE", [(c, 16.0, 131072), (k, 10.0), (c, 57.0, 131072), (c, 3.0, 512),
                                             (c, 512.0, 131072), (c, 512.0, 131072)])
    _dump(tmp_path / "w.csv", "WRITE_SIZE", [(c, 16.0, 131072), (k, 10.0), (c, 57.0, 131072), (c, 3.0, 512),
                                             (c, 1024.0, 131072), (c, 1024.0, 131072)])
    s = profiling.summarize(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), 1024 * 1024, "cmd")
    assert s["fetch_scale"] == 2.0 and s["write_scale"] == 1.0
    assert profiling.counter_means(str(tmp_path / "f.csv"))[c]["dispatches"] == 2


def test_label_matching():
    m = profiling.label_matches
    assert m("wide_kd256<64>", "wide_kd256")
    assert m("wide_mn256<true, 32>", "wide_mn256<true>/bk32")
    assert not m("wide_mn256<false, 64>", "wide_mn256<true>")
    assert not m("wide_gemv_n_finish<true>", "wide_gemv_n<true>")
    assert m("wide_gemv_n<true, 4, 2>", "wide_gemv_n<true>")
    assert m("wide_reorder_count", "wide_reorder_count")
    # dense-masked K-axis variants: the label carries the leading template argument
    assert m("wide_kd256<1, 64>", "wide_kd256<1>/bk64")
    assert m("wide_kd256<4, 32>", "wide_kd256<4>")
    assert not m("wide_kd256<4, 64>", "wide_kd256<1>/bk64")
    assert m("wide_kd256<0, 64>", "wide_kd256")


def test_kernel_key_strips_namespaces_and_arguments():
    from paper_2607_28418_amd.profiling import kernel_key, label_matches
    assert kernel_key("void wide::wide_mn256<true, 64>(wide::MN256Args)") == "wide_mn256<true, 64>"
    assert kernel_key("void wide::(anonymous namespace)::wide_attn_fwd<4>(wide::AttnArgs)") == "wide_attn_fwd<4>"
    assert kernel_key("wide::(anonymous namespace)::wide_attn_prep(wide::AttnArgs, unsigned short const*, int*, int)") \
        == "wide_attn_prep"
    assert label_matches("wide_attn_fwd<4>", "wide_attn_fwd")
    assert not label_matches("wide_attn_fwd<4>", "wide_attn_prep")


def test_mfma_summary_normalisation(tmp_path):
    """Utilisation from two counter passes: GRBM_GUI_ACTIVE counts cycles on
    each of 8 XCDs, SQ_VALU_MFMA_BUSY_CYCLES on each of 1024 SIMDs."""
    fields = ["Kernel_Name", "Dispatch_Id", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    k = "void wide::wide_kd256<4, 64>(wide::KArgs)"
    cycles = 2_000_000  # 1 ms at 2 GHz

    def dump(path, counters):
        with open(path, "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=fields)
            w.writeheader()
            for d in (1, 2):
                for c, v in counters.items():
                    w.writerow({"Kernel_Name": k, "Dispatch_Id": d, "Counter_Name": c, "Counter_Value": v,
                                "Start_Timestamp": 0, "End_Timestamp": 1_000_000})

    dump(tmp_path / "a.csv", {"GRBM_GUI_ACTIVE": 8 * cycles, "SQ_VALU_MFMA_BUSY_CYCLES": 0.75 * 1024 * cycles,
                              "SQ_WAVE_CYCLES": 1000.0, "SQ_WAIT_ANY": 250.0})
    dump(tmp_path / "b.csv", {"GRBM_GUI_ACTIVE": 8 * cycles, "SQ_LDS_CMD_FIFO_FULL": 0.1 * 256 * cycles})
    s = profiling.mfma_summary([str(tmp_path / "a.csv"), str(tmp_path / "b.csv")], "cmd")
    r = s["kernels"]["wide_kd256<4, 64>"]
    assert r["dispatches"] == 2 and r["avg_us"] == 1000.0
    assert r["clock_GHz"] == 2.0
    assert r["mfma_busy"] == 0.75
    assert r["wait_any"] == 0.25
    assert r["lds_fifo_full"] == 0.1


def test_source_digest_ignores_comments_not_code():
    a = 'int f() { return 1; } // one\n/* block\n comment */ const char* s = "// not a comment";\n'
    b = 'int f() {   return 1; }\n\n// a different comment\nconst char* s = "// not a comment";'
    c = 'int f() { return 2; } // one\nconst char* s = "// not a comment";\n'
    d = 'int f() { return 1; }\nconst char* s = "// changed";\n'
    assert profiling.code_text(a) == profiling.code_text(b)
    assert profiling.code_text(a) != profiling.code_text(c)
    assert profiling.code_text(a) != profiling.code_text(d)
    assert profiling.code_text("char q = '\\\"'; x(); // c") == "char q = '\\\"'; x();"

"""bench.py's kernel naming (CPU): the keys that tie rocprofv3 counter rows and
kernel traces to one kernel instantiation."""
import bench


def test_kernel_key_demangled_and_mangled():
    cases = {
        "void fox::bwd_dkdv_bf16_kernel<128, false, false, true>(__bf16 const*, int)":
            "bwd_dkdv_bf16_kernel<128,false,false,true>",
        "_ZN3fox20bwd_dkdv_bf16_kernelILi128ELb0ELb0ELb1EEEvPKDF16bS2_":
            "bwd_dkdv_bf16_kernel<128,false,false,true>",
        "_ZN3fox20bwd_dkdv_bf16_kernelILi128ELb0ELb0ELb0EEEvPKDF16bS2_":
            "bwd_dkdv_bf16_kernel<128,false,false,false>",
        "void fox::bwd_dq_stored_kernel<128, false>(__bf16 const*, float)":
            "bwd_dq_stored_kernel<128,false>",
        "_ZN3fox20bwd_dq_stored_kernelILi128ELb1EEEvPKDF16bPKDv8_DF16bPKiPDF16bPfiiif":
            "bwd_dq_stored_kernel<128,true>",
        "_ZN3fox19decode_split_kernelIDF16bLi128ELb0ELb1EEEv": "decode_split_kernel<__bf16,128,false,true>",
        "fox::gate_proj_reduce_kernel(float const*, float const*, float*, float*, int, int, int)":
            "gate_proj_reduce_kernel",
        "void fox::log_sigmoid_kernel(float const*, float*, float*, unsigned long)":
            "log_sigmoid_kernel",
        "__amd_rocclr_copyBuffer": "copy",
        "void at::native::vectorized_elementwise_kernel<4>": None,
    }
    for name, key in cases.items():
        assert bench._kernel_key(name) == key, name


def test_every_traffic_kernel_has_sources():
    for k in bench.SQ_KERNELS + bench.ROOFLINE_KERNELS:
        assert k.split("<")[0] in bench.KERNEL_SOURCES


def test_traffic_file_names_the_benchmarked_kernels():
    """Every kernel whose measured traffic the benchmark reports has a row in the
    committed traffic summary (the hash that gates its use is checked at run time)."""
    rows = [line.split()[0] for line in open(bench.TRAFFIC_FILE)
            if line.strip() and not line.startswith("#")]
    for k in bench.ROOFLINE_KERNELS:
        assert k in rows, k


def test_trace_summary_counts_every_grid_dimension(tmp_path):
    """A kernel trace row gives the grid in work-items per dimension: a 2D launch
    of (16, 256) workgroups of 256 threads is 4096 workgroups."""
    import sqlite3
    db = tmp_path / "t.db"
    con = sqlite3.connect(db)
    con.execute("create table kernels (name text, grid_x int, grid_y int, grid_z int, "
                "workgroup_x int, workgroup_y int, workgroup_z int, duration int, lds_size int)")
    rows = [("void fox::gate_proj_bwd_kernel<true, 1>(float const*)", 4096, 256, 1, 256, 1, 1,
             27000, 37888),
            ("void fox::gate_proj_bwd_kernel<true, 1>(float const*)", 4096, 256, 1, 256, 1, 1,
             29000, 37888),
            ("fox::gate_proj_reduce_kernel(float const*)", 262400, 1, 1, 256, 1, 1, 3000, 0),
            ("__amd_rocclr_copyBuffer", 1024, 1, 1, 256, 1, 1, 5000, 0)]
    con.executemany("insert into kernels values (?, ?, ?, ?, ?, ?, ?, ?, ?)", rows)
    con.commit()
    con.close()
    text = bench.trace_summary(str(db), "cmd")
    assert "| gate_proj_bwd_kernel<true,1> | 4096 | 256 | 2 | 28.0 | 27.0 | 29.0 | 37888 |" in text
    assert "| gate_proj_reduce_kernel | 1025 | 256 | 1 | 3.0 | 3.0 | 3.0 | 0 |" in text
    assert "copy" not in text.split("|---|")[-1]


def test_training_leg_reports_the_faster_backward():
    import paper_2503_02130_amd.inputs as inputs
    w = inputs.WORKLOADS["fwdbwd_bf16_b8_h12_l2048_d64"]
    r = {"gate_prefix": 0.006, "fwd": 0.07, "delta": 0.009, "dkdv_store": 0.178,
         "dq_stored": 0.081, "dkdv": 0.155, "dq": 0.095, "scan": 0.007, "store_bytes": 4.3e8}
    fl = bench.fwd_flops(8, 12, 2048, 64) + bench.bwd_flops(8, 12, 2048, 64)
    for stored_ms, recompute_ms, main, other in ((0.36, 0.35, "recompute", "stored"),
                                                 (0.34, 0.35, "stored", "recompute")):
        out = bench.train_graph_summary(w, dict(r, stored_ms=stored_ms, recompute_ms=recompute_ms))
        assert out["ms_per_step"] == min(stored_ms, recompute_ms)
        assert abs(out["TFLOP/s"] - fl / (min(stored_ms, recompute_ms) * 1e-3) / 1e12) < 0.01
        assert out[other]["ms_per_step"] == max(stored_ms, recompute_ms)
        kernel = "true" if main == "stored" else "false"
        assert out["roofline"]["kernel"].startswith(f"bwd_dkdv_bf16_kernel<64,false,false,{kernel}>")

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

"""Host-side helpers that turn rocprofv3 output into the committed summaries."""
import csv

from paper_2606_19025_amd import profiling as P


def test_symbols_map_to_timing_names():
    assert P.timing_name("void moe::(anonymous namespace)::gemm_bf16_kernel<5>("
                         "moe::(anonymous namespace)::GemmArgs)") == "gemm_dwgu"
    assert P.timing_name("_ZN3moe12_GLOBAL__N_116gemm_bf16_kernelILi2EEEvNS0_8GemmArgsE") \
        == "gemm_dhh_bwd"
    assert P.timing_name("void moe::(anonymous namespace)::gemm_bf16_kernel<1, 1>("
                         "moe::(anonymous namespace)::GemmLaunch)") == "gemm_down_fwd"
    assert P.timing_name("_ZN3moe12_GLOBAL__N_116gemm_bf16_kernelILi3ELi5EEEvNS0_10GemmLaunchE") \
        == "gemm_dx_dwgu"
    assert P.timing_name("void moe::(anonymous namespace)::gemm_bf16_kernel<2, 4>(x)") \
        == "gemm_dhh_dwd"
    assert P.timing_name("_ZN3moe12_GLOBAL__N_118combine_fwd_kernelIDF16bEEvPKT_") == "combine_fwd"
    assert P.timing_name("moe::(anonymous namespace)::route_bwd_mfma_kernel(x)") == "route_bwd_mfma"
    assert P.timing_name("_ZN3moe12_GLOBAL__N_123combine_bwd_rows_kernelIDF16bEEvPKT_S4_") \
        == "combine_bwd"
    assert P.timing_name("moe::(anonymous namespace)::splitk_rows_reduce_kernel(x)") \
        == "splitk_rows_reduce"
    assert P.timing_name("__amd_rocclr_copyBuffer") is None
    assert P.source_digest("gemm_gu_fwd") != P.source_digest("route_fwd")


def test_traffic_summary_is_scaled_by_the_calibration_copy(tmp_path):
    kib = P.CALIBRATION_BYTES / 1024

    def write(path, counter, copy_kib, kern_kib):
        with open(path, "w", newline="") as f:
            w = csv.writer(f)
            w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
            w.writerow([1, "__amd_rocclr_copyBuffer", counter, copy_kib])
            for i, v in enumerate(kern_kib):  # two dimensions of one dispatch are summed
                w.writerow([2 + i, "void moe::(anonymous namespace)::gemm_bf16_kernel<0>(a)",
                            counter, v / 2])
                w.writerow([2 + i, "void moe::(anonymous namespace)::gemm_bf16_kernel<0>(a)",
                            counter, v / 2])

    fc, wc, out = tmp_path / "f.csv", tmp_path / "w.csv", tmp_path / "t.txt"
    write(fc, "FETCH_SIZE", kib / 2, [100.0, 300.0])   # counter reads half of a copy's bytes
    write(wc, "WRITE_SIZE", kib, [50.0, 50.0])
    P.traffic(str(fc), str(wc), str(out), "rocprofv3 --pmc {COUNTER} -- prog")
    t = P.load_traffic(str(out))
    b, dg = t["gemm_gu_fwd"]
    assert abs(b - (200.0 * 1024 * 2 + 50.0 * 1024)) < 1.0
    assert dg == P.source_digest("gemm_gu_fwd")
    assert "FETCH_SIZE" in out.read_text()


def test_digest_ignores_comments_and_layout():
    a = "int f(int x) {  // doubles x\n  return 2 * x; /* no overflow check */\n}\n"
    b = "// header\nint f(int x) {\n    return 2 * x;\n}"
    c = "int f(int x) { return 3 * x; }"
    assert P._code_only(a) == P._code_only(b)
    assert P._code_only(a) != P._code_only(c)


def test_every_kernel_of_the_library_has_a_timing_name():
    """Each __global__ kernel in csrc/ maps to a name, so that no kernel is
    missing from the committed summaries."""
    import glob
    import os
    import re
    names = set()
    for f in glob.glob(os.path.join(P.CSRC, "*.hip")):
        src = open(f).read()
        names |= set(re.findall(r"__global__\s+(?:__launch_bounds__\([^)]*\)\s+)?void\s+(\w+_kernel)\s*\(", src))
    assert len(names) >= 15
    for n in sorted(names):
        # (template arguments as a templated kernel would carry them)
        assert P.timing_name(f"void moe::(anonymous namespace)::{n}<0, 0>(x)") is not None, n


def test_mangled_names_shorten_to_the_kernel():
    assert P._mangled_kernel_name(
        "_ZN3moe12_GLOBAL__N_123combine_bwd_rows_kernelIDF16bEEvPKT_S4_") == "combine_bwd_rows_kernel"
    assert P._mangled_kernel_name("not_mangled") == "not_mangled"

"""Host logic of the rocprofv3 summary (paper_2405_14009_amd/profile_summary.py):
kernel classes of the library's kernel names, the arithmetic of the MFMA and
L1 -> L2 counter passes on small synthetic counter files, and the source
digest that ties a summary to the kernel code it was taken with."""
import csv

import pytest

from paper_2405_14009_amd import profile_summary as ps

NS = "void (anonymous namespace)::"


@pytest.mark.parametrize("name, cls", [
    (NS + "gemm_bf16_persist_kernel<5, false, false, true>(GemmParams)", "gemm_wgrad"),
    (NS + "gemm_bf16_persist_kernel<5, false, false, false>(GemmParams)", "gemm_wgrad"),
    (NS + "gemm_bf16_persist_kernel<5, false, false>(GemmParams)", "gemm_wgrad"),
    (NS + "gemm_bf16_pp_kernel<128, 2, 3, 4, true, true, 0>(GemmParams)", "gemm_dgrad"),
    (NS + "gemm_bf16_pp_kernel<128, 2, 3, 4, true, false, 2>(GemmParams)", "gemm_fwd"),
    (NS + "gemm_bf16_pp_kernel<128, 2, 3, 4, true, false, 1>(GemmParams)", "gemm_fwd"),
    (NS + "gemm_bf16_pp_kernel<128, 2, 3, 4, false, false, 5>(GemmParams)", "gemm_wgrad"),
    (NS + "gemm_bf16_kernel<256, 256, 8, 1, 64, 2, true, false, 3>(GemmParams)", "gemm_fwd"),
    (NS + "gemm_bf16_kernel<256, 256, 8, 1, 64, 2, true, true, 4>(GemmParams)", "gemm_dgrad"),
    (NS + "gemm_bf16_kernel<256, 256, 8, 1, 64, 2, false, false, 5>(GemmParams)", "gemm_wgrad"),
    (NS + "gemm_bf16_kernel<256, 256, 8, 1, 64, 2, true, false, 6>(GemmParams)", "gemm_other"),
    ("(anonymous namespace)::attn_bwd_kv_k<true>((anonymous namespace)::AttnArgs)", "attn_bwd"),
    ("(anonymous namespace)::attn_bwd_q_pair_k((anonymous namespace)::AttnArgs)", "attn_bwd"),
    ("(anonymous namespace)::attn_fwd_pair_k((anonymous namespace)::AttnArgs)", "attn_fwd"),
    ("(anonymous namespace)::attn_fwd_k<true>((anonymous namespace)::AttnArgs)", "attn_fwd"),
    ("_ZN12_GLOBAL__N_113ln_bwd_wave_kIDF16bLi8EEEvPKT_S3_PKfS5_S5_S3_PS1_S6_li", "layernorm"),
    ("_ZN12_GLOBAL__N_113ln_fwd_wave_kIDF16bLi8EEEvPKT_PKfS5_PS1_S6_PfS7_lif", "layernorm"),
    ("void colsum_part16_k<bool _Accum, bool, E>(ColSegs, long, long, int, int, float*, ColSegs)", "reduce"),
    ("(anonymous namespace)::adamw_k(HIP_vector_type<float, 4u>*)", "adamw"),
    ("__amd_rocclr_copyBuffer", "copy"),
])
def test_kernel_class(name, cls):
    assert ps.kernel_class(name) == cls


def _write(path, rows):
    cols = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(cols, r)))


def test_mfma_pass_arithmetic(tmp_path):
    # one 100 us forward GEMM dispatch: 8 XCDs x 200000 active cycles (2 GHz),
    # half of the 1024 SIMDs' cycles busy, 2^30 bf16 MOPS (512 flop each)
    name = NS + "gemm_bf16_kernel<256, 256, 8, 1, 64, 2, true, false, 3>(GemmParams)"
    cyc = 200000
    rows = [(1, name, "GRBM_GUI_ACTIVE", 8 * cyc, 0, 100000),
            (1, name, "SQ_VALU_MFMA_BUSY_CYCLES", 0.5 * cyc * 1024, 0, 100000),
            (1, name, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 2 ** 30, 0, 100000)]
    p = tmp_path / "mfma.csv"
    _write(p, rows)
    out = ps.mfma_classes(str(p))["gemm_fwd"]
    assert out["mfma_busy_pct"] == 50.0
    assert out["mfma_bf16_flops_per_dispatch"] == 512 * 2 ** 30
    assert out["mfma_bf16_tflops_executed"] == round(512 * 2 ** 30 / 100000 / 1e3, 1)
    assert out["sclk_ghz"] == 2.0


def test_l2_pass_arithmetic(tmp_path):
    # 256 CUs x 1000 cycles; 64 requests in flight per CU at 400 cycles each
    name = NS + "gemm_bf16_pp_kernel<128, 2, 3, 4, true, true, 0>(GemmParams)"
    cyc, lat, infl = 1000, 400, 64
    req = infl * 256 * cyc / lat
    rows = [(1, name, "GRBM_GUI_ACTIVE", 8 * cyc, 0, 1),
            (1, name, "TCP_TCC_READ_REQ_sum", req, 0, 1),
            (1, name, "TCP_TCC_READ_REQ_LATENCY_sum", req * lat, 0, 1),
            (1, name, "TCC_HIT_sum", 80, 0, 1),
            (1, name, "TCC_MISS_sum", 20, 0, 1)]
    # the copy probe: 1 GiB read in 128-byte requests
    copy = [(1, "__amd_rocclr_copyBuffer", "TCP_TCC_READ_REQ_sum", ps.COPY_BYTES / 128, 0, 1)]
    p, c = tmp_path / "l2.csv", tmp_path / "copy.csv"
    _write(p, rows)
    _write(c, copy)
    out = ps.l2_classes(str(p), str(c))["gemm_dgrad"]
    assert out["l2_hit_pct"] == 80.0
    assert out["l1_l2_read_latency_cycles"] == lat
    assert out["read_requests_in_flight_per_cu"] == infl
    assert out["read_request_bytes"] == 128.0
    assert out["read_bytes_per_clk_per_cu"] == round(infl * 128 / lat, 2)


def test_sources_digest_is_stable():
    assert ps.sources_digest() == ps.sources_digest()
    assert len(ps.sources_digest()) == 64


def test_sources_digest_ignores_comments_only(tmp_path):
    src = tmp_path / "k.hip"
    src.write_text("// header\n__global__ void k(int* p) {\n  p[0] = 1;  // store\n}\n")
    base = ps.sources_digest(str(tmp_path))
    src.write_text("// a new header\n/* and a block\n comment */\n__global__ void k(int* p) {\n  p[0] = 1;\n}\n")
    assert ps.sources_digest(str(tmp_path)) == base
    src.write_text("// header\n__global__ void k(int* p) {\n  p[0] = 2;  // store\n}\n")
    assert ps.sources_digest(str(tmp_path)) != base

"""Host logic of the measurement tools (no GPU): the counter summaries that
bench.py attaches to its line are computed from rocprofv3 CSV files; here
from small synthetic files whose figures are worked out by hand."""
import csv
import json
import os

import pytest

from paper_2608_13057_amd import measure

GU = "void tempo::(anonymous namespace)::k_gemm_big_f8<true>(tempo::(anonymous namespace)::F8Args)"
COPY = "void at::native::vectorized_elementwise_kernel<4, at::native::AUnaryFunctor<float, float, float, " \
       "at::native::binary_internal::MulFunctor<float> >, std::array<char*, 2ul> >(int, ...)"


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(header)
        w.writerows(rows)


def _counters(d, rows):
    _write(os.path.join(d, "run_counter_collection.csv"), ["Kernel_Name", "Counter_Name", "Counter_Value"], rows)


def _agent(d):
    _write(os.path.join(d, "run_agent_info.csv"), ["Name", "Num_Xcc", "Simd_Count", "Max_Engine_Clk_Fcompute"],
           [["gfx950", 8, 1024, 2400]])


def test_kernel_classification():
    assert measure._is_gateup(GU)
    assert measure._is_gateup("void tempo::(anonymous namespace)::k_gemm_big<true>(tempo::gemm::GemmArgs)")
    assert not measure._is_gateup("void tempo::(anonymous namespace)::k_gemm_big<false>(tempo::gemm::GemmArgs)")
    assert measure._is_gateup("void tempo::gemm::k_gemm<false, 64, true, false>(tempo::gemm::GemmArgs)")
    assert not measure._is_gateup("void tempo::gemm::k_gemm<false, 64, false, false>(tempo::gemm::GemmArgs)")
    assert measure._is_copy(COPY) and not measure._is_copy(GU)


def test_mfma_summary_arithmetic(tmp_path):
    """Two dispatches: busy cycles 2e8 / 3e8, GRBM_GUI_ACTIVE (summed over 8
    XCDs) 3.2e6 / 4.8e6, MOPS 1e8 / 1e8, mean duration 200 us.  Mean busy
    2.5e8 over 4e6 / 8 = 5e5 dispatch cycles x 1024 SIMDs: 0.48828125;
    clock 5e5 cycles / 200 us = 2.5 GHz; executed 1e8 x 512 flops in 200 us:
    256 TFLOP/s."""
    pmc, kt = str(tmp_path / "pmc"), str(tmp_path / "kt")
    _counters(pmc, [[GU, "SQ_VALU_MFMA_BUSY_CYCLES", 2e8], [GU, "SQ_VALU_MFMA_BUSY_CYCLES", 3e8],
                    [GU, "GRBM_GUI_ACTIVE", 3.2e6], [GU, "GRBM_GUI_ACTIVE", 4.8e6],
                    [GU, "SQ_INSTS_VALU_MFMA_MOPS_F8", 1e8], [GU, "SQ_INSTS_VALU_MFMA_MOPS_F8", 1e8],
                    ["other", "GRBM_GUI_ACTIVE", 1.0]])
    _agent(pmc)
    _write(os.path.join(kt, "run_kernel_stats.csv"), ["Name", "Calls", "AverageNs", "MinNs", "MaxNs", "Percentage"],
           [[GU, 2, 200000.0, 190000.0, 210000.0, 50.0]])
    out = str(tmp_path / "m.md")

    class A:
        pass

    a = A()
    a.pmc_dir, a.trace_dir, a.workload, a.m_tile, a.out, a.command1, a.command2 = \
        pmc, kt, "qwen3_prefill_fp8mx", 256, out, "c1", "c2"
    assert measure._mfma(a) == 0
    line = [l for l in open(out) if l.startswith("mfma_json: ")][0]
    d = json.loads(line[len("mfma_json: "):])
    assert d["mfma_busy"] == pytest.approx(0.48828125)
    assert d["clock_ghz"] == pytest.approx(2.5)
    assert d["executed_tflops"] == pytest.approx(256.0)
    assert d["dispatches"] == 2 and d["source_hash"] == measure.gemm_source_hash()


def test_traffic_summary_scales_by_the_copy(tmp_path):
    """The gate/up kernel's FETCH_SIZE (KiB per dispatch) is scaled by what the
    counter reads for the 256 MiB copy: a copy reading 131072 KiB where
    262144 KiB were read gives 2.0, so 1000 KiB of the kernel are 2048000
    bytes; WRITE_SIZE of the copy reads its true 262144 KiB (factor 1)."""
    fe, wr = str(tmp_path / "fe"), str(tmp_path / "wr")
    _counters(fe, [[GU, "FETCH_SIZE", 1000.0], [GU, "FETCH_SIZE", 1000.0], [COPY, "FETCH_SIZE", 131072.0]])
    _counters(wr, [[GU, "WRITE_SIZE", 50.0], [COPY, "WRITE_SIZE", 262144.0]])
    out = str(tmp_path / "t.md")

    class A:
        pass

    a = A()
    a.fetch_dir, a.write_dir, a.workload, a.m_tile, a.out, a.command1, a.command2 = \
        fe, wr, "qwen3_prefill_fp8mx", 256, out, "c1", "c2"
    assert measure._traffic(a) == 0
    line = [l for l in open(out) if l.startswith("traffic_json: ")][0]
    d = json.loads(line[len("traffic_json: "):])
    assert d["copy_fetch_factor"] == pytest.approx(2.0) and d["copy_write_factor"] == pytest.approx(1.0)
    assert d["fetch_bytes"] == pytest.approx(2048000.0) and d["write_bytes"] == pytest.approx(51200.0)
    assert d["bytes_per_launch"] == pytest.approx(2099200.0)


def test_committed_summaries_match_their_sources():
    """Every committed counter summary names the stage-2 source hash it was
    taken with; bench.py drops figures whose hash differs."""
    for name, m in (("qwen3_prefill_fp8mx", 256), ("qwen3_prefill_bf16", 256)):
        d = measure.committed_mfma(name, m)
        if d is not None:
            assert d["source_hash"] == measure.gemm_source_hash()
    b, current = measure.committed_traffic("qwen3_decode_bf16", 64)
    assert b is None or b > 0

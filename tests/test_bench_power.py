"""bench.py --power: parsing of the board readings (no GPU, no amd-smi call)."""
import bench

HEADER = ("gpu,socket_power,gfx_voltage,soc_voltage,mem_voltage,throttle_status,power_management,"
          + ",".join("gfx_%d_clk,gfx_%d_min_clk,gfx_%d_max_clk,gfx_%d_clk_locked,gfx_%d_deep_sleep"
                     % ((i,) * 5) for i in range(8))
          + ",mem_0_clk")


def _row(power, clocks):
    return ("0,%s,N/A,N/A,N/A,N/A,N/A," % power
            + ",".join("%s,500,2400,DISABLED,DISABLED" % c for c in clocks) + ",2000")


def test_parse_reads_power_and_every_xcd_clock():
    clocks = [1646, 1567, 1692, 1609, 1728, 1639, 1666, 1604]
    power, got = bench.parse_smi_csv(HEADER + "\n" + _row(1396, clocks) + "\n")
    assert power == 1396.0
    assert got == [float(c) for c in clocks]  # gfx_N_clk only, not min/max/mem clocks


def test_parse_rejects_missing_or_unreadable_fields():
    assert bench.parse_smi_csv("") is None
    assert bench.parse_smi_csv("gpu,gfx_0_clk\n0,1600\n") is None      # no socket_power
    assert bench.parse_smi_csv(HEADER + "\n" + _row("N/A", [1600] * 8)) is None


def test_mfma_ceiling_reads_the_program_output(tmp_path, monkeypatch):
    # A stand-in for the measuring program: the wrapper runs it with the run
    # length and keeps the rate of each data kind (no GPU involved).
    fake = tmp_path / "mfma_ceiling"
    line = "echo '{\"mfma\": \"%s\", \"data\": \"%s\", \"ms\": 20.1, \"tflops\": %s, \"frac_nominal\": 0.7, \"iters\": 9}'\n"
    fake.write_text("#!/bin/sh\n" + line % ("32x32x16", "random", "1702.5") + line % ("32x32x16", "zero", "2450.0")
                    + line % ("16x16x32", "random", "2090.0") + line % ("16x16x32", "zero", "2470.0"))
    fake.chmod(0o755)
    monkeypatch.setattr(bench, "MFMA_CEILING", str(fake))
    got = bench.mfma_ceiling(20.0)
    assert got["random_data_tflops"] == 1702.5 and got["zero_data_tflops"] == 2450.0
    assert got["random_data_tflops_16x16x32"] == 2090.0 and got["zero_data_tflops_16x16x32"] == 2470.0
    monkeypatch.setattr(bench, "MFMA_CEILING", str(tmp_path / "missing"))
    assert "error" in bench.mfma_ceiling()


def test_mfma_instruction_of_a_kernel_name():
    assert bench.mfma_instruction("gemm_mfma_kernel<GemmShape<2, 4, 2, 1, 4, 2, 64>, 0, false, false>") == "16x16x32"
    assert bench.mfma_instruction("gemm_mfma_kernel<GemmShape<1, 4, 2, 2, 2, 3, 64>, 1, true, false>") == "16x16x32"
    assert bench.mfma_instruction("gemm_mfma_kernel<GemmShape<2, 4, 2, 1, 2, 3, 64>, 0, true, true>") == "32x32x16"
    assert bench.mfma_instruction("gemv_splitk_kernel<1, 2, 0, false>") == "32x32x16"

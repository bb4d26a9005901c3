"""The measurement aids on the GPU: gemm_probe_read reads every byte of its range once
(the XOR of its per-thread outputs equals the XOR of the buffer's dwords) and rejects
bad arguments; gemm_probe_mfma reports a sustained rate and clock (needs an MI355X)."""
import numpy as np
import pytest
import torch

from paper_2512_13282_amd import binding as b

pytestmark = pytest.mark.gpu


def _threads():
    return torch.cuda.get_device_properties(0).multi_processor_count * 2048


@pytest.mark.parametrize("nbytes", [16, 4096 * 16 + 48, 64 << 20])
def test_read_probe_reads_every_byte_once(nbytes):
    g = torch.Generator(device="cuda:0")
    g.manual_seed(nbytes)
    buf = torch.randint(-2 ** 31, 2 ** 31 - 1, (nbytes // 4 + 4,), dtype=torch.int32, device="cuda:0", generator=g)
    sink = torch.full((_threads(),), 12345, dtype=torch.int32, device="cuda:0")
    st = torch.cuda.current_stream().cuda_stream
    assert b.gemm_probe_read(buf.data_ptr(), nbytes, sink.data_ptr(), sink.numel(), st) == b.GEMM_OK
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(buf[: nbytes // 4].cpu().numpy().view(np.uint32))
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == want


def test_read_probe_rejects_bad_arguments():
    buf = torch.zeros(64, dtype=torch.int32, device="cuda:0")
    sink = torch.zeros(_threads(), dtype=torch.int32, device="cuda:0")
    p, s, n = buf.data_ptr(), sink.data_ptr(), sink.numel()
    assert b.gemm_probe_read(p + 4, 64, s, n) == b.GEMM_ERR_INVALID_VALUE      # misaligned source
    assert b.gemm_probe_read(p, 60, s, n) == b.GEMM_ERR_INVALID_VALUE          # not a multiple of 16
    assert b.gemm_probe_read(p, -16, s, n) == b.GEMM_ERR_INVALID_VALUE
    assert b.gemm_probe_read(p, 64, s, n - 1) == b.GEMM_ERR_INVALID_VALUE      # sink too small
    assert b.gemm_probe_read(p, 64, 0, n) == b.GEMM_ERR_INVALID_VALUE


@pytest.mark.parametrize("dtype", [b.GEMM_DTYPE_I8_I32, b.GEMM_DTYPE_BF16_F32], ids=["i8", "bf16"])
def test_mfma_probe_reports_a_plausible_rate(dtype):
    rc, info = b.gemm_probe_mfma(dtype, True, 2000)
    assert rc == b.GEMM_OK
    wg = int(info["workgroups"])
    clocks = torch.zeros(2 * wg, dtype=torch.int64, device="cuda:0")
    sink = torch.zeros(wg * int(info["threads_per_workgroup"]), dtype=torch.int32, device="cuda:0")
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    rc, _ = b.gemm_probe_mfma(dtype, True, 2000, clocks.data_ptr(), sink.data_ptr(), st.cuda_stream)
    e1.record(st)
    torch.cuda.synchronize()
    assert rc == b.GEMM_OK
    rate = info["ops_per_launch"] / (e0.elapsed_time(e1) * 1e-3) / 1e12
    peak = 5000.0 if dtype == b.GEMM_DTYPE_I8_I32 else 2500.0
    assert 0.2 * peak < rate < 1.05 * peak
    c = clocks.view(wg, 2).double().cpu()
    ghz = float((c[:, 0] / c[:, 1]).mean()) * info["wall_clock_hz"] / 1e9
    assert 0.5 < ghz < 2.6

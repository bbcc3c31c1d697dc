"""The achievable-peak calibration kernels (include/kvp_calib.h) on the GPU: they launch,
leave their sink untouched (it is written only on an impossible value), and the rates they
imply are below the datasheet peaks."""
import pytest
import torch

from paper_2608_15943_amd import binding as kb

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kb.lib()


def _time_ms(fn):
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    fn()
    e0.record(st)
    fn()
    e1.record(st)
    e1.synchronize()
    return e0.elapsed_time(e1)


def test_calibration_kernels_run_and_stay_below_datasheet_peaks():
    st = torch.cuda.current_stream().cuda_stream
    sink = torch.zeros(64, dtype=torch.uint8, device="cuda")
    flops = {}

    def mfma():
        flops["n"] = kb.kvp_calib_mfma_bf16(2000, sink.data_ptr(), st)
    ms = _time_ms(mfma)
    tflops = flops["n"] / (ms * 1e-3) / 1e12
    n = 1 << 30
    buf = torch.ones(n // 4, dtype=torch.int32, device="cuda")
    ms_r = _time_ms(lambda: kb.kvp_calib_stream_read(buf.data_ptr(), n, sink.data_ptr(), st))
    gbs = n / (ms_r * 1e-3) / 1e9
    torch.cuda.synchronize()
    print(f"  calibration: {tflops:.0f} TFLOP/s bf16, {gbs:.0f} GB/s read (1 GiB)")
    assert int(sink.sum().item()) == 0
    assert 100 < tflops < 2516.6
    assert 500 < gbs < 8000

"""The stream probe (a measurement aid beside the roofline): it reads a device buffer through
LDS the way the GEMM and attention kernels load operands, writes nothing, and its rate with
every CU streaming stays between a floor no working HBM path misses and the published peak."""
import pytest
import torch

from paper_2607_14647_amd import lib as L
from tests.gpu_common import need_gpu, note

pytestmark = pytest.mark.gpu


def _rate(buf, workgroups, reps=3):
    L.stream_probe(buf, workgroups)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        L.stream_probe(buf, workgroups)
    b.record()
    torch.cuda.synchronize()
    return buf.numel() * reps / (a.elapsed_time(b) * 1e-3) / 1e9


def test_stream_probe_reads_at_hbm_rates_and_writes_nothing():
    need_gpu()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    buf = torch.arange(1 << 28, dtype=torch.int32, device="cuda").view(torch.uint8)   # 1 GiB
    before = buf[:: 1 << 20].clone()
    full = _rate(buf, 2 * cus)
    one = _rate(buf[: 32 * 4096 * 256], 32)       # 32 workgroups: about one CU each
    note(f"stream probe: {full:.0f} GB/s with {2 * cus} workgroups, {one / 32:.1f} GB/s per workgroup with 32")
    assert 1000.0 < full < 8000.0
    assert one < full
    assert torch.equal(buf[:: 1 << 20], before)


def test_stream_probe_ragged_sizes_are_rejected():
    need_gpu()
    buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    with pytest.raises(L.DcutError):
        L.stream_probe(buf[: (1 << 20) - 1024], 4)    # not a whole number of 1 KB loads per wave
    with pytest.raises(L.DcutError):
        L.stream_probe(buf[8:], 1)                    # misaligned
    L.stream_probe(buf, 256)                          # 1 KB per wave: one load each
    torch.cuda.synchronize()

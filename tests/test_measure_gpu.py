"""The measurement calls of include/mg3m_measure.h on the GPU: the copy and
fill probes move exactly their bytes, the MFMA probe reports its flops, and
the timing events (no system-scope fence) time a kernel and the hooked main
convolution kernel of a call."""
import numpy as np
import pytest

from paper_2307_04941_amd import mg3m
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def test_copy_and_fill_probes():
    import torch
    n = (1 << 20) + 4                        # 16-byte multiple, not a whole number of blocks
    src = torch.arange(n, dtype=torch.float32, device="cuda")
    dst = torch.full((n,), -1.0, device="cuda")
    mg3m.mg3m_probe_copy(src, dst, 4 * n)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    mg3m.mg3m_probe_fill(dst, 4 * (n - 4))
    torch.cuda.synchronize()
    assert float(dst[: n - 4].abs().max()) == 0.0 and torch.equal(dst[n - 4:], src[n - 4:])


def test_mfma_probe_and_empty_launch():
    import torch
    sink = torch.zeros(64 * 256, dtype=torch.float32, device="cuda")
    flops = mg3m.mg3m_probe_mfma_f32(sink, 64, 100)
    mg3m.mg3m_launch_empty()
    torch.cuda.synchronize()
    assert flops == 64 * 4 * 100 * 8 * 4096
    assert np.isfinite(sink.cpu().numpy()).all()


def test_timing_events():
    import torch
    n = 1 << 26                              # 256 MiB copied: a few tens of microseconds
    src = torch.zeros(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    mg3m.mg3m_probe_copy(src, dst, 4 * n)    # untimed: the first touch of dst is slower
    torch.cuda.synchronize()
    e0, e1, e2 = mg3m.TimingEvent(), mg3m.TimingEvent(), mg3m.TimingEvent()
    e0.record()
    mg3m.mg3m_probe_copy(src, dst, 4 * n)
    e1.record()
    mg3m.mg3m_probe_copy(src, dst, 4 * n)
    mg3m.mg3m_probe_copy(src, dst, 4 * n)
    e2.record()
    torch.cuda.synchronize()
    one, two = e0.elapsed_ms(e1), e1.elapsed_ms(e2)
    say(f"copy of 256 MiB: {1e3 * one:.1f} us, two copies: {1e3 * two:.1f} us")
    assert 0.0 < one and 1.2 * one < two < 4.0 * one
    # the hook around a call's main kernel, with timing events
    x = torch.rand((14, 14, 64, 32), device="cuda")
    w = torch.rand((3, 3, 64, 64), device="cuda")
    y = torch.empty((14, 14, 64, 32), device="cuda")
    k0, k1, c0, c1 = (mg3m.TimingEvent() for _ in range(4))
    c0.record()
    mg3m.mg3m_time_next_kernel(k0, k1)
    mg3m.conv2d_fwd_f32(x, w, y, 32, 64, 14, 14, 64, 3, 3, 1, 1, "HWCN")
    c1.record()
    torch.cuda.synchronize()
    kernel, call = k0.elapsed_ms(k1), c0.elapsed_ms(c1)
    assert 0.0 < kernel <= call, (kernel, call)
    for e in (e0, e1, e2, k0, k1, c0, c1):
        e.close()

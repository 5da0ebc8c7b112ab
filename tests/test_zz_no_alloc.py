"""conv2d_fwd_f32_noalloc: the convolution for callers that cannot allocate
device memory, whose plan workspace lives in the library's fixed per-device
scratch array.  Checked through the C ABI against conv2d_fwd_f32 (the entry
point it is a variant of) and the fp64 oracle: on small-integer data every
partial sum is exact in fp32, so both entry points must match the oracle bit
for bit whatever plans they run; on uniform data both must lie within
1e-5 * sum|x*w| of it.  Two calls in a row, the second on a smaller input,
so that the second reads a scratch array still holding the first call's
partials."""
import numpy as np
import pytest

import oracle
from paper_2307_04941_amd import mg3m
from tests.gpu_util import assert_parity, make, say, to_dev

pytestmark = pytest.mark.gpu

SCRATCH = 128 << 20

# (larger, smaller) pairs whose selector plans use a workspace: split-K
# partials (HWCN), and the filter copy plus partials of tap-major NCHW.
PAIRS = [
    ("HWCN", (16, 256, 14, 14, 256, 3, 3, 1, 1), (4, 128, 9, 11, 96, 3, 3, 1, 1)),
    ("NCHW", (8, 128, 14, 14, 256, 3, 3, 1, 1), (2, 64, 10, 9, 40, 3, 3, 1, 1)),
    ("HWCN", (32, 512, 7, 7, 512, 3, 3, 1, 1), (8, 256, 7, 7, 64, 1, 1, 1, 0)),
]


def _noalloc(x, w, shape, layout):
    import torch
    N, C, H, W, K, R, S, st, pd = shape
    Ho, Wo = mg3m.conv2d_out_dims(H, W, R, S, st, pd)
    ys = (Ho, Wo, K, N) if layout == "HWCN" else (N, K, Ho, Wo)
    xd, wd = to_dev(x), to_dev(w)
    y = torch.full(ys, float("nan"), dtype=torch.float32, device="cuda")
    mg3m.conv2d_fwd_f32_noalloc(xd, wd, y, N, C, H, W, K, R, S, st, pd, layout,
                                torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def _plain(x, w, shape, layout):
    import torch
    N, C, H, W, K, R, S, st, pd = shape
    Ho, Wo = mg3m.conv2d_out_dims(H, W, R, S, st, pd)
    ys = (Ho, Wo, K, N) if layout == "HWCN" else (N, K, Ho, Wo)
    xd, wd = to_dev(x), to_dev(w)
    y = torch.full(ys, float("nan"), dtype=torch.float32, device="cuda")
    mg3m.conv2d_fwd_f32(xd, wd, y, N, C, H, W, K, R, S, st, pd, layout,
                        torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("case", range(len(PAIRS)))
@pytest.mark.parametrize("dist", ["int", "uniform"])
def test_noalloc_matches_plain_entry_point(case, dist):
    layout, big, small = PAIRS[case]
    for shape in (big, small):
        ws = mg3m.conv2d_fwd_f32_workspace_bytes(*shape, layout)
        assert 0 < ws <= SCRATCH, (shape, ws)
    for k, shape in enumerate((big, small)):
        say(f"noalloc {layout} {dist} call {k + 1} shape={shape}")
        x, w, st, pd = make(shape, 3100 + 10 * case + k, layout, dist=None if dist == "uniform" else "int")
        acc, mag = oracle.conv2d(x, w, st, pd, layout)
        y_na = _noalloc(x, w, shape, layout)
        y_pl = _plain(x, w, shape, layout)
        if dist == "int":
            exact = acc.astype(np.float32)
            assert np.array_equal(y_na, exact), f"{shape}: noalloc not bit-exact"
            assert np.array_equal(y_pl, exact), f"{shape}: conv2d_fwd_f32 not bit-exact"
        else:
            assert_parity(y_na, acc, mag, f"noalloc {shape} {layout}")
            assert_parity(y_pl, acc, mag, f"conv2d_fwd_f32 {shape} {layout}")


def test_noalloc_rejects_filter_copy_over_scratch():
    """A tap-major NCHW plan whose filter copy alone exceeds the scratch:
    MG3M_ERR_WORKSPACE, with nothing launched (the output keeps its NaNs)."""
    import torch
    lib = mg3m.load_library()
    N, C, H, W, K, R, S = 1, 1024, 3, 3, 4096, 3, 3      # filter 151 MB
    x = torch.zeros(N * C * H * W, dtype=torch.float32, device="cuda")
    w = torch.zeros(K * C * R * S, dtype=torch.float32, device="cuda")
    y = torch.full((N * K * H * W,), float("nan"), dtype=torch.float32, device="cuda")
    rc = lib.conv2d_fwd_f32_noalloc(x.data_ptr(), w.data_ptr(), y.data_ptr(), N, C, H, W, K, R, S, 1, 1,
                                    1, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 6, mg3m.mg3m_last_error()
    assert "workspace" in mg3m.mg3m_last_error()
    assert torch.isnan(y).all()

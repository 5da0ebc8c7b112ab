"""GPU parity of the tail schedule: the reduction steps of the tiles left
over after whole rounds of work-groups shared out in runs, either stream-K
(equal runs over all the tail's steps, crossing tile boundaries; one-tap HWCN
loader) or split (each tile cut into runs of nearly equal length; every
kernel), the pieces summed by the tail reduction in a fixed order.  Against
the fp64 oracle, bit-exact on small-integer data."""
import numpy as np
import pytest

import oracle
from paper_2307_04941_amd import mg3m
from tests.gpu_util import assert_parity, assert_parity_acc64, make, run_gpu, say, to_dev

pytestmark = pytest.mark.gpu

# Fewer tiles than one round (every tile is a tail tile): 256x64 tiles give
# 1 x 13 tiles of 36 k-tiles.
SK_SMALL = (4, 64, 14, 14, 256, 3, 3, 1, 1)
# More tiles than one round (whole rounds, then a tail of 525 tiles for 256x64).
SK_ROUNDS = (24, 16, 111, 111, 32, 3, 3, 1, 1)
# N = 3: the element-wise patch loader (one piece per tail work-group).
SK_SCALAR = (3, 20, 14, 14, 96, 3, 3, 1, 1)


def _tail(shape, layout, tile):
    info = mg3m.conv2d_fwd_f32_plan_info(*shape, layout, f"tile={tile},tail=2")
    return info["dp_tiles"], info["tail_tiles"], info["k_tiles"]


def _sk_counts(tail, k):
    """Work-group counts from one more than the tail tiles (runs nearly a
    tile long, every one crossing a boundary) to one per k-tile."""
    steps = tail * k
    return sorted({tail + 1, 2 * tail + 1, (5 * tail) // 2 + 3, max(tail + 1, steps // 7), steps})


SK_CASES = [(shape, tile, g) for shape in (SK_SMALL, SK_ROUNDS) for tile in ("256x64", "128x32") for g in range(5)]


@pytest.mark.parametrize("case", range(len(SK_CASES)))
def test_stream_k_runs(case):
    shape, tile, gi = SK_CASES[case]
    dp, tail, k = _tail(shape, "HWCN", tile)
    counts = _sk_counts(tail, k)
    g = counts[min(gi, len(counts) - 1)]
    plan = f"tile={tile},sk={g}"
    info = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", plan)
    say(f"stream-K {shape} {plan}: dp {info['dp_tiles']} tail {info['tail_tiles']} "
        f"wgs {info['tail_wgs']} k/wg {info['k_tiles_per_wg']}")
    assert (info["dp_tiles"], info["tail_tiles"], info["tail_wgs"]) == (dp, tail, g)
    x, w, st, pd = make(shape, 700 + case, "HWCN")
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    y = run_gpu(x, w, st, pd, "HWCN", plan=plan)
    assert_parity(y, acc, mag, f"{shape} {plan}")


# Split runs of unequal length (k-tiles not a multiple of the runs per tile)
# for every kind of kernel: one-tap HWCN, element-wise HWCN, NCHW.
SPLIT_CASES = [(shape, layout, plan + (",via=none" if layout == "NCHW" else ""))
               for shape, layout in ((SK_SMALL, "HWCN"), (SK_SCALAR, "HWCN"), (SK_SMALL, "NCHW"),
                                     (SK_ROUNDS, "NCHW"))
               for plan in ("tile=256x64,tail=5", "tile=128x32,tail=7", "tile=64x64,split=8")]


@pytest.mark.parametrize("case", range(len(SPLIT_CASES)))
def test_split_runs_uneven(case):
    shape, layout, plan = SPLIT_CASES[case]
    info = mg3m.conv2d_fwd_f32_plan_info(*shape, layout, plan)
    say(f"split {shape} {layout} {plan}: dp {info['dp_tiles']} tail {info['tail_tiles']} "
        f"wgs {info['tail_wgs']} k {info['k_tiles']} b_mode {info['b_mode']}")
    assert info["tail_tiles"] > 0 and info["tail_wgs"] == info["split"] * info["tail_tiles"]
    assert info["k_tiles"] % info["split"] != 0
    x, w, st, pd = make(shape, 730 + case, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=plan)
    assert_parity(y, acc, mag, f"{shape} {layout} {plan}")


def test_stream_k_bit_exact_and_deterministic():
    x, w, st, pd = make(SK_SMALL, 760, "HWCN", dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, "HWCN")
    _, tail, k = _tail(SK_SMALL, "HWCN", "256x64")
    for g in _sk_counts(tail, k):
        plan = f"tile=256x64,sk={g}"
        y1 = run_gpu(x, w, st, pd, "HWCN", plan=plan)
        assert np.array_equal(y1.astype(np.float64), acc), f"{plan}: not bit-exact"
    # random data: the same plan gives the same bits run to run
    x, w, st, pd = make(SK_SMALL, 761, "HWCN")
    plan = f"tile=256x64,sk={2 * tail + 1}"
    y1 = run_gpu(x, w, st, pd, "HWCN", plan=plan)
    y2 = run_gpu(x, w, st, pd, "HWCN", plan=plan)
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_split_runs_bit_exact(layout):
    x, w, st, pd = make(SK_SMALL, 762, layout, dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, layout)
    for plan in ("tile=256x64,tail=5", "tile=256x64,split=36", "tile=128x32,tail=7"):
        plan += ",via=none" if layout == "NCHW" else ""
        y = run_gpu(x, w, st, pd, layout, plan=plan)
        assert np.array_equal(y.astype(np.float64), acc), f"{plan}: not bit-exact"


@pytest.mark.parametrize("layout,plan", [("HWCN", "sk"), ("NCHW", "tile=256x64,tail=5,via=none"),
                                         ("NCHW", "tile=256x64,tail=5,via=hwcn")])
def test_tail_fused_add_relu(layout, plan):
    """The fused output stage is applied by the tail reduction (an NCHW call
    run as HWCN: by the layout change back to NCHW)."""
    import torch
    x, w, st, pd = make(SK_SMALL, 770, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    rng = np.random.Generator(np.random.PCG64(771))
    add = rng.standard_normal(acc.shape).astype(np.float32)
    N, C, H, W, K, R, S = mg3m.dims_of(x, w, layout)
    if plan == "sk":
        _, tail, _ = _tail(SK_SMALL, layout, "256x64")
        plan = f"tile=256x64,sk={2 * tail + 1}"
    wsb = mg3m.conv2d_fwd_f32_hw_workspace_bytes(N, C, H, W, K, R, S, 1, 1, 1, 1, layout, plan)
    ws = torch.empty((wsb + 3) // 4, dtype=torch.float32, device="cuda")
    y = torch.empty(acc.shape, dtype=torch.float32, device="cuda")
    mg3m.conv2d_fwd_f32_fused(to_dev(x), to_dev(w), y, to_dev(add), 1, N, C, H, W, K, R, S, 1, 1, 1, 1,
                              layout, ws, ws.numel() * 4, plan)
    ref = np.maximum(acc + add.astype(np.float64), 0.0)
    tol = 1e-5 * mag + 2.0 ** -23 * (np.abs(acc) + np.abs(add))
    assert np.all(np.abs(y.cpu().numpy() - ref) <= tol)


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("plan", ["tile=256x64,tail=5", "tile=64x32,split=7", "tile=256x64,sk=52"])
def test_split_runs_acc64(plan, layout):
    """fp64 pieces of uneven split runs added in fp64 and rounded once (sk=52:
    runs that fall on tile boundaries, taken as a split)."""
    x, w, st, pd = make(SK_SMALL, 780, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=plan, acc64=True)
    assert_parity_acc64(y, acc, mag, 9 * 64, f"{plan} {layout}")


# Plain calls whose selector plan shares tiles out: their partials come from
# the library's per-device pool, which keeps freed blocks for the next call.
POOL_SEQ = [SK_SMALL, (8, 256, 14, 14, 256, 3, 3, 1, 1), SK_SCALAR, (8, 256, 14, 14, 256, 3, 3, 1, 1)]


def test_workspace_pool_reuse_and_trim():
    for i, shape in enumerate(POOL_SEQ):
        info = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN")
        say(f"pool call {i}: {shape} tail_wgs {info['tail_wgs']} ws {info['workspace_bytes']}")
        assert info["tail_wgs"] > 0 and info["workspace_bytes"] > 0
        x, w, st, pd = make(shape, 780 + i, "HWCN")
        acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
        y = run_gpu(x, w, st, pd, "HWCN")          # plan None: conv2d_fwd_f32, own workspace
        assert_parity(y, acc, mag, f"pool call {i} {shape}")
        if i == 1:
            mg3m.mg3m_trim_workspace_pool()
    x, w, st, pd = make(SK_SMALL, 790, "HWCN")
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    Kg = SK_SMALL[1] * SK_SMALL[5] * SK_SMALL[6]
    assert_parity_acc64(run_gpu(x, w, st, pd, "HWCN", acc64=True), acc, mag, Kg, "acc64 after trim")
    mg3m.mg3m_trim_workspace_pool()


def _launch_plain(case, stream):
    """conv2d_fwd_f32 of one prepared case on `stream`, into a fresh output
    made on that stream."""
    import torch
    (N, C, H, W, K, R, S, st, pd), xd, wd = case[0], case[1], case[2]
    Ho, Wo = mg3m.conv2d_out_dims(H, W, R, S, st, pd)
    with torch.cuda.stream(stream):
        y = torch.full((Ho, Wo, K, N), float("nan"), dtype=torch.float32, device="cuda")
    mg3m.conv2d_fwd_f32(xd, wd, y, N, C, H, W, K, R, S, st, pd, "HWCN", stream=stream)
    return y


def _plain_cases(seed):
    shapes = [SK_SMALL, (8, 256, 14, 14, 256, 3, 3, 1, 1), SK_SMALL, SK_SCALAR]
    cases = []
    for i, shape in enumerate(shapes):
        info = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN")
        assert info["workspace_bytes"] > 0, info
        x, w, st, pd = make(shape, seed + i, "HWCN")
        acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
        cases.append((shape, to_dev(x), to_dev(w), acc, mag))
    return cases


def test_workspace_per_stream():
    """conv2d_fwd_f32 keeps one workspace per stream and reuses it: calls
    queued on two streams at once, each stream's buffer grown while earlier
    calls that use it are still queued, more streams than get a buffer of
    their own (those take a pool block per call), and new buffers after the
    trim call has given the old ones back."""
    import torch
    cases = _plain_cases(800)
    streams = [torch.cuda.Stream() for _ in range(2)]
    extra = [torch.cuda.Stream() for _ in range(34)]
    torch.cuda.synchronize()
    jobs = []
    for rep in range(2):
        for k, s in enumerate(streams):
            for i in range(len(cases)):
                c = cases[(i + k) % len(cases)]
                jobs.append((c, _launch_plain(c, s)))
    for j, s in enumerate(extra):
        c = cases[j % len(cases)]
        jobs.append((c, _launch_plain(c, s)))
    say(f"{len(jobs)} calls queued on {len(streams) + len(extra)} streams")
    torch.cuda.synchronize()
    for (shape, _, _, acc, mag), y in jobs:
        assert_parity(y.cpu().numpy(), acc, mag, f"{shape}")
    mg3m.mg3m_trim_workspace_pool()
    for c in cases[:2]:
        y = _launch_plain(c, streams[0])
        torch.cuda.synchronize()
        assert_parity(y.cpu().numpy(), c[3], c[4], f"after trim {c[0]}")


def test_workspace_under_graph_capture():
    """A captured conv2d_fwd_f32 takes its workspace from the pool inside the
    graph, not from the stream's buffer; every replay, with eager calls on
    the same stream between them, equals the eager result bit for bit."""
    import torch
    cases = _plain_cases(820)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    c = cases[1]
    (N, C, H, W, K, R, S, st, pd), xd, wd = c[0], c[1], c[2]
    y = _launch_plain(c, s)                    # the stream's buffer, sized for this shape
    torch.cuda.synchronize()
    assert_parity(y.cpu().numpy(), c[3], c[4], "eager")
    ref = y.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        mg3m.conv2d_fwd_f32(xd, wd, y, N, C, H, W, K, R, S, st, pd, "HWCN", stream=s)
    for rep in range(3):
        other = _launch_plain(cases[3], s)     # eager work on the stream's own buffer
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), f"replay {rep}"
        assert_parity(other.cpu().numpy(), cases[3][3], cases[3][4], f"eager call between replays {rep}")
    del g
    mg3m.mg3m_trim_workspace_pool()


def test_workspace_per_stream_from_host_threads():
    """Host threads calling conv2d_fwd_f32 at once, each on its own stream
    (and two of them sharing one): every result equals the oracle's."""
    import threading
    import torch
    cases = _plain_cases(840)
    streams = [torch.cuda.Stream() for _ in range(3)]
    torch.cuda.synchronize()
    results, errors = [], []

    def worker(k):
        try:
            s = streams[min(k, 2)]          # threads 2 and 3 share a stream
            for i in range(6):
                c = cases[(i + k) % len(cases)]
                results.append((c, _launch_plain(c, s)))
        except Exception as e:               # reported below, on the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    torch.cuda.synchronize()
    say(f"{len(results)} calls from 4 host threads")
    assert len(results) == 24
    for (shape, _, _, acc, mag), y in results:
        assert_parity(y.cpu().numpy(), acc, mag, f"{shape}")

"""pk_conv2d_fwd_noalloc (the convolution for callers that cannot allocate)
through the C-ABI against pk_conv2d_fwd given the workspace the library asks
for: two calls in a row, the second on a smaller input, then the first again
over the stale scratch; configurations that use the workspace (stream-K
partial tiles and arrival counters, split-K partial sums); outputs equal bit
for bit, and on integer data equal to the oracle."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import dev, host, require_gpu
from paper_1904_05347_amd import workloads as wl

pytestmark = pytest.mark.gpu

# (N, H, W, Cin, Cout): 3x3 stride 1, one pixel of padding on every side
BIG = (4, 56, 56, 256, 256)     # stream-K: about 64 MiB of partial tiles and counters
SMALL = (4, 28, 28, 256, 512)   # split-K: about 18 MiB of partial sums


def _geometry(shape):
    N, H, W, Cin, Cout = shape
    return N, H, W, Cin, 3, 3, Cout, 1, 1, 1, 1, 1, 1


def _inputs(shape, seed):
    N, H, W, Cin, Cout = shape
    rng = np.random.default_rng(seed)
    x = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.integers(rng, 9 * Cin * Cout).reshape(3, 3, Cin, Cout)
    return x, f


def _call(torch, pk, shape, dx, df, noalloc):
    N, H, W, Cin, KH, KW, Cout, sh, sw, pt, pl, pb, pr = _geometry(shape)
    y = torch.full((N, H, W, Cout), float("nan"), device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    if noalloc:
        st = pk.binding.conv2d_fwd_noalloc_raw(dx.data_ptr(), N, H, W, Cin, df.data_ptr(), KH, KW, Cout,
                                               sh, sw, pt, pl, pb, pr, y.data_ptr(), H, W, stream)
    else:
        need = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, sh, sw, pt, pl, pb, pr)
        assert need > 0
        ws = torch.empty(need // 4 + 1, dtype=torch.float32, device="cuda")
        st = pk.binding.conv2d_fwd_raw(dx.data_ptr(), N, H, W, Cin, df.data_ptr(), KH, KW, Cout,
                                       sh, sw, pt, pl, pb, pr, y.data_ptr(), H, W,
                                       ws.data_ptr(), need, stream)
    assert st == 0, (shape, noalloc, st, pk.last_invalid_param())
    return host(y), pk.last_config_name()


def test_noalloc_matches_workspace_entry_point():
    torch, pk = require_gpu()
    data = {}
    for shape, seed in ((BIG, 401), (SMALL, 402)):
        x, f = _inputs(shape, seed)
        ref, _ = oracle.conv2d(x, f, (1, 1), (1, 1, 1, 1))
        dx, df = dev(x), dev(f)
        want, cfg = _call(torch, pk, shape, dx, df, noalloc=False)
        assert np.array_equal(want.astype(np.float64), ref), (shape, cfg)
        data[shape] = (dx, df, want, cfg)
    names = {c["name"]: c for c in pk.configs()}
    assert names[data[BIG][3]]["streamk"] == 1, data[BIG][3]
    # BIG, then the smaller SMALL over BIG's scratch, then BIG again over SMALL's
    for shape in (BIG, SMALL, BIG):
        dx, df, want, cfg = data[shape]
        got, used = _call(torch, pk, shape, dx, df, noalloc=True)
        assert used == cfg, (shape, used, cfg)
        assert np.array_equal(got, want), (shape, cfg)


def test_noalloc_limits_and_quick_returns():
    torch, pk = require_gpu()
    # a forced split whose partial sums exceed the static scratch is refused
    # before any work is queued
    N, H, W, Cin, Cout = 32, 56, 56, 64, 64
    x = torch.zeros((N, H, W, Cin), device="cuda")
    f = torch.zeros((3, 3, Cin, Cout), device="cuda")
    y = torch.full((N, H, W, Cout), 3.0, device="cuda")
    pk.force_config("conv_64x64x32_w2x2_v44")
    pk.force_splits(8)
    try:
        st = pk.binding.conv2d_fwd_noalloc_raw(x.data_ptr(), N, H, W, Cin, f.data_ptr(), 3, 3, Cout,
                                               1, 1, 1, 1, 1, 1, y.data_ptr(), H, W, None)
    finally:
        pk.force_config(None)
        pk.force_splits(0)
    assert st == 5
    torch.cuda.synchronize()
    assert bool(torch.all(y == 3.0))
    # an empty batch does nothing; a bad argument keeps pk_conv2d_fwd's position
    st = pk.binding.conv2d_fwd_noalloc_raw(x.data_ptr(), 0, H, W, Cin, f.data_ptr(), 3, 3, Cout,
                                           1, 1, 1, 1, 1, 1, y.data_ptr(), H, W, None)
    assert st == 0
    st = pk.binding.conv2d_fwd_noalloc_raw(x.data_ptr(), N, H, W, Cin, f.data_ptr(), 3, 3, Cout,
                                           1, 1, 1, 1, 1, 1, y.data_ptr(), H + 1, W, None)
    assert st == 1 and pk.last_invalid_param() == 17

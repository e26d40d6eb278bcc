"""Winograd F(2x2, 3x3) and F(4x4, 3x3) convolution (Section 4.1.2: the
output-tile size is the parameter) on the GPU through the C-ABI.  The
reference is the convolution's definition (the direct-sum oracle); the
tolerance is 1e-5 times the oracle's Winograd error scale for that tile size
(the transform chain on absolute values), which bounds the rounding of the
transformed computation as sum |a*b| bounds the direct one.  For F(2x2, 3x3)
every intermediate is exact on small integers, so there the result must
equal the definition bit for bit; F(4x4, 3x3)'s filter transform has the
non-dyadic entries 1/6, 1/12, 1/24, so it is held to the bound there too."""
import numpy as np
import pytest

import oracle
from paper_1904_05347_amd import workloads as wl
from tests.gpu_util import assert_parity, dev, host, require_gpu, sample_conv_outputs

pytestmark = pytest.mark.gpu


TILES = (2, 4)


def _scale(tile, x, f, pads, idx=None):
    if idx is None:
        return oracle.winograd(tile, x, f, pads)[1]
    return oracle.winograd_at(tile, x, f, pads, idx)[1]


def _check_integers(tile, out, ref, scale, what):
    if tile == 2:
        assert np.array_equal(out.astype(np.float64), ref), what
    else:
        assert_parity(out, ref, scale, what)


def _run(pk, x, f, pads, force=None, out=None, tile=2):
    if force:
        pk.force_config(force)
    try:
        y = pk.conv2d_winograd(dev(x), dev(f), padding=pads, out=out, tile=tile)
    finally:
        if force:
            pk.force_config(None)
    return host(y), pk.last_config_name()


GEOMS = [
    # (N, H, W, Cin, Cout, pads): ragged 2x2 tiles, scalar and 16-byte channels
    (2, 9, 7, 8, 12, (1, 1, 1, 1)),
    (1, 6, 6, 4, 64, (0, 0, 0, 0)),
    (3, 5, 8, 3, 5, (1, 1, 1, 1)),      # Cin = 3, Cout = 5: 4-byte transforms and loads
    (1, 11, 4, 1, 1, (2, 0, 1, 2)),     # asymmetric padding, one channel
    (2, 7, 10, 64, 68, (0, 2, 2, 1)),
    (1, 3, 3, 16, 8, (0, 0, 0, 0)),     # a single output
    (2, 14, 14, 128, 96, (1, 1, 1, 1)),
]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("geom", GEOMS, ids=lambda g: "x".join(map(str, g[:5])) + "_p" + "".join(map(str, g[5])))
def test_winograd_small_geometries(geom, tile):
    torch, pk = require_gpu()
    N, H, W, Cin, Cout, pads = geom
    rng = np.random.default_rng(sum(geom[:5]) + 7)
    x = wl.uniform(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.uniform(rng, 9 * Cin * Cout).reshape(3, 3, Cin, Cout)
    Ho, Wo = oracle.conv2d_out_dims(H, W, 3, 3, 1, 1, *pads)
    y = torch.full((N, Ho, Wo, Cout), float("nan"), dtype=torch.float32, device="cuda")
    out, cfg = _run(pk, x, f, pads, out=y, tile=tile)
    ref, _ = oracle.conv2d(x, f, (1, 1), pads)
    assert out.shape == ref.shape
    assert_parity(out, ref, _scale(tile, x, f, pads), "F(%d) %s %s" % (tile, geom, cfg))
    xi = wl.integers(rng, x.size).reshape(x.shape)
    fi = wl.integers(rng, f.size).reshape(f.shape)
    out, cfg = _run(pk, xi, fi, pads, tile=tile)
    ref, _ = oracle.conv2d(xi, fi, (1, 1), pads)
    _check_integers(tile, out, ref, _scale(tile, xi, fi, pads), "F(%d) %s %s" % (tile, geom, cfg))


@pytest.mark.parametrize("tile", TILES)
def test_winograd_every_product_config_forced(tile):
    """Every non-persistent NN contraction instance runs the batched product."""
    torch, pk = require_gpu()
    rng = np.random.default_rng(71)
    x = wl.integers(rng, 2 * 9 * 11 * 8).reshape(2, 9, 11, 8)
    f = wl.integers(rng, 9 * 8 * 20).reshape(3, 3, 8, 20)
    ref, _ = oracle.conv2d(x, f, (1, 1), (1, 1, 1, 1))
    sc = _scale(tile, x, f, (1, 1, 1, 1))
    xs = wl.integers(rng, 1 * 7 * 6 * 3).reshape(1, 7, 6, 3)
    fs = wl.integers(rng, 9 * 3 * 5).reshape(3, 3, 3, 5)
    ref_s, _ = oracle.conv2d(xs, fs, (1, 1), (1, 1, 1, 1))
    sc_s = _scale(tile, xs, fs, (1, 1, 1, 1))
    ran = 0
    for cfg in pk.configs():
        if cfg["kind"] != 0 or cfg["trans_a"] or cfg["trans_b"] or cfg["persistent"] or cfg["streamk"] or cfg["bres"]:
            continue
        out, used = _run(pk, x, f, (1, 1, 1, 1), force=cfg["name"], tile=tile)
        assert used == cfg["name"]
        _check_integers(tile, out, ref, sc, cfg["name"])
        if cfg["vec_a"] == 1 and cfg["vec_b"] == 1:
            out, used = _run(pk, xs, fs, (1, 1, 1, 1), force=cfg["name"], tile=tile)
            _check_integers(tile, out, ref_s, sc_s, cfg["name"])
        ran += 1
    assert ran >= 10


def test_winograd_rejects_other_windows_and_workspace():
    torch, pk = require_gpu()
    from paper_1904_05347_amd import binding
    x = torch.zeros((1, 8, 8, 4), dtype=torch.float32, device="cuda")
    f5 = torch.zeros((5, 5, 4, 4), dtype=torch.float32, device="cuda")
    with pytest.raises(pk.PkError):
        pk.conv2d_winograd(x, f5, padding="SAME")
    f = torch.zeros((3, 3, 4, 4), dtype=torch.float32, device="cuda")
    y = torch.zeros((1, 8, 8, 4), dtype=torch.float32, device="cuda")
    need = pk.conv2d_winograd_workspace_bytes(1, 8, 8, 4, 4, 1, 1, 1, 1)
    ws = torch.zeros(need // 4, dtype=torch.float32, device="cuda")
    st = binding.conv2d_winograd_raw(x.data_ptr(), 1, 8, 8, 4, f.data_ptr(), 3, 3, 4, 1, 1, 1, 1, 1, 1,
                                     y.data_ptr(), 8, 8, ws.data_ptr(), need - 4)
    assert st == 3
    st = binding.conv2d_winograd_raw(x.data_ptr(), 1, 8, 8, 4, f.data_ptr(), 3, 3, 4, 2, 2, 1, 1, 1, 1,
                                     y.data_ptr(), 4, 4, ws.data_ptr(), need)
    assert st == 2
    # batch 0: nothing to do, nothing written
    x0 = torch.zeros((0, 8, 8, 4), dtype=torch.float32, device="cuda")
    assert tuple(pk.conv2d_winograd(x0, f).shape) == (0, 8, 8, 4)
    assert tuple(pk.conv2d_winograd(x0, f, tile=4).shape) == (0, 8, 8, 4)
    # the tile-size entry point: m is argument 19, the workspace 20
    need4 = pk.conv2d_winograd_workspace_bytes(1, 8, 8, 4, 4, 1, 1, 1, 1, 4)
    assert need4 > 0 and pk.conv2d_winograd_workspace_bytes(1, 8, 8, 4, 4, 1, 1, 1, 1, 3) == 0
    ws4 = torch.zeros(need4 // 4 + 4, dtype=torch.float32, device="cuda")
    st = binding.conv2d_winograd_tile_raw(x.data_ptr(), 1, 8, 8, 4, f.data_ptr(), 3, 3, 4, 1, 1, 1, 1, 1, 1,
                                          y.data_ptr(), 8, 8, 3, ws4.data_ptr(), need4)
    assert st == 1 and pk.last_invalid_param() == 19
    st = binding.conv2d_winograd_tile_raw(x.data_ptr(), 1, 8, 8, 4, f.data_ptr(), 3, 3, 4, 1, 1, 1, 1, 1, 1,
                                          y.data_ptr(), 8, 8, 4, ws4.data_ptr() + 4, need4)
    assert st == 1 and pk.last_invalid_param() == 20
    st = binding.conv2d_winograd_tile_raw(x.data_ptr(), 1, 8, 8, 4, f.data_ptr(), 3, 3, 4, 1, 1, 1, 1, 1, 1,
                                          y.data_ptr(), 8, 8, 4, ws4.data_ptr(), need4 - 4)
    assert st == 3


@pytest.mark.parametrize("tile", TILES)
def test_winograd_deterministic(tile):
    torch, pk = require_gpu()
    rng = np.random.default_rng(5)
    x = dev(wl.uniform(rng, 4 * 28 * 28 * 64).reshape(4, 28, 28, 64))
    f = dev(wl.uniform(rng, 9 * 64 * 128).reshape(3, 3, 64, 128))
    a = pk.conv2d_winograd(x, f, tile=tile)
    b = pk.conv2d_winograd(x, f, tile=tile)
    assert torch.equal(a, b)


WINO_LAYERS = [c for c in wl.STEP_CONVS if c.f_shape[0] == 3 and c.f_shape[1] == 3 and c.stride == (1, 1)
               and c.x_shape[3] >= 64]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("case", WINO_LAYERS, ids=[c.name for c in WINO_LAYERS])
def test_winograd_benchmark_layers_sampled(case, tile):
    """The 3x3 layers of the benchmark at batch 32 into a NaN-filled output:
    the corners of every m x m output tile of a band of tile rows at the top,
    middle and bottom of each image, and random outputs (every border class
    included), in the configuration the Winograd suite times."""
    torch, pk = require_gpu()
    x, f = case.inputs()
    N, H, W, Cin = case.x_shape
    Cout = case.f_shape[3]
    Ho, Wo = case.out_hw
    y = torch.full((N, Ho, Wo, Cout), float("nan"), dtype=torch.float32, device="cuda")
    out, cfg = _run(pk, x, f, case.pads, out=y, tile=tile)
    assert out.shape == (N, Ho, Wo, Cout)
    assert np.all(np.isfinite(out))
    rows = sorted({r for t in (0, (Ho // tile) // 2, (Ho - 1) // tile) for r in (t * tile, min(t * tile + tile, Ho) - 1)})
    cols = sorted({c for t in range(0, (Wo + tile - 1) // tile) for c in (t * tile, min(t * tile + tile, Wo) - 1)})
    n, h, w, c = np.meshgrid([0, N - 1], rows, cols, [0, Cout - 1], indexing="ij")
    idx = np.concatenate([(((n * Ho + h) * Wo + w) * Cout + c).reshape(-1),
                          sample_conv_outputs(N, Ho, Wo, Cout, 2500, case.seed)])
    ref, _ = oracle.conv2d_at(x, f, (1, 1), case.pads, idx)
    assert_parity(out.reshape(-1)[idx], ref, _scale(tile, x, f, case.pads, idx),
                  "F(%d) %s %s" % (tile, case.name, cfg))


SUITE = [(b, c) for b in (1, 4) for c in wl.layer_suite(b)
         if c.f_shape[0] == 3 and c.f_shape[1] == 3 and c.stride == (1, 1)]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("batch,case", SUITE, ids=[c.name for _, c in SUITE])
def test_winograd_paper_layers_batch_1_4(batch, case, tile):
    """Every 3x3 stride-1 layer of the paper's tables at batch 1 and 4."""
    torch, pk = require_gpu()
    x, f = case.inputs()
    N, H, W, Cin = case.x_shape
    Cout = case.f_shape[3]
    Ho, Wo = oracle.conv2d_out_dims(H, W, 3, 3, 1, 1, *case.pads)
    y = torch.full((N, Ho, Wo, Cout), float("nan"), dtype=torch.float32, device="cuda")
    out, cfg = _run(pk, x, f, case.pads, out=y, tile=tile)
    assert np.all(np.isfinite(out))
    idx = sample_conv_outputs(N, Ho, Wo, Cout, 1500, case.seed)
    ref, _ = oracle.conv2d_at(x, f, (1, 1), case.pads, idx)
    assert_parity(out.reshape(-1)[idx], ref, _scale(tile, x, f, case.pads, idx),
                  "F(%d) %s %s" % (tile, case.name, cfg))

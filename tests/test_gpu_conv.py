"""Convolution forward on the GPU through the C-ABI against the CPU oracle."""
import numpy as np
import pytest

import oracle
from paper_1904_05347_amd import workloads as wl
from tests.gpu_util import assert_parity, dev, host, require_gpu, sample_conv_outputs

pytestmark = pytest.mark.gpu


def _run(pk, x, f, stride, pads, workspace=None, force=None, splits=0):
    if force:
        pk.force_config(force)
    if splits:
        pk.force_splits(splits)
    try:
        y = pk.conv2d_fwd(dev(x), dev(f), stride=stride, padding=pads, workspace=workspace)
    finally:
        if force:
            pk.force_config(None)
        if splits:
            pk.force_splits(0)
    return host(y), pk.last_config_name()


def test_conv_b1_56x56x64_whole_output():
    torch, pk = require_gpu()
    case = wl.CONV_SMALL
    x, f = case.inputs()
    out, cfg = _run(pk, x, f, case.stride, case.pads)
    ref, scale = oracle.conv2d(x, f, case.stride, case.pads)
    assert out.shape == ref.shape == (1, 56, 56, 64)
    mx = assert_parity(out, ref, scale, case.name + " " + cfg)
    assert mx < 1e-6


def test_conv_b1_integer_exact():
    torch, pk = require_gpu()
    case = wl.CONV_SMALL
    x, f = case.inputs(kind="int")
    out, cfg = _run(pk, x, f, case.stride, case.pads)
    ref, _ = oracle.conv2d(x, f, case.stride, case.pads)
    assert np.array_equal(out.astype(np.float64), ref), cfg


SMALL_GEOMS = [
    # (N, H, W, Cin, KH, KW, Cout, stride, pads)
    (2, 9, 7, 8, 3, 3, 12, (1, 1), (1, 1, 1, 1)),
    (1, 13, 11, 4, 3, 3, 68, (2, 2), (0, 0, 1, 1)),
    (3, 8, 8, 3, 3, 3, 64, (1, 1), (1, 1, 1, 1)),       # Cin = 3: scalar gather
    (2, 10, 10, 3, 7, 7, 16, (2, 2), (3, 3, 3, 3)),     # 7x7 stride 2
    (1, 12, 9, 16, 1, 1, 20, (2, 2), (0, 0, 0, 0)),     # 1x1 stride 2: row gather
    (2, 7, 7, 36, 1, 1, 132, (1, 1), (0, 0, 0, 0)),     # 1x1 stride 1: plain GEMM
    (1, 6, 5, 5, 2, 3, 7, (1, 2), (1, 0, 0, 2)),        # odd everything: scalar B too
    (1, 5, 5, 12, 5, 5, 8, (1, 1), (0, 0, 0, 0)),       # window = image
]


@pytest.mark.parametrize("geom", SMALL_GEOMS, ids=lambda g: "x".join(map(str, g[:7])) + "_s%d%d" % g[7])
def test_conv_small_geometries(geom):
    torch, pk = require_gpu()
    N, H, W, Cin, KH, KW, Cout, stride, pads = geom
    rng = np.random.default_rng(sum(geom[:7]))
    x = wl.uniform(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.uniform(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
    out, cfg = _run(pk, x, f, stride, pads)
    ref, scale = oracle.conv2d(x, f, stride, pads)
    assert out.shape == ref.shape
    assert_parity(out, ref, scale, str(geom) + " " + cfg)
    xi = wl.integers(rng, x.size).reshape(x.shape)
    fi = wl.integers(rng, f.size).reshape(f.shape)
    out, cfg = _run(pk, xi, fi, stride, pads)
    ref, _ = oracle.conv2d(xi, fi, stride, pads)
    assert np.array_equal(out.astype(np.float64), ref), (geom, cfg)


def test_every_conv_config_forced():
    torch, pk = require_gpu()
    rng = np.random.default_rng(77)
    x = wl.integers(rng, 2 * 11 * 10 * 8).reshape(2, 11, 10, 8)
    f = wl.integers(rng, 3 * 3 * 8 * 20).reshape(3, 3, 8, 20)
    ref, _ = oracle.conv2d(x, f, (1, 1), (1, 1, 1, 1))
    # a window the direct kernel takes (KH*KW*Cin <= 32)
    xs = wl.integers(rng, 2 * 11 * 10 * 3).reshape(2, 11, 10, 3)
    fs = wl.integers(rng, 3 * 3 * 3 * 20).reshape(3, 3, 3, 20)
    ref_s, _ = oracle.conv2d(xs, fs, (1, 1), (1, 1, 1, 1))
    for cfg in pk.configs():
        if cfg["kind"] == 1:
            out, used = _run(pk, x, f, (1, 1), (1, 1, 1, 1), force=cfg["name"])
            assert used == cfg["name"]
            assert np.array_equal(out.astype(np.float64), ref), cfg["name"]
        if cfg["kind"] in (1, 2) and cfg["vec_a"] == 1:
            out, used = _run(pk, xs, fs, (1, 1), (1, 1, 1, 1), force=cfg["name"])
            assert used == cfg["name"]
            assert np.array_equal(out.astype(np.float64), ref_s), cfg["name"]


DIRECT_GEOMS = [
    # (N, H, W, Cin, KH, KW, Cout, stride, pads): ragged tiles, channel groups, strides
    (3, 13, 45, 3, 3, 3, 100, (1, 1), (1, 1, 1, 1)),
    (2, 17, 70, 3, 3, 3, 64, (2, 2), (0, 0, 1, 1)),
    (1, 9, 33, 1, 5, 5, 7, (1, 1), (2, 2, 2, 2)),
    (2, 8, 31, 4, 2, 4, 130, (2, 1), (1, 0, 0, 3)),
    (1, 40, 40, 2, 4, 4, 32, (3, 3), (0, 0, 0, 0)),
]


DIRECT_CONFIGS = ["direct_8x32x64_k32", "direct_8x32x64_k32_p"]


def _direct_patch_floats(KH, KW, Cin, stride):
    return (7 * stride[0] + KH) * (31 * stride[1] + KW) * Cin


@pytest.mark.parametrize("name", DIRECT_CONFIGS)
@pytest.mark.parametrize("geom", DIRECT_GEOMS, ids=lambda g: "x".join(map(str, g[:7])) + "_s%d%d" % g[7])
def test_direct_conv_geometries(geom, name):
    torch, pk = require_gpu()
    N, H, W, Cin, KH, KW, Cout, stride, pads = geom
    rng = np.random.default_rng(sum(geom[:7]) + 1)
    x = wl.uniform(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.uniform(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
    if name.endswith("_p") and _direct_patch_floats(KH, KW, Cin, stride) > 2048:
        # the persistent form stages at most 2048 patch floats: a forced call is refused
        with pytest.raises(pk.PkError):
            _run(pk, x, f, stride, pads, force=name)
        return
    out, cfg = _run(pk, x, f, stride, pads, force=name)
    assert cfg == name
    ref, scale = oracle.conv2d(x, f, stride, pads)
    assert out.shape == ref.shape
    assert_parity(out, ref, scale, str(geom) + " " + cfg)
    xi = wl.integers(rng, x.size).reshape(x.shape)
    fi = wl.integers(rng, f.size).reshape(f.shape)
    out, cfg = _run(pk, xi, fi, stride, pads, force=name)
    ref, _ = oracle.conv2d(xi, fi, stride, pads)
    assert np.array_equal(out.astype(np.float64), ref), (geom, cfg)


def test_direct_conv_default_choice():
    """The selector takes the persistent direct form where its patch fits and
    the one-tile-per-work-group form otherwise."""
    torch, pk = require_gpu()
    rng = np.random.default_rng(5)
    for geom, want in [((1, 9, 40, 3, 3, 3, 16, (1, 1), (1, 1, 1, 1)), "direct_8x32x64_k32_p"),
                       ((1, 40, 40, 2, 4, 4, 32, (3, 3), (0, 0, 0, 0)), "direct_8x32x64_k32")]:
        N, H, W, Cin, KH, KW, Cout, stride, pads = geom
        x = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
        f = wl.integers(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
        out, cfg = _run(pk, x, f, stride, pads)
        assert cfg == want, (geom, cfg)
        ref, _ = oracle.conv2d(x, f, stride, pads)
        assert np.array_equal(out.astype(np.float64), ref), (geom, cfg)


# Enough tiles that every resident work-group of the persistent direct form
# walks several, with channel-block changes inside a work-group's run (Cout =
# 130: three blocks of 64) and both patch sizes (4 and 8 floats per thread).
DIRECT_LOOP_GEOMS = [
    (32, 56, 56, 3, 3, 3, 130, (1, 1), (1, 1, 1, 1)),
    (96, 64, 70, 3, 3, 3, 64, (1, 2), (1, 1, 1, 1)),
    (8, 224, 224, 3, 3, 3, 64, (1, 1), (1, 1, 1, 1)),
]


@pytest.mark.parametrize("geom", DIRECT_LOOP_GEOMS, ids=lambda g: "x".join(map(str, g[:7])) + "_s%d%d" % g[7])
def test_direct_persistent_loops_over_tiles(geom):
    torch, pk = require_gpu()
    N, H, W, Cin, KH, KW, Cout, stride, pads = geom
    rng = np.random.default_rng(sum(geom[:7]) + 7)
    x = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.integers(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
    Ho, Wo = oracle.conv2d_out_dims(H, W, KH, KW, *stride, *pads)
    y = torch.full((N, Ho, Wo, Cout), float("nan"), dtype=torch.float32, device="cuda")
    pk.force_config("direct_8x32x64_k32_p")
    try:
        pk.conv2d_fwd(dev(x), dev(f), stride=stride, padding=pads, out=y)
        used = pk.last_config_name()
    finally:
        pk.force_config(None)
    assert used == "direct_8x32x64_k32_p"
    out = host(y)
    assert np.all(np.isfinite(out))
    idx = sample_conv_outputs(N, Ho, Wo, Cout, 6000, sum(geom[:7]))
    ref, _ = oracle.conv2d_at(x, f, stride, pads, idx)
    assert np.array_equal(out.reshape(-1)[idx].astype(np.float64), ref)


DMA_GEOMS = [
    # N, H, W, Cin, KH, KW, Cout, stride, pads (t, l, b, r)
    (2, 13, 9, 12, 3, 3, 36, (2, 2), (1, 0, 1, 1)),
    (3, 10, 10, 64, 1, 1, 68, (2, 2), (0, 0, 0, 0)),
    (1, 12, 11, 4, 5, 5, 8, (1, 1), (2, 2, 2, 2)),
    (2, 7, 7, 132, 3, 3, 260, (1, 1), (1, 1, 1, 1)),
]


@pytest.mark.parametrize("geom", DMA_GEOMS, ids=lambda g: "%dx%dx%dx%d_k%d_s%d" % (g[0], g[1], g[2], g[3], g[4], g[7][0]))
def test_conv_dma_geometries(geom):
    """The direct-to-LDS gather forms on windows beside the 3x3 stride-1 one:
    stride 2 with asymmetric padding, a strided 1x1, a 5x5, channel counts
    that are not multiples of the K-block, and a forced split of the
    reduction (stream-K forms: their own partition); integer data, so every
    output must equal the oracle bit for bit."""
    torch, pk = require_gpu()
    N, H, W, Cin, KH, KW, Cout, stride, pads = geom
    rng = np.random.default_rng(H * 31 + Cin)
    x = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.integers(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
    ref, _ = oracle.conv2d(x, f, stride, pads)
    Ho, Wo = ref.shape[1], ref.shape[2]
    ws = torch.empty(2 * N * Ho * Wo * Cout, dtype=torch.float32, device="cuda")
    ran = 0
    for cfg in pk.configs():
        if cfg["kind"] != 1 or not cfg["dma"]:
            continue
        # stream-K forms take no split; the binding sizes their workspace
        for splits in ((0,) if cfg["streamk"] else (0, 2)):
            out, used = _run(pk, x, f, stride, pads, workspace=ws if splits else None, force=cfg["name"],
                             splits=splits)
            assert used == cfg["name"]
            assert np.array_equal(out.astype(np.float64), ref), (cfg["name"], splits)
            ran += 1
    assert ran >= 8


@pytest.mark.parametrize("splits", [2, 3, 5])
def test_conv_split_k_forced(splits):
    torch, pk = require_gpu()
    rng = np.random.default_rng(splits)
    N, H, W, Cin, Cout = 1, 9, 9, 64, 96
    x = wl.uniform(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.uniform(rng, 9 * Cin * Cout).reshape(3, 3, Cin, Cout)
    ws = torch.empty(splits * N * H * W * Cout, dtype=torch.float32, device="cuda")
    outs = []
    for _ in range(2):
        out, cfg = _run(pk, x, f, (1, 1), (1, 1, 1, 1), workspace=ws, splits=splits)
        outs.append(out)
    assert np.array_equal(outs[0], outs[1]), "split-K must be deterministic"
    ref, scale = oracle.conv2d(x, f, (1, 1), (1, 1, 1, 1))
    assert_parity(outs[0], ref, scale, "split %d %s" % (splits, cfg))
    # too little workspace for a forced split is an error, not a silent fallback
    with pytest.raises(pk.PkError):
        _run(pk, x, f, (1, 1), (1, 1, 1, 1), workspace=ws[: N * H * W * Cout], splits=splits)


def test_conv_batch_zero_and_errors():
    torch, pk = require_gpu()
    x = torch.zeros((0, 5, 5, 4), dtype=torch.float32, device="cuda")
    f = torch.zeros((3, 3, 4, 4), dtype=torch.float32, device="cuda")
    y = pk.conv2d_fwd(x, f, padding="SAME")
    assert tuple(y.shape) == (0, 5, 5, 4)
    xx = torch.zeros((1, 5, 5, 4), dtype=torch.float32, device="cuda")
    yy = torch.zeros((1, 5, 5, 4), dtype=torch.float32, device="cuda")
    st = pk.binding.conv2d_fwd_raw(xx.data_ptr(), 1, 5, 5, 4, f.data_ptr(), 3, 3, 4, 1, 1, 1, 1, 1, 1,
                                   yy.data_ptr(), 4, 5)  # wrong Ho
    assert st == 1 and pk.last_invalid_param() == 17
    st = pk.binding.conv2d_fwd_raw(xx.data_ptr(), 1, 5, 5, 4, f.data_ptr(), 3, 3, 4, 1, 1, 1, 1, 1, 1,
                                   xx.data_ptr(), 5, 5)  # output aliases input
    assert st == 1 and pk.last_invalid_param() == 16


@pytest.mark.parametrize("splits", [1, 3])
def test_persistent_conv_configs_loop_over_tiles(splits):
    """Persistent convolution configurations with several tiles (and split-K
    items) per resident work-group; NaN-prefilled output, sampled bit-exact
    parity on integer data."""
    torch, pk = require_gpu()
    rng = np.random.default_rng(90 + splits)
    N, H, W, Cin, Cout = 16, 96, 96, 16, 68
    x = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
    f = wl.integers(rng, 9 * Cin * Cout).reshape(3, 3, Cin, Cout)
    dx, df = dev(x), dev(f)
    ws = torch.empty(splits * N * H * W * Cout, dtype=torch.float32, device="cuda")
    idx = sample_conv_outputs(N, H, W, Cout, 4000, splits)
    ref, _ = oracle.conv2d_at(x, f, (1, 1), (1, 1, 1, 1), idx)
    for cfg in pk.configs():
        if cfg["kind"] != 1 or not cfg["persistent"]:
            continue
        y = torch.full((N, H, W, Cout), float("nan"), dtype=torch.float32, device="cuda")
        pk.force_config(cfg["name"])
        pk.force_splits(splits)
        try:
            pk.conv2d_fwd(dx, df, padding=(1, 1, 1, 1), out=y, workspace=ws)
            used = pk.last_config_name()
        finally:
            pk.force_config(None)
            pk.force_splits(0)
        assert used == cfg["name"]
        out = host(y)
        assert np.all(np.isfinite(out)), cfg["name"]
        assert np.array_equal(out.reshape(-1)[idx].astype(np.float64), ref), cfg["name"]


# batch 1, 4 and 32 (the built-in table's shapes) and 2 and 12 (shapes the
# table does not hold: the selection rules' own configurations and splits)
SUITE = [(b, c) for b in (1, 2, 4, 12, 32) for c in wl.layer_suite(b)]


@pytest.mark.parametrize("batch,case", SUITE, ids=[c.name for _, c in SUITE])
def test_paper_layer_suite(batch, case):
    """Every distinct VGG-16 / ResNet-50 layer of the paper at batch 1, 2, 4,
    12 and 32, into a NaN-filled output: the whole output where the oracle is
    quick, else the corners of every output tile and sampled outputs (every
    border class included)."""
    from tests.test_gpu_fullsize import _conv_tile_corners
    torch, pk = require_gpu()
    x, f = case.inputs()
    N, H, W, Cin = case.x_shape
    KH, KW, _, Cout = case.f_shape
    Ho, Wo = oracle.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
    y = torch.full((N, Ho, Wo, Cout), float("nan"), device="cuda")
    pk.conv2d_fwd(dev(x), dev(f), stride=case.stride, padding=case.pads, out=y)
    cfg = pk.last_config_name()
    out = host(y)
    assert np.all(np.isfinite(out)), cfg
    macs = N * Ho * Wo * Cout * KH * KW * Cin
    if macs <= 4e8:
        ref, scale = oracle.conv2d(x, f, case.stride, case.pads)
        assert_parity(out, ref, scale, case.name + " " + cfg)
    else:
        info = {c["name"]: c for c in pk.configs()}[cfg]
        idx = np.concatenate([_conv_tile_corners(info, N, Ho, Wo, Cout),
                              sample_conv_outputs(N, Ho, Wo, Cout, 1000, case.seed)])
        ref, scale = oracle.conv2d_at(x, f, case.stride, case.pads, idx)
        assert_parity(out.reshape(-1)[idx], ref, scale, case.name + " " + cfg)


STREAMK_GEOMS = [
    # (N, H, W, Cin, KH, KW, Cout, stride, pads)
    (4, 24, 24, 64, 3, 3, 68, (1, 1), (1, 1, 1, 1)),   # many iterations per work-group, ragged Cout
    (1, 9, 11, 8, 3, 3, 20, (1, 1), (1, 1, 1, 1)),     # fewer iterations than resident work-groups
    (2, 14, 14, 64, 1, 1, 136, (1, 1), (0, 0, 0, 0)),  # 1x1 stride 1: the NN GEMM instances
    (2, 15, 13, 32, 1, 1, 40, (2, 2), (0, 0, 0, 0)),   # strided 1x1: row gather
]


def test_streamk_configs_partial_tiles():
    """Every stream-K configuration on problems whose (tile, K-block)
    iterations cut tiles between work-groups: NaN-prefilled output, whole
    output bit-exact against the oracle on integer data (a lost, doubled or
    misplaced partial sum shows), and a second call gives the same bits."""
    torch, pk = require_gpu()
    ran = 0
    for gi, (N, H, W, Cin, KH, KW, Cout, stride, pads) in enumerate(STREAMK_GEOMS):
        rng = np.random.default_rng(300 + gi)
        x = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
        f = wl.integers(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
        ref, _ = oracle.conv2d(x, f, stride, pads)
        dx, df = dev(x), dev(f)
        gemm_path = KH == 1 and KW == 1 and stride == (1, 1) and pads == (0, 0, 0, 0)
        for cfg in pk.configs():
            if not cfg["streamk"] or (cfg["kind"] == 0) != gemm_path:
                continue
            outs = []
            pk.force_config(cfg["name"])
            try:
                for _ in range(2):
                    y = torch.full(ref.shape, float("nan"), dtype=torch.float32, device="cuda")
                    pk.conv2d_fwd(dx, df, stride=stride, padding=pads, out=y)
                    assert pk.last_config_name() == cfg["name"]
                    outs.append(host(y))
            finally:
                pk.force_config(None)
            assert np.array_equal(outs[0].astype(np.float64), ref), (cfg["name"], gi)
            assert np.array_equal(outs[0], outs[1]), (cfg["name"], gi)
            ran += 1
    assert ran >= 8


def test_streamk_needs_workspace():
    """A forced stream-K configuration without room for its partial tiles
    reports PK_ERR_WORKSPACE; the selector's own choices fall back."""
    torch, pk = require_gpu()
    x = torch.ones((1, 8, 8, 16), dtype=torch.float32, device="cuda")
    f = torch.ones((3, 3, 16, 16), dtype=torch.float32, device="cuda")
    y = torch.empty((1, 8, 8, 16), dtype=torch.float32, device="cuda")
    name = next(c["name"] for c in pk.configs() if c["streamk"] and c["kind"] == 1)
    pk.force_config(name)
    try:
        st = pk.binding.conv2d_fwd_raw(x.data_ptr(), 1, 8, 8, 16, f.data_ptr(), 3, 3, 16, 1, 1, 1, 1, 1, 1,
                                       y.data_ptr(), 8, 8, None, 0)
    finally:
        pk.force_config(None)
    assert st == 3


TILED_GEOMS = [
    # (N, H, W, Cin, KH, KW, Cout, stride, pads)
    (2, 37, 45, 3, 7, 7, 64, (2, 2), (3, 3, 3, 3)),     # ResNet-50's first-layer window, ragged tiles
    (1, 30, 70, 3, 3, 3, 72, (1, 1), (1, 1, 1, 1)),     # VGG's first-layer window, ragged channel block
    (2, 19, 21, 16, 3, 3, 40, (1, 1), (1, 1, 1, 1)),    # Cin = 16: 4-wide channel loads, K = 144
    (1, 12, 9, 5, 5, 3, 7, (2, 1), (2, 0, 1, 2)),       # odd window, odd K, asymmetric padding
    (3, 8, 8, 4, 1, 1, 33, (2, 2), (0, 0, 0, 0)),       # 1x1 stride 2, K = 4
]


def test_tiled_direct_configs_every_instance():
    """Every tiled direct-convolution instance (output tile x channel widths
    of Section 4.1.1; one tile per work-group, and the persistent form with
    double-buffered patches, _tp) on windows up to 7x7 stride 2, ragged output tiles and
    channel blocks, odd reductions and asymmetric padding: integer data
    bit-exact against the oracle into a NaN-filled output, and uniform data
    within the bound.  An instance that cannot take a window (LDS, channel
    width) must say so with PK_ERR_NOT_SUPPORTED, never run."""
    torch, pk = require_gpu()
    tiled = [c for c in pk.configs() if c["kind"] == 2 and c["name"].endswith(("_v1", "_v4", "_tp"))]
    assert len(tiled) >= 30
    ran = 0
    for gi, (N, H, W, Cin, KH, KW, Cout, stride, pads) in enumerate(TILED_GEOMS):
        rng = np.random.default_rng(500 + gi)
        xi = wl.integers(rng, N * H * W * Cin).reshape(N, H, W, Cin)
        fi = wl.integers(rng, KH * KW * Cin * Cout).reshape(KH, KW, Cin, Cout)
        xu = wl.uniform(rng, xi.size).reshape(xi.shape)
        fu = wl.uniform(rng, fi.size).reshape(fi.shape)
        ref_i, _ = oracle.conv2d(xi, fi, stride, pads)
        ref_u, scale_u = oracle.conv2d(xu, fu, stride, pads)
        dxi, dfi, dxu, dfu = dev(xi), dev(fi), dev(xu), dev(fu)
        for cfg in tiled:
            if Cin % cfg["vec_a"]:
                continue
            pk.force_config(cfg["name"])
            try:
                y = torch.full(ref_i.shape, float("nan"), device="cuda")
                try:
                    pk.conv2d_fwd(dxi, dfi, stride=stride, padding=pads, out=y)
                except pk.PkError as e:
                    assert e.status == 2, (cfg["name"], gi, e)
                    continue
                assert pk.last_config_name() == cfg["name"]
                out = host(y)
                assert np.array_equal(out.astype(np.float64), ref_i), (cfg["name"], gi)
                yu = pk.conv2d_fwd(dxu, dfu, stride=stride, padding=pads)
                assert_parity(host(yu), ref_u, scale_u, "%s %d" % (cfg["name"], gi))
                ran += 1
            finally:
                pk.force_config(None)
    assert ran >= 70

"""The workload tables against the paper's layer tables (tests/golden) and the
oracle's own shape rules: the suite runs exactly the paper's layers."""
import oracle
from paper_1904_05347_amd import workloads as wl
from tests import pins


def test_layer_suite_matches_paper_tables():
    rows = {("vgg16", r["layer"]): r for r in pins.read_golden("vgg16_layers.csv")}
    rows.update({("resnet50", r["layer"]): r for r in pins.read_golden("resnet50_layers.csv")})
    cases = wl.layer_suite(1)
    assert len(cases) == len(rows) == 35
    for c in cases:
        net, name = c.name.split()[:2]
        r = rows[(net, name)]
        assert (c.H, c.W, c.Cin, c.KH, c.KW, c.stride, c.Cout) == (
            int(r["in_h"]), int(r["in_w"]), int(r["in_c"]), int(r["window"]), int(r["window"]),
            (int(r["stride"]),) * 2, int(r["out_c"])), c.name
        assert oracle.conv2d_out_dims(c.H, c.W, c.KH, c.KW, *c.stride, *c.pads) == (int(r["out_h"]), int(r["out_w"]))
        if c.KH != 7:  # "same" padding written out in the table equals the rule
            assert c.pads == oracle.same_pads(c.H, c.W, c.KH, c.KW, *c.stride), c.name


def test_step_layers_are_paper_layers():
    suite = {(c.H, c.Cin, c.KH, c.stride, c.Cout, c.pads) for c in wl.layer_suite(32)}
    for c in wl.STEP_CONVS:
        if c.name.startswith("resnet50 b32 56x56x256->128 1x1 s2"):
            continue  # the down-sampling branch reading (not a row of the paper's table)
        assert (c.H, c.Cin, c.KH, c.stride, c.Cout, c.pads) in suite, c.name


def test_gemm_sweep_is_the_papers():
    cases = wl.gemm_sweep()
    assert len(cases) == 125
    assert {c.M for c in cases} == {64, 128, 256, 512, 1024}

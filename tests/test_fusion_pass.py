"""The pass that picks which residual adds run inside a conv's epilogue
(host logic, no GPU): small graphs for each rule, and the chained networks."""
import workloads as W
from paper_2006_10226_amd.fusion import residual_fusions


def test_identity_shortcut():
    # block input read by the first conv and the add: the last conv takes it
    g = [("conv", ("x",), "a"), ("conv", ("a",), "b"), ("conv", ("b",), "c"), ("add", ("c", "x"), "y")]
    assert residual_fusions(g) == {3: (2, "x")}


def test_projection_shortcut_goes_to_the_later_conv():
    # both operands are conv outputs read only by the add: the conv that
    # runs later takes it, with the earlier one's output as residual
    g = [("conv", ("x",), "a"), ("conv", ("a",), "c"), ("conv", ("x",), "p"), ("add", ("c", "p"), "y")]
    assert residual_fusions(g) == {3: (2, "c")}


def test_residual_not_ready_when_the_conv_runs():
    # the residual is written after the conv: no fusion
    g = [("conv", ("x",), "c"), ("pool", ("x",), "r"), ("add", ("c", "r"), "y")]
    assert residual_fusions(g) == {}


def test_conv_output_read_elsewhere():
    g = [("conv", ("x",), "c"), ("pool", ("c",), "q"), ("add", ("c", "x"), "y")]
    assert residual_fusions(g) == {}


def test_only_convs_take_adds():
    g = [("dw", ("x",), "c"), ("add", ("c", "x"), "y"),
         ("conv_slice", ("y",), "cat"), ("add", ("cat", "y"), "z")]
    assert residual_fusions(g) == {}


def test_slices_and_rewritten_outputs():
    # the residual is a concat written by two steps, one of them after the conv
    g = [("conv_slice", ("x",), "cat"), ("conv", ("x",), "c"), ("conv_slice", ("x",), "cat"),
         ("add", ("c", "cat"), "y")]
    assert residual_fusions(g) == {}
    # the add's output name is written by another step too
    g = [("conv", ("x",), "c"), ("add", ("c", "x"), "y"), ("pool", ("x",), "y")]
    assert residual_fusions(g) == {}


def test_same_operand_twice_and_one_add_per_conv():
    g = [("conv", ("x",), "c"), ("add", ("c", "c"), "y")]
    assert residual_fusions(g) == {}
    # adds after the conv's only reader are not its to take
    g = [("conv", ("x",), "c"), ("add", ("c", "x"), "y"), ("add", ("y", "x"), "z")]
    assert residual_fusions(g) == {1: (0, "x")}


def test_chained_networks():
    for chain, adds in ((W.resnet50_chain(1), 16), (W.mobilenet_v2_chain(1), 10),
                        (W.inception_v3_mixed5_chain(1), 0)):
        g = chain.graph()
        f = residual_fusions(g)
        assert sum(1 for k, _, _ in g if k == "add") == adds
        assert len(f) == adds   # every residual add of these bodies has a conv to run in
        for i, (c, r) in f.items():
            kind, ins, out = g[c]
            assert kind == "conv" and c < i and set(g[i][1]) == {out, r}

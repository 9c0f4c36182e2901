"""Pins for the MobileNetV2 pointwise workload's layer table.

The paper's appendix table of lightweight-architecture benchmarks prints
the weight and multiply-accumulate counts of MobileNetV2 with CCI sparsity
(G = 8, s kept weights per group) on its pointwise layers.  The layer table
that the workload is built from must reproduce them; the dense network must
reproduce the published MobileNetV2 counts."""
import os

import pytest

from paper_1910_11971_amd import workloads as wl

HERE = os.path.dirname(os.path.abspath(__file__))


def printed_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "tab_lightweight_mobilenetv2.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                label, G, s, p, m = line.split()
                rows.append((label, int(G), int(s), p, m))
    return rows


def ulp(printed: str) -> float:
    """One unit in the last printed place ("2.19" -> 0.01, "120" -> 1)."""
    return 10.0 ** -len(printed.split(".")[1]) if "." in printed else 1.0


def cci_counts(G, s, cci_layers, layers):
    """Weights and MACs of the network once the CCI layers keep s of every G."""
    w = sum(l.weights for l in layers) - sum(l.weights for l in cci_layers) * (G - s) / G
    m = sum(l.macs for l in layers) - sum(l.macs for l in cci_layers) * (G - s) / G
    return w, m


def test_dense_network_matches_published_counts():
    L = wl.mobilenetv2_layers()
    assert len(L) == 53 and sum(l.kind == "depthwise" for l in L) == 17
    assert L[-2].H == 7 and L[-2].Ho == 7
    w = sum(l.weights for l in L)
    # + batch-norm scale and shift per channel: torchvision's 3 504 872
    assert w + 2 * sum(l.Cout for l in L if l.kind != "fc") == 3_504_872
    assert sum(l.macs for l in L) == 300_774_272


@pytest.mark.parametrize("row", printed_rows(), ids=lambda r: r[0])
def test_counts_match_the_paper_table(row):
    label, G, s, p, m = row
    L = wl.mobilenetv2_layers()
    if G == 0:
        w, macs = sum(l.weights for l in L), sum(l.macs for l in L)
    else:
        w, macs = cci_counts(G, s, wl.mobilenetv2_cci_layers(), L)
    assert abs(w / 1e6 - float(p)) <= ulp(p), (label, w)
    assert abs(macs / 1e6 - float(m)) <= ulp(m), (label, macs)


def test_other_readings_of_the_sparse_layer_set_do_not_match():
    """Sparsifying the 1280-channel conv too, or block 1's projection, misses
    the printed counts (so the table fixes the layer set)."""
    L = wl.mobilenetv2_layers()
    cci = wl.mobilenetv2_cci_layers()
    with_last = cci + [l for l in L if l.kind == "last"]
    with_first = cci + [l for l in L if l.name == "b1.0.project"]
    w, _ = cci_counts(8, 2, with_last, L)
    assert abs(w / 1e6 - 2.19) > 0.2
    _, m = cci_counts(8, 1, with_first, L)
    assert abs(m / 1e6 - 90) > 5


def test_pointwise_workloads():
    P = wl.mobilenetv2_pointwise(B=64, K=3)
    cci = wl.mobilenetv2_cci_layers()
    assert len(P) == len(cci) == 32
    for w, l in zip(P, cci):
        assert (w.Cin, w.O, w.H, w.KH, w.G, w.K) == (l.Cin, l.Cout, l.H, 1, 8, 3)
        assert w.N == 64 * l.H * l.H and w.C == l.Cin
        assert w.x_dist == ("relu_normal" if l.kind == "project" else "normal")
    assert len({w.seed for w in P}) == 32
    assert sum(w.N * w.C * w.O for w in P) == 64 * sum(l.macs for l in cci)
    # channel counts of the width multipliers round to multiples of 8
    assert [wl.round_channels(c * 1.4) for c in (32, 16, 24, 320)] == [48, 24, 32, 448]

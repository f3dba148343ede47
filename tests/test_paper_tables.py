"""The paper's VGG variant shapes against Table 1 (tests/golden/table1_params.txt)."""
import os

from paper_2112_15317_amd import configs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_params.txt")


def _golden():
    rows, pct = [], {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        a, b, c = line.split()
        if a == "PCT":
            pct[b] = float(c)
        else:
            rows.append((a, b, int(c)))
    return rows, pct


def test_variant_layer_shapes_reproduce_table1_counts():
    rows, pct = _golden()
    convs = configs.conv_layers(configs.PAPER_VARIANT_CONV, 3, 32)
    got = [(f"Conv{L.index}", f"{L.c}x{L.k}", L.k * L.c * 9) for L in convs]
    got += [(f"FC{j}", f"{i}x{o}", i * o) for j, (i, o) in enumerate(configs.PAPER_VARIANT_FC)]
    assert got == rows
    # FC0's 4096 inputs are the flattened 256 x 4 x 4 output of the last pool.
    last = convs[-1]
    assert last.pool_after and last.k * (last.h // 2) * (last.w // 2) == 4096
    conv_p = sum(L.k * L.c * 9 + L.k for L in convs)
    fc_p = sum(i * o + o for i, o in configs.PAPER_VARIANT_FC)
    assert round(100 * conv_p / (conv_p + fc_p), 2) == pct["conv"]
    assert round(100 * fc_p / (conv_p + fc_p), 2) == pct["fc"]

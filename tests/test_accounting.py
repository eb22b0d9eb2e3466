"""The traffic and parameter accounting reproduce the numbers the paper prints
(tests/golden/paper_printed_values.txt, each group with its citation)."""

import os

import pytest

from paper_2607_14530_amd import accounting as A
from paper_2607_14530_amd import synth


def _golden():
    path = os.path.join(os.path.dirname(__file__), "golden", "paper_printed_values.txt")
    vals = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                key, val = (x.strip() for x in line.split("="))
                vals[key] = float(val)
    return vals


G = _golden()


def test_table4_mhc_totals():
    r, w = A.paper_table4_mhc(4)
    assert (r, w) == (G["mhc_n4_read"], G["mhc_n4_write"])
    assert r + w == G["mhc_n4_total"]
    assert sum(A.paper_table4_mhc(16)) == G["mhc_n16_total"]


def test_table4_xhc_totals():
    r, w = A.paper_table4_xhc(16, 4)
    assert (r, w) == (G["xhc_read"], G["xhc_write"])
    assert r + w == G["xhc_total"]


def test_table4_flash_totals():
    r, w = A.paper_table4_flash(16, 4, Q=2)
    assert (r, w) == (G["flash_q2_read"], G["flash_q2_write"])
    assert r + w == G["flash_q2_total"]
    r4, w4 = A.paper_table4_flash(16, 4, Q=4)
    assert r4 == G["flash_q4_read"]
    # the printed write column is 13.5C; the per-operation sum gives 13.25C
    assert abs((r4 + w4) - G["flash_q4_total"]) <= 0.25


@pytest.mark.parametrize("N,k,key", [(16, 4, "xhc_params_n16_k4"), (4, 2, "xhc_params_n4_k2")])
def test_xhc_param_count(N, k, key):
    assert A.param_count_xhc_layer(N, k, 4, (4, 8, 12), 1) == G[key]


@pytest.mark.parametrize("N,key", [(4, "mhc_params_n4"), (16, "mhc_params_n16")])
def test_mhc_param_count(N, key):
    assert A.param_count_mhc_layer(N, 1) == G[key]


@pytest.mark.parametrize("C", [2112, 2560])
def test_param_counts_at_model_widths(C):
    """Table "Parameter and training FLOPs overhead": P/layer at the 18B and 28B widths."""
    assert A.param_count_xhc_layer(16, 4, 4, (4, 8, 12), C) == pytest.approx(G[f"params_c{C}_xhc"], rel=5e-3)
    assert A.param_count_mhc_layer(4, C) == pytest.approx(G[f"params_c{C}_mhc4"], rel=5e-3)
    assert A.param_count_mhc_layer(16, C) == pytest.approx(G[f"params_c{C}_mhc16"], rel=5e-3)


def test_param_count_matches_generated_weight_shapes():
    """The weights the library consumes have exactly the counted sizes."""
    C = 64
    n = 0
    for Kr in (1, 4):
        w = synth.Workload(T=2, N=16, k=4, m=2, C=C, Kr=Kr)
        d = synth.sublayer_inputs(w, 0)
        n += sum(d[x].numel() for x in ("W_r", "W_pre", "W_res", "W_post"))
        n += d["conv_w"].numel() if d["conv_w"] is not None else 0
    assert n == 1256 * C


def test_algorithmic_bytes_sum_to_26C_for_xhc():
    C = 4096
    unit = 2 * C
    b = A.algorithmic_bytes_sublayer(16, 4, C, 1)
    coef = 4 * (A.coef_floats(16, 4, 1) + 4 + 4 + 16 + 4)
    assert b - coef == 26 * unit

"""The traffic and parameter accounting reproduce the numbers the paper prints."""

import pytest

from paper_2607_14530_amd import accounting as A
from paper_2607_14530_amd import synth


def test_table4_mhc_totals():
    r, w = A.paper_table4_mhc(4)
    assert (r, w) == (21, 13)          # 21C R + 13C W = 34C
    assert sum(A.paper_table4_mhc(16)) == 130


def test_table4_xhc_totals():
    r, w = A.paper_table4_xhc(16, 4)
    assert (r, w) == (55, 18.5)        # 73.5C


def test_table4_flash_totals():
    r, w = A.paper_table4_flash(16, 4, Q=2)
    assert (r, w) == (36, 15)          # 51C
    r4, w4 = A.paper_table4_flash(16, 4, Q=4)
    assert r4 == 26.5
    # the printed write column is 13.5C; the per-operation sum gives 13.25C
    assert abs((r4 + w4) - 40) <= 0.25


@pytest.mark.parametrize("N,k,expect", [(16, 4, 1256), (4, 2, 124)])
def test_xhc_param_count(N, k, expect):
    assert A.param_count_xhc_layer(N, k, 4, (4, 8, 12), 1) == expect


@pytest.mark.parametrize("N,expect", [(4, 192), (16, 9216)])
def test_mhc_param_count(N, expect):
    assert A.param_count_mhc_layer(N, 1) == expect


@pytest.mark.parametrize("C,xhc,mhc4,mhc16", [(2112, 2.65e6, 405e3, 19.5e6), (2560, 3.22e6, 492e3, 23.6e6)])
def test_param_counts_at_model_widths(C, xhc, mhc4, mhc16):
    """Table "Parameter and training FLOPs overhead": P/layer at 18B and 28B widths."""
    assert A.param_count_xhc_layer(16, 4, 4, (4, 8, 12), C) == pytest.approx(xhc, rel=5e-3)
    assert A.param_count_mhc_layer(4, C) == pytest.approx(mhc4, rel=5e-3)
    assert A.param_count_mhc_layer(16, C) == pytest.approx(mhc16, rel=5e-3)


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

"""Central finite differences pin the oracle's backward (reverse mode of the forward)."""

import pytest
import torch

from oracle import xhc_oracle as O
from paper_2607_14530_amd import synth

F64 = torch.float64


def _setup(N, Kr, stress, seed, router="sigmoid"):
    w = synth.Workload(T=8, S=8, N=N, k=4, m=2, C=32, Kr=Kr,
                       alpha=(0.5, 1.0, 0.5) if stress else (0.01, 0.01, 0.01), router=router)
    d = synth.sublayer_inputs(w, seed, grads=True, bias_std=2.0 if stress else 0.0)
    vals = {
        "X": d["X"].to(F64), "F": d["F"].to(F64),
        "conv_w": d["conv_w"].to(F64) if d["conv_w"] is not None else None,
        "W_r": O.bf16_operand(d["W_r"]), "W_pre": O.bf16_operand(d["W_pre"]),
        "W_res": O.bf16_operand(d["W_res"]), "W_post": O.bf16_operand(d["W_post"]),
        "alpha": d["alpha"].to(F64), "b_pre": d["b_pre"].to(F64),
        "b_res": d["b_res"].to(F64), "b_post": d["b_post"].to(F64),
    }
    return w, d, vals


def _objective(w, d, vals):
    return O.sublayer_objective(
        vals["X"], vals["F"], vals["conv_w"], vals["W_r"], vals["W_pre"], vals["W_res"],
        vals["W_post"], vals["alpha"], vals["b_pre"], vals["b_res"], vals["b_post"],
        d["G_X"], d["G_in"], m=w.m, k=w.k, Kr=w.Kr, S=w.S, router=w.router)


@pytest.mark.parametrize("N,Kr,stress,seed,router", [(4, 4, False, 0, "sigmoid"), (8, 4, False, 1, "sigmoid"),
                                                      (8, 1, False, 2, "sigmoid"), (8, 4, True, 3, "sigmoid"),
                                                      (8, 4, True, 4, "softmax")])
def test_backward_matches_central_differences(N, Kr, stress, seed, router):
    w, d, vals = _setup(N, Kr, stress, seed, router)
    g = O.xhc_sublayer_grads(d["X"], d["F"], d["conv_w"], d["W_r"], d["W_pre"], d["W_res"],
                             d["W_post"], d["alpha"], d["b_pre"], d["b_res"], d["b_post"],
                             d["G_X"], d["G_in"], m=w.m, k=w.k, Kr=w.Kr, S=w.S, router=w.router)
    gen = torch.Generator().manual_seed(100 + seed)
    for name in O.GRAD_NAMES:
        if vals[name] is None:
            continue
        base = vals[name]
        direction = torch.randn(base.shape, generator=gen, dtype=F64)
        h = 1e-6 * max(1.0, base.abs().max().item())
        plus = dict(vals, **{name: base + h * direction})
        minus = dict(vals, **{name: base - h * direction})
        Lp, fp = _objective(w, d, plus)
        Lm, fm = _objective(w, d, minus)
        # the piecewise-constant routing decision must not flip inside the probe
        assert torch.equal(fp["idx"], fm["idx"]), name
        fd = ((Lp - Lm) / (2 * h)).item()
        an = (g[name] * direction).sum().item()
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, fd, an)


def test_backward_routes_gradient_only_through_selected_logits():
    """W_r receives gradient only via p of routed slots: with m = k there is none."""
    w = synth.Workload(T=8, S=8, N=6, k=4, m=4, C=16, Kr=1)
    d = synth.sublayer_inputs(w, 9, grads=True)
    g = O.xhc_sublayer_grads(d["X"], d["F"], None, d["W_r"], d["W_pre"], d["W_res"],
                             d["W_post"], d["alpha"], d["b_pre"], d["b_res"], d["b_post"],
                             d["G_X"], d["G_in"], m=w.m, k=w.k, Kr=w.Kr, S=w.S)
    assert torch.equal(g["W_r"], torch.zeros_like(g["W_r"]))


def test_stress_case_exercises_the_row_clamp():
    """The stressed finite-difference case must actually take the clamp branch."""
    w, d, vals = _setup(8, 4, True, 3)
    _, f = _objective(w, d, vals)
    a_n = O.rms_norm(O.gather_rows(vals["X"], f["idx"]).reshape(w.T, -1), 1e-5)
    logits = vals["alpha"][1] * (a_n @ vals["W_res"]) + vals["b_res"]
    raw = O.sinkhorn(torch.exp(logits).reshape(w.T, w.k, w.k), 20)
    assert (raw.sum(-1) > 1 + 1e-6).any()


def _stack_layers(N, C, seed):
    """Two chained sublayers (attention-type, then MLP-type) with a smooth
    stand-in for the sublayer function: out = tanh(input @ W_l)."""
    layers = []
    for l, Kr in enumerate((1, 4)):
        w = synth.Workload(T=8, S=8, N=N, k=4, m=2, C=C, Kr=Kr, alpha=(0.5, 1.0, 0.5))
        d = synth.sublayer_inputs(w, seed + l, grads=True)
        gen = torch.Generator().manual_seed(seed + 10 + l)
        Wl = torch.randn(C, C, generator=gen, dtype=F64) / C ** 0.5
        lay = {"fn": (lambda Wl: (lambda inp: torch.tanh(inp @ Wl)))(Wl), "m": w.m, "k": w.k, "Kr": Kr,
               "conv_w": d["conv_w"].to(F64) if d["conv_w"] is not None else None,
               "W_r": O.bf16_operand(d["W_r"]), "W_pre": O.bf16_operand(d["W_pre"]),
               "W_res": O.bf16_operand(d["W_res"]), "W_post": O.bf16_operand(d["W_post"]),
               "alpha": d["alpha"].to(F64), "b_pre": d["b_pre"].to(F64), "b_res": d["b_res"].to(F64),
               "b_post": d["b_post"].to(F64)}
        layers.append(lay)
        if l == 0:
            X0 = d["X"].to(F64)
    return X0, layers


def test_stack_backward_matches_central_differences():
    """Two sublayers chained on one state plus the final stream reduction:
    the oracle's gradients (entry state, every weight of both layers) against
    central differences of the chained objective."""
    N, C = 8, 32
    X0, layers = _stack_layers(N, C, 20)
    G = torch.randn(8, C, generator=torch.Generator().manual_seed(21), dtype=F64)
    dX0, per, _, _ = O.stack_grads(X0, layers, G, S=8, round_state=False)
    gen = torch.Generator().manual_seed(22)

    def L_of(X0v, lays):
        L, f, _ = O.stack_objective(X0v, lays, G, S=8, round_state=False)
        return L.item(), [x["idx"] for x in f]

    probes = [("X0", None)] + [(n, l) for l in range(2) for n in O.STACK_WEIGHTS if layers[l][n] is not None]
    for name, l in probes:
        base = X0 if l is None else layers[l][name]
        direction = torch.randn(base.shape, generator=gen, dtype=F64)
        h = 1e-6 * max(1.0, base.abs().max().item())

        def shifted(sign):
            if l is None:
                return X0 + sign * h * direction, layers
            lays = [dict(q) for q in layers]
            lays[l][name] = base + sign * h * direction
            return X0, lays
        Lp, ip = L_of(*shifted(1))
        Lm, im = L_of(*shifted(-1))
        assert all(torch.equal(a, b) for a, b in zip(ip, im)), (name, l)
        fd = (Lp - Lm) / (2 * h)
        g = dX0 if l is None else per[l][name]
        an = (g * direction).sum().item()
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, l, fd, an)


def test_single_layer_stack_is_the_sublayer_objective():
    """With one layer, <G, sum_i X'_i> = <G broadcast over the streams, X'>:
    the stack objective equals the sublayer objective with that G_X, G_in = 0
    and the layer's output as F."""
    X0, layers = _stack_layers(8, 32, 30)
    lay = layers[1]
    G = torch.randn(8, 32, generator=torch.Generator().manual_seed(31), dtype=F64)
    L1, f1, _ = O.stack_objective(X0, [lay], G, S=8, round_state=False)
    F = lay["fn"](f1[0]["input"])
    L2, _ = O.sublayer_objective(X0, F, lay["conv_w"], lay["W_r"], lay["W_pre"], lay["W_res"], lay["W_post"],
                                 lay["alpha"], lay["b_pre"], lay["b_res"], lay["b_post"],
                                 G[:, None, :].expand(8, 8, 32), torch.zeros(8, 32, dtype=F64),
                                 m=lay["m"], k=lay["k"], Kr=lay["Kr"], S=8)
    assert abs(L1.item() - L2.item()) <= 1e-12 * max(1.0, abs(L2.item()))

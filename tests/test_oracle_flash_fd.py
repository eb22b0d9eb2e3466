"""Central finite differences pin the oracle's xHC-Flash backward (reverse
mode of the sharing-group forward: one routing and Q pre-maps from the entry
state, Q write-backs on the active rows, H^res before the last)."""

import pytest
import torch

from oracle import xhc_oracle as O
from paper_2607_14530_amd import synth

F64 = torch.float64


def _setup(Q, N, stress, seed, router="sigmoid", attn_aug=0):
    w = synth.Workload(T=8, S=8, N=N, k=4, m=2, C=32, Kr=4,
                       alpha=(0.5, 1.0, 0.5) if stress else (0.01, 0.01, 0.01), router=router, attn_aug=attn_aug)
    d = synth.flash_inputs(w, Q, seed, grads=True, bias_std=2.0 if stress else 0.0)
    vals = O.flash_leaves(d["X"], d["F_list"], d["conv_w_list"], d["W_r"], d["W_pre_list"], d["W_post_list"],
                          d["W_res"], d["alpha_pre"], d["b_pre"], d["alpha_post"], d["b_post"], d["alpha_res"],
                          d["b_res"])
    kw = dict(m=w.m, k=w.k, S=w.S, round_state=False, router=router)
    return w, d, vals, kw


def _probes(vals):
    for name in O.FLASH_GRAD_NAMES:
        v = vals[name]
        if isinstance(v, list):
            for i, t in enumerate(v):
                if t is not None:
                    yield name, i
        else:
            yield name, None


@pytest.mark.parametrize("Q,N,stress,seed,router,attn_aug", [(2, 8, False, 0, "sigmoid", 0),
                                                              (4, 8, False, 1, "sigmoid", 0),
                                                              (2, 4, False, 2, "sigmoid", 0),
                                                              (4, 8, True, 3, "sigmoid", 0),
                                                              (2, 8, True, 4, "softmax", 0),
                                                              (4, 8, False, 5, "sigmoid", 1)])
def test_flash_backward_matches_central_differences(Q, N, stress, seed, router, attn_aug):
    w, d, vals, kw = _setup(Q, N, stress, seed, router, attn_aug)
    if attn_aug:   # the attention-side augmentation: every sublayer has K_r components
        assert all(c is not None for c in d["conv_w_list"])
    g, fwd, _ = O.flash_group_grads(vals, d["G_X"], d["G_in_list"], **kw)
    gen = torch.Generator().manual_seed(200 + seed)
    for name, i in _probes(vals):
        base = vals[name] if i is None else vals[name][i]
        direction = torch.randn(base.shape, generator=gen, dtype=F64)
        h = 1e-6 * max(1.0, base.abs().max().item())

        def at(sign):
            v = dict(vals)
            if i is None:
                v[name] = base + sign * h * direction
            else:
                v[name] = list(vals[name])
                v[name][i] = base + sign * h * direction
            return O.flash_objective(v, d["G_X"], d["G_in_list"], **kw)
        Lp, fp = at(1)
        Lm, fm = at(-1)
        assert torch.equal(fp["idx"], fm["idx"]), (name, i)   # the routing must not flip inside the probe
        fd = ((Lp - Lm) / (2 * h)).item()
        gr = g[name] if i is None else g[name][i]
        an = (gr * direction).sum().item()
        assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, i, fd, an)


def test_flash_forward_is_the_group_forward():
    """The differentiable forward and xhc_flash_group give the same state and
    inputs (both round the written rows to bf16)."""
    w, d, vals, _ = _setup(4, 8, True, 7)
    ref = O.xhc_flash_group(d["X"].to(F64), d["F_list"], d["W_r"], d["W_pre_list"], d["W_post_list"], d["W_res"],
                            d["conv_w_list"], d["alpha_pre"], d["b_pre"], d["alpha_post"], d["b_post"],
                            d["alpha_res"], d["b_res"], m=w.m, k=w.k, S=w.S)
    Xn, inputs, f = O.flash_forward(vals["X"], vals["F_list"], vals["conv_w_list"], vals["W_r"], vals["W_pre_list"],
                                    vals["W_post_list"], vals["W_res"], vals["alpha_pre"], vals["b_pre"],
                                    vals["alpha_post"], vals["b_post"], vals["alpha_res"], vals["b_res"],
                                    m=w.m, k=w.k, S=w.S)
    assert torch.equal(Xn, ref["X"])
    for a, b in zip(inputs, ref["inputs"]):
        assert torch.equal(a, b)
    assert torch.equal(f["idx"], ref["idx"])


def test_flash_untouched_rows_pass_the_state_gradient_through_plus_base_readouts():
    """A non-active stream i enters the group only through the pre-maps and
    the base readouts, so with the pre-map and router weights zeroed its
    gradient is G_X[i] + sum_q H^pre,q_i G_in_q exactly (H^pre,q = sigma(b))."""
    w, d, vals, kw = _setup(4, 8, True, 8)
    vals = dict(vals)
    vals["W_r"] = torch.zeros_like(vals["W_r"])
    vals["W_pre_list"] = [torch.zeros_like(t) for t in vals["W_pre_list"]]
    g, fwd, _ = O.flash_group_grads(vals, d["G_X"], d["G_in_list"], **kw)
    T, N, _ = vals["X"].shape
    idx = fwd["idx"]
    for t in range(T):
        for i in range(N):
            if (idx[t] == i).any():
                continue
            want = d["G_X"][t, i].to(F64).clone()
            for q in range(len(d["F_list"])):
                h = 1.0 / (1.0 + torch.exp(-vals["b_pre"][q][i]))
                want += h * d["G_in_list"][q][t].to(F64)
            assert torch.allclose(g["X"][t, i], want, rtol=0, atol=1e-12), (t, i)


def test_flash_sampled_tokens_equal_the_full_group():
    """Evaluating the group on a subset of tokens (their states only, every F
    whole) gives those tokens' outputs and state gradients of the full
    evaluation: every step is per token except the causal convolutions, which
    read the same sequence's earlier F rows (tokens on both sides of a
    sequence start are sampled)."""
    w = synth.Workload(T=24, S=12, N=8, k=4, m=2, C=32, Kr=4)
    d = synth.flash_inputs(w, 4, 21, grads=True, bias_std=0.5)
    vals = O.flash_leaves(d["X"], d["F_list"], d["conv_w_list"], d["W_r"], d["W_pre_list"], d["W_post_list"],
                          d["W_res"], d["alpha_pre"], d["b_pre"], d["alpha_post"], d["b_post"], d["alpha_res"],
                          d["b_res"])
    kw = dict(m=w.m, k=w.k, S=w.S)
    full, ffwd, _ = O.flash_group_grads(vals, d["G_X"], d["G_in_list"], wrt=("X",), **kw)
    tok = torch.tensor([0, 5, 11, 12, 13, 23])
    sub = dict(vals, X=vals["X"][tok])
    part, pfwd, _ = O.flash_group_grads(sub, d["G_X"][tok], [g[tok] for g in d["G_in_list"]], wrt=("X",),
                                        tokens=tok, **kw)
    assert part["W_r"] is None and part["F_list"] is None
    assert torch.equal(pfwd["idx"], ffwd["idx"][tok])
    torch.testing.assert_close(pfwd["X_new"], ffwd["X_new"][tok], rtol=1e-12, atol=1e-12)
    for a, b in zip(pfwd["inputs"], ffwd["inputs"]):
        torch.testing.assert_close(a, b[tok], rtol=1e-12, atol=1e-12)
    torch.testing.assert_close(part["X"], full["X"][tok], rtol=1e-10, atol=1e-12)

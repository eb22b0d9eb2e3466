"""xHC-Flash groups (Q = 2, 4) on the GPU vs the fp64 oracle, through the C ABI."""

import pytest
import torch

from oracle import xhc_oracle as O
from paper_2607_14530_amd import synth
from paper_2607_14530_amd import xhc as X
from tests.parity_util import BF16_ULP_REL, assert_bf16_close, assert_coef_close, compare_routing

pytestmark = pytest.mark.gpu
F64 = torch.float64
W = synth.Workload


def _run_group(w, Q, seed):
    d = synth.flash_inputs(w, Q, seed, device="cuda")
    g = X.FlashGroup(X.dims_for(w), Q, d, "cuda")
    state = d["X"].clone()
    states = []
    g.pre(state)
    for q in range(1, Q + 1):
        g.step(q, state, d["F_list"][q - 1])
        states.append(state.clone())
    torch.cuda.synchronize()
    return d, g, states


def _oracle(w, d, Q, tokens=None):
    X0 = d["X"] if tokens is None else d["X"][tokens.to(d["X"].device)]
    cpu = lambda v: v.cpu() if torch.is_tensor(v) else v
    return O.xhc_flash_group(
        X0.to("cpu", F64), [f.cpu() for f in d["F_list"]], d["W_r"].cpu(), [cpu(v) for v in d["W_pre_list"]],
        [cpu(v) for v in d["W_post_list"]], d["W_res"].cpu(), [cpu(v) for v in d["conv_w_list"]],
        d["alpha_pre"], [cpu(v) for v in d["b_pre"]], d["alpha_post"], [cpu(v) for v in d["b_post"]],
        d["alpha_res"], d["b_res"].cpu(), m=w.m, k=w.k, S=w.S, kappa=w.kappa, tokens=tokens,
        router=w.router, gram_schmidt_on=bool(w.gram_schmidt),
        round_state=w.state != "f32")   # an fp32 state stores the written rows unrounded


def _check(w, Q, d, g, states, tokens=None):
    sel = (lambda t: t.cpu()) if tokens is None else (lambda t: t[tokens.to(t.device)].cpu())
    ref = _oracle(w, d, Q, tokens)
    same = compare_routing(sel(g.idx), ref, w.m)
    assert_coef_close(sel(g.p)[same], ref["p"][same], "p")
    X0r = ref_state = d["X"] if tokens is None else d["X"][tokens.to(d["X"].device)]
    prev = X0r.to("cpu", F64)
    idx = ref["idx"]
    ar = torch.arange(idx.shape[0])[:, None]
    for q in range(Q):
        assert_coef_close(sel(g.Hpre[q]), ref["Hpre"][q], f"Hpre[{q}]")
        # input of sublayer q+1 reads the active rows after q rounded writes
        a_prev = prev[ar, idx]                                                   # [T, k, C]
        hsel = torch.gather(ref["Hpre"][q], 1, idx)                              # [T, k]
        slack_in = q * BF16_ULP_REL * (hsel[:, :, None] * a_prev.abs()).sum(1)
        assert_bf16_close(sel(g.inputs[q])[same], ref["inputs"][q][same], f"input[{q + 1}]",
                          slack=slack_in[same])
        assert_coef_close(sel(g.Hpost[q])[same], ref["Hpost"][q][same], f"Hpost[{q + 1}]")
        got = sel(states[q])
        slack_x = q * BF16_ULP_REL * prev.abs()
        assert_bf16_close(got[same], ref["X_steps"][q][same], f"state after sublayer {q + 1}",
                          slack=slack_x[same])
        prev = ref["X_steps"][q]
    assert_coef_close(sel(g.Hres)[same], ref["Hres"][same], "Hres")
    # rows outside the shared routing are never written
    X0 = sel(d["X"])
    act = torch.zeros(X0.shape[0], X0.shape[1], dtype=torch.bool)
    act[torch.arange(X0.shape[0])[:, None], sel(g.idx).long()] = True
    assert torch.equal(sel(states[-1])[~act], X0[~act])


@pytest.mark.parametrize("Q", [2, 4])
@pytest.mark.parametrize("w", [
    W(T=96, S=48, N=16, k=4, m=2, C=256, Kr=4, name="flash-small"),
    W(T=50, N=8, k=4, m=1, C=128, Kr=3, kappa=(3, 6), name="flash-odd"),
    W(T=96, S=48, N=16, k=4, m=2, C=256, Kr=4, router="softmax", name="flash-softmax"),
    W(T=64, S=32, N=8, k=4, m=2, C=256, Kr=4, gram_schmidt=0, name="flash-gs-off"),
    W(T=64, S=32, N=8, k=4, m=2, C=256, Kr=4, state="f32", name="flash-f32"),
], ids=lambda w: w.name)
def test_flash_group_matches_oracle(w, Q):
    print(f"[flash] {w.name} Q={Q}", flush=True)
    d, g, states = _run_group(w, Q, seed=21)
    _check(w, Q, d, g, states)


def test_flash_full_size_sampled_tokens():
    """The 4-sublayer group at T=16384 (2 x 8192), N=16, k=4, C=4096, on sampled tokens."""
    w = synth.sparse_c4096(4)
    print(f"[flash-full] {w.name} Q=4", flush=True)
    d, g, states = _run_group(w, 4, seed=4)
    gen = torch.Generator().manual_seed(17)
    tok = torch.tensor(sorted(set([0, 1, 8191, 8192, 8193, 16383] + torch.randint(0, 16384, (24,), generator=gen).tolist())))
    _check(w, 4, d, g, states, tokens=tok)

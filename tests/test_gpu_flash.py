"""xHC-Flash groups (Q = 2, 4) on the GPU vs the fp64 oracle, through the C ABI."""

import pytest
import torch

from oracle import xhc_oracle as O
from paper_2607_14530_amd import synth
from paper_2607_14530_amd import xhc as X
from tests.parity_util import assert_bf16_close, assert_coef_close, compare_routing

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
    """Routing and pre-maps against the oracle's group; then each sublayer q
    teacher-forced: the oracle runs step q from the active rows the GPU
    stored before it (xhc_flash_step), so the input, mappings and written
    rows of q are compared at the plain bounds, with no allowance for earlier
    rounded rows."""
    sel = (lambda t: t.cpu()) if tokens is None else (lambda t: t[tokens.to(t.device)].cpu())
    ref = _oracle(w, d, Q, tokens)
    same = compare_routing(sel(g.idx), ref, w.m)
    assert_coef_close(sel(g.p)[same], ref["p"][same], "p")
    for q in range(Q):
        assert_coef_close(sel(g.Hpre[q]), ref["Hpre"][q], f"Hpre[{q}]")
    X0 = sel(d["X"]).to(F64)
    idx = sel(g.idx).long()
    ar = torch.arange(idx.shape[0])[:, None]
    p, Hpre = sel(g.p).to(F64), torch.stack([sel(h) for h in g.Hpre]).to(F64)
    cpu = lambda v: v.cpu() if torch.is_tensor(v) else v
    prev = X0
    for q in range(2, Q + 1):   # the non-active base readouts of the entry pass
        assert_bf16_close(sel(g.base[q - 2])[same], ref["bases"][q - 1][same], f"base[{q}]")
    for q in range(1, Q + 1):
        last = q == Q
        # base^(q) as the GPU stored it (state dtype) enters input_q
        base = sel(g.base[q - 2]).to(F64) if q >= 2 else None
        st = O.xhc_flash_step(prev[ar, idx], q, X0, idx, p, Hpre, d["F_list"][q - 1].cpu(),
                              cpu(d["conv_w_list"][q - 1]), cpu(d["W_post_list"][q - 1]), d["alpha_post"][q - 1],
                              cpu(d["b_post"][q - 1]), cpu(d["W_res"]) if last else None,
                              d["alpha_res"] if last else None, cpu(d["b_res"]) if last else None,
                              Q=Q, S=w.S, kappa=w.kappa, gram_schmidt_on=bool(w.gram_schmidt), tokens=tokens,
                              base=base)
        # the step runs on the GPU's own routing, so every token is compared
        assert_bf16_close(sel(g.inputs[q - 1]), st["input"], f"input[{q}]")
        assert_coef_close(sel(g.Hpost[q - 1]), st["Hpost"], f"Hpost[{q}]")
        if last:
            assert_coef_close(sel(g.Hres), st["Hres"], "Hres")
        got = sel(states[q - 1]).to(F64)
        assert_bf16_close(got[ar, idx], st["a_new"], f"rows after sublayer {q}")
        prev = got
    # rows outside the shared routing are never written
    X0b = sel(d["X"])
    act = torch.zeros(X0b.shape[0], X0b.shape[1], dtype=torch.bool)
    act[torch.arange(X0b.shape[0])[:, None], idx] = True
    assert torch.equal(sel(states[-1])[~act], X0b[~act])


@pytest.mark.parametrize("Q", [2, 4])
@pytest.mark.parametrize("w", [
    W(T=96, S=48, N=16, k=4, m=2, C=256, Kr=4, name="flash-small"),
    W(T=50, N=8, k=4, m=1, C=128, Kr=3, kappa=(3, 6), name="flash-odd"),
    W(T=96, S=48, N=16, k=4, m=2, C=256, Kr=4, router="softmax", name="flash-softmax"),
    W(T=64, S=32, N=8, k=4, m=2, C=256, Kr=4, gram_schmidt=0, name="flash-gs-off"),
    W(T=64, S=32, N=8, k=4, m=2, C=256, Kr=4, state="f32", name="flash-f32"),
    # attention-side temporal augmentation (ablation): every sublayer has K_r components
    W(T=96, S=48, N=16, k=4, m=2, C=256, Kr=4, attn_aug=1, name="flash-attn-aug"),
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

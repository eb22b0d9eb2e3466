"""NaN and +-Inf in the state and the sublayer output, HIP path vs the oracle.

A NaN or an infinity in a token's state makes all its router logits NaN
(through the LayerNorm statistics).  Routing then still assigns each slot
one distinct stream (NaN ranks below every number, ties to the lower index,
so the routed slots take streams m, m+1, ...), p of a routed slot is NaN,
and the NaN propagates into H^pre, the input and the written rows; nothing
indexes out of range and no wait of the single-pass kernel gives up.  Other
tokens are unaffected.  Compared element by element: idx exactly, NaN
positions exactly, finite values at the usual tolerances, unwritten rows bit
for bit."""

import pytest
import torch

from paper_2607_14530_amd import synth
from paper_2607_14530_amd import xhc as X
from tests.parity_util import (BF16_ATOL, BF16_RTOL, COEF_ATOL, compare_routing, oracle_post,
                               oracle_pre)

pytestmark = pytest.mark.gpu
F64 = torch.float64
NAN, INF = float("nan"), float("inf")


def _poison(inp):
    Xs, F = inp["X"], inp["F"]
    Xs[3, 5, 17] = NAN        # a stream the routing will not pick
    Xs[10, 0, 3] = INF        # a fixed (always active) stream
    Xs[20, 9, 100] = -INF
    Xs[33, 2, 0] = NAN        # the first routed stream of a NaN token
    F[40, 7] = NAN            # the conv window carries it to tokens 40..51
    return inp


def _close(got, ref, atol, rtol, what):
    got = got.detach().to("cpu", F64)
    ref = ref.detach().to("cpu", F64)
    diff = torch.isnan(got) != torch.isnan(ref)
    assert not bool(diff.any()), f"{what}: NaN positions differ, first at {diff.nonzero()[:6].tolist()}"
    fin = torch.isfinite(ref)
    assert torch.equal(torch.isinf(got), torch.isinf(ref)), f"{what}: infinite positions differ"
    d = (got[fin] - ref[fin]).abs()
    bound = torch.maximum(torch.full_like(ref[fin], atol), rtol * ref[fin].abs())
    assert bool((d <= bound).all()), f"{what}: max |d| = {d.max().item():.3e}"


@pytest.mark.parametrize("impl", [X.XHC_IMPL_FUSED, X.XHC_IMPL_MULTI], ids=["fused", "multi"])
@pytest.mark.parametrize("Kr", [1, 4])
def test_nan_and_inf_propagate_without_bad_indices(Kr, impl):
    w = synth.Workload(T=64, S=32, N=16, k=4, m=2, C=256, Kr=Kr, name=f"nan-Kr{Kr}")
    print(f"[nan] Kr={Kr} impl={impl}", flush=True)
    inp = _poison(synth.sublayer_inputs(w, 31))
    dev = {n: (v.to("cuda") if v is not None else None) for n, v in inp.items()}
    sub = X.Sublayer(X.dims_for(w, impl=impl), dev, "cuda")
    Xs = dev["X"].clone()
    sub.pre(Xs)
    before = Xs.clone()
    sub.post(Xs, dev["F"])
    torch.cuda.synchronize()
    assert sub.pre_failures() == 0
    ref = oracle_pre(inp, w)
    idx = sub.idx.cpu().long()
    assert int(idx.min()) >= 0 and int(idx.max()) < w.N
    for t in (3, 10, 20, 33):   # every router logit NaN: the routed slots take streams 2, 3
        assert idx[t].tolist() == [0, 1, 2, 3], (t, idx[t].tolist())
    same = compare_routing(sub.idx, ref, w.m)
    assert bool(same.all())
    _close(sub.p, ref["p"], COEF_ATOL, 0.0, "p")
    _close(sub.Hpre, ref["Hpre"], COEF_ATOL, 0.0, "Hpre")
    _close(sub.Hres, ref["Hres"], COEF_ATOL, 0.0, "Hres")
    _close(sub.Hpost, ref["Hpost"], COEF_ATOL, 0.0, "Hpost")
    _close(sub.input, ref["input"], BF16_ATOL, BF16_RTOL, "input")
    ref_X = oracle_post(inp, w, ref)
    _close(Xs, ref_X, BF16_ATOL, BF16_RTOL, "state after post")
    act = torch.zeros(w.T, w.N, dtype=torch.bool)
    act[torch.arange(w.T)[:, None], idx] = True
    got16 = Xs.cpu().view(torch.int16)
    before16 = before.cpu().view(torch.int16)
    assert torch.equal(got16[~act], before16[~act]), "unwritten rows changed"
    assert torch.isnan(Xs[3].float()).any() and torch.isnan(Xs[45].float()).any() == (Kr > 1)

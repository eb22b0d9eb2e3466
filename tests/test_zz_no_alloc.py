"""xhc_post_noalloc (no workspace, nothing allocated) against xhc_post,
through the C ABI: the same kernels run on the library's static scratch
instead of a caller workspace, so the state after the write-back must be
bit-identical.  Two calls in a row, the second on a smaller input (the
scratch keeps the first call's contents); MLP-type (the scratch holds the
Gram partials and write-back weights) and attention-type (no scratch)."""

import ctypes

import pytest
import torch

from paper_2607_14530_amd import synth
from paper_2607_14530_amd import xhc as X

pytestmark = pytest.mark.gpu


def _pre(w, seed):
    inp = synth.sublayer_inputs(w, seed, device="cuda")
    sub = X.Sublayer(X.dims_for(w), inp, "cuda")
    Xs = inp["X"].clone()
    sub.pre(Xs)
    return inp, sub, Xs


def _noalloc(sub, Xs, F, save=None):
    st = X.lib().xhc_post_noalloc(ctypes.byref(sub.d), Xs.data_ptr(), F.data_ptr(),
                                  sub.conv_w.data_ptr() if sub.conv_w is not None else None,
                                  sub.idx.data_ptr(), sub.p.data_ptr(), sub.Hres.data_ptr(), sub.Hpost.data_ptr(),
                                  save.data_ptr() if save is not None else None,
                                  torch.cuda.current_stream().cuda_stream)
    assert st == X.XHC_OK, X.STATUS_NAMES.get(st, st)


@pytest.mark.parametrize("Kr", [4, 1])
def test_post_noalloc_matches_post_on_two_calls(Kr):
    for T, S, C, seed in ((2048, 1024, 4096, 3), (300, 100, 768, 4)):
        w = synth.Workload(T=T, S=S, N=16, k=4, m=2, C=C, Kr=Kr, name=f"noalloc-T{T}")
        print(f"[noalloc] Kr={Kr} T={T} C={C}", flush=True)
        inp, sub, Xs = _pre(w, seed)
        a, b = Xs.clone(), Xs.clone()
        sa = torch.empty(T, 4, C, dtype=torch.bfloat16, device="cuda")
        sb = torch.empty_like(sa)
        sub.post(a, inp["F"], Xact_save=sa)
        _noalloc(sub, b, inp["F"], sb)
        torch.cuda.synchronize()
        assert torch.equal(a, b), "state after the write-back differs"
        assert torch.equal(sa, sb), "saved active rows differ"


def test_post_noalloc_rejects_shapes_beyond_its_scratch():
    # T = 2^20 tokens at C = 4096, K_r = 4 needs about 220 MiB of scratch
    d = X.make_dims(1 << 20, 16, 4, 2, 4096, Kr=4, S=8192)
    assert X.xhc_workspace_bytes(d, X.XHC_OP_POST) > X.NOALLOC_SCRATCH_BYTES
    st = X.lib().xhc_post_noalloc(ctypes.byref(d), 16, 16, 16, 16, 16, 16, 16, None, None)
    assert st == X.XHC_EWORKSPACE

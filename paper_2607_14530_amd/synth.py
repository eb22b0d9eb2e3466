"""Seeded synthetic inputs for the xHC connection.

Holds none of the method's arithmetic: it only draws tensors of the shapes
and distributions of the workloads (state and sublayer output ~ N(0, 1) in
bf16, projection weights ~ N(0, 0.02) in fp32, gating scalars 0.01, biases
0, conv kernels ~ N(0, 1), upstream gradients ~ N(0, 1)).  Both the HIP
path and the CPU oracle consume what is drawn here.

Every draw uses a torch.Generator seeded by the caller on the device where
the tensors are made; on the CPU the stream is reproducible across runs and
machines.  Draw order is fixed: X, F, W_r, W_pre, W_res, W_post, conv_w,
then gradients.
"""

from __future__ import annotations

from dataclasses import dataclass

import torch

KAPPA_DEFAULT = (4, 8, 12)


@dataclass
class Workload:
    """Shape of one sublayer workload (notation of the paper)."""
    T: int
    N: int
    k: int
    m: int
    C: int
    Kr: int = 1
    S: int = 0                      # tokens per sequence; 0 means S = T
    kappa: tuple = KAPPA_DEFAULT
    state: str = "bf16"             # "bf16" or "f32"
    alpha: tuple = (0.01, 0.01, 0.01)
    name: str = ""
    router: str = "sigmoid"         # "sigmoid" (eq:router) or "softmax" (ablation)
    gram_schmidt: int = 1           # 0: components used as they are (the Muon-trained variant)
    attn_aug: int = 0               # 1: attention-type sublayers of a Flash group augmented too (ablation)

    def __post_init__(self):
        if self.S == 0:
            self.S = self.T

    @property
    def dtype(self):
        return torch.bfloat16 if self.state == "bf16" else torch.float32


def _randn(shape, g, device, std=1.0):
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    return t * std if std != 1.0 else t


def sublayer_inputs(w: Workload, seed: int, device="cpu", weight_std=0.02,
                    grads=False, bias_std=0.0):
    """Inputs of one full xHC sublayer.

    Returns a dict: X [T,N,C], F [T,C] in the state dtype; W_r, W_pre [N*C,N],
    W_res [k*C,k*k], W_post [k*C,k*Kr] fp32; conv_w [sum kappa, C] fp32 or
    None (Kr == 1); alpha [3] = (pre, res, post) fp32; b_pre [N], b_res
    [k*k], b_post [k*Kr] fp32 (zero unless bias_std > 0); with grads=True
    also G_X [T,N,C] and G_in [T,C] in the state dtype.
    """
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    T, N, k, C, Kr = w.T, w.N, w.k, w.C, w.Kr
    d = {}
    d["X"] = _randn((T, N, C), g, device).to(w.dtype)
    d["F"] = _randn((T, C), g, device).to(w.dtype)
    d["W_r"] = _randn((N * C, N), g, device, weight_std)
    d["W_pre"] = _randn((N * C, N), g, device, weight_std)
    d["W_res"] = _randn((k * C, k * k), g, device, weight_std)
    d["W_post"] = _randn((k * C, k * Kr), g, device, weight_std)
    d["conv_w"] = _randn((sum(w.kappa), C), g, device) if Kr > 1 else None
    d["alpha"] = torch.tensor(w.alpha, dtype=torch.float32, device=device)
    if bias_std > 0:
        d["b_pre"] = _randn((N,), g, device, bias_std)
        d["b_res"] = _randn((k * k,), g, device, bias_std)
        d["b_post"] = _randn((k * Kr,), g, device, bias_std)
    else:
        d["b_pre"] = torch.zeros(N, device=device)
        d["b_res"] = torch.zeros(k * k, device=device)
        d["b_post"] = torch.zeros(k * Kr, device=device)
    if grads:
        d["G_X"] = _randn((T, N, C), g, device).to(w.dtype)
        d["G_in"] = _randn((T, C), g, device).to(w.dtype)
    return d


def flash_inputs(w: Workload, Q: int, seed: int, device="cpu", weight_std=0.02, grads=False,
                 bias_std=0.0):
    """Inputs of one xHC-Flash sharing group of Q sublayers (Q = 2 or 4).

    Sublayer q (1-based) is attention-type (one write-back component, or
    1 + len(kappa) with w.attn_aug) when q is odd and MLP-type
    (1 + len(kappa) components) when q is even.  Returns
    X, F_list (Q x [T,C]), W_r, W_pre_list (Q x [N*C,N]), W_post_list
    (Q x [k*C, k*K_q]), W_res [k*C,k*k], conv_w_list (None for attention),
    alpha_pre/alpha_post (Q floats), alpha_res, b_pre (Q x [N]),
    b_post (Q x [k*K_q]), b_res [k*k].  With grads=True also the upstream
    gradients G_X [T,N,C] (of the state after the group) and G_in_list
    (Q x [T,C], of each sublayer input), drawn after everything above; with
    bias_std > 0 the biases are drawn last ~ N(0, bias_std).
    """
    assert Q in (2, 4)
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    T, N, k, C = w.T, w.N, w.k, w.C
    Kq = [1 if (q % 2 == 1 and not w.attn_aug) else 1 + len(w.kappa) for q in range(1, Q + 1)]
    d = {"Kq": Kq}
    d["X"] = _randn((T, N, C), g, device).to(w.dtype)
    d["F_list"] = [_randn((T, C), g, device).to(w.dtype) for _ in range(Q)]
    d["W_r"] = _randn((N * C, N), g, device, weight_std)
    d["W_pre_list"] = [_randn((N * C, N), g, device, weight_std) for _ in range(Q)]
    d["W_post_list"] = [_randn((k * C, k * Kq[q]), g, device, weight_std) for q in range(Q)]
    d["W_res"] = _randn((k * C, k * k), g, device, weight_std)
    d["conv_w_list"] = [(_randn((sum(w.kappa), C), g, device) if Kq[q] > 1 else None)
                        for q in range(Q)]
    d["alpha_pre"] = [w.alpha[0]] * Q
    d["alpha_post"] = [w.alpha[2]] * Q
    d["alpha_res"] = w.alpha[1]
    d["b_pre"] = [torch.zeros(N, device=device) for _ in range(Q)]
    d["b_post"] = [torch.zeros(k * Kq[q], device=device) for q in range(Q)]
    d["b_res"] = torch.zeros(k * k, device=device)
    if grads:
        d["G_X"] = _randn((T, N, C), g, device).to(w.dtype)
        d["G_in_list"] = [_randn((T, C), g, device).to(w.dtype) for _ in range(Q)]
    if bias_std > 0:
        d["b_pre"] = [_randn((N,), g, device, bias_std) for _ in range(Q)]
        d["b_post"] = [_randn((k * Kq[q],), g, device, bias_std) for q in range(Q)]
        d["b_res"] = _randn((k * k,), g, device, bias_std)
    return d


# Named workloads: the paper's default connection shape (N=16, k=4, m=2,
# kappa = 4/8/12, 8192-token sequences) at the widths exercised here.
def tiny_dense():
    """Dense mHC-equivalent: every stream active and fixed, fp32 state."""
    return Workload(T=64, N=4, k=4, m=4, C=256, Kr=1, state="f32", name="tiny-dense-T64-N4-C256")


def sparse_c1024(Kr):
    return Workload(T=4096, N=16, k=4, m=2, C=1024, Kr=Kr, name=f"xhc-T4096-N16-k4-C1024-Kr{Kr}")


def sparse_c4096(Kr):
    return Workload(T=16384, S=8192, N=16, k=4, m=2, C=4096, Kr=Kr,
                    name=f"xhc-T16384-N16-k4-C4096-Kr{Kr}")


def bwd_sweep(N, Kr):
    return Workload(T=8192, N=N, k=4, m=2, C=4096, Kr=Kr, name=f"xhc-bwd-T8192-N{N}-k4-C4096-Kr{Kr}")

"""Oracle for the xHC / xHC-Flash per-sublayer residual-stream connection.

TEST INFRASTRUCTURE ONLY.  This module is a plain, slow, CPU, float64
implementation of what the paper (xHC: Expanded Hyper-Connections,
arXiv 2607.14530) defines, used to check the HIP library.  Only the test
suite, the smoke check and the CPU-baseline leg of the benchmark may import
it.  It shares no code with the HIP path: no kernels, no packing, no helpers.

Conventions (readings of the paper where it is silent, see the ambiguity
register in the design notes; each is repeated at the line that uses it):

* The state of one token is X in R^{N x C}; ``flatten`` is stream-major,
  x[i*C + c] = X[i, c].  The active state is gathered in slot order and
  ``vec`` is slot-major, a[j*C + c] = X[I_j, c].
* Projection operands are bfloat16 (Sec. "Infrastructure Design"): the
  state already is; every projection weight is rounded fp32 -> bf16 (round
  to nearest even) before use.  Everything else is exact float64 here.
* ``mat_{k x k}`` and ``mat_{k x K_r}`` are row-major: H^res[j, l] =
  z[j*k + l], H^post[j, r] = z[j*K_r + r].
* Routing: slots 0..m-1 hold the fixed streams 0..m-1 (p = 1); slots
  m..k-1 hold the k-m streams among m..N-1 with the largest router logit,
  in descending logit order, ties to the lower stream index (eq:router_topk;
  sigma is monotone, so ordering logits orders the scores).  The softmax
  router of the ablation table (row 11) replaces sigma by a softmax over all
  N logits (the projection scores every stream); it is monotone too, so the
  selection is the same and only p changes.
* Sinkhorn: each iteration normalises rows, then columns (eq:mhc_sinkhorn,
  20 iterations per the hyperparameter table); afterwards each row i is
  divided by its sum s_i when s_i > 1 + clamp_delta (the row-sum clamp of
  App. A, "xHC Configuration"; clamp_delta = 0 is the literal max(s_i, 1)).
* Temporal augmentation: g_j[t] = sum_{i < kappa_j} w_j[i] * out[t - i],
  per channel, with out[t - i] = 0 before the start of t's sequence
  (eq:aug and Sec. "Parameterization Details").  conv_w stacks the branch
  kernels row-wise: rows [0, kappa_1) are w_1, the next kappa_2 rows w_2 ...
* Gram-Schmidt follows the printed formula eq:gs; a coefficient whose
  denominator <v_i, v_i> is zero is taken as zero.

Parity status of each function is stated in its docstring; the pins live in
``tests/test_oracle_*.py``.
"""

from __future__ import annotations

import torch

F64 = torch.float64


# --------------------------------------------------------------------------
# small pieces
# --------------------------------------------------------------------------

def bf16_operand(w: torch.Tensor) -> torch.Tensor:
    """Round fp32 values to bfloat16 (nearest even) and return them as fp64.

    The paper keeps projection operands in bfloat16 (Sec. "Infrastructure
    Design").  The conversion is done from float32 so that a value is rounded
    exactly once.
    """
    return w.to(torch.float32).to(torch.bfloat16).to(F64)


def round_state_bf16(x: torch.Tensor) -> torch.Tensor:
    """Round values of the residual state to bfloat16 (stored precision)."""
    return x.to(torch.bfloat16).to(F64)


def sigmoid(z: torch.Tensor) -> torch.Tensor:
    return 1.0 / (1.0 + torch.exp(-z))


def router_scores(z_r: torch.Tensor, router: str = "sigmoid") -> torch.Tensor:
    """Per-stream router scores s from the logits z_r [T, N]: sigma
    (eq:router) or, for the ablation (ablation table, row 11), a softmax over
    the N streams of each token.  Parity: pinned (see tests)."""
    if router == "sigmoid":
        return sigmoid(z_r)
    if router == "softmax":
        return torch.softmax(z_r, dim=1)
    raise ValueError(router)


def layer_norm(x: torch.Tensor, eps: float) -> torch.Tensor:
    """LayerNorm over the last axis, biased variance, no affine (eq:router)."""
    mu = x.mean(-1, keepdim=True)
    var = ((x - mu) ** 2).mean(-1, keepdim=True)
    return (x - mu) / torch.sqrt(var + eps)


def rms_norm(x: torch.Tensor, eps: float) -> torch.Tensor:
    """RMSNorm over the last axis, no gain (eq:param_pre, eq:param_res)."""
    return x / torch.sqrt((x * x).mean(-1, keepdim=True) + eps)


def sinkhorn(M: torch.Tensor, iters: int) -> torch.Tensor:
    """Sinkhorn-Knopp on the last two axes: rows, then columns, per iteration."""
    for _ in range(iters):
        M = M / M.sum(-1, keepdim=True)
        M = M / M.sum(-2, keepdim=True)
    return M


def row_clamp(H: torch.Tensor, delta: float) -> torch.Tensor:
    """Divide each row by its sum when the sum exceeds 1 + delta (App. A)."""
    s = H.sum(-1, keepdim=True)
    return torch.where(s > 1.0 + delta, H / s, H)


def residual_mapping(z_res: torch.Tensor, alpha_res, b_res, k: int,
                     iters: int, delta: float) -> torch.Tensor:
    """H^res = clamp(SK(exp(alpha * mat_{k x k}(z) + b)))  (eq:param_res)."""
    T = z_res.shape[0]
    logits = alpha_res * z_res + b_res
    return row_clamp(sinkhorn(torch.exp(logits).reshape(T, k, k), iters), delta)


def post_mapping(z_post: torch.Tensor, alpha_post, b_post, k: int, Kr: int) -> torch.Tensor:
    """H^post = 2 sigma(alpha * mat_{k x K_r}(z) + b)  (eq:param_post)."""
    T = z_post.shape[0]
    return (2.0 * sigmoid(alpha_post * z_post + b_post)).reshape(T, k, Kr)


def route(z_r: torch.Tensor, m: int, k: int, router: str = "sigmoid"):
    """Fixed-plus-TopK routing (eq:router_topk); ``router`` picks the score
    function (see router_scores).

    Returns (idx [T,k] int64, p [T,k] fp64, gap [T] fp64).  ``gap`` is the
    smallest difference between neighbouring logits in the sorted routed
    list, taken over the k-m selected ones and the first unselected one; it
    is +inf when nothing is routed.  A small gap marks a near-tie, where more
    than one slot assignment is correct within rounding.
    """
    T, N = z_r.shape
    idx = torch.empty(T, k, dtype=torch.int64)
    idx[:, :m] = torch.arange(m)
    gap = torch.full((T,), float("inf"), dtype=F64)
    if k > m:
        cand = z_r[:, m:]
        order = torch.sort(-cand, dim=1, stable=True).indices   # ties keep lower index first
        idx[:, m:] = order[:, : k - m] + m
        n_look = min(k - m + 1, N - m)
        srt = torch.gather(cand, 1, order[:, :n_look])
        if n_look > 1:
            gap = (srt[:, :-1] - srt[:, 1:]).min(dim=1).values
    s = router_scores(z_r, router)
    p = torch.ones(T, k, dtype=F64)
    if k > m:
        p[:, m:] = torch.gather(s, 1, idx[:, m:])
    return idx, p, gap


def gather_rows(X: torch.Tensor, idx: torch.Tensor) -> torch.Tensor:
    """X_act[t, j, :] = X[t, idx[t, j], :]."""
    T = X.shape[0]
    return X[torch.arange(T)[:, None], idx]


# --------------------------------------------------------------------------
# temporal feature augmentation + Gram-Schmidt
# --------------------------------------------------------------------------

def temporal_branches(F: torch.Tensor, conv_w: torch.Tensor, kappa, S: int,
                      tokens: torch.Tensor) -> list:
    """g_j[t] for t in ``tokens`` (eq:aug, Sec. "Parameterization Details").

    F: [T, C] sublayer output of the whole batch (any float dtype); conv_w:
    [sum(kappa), C].  Causal, per channel, zero before each sequence start.
    """
    w = conv_w.to(F64)
    pos = tokens % S
    out = []
    row = 0
    for kap in kappa:
        g = torch.zeros(tokens.shape[0], F.shape[1], dtype=F64)
        for i in range(kap):
            valid = pos >= i
            src = torch.where(valid, tokens - i, tokens)
            g = g + torch.where(valid[:, None], w[row + i] * F[src].to(F64), 0.0)
        out.append(g)
        row += kap
    return out


def gram_schmidt(components: list) -> list:
    """Orthogonalise [out, g_1, ..., g_r] per token over C (eq:gs).

    A coefficient is 0 only where <v_i, v_i> is exactly 0 (the printed
    quotient is undefined there); a NaN norm gives a NaN coefficient, as the
    printed quotient does."""
    v = [components[0]]
    for g in components[1:]:
        u = g
        for vi in v:
            nn = (vi * vi).sum(-1, keepdim=True)
            dot = (g * vi).sum(-1, keepdim=True)
            coef = torch.where(nn != 0, dot / torch.where(nn != 0, nn, 1.0), 0.0)
            u = u - coef * vi
        v.append(u)
    return v


def augmented_output(F, conv_w, kappa, S, tokens, gram_schmidt_on=True) -> list:
    """out_aug for token list ``tokens``: K_r components, each [len(tokens), C]."""
    out = F[tokens].to(F64)
    if conv_w is None:
        return [out]
    comps = [out] + temporal_branches(F, conv_w, kappa, S, tokens)
    return gram_schmidt(comps) if gram_schmidt_on else comps


# --------------------------------------------------------------------------
# full xHC sublayer (Alg. "Forward pass of one xHC sublayer")
# --------------------------------------------------------------------------

def xhc_pre(X, W_r, W_pre, W_res, W_post, alpha, b_pre, b_res, b_post, *,
            m, k, Kr, eps=1e-5, sinkhorn_iters=20, clamp_delta=1e-6, router="sigmoid"):
    """Mapping generation + dense read of one xHC sublayer.

    X: [T, N, C] float64 holding the exact state values.  W_r, W_pre: [N*C, N]
    fp32; W_res: [k*C, k*k]; W_post: [k*C, k*Kr]; alpha = (alpha_pre,
    alpha_res, alpha_post); b_pre [N], b_res [k*k], b_post [k*Kr].

    Follows eq:router, eq:router_topk, eq:param_pre, eq:dense_read,
    eq:param_res, eq:param_post.  Parity: pinned (see tests).
    """
    T, N, C = X.shape
    a_pre, a_res, a_post = alpha
    x = X.reshape(T, N * C)                                   # flatten, stream-major
    z_r = layer_norm(x, eps) @ bf16_operand(W_r)              # router logits
    z_pre = rms_norm(x, eps) @ bf16_operand(W_pre)
    Hpre = sigmoid(a_pre * z_pre + torch.as_tensor(b_pre, dtype=F64))
    idx, p, gap = route(z_r, m, k, router)
    act = gather_rows(X, idx)                                 # [T, k, C]
    a_n = rms_norm(act.reshape(T, k * C), eps)                # vec, slot-major
    z_res = a_n @ bf16_operand(W_res)
    z_post = a_n @ bf16_operand(W_post)
    Hres = residual_mapping(z_res, a_res, torch.as_tensor(b_res, dtype=F64), k,
                            sinkhorn_iters, clamp_delta)
    Hpost = post_mapping(z_post, a_post, torch.as_tensor(b_post, dtype=F64), k, Kr)
    inp = torch.einsum("tn,tnc->tc", Hpre, X)                 # dense read
    return dict(input=inp, idx=idx, p=p, Hpre=Hpre, Hres=Hres, Hpost=Hpost,
                z_r=z_r, z_pre=z_pre, z_res=z_res, z_post=z_post, gap=gap)


def xhc_post(X, F, conv_w, idx, p, Hres, Hpost, *, S, kappa=(4, 8, 12),
             tokens=None, gram_schmidt_on=True):
    """Sparse write-back of one xHC sublayer (eq:sparse_write_delta, eq:sparse_write).

    X: [Tt, N, C] float64 state of the tokens ``tokens`` (all tokens when
    None) before the update; F: [T, C] sublayer output of the whole batch
    (needed for the causal window); conv_w: [sum(kappa), C] or None (K_r = 1).
    idx, p, Hres, Hpost belong to the same tokens as X.  Returns the updated
    state (float64): rows idx replaced, every other row returned unchanged.
    Parity: pinned (see tests).
    """
    Tt, N, C = X.shape
    if tokens is None:
        tokens = torch.arange(Tt)
    comps = augmented_output(F, conv_w, kappa, S, tokens, gram_schmidt_on)
    Kr = len(comps)
    assert Hpost.shape[-1] == Kr
    act = gather_rows(X, idx)                                            # [Tt, k, C]
    mixed = torch.einsum("tjl,tlc->tjc", Hres, act)                      # H^res X_act
    wb = sum(Hpost[:, :, r, None] * comps[r][:, None, :] for r in range(Kr))
    Y = mixed + p[:, :, None] * wb                                       # p on write-back only
    Xn = X.clone()
    Xn[torch.arange(Tt)[:, None], idx] = Y
    return Xn


# --------------------------------------------------------------------------
# dense mHC (separately written, used as a special-case pin)
# --------------------------------------------------------------------------

def mhc_dense(X, F, W_pre, W_post, W_res, alpha, b_pre, b_post, b_res, *,
              eps=1e-5, sinkhorn_iters=20, clamp_delta=1e-6):
    """Dense mHC sublayer, k = N, no router, one write-back component.

    eq:hc with the mappings of eq:mhc_sinkhorn and the gated sigmoid
    parameterisation of Sec. "Parameterization Details" applied to the full
    RMS-normalised state.  X: [T, N, C]; F: [T, C]; W_pre, W_post: [N*C, N];
    W_res: [N*C, N*N].  Returns (input, X_new, Hpre, Hpost, Hres).
    """
    T, N, C = X.shape
    a_pre, a_res, a_post = alpha
    xn = rms_norm(X.reshape(T, N * C), eps)
    Hpre = sigmoid(a_pre * (xn @ bf16_operand(W_pre)) + torch.as_tensor(b_pre, dtype=F64))
    Hpost = 2.0 * sigmoid(a_post * (xn @ bf16_operand(W_post)) + torch.as_tensor(b_post, dtype=F64))
    E = torch.exp(a_res * (xn @ bf16_operand(W_res)) + torch.as_tensor(b_res, dtype=F64))
    Hres = row_clamp(sinkhorn(E.reshape(T, N, N), sinkhorn_iters), clamp_delta)
    inp = (Hpre[:, :, None] * X).sum(1)
    Xn = torch.bmm(Hres, X) + Hpost[:, :, None] * F.to(F64)[:, None, :]
    return inp, Xn, Hpre, Hpost, Hres


# --------------------------------------------------------------------------
# xHC-Flash (Alg. "xHC-Flash: one Transformer block"; App. E.1, E.2)
# --------------------------------------------------------------------------

def flash_sublayer_kind(q: int) -> str:
    """Sublayer q (1-based) of a sharing group: odd = attention, even = MLP."""
    return "attn" if q % 2 == 1 else "mlp"


def xhc_flash_group(X0, F_list, W_r, W_pre_list, W_post_list, W_res, conv_w_list,
                    alpha_pre, b_pre, alpha_post, b_post, alpha_res, b_res, *,
                    m, k, S, kappa=(4, 8, 12), eps=1e-5, sinkhorn_iters=20,
                    clamp_delta=1e-6, round_state=True, gram_schmidt_on=True, tokens=None,
                    router="sigmoid"):
    """One xHC-Flash sharing group of Q = len(F_list) sublayers (Q = 2 or 4).

    Shared routing and Q pre-mappings come from the group-entry state X0
    (eq:flash_dual_read, App. E.2 eq:app_four_sub_base).  Sublayers before
    the last update the active rows without residual mixing
    (eq:flash_attn_update, eq:app_general_writeback); the last sublayer
    applies H^res (Alg. "xHC-Flash", MLP step).  Inputs of later sublayers
    use the active-state form (eq:app_active_state_correction); for Q = 2
    the scalar form of eq:read_reuse is also returned for comparison.

    X0: [T, N, C] float64; F_list[q-1]: [T, C] output of sublayer q;
    W_pre_list[q-1]: [N*C, N]; W_post_list[q-1]: [k*C, k*K_q] with K_q = 1 for
    attention and 1 + len(kappa) for MLP; conv_w_list[q-1]: [sum kappa, C] or
    None; alpha_pre/b_pre/alpha_post/b_post: per-sublayer lists.
    ``round_state`` rounds each written active row to bfloat16 (the stored
    state precision); pins of exact identities switch it off.  With
    ``tokens`` (positions in the batch), X0 holds only those tokens' states
    while F_list keeps the whole batch (the causal window needs it).

    Returns a dict with idx, p, Hpre [Q,T,N], inputs (list of Q [T,C]), bases
    (list, entry 0 is None), Hpost (list), Hres, X (final state), X_steps
    (state after each sublayer) and, for Q = 2, input_scalar_form.
    Parity: pinned (see tests).
    """
    Q = len(F_list)
    assert Q in (2, 4), "a sharing group holds 2 or 4 sublayers"
    T, N, C = X0.shape
    x = X0.reshape(T, N * C)
    z_r = layer_norm(x, eps) @ bf16_operand(W_r)
    xr = rms_norm(x, eps)
    Hpre = torch.stack([
        sigmoid(alpha_pre[q] * (xr @ bf16_operand(W_pre_list[q])) +
                torch.as_tensor(b_pre[q], dtype=F64))
        for q in range(Q)])
    idx, p, gap = route(z_r, m, k, router)
    active = torch.zeros(T, N, dtype=torch.bool)
    active[torch.arange(T)[:, None], idx] = True
    inputs = [torch.einsum("tn,tnc->tc", Hpre[0], X0)]
    bases = [None] + [torch.einsum("tn,tnc->tc", Hpre[q] * (~active), X0) for q in range(1, Q)]
    inp_full = [torch.einsum("tn,tnc->tc", Hpre[q], X0) for q in range(Q)]

    def post_from(a, q):
        Kq = W_post_list[q].shape[1] // k
        z = rms_norm(a.reshape(T, k * C), eps) @ bf16_operand(W_post_list[q])
        return post_mapping(z, alpha_post[q], torch.as_tensor(b_post[q], dtype=F64), k, Kq)

    def res_from(a):
        z = rms_norm(a.reshape(T, k * C), eps) @ bf16_operand(W_res)
        return residual_mapping(z, alpha_res, torch.as_tensor(b_res, dtype=F64), k,
                                sinkhorn_iters, clamp_delta)

    a = gather_rows(X0, idx)
    Hpost = [post_from(a, 0)]
    Hres = None
    X = X0.clone()
    X_steps = []
    if tokens is None:
        tokens = torch.arange(T)
    ar = torch.arange(T)[:, None]
    input_scalar = None
    for q in range(Q):
        comps = augmented_output(F_list[q], conv_w_list[q], kappa, S, tokens, gram_schmidt_on)
        Hp = Hpost[q]
        wb = sum(Hp[:, :, r, None] * comps[r][:, None, :] for r in range(len(comps)))
        if q < Q - 1:
            a_new = a + p[:, :, None] * wb
        else:
            a_new = torch.einsum("tjl,tlc->tjc", Hres, a) + p[:, :, None] * wb
        if round_state:
            a_new = round_state_bf16(a_new)
        X = X.clone()
        X[ar, idx] = a_new
        X_steps.append(X)
        if q < Q - 1:
            hsel = torch.gather(Hpre[q + 1], 1, idx)                    # H^pre,q+1 at I_j
            inputs.append(bases[q + 1] + (hsel[:, :, None] * a_new).sum(1))
            if Q == 2:
                gamma = (hsel * p * Hp[:, :, 0]).sum(1)                # eq:read_reuse
                input_scalar = inp_full[1] + gamma[:, None] * F_list[0][tokens].to(F64)
            Hpost.append(post_from(a_new, q + 1))
            if q + 1 == Q - 1:
                Hres = res_from(a_new)
        a = a_new
    return dict(idx=idx, p=p, gap=gap, Hpre=Hpre, inputs=inputs, bases=bases,
                inp_full=inp_full, Hpost=Hpost, Hres=Hres, X=X, X_steps=X_steps,
                input_scalar_form=input_scalar, z_r=z_r)


def xhc_flash_step(a, q, X0, idx, p, Hpre, F, conv_w, W_post, alpha_post, b_post,
                   W_res=None, alpha_res=None, b_res=None, *, Q, S, kappa=(4, 8, 12), eps=1e-5,
                   sinkhorn_iters=20, clamp_delta=1e-6, gram_schmidt_on=True, tokens=None, base=None):
    """Sublayer q (1-based) of a sharing group, from the active rows a =
    a^(q-1) [T, k, C] as they are stored before it (float64 values).

    The routing (idx, p) and the pre-maps Hpre [Q, T, N] come from the
    group-entry state X0 (eq:flash_dual_read).  The input of sublayer q is
    the dense read of X0 for q = 1 and base^(q) + sum_j H^pre,q_{I_j} a_j for
    q >= 2 (eq:app_four_sub_base, eq:app_active_state_correction); H^post,q
    (and H^res for q = Q) come from RMS(a) (eq:param_post, eq:param_res, App.
    E.2); the rows become a + p H^post,q out_aug for q < Q and H^res a + p
    H^post,Q out_aug for q = Q (eq:flash_attn_update,
    eq:app_general_writeback).  ``base`` (q >= 2, optional) is base^(q) as
    stored by whoever formed it; when None it is computed from X0.  Returns
    dict(input, Hpost, Hres (q = Q, else None), a_new), a_new unrounded.
    Parity: pinned (chaining it reproduces xhc_flash_group, see tests)."""
    T, N, C = X0.shape
    k = idx.shape[1]
    Kq = W_post.shape[1] // k
    active = torch.zeros(T, N, dtype=torch.bool)
    active[torch.arange(T)[:, None], idx] = True
    if q == 1:
        inp = torch.einsum("tn,tnc->tc", Hpre[0], X0)
    else:
        if base is None:
            base = torch.einsum("tn,tnc->tc", Hpre[q - 1] * (~active), X0)
        hsel = torch.gather(Hpre[q - 1], 1, idx)
        inp = base + (hsel[:, :, None] * a).sum(1)
    a_n = rms_norm(a.reshape(T, k * C), eps)
    Hpost = post_mapping(a_n @ bf16_operand(W_post), alpha_post, torch.as_tensor(b_post, dtype=F64), k, Kq)
    Hres = None
    if q == Q:
        Hres = residual_mapping(a_n @ bf16_operand(W_res), alpha_res, torch.as_tensor(b_res, dtype=F64), k,
                                sinkhorn_iters, clamp_delta)
    if tokens is None:
        tokens = torch.arange(T)
    comps = augmented_output(F, conv_w, kappa, S, tokens, gram_schmidt_on)
    wb = sum(Hpost[:, :, r, None] * comps[r][:, None, :] for r in range(len(comps)))
    mixed = a if q < Q else torch.einsum("tjl,tlc->tjc", Hres, a)
    return dict(input=inp, Hpost=Hpost, Hres=Hres, a_new=mixed + p[:, :, None] * wb)


# --------------------------------------------------------------------------
# backward (reverse mode of the forward above)
# --------------------------------------------------------------------------

def sublayer_forward(Xv, F, cw, Wr, Wp, Wre, Wpo, al, bp, bre, bpo, *, m, k, Kr, S, kappa=(4, 8, 12),
                     eps=1e-5, sinkhorn_iters=20, clamp_delta=1e-6, gram_schmidt_on=True, tokens=None,
                     router="sigmoid"):
    """One full xHC sublayer (Alg. "Forward pass of one xHC sublayer"), float64.

    Same steps as xhc_pre followed by xhc_post, except that the projection
    weights are taken as given (already the bf16 operand values), so that a
    finite-difference probe can perturb them.  ``F`` is the sublayer output
    [T, C], or a callable that forms it from the dense-read input.  ``al`` =
    (alpha_pre, alpha_res, alpha_post).  With ``tokens`` (positions in the
    batch), Xv holds only those tokens while F is the whole batch.  Returns
    (X after the write-back, forward results dict).
    """
    T, N, C = Xv.shape
    x = Xv.reshape(T, N * C)
    z_r = layer_norm(x, eps) @ Wr
    Hpre = sigmoid(al[0] * (rms_norm(x, eps) @ Wp) + bp)
    idx, _, gap = route(z_r.detach(), m, k)       # piecewise constant decision
    s = router_scores(z_r, router)
    p = torch.ones(T, k, dtype=F64)
    if k > m:
        p = torch.cat([p[:, :m], torch.gather(s, 1, idx[:, m:])], dim=1)
    a_n = rms_norm(gather_rows(Xv, idx).reshape(T, k * C), eps)
    Hres = residual_mapping(a_n @ Wre, al[1], bre, k, sinkhorn_iters, clamp_delta)
    Hpost = post_mapping(a_n @ Wpo, al[2], bpo, k, Kr)
    inp = torch.einsum("tn,tnc->tc", Hpre, Xv)
    Fv = F(inp) if callable(F) else F
    Xn = xhc_post(Xv, Fv, cw, idx, p, Hres, Hpost, S=S, kappa=kappa,
                  gram_schmidt_on=gram_schmidt_on, tokens=tokens)
    return Xn, dict(idx=idx, p=p, Hpre=Hpre, Hres=Hres, Hpost=Hpost, input=inp, X_new=Xn, out=Fv, gap=gap)


def sublayer_objective(Xv, Fv, cw, Wr, Wp, Wre, Wpo, al, bp, bre, bpo, G_X, G_in, **kw):
    """L = <G_X, X'> + <G_in, input> for one full xHC sublayer (see
    sublayer_forward), float64.  Returns (L, forward results dict)."""
    Xn, fwd = sublayer_forward(Xv, Fv, cw, Wr, Wp, Wre, Wpo, al, bp, bre, bpo, **kw)
    L = (G_X.to(F64) * Xn).sum() + (G_in.to(F64) * fwd["input"]).sum()
    return L, fwd


def stream_sum(X: torch.Tensor) -> torch.Tensor:
    """Final stream reduction (App. "Final Stream Reduction"): the N streams of
    each token are summed before the last RMSNorm.  [T, N, C] -> [T, C].
    Parity: pinned (see tests)."""
    return X.sum(dim=1)


STACK_WEIGHTS = ("conv_w", "W_r", "W_pre", "W_res", "W_post", "alpha", "b_pre", "b_res", "b_post")


def stack_objective(X0, layers, G_out, *, S, round_state=True):
    """L = <G_out, stream_sum(X_L)> after L sublayers chained on one state,
    float64.  Sublayer l reads the state sublayer l - 1 wrote (Alg. "Forward
    pass of one xHC sublayer" per layer); with ``round_state`` each written
    state is rounded to bfloat16, the stored precision.

    layers[l] is a dict of STACK_WEIGHTS (weights already the bf16 operand
    values; conv_w None for K_r = 1), 'fn' (callable: dense-read input [T, C]
    -> sublayer output [T, C]) and the shape keys m, k, Kr, kappa and
    optionally router, gram_schmidt_on.  Returns (L, per-layer forward dicts,
    reduced output).
    """
    X = X0
    fwds = []
    for lay in layers:
        X, fwd = sublayer_forward(
            X, lay["fn"], lay["conv_w"], lay["W_r"], lay["W_pre"], lay["W_res"], lay["W_post"], lay["alpha"],
            lay["b_pre"], lay["b_res"], lay["b_post"], m=lay["m"], k=lay["k"], Kr=lay["Kr"], S=S,
            kappa=lay.get("kappa", (4, 8, 12)), router=lay.get("router", "sigmoid"),
            gram_schmidt_on=lay.get("gram_schmidt_on", True))
        if round_state:
            X = round_state_bf16(X)
        fwds.append(fwd)
    out = stream_sum(X)
    return (G_out.to(F64) * out).sum(), fwds, out


def stack_grads(X0, layers, G_out, *, S, round_state=True):
    """Gradients of stack_objective with respect to the entry state and every
    layer's weights (reverse mode of the forward; routing piecewise constant).
    Returns (dX0, list of per-layer dicts keyed by STACK_WEIGHTS, forward
    dicts, reduced output).  Parity: pinned by central differences (tests)."""
    leaf = lambda t: None if t is None else torch.as_tensor(t).detach().to(F64).clone().requires_grad_(True)
    X0l = leaf(X0)
    lays = []
    for lay in layers:
        q = dict(lay)
        for n in STACK_WEIGHTS:
            q[n] = leaf(lay[n])
        lays.append(q)
    L, fwds, out = stack_objective(X0l, lays, G_out, S=S, round_state=round_state)
    leaves = [X0l] + [q[n] for q in lays for n in STACK_WEIGHTS if q[n] is not None]
    grads = torch.autograd.grad(L, leaves, allow_unused=True)
    grads = [torch.zeros_like(v) if g is None else g for g, v in zip(grads, leaves)]
    it = iter(grads[1:])
    per = [{n: (next(it) if q[n] is not None else None) for n in STACK_WEIGHTS} for q in lays]
    return grads[0], per, fwds, out.detach()


GRAD_NAMES = ("X", "F", "W_r", "W_pre", "W_res", "W_post", "alpha", "b_pre", "b_res",
              "b_post", "conv_w")


def xhc_sublayer_grads(X, F, conv_w, W_r, W_pre, W_res, W_post, alpha, b_pre, b_res,
                       b_post, G_X, G_in, **kw):
    """Gradients of sublayer_objective with respect to every input.

    The sublayer output F stands in as an independent input.  The routing
    decision is piecewise constant, so gradients reach the router only
    through p of the routed slots (Sec. "Infrastructure Design").  Weights
    enter as their bf16 operand values and their gradients are taken with
    respect to those values.  The derivative is the plain definition
    (reverse mode of the forward); the tests pin it by central finite
    differences.  Returns a dict of float64 gradients keyed by GRAD_NAMES
    (conv_w is None for K_r = 1) plus the forward results and the loss.
    """
    leaf = lambda t: torch.as_tensor(t).detach().to(F64).clone().requires_grad_(True)
    vals = [leaf(X), leaf(F), leaf(conv_w) if conv_w is not None else None,
            leaf(bf16_operand(W_r)), leaf(bf16_operand(W_pre)),
            leaf(bf16_operand(W_res)), leaf(bf16_operand(W_post)),
            leaf(alpha), leaf(b_pre), leaf(b_res), leaf(b_post)]
    L, fwd = sublayer_objective(*vals, G_X, G_in, **kw)
    order = [0, 1, 3, 4, 5, 6, 7, 8, 9, 10] + ([2] if conv_w is not None else [])
    leaves = [vals[i] for i in order]
    grads = torch.autograd.grad(L, leaves, allow_unused=True)
    # an input the loss does not reach (W_r when every slot is fixed) has zero gradient
    grads = [torch.zeros_like(v) if gr is None else gr for gr, v in zip(grads, leaves)]
    out = dict(zip(GRAD_NAMES, grads))
    if conv_w is None:
        out["conv_w"] = None
    out.update({k_: (v.detach() if torch.is_tensor(v) else v) for k_, v in fwd.items()})
    out["loss"] = L.detach()
    return out


# --------------------------------------------------------------------------
# xHC-Flash backward (reverse mode of the group forward)
# --------------------------------------------------------------------------

def flash_forward(X0, F_list, conv_w_list, W_r, W_pre_list, W_post_list, W_res, alpha_pre, b_pre,
                  alpha_post, b_post, alpha_res, b_res, *, m, k, S, kappa=(4, 8, 12), eps=1e-5,
                  sinkhorn_iters=20, clamp_delta=1e-6, round_state=True, gram_schmidt_on=True,
                  router="sigmoid", tokens=None):
    """One xHC-Flash sharing group, float64, with every weight taken as given
    (already the bf16 operand values) so that it can be differentiated.

    Same steps as xhc_flash_group (Alg. "xHC-Flash: one Transformer block";
    eq:flash_dual_read, eq:flash_attn_update, App. E.2 eq:app_four_sub_base,
    eq:app_general_writeback, eq:app_active_state_correction): one routing
    and Q pre-maps from the entry state X0; sublayers q < Q add
    p (H^post,q out_aug^(q)) to the active rows, the last applies H^res
    first; the input of sublayer q + 1 is its non-active base readout plus
    the pre-map weights of the active streams on the updated active rows;
    H^post,q+1 (and H^res before the last sublayer) come from the updated
    active rows.  The routing decision is taken on detached logits
    (piecewise constant); p is the score of the routed stream.  With
    ``round_state`` each written active row passes through a bfloat16
    rounding, which the reverse mode treats as the identity (the stored
    state is what the next step reads).  With ``tokens`` (positions in the
    batch), X0 holds only those tokens' states while every F is the whole
    batch: each step is per token except the causal convolutions, which
    read the same sequence's earlier F rows.  Returns (X after the group,
    list of the Q inputs, dict of idx, p, Hpre [Q,T,N], Hpost list, Hres and
    acts, the active rows before each sublayer).
    """
    Q = len(F_list)
    T, N, C = X0.shape
    x = X0.reshape(T, N * C)
    z_r = layer_norm(x, eps) @ W_r
    xr = rms_norm(x, eps)
    Hpre = torch.stack([sigmoid(alpha_pre[q] * (xr @ W_pre_list[q]) + b_pre[q]) for q in range(Q)])
    idx, _, gap = route(z_r.detach(), m, k, router)
    s = router_scores(z_r, router)
    p = torch.ones(T, k, dtype=F64)
    if k > m:
        p = torch.cat([p[:, :m], torch.gather(s, 1, idx[:, m:])], dim=1)
    active = torch.zeros(T, N, dtype=torch.bool)
    active[torch.arange(T)[:, None], idx] = True
    keep = (~active).to(F64)
    ar = torch.arange(T)[:, None]

    def post_from(a, q):
        Kq = W_post_list[q].shape[1] // k
        return post_mapping(rms_norm(a.reshape(T, k * C), eps) @ W_post_list[q], alpha_post[q], b_post[q], k, Kq)

    def res_from(a):
        return residual_mapping(rms_norm(a.reshape(T, k * C), eps) @ W_res, alpha_res, b_res, k,
                                sinkhorn_iters, clamp_delta)

    if tokens is None:
        tokens = torch.arange(T)
    inputs = [torch.einsum("tn,tnc->tc", Hpre[0], X0)]
    a = gather_rows(X0, idx)
    acts = [a]
    Hpost = [post_from(a, 0)]
    Hres = res_from(a) if Q == 1 else None
    for q in range(Q):
        comps = augmented_output(F_list[q], conv_w_list[q], kappa, S, tokens, gram_schmidt_on)
        wb = sum(Hpost[q][:, :, r, None] * comps[r][:, None, :] for r in range(len(comps)))
        if q < Q - 1:
            a_new = a + p[:, :, None] * wb
        else:
            a_new = torch.einsum("tjl,tlc->tjc", Hres, a) + p[:, :, None] * wb
        if round_state:
            a_new = a_new + (round_state_bf16(a_new.detach()) - a_new.detach())
        if q < Q - 1:
            hsel = torch.gather(Hpre[q + 1], 1, idx)
            base = torch.einsum("tn,tnc->tc", Hpre[q + 1] * keep, X0)
            inputs.append(base + (hsel[:, :, None] * a_new).sum(1))
            Hpost.append(post_from(a_new, q + 1))
            if q + 1 == Q - 1:
                Hres = res_from(a_new)
            acts.append(a_new)
        a = a_new
    Xn = X0.clone()
    Xn[ar, idx] = a
    return Xn, inputs, dict(idx=idx, p=p, gap=gap, Hpre=Hpre, Hpost=Hpost, Hres=Hres, acts=acts, z_r=z_r)


def flash_objective(vals, G_X, G_in_list, **kw):
    """L = <G_X, X after the group> + sum_q <G_in_q, input_q> for one
    xHC-Flash group (see flash_forward); ``vals`` holds the leaves named in
    FLASH_GRAD_NAMES.  Returns (L, forward dict)."""
    Xn, inputs, fwd = flash_forward(vals["X"], vals["F_list"], vals["conv_w_list"], vals["W_r"],
                                    vals["W_pre_list"], vals["W_post_list"], vals["W_res"], vals["alpha_pre"],
                                    vals["b_pre"], vals["alpha_post"], vals["b_post"], vals["alpha_res"],
                                    vals["b_res"], **kw)
    L = (G_X.to(F64) * Xn).sum()
    for g, inp in zip(G_in_list, inputs):
        L = L + (g.to(F64) * inp).sum()
    fwd["X_new"], fwd["inputs"] = Xn, inputs
    return L, fwd


FLASH_GRAD_NAMES = ("X", "F_list", "conv_w_list", "W_r", "W_pre_list", "W_post_list", "W_res", "alpha_pre",
                    "b_pre", "alpha_post", "b_post", "alpha_res", "b_res")


def flash_leaves(X0, F_list, conv_w_list, W_r, W_pre_list, W_post_list, W_res, alpha_pre, b_pre, alpha_post,
                 b_post, alpha_res, b_res):
    """float64 copies of a group's inputs, the projection weights rounded to
    their bf16 operand values; lists stay lists, None stays None."""
    def one(t, op=False):
        if t is None:
            return None
        t = torch.as_tensor(t)
        return (bf16_operand(t) if op else t.to(F64)).detach().clone()
    return {"X": one(X0), "F_list": [one(f) for f in F_list], "conv_w_list": [one(c) for c in conv_w_list],
            "W_r": one(W_r, True), "W_pre_list": [one(w, True) for w in W_pre_list],
            "W_post_list": [one(w, True) for w in W_post_list], "W_res": one(W_res, True),
            "alpha_pre": one(torch.as_tensor(alpha_pre, dtype=F64)), "b_pre": [one(b) for b in b_pre],
            "alpha_post": one(torch.as_tensor(alpha_post, dtype=F64)), "b_post": [one(b) for b in b_post],
            "alpha_res": one(torch.as_tensor(alpha_res, dtype=F64)), "b_res": one(b_res)}


def flash_group_grads(vals, G_X, G_in_list, wrt=FLASH_GRAD_NAMES, **kw):
    """Gradients of flash_objective with respect to the entries of ``vals``
    named in ``wrt`` (as made by flash_leaves; the others are held constant
    and get None): the reverse mode of the group forward, the routing
    decision piecewise constant.  Returns (dict of gradients with the
    structure of vals, forward dict, loss).  Parity: pinned by central
    differences (tests)."""
    leaves, paths = [], []
    lv = {}
    for name in FLASH_GRAD_NAMES:
        v = vals[name]
        if name not in wrt:
            lv[name] = v
            continue
        if isinstance(v, list):
            lv[name] = []
            for i, t in enumerate(v):
                if t is None:
                    lv[name].append(None)
                    continue
                t = t.detach().clone().requires_grad_(True)
                lv[name].append(t)
                leaves.append(t)
                paths.append((name, i))
        else:
            t = v.detach().clone().requires_grad_(True)
            lv[name] = t
            leaves.append(t)
            paths.append((name, None))
    L, fwd = flash_objective(lv, G_X, G_in_list, **kw)
    grads = torch.autograd.grad(L, leaves, allow_unused=True)
    out = {n: ([None] * len(vals[n]) if isinstance(vals[n], list) else None) for n in FLASH_GRAD_NAMES}
    out.update({n: None for n in FLASH_GRAD_NAMES if n not in wrt})
    for (name, i), g, t in zip(paths, grads, leaves):
        g = torch.zeros_like(t) if g is None else g
        if i is None:
            out[name] = g
        else:
            out[name][i] = g
    fwd = {k_: (v.detach() if torch.is_tensor(v) else v) for k_, v in fwd.items()}
    return out, fwd, L.detach()

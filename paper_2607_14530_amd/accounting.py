"""Per-token memory-traffic and parameter accounting.

Two yardsticks:

* ``paper_table4_*`` rebuild the per-operation element counts of the
  paper's per-token memory-access table (Sec. "Efficiency Analysis",
  Table "Per-token memory access of residual-stream operations") so that its
  totals (34C, 130C, 73.5C, 51C, 40C) can be set beside measured traffic.
* ``algorithmic_bytes_*`` count the bytes each entry point of this library
  must read and write by its contract (every distinct tensor once), the
  figure the roofline fraction is taken against.

``param_count_*`` rebuild eq:xhc_params / eq:mhc_params from the weight
shapes used by the library.
"""

from __future__ import annotations


# ---------------------------------------------------------------- paper table

def paper_table4_mhc(N: int):
    """(reads, writes) in units of C per token for dense mHC (O(N^2) scalars dropped)."""
    ops = {
        "mapping generation": (N, 0),
        "pre dense read": (N, 1),
        "residual mixing": (N, N),
        "post write-back": (1, N),
        "merge and scatter": (2 * N, N),
    }
    return sum(r for r, _ in ops.values()), sum(w for _, w in ops.values())


def _xhc_sublayer(N, k, Kr):
    ops = {
        "mapping generation": (N, 0),
        "pre dense read": (N, 1),
        "gather active": (k, k),
        "active mapping generation": (k, 0),
        "residual mixing": (k, k),
        "post write-back": (Kr, k),
        "merge and scatter": (2 * k, k),
    }
    return sum(r for r, _ in ops.values()), sum(w for _, w in ops.values())


def paper_table4_xhc(N: int, k: int, Kr_mlp: int = 4):
    """Average per sublayer over one attention (K_r = 1) + MLP (K_r = Kr_mlp) block.

    The MLP sublayer also pays the temporal-augmentation kernel (C read,
    3C written, table footnote).
    """
    ra, wa = _xhc_sublayer(N, k, 1)
    rm, wm = _xhc_sublayer(N, k, Kr_mlp)
    rm, wm = rm + 1, wm + (Kr_mlp - 1)
    return (ra + rm) / 2, (wa + wm) / 2


def paper_table4_flash(N: int, k: int, Q: int, Kr_mlp: int = 4):
    """Per-sublayer average for xHC-Flash (Q = 2) or xHC-Flash-4sub (Q = 4).

    Once per group: the joint mapping generation (NC read), the joint dense
    read (NC read, Q readouts written), the gather (kC R/W) and one residual
    mixing (kC R/W).  Per sublayer: active mapping generation (kC read),
    post write-back (K_q C read, kC written), merge and scatter (2kC read,
    kC written).  Per MLP sublayer: the conv (C read, 3C written).  Per
    later sublayer: the input correction (2C read, C written).
    """
    r = N + N + k + k
    w = Q + k + k
    for q in range(1, Q + 1):
        Kq = 1 if q % 2 == 1 else Kr_mlp
        r += k + Kq + 2 * k
        w += k + k
        if Kq > 1:
            r += 1
            w += Kq - 1
        if q > 1:
            r += 2
            w += 1
    return r / Q, w / Q


# ---------------------------------------------------------------- this library

def coef_floats(N: int, k: int, Kr: int) -> int:
    """fp32/int32 words per token written by the pre step: idx, p, H^pre, H^res, H^post."""
    return k + k + N + k * k + k * Kr


def algorithmic_bytes_pre(N, k, C, Kr, state_bytes=2):
    """xhc_pre: read the state once, write the input and the coefficients."""
    return N * C * state_bytes + C * state_bytes + 4 * coef_floats(N, k, Kr)


def algorithmic_bytes_post(N, k, C, Kr, state_bytes=2):
    """xhc_post: read k rows and F, write k rows; read idx, p, H^res, H^post."""
    return (2 * k + 1) * C * state_bytes + 4 * (k + k + k * k + k * Kr)


def algorithmic_bytes_sublayer(N, k, C, Kr, state_bytes=2):
    return algorithmic_bytes_pre(N, k, C, Kr, state_bytes) + algorithmic_bytes_post(N, k, C, Kr, state_bytes)


def algorithmic_bytes_flash_pre(N, k, C, Q, Kq0=1, state_bytes=2):
    """xhc_flash_pre: read the state once; write input^(1) and Q-1 bases, idx, p,
    Q pre-maps and the first sublayer's post-map."""
    return (N * C + Q * C) * state_bytes + 4 * (k + k + Q * N + k * Kq0)


def algorithmic_bytes_flash_post(N, k, C, Kq, last, Kq_next=0, state_bytes=2):
    """xhc_flash_post for one sublayer: k rows R/W, F R; for a non-last sublayer also
    the next base R and next input W and the next coefficient outputs."""
    b = (2 * k + 1) * C * state_bytes + 4 * (k + k * Kq)
    if last:
        b += 4 * k * k
    else:
        b += 2 * C * state_bytes + 4 * (N + k * Kq_next)
    return b


# ---------------------------------------------------------------- parameters

def param_count_xhc_layer(N: int, k: int, Kr: int, kappa, C: int) -> int:
    """Parameters of one layer (attention + MLP sublayer) from the weight shapes.

    Each sublayer: W_r [NC, N], W_pre [NC, N], W_res [kC, k^2]; post [kC, k*K]
    with K = 1 (attention) or Kr (MLP); conv kernels [sum kappa, C] on MLP.
    Gating scalars and biases are O(N^2), not counted (as in eq:xhc_params).
    """
    per = 2 * (N * C) * N + (k * C) * (k * k)
    return 2 * per + (k * C) * (k * 1) + (k * C) * (k * Kr) + sum(kappa) * C


def param_count_mhc_layer(N: int, C: int) -> int:
    """Dense mHC: W_pre, W_post [NC, N], W_res [NC, N^2] on both sublayers."""
    return 2 * ((N * C) * N * 2 + (N * C) * (N * N))

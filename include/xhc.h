/*
 * xhc.h - C ABI of the MI355X (gfx950) implementation of the xHC per-sublayer
 * residual-stream connection (xHC: Expanded Hyper-Connections, arXiv
 * 2607.14530), in its full xHC and xHC-Flash forms.
 *
 * Notation follows the paper: T tokens (token t = b*S + s, S tokens per
 * sequence), N residual streams of width C, k active streams of which m are
 * fixed, K_r write-back components (1 for attention-type sublayers, 1 + r for
 * MLP-type sublayers with r causal depthwise convolutions), Q sublayers per
 * xHC-Flash sharing group.
 *
 * Conventions for every entry point:
 *  - All tensor pointers are DEVICE pointers owned by the caller; the library
 *    never allocates or frees memory inside a call.  `workspace` is caller
 *    device memory of at least xhc_workspace_bytes() bytes, 16-byte aligned
 *    (hipMalloc gives 256); its contents on entry are ignored and on return
 *    are unspecified.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).  Calls
 *    are asynchronous on that stream and enqueue device work only.
 *  - Layouts are row-major and contiguous: X [T,N,C]; F, input [T,C];
 *    idx [T,k] int32; p [T,k]; Hpre [T,N]; Hres [T,k,k]; Hpost [T,k,K].
 *    The state X and the tensors F, input and base use `state_dtype`
 *    (bf16 or fp32); coefficients are fp32.
 *  - Slot order of idx (reading of eq:router_topk): slots 0..m-1 hold the
 *    fixed streams 0..m-1 with p = 1; slots m..k-1 hold the routed streams in
 *    descending router logit, ties to the lower stream index.
 *  - Errors: arguments are validated before any device work is enqueued, so
 *    an error return leaves every output untouched.  XHC_EINVAL: violated
 *    constraint or NULL required pointer; XHC_EUNSUPPORTED: valid shape this
 *    library does not implement; XHC_EWORKSPACE: workspace too small;
 *    XHC_EHIP: a HIP launch failed (outputs unspecified).
 *  - Thread safety: the library holds no mutable global state (apart from a
 *    per-device cache of the scratch address of xhc_post_noalloc); calls on
 *    different streams may overlap provided their buffers do not.
 */
#ifndef XHC_H_
#define XHC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  XHC_OK = 0,
  XHC_EINVAL = 1,
  XHC_EUNSUPPORTED = 2,
  XHC_EWORKSPACE = 3,
  XHC_EHIP = 4
} xhc_status;

typedef enum { XHC_BF16 = 0, XHC_F32 = 1 } xhc_dtype;

/* Shape and hyperparameters of one sublayer connection (Sec. "Parameterization
 * Details" and the hyperparameter table: N = 16, k = 4, m = 2, r = 3,
 * kappa = {4, 8, 12}, 20 Sinkhorn iterations).  Constraints:
 *   T >= 0, S >= 1, T % S == 0;  1 <= k <= N <= 64;  0 <= m <= k;  k <= 8;
 *   C >= 32, C % 32 == 0;  Kr in 1..4;  kappa[j] in 1..16 for j < Kr - 1;
 *   sinkhorn_iters in 0..1000;  eps > 0;  clamp_delta >= 0;  router 0 or 1;
 *   attn_aug 0 or 1.                                                         */
typedef struct xhc_dims {
  int64_t T;              /* tokens                                              */
  int64_t S;              /* tokens per sequence (causal conv window resets)     */
  int32_t N;              /* residual streams                                    */
  int32_t k;              /* active streams                                      */
  int32_t m;              /* fixed (always active) streams                       */
  int32_t C;              /* width                                               */
  int32_t Kr;             /* write-back components of an MLP-type sublayer       */
  int32_t kappa[3];       /* conv kernel sizes of the Kr - 1 branches            */
  int32_t sinkhorn_iters; /* Sinkhorn iterations (row then column normalisation) */
  int32_t gram_schmidt;   /* 1: orthogonalise the components (eq:gs); 0: skip    */
  float eps;              /* epsilon of the LayerNorm / RMSNorm statistics       */
  float clamp_delta;      /* row clamp applies when a row sum exceeds 1 + delta  */
  int32_t state_dtype;    /* xhc_dtype of X, F, input, base                      */
  int32_t impl;           /* xhc_impl: which kernels run (same results)          */
  int32_t router;         /* xhc_router: score function of the router            */
  int32_t attn_aug;       /* xHC-Flash groups: 0 = attention-type sublayers have */
                          /* one write-back component (the paper's design); 1 =  */
                          /* they get the Kr components of the temporal          */
                          /* augmentation too (the attention-side ablation)      */
} xhc_dims;

/* Router score function.  SIGMOID is eq:router; SOFTMAX is the ablation of
 * the ablation table (row 11): a softmax over all N router logits of a token.
 * Both are monotone, so TopK selects the same streams; p of a routed slot is
 * the stream's score.                                                      */
typedef enum { XHC_ROUTER_SIGMOID = 0, XHC_ROUTER_SOFTMAX = 1 } xhc_router;

/* Kernel selection for xhc_pre.  AUTO takes the single-pass cooperative
 * kernel where it applies (bf16 state, N = 16, k = 4, C = 128 G with G
 * dividing 32) and the multi-kernel path elsewhere, or when the device cannot
 * hold the single-pass grid.  MULTI forces the multi-kernel path.  FUSED
 * forces the single-pass kernel and returns XHC_EUNSUPPORTED where it does
 * not apply.  All give the same results within rounding.  If a wait of the
 * single-pass kernel ever gives up (bounded spin), H^post and H^res come out
 * as NaN rather than as silently wrong values.                              */
typedef enum { XHC_IMPL_AUTO = 0, XHC_IMPL_MULTI = 1, XHC_IMPL_FUSED = 2 } xhc_impl;

/* Name of a status code, and the name of the HIP error behind the last
 * XHC_EHIP returned on the calling thread (static strings).               */
const char* xhc_status_string(int32_t status);
const char* xhc_last_hip_error(void);

/* ------------------------------------------------------------------ packing
 * Projection operands are bf16 (Sec. "Infrastructure Design"): the packers
 * round fp32 weights to bf16 (nearest even) into an opaque device layout used
 * by the projection kernels.  Sizes come from the *_bytes queries.
 *
 * Full-state projection (eq:fused_normalized_projection): columns are
 * [W_r | W_pre,1 | ... | W_pre,npre], W_r and each W_pre [N*C, N] fp32 with
 * row index i*C + c (stream-major flatten).  Full xHC uses npre = 1;
 * xHC-Flash uses npre = Q.  W_pre points at npre contiguous matrices.
 * Also stores the column sums of bf16(W_r) used by the LayerNorm correction.
 *
 * Active projection (Sec. "Infrastructure Design", [W^post, W^res]): columns
 * [W_post | W_res], W_post [k*C, k*Kq] and W_res [k*C, k*k] (may be NULL when
 * the sublayer has no residual mixing), row index j*C + c (slot-major vec).  */
size_t xhc_packed_full_bytes(const xhc_dims* d, int32_t npre);
size_t xhc_packed_active_bytes(const xhc_dims* d, int32_t Kq, int32_t with_res);
xhc_status xhc_pack_full(const xhc_dims* d, int32_t npre, const float* W_r, const float* W_pre,
                         void* packed, void* stream);
xhc_status xhc_pack_active(const xhc_dims* d, int32_t Kq, const float* W_post, const float* W_res,
                           void* packed, void* stream);

/* Workspace needed by an entry point (op: one of the XHC_OP_* values).        */
enum {
  XHC_OP_PRE = 0, XHC_OP_POST = 1, XHC_OP_FLASH_PRE = 2, XHC_OP_FLASH_POST = 3,
  XHC_OP_POST_BWD = 4, XHC_OP_PRE_BWD = 5, XHC_OP_FLASH_POST_BWD = 6, XHC_OP_FLASH_PRE_BWD = 7
};
size_t xhc_workspace_bytes(const xhc_dims* d, int32_t op, int32_t Q);

/* ------------------------------------------------------------------ full xHC
 * xhc_pre - mapping generation and dense read of one xHC sublayer
 * (Alg. "Forward pass of one xHC sublayer", routing / mapping-generation / dense
 * read steps; eq:router, eq:router_topk, eq:param_pre, eq:dense_read,
 * eq:param_res, eq:param_post, row clamp of App. A).
 *   X          [T,N,C] state (read only)
 *   packed_full  xhc_pack_full(npre = 1) of W_r, W_pre
 *   packed_act   xhc_pack_active(Kq = d->Kr, with_res = 1) of W_post, W_res
 *   alpha      [3] fp32 device: alpha_pre, alpha_res, alpha_post
 *   b_pre [N], b_res [k*k], b_post [k*Kr] fp32 device
 * Outputs: input [T,C] (state dtype), idx [T,k], p [T,k], Hpre [T,N],
 * Hres [T,k,k], Hpost [T,k,Kr].  Uses d->Kr as this sublayer's K_r.          */
xhc_status xhc_pre(const xhc_dims* d, const void* X, const void* packed_full, const void* packed_act,
                   const float* alpha, const float* b_pre, const float* b_res, const float* b_post,
                   void* input, int32_t* idx, float* p, float* Hpre, float* Hres, float* Hpost,
                   float* saved, void* workspace, size_t workspace_bytes, void* stream);

/* xhc_pre_failures - waits until the work enqueued on `stream` so far has
 * finished, then sets *failures to the number of bounded waits that gave up
 * in the last xhc_pre call that used `workspace` (that call's own workspace
 * pointer).  The single-pass kernel's members exchange partial sums through
 * device memory and every wait on another member is bounded; a wait that
 * gives up leaves NaN in H^post and H^res, and this count says that it
 * happened.  The multi-kernel path has no such waits and reports 0.
 * Errors: XHC_EINVAL (NULL pointer), XHC_EUNSUPPORTED (workspace not 16-byte
 * aligned), XHC_EHIP (the copy or the synchronisation failed).            */
xhc_status xhc_pre_failures(const void* workspace, int32_t* failures, void* stream);

/* Floats per token that xhc_pre writes to `saved` when it is non-NULL (for
 * xhc_pre_bwd): [z_r (N) | z_pre (N) | z_post, z_res (k*Kr + k*k) | mu | nu |
 * nu_a | pad], z = the normalised logits before gating, mu / nu = mean and
 * mean square of the flattened state, nu_a = mean square of the active rows.
 * Both xhc_pre implementations write it.                                   */
size_t xhc_saved_floats(const xhc_dims* d);

/* xhc_post - sparse write-back of one xHC sublayer (eq:aug, eq:gs,
 * eq:sparse_write_delta, eq:sparse_write; Alg. "Forward pass of one xHC
 * sublayer", write-back and scatter steps).
 *   X       [T,N,C] in/out: only rows X[t, idx[t,j], :] are written, each to
 *           sum_l Hres[t,j,l] X[t,idx[t,l],:] + p[t,j] sum_r Hpost[t,j,r] v_r[t]
 *   F       [T,C] sublayer output (must not alias X)
 *   conv_w  [sum_{j<Kr-1} kappa[j], C] fp32 (branch kernels stacked, row i of
 *           branch j multiplies F[t-i]); NULL iff d->Kr == 1
 *   idx, p, Hres, Hpost as produced by xhc_pre.
 *   Xact_save  [T,k,C] or NULL: receives the active rows before the update
 *           (slot order), as xhc_post_bwd needs them.                          */
xhc_status xhc_post(const xhc_dims* d, void* X, const void* F, const float* conv_w,
                    const int32_t* idx, const float* p, const float* Hres, const float* Hpost,
                    void* Xact_save, void* workspace, size_t workspace_bytes, void* stream);

/* xhc_post_noalloc - xhc_post for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and errors as xhc_post, without the
 * workspace: the MLP-type write-back's scratch (Gram partials and write-back
 * weights, xhc_workspace_bytes(d, XHC_OP_POST, 0) bytes) lives in a static
 * device array of XHC_NOALLOC_SCRATCH_BYTES that every GPU the library runs
 * on holds until the process ends.  The call allocates nothing.  Shapes whose
 * scratch exceeds that size return XHC_EWORKSPACE before any work is
 * enqueued (at C = 4096, K_r = 4: T up to about 72K tokens).  All calls on
 * one GPU share its array: calls that overlap on one GPU (different streams
 * without ordering between them) race and must not be made.            */
#define XHC_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
xhc_status xhc_post_noalloc(const xhc_dims* d, void* X, const void* F, const float* conv_w,
                            const int32_t* idx, const float* p, const float* Hres, const float* Hpost,
                            void* Xact_save, void* stream);

/* ------------------------------------------------------------------ backward
 * Reverse mode of xhc_pre + xhc_post for a loss L(X', input) (X' = state after
 * xhc_post, input = xhc_pre's output).  Routing is piecewise constant: the
 * router receives gradient only through p of the routed slots; Sinkhorn is
 * differentiated through its unrolled iterations (recomputed); projection
 * weights receive the gradient of their bf16 operand values.  Call
 * xhc_post_bwd first (it also gives dL/dF for the sublayer's own backward),
 * then xhc_pre_bwd with dL/d input.
 *
 * xhc_post_bwd
 *   dXn     [T,N,C] dL/dX' (read)
 *   X       [T,N,C] in/out: the state after xhc_post; on return its active rows
 *           are restored from Xact, i.e. X holds the state xhc_pre saw
 *   Xact    [T,k,C] the active rows before the update (xhc_post's Xact_save)
 *   F, conv_w, idx, p, Hres, Hpost as in xhc_post
 * Outputs: dX [T,N,C] = dXn on untouched rows and sum_j Hres[t,j,l] dXn[t,I_j]
 * on active row I_l (xhc_pre_bwd adds the rest).  dX may be dXn itself (in
 * place, the sparse form of eq:sparse_write): then only the k active rows of
 * each token are written and the untouched rows are not moved at all.
 * dF [T,C]; dHres [T,k,k];
 * dHpost [T,k,Kr]; dp [T,k]; dconv_w [sum kappa, C] (NULL iff Kr == 1).
 *
 * xhc_pre_bwd (N in {4, 8, 16, 32}, C % 256 == 0, k*Kr + k*k <= 32)
 *   X           [T,N,C] the state xhc_pre saw (after xhc_post_bwd's restore)
 *   packed_full the packed [W_r | W_pre] of the forward (for sum_K bf16(W_r))
 *   W_r, W_pre [N*C,N], W_res [k*C,k*k], W_post [k*C,k*Kr] fp32 (used as bf16)
 *   alpha [3], b_res [k*k]; saved [T, xhc_saved_floats] from xhc_pre
 *   idx, p, Hpre, Hpost from xhc_pre; d_input [T,C] dL/d input
 *   dHres, dHpost, dp from xhc_post_bwd
 *   dX [T,N,C] in/out: xhc_post_bwd's dX; on return the full dL/dX
 * Outputs (overwritten): dW_r, dW_pre, dW_res, dW_post (shapes of the weights);
 * dalpha [3]; db_pre [N]; db_res [k*k]; db_post [k*Kr].  Weight and bias
 * gradients are summed over tokens in a fixed order (deterministic).       */
xhc_status xhc_post_bwd(const xhc_dims* d, const void* dXn, void* X, const void* Xact, const void* F,
                        const float* conv_w, const int32_t* idx, const float* p, const float* Hres,
                        const float* Hpost, void* dX, void* dF, float* dHres, float* dHpost, float* dp,
                        float* dconv_w, void* workspace, size_t workspace_bytes, void* stream);
xhc_status xhc_pre_bwd(const xhc_dims* d, const void* X, const void* packed_full, const float* W_r,
                       const float* W_pre, const float* W_res, const float* W_post, const float* alpha,
                       const float* b_res, const float* saved, const int32_t* idx, const float* p,
                       const float* Hpre, const float* Hpost, const void* d_input, const float* dHres,
                       const float* dHpost, const float* dp, void* dX, float* dW_r, float* dW_pre, float* dW_res,
                       float* dW_post, float* dalpha, float* db_pre, float* db_res, float* db_post, void* workspace,
                       size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ xHC-Flash
 * A sharing group of Q = 2 or 4 consecutive sublayers (Sec. "xHC-Flash",
 * Alg. "xHC-Flash: one Transformer block", App. E).  Sublayer q (1-based) is
 * attention-type (one write-back component) for odd q and MLP-type (d->Kr
 * components with the temporal augmentation) for even q; with d->attn_aug = 1
 * the attention-type sublayers get the same d->Kr components (the
 * attention-side temporal augmentation of the additional-ablations table).
 * K_q below is the component count of sublayer q.  One routing
 * decision and Q pre-maps come from the group-entry state; intermediate
 * sublayers write the active rows without residual mixing; the last applies
 * H^res.  Later inputs are formed from non-active base readouts plus the
 * active rows as stored (eq:app_four_sub_base, eq:app_active_state_correction).
 *
 * xhc_flash_pre - once per group.
 *   X            [T,N,C] group-entry state (read only)
 *   packed_full  xhc_pack_full(npre = Q) of W_r and the Q matrices W_pre,q
 *   packed_act1  xhc_pack_active(Kq = K_1, W_res = NULL) of W_post,1
 *   alpha_pre [Q], b_pre [Q,N], alpha_post1 [1], b_post1 [k K_1] fp32 device
 * Outputs: input1 [T,C] = sum_i H^pre,1_i x_i; base [Q-1,T,C] where base[q-2] =
 * sum_{i not in I} H^pre,q_i x_i (q = 2..Q); idx, p as in xhc_pre; Hpre [Q,T,N];
 * Hpost1 [T,k,K_1].  saved [Q,T,2N + k + k*k + 4] fp32 or NULL: per pre-map q
 * and token the router logits, the pre-map logits and the norm statistics
 * (the other fields zero), which xhc_flash_pre_bwd then reads instead of
 * recomputing them from X.  saved_act1 [T, 2k + k*K_1 + k*k + 4] fp32 or NULL:
 * per token the logits and the RMS statistic of sublayer 1's H^post (the
 * other fields zero), which xhc_flash_post_bwd(q = 1) reads instead of
 * reprojecting the active rows.                                               */
xhc_status xhc_flash_pre(const xhc_dims* d, int32_t Q, const void* X, const void* packed_full,
                         const void* packed_act1, const float* alpha_pre, const float* b_pre,
                         const float* alpha_post1, const float* b_post1, void* input1, void* base, int32_t* idx,
                         float* p, float* Hpre, float* Hpost1, float* saved, float* saved_act1, void* workspace,
                         size_t workspace_bytes, void* stream);

/* xhc_flash_post - after sublayer q of the group (1 <= q <= Q).
 *   X       [T,N,C] in/out: rows X[t, idx[t,j], :] <- (q == Q ? sum_l Hres[t,j,l]
 *           X[t,idx[t,l],:] : X[t,idx[t,j],:]) + p[t,j] sum_r Hpost[t,j,r] v_r[t]
 *   F       [T,C] output of sublayer q; conv_w as in xhc_post, non-NULL iff K_q > 1
 *   Hpost   [T,k,K_q] of sublayer q; Hres [T,k,k] iff q == Q (else NULL)
 * For q < Q (else all NULL):
 *   Hpre_next [T,N] = Hpre[q] from xhc_flash_pre; base_next [T,C] = base[q-1];
 *   input_next [T,C] out: base_next + sum_j Hpre_next[t, idx[t,j]] X[t, idx[t,j], :]
 *   packed_act_next  xhc_pack_active(K_{q+1}, W_res iff q + 1 == Q) of sublayer q+1
 *   alpha_next [2] = (alpha_post_{q+1}, alpha_res); b_post_next [k*K_{q+1}];
 *   b_res_next [k*k] iff q + 1 == Q; outputs Hpost_next [T,k,K_{q+1}] and
 *   Hres_next [T,k,k] iff q + 1 == Q, both from the updated active rows.
 *   Xact_save [T,k,C] or NULL: receives the active rows before this sublayer's
 *   write-back (slot order), as xhc_flash_post_bwd needs them.
 *   saved_next [T, 2k + k*K_{q+1} + k*k + 4] fp32 or NULL (q < Q only): the
 *   logits and statistic of the next mappings, as saved_act1 for sublayer 1. */
xhc_status xhc_flash_post(const xhc_dims* d, int32_t Q, int32_t q, void* X, const void* F, const float* conv_w,
                          const int32_t* idx, const float* p, const float* Hpost, const float* Hres,
                          const float* Hpre_next, const void* base_next, void* input_next,
                          const void* packed_act_next, const float* alpha_next, const float* b_post_next,
                          const float* b_res_next, float* Hpost_next, float* Hres_next, void* Xact_save,
                          float* saved_next, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------ xHC-Flash backward
 * Reverse mode of one sharing group (xhc_flash_pre, then xhc_flash_post for
 * q = 1..Q) for a loss L(X', input_1 .. input_Q), X' the state after the
 * group.  Routing is piecewise constant (the router gets gradient only
 * through p of routed slots); written rows are taken as stored (their bf16
 * rounding passes the gradient through).  The sweep runs sublayer by
 * sublayer on the active rows a^(q) [T,k,C] (slot order), their gradient
 * held in fp32 between the calls: call
 * xhc_flash_post_bwd for q = Q, Q-1, .., 1 (each may run right after the
 * sublayer's own backward has produced dL/d input_q from dL/dF_q), then
 * xhc_flash_pre_bwd once.  a^(0) = X[idx] is the group-entry active state,
 * a^(q) the active rows after sublayer q.  Supported: k = 4 (or 8 with
 * k K_r + k k <= 32), N in {4, 8, 16, 32}, C % 256 == 0.
 *
 * xhc_flash_post_bwd - sublayer q (1 <= q <= Q)
 *   dXn     [T,N,C] dL/dX' (read), iff q == Q (else NULL): da is then set to
 *           its active rows before the sweep starts
 *   da      [T,k,C] fp32 in/out: on entry dL/da^(q) (ignored when q == Q), on
 *           return dL/da^(q-1) through this sublayer: the write-back reverse
 *           (H^res^T at q == Q, pass-through before), the reverse of H^post,q
 *           (and H^res) computed from a^(q-1) (eq:param_post, eq:param_res),
 *           and for q >= 2 the active part of input_q (H^pre,q_{I_j} d input_q)
 *   Xact    [T,k,C] a^(q-1): xhc_flash_post's Xact_save of sublayer q
 *   F, conv_w (iff q is even), idx, p, Hpost [T,k,K_q], Hres (iff q == Q) as
 *           in the forward; packed_act: the forward's packed [W_post,q | W_res];
 *           W_post [k*C, k*K_q] and W_res [k*C,k*k] (iff q == Q) fp32;
 *           alpha_post [1], b_post [k*K_q]; alpha_res [1], b_res [k*k] iff q == Q
 *   Hpre_q  [T,N] = Hpre[q-1] of xhc_flash_pre and d_input [T,C] = dL/d input_q,
 *           both iff q >= 2 (input_1 is reversed by xhc_flash_pre_bwd)
 *   saved_act  sublayer q's mapping record (saved_act1 of xhc_flash_pre for
 *           q = 1, saved_next of xhc_flash_post q - 1 otherwise) or NULL (the
 *           logits are then recomputed from Xact)
 * Outputs (overwritten): dF [T,C]; dconv_w (iff q is even); dW_post,
 * dalpha_post [1], db_post; dW_res, dalpha_res [1], db_res iff q == Q;
 * dHpre_act [T,k] = <d input_q, a^(q-1)_j> iff q >= 2.  dp [T,k] is
 * accumulated (+=): zero it before the sweep.
 *
 * xhc_flash_pre_bwd - the group-entry state
 *   X [T,N,C] group-entry state; packed_full, W_r [N*C,N], W_pre [Q,N*C,N]
 *   fp32, alpha_pre [Q], b_pre [Q,N] as in the forward; idx, p, Hpre [Q,T,N]
 *   from xhc_flash_pre; d_input [Q,T,C] = dL/d input_q; dHpre_act [Q-1,T,k]
 *   from xhc_flash_post_bwd (q = 2..Q); dp [T,k] the accumulated dp;
 *   dXn [T,N,C] dL/dX'; da0 [T,k,C] fp32 dL/da^(0) (da after the q = 1 reverse)
 * Outputs (overwritten): dX [T,N,C] = dL/dX; dW_r; dW_pre [Q,N*C,N];
 * dalpha_pre [Q]; db_pre [Q,N].  saved: the records xhc_flash_pre wrote for
 * this group, or NULL (they are then recomputed from X, one more read of
 * the state).  dX may be dXn itself (in place): the
 * untouched streams then keep their gradient without a copy and only the k
 * active rows of each token are first overwritten with da0.  Token sums run
 * in a fixed order (deterministic).                                         */
xhc_status xhc_flash_post_bwd(const xhc_dims* d, int32_t Q, int32_t q, const void* dXn, void* da, const void* Xact,
                              const void* F, const float* conv_w, const int32_t* idx, const float* p,
                              const float* Hpost, const float* Hres, const void* packed_act, const float* W_post,
                              const float* W_res, const float* alpha_post, const float* alpha_res,
                              const float* b_post, const float* b_res, const float* Hpre_q, const void* d_input,
                              const float* saved_act, void* dF, float* dconv_w, float* dW_post,
                              float* dalpha_post, float* db_post, float* dW_res, float* dalpha_res, float* db_res,
                              float* dp, float* dHpre_act, void* workspace, size_t workspace_bytes, void* stream);
xhc_status xhc_flash_pre_bwd(const xhc_dims* d, int32_t Q, const void* X, const void* packed_full, const float* W_r,
                             const float* W_pre, const float* alpha_pre, const float* b_pre, const int32_t* idx,
                             const float* p, const float* Hpre, const float* saved, const void* d_input,
                             const float* dHpre_act, const float* dp, const void* dXn, const void* da0, void* dX,
                             float* dW_r, float* dW_pre, float* dalpha_pre, float* db_pre, void* workspace,
                             size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------ final stream reduction
 * App. "Final Stream Reduction": before the last RMSNorm and the unembedding
 * the N streams of each token are summed into one C-vector.
 *
 * xhc_stream_sum: out [T,C] = sum_{i<N} X[t,i,:] (fp32 accumulation over
 *   i ascending, rounded to state_dtype).  Only T, N, C and state_dtype of d
 *   are used.  X, out: 16-byte aligned, not overlapping.
 * xhc_stream_sum_bwd: its backward, dX[t,i,:] = dout[t,:] for every i, or
 *   dX[t,i,:] += dout[t,:] with accumulate = 1 (dX then holds a gradient
 *   already, in state_dtype).  dout, dX: 16-byte aligned, not overlapping.
 * Errors as for every entry point (XHC_EINVAL for NULL pointers or
 * accumulate outside {0, 1}, XHC_EUNSUPPORTED for misaligned pointers).     */
xhc_status xhc_stream_sum(const xhc_dims* d, const void* X, void* out, void* stream);
xhc_status xhc_stream_sum_bwd(const xhc_dims* d, const void* dout, void* dX, int32_t accumulate, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* XHC_H_ */

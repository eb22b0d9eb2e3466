// C ABI of the xHC library: argument validation, workspace sizing, dispatch.
// Every check happens before the first launch, so an error return leaves
// all outputs untouched.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include <algorithm>

#include "xhc.h"
#include "xhc_launch.h"

using namespace xhc;

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// shape constraints shared by every entry point (see xhc_dims in xhc.h)
xhc_status check_dims(const xhc_dims* d) {
  if (!d) return XHC_EINVAL;
  if (d->T < 0 || d->S < 1 || (d->T % d->S) != 0) return XHC_EINVAL;
  if (d->N < 1 || d->k < 1 || d->k > d->N || d->m < 0 || d->m > d->k) return XHC_EINVAL;
  if (d->C < 1 || d->Kr < 1 || d->sinkhorn_iters < 0 || !(d->eps > 0.f) || !(d->clamp_delta >= 0.f))
    return XHC_EINVAL;
  if (d->state_dtype != XHC_BF16 && d->state_dtype != XHC_F32) return XHC_EINVAL;
  if (d->impl < XHC_IMPL_AUTO || d->impl > XHC_IMPL_FUSED) return XHC_EINVAL;
  if (d->router != XHC_ROUTER_SIGMOID && d->router != XHC_ROUTER_SOFTMAX) return XHC_EINVAL;
  if (d->N > kMaxN || d->k > kMaxK || d->Kr > kMaxKr || d->sinkhorn_iters > 1000) return XHC_EUNSUPPORTED;
  if (d->C % 32 != 0) return XHC_EUNSUPPORTED;
  for (int j = 0; j < d->Kr - 1; ++j)
    if (d->kappa[j] < 1 || d->kappa[j] > 16) return XHC_EUNSUPPORTED;
  return XHC_OK;
}

thread_local hipError_t g_last_hip_error = hipSuccess;
thread_local const char* g_failed_step = "";
thread_local char g_error_text[160];

// run one launcher unless an earlier one failed; remember which one failed
#define XHC_STEP(name, call)              \
  do {                                    \
    if (e == hipSuccess) {                \
      e = (call);                         \
      if (e != hipSuccess) g_failed_step = name; \
    }                                     \
  } while (0)

xhc_status hip_status(hipError_t e) {
  if (e == hipSuccess) return XHC_OK;
  g_last_hip_error = e;
  return XHC_EHIP;
}

// A runtime error left by an unrelated earlier call on this thread would be
// reported by the first hipGetLastError() after our launch; clear it first.
void clear_stale_error() { (void)hipGetLastError(); }

int64_t NC_of(const xhc_dims* d) { return (int64_t)d->N * d->C; }
int64_t kC_of(const xhc_dims* d) { return (int64_t)d->k * d->C; }
int64_t act_outs(const xhc_dims* d, int Kq, int with_res) { return (int64_t)d->k * Kq + (with_res ? d->k * d->k : 0); }

size_t part_bytes(const xhc_dims* d, bool gather, int64_t K, int64_t nout) {
  return align_up((size_t)proj_chunks(d->state_dtype, gather, K, d->C, nout, d->T) * (size_t)(out_blocks(nout) * 16 + 2) *
                  (size_t)d->T * sizeof(float));
}

// partials of the larger projection, then the per-token sums of either one
size_t sums_bytes(int64_t nout, int64_t T) { return align_up((size_t)(out_blocks(nout) * 16 + 2) * T * sizeof(float)); }

size_t pre_ws_multi(const xhc_dims* d) {
  const size_t full = part_bytes(d, false, NC_of(d), 2 * d->N);
  const size_t act = part_bytes(d, true, kC_of(d), act_outs(d, d->Kr, 1));
  const size_t sf = sums_bytes(2 * d->N, d->T), sa = sums_bytes(act_outs(d, d->Kr, 1), d->T);
  return (full > act ? full : act) + (sf > sa ? sf : sa);
}

// The single-pass path may fall back to the multi-kernel path at run time
// (device too small for its grid), so AUTO sizes for both.
size_t pre_ws(const xhc_dims* d) {
  size_t need = 0;
  if (d->impl != XHC_IMPL_FUSED) need = pre_ws_multi(d);
  if (d->impl != XHC_IMPL_MULTI && fused_pre_supported(d)) {
    const size_t f = fused_pre_ws_bytes(d);
    need = need > f ? need : f;
  }
  return need;
}

// write-back components of sublayer q (1-based) of an xHC-Flash group:
// attention-type (odd q) has one, MLP-type (even q) has d->Kr
int flash_Kq(const xhc_dims* d, int q) { return (q % 2 == 1) ? 1 : d->Kr; }

size_t flash_pre_ws(const xhc_dims* d, int Q) {
  const int64_t nf = (int64_t)(Q + 1) * d->N, na = act_outs(d, 1, 0);
  const size_t full = part_bytes(d, false, NC_of(d), nf), act = part_bytes(d, true, kC_of(d), na);
  const size_t sf = sums_bytes(nf, d->T), sa = sums_bytes(na, d->T);
  return (full > act ? full : act) + (sf > sa ? sf : sa);
}

size_t gram_bytes(const xhc_dims* d, int Kq) {
  const int np = Kq * (Kq + 1) / 2;
  return align_up((size_t)gram_chunks(d->C, d->S, Kq, d->kappa) * np * (size_t)d->T * sizeof(float)) +
         align_up((size_t)d->T * d->k * Kq * sizeof(float));
}

size_t flash_post_ws(const xhc_dims* d, int Q, int q) {
  const int Kq = flash_Kq(d, q);
  size_t need = Kq > 1 ? gram_bytes(d, Kq) : 0;
  if (q < Q) {
    const int64_t na = act_outs(d, flash_Kq(d, q + 1), q + 1 == Q);
    need = std::max(need, part_bytes(d, true, kC_of(d), na) + sums_bytes(na, d->T));
  }
  return need;
}

size_t post_ws(const xhc_dims* d) {
  if (d->Kr == 1) return 0;
  const int np = d->Kr * (d->Kr + 1) / 2;
  return align_up((size_t)gram_chunks(d->C, d->S, d->Kr, d->kappa) * np * (size_t)d->T * sizeof(float)) +
         align_up((size_t)d->T * d->k * d->Kr * sizeof(float));
}

}  // namespace

extern "C" {

const char* xhc_status_string(int32_t status) {
  switch (status) {
    case XHC_OK: return "XHC_OK";
    case XHC_EINVAL: return "XHC_EINVAL";
    case XHC_EUNSUPPORTED: return "XHC_EUNSUPPORTED";
    case XHC_EWORKSPACE: return "XHC_EWORKSPACE";
    case XHC_EHIP: return "XHC_EHIP";
    default: return "unknown xhc_status";
  }
}

const char* xhc_last_hip_error(void) {
  snprintf(g_error_text, sizeof(g_error_text), "%s in %s", hipGetErrorName(g_last_hip_error), g_failed_step);
  return g_error_text;
}

size_t xhc_packed_full_bytes(const xhc_dims* d, int32_t npre) {
  if (check_dims(d) != XHC_OK || npre < 1) return 0;
  return packed_frag_bytes(NC_of(d), (int64_t)(1 + npre) * d->N) + kColsumBytes;
}

size_t xhc_packed_active_bytes(const xhc_dims* d, int32_t Kq, int32_t with_res) {
  if (check_dims(d) != XHC_OK || Kq < 1 || Kq > kMaxKr) return 0;
  return packed_frag_bytes(kC_of(d), act_outs(d, Kq, with_res));
}

xhc_status xhc_pack_full(const xhc_dims* d, int32_t npre, const float* W_r, const float* W_pre, void* packed,
                         void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (npre < 1 || !W_r || !W_pre || !packed) return XHC_EINVAL;
  if ((int64_t)(1 + npre) * d->N > 128) return XHC_EUNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  const int64_t K = NC_of(d);
  hipError_t e = hipSuccess;
  XHC_STEP("pack", launch_pack(K, (int64_t)(1 + npre) * d->N, d->N, W_r, d->N, W_pre, npre,
                               full_grouped(d->state_dtype, K), packed, s));
  float* colsum = reinterpret_cast<float*>(reinterpret_cast<char*>(packed) +
                                           packed_frag_bytes(K, (int64_t)(1 + npre) * d->N));
  XHC_STEP("colsum", launch_colsum(K, d->N, W_r, colsum, s));
  return hip_status(e);
}

xhc_status xhc_pack_active(const xhc_dims* d, int32_t Kq, const float* W_post, const float* W_res, void* packed,
                           void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (Kq < 1 || Kq > kMaxKr || !W_post || !packed) return XHC_EINVAL;
  const int with_res = W_res != nullptr;
  clear_stale_error();
  hipError_t e = hipSuccess;
  XHC_STEP("pack", launch_pack(kC_of(d), act_outs(d, Kq, with_res), d->k * Kq, W_post, d->k * d->k, W_res,
                               with_res ? 1 : 0, act_grouped(d->state_dtype, d->C), packed,
                               reinterpret_cast<hipStream_t>(stream)));
  return hip_status(e);
}

size_t xhc_workspace_bytes(const xhc_dims* d, int32_t op, int32_t Q) {
  if (check_dims(d) != XHC_OK) return 0;
  switch (op) {
    case XHC_OP_PRE: return pre_ws(d);
    case XHC_OP_POST: return post_ws(d);
    case XHC_OP_POST_BWD: return bwd_post_ws_bytes(d);
    case XHC_OP_PRE_BWD: return bwd_pre_supported(d) ? bwd_pre_ws_bytes(d) : 0;
    case XHC_OP_FLASH_PRE: return (Q == 2 || Q == 4) ? flash_pre_ws(d, Q) : 0;
    case XHC_OP_FLASH_POST: {
      if (Q != 2 && Q != 4) return 0;
      size_t need = 0;
      for (int q = 1; q <= Q; ++q) need = std::max(need, flash_post_ws(d, Q, q));
      return need;
    }
    default: return 0;
  }
}

size_t xhc_saved_floats(const xhc_dims* d) {
  if (check_dims(d) != XHC_OK) return 0;
  return (size_t)saved_floats(d->N, d->k, d->Kr);
}

xhc_status xhc_pre(const xhc_dims* d, const void* X, const void* packed_full, const void* packed_act,
                   const float* alpha, const float* b_pre, const float* b_res, const float* b_post, void* input,
                   int32_t* idx, float* p, float* Hpre, float* Hres, float* Hpost, float* saved, void* workspace,
                   size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (d->T == 0) return XHC_OK;
  if (!X || !packed_full || !packed_act || !alpha || !b_pre || !b_res || !b_post || !input || !idx || !p ||
      !Hpre || !Hres || !Hpost || !workspace)
    return XHC_EINVAL;
  if (!aligned16(X) || !aligned16(input) || !aligned16(packed_full) || !aligned16(packed_act) ||
      !aligned16(workspace))
    return XHC_EUNSUPPORTED;
  if (d->impl == XHC_IMPL_FUSED && !fused_pre_supported(d)) return XHC_EUNSUPPORTED;
  if (workspace_bytes < pre_ws(d)) return XHC_EWORKSPACE;
  // AUTO takes the single-pass kernel where it applies (it reads X once) and
  // the multi-kernel path elsewhere
  if (d->impl == XHC_IMPL_AUTO && !fused_pre_supported(d)) {
    xhc_dims m = *d;
    m.impl = XHC_IMPL_MULTI;
    return xhc_pre(&m, X, packed_full, packed_act, alpha, b_pre, b_res, b_post, input, idx, p, Hpre, Hres, Hpost,
                   saved, workspace, workspace_bytes, stream);
  }
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  float* part = reinterpret_cast<float*>(workspace);
  const size_t part_max = std::max(part_bytes(d, false, NC_of(d), 2 * d->N),
                                   part_bytes(d, true, kC_of(d), act_outs(d, d->Kr, 1)));
  float* sums = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + part_max);
  const int64_t NC = NC_of(d), kC = kC_of(d);
  const int64_t nout_full = 2 * d->N, nout_act = act_outs(d, d->Kr, 1);
  const int nsave = saved_floats(d->N, d->k, d->Kr);
  const float* colsum = reinterpret_cast<const float*>(reinterpret_cast<const char*>(packed_full) +
                                                       packed_frag_bytes(NC, nout_full));
  hipError_t e = hipSuccess;
  if (d->impl != XHC_IMPL_MULTI) {
    e = launch_pre_fused(d, X, packed_full, colsum, packed_act, alpha, b_pre, b_res, b_post, input, idx, p, Hpre,
                         Hres, Hpost, saved, workspace, s);
    if (e == hipSuccess) return XHC_OK;
    if (d->impl == XHC_IMPL_FUSED || e != hipErrorInvalidConfiguration) {
      g_failed_step = "pre_fused";
      return hip_status(e);
    }
    e = hipSuccess;   // the device cannot hold the single-pass grid: multi-kernel path
    clear_stale_error();
  }
  XHC_STEP("proj_full", launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, NC, packed_full, nout_full,
                                            nullptr, d->k, part, s));
  XHC_STEP("pre_route", launch_pre_route(part, proj_chunks(d->state_dtype, false, NC, d->C, nout_full, d->T), nout_full, d->T, d->N, d->m, d->k, 1, d->C, colsum,
                                         alpha, 1, b_pre, d->eps, idx, p, Hpre, sums, saved, nsave,
                                         nsave - 4, d->router, s));
  XHC_STEP("proj_active", launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, kC, packed_act, nout_act, idx,
                                              d->k, part, s));
  XHC_STEP("pre_coef", launch_pre_coef(part, proj_chunks(d->state_dtype, true, kC, d->C, nout_act, d->T), nout_act,
                                       d->T, d->k, d->Kr, 1, d->C, alpha + 2, alpha + 1, b_post, b_res, d->eps,
                                       d->sinkhorn_iters, d->clamp_delta, Hpost, Hres, sums, saved, nsave, 2 * d->N,
                                       nsave - 2, s));
  XHC_STEP("dense_read",
           launch_dense_read(d->state_dtype, X, d->T, d->N, d->C, Hpre, 1, idx, d->k, input, nullptr, s));
  return hip_status(e);
}

xhc_status xhc_post(const xhc_dims* d, void* X, const void* F, const float* conv_w, const int32_t* idx,
                    const float* p, const float* Hres, const float* Hpost, void* Xact_save, void* workspace,
                    size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (d->T == 0) return XHC_OK;
  if (!X || !F || !idx || !p || !Hres || !Hpost) return XHC_EINVAL;
  if ((d->Kr > 1) != (conv_w != nullptr)) return XHC_EINVAL;
  if (X == F) return XHC_EINVAL;
  if (!aligned16(X) || !aligned16(F) || (conv_w && !aligned16(conv_w)) || (Xact_save && !aligned16(Xact_save)))
    return XHC_EUNSUPPORTED;
  const size_t need = post_ws(d);
  if (need > 0 && (!workspace || workspace_bytes < need)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  float* wb = nullptr;
  hipError_t e = hipSuccess;
  if (d->Kr > 1) {
    const int np = d->Kr * (d->Kr + 1) / 2;
    float* gpart = reinterpret_cast<float*>(workspace);
    wb = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                  align_up((size_t)gram_chunks(d->C, d->S, d->Kr, d->kappa) * np * (size_t)d->T *
                                           sizeof(float)));
    XHC_STEP("post_gram", launch_post_gram(d->state_dtype, F, d->T, d->S, d->C, d->Kr, d->kappa, conv_w, gpart, s));
    XHC_STEP("post_coef", launch_post_coef(gpart, gram_chunks(d->C, d->S, d->Kr, d->kappa), d->T, d->k, d->Kr,
                                           d->gram_schmidt, p, Hpost, wb, s));
  }
  XHC_STEP("post_apply", launch_post_apply(d->state_dtype, X, F, d->T, d->S, d->N, d->C, d->k, d->Kr, d->kappa,
                                           conv_w, idx, p, Hres, Hpost, wb, nullptr, nullptr, nullptr, Xact_save,
                                           s));
  return hip_status(e);
}

// ---------------------------------------------------------------- xHC-Flash

xhc_status xhc_flash_pre(const xhc_dims* d, int32_t Q, const void* X, const void* packed_full,
                         const void* packed_act1, const float* alpha_pre, const float* b_pre,
                         const float* alpha_post1, const float* b_post1, void* input1, void* base, int32_t* idx,
                         float* p, float* Hpre, float* Hpost1, void* workspace, size_t workspace_bytes,
                         void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (Q != 2 && Q != 4) return XHC_EINVAL;
  if ((int64_t)(Q + 1) * d->N > 128) return XHC_EUNSUPPORTED;
  if (d->T == 0) return XHC_OK;
  if (!X || !packed_full || !packed_act1 || !alpha_pre || !b_pre || !alpha_post1 || !b_post1 || !input1 || !base ||
      !idx || !p || !Hpre || !Hpost1 || !workspace)
    return XHC_EINVAL;
  if (!aligned16(X) || !aligned16(input1) || !aligned16(base) || !aligned16(packed_full) || !aligned16(packed_act1))
    return XHC_EUNSUPPORTED;
  if (workspace_bytes < flash_pre_ws(d, Q)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  const int64_t NC = NC_of(d), kC = kC_of(d);
  const int64_t nf = (int64_t)(Q + 1) * d->N, na = act_outs(d, 1, 0);
  float* part = reinterpret_cast<float*>(workspace);
  float* sums = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                         std::max(part_bytes(d, false, NC, nf), part_bytes(d, true, kC, na)));
  const float* colsum = reinterpret_cast<const float*>(reinterpret_cast<const char*>(packed_full) +
                                                       packed_frag_bytes(NC, nf));
  hipError_t e = hipSuccess;
  XHC_STEP("flash_proj_full",
           launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, NC, packed_full, nf, nullptr, d->k, part, s));
  XHC_STEP("flash_route", launch_pre_route(part, proj_chunks(d->state_dtype, false, NC, d->C, nf, d->T), nf, d->T, d->N, d->m, d->k, Q, d->C, colsum,
                                           alpha_pre, 1, b_pre, d->eps, idx, p, Hpre, sums, nullptr, 0, 0,
                                           d->router, s));
  XHC_STEP("flash_proj_active",
           launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, kC, packed_act1, na, idx, d->k, part, s));
  XHC_STEP("flash_coef1", launch_pre_coef(part, proj_chunks(d->state_dtype, true, kC, d->C, na, d->T), na, d->T,
                                          d->k, 1, 0, d->C, alpha_post1, nullptr, b_post1, nullptr, d->eps,
                                          d->sinkhorn_iters, d->clamp_delta, Hpost1, nullptr, sums, nullptr, 0, 0, 0,
                                          s));
  XHC_STEP("flash_dense_read",
           launch_dense_read(d->state_dtype, X, d->T, d->N, d->C, Hpre, Q, idx, d->k, input1, base, s));
  return hip_status(e);
}

xhc_status xhc_flash_post(const xhc_dims* d, int32_t Q, int32_t q, void* X, const void* F, const float* conv_w,
                          const int32_t* idx, const float* p, const float* Hpost, const float* Hres,
                          const float* Hpre_next, const void* base_next, void* input_next,
                          const void* packed_act_next, const float* alpha_next, const float* b_post_next,
                          const float* b_res_next, float* Hpost_next, float* Hres_next, void* workspace,
                          size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if ((Q != 2 && Q != 4) || q < 1 || q > Q) return XHC_EINVAL;
  if (d->T == 0) return XHC_OK;
  const int Kq = flash_Kq(d, q);
  const bool last = q == Q;
  if (!X || !F || !idx || !p || !Hpost || X == F) return XHC_EINVAL;
  if ((Kq > 1) != (conv_w != nullptr)) return XHC_EINVAL;
  if (last != (Hres != nullptr)) return XHC_EINVAL;
  if (!last) {
    if (!Hpre_next || !base_next || !input_next || !packed_act_next || !alpha_next || !b_post_next || !Hpost_next)
      return XHC_EINVAL;
    if ((q + 1 == Q) != (b_res_next != nullptr && Hres_next != nullptr)) return XHC_EINVAL;
    if (!aligned16(base_next) || !aligned16(input_next) || !aligned16(packed_act_next)) return XHC_EUNSUPPORTED;
  }
  if (!aligned16(X) || !aligned16(F) || (conv_w && !aligned16(conv_w))) return XHC_EUNSUPPORTED;
  const size_t need = flash_post_ws(d, Q, q);
  if (need > 0 && (!workspace || workspace_bytes < need)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  hipError_t e = hipSuccess;
  float* wb = nullptr;
  if (Kq > 1) {
    const int np = Kq * (Kq + 1) / 2;
    float* gpart = reinterpret_cast<float*>(workspace);
    wb = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                  align_up((size_t)gram_chunks(d->C, d->S, Kq, d->kappa) * np * (size_t)d->T *
                                           sizeof(float)));
    XHC_STEP("flash_post_gram", launch_post_gram(d->state_dtype, F, d->T, d->S, d->C, Kq, d->kappa, conv_w, gpart, s));
    XHC_STEP("flash_post_coef", launch_post_coef(gpart, gram_chunks(d->C, d->S, Kq, d->kappa), d->T, d->k, Kq,
                                                 d->gram_schmidt, p, Hpost, wb, s));
  }
  XHC_STEP("flash_post_apply", launch_post_apply(d->state_dtype, X, F, d->T, d->S, d->N, d->C, d->k, Kq, d->kappa,
                                                 conv_w, idx, p, Hres, Hpost, wb, last ? nullptr : Hpre_next,
                                                 last ? nullptr : base_next, last ? nullptr : input_next, nullptr, s));
  if (!last) {
    // mappings of sublayer q + 1 from the updated active rows (Alg. xHC-Flash, MLP step; App. E.2)
    const int Kn = flash_Kq(d, q + 1);
    const int with_res = (q + 1 == Q);
    const int64_t kC = kC_of(d), na = act_outs(d, Kn, with_res);
    float* part = reinterpret_cast<float*>(workspace);
    float* sums = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + part_bytes(d, true, kC, na));
    XHC_STEP("flash_proj_next",
             launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, kC, packed_act_next, na, idx, d->k, part, s));
    XHC_STEP("flash_coef_next",
             launch_pre_coef(part, proj_chunks(d->state_dtype, true, kC, d->C, na, d->T), na, d->T, d->k, Kn, with_res, d->C, alpha_next,
                             with_res ? alpha_next + 1 : nullptr, b_post_next, b_res_next, d->eps, d->sinkhorn_iters,
                             d->clamp_delta, Hpost_next, Hres_next, sums, nullptr, 0, 0, 0, s));
  }
  return hip_status(e);
}

// ---------------------------------------------------------------- backward

xhc_status xhc_post_bwd(const xhc_dims* d, const void* dXn, void* X, const void* Xact, const void* F,
                        const float* conv_w, const int32_t* idx, const float* p, const float* Hres,
                        const float* Hpost, void* dX, void* dF, float* dHres, float* dHpost, float* dp,
                        float* dconv_w, void* workspace, size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (d->T == 0) return XHC_OK;
  if (!dXn || !X || !Xact || !F || !idx || !p || !Hres || !Hpost || !dX || !dF || !dHres || !dHpost || !dp ||
      !workspace)
    return XHC_EINVAL;
  if ((d->Kr > 1) != (conv_w != nullptr) || (d->Kr > 1) != (dconv_w != nullptr)) return XHC_EINVAL;
  if (dX == dXn || dX == X || dF == F) return XHC_EINVAL;
  if (!aligned16(dXn) || !aligned16(X) || !aligned16(Xact) || !aligned16(F) || !aligned16(dX) || !aligned16(dF) ||
      (conv_w && !aligned16(conv_w)) || (dconv_w && !aligned16(dconv_w)))
    return XHC_EUNSUPPORTED;
  if (workspace_bytes < bwd_post_ws_bytes(d)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  hipError_t e = hipSuccess;
  XHC_STEP("post_bwd", launch_bwd_post(d, dXn, X, Xact, F, conv_w, idx, p, Hres, Hpost, dX, dF, dHres, dHpost, dp,
                                       dconv_w, reinterpret_cast<char*>(workspace), s));
  return hip_status(e);
}

xhc_status xhc_pre_bwd(const xhc_dims* d, const void* X, const void* packed_full, const float* W_r,
                       const float* W_pre, const float* W_res, const float* W_post, const float* alpha,
                       const float* b_res, const float* saved, const int32_t* idx, const float* p,
                       const float* Hpre, const float* Hpost, const void* d_input, const float* dHres,
                       const float* dHpost, const float* dp, void* dX, float* dW_r, float* dW_pre, float* dW_res,
                       float* dW_post, float* dalpha, float* db_pre, float* db_res, float* db_post, void* workspace,
                       size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (!bwd_pre_supported(d)) return XHC_EUNSUPPORTED;
  if (d->T == 0) return XHC_OK;
  if (!X || !packed_full || !W_r || !W_pre || !W_res || !W_post || !alpha || !b_res || !saved || !idx || !p ||
      !Hpre || !Hpost || !d_input || !dHres || !dHpost || !dp || !dX || !dW_r || !dW_pre || !dW_res || !dW_post ||
      !dalpha || !db_pre || !db_res || !db_post || !workspace)
    return XHC_EINVAL;
  if (dX == X) return XHC_EINVAL;
  if (!aligned16(X) || !aligned16(d_input) || !aligned16(dX)) return XHC_EUNSUPPORTED;
  if (workspace_bytes < bwd_pre_ws_bytes(d)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  const float* colsum = reinterpret_cast<const float*>(reinterpret_cast<const char*>(packed_full) +
                                                       packed_frag_bytes(NC_of(d), 2 * d->N));
  hipError_t e = hipSuccess;
  XHC_STEP("pre_bwd", launch_bwd_pre(d, X, colsum, W_r, W_pre, W_res, W_post, alpha, b_res, saved, idx, p, Hpre,
                                     Hpost, d_input, dHres, dHpost, dp, dX, dW_r, dW_pre, dW_res, dW_post, dalpha,
                                     db_pre, db_res, db_post, reinterpret_cast<char*>(workspace), s));
  return hip_status(e);
}

xhc_status xhc_stream_sum(const xhc_dims* d, const void* X, void* out, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (d->T == 0) return XHC_OK;
  if (!X || !out || X == out) return XHC_EINVAL;
  if (!aligned16(X) || !aligned16(out)) return XHC_EUNSUPPORTED;
  clear_stale_error();
  hipError_t e = hipSuccess;
  XHC_STEP("stream_sum", launch_stream_sum(d->state_dtype, X, d->T, d->N, d->C, out,
                                           reinterpret_cast<hipStream_t>(stream)));
  return hip_status(e);
}

xhc_status xhc_stream_sum_bwd(const xhc_dims* d, const void* dout, void* dX, int32_t accumulate, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (accumulate != 0 && accumulate != 1) return XHC_EINVAL;
  if (d->T == 0) return XHC_OK;
  if (!dout || !dX || dout == dX) return XHC_EINVAL;
  if (!aligned16(dout) || !aligned16(dX)) return XHC_EUNSUPPORTED;
  clear_stale_error();
  hipError_t e = hipSuccess;
  XHC_STEP("stream_sum_bwd", launch_stream_bcast(d->state_dtype, dout, d->T, d->N, d->C, accumulate, dX,
                                                 reinterpret_cast<hipStream_t>(stream)));
  return hip_status(e);
}

}  // extern "C"

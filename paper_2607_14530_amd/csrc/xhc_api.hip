// C ABI of the xHC library: argument validation, workspace sizing, dispatch.
// Every check happens before the first launch, so an error return leaves
// all outputs untouched.
#include <hip/hip_runtime.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>

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
  if (d->attn_aug != 0 && d->attn_aug != 1) return XHC_EINVAL;
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

// The first kPreErrBytes of an xhc_pre workspace hold the count of bounded
// waits that gave up (xhc_pre_failures); both paths clear it.
constexpr size_t kPreErrBytes = 256;

size_t pre_ws_multi(const xhc_dims* d) {
  const size_t full = part_bytes(d, false, NC_of(d), 2 * d->N);
  const size_t act = part_bytes(d, true, kC_of(d), act_outs(d, d->Kr, 1));
  const size_t sf = sums_bytes(2 * d->N, d->T), sa = sums_bytes(act_outs(d, d->Kr, 1), d->T);
  return kPreErrBytes + (full > act ? full : act) + (sf > sa ? sf : sa);
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
// attention-type (odd q) has one, MLP-type (even q) has d->Kr; with attn_aug
// the attention-type sublayers have d->Kr too (the ablation of
// attention-side temporal augmentation)
int flash_Kq(const xhc_dims* d, int q) { return (q % 2 == 1 && !d->attn_aug) ? 1 : d->Kr; }

size_t flash_pre_ws(const xhc_dims* d, int Q) {
  const int64_t nf = (int64_t)(Q + 1) * d->N, na = act_outs(d, flash_Kq(d, 1), 0);
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

// ---- xHC-Flash backward: the per-sublayer reverse runs the single-sublayer
// kernels on the k active rows ([T, k, C], every row active, identity slot
// map); dims_rows() is that view.  Its post part sees the sublayer's K_q, its
// pre part sees K_q with every stream fixed (no router).
xhc_dims dims_rows(const xhc_dims* d, int Kq) {
  xhc_dims r = *d;
  r.N = d->k;
  r.m = d->k;
  r.Kr = Kq;
  r.router = XHC_ROUTER_SIGMOID;
  r.impl = XHC_IMPL_MULTI;
  return r;
}

// the entry-state reverse: the single-sublayer pre reverse with one
// write-back component (its active mapping receives no gradient here)
xhc_dims dims_entry(const xhc_dims* d) {
  xhc_dims r = *d;
  r.Kr = 1;
  r.impl = XHC_IMPL_MULTI;
  return r;
}

bool flash_bwd_supported(const xhc_dims* d) {
  if ((d->k != 4 && d->k != 8) || !bwd_pre_supported(d)) return false;
  const xhc_dims r = dims_rows(d, d->Kr);
  return bwd_pre_supported(&r);
}

// sequential carve of a workspace into 256-byte aligned pieces
struct Carve {
  size_t total = 0;
  size_t take(size_t bytes) {
    const size_t at = total;
    total += align_up(bytes);
    return at;
  }
};

// The active-row gradient between sublayers is kept in fp32, so the per-row
// reverses run on fp32 copies of the slice (dims with state_dtype fp32).
xhc_dims dims_rows32(const xhc_dims* d, int Kq) {
  xhc_dims r = dims_rows(d, Kq);
  r.state_dtype = XHC_F32;
  return r;
}

struct FlashPostBwdWs {
  size_t post, pre, part, sums, idx_id, hres_id, hsel, da_out, dhpost, dhres, dp,
      saved, hpost_re, hres_re, w0, colsum0, wres0, bres0, alpha2, dwr, dwpre, dbpre, dwres, dbres, dalpha2, total;
};

FlashPostBwdWs flash_post_bwd_ws(const xhc_dims* d, int Q, int q) {
  const int Kq = flash_Kq(d, q);
  const xhc_dims r = dims_rows32(d, Kq);
  const int64_t T = d->T, k = d->k, C = d->C, kC = k * C;
  const size_t f = sizeof(float);
  const int64_t na = act_outs(d, Kq, q == Q);
  Carve c;
  FlashPostBwdWs w;
  w.post = c.take(bwd_post_ws_bytes(&r));
  w.pre = c.take(bwd_pre_ws_bytes(&r));
  w.part = c.take(part_bytes(d, true, kC, na));
  w.sums = c.take(sums_bytes(na, T));
  w.idx_id = c.take((size_t)T * k * sizeof(int32_t));
  w.hres_id = c.take((size_t)T * k * k * f);
  w.hsel = c.take((size_t)T * k * f);
  w.da_out = c.take((size_t)T * kC * f);
  w.dhpost = c.take((size_t)T * k * Kq * f);
  w.dhres = c.take((size_t)T * k * k * f);
  w.dp = c.take((size_t)T * k * f);
  w.saved = c.take((size_t)T * saved_floats(k, k, Kq) * f);
  w.hpost_re = c.take((size_t)T * k * Kq * f);
  w.hres_re = c.take((size_t)T * k * k * f);
  w.w0 = c.take((size_t)kC * k * f);
  w.colsum0 = c.take((size_t)k * f);
  w.wres0 = c.take((size_t)kC * k * k * f);
  w.bres0 = c.take((size_t)k * k * f);
  w.alpha2 = c.take(3 * f);
  w.dwr = c.take((size_t)kC * k * f);
  w.dwpre = c.take((size_t)kC * k * f);
  w.dbpre = c.take((size_t)k * f);
  w.dwres = c.take((size_t)kC * k * k * f);
  w.dbres = c.take((size_t)k * k * f);
  w.dalpha2 = c.take(3 * f);
  w.total = c.total;
  return w;
}

struct FlashPreBwdWs {
  size_t pre_slice;   // one pre-map reverse's workspace (Q of them when the row passes are fused)
  bool fused;
  size_t multi;       // the fused row pass's per-token inputs
  size_t pre, part, sums, saved, idx_s, p_s, hpre_s, hmask, wpost0, wres0, bres0, hpost0, dhpost0, dhres0, dp0,
      alpha_e, dwr, dwres, dwpost, dalpha, dbres, dbpost, total;
};

FlashPreBwdWs flash_pre_bwd_ws(const xhc_dims* d, int Q) {
  const xhc_dims e = dims_entry(d);
  const int64_t T = d->T, N = d->N, k = d->k, C = d->C, NC = N * C, kC = k * C;
  const size_t f = sizeof(float);
  const int64_t nf = (int64_t)(Q + 1) * N;
  Carve c;
  FlashPreBwdWs w;
  w.fused = bwd_rows_multi_supported(&e, Q);
  w.pre_slice = align_up(bwd_pre_ws_bytes(&e));
  w.pre = c.take((w.fused ? Q : 1) * w.pre_slice);
  w.multi = c.take(w.fused ? bwd_rows_multi_ws_bytes(&e, Q) : 0);
  w.part = c.take(part_bytes(d, false, NC, nf));
  w.sums = c.take(sums_bytes(nf, T));
  w.saved = c.take((size_t)T * saved_floats(N, k, 1) * f);
  w.idx_s = c.take((size_t)T * k * sizeof(int32_t));
  w.p_s = c.take((size_t)T * k * f);
  w.hpre_s = c.take((size_t)Q * T * N * f);
  w.hmask = c.take((size_t)Q * T * N * f);   // [Q][T, N]: the masked dense-read weights of pre-map q >= 1
  w.wpost0 = c.take((size_t)kC * k * f);
  w.wres0 = c.take((size_t)kC * k * k * f);
  w.bres0 = c.take((size_t)k * k * f);
  w.hpost0 = c.take((size_t)T * k * f);
  w.dhpost0 = c.take((size_t)T * k * f);
  w.dhres0 = c.take((size_t)T * k * k * f);
  w.dp0 = c.take((size_t)T * k * f);
  w.alpha_e = c.take(3 * f);
  w.dwr = c.take((size_t)NC * N * f);
  w.dwres = c.take((size_t)kC * k * k * f);
  w.dwpost = c.take((size_t)kC * k * f);
  w.dalpha = c.take(3 * f);
  w.dbres = c.take((size_t)k * k * f);
  w.dbpost = c.take((size_t)k * f);
  w.total = c.total;
  return w;
}

size_t post_ws(const xhc_dims* d) {
  if (d->Kr == 1) return 0;
  const int np = d->Kr * (d->Kr + 1) / 2;
  return align_up((size_t)gram_chunks(d->C, d->S, d->Kr, d->kappa) * np * (size_t)d->T * sizeof(float)) +
         align_up((size_t)d->T * d->k * d->Kr * sizeof(float));
}

// xhc_post's work on a given scratch buffer (the caller's workspace, or the
// library's static one for xhc_post_noalloc)
xhc_status post_impl(const xhc_dims* d, void* X, const void* F, const float* conv_w, const int32_t* idx,
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
  const float* gp = nullptr;
  hipError_t e = hipSuccess;
  if (d->Kr > 1) {
    const int np = d->Kr * (d->Kr + 1) / 2;
    float* gpart = reinterpret_cast<float*>(workspace);
    wb = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                  align_up((size_t)gram_chunks(d->C, d->S, d->Kr, d->kappa) * np * (size_t)d->T *
                                           sizeof(float)));
    gp = gpart;
    XHC_STEP("post_gram", launch_post_gram(d->state_dtype, F, d->T, d->S, d->C, d->Kr, d->kappa, conv_w, gpart, s));
  }
  XHC_STEP("post_apply", launch_post_apply(d->state_dtype, X, F, d->T, d->S, d->N, d->C, d->k, d->Kr, d->kappa,
                                           conv_w, idx, p, Hres, Hpost, gp,
                                           gram_chunks(d->C, d->S, d->Kr, d->kappa), d->gram_schmidt, wb, nullptr,
                                           nullptr, nullptr, Xact_save, s));
  return hip_status(e);
}


// ---- scratch of xhc_post_noalloc: a fixed device array instead of a caller
// workspace.  Each device holds its own copy of the array for the life of the
// process; host code reaches it only through the address hipGetSymbolAddress
// returns on that device (the array's name is not a device address in host
// code).
constexpr size_t kNoAllocScratchBytes = XHC_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// the address of `scratch` on the current device, looked up once per device
xhc_status noalloc_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess && (dev < 0 || dev >= kMaxDevices)) e = hipErrorInvalidDevice;
  if (e != hipSuccess) {
    g_failed_step = "noalloc_device";
    return hip_status(e);
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      g_failed_step = "noalloc_symbol";
      return hip_status(e != hipSuccess ? e : hipErrorInvalidSymbol);
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return XHC_OK;
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
    case XHC_OP_FLASH_POST_BWD: {
      if ((Q != 2 && Q != 4) || !flash_bwd_supported(d)) return 0;
      size_t need = 0;
      for (int q = 1; q <= Q; ++q) need = std::max(need, flash_post_bwd_ws(d, Q, q).total);
      return need;
    }
    case XHC_OP_FLASH_PRE_BWD:
      return ((Q == 2 || Q == 4) && flash_bwd_supported(d)) ? flash_pre_bwd_ws(d, Q).total : 0;
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
  float* part = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + kPreErrBytes);
  const size_t part_max = std::max(part_bytes(d, false, NC_of(d), 2 * d->N),
                                   part_bytes(d, true, kC_of(d), act_outs(d, d->Kr, 1)));
  float* sums = reinterpret_cast<float*>(reinterpret_cast<char*>(part) + part_max);
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
  XHC_STEP("pre_clear", launch_fill0(workspace, kPreErrBytes, s));   // no waits here: no failures
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

xhc_status xhc_pre_failures(const void* workspace, int32_t* failures, void* stream) {
  if (!workspace || !failures) return XHC_EINVAL;
  if (!aligned16(workspace)) return XHC_EUNSUPPORTED;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  int32_t n = 0;
  hipError_t e = hipMemcpyAsync(&n, workspace, sizeof(n), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    g_failed_step = "pre_failures";
    return hip_status(e);
  }
  *failures = n;
  return XHC_OK;
}

xhc_status xhc_post(const xhc_dims* d, void* X, const void* F, const float* conv_w, const int32_t* idx,
                    const float* p, const float* Hres, const float* Hpost, void* Xact_save, void* workspace,
                    size_t workspace_bytes, void* stream) {
  return post_impl(d, X, F, conv_w, idx, p, Hres, Hpost, Xact_save, workspace, workspace_bytes, stream);
}

xhc_status xhc_post_noalloc(const xhc_dims* d, void* X, const void* F, const float* conv_w, const int32_t* idx,
                            const float* p, const float* Hres, const float* Hpost, void* Xact_save, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (post_ws(d) > kNoAllocScratchBytes) return XHC_EWORKSPACE;
  void* scr = nullptr;
  if (post_ws(d) > 0 && d->T > 0) {
    st = noalloc_scratch(&scr);
    if (st != XHC_OK) return st;
  }
  return post_impl(d, X, F, conv_w, idx, p, Hres, Hpost, Xact_save, scr, scr ? kNoAllocScratchBytes : 0, stream);
}

// ---------------------------------------------------------------- xHC-Flash

xhc_status xhc_flash_pre(const xhc_dims* d, int32_t Q, const void* X, const void* packed_full,
                         const void* packed_act1, const float* alpha_pre, const float* b_pre,
                         const float* alpha_post1, const float* b_post1, void* input1, void* base, int32_t* idx,
                         float* p, float* Hpre, float* Hpost1, float* saved, float* saved_act1, void* workspace,
                         size_t workspace_bytes, void* stream) {
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
  const int K1 = flash_Kq(d, 1);
  const int64_t nf = (int64_t)(Q + 1) * d->N, na = act_outs(d, K1, 0);
  float* part = reinterpret_cast<float*>(workspace);
  float* sums = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                         std::max(part_bytes(d, false, NC, nf), part_bytes(d, true, kC, na)));
  const float* colsum = reinterpret_cast<const float*>(reinterpret_cast<const char*>(packed_full) +
                                                       packed_frag_bytes(NC, nf));
  hipError_t e = hipSuccess;
  XHC_STEP("flash_proj_full",
           launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, NC, packed_full, nf, nullptr, d->k, part, s));
  // the records the backward reads (one per pre-map; fields it does not use stay zero)
  const int nsave = saved_floats(d->N, d->k, 1);
  if (saved) XHC_STEP("flash_save_zero", launch_fill0(saved, (size_t)Q * d->T * nsave * sizeof(float), s));
  XHC_STEP("flash_route", launch_pre_route(part, proj_chunks(d->state_dtype, false, NC, d->C, nf, d->T), nf, d->T, d->N, d->m, d->k, Q, d->C, colsum,
                                           alpha_pre, 1, b_pre, d->eps, idx, p, Hpre, sums, saved,
                                           saved ? nsave : 0, saved ? nsave - 4 : 0, d->router, s, -1));
  XHC_STEP("flash_proj_active",
           launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, kC, packed_act1, na, idx, d->k, part, s));
  // sublayer 1's mapping record for the backward (the layout its reverse uses)
  const int nsave1 = saved_floats(d->k, d->k, K1);
  if (saved_act1)
    XHC_STEP("flash_save_zero", launch_fill0(saved_act1, (size_t)d->T * nsave1 * sizeof(float), s));
  XHC_STEP("flash_coef1", launch_pre_coef(part, proj_chunks(d->state_dtype, true, kC, d->C, na, d->T), na, d->T,
                                          d->k, K1, 0, d->C, alpha_post1, nullptr, b_post1, nullptr, d->eps,
                                          d->sinkhorn_iters, d->clamp_delta, Hpost1, nullptr, sums, saved_act1,
                                          saved_act1 ? nsave1 : 0, 2 * d->k, nsave1 - 2, s));
  XHC_STEP("flash_dense_read",
           launch_dense_read(d->state_dtype, X, d->T, d->N, d->C, Hpre, Q, idx, d->k, input1, base, s));
  return hip_status(e);
}

xhc_status xhc_flash_post(const xhc_dims* d, int32_t Q, int32_t q, void* X, const void* F, const float* conv_w,
                          const int32_t* idx, const float* p, const float* Hpost, const float* Hres,
                          const float* Hpre_next, const void* base_next, void* input_next,
                          const void* packed_act_next, const float* alpha_next, const float* b_post_next,
                          const float* b_res_next, float* Hpost_next, float* Hres_next, void* Xact_save,
                          float* saved_next, void* workspace, size_t workspace_bytes, void* stream) {
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
  if (!aligned16(X) || !aligned16(F) || (conv_w && !aligned16(conv_w)) || (Xact_save && !aligned16(Xact_save)))
    return XHC_EUNSUPPORTED;
  const size_t need = flash_post_ws(d, Q, q);
  if (need > 0 && (!workspace || workspace_bytes < need)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  hipError_t e = hipSuccess;
  float* wb = nullptr;
  const float* gp = nullptr;
  if (Kq > 1) {
    const int np = Kq * (Kq + 1) / 2;
    float* gpart = reinterpret_cast<float*>(workspace);
    wb = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) +
                                  align_up((size_t)gram_chunks(d->C, d->S, Kq, d->kappa) * np * (size_t)d->T *
                                           sizeof(float)));
    gp = gpart;
    XHC_STEP("flash_post_gram", launch_post_gram(d->state_dtype, F, d->T, d->S, d->C, Kq, d->kappa, conv_w, gpart, s));
  }
  XHC_STEP("flash_post_apply", launch_post_apply(d->state_dtype, X, F, d->T, d->S, d->N, d->C, d->k, Kq, d->kappa,
                                                 conv_w, idx, p, Hres, Hpost, gp,
                                                 gram_chunks(d->C, d->S, Kq, d->kappa), d->gram_schmidt, wb,
                                                 last ? nullptr : Hpre_next,
                                                 last ? nullptr : base_next, last ? nullptr : input_next, Xact_save,
                                                 s));
  if (!last) {
    // mappings of sublayer q + 1 from the updated active rows (Alg. xHC-Flash, MLP step; App. E.2)
    const int Kn = flash_Kq(d, q + 1);
    const int with_res = (q + 1 == Q);
    const int64_t kC = kC_of(d), na = act_outs(d, Kn, with_res);
    float* part = reinterpret_cast<float*>(workspace);
    float* sums = reinterpret_cast<float*>(reinterpret_cast<char*>(workspace) + part_bytes(d, true, kC, na));
    XHC_STEP("flash_proj_next",
             launch_proj_partial(d->state_dtype, X, d->T, d->N, d->C, kC, packed_act_next, na, idx, d->k, part, s));
    const int nsn = saved_floats(d->k, d->k, Kn);   // the next sublayer's mapping record
    if (saved_next)
      XHC_STEP("flash_save_zero", launch_fill0(saved_next, (size_t)d->T * nsn * sizeof(float), s));
    XHC_STEP("flash_coef_next",
             launch_pre_coef(part, proj_chunks(d->state_dtype, true, kC, d->C, na, d->T), na, d->T, d->k, Kn, with_res, d->C, alpha_next,
                             with_res ? alpha_next + 1 : nullptr, b_post_next, b_res_next, d->eps, d->sinkhorn_iters,
                             d->clamp_delta, Hpost_next, Hres_next, sums, saved_next, saved_next ? nsn : 0,
                             2 * d->k, nsn - 2, s));
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
  if (dX == X || dF == F) return XHC_EINVAL;   // dX == dXn: in place
  if (!aligned16(dXn) || !aligned16(X) || !aligned16(Xact) || !aligned16(F) || !aligned16(dX) || !aligned16(dF) ||
      (conv_w && !aligned16(conv_w)) || (dconv_w && !aligned16(dconv_w)))
    return XHC_EUNSUPPORTED;
  if (workspace_bytes < bwd_post_ws_bytes(d)) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  hipError_t e = hipSuccess;
  XHC_STEP("post_bwd", launch_bwd_post(d, dXn, X, Xact, F, conv_w, idx, p, Hres, Hpost, dX, dF, dHres, dHpost, dp,
                                       dconv_w, reinterpret_cast<char*>(workspace), s, /*grad_f32=*/false));
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

// ---------------------------------------------------------------- xHC-Flash backward

xhc_status xhc_flash_post_bwd(const xhc_dims* d, int32_t Q, int32_t q, const void* dXn, void* da, const void* Xact,
                              const void* F, const float* conv_w, const int32_t* idx, const float* p,
                              const float* Hpost, const float* Hres, const void* packed_act, const float* W_post,
                              const float* W_res, const float* alpha_post, const float* alpha_res,
                              const float* b_post, const float* b_res, const float* Hpre_q, const void* d_input,
                              const float* saved_act, void* dF, float* dconv_w, float* dW_post,
                              float* dalpha_post, float* db_post, float* dW_res, float* dalpha_res, float* db_res,
                              float* dp, float* dHpre_act, void* workspace, size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if ((Q != 2 && Q != 4) || q < 1 || q > Q) return XHC_EINVAL;
  if (!flash_bwd_supported(d)) return XHC_EUNSUPPORTED;
  if (d->T == 0) return XHC_OK;
  const int Kq = flash_Kq(d, q);
  const bool last = q == Q, reads = q >= 2;
  if (!da || !Xact || !F || !idx || !p || !Hpost || !packed_act || !W_post || !alpha_post || !b_post || !dF ||
      !dW_post || !dalpha_post || !db_post || !dp || !workspace)
    return XHC_EINVAL;
  if ((Kq > 1) != (conv_w != nullptr) || (Kq > 1) != (dconv_w != nullptr)) return XHC_EINVAL;
  if (last != (dXn != nullptr) || last != (Hres != nullptr) || last != (W_res != nullptr) ||
      last != (alpha_res != nullptr) || last != (b_res != nullptr) || last != (dW_res != nullptr) ||
      last != (dalpha_res != nullptr) || last != (db_res != nullptr))
    return XHC_EINVAL;
  if (reads != (Hpre_q != nullptr) || reads != (d_input != nullptr) || reads != (dHpre_act != nullptr))
    return XHC_EINVAL;
  if (da == Xact || dF == F) return XHC_EINVAL;
  if (!aligned16(da) || !aligned16(Xact) || !aligned16(F) || !aligned16(dF) || !aligned16(packed_act) ||
      (dXn && !aligned16(dXn)) || (d_input && !aligned16(d_input)) || (conv_w && !aligned16(conv_w)) ||
      (dconv_w && !aligned16(dconv_w)) || !aligned16(workspace))
    return XHC_EUNSUPPORTED;
  const FlashPostBwdWs w = flash_post_bwd_ws(d, Q, q);
  if (workspace_bytes < w.total) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  char* ws = reinterpret_cast<char*>(workspace);
  auto F32 = [&](size_t at) { return reinterpret_cast<float*>(ws + at); };
  const int64_t T = d->T, k = d->k, C = d->C, kC = k * C;
  const xhc_dims r = dims_rows32(d, Kq);
  float* dA = reinterpret_cast<float*>(da);
  // a bf16 state: the reverse runs in place on da and the active-row pass adds
  // the read of input_q (no separate pass)
  const bool fold_read = d->state_dtype == XHC_BF16;
  int32_t* idx_id = reinterpret_cast<int32_t*>(ws + w.idx_id);
  float* hres_use = last ? const_cast<float*>(Hres) : F32(w.hres_id);
  hipError_t e = hipSuccess;
  // zero the dummy operands (weights of the absent pre-map and router, the
  // saved logits the recompute leaves empty), and for q < Q the residual
  // mapping that sublayer does not have
  if (!saved_act)
    XHC_STEP("fbwd_zero", launch_fill0(ws + w.saved, (size_t)T * saved_floats(k, k, Kq) * sizeof(float), s));
  XHC_STEP("fbwd_zero", launch_fill0(ws + w.w0, w.wres0 - w.w0, s));   // w0, colsum0
  if (!last) XHC_STEP("fbwd_zero", launch_fill0(ws + w.wres0, w.alpha2 - w.wres0, s));   // wres0, bres0
  // slot map, identity mixing, pre-map weights of the active streams, <d input_q, a_j>
  XHC_STEP("fbwd_token", launch_fbwd_token(d->state_dtype, T, d->N, (int)k, (int)C, idx, Hpre_q, d_input, Xact,
                                           idx_id, last ? nullptr : F32(w.hres_id), F32(w.hsel), dHpre_act, s));
  if (last) XHC_STEP("fbwd_gather", launch_fbwd_gather(d->state_dtype, T, d->N, (int)k, (int)C, idx, dXn, dA, s));
  // write-back reverse on the active rows: dF, dH^post, dp and the mixing
  // transpose, reading the saved rows and F in the state dtype, the fp32
  // active-row gradient, and writing dF in the state dtype (in place for a
  // bf16 state: each thread reads all k incoming rows of its chunk before it
  // writes the outgoing ones)
  float* const dA_out = fold_read ? dA : F32(w.da_out);
  const xhc_dims rs = dims_rows(d, Kq);
  XHC_STEP("fbwd_post", launch_bwd_post(&rs, dA, nullptr, Xact, F, conv_w, idx_id, p, hres_use, Hpost, dA_out,
                                        dF, F32(w.dhres), F32(w.dhpost), F32(w.dp), dconv_w, ws + w.post, s,
                                        /*grad_f32=*/true));
  XHC_STEP("fbwd_dp", launch_fbwd_add(dp, F32(w.dp), T * k, s));
  if (!last) XHC_STEP("fbwd_zero", launch_fill0(ws + w.dhres, (size_t)T * k * k * sizeof(float), s));
  // the mapping logits of sublayer q: saved by the forward, or recomputed
  // from a^(q-1) (same kernels and operands as the forward)
  const int64_t na = act_outs(d, Kq, last);
  const int nsave = saved_floats((int)k, (int)k, Kq);
  const float* rec = saved_act ? saved_act : F32(w.saved);
  if (!saved_act) {
    XHC_STEP("fbwd_proj", launch_proj_partial(d->state_dtype, Xact, T, (int)k, (int)C, kC, packed_act, na, idx_id,
                                              (int)k, F32(w.part), s));
    XHC_STEP("fbwd_coef", launch_pre_coef(F32(w.part), proj_chunks(d->state_dtype, true, kC, (int)C, na, T), na, T,
                                          (int)k, Kq, last, C, alpha_post, last ? alpha_res : nullptr, b_post,
                                          last ? b_res : nullptr, d->eps, d->sinkhorn_iters, d->clamp_delta,
                                          F32(w.hpost_re), last ? F32(w.hres_re) : nullptr, F32(w.sums), F32(w.saved),
                                          nsave, 2 * (int)k, nsave - 2, s));
  }
  XHC_STEP("fbwd_alpha", launch_fbwd_alpha(nullptr, alpha_res, alpha_post, F32(w.alpha2), s));
  // mapping reverse through a^(q-1) (its dense-row terms are all zero here:
  // no router or pre-map weights)
  // (the fp32 view's own row pass reads Xact only for an fp32 state; a bf16
  // state goes through the MFMA pass on Xact as saved)
  XHC_STEP("fbwd_pre", launch_bwd_pre(&r, Xact, F32(w.colsum0), F32(w.w0), F32(w.w0),
                                      last ? W_res : F32(w.wres0), W_post, F32(w.alpha2),
                                      last ? b_res : F32(w.bres0), rec, idx_id, p, F32(w.hsel), Hpost,
                                      nullptr, F32(w.dhres), F32(w.dhpost), F32(w.dp), dA_out,
                                      F32(w.dwr), F32(w.dwpre), last ? dW_res : F32(w.dwres), dW_post,
                                      F32(w.dalpha2), F32(w.dbpre), last ? db_res : F32(w.dbres), db_post,
                                      ws + w.pre, s, nullptr, nullptr, /*dense_rows=*/false,
                                      d->state_dtype == XHC_BF16 ? Xact : nullptr, /*act_rows=*/true, kBwdPreAll,
                                      fold_read && reads ? d_input : nullptr));
  XHC_STEP("fbwd_copy", hipMemcpyAsync(dalpha_post, F32(w.dalpha2) + 2, sizeof(float), hipMemcpyDeviceToDevice, s));
  if (last)
    XHC_STEP("fbwd_copy", hipMemcpyAsync(dalpha_res, F32(w.dalpha2) + 1, sizeof(float), hipMemcpyDeviceToDevice, s));
  // da = (reverse so far) + H^pre,q_{I_j} d input_q (the active part of
  // input_q's read): added by the active-row pass for a bf16 state, here
  // otherwise
  if (!fold_read)
    XHC_STEP("fbwd_finish", launch_fbwd_finish(d->state_dtype, T, (int)k, (int)C, F32(w.da_out), F32(w.hsel),
                                               reads ? d_input : nullptr, dA, s));
  return hip_status(e);
}

xhc_status xhc_flash_pre_bwd(const xhc_dims* d, int32_t Q, const void* X, const void* packed_full, const float* W_r,
                             const float* W_pre, const float* alpha_pre, const float* b_pre, const int32_t* idx,
                             const float* p, const float* Hpre, const float* saved, const void* d_input,
                             const float* dHpre_act, const float* dp, const void* dXn, const void* da0, void* dX,
                             float* dW_r, float* dW_pre, float* dalpha_pre, float* db_pre, void* workspace,
                             size_t workspace_bytes, void* stream) {
  xhc_status st = check_dims(d);
  if (st != XHC_OK) return st;
  if (Q != 2 && Q != 4) return XHC_EINVAL;
  if ((int64_t)(Q + 1) * d->N > 128 || !flash_bwd_supported(d)) return XHC_EUNSUPPORTED;
  if (d->T == 0) return XHC_OK;
  if (!X || !packed_full || !W_r || !W_pre || !alpha_pre || !b_pre || !idx || !p || !Hpre || !d_input ||
      !dHpre_act || !dp || !dXn || !da0 || !dX || !dW_r || !dW_pre || !dalpha_pre || !db_pre || !workspace)
    return XHC_EINVAL;
  if (dX == X || dX == da0) return XHC_EINVAL;   // dX == dXn: in place
  if (!aligned16(X) || !aligned16(packed_full) || !aligned16(d_input) || !aligned16(dXn) || !aligned16(da0) ||
      !aligned16(dX) || !aligned16(workspace))
    return XHC_EUNSUPPORTED;
  const FlashPreBwdWs w = flash_pre_bwd_ws(d, Q);
  if (workspace_bytes < w.total) return XHC_EWORKSPACE;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  clear_stale_error();
  char* ws = reinterpret_cast<char*>(workspace);
  auto F32 = [&](size_t at) { return reinterpret_cast<float*>(ws + at); };
  const int64_t T = d->T, N = d->N, k = d->k, C = d->C, NC = N * C;
  const size_t es = d->state_dtype == XHC_BF16 ? 2 : 4;   // d_input
  const int64_t nf = (int64_t)(Q + 1) * N;
  const xhc_dims en = dims_entry(d);
  const int nsave = saved_floats((int)N, (int)k, 1);
  const float* colsum = reinterpret_cast<const float*>(reinterpret_cast<const char*>(packed_full) +
                                                       packed_frag_bytes(NC, nf));
  hipError_t e = hipSuccess;
  if (!saved) XHC_STEP("fpbwd_zero", launch_fill0(ws + w.saved, (size_t)T * nsave * sizeof(float), s));
  XHC_STEP("fpbwd_zero", launch_fill0(ws + w.wpost0, w.alpha_e - w.wpost0, s));   // zero operands
  // the group-entry logits and statistics: saved by the forward, or
  // recomputed as the forward made them
  if (!saved)
    XHC_STEP("fpbwd_proj", launch_proj_partial(d->state_dtype, X, T, (int)N, (int)C, NC, packed_full, nf, nullptr,
                                               (int)k, F32(w.part), s));
  // dL/dX starts as the gradient of the state after the group: the untouched
  // streams pass it through, the active ones carry the reverse of the group
  XHC_STEP("fpbwd_scatter", launch_fbwd_scatter(d->state_dtype, T, (int)N, (int)k, (int)C, idx,
                                                 dX == dXn ? nullptr : dXn, reinterpret_cast<const float*>(da0), dX,
                                                 s));
  // pre-map q + 1 (and the router with the first): dL/dH^pre,q+1 of the active
  // streams comes from the sublayer reverse (q >= 1); the base readouts of q >=
  // 1 leave the active streams out.  This view has no active-row projection
  // (H^post and H^res are reversed per sublayer), so the active-row pass is
  // left out.  Where supported the Q full-row passes run as one pass over the
  // state (token records first, then the fused rows, then the reductions).
  const float* hrd[4] = {nullptr, nullptr, nullptr, nullptr};
  char* wsq[4] = {nullptr, nullptr, nullptr, nullptr};
  auto pass = [&](int q, int phase) -> hipError_t {
    char* wq = ws + w.pre + (w.fused ? (size_t)q * w.pre_slice : 0);
    float* hm = F32(w.hmask) + (int64_t)q * T * N;
    const float* rec = saved ? saved + (int64_t)q * T * nsave : F32(w.saved);   // pre-map q's records
    if (phase != kBwdPreReduce) {
      hipError_t e1 = hipSuccess;
      if (!saved)
        e1 = launch_pre_route(F32(w.part), proj_chunks(d->state_dtype, false, NC, (int)C, nf, T), nf, T,
                              (int)N, d->m, (int)k, Q, C, colsum, alpha_pre, 1, b_pre, d->eps,
                              reinterpret_cast<int32_t*>(ws + w.idx_s), F32(w.p_s), F32(w.hpre_s),
                              F32(w.sums), F32(w.saved), nsave, nsave - 4, d->router, s, q);
      if (e1 == hipSuccess) e1 = launch_fbwd_alpha(alpha_pre + q, nullptr, nullptr, F32(w.alpha_e), s);
      if (e1 == hipSuccess && q >= 1) e1 = launch_fbwd_mask(T, (int)N, (int)k, idx, Hpre + (int64_t)q * T * N, hm, s);
      if (e1 != hipSuccess) return e1;
    }
    hrd[q] = q >= 1 ? hm : Hpre;
    wsq[q] = wq;
    return launch_bwd_pre(&en, X, colsum, W_r, W_pre + (int64_t)q * NC * N, F32(w.wres0), F32(w.wpost0),
                          F32(w.alpha_e), F32(w.bres0), rec, idx, p, Hpre + (int64_t)q * T * N,
                          F32(w.hpost0), reinterpret_cast<const char*>(d_input) + (size_t)q * T * C * es,
                          F32(w.dhres0), F32(w.dhpost0), q == 0 ? dp : F32(w.dp0), dX, q == 0 ? dW_r : F32(w.dwr),
                          dW_pre + (int64_t)q * NC * N, F32(w.dwres), F32(w.dwpost), F32(w.dalpha),
                          db_pre + (int64_t)q * N, F32(w.dbres), F32(w.dbpost), wq, s,
                          q >= 1 ? dHpre_act + (int64_t)(q - 1) * T * k : nullptr, q >= 1 ? hm : nullptr,
                          /*dense_rows=*/true, /*X_bf16=*/nullptr, /*act_rows=*/false, phase);
  };
  if (w.fused) {
    for (int q = 0; q < Q; ++q) wsq[q] = ws + w.pre + (size_t)q * w.pre_slice;
    XHC_STEP("fpbwd_dhpre", launch_bwd_dhpre_multi(&en, Q, X, d_input, wsq, s));
    for (int q = 0; q < Q && e == hipSuccess; ++q) XHC_STEP("fpbwd_tokens", pass(q, kBwdPreTokensGiven));
    XHC_STEP("fpbwd_rows", launch_bwd_rows_multi(&en, Q, X, dX, W_r, W_pre, d_input, hrd, wsq, F32(w.multi), s));
    for (int q = 0; q < Q && e == hipSuccess; ++q) {
      XHC_STEP("fpbwd_reduce", pass(q, kBwdPreReduce));
      XHC_STEP("fpbwd_copy", hipMemcpyAsync(dalpha_pre + q, F32(w.dalpha), sizeof(float), hipMemcpyDeviceToDevice, s));
    }
  } else {
    for (int q = 0; q < Q && e == hipSuccess; ++q) {
      XHC_STEP("fpbwd_pre", pass(q, kBwdPreAll));
      XHC_STEP("fpbwd_copy", hipMemcpyAsync(dalpha_pre + q, F32(w.dalpha), sizeof(float), hipMemcpyDeviceToDevice, s));
    }
  }
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

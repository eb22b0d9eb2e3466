// Helpers of the xHC-Flash backward (reverse mode of xhc_flash_pre and
// xhc_flash_post; Alg. "xHC-Flash: one Transformer block", App. E.2).
//
// The group is reversed sublayer by sublayer on the k active rows of each
// token, slot order, [T, k, C]:
//  - the write-back of sublayer q (a^(q) = M_q a^(q-1) + p (H^post,q out_aug),
//    M_q = H^res for q = Q, the identity before) is the single-sublayer
//    post reverse on a state of k rows that are all active (identity slot map);
//  - the mappings H^post,q (and H^res) come from a^(q-1) through the
//    active-row projection, so their reverse is the single-sublayer pre
//    reverse on that k-row state with every stream fixed (no router) and no
//    pre-map weights;
//  - the input of sublayer q >= 2 reads the active rows a^(q-1) with the
//    weights H^pre,q of their streams (eq:app_active_state_correction):
//    their gradient adds H^pre,q_{I_j} d input_q, and the weights receive
//    <d input_q, a^(q-1)_j>.
// The group-entry state is then reversed once per pre-map (router with the
// first), with dH^pre,q of the active streams taken from the step above and
// the base readouts leaving the active streams out.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {
namespace {

__global__ __launch_bounds__(256) void k_fill0(uint4* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = make_uint4(0, 0, 0, 0);
}

// Per token (one workgroup): the identity slot map, the identity mixing
// matrix (when Hres_id is given), the pre-map weights of the active streams
// Hsel[t, j] = Hpre_q[t, idx[t, j]] (0 without Hpre_q) and, when din is
// given, dhact[t, j] = <din[t], Xact[t, j]> summed in a fixed order.
template <typename TS>
__global__ __launch_bounds__(256) void k_fbwd_token(int64_t T, int N, int k, int C, const int32_t* __restrict__ idx,
                                                    const float* __restrict__ Hpre_q, const TS* __restrict__ din,
                                                    const TS* __restrict__ Xact, int32_t* __restrict__ idx_id,
                                                    float* __restrict__ Hres_id, float* __restrict__ Hsel,
                                                    float* __restrict__ dhact) {
  const int64_t t = blockIdx.x;
  if (t >= T) return;
  if (threadIdx.x < k) {
    const int j = threadIdx.x;
    idx_id[t * k + j] = j;
    if (Hres_id)
      for (int l = 0; l < k; ++l) Hres_id[(t * k + j) * k + l] = (j == l) ? 1.0f : 0.0f;
    Hsel[t * k + j] = Hpre_q ? Hpre_q[t * N + idx[t * k + j]] : 0.0f;
  }
  if (!din) return;
  __shared__ float red[kMaxK][256 / kWave];
  float acc[kMaxK];
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) acc[j] = 0.f;
  for (int c = threadIdx.x * 8; c < C; c += 256 * 8) {
    float g[8];
    Vec8<TS>::load(din + t * C + c, g);
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j >= k) break;
      float a[8];
      Vec8<TS>::load(Xact + (t * k + j) * (int64_t)C + c, a);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[j] = fmaf(g[e], a[e], acc[j]);
    }
  }
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j >= k) break;
    const float v = wave_sum(acc[j]);
    if (lane == 0) red[j][wave] = v;
  }
  __syncthreads();
  if (threadIdx.x < k) {
    float v = 0.f;
    for (int w = 0; w < 256 / kWave; ++w) v += red[threadIdx.x][w];
    dhact[t * k + threadIdx.x] = v;
  }
}

// da[t, j, :] = dXn[t, idx[t, j], :] as fp32 (one workgroup per active row)
template <typename TS>
__global__ __launch_bounds__(256) void k_fbwd_gather(int64_t T, int N, int k, int C, const int32_t* __restrict__ idx,
                                                     const TS* __restrict__ dXn, float* __restrict__ da) {
  const int64_t r = blockIdx.x, t = r / k;
  const int j = (int)(r % k), i = idx[t * k + j];
  const TS* src = dXn + (t * N + i) * (int64_t)C;
  float* dst = da + (t * k + j) * (int64_t)C;
  for (int c = threadIdx.x * 8; c < C; c += 256 * 8) {
    float f[8];
    Vec8<TS>::load(src + c, f);
    Vec8<float>::store(dst + c, f);
  }
}

// dX[t, i, :] = da0[t, j, :] (fp32, rounded to the state dtype) where stream
// i sits in slot j, else GX[t, i, :] (one workgroup per state row)
template <typename TS>
__global__ __launch_bounds__(256) void k_fbwd_scatter(int64_t T, int N, int k, int C, const int32_t* __restrict__ idx,
                                                      const TS* __restrict__ GX, const float* __restrict__ da0,
                                                      TS* __restrict__ dX) {
  const int64_t row = blockIdx.x, t = row / N;
  const int i = (int)(row % N);
  int slot = -1;
  for (int j = 0; j < k; ++j)
    if (idx[t * k + j] == i) slot = j;
  TS* dst = dX + row * (int64_t)C;
  for (int c = threadIdx.x * 8; c < C; c += 256 * 8) {
    float f[8];
    if (slot >= 0) Vec8<float>::load(da0 + (t * k + slot) * (int64_t)C + c, f);
    else Vec8<TS>::load(GX + row * (int64_t)C + c, f);
    Vec8<TS>::store(dst + c, f);
  }
}

// the same in place: row (t, I_j) of dX = slot j of da0 (one workgroup per
// active row; the other rows already hold G_X)
template <typename TS>
__global__ __launch_bounds__(256) void k_fbwd_scatter_act(int64_t T, int N, int k, int C,
                                                          const int32_t* __restrict__ idx,
                                                          const float* __restrict__ da0, TS* __restrict__ dX) {
  const int64_t r = blockIdx.x, t = r / k;
  const int j = (int)(r % k);
  TS* dst = dX + (t * N + idx[t * k + j]) * (int64_t)C;
  for (int c = threadIdx.x * 8; c < C; c += 256 * 8) {
    float f[8];
    Vec8<float>::load(da0 + r * (int64_t)C + c, f);
    Vec8<TS>::store(dst + c, f);
  }
}

// Hm[t, i] = 0 for the active streams of token t, Hpre[t, i] otherwise
__global__ __launch_bounds__(256) void k_fbwd_mask(int64_t T, int N, int k, const int32_t* __restrict__ idx,
                                                   const float* __restrict__ Hpre, float* __restrict__ Hm) {
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= T * N) return;
  const int64_t t = u / N;
  const int i = (int)(u % N);
  bool act = false;
  for (int j = 0; j < k; ++j) act = act || idx[t * k + j] == i;
  Hm[u] = act ? 0.0f : Hpre[u];
}

__global__ __launch_bounds__(256) void k_fbwd_add(float* __restrict__ dst, const float* __restrict__ src, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] += src[i];
}

// out = (a0, a1, a2), each from its device scalar or 0 where the pointer is null
__global__ void k_fbwd_alpha(const float* a0, const float* a1, const float* a2, float* out) {
  if (threadIdx.x == 0) {
    out[0] = a0 ? *a0 : 0.0f;
    out[1] = a1 ? *a1 : 0.0f;
    out[2] = a2 ? *a2 : 0.0f;
  }
}

// da[t, j, :] = da_rev[t, j, :] + Hsel[t, j] din[t, :] (din null: a copy),
// one workgroup per active row
template <typename TS>
__global__ __launch_bounds__(256) void k_fbwd_finish(int k, int C, const float* __restrict__ da_rev,
                                                     const float* __restrict__ Hsel, const TS* __restrict__ din,
                                                     float* __restrict__ da) {
  const int64_t r = blockIdx.x, t = r / k;
  const float h = din ? Hsel[r] : 0.0f;
  for (int c = threadIdx.x * 8; c < C; c += 256 * 8) {
    float f[8], g[8];
    Vec8<float>::load(da_rev + r * C + c, f);
    if (din) {
      Vec8<TS>::load(din + t * C + c, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = fmaf(h, g[e], f[e]);
    }
    Vec8<float>::store(da + r * C + c, f);
  }
}

unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

#define XHC_FTS(dt, ...)                    \
  do {                                      \
    if ((dt) == XHC_BF16) {                 \
      using TS = uint16_t;                  \
      __VA_ARGS__;                          \
    } else {                                \
      using TS = float;                     \
      __VA_ARGS__;                          \
    }                                       \
  } while (0)

hipError_t launch_fill0(void* p, size_t bytes, hipStream_t s) {
  const int64_t n = (int64_t)(bytes / 16);
  if (n == 0) return hipSuccess;
  k_fill0<<<dim3(blocks_for(n, 256)), dim3(256), 0, s>>>(reinterpret_cast<uint4*>(p), n);
  return hipGetLastError();
}

hipError_t launch_fbwd_token(int state_dtype, int64_t T, int N, int k, int C, const int32_t* idx,
                             const float* Hpre_q, const void* din, const void* Xact, int32_t* idx_id, float* Hres_id,
                             float* Hsel, float* dhact, hipStream_t s) {
  XHC_FTS(state_dtype, k_fbwd_token<TS><<<dim3((unsigned)T), dim3(256), 0, s>>>(
                           T, N, k, C, idx, Hpre_q, reinterpret_cast<const TS*>(din),
                           reinterpret_cast<const TS*>(Xact), idx_id, Hres_id, Hsel, dhact));
  return hipGetLastError();
}

hipError_t launch_fbwd_gather(int state_dtype, int64_t T, int N, int k, int C, const int32_t* idx, const void* dXn,
                              float* da, hipStream_t s) {
  XHC_FTS(state_dtype, k_fbwd_gather<TS><<<dim3((unsigned)(T * k)), dim3(256), 0, s>>>(
                           T, N, k, C, idx, reinterpret_cast<const TS*>(dXn), da));
  return hipGetLastError();
}

hipError_t launch_fbwd_scatter(int state_dtype, int64_t T, int N, int k, int C, const int32_t* idx, const void* GX,
                               const float* da0, void* dX, hipStream_t s) {
  if (!GX) {   // in place: dX holds G_X; only the active rows change
    XHC_FTS(state_dtype, k_fbwd_scatter_act<TS><<<dim3((unsigned)(T * k)), dim3(256), 0, s>>>(
                             T, N, k, C, idx, da0, reinterpret_cast<TS*>(dX)));
    return hipGetLastError();
  }
  XHC_FTS(state_dtype, k_fbwd_scatter<TS><<<dim3((unsigned)(T * N)), dim3(256), 0, s>>>(
                           T, N, k, C, idx, reinterpret_cast<const TS*>(GX), da0, reinterpret_cast<TS*>(dX)));
  return hipGetLastError();
}

hipError_t launch_fbwd_mask(int64_t T, int N, int k, const int32_t* idx, const float* Hpre, float* Hm, hipStream_t s) {
  k_fbwd_mask<<<dim3(blocks_for(T * N, 256)), dim3(256), 0, s>>>(T, N, k, idx, Hpre, Hm);
  return hipGetLastError();
}

hipError_t launch_fbwd_add(float* dst, const float* src, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  k_fbwd_add<<<dim3(blocks_for(n, 256)), dim3(256), 0, s>>>(dst, src, n);
  return hipGetLastError();
}

hipError_t launch_fbwd_alpha(const float* a0, const float* a1, const float* a2, float* out, hipStream_t s) {
  k_fbwd_alpha<<<dim3(1), dim3(64), 0, s>>>(a0, a1, a2, out);
  return hipGetLastError();
}

hipError_t launch_fbwd_finish(int state_dtype, int64_t T, int k, int C, const float* da_rev, const float* Hsel,
                              const void* din, float* da, hipStream_t s) {
  XHC_FTS(state_dtype, k_fbwd_finish<TS><<<dim3((unsigned)(T * k)), dim3(256), 0, s>>>(
                           k, C, da_rev, Hsel, reinterpret_cast<const TS*>(din), da));
  return hipGetLastError();
}

#undef XHC_FTS

}  // namespace xhc

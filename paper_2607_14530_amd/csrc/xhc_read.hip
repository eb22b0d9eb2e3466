// Dense read of eq:dense_read (and the xHC-Flash non-active bases): the
// pre-mapped combination of the N streams of every token.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {

// ----------------------------------------------------------------- dense read
// out[q][t][c] = sum_i w_q[t][i] X[t][i][c] with w_q = Hpre[q][t][:]; for q >= 1
// the active streams idx[t][:] are left out (xHC-Flash non-active bases,
// App. E.2 eq:app_four_sub_base).  One thread per 8 channels of one token.

template <typename TS, int NMAP>
__global__ __launch_bounds__(256) void k_dense_read(const TS* __restrict__ X, int64_t T, int N, int C,
                                                    const float* __restrict__ Hpre,
                                                    const int32_t* __restrict__ idx, int k,
                                                    TS* __restrict__ out0, TS* __restrict__ outr) {
  const int64_t ncb = ((int64_t)C / 8 + 255) / 256;
  const int64_t t = blockIdx.x / ncb;
  const int c = (int)((blockIdx.x % ncb) * 256 + threadIdx.x) * 8;
  if (c >= C) return;
  uint64_t act = 0;
  if (NMAP > 1)
    for (int j = 0; j < k; ++j) act |= 1ull << idx[t * k + j];
  float acc[NMAP][8];
#pragma unroll
  for (int q = 0; q < NMAP; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[q][e] = 0.f;
  const TS* xt = X + t * (int64_t)N * C + c;
  // stream rows loaded before use, kept in the storage format until then
  constexpr int UNR = 8;
  using R8 = Raw8<TS>;
  for (int i0 = 0; i0 < N; i0 += UNR) {
    typename R8::raw r[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (i0 + u < N) r[u] = R8::load(xt + (int64_t)(i0 + u) * C);
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u;
      if (i < N) {
        float f[8];
        R8::unpack(r[u], f);
#pragma unroll
        for (int q = 0; q < NMAP; ++q) {
          float w = Hpre[((int64_t)q * T + t) * N + i];
          if (q > 0 && ((act >> i) & 1ull)) w = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[q][e] = fmaf(w, f[e], acc[q][e]);
        }
      }
    }
  }
  Vec8<TS>::store(out0 + t * C + c, acc[0]);
#pragma unroll
  for (int q = 1; q < NMAP; ++q) Vec8<TS>::store(outr + ((int64_t)(q - 1) * T + t) * C + c, acc[q]);
}

template <typename TS>
static hipError_t dense_dispatch(const TS* X, int64_t T, int N, int C, const float* Hpre, int nmap,
                                 const int32_t* idx, int k, TS* out0, TS* outr, hipStream_t s) {
  const dim3 grid((unsigned)(T * ((C / 8 + 255) / 256)));
  switch (nmap) {
    case 1: k_dense_read<TS, 1><<<grid, dim3(256), 0, s>>>(X, T, N, C, Hpre, idx, k, out0, outr); break;
    case 2: k_dense_read<TS, 2><<<grid, dim3(256), 0, s>>>(X, T, N, C, Hpre, idx, k, out0, outr); break;
    case 4: k_dense_read<TS, 4><<<grid, dim3(256), 0, s>>>(X, T, N, C, Hpre, idx, k, out0, outr); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_dense_read(int state_dtype, const void* X, int64_t T, int N, int C, const float* Hpre,
                             int nmap, const int32_t* idx, int k, void* out0, void* outr, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (state_dtype == XHC_BF16)
    return dense_dispatch<uint16_t>(reinterpret_cast<const uint16_t*>(X), T, N, C, Hpre, nmap, idx, k,
                                    reinterpret_cast<uint16_t*>(out0), reinterpret_cast<uint16_t*>(outr), s);
  return dense_dispatch<float>(reinterpret_cast<const float*>(X), T, N, C, Hpre, nmap, idx, k,
                               reinterpret_cast<float*>(out0), reinterpret_cast<float*>(outr), s);
}

// ----------------------------------------------------------------- final stream reduction
// out[t, c] = sum_{i < N} X[t, i, c] (fp32, streams in order), one thread per
// 8 channels of a token, 8 rows in flight.
template <typename TS>
__global__ __launch_bounds__(256) void k_stream_sum(const TS* __restrict__ X, int64_t T, int N, int C,
                                                    TS* __restrict__ out) {
  using R8 = Raw8<TS>;
  constexpr int UNR = 8;
  const int64_t cb = (C / 8 + 255) / 256;
  const int64_t t = blockIdx.x / cb;
  const int c = (int)((blockIdx.x % cb) * 256 + threadIdx.x) * 8;
  if (t >= T || c >= C) return;
  const TS* xt = X + t * N * (int64_t)C + c;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int i0 = 0; i0 < N; i0 += UNR) {
    typename R8::raw r[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (i0 + u < N) r[u] = R8::load(xt + (int64_t)(i0 + u) * C);
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (i0 + u < N) {
        float f[8];
        R8::unpack(r[u], f);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += f[e];
      }
  }
  Vec8<TS>::store(out + t * C + c, acc);
}

// dX[t, i, c] = dout[t, c] (or += with accumulate) for every stream i
template <typename TS>
__global__ __launch_bounds__(256) void k_stream_bcast(const TS* __restrict__ dout, int64_t T, int N, int C,
                                                      int accumulate, TS* __restrict__ dX) {
  const int64_t cb = (C / 8 + 255) / 256;
  const int64_t t = blockIdx.x / cb;
  const int c = (int)((blockIdx.x % cb) * 256 + threadIdx.x) * 8;
  if (t >= T || c >= C) return;
  float g[8];
  Vec8<TS>::load(dout + t * C + c, g);
  for (int i = 0; i < N; ++i) {
    TS* p = dX + (t * N + i) * (int64_t)C + c;
    float f[8];
    if (accumulate) {
      Vec8<TS>::load(p, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] += g[e];
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = g[e];
    }
    Vec8<TS>::store(p, f);
  }
}

hipError_t launch_stream_sum(int state_dtype, const void* X, int64_t T, int N, int C, void* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)(T * ((C / 8 + 255) / 256)));
  if (state_dtype == XHC_BF16)
    k_stream_sum<uint16_t><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const uint16_t*>(X), T, N, C,
                                                        reinterpret_cast<uint16_t*>(out));
  else
    k_stream_sum<float><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const float*>(X), T, N, C,
                                                     reinterpret_cast<float*>(out));
  return hipGetLastError();
}

hipError_t launch_stream_bcast(int state_dtype, const void* dout, int64_t T, int N, int C, int accumulate, void* dX,
                               hipStream_t s) {
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)(T * ((C / 8 + 255) / 256)));
  if (state_dtype == XHC_BF16)
    k_stream_bcast<uint16_t><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const uint16_t*>(dout), T, N, C,
                                                          accumulate, reinterpret_cast<uint16_t*>(dX));
  else
    k_stream_bcast<float><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const float*>(dout), T, N, C, accumulate,
                                                       reinterpret_cast<float*>(dX));
  return hipGetLastError();
}

}  // namespace xhc

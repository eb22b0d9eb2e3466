// Sparse write-back of an xHC sublayer (eq:aug, eq:gs, eq:sparse_write_delta,
// eq:sparse_write).
//
//  k_post_gram   MLP-type only: per token and channel chunk, the Gram matrix of
//                the components e_0 = out, e_j = DWConv_kappa_j(out) (fp32)
//  k_post_coef   per token: Gram-Schmidt in the component basis folded with p
//                and H^post into write-back weights wb[t][j][b]
//  k_post_apply  X[t, I_j, :] <- sum_l H^res[j,l] X[t, I_l, :] + sum_b wb[j][b] e_b;
//                the other N - k rows are never touched
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {

// Gram partials: gpart[chunk][pair][t], pairs (a <= b) in row-major upper order.
template <typename TS, int KR>
__global__ __launch_bounds__(256) void k_post_gram(const TS* __restrict__ F, int64_t T, int64_t S, int C,
                                                   int kap0, int kap1, int kap2, const float* __restrict__ conv_w,
                                                   float* __restrict__ gpart) {
  constexpr int NP = KR * (KR + 1) / 2;
  __shared__ float red[4][NP];
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb;
  const int64_t cb = blockIdx.x % ncb;
  const int c = (int)(cb * 256 + threadIdx.x) * 8;
  const int kap[3] = {kap0, kap1, kap2};
  float g[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) g[i] = 0.f;
  if (c < C) {
    float e[KR][8];
    components<TS, KR>(F, conv_w, t, t % S, C, c, kap, e);
    int pi = 0;
#pragma unroll
    for (int a = 0; a < KR; ++a)
#pragma unroll
      for (int b = a; b < KR; ++b, ++pi)
#pragma unroll
        for (int q = 0; q < 8; ++q) g[pi] = fmaf(e[a][q], e[b][q], g[pi]);
  }
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    float v = g[i];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    g[i] = v;
  }
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (lane == 0)
#pragma unroll
    for (int i = 0; i < NP; ++i) red[wave][i] = g[i];
  __syncthreads();
  if ((int)threadIdx.x < NP) {
    const int i = threadIdx.x;
    gpart[(cb * NP + i) * T + t] = red[0][i] + red[1][i] + red[2][i] + red[3][i];
  }
}

hipError_t launch_post_gram(int state_dtype, const void* F, int64_t T, int64_t S, int C, int Kr,
                            const int32_t* kappa, const float* conv_w, float* gpart, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)(T * post_chunks(C)));
#define XHC_GRAM(TS, KR)                                                                                   \
  k_post_gram<TS, KR><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const TS*>(F), T, S, C, kappa[0], kappa[1], \
                                                 kappa[2], conv_w, gpart)
  if (state_dtype == XHC_BF16) {
    if (Kr == 2) XHC_GRAM(uint16_t, 2); else if (Kr == 3) XHC_GRAM(uint16_t, 3); else XHC_GRAM(uint16_t, 4);
  } else {
    if (Kr == 2) XHC_GRAM(float, 2); else if (Kr == 3) XHC_GRAM(float, 3); else XHC_GRAM(float, 4);
  }
#undef XHC_GRAM
  return hipGetLastError();
}

// Per token: G = sum over chunks; v_r = sum_b V[r][b] e_b (Gram-Schmidt, eq:gs);
// wb[j][b] = p_j sum_r H^post[j][r] V[r][b]  (p gates only the write-back term).
__global__ __launch_bounds__(128) void k_post_coef(const float* __restrict__ gpart, int64_t nchunk, int64_t T,
                                                   int k, int Kr, int gram_schmidt, const float* __restrict__ p,
                                                   const float* __restrict__ Hpost, float* __restrict__ wb) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int NP = Kr * (Kr + 1) / 2;
  double G[kMaxKr][kMaxKr];
  int pi = 0;
#pragma unroll
  for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
    for (int b = a; b < kMaxKr; ++b) {
      if (a < Kr && b < Kr) {
        float s = 0.f;
        for (int64_t c = 0; c < nchunk; ++c) s += gpart[(c * NP + pi) * T + t];
        G[a][b] = G[b][a] = s;
        ++pi;
      } else {
        G[a][b] = G[b][a] = 0.0;
      }
    }
  double V[kMaxKr][kMaxKr];
  if (gram_schmidt) {
    gram_schmidt_basis(G, Kr, V);
  } else {
#pragma unroll
    for (int i = 0; i < kMaxKr; ++i)
#pragma unroll
      for (int b = 0; b < kMaxKr; ++b) V[i][b] = (i == b) ? 1.0 : 0.0;
  }
  for (int j = 0; j < k; ++j) {
    const double pj = p[t * k + j];
    for (int b = 0; b < Kr; ++b) {
      double s = 0.0;
      for (int r = 0; r < Kr; ++r) s += (double)Hpost[(t * k + j) * Kr + r] * V[r][b];
      wb[(t * k + j) * Kr + b] = (float)(pj * s);
    }
  }
}

hipError_t launch_post_coef(const float* gpart, int64_t nchunk, int64_t T, int k, int Kr, int gram_schmidt,
                            const float* p, const float* Hpost, float* wb, hipStream_t s) {
  if (T == 0) return hipSuccess;
  k_post_coef<<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(gpart, nchunk, T, k, Kr, gram_schmidt, p,
                                                                      Hpost, wb);
  return hipGetLastError();
}

// In-place update of the k active rows of one token, 8 channels per thread.
// All k rows are read before any is written; each thread owns its channels.
// Hres == nullptr means no residual mixing (an intermediate xHC-Flash
// sublayer, eq:flash_attn_update).  With input_next, the thread also forms
// the next sublayer's input from its non-active base and the active rows as
// stored (App. E.2, eq:app_active_state_correction).
template <typename TS, int KR>
__global__ __launch_bounds__(256) void k_post_apply(TS* __restrict__ X, const TS* __restrict__ F, int64_t T,
                                                    int64_t S, int N, int C, int k, int kap0, int kap1, int kap2,
                                                    const float* __restrict__ conv_w,
                                                    const int32_t* __restrict__ idx, const float* __restrict__ p,
                                                    const float* __restrict__ Hres,
                                                    const float* __restrict__ Hpost,
                                                    const float* __restrict__ wb,
                                                    const float* __restrict__ Hpre_next,
                                                    const TS* __restrict__ base_next,
                                                    TS* __restrict__ input_next, TS* __restrict__ Xact_save) {
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb;
  const int c = (int)((blockIdx.x % ncb) * 256 + threadIdx.x) * 8;
  if (c >= C) return;
  const int kap[3] = {kap0, kap1, kap2};
  float e[KR][8];
  components<TS, KR>(F, conv_w, t, t % S, C, c, kap, e);
  float a[kMaxK][8];
  int32_t rows[kMaxK];
#pragma unroll
  for (int l = 0; l < kMaxK; ++l) {
    if (l < k) {
      rows[l] = idx[t * k + l];
      Vec8<TS>::load(X + (t * N + rows[l]) * (int64_t)C + c, a[l]);
      if (Xact_save) Vec8<TS>::store(Xact_save + (t * k + l) * (int64_t)C + c, a[l]);
    }
  }
  float nxt[8];
  if (input_next) Vec8<TS>::load(base_next + t * C + c, nxt);
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j >= k) break;
    float y[8];
    if (Hres) {
#pragma unroll
      for (int q = 0; q < 8; ++q) y[q] = 0.f;
#pragma unroll
      for (int l = 0; l < kMaxK; ++l) {
        if (l < k) {
          const float h = Hres[(t * k + j) * k + l];
#pragma unroll
          for (int q = 0; q < 8; ++q) y[q] = fmaf(h, a[l][q], y[q]);
        }
      }
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) y[q] = a[j][q];
    }
#pragma unroll
    for (int b = 0; b < KR; ++b) {
      const float w = (KR == 1) ? p[t * k + j] * Hpost[t * k + j] : wb[(t * k + j) * KR + b];
#pragma unroll
      for (int q = 0; q < 8; ++q) y[q] = fmaf(w, e[b][q], y[q]);
    }
    Vec8<TS>::store(X + (t * N + rows[j]) * (int64_t)C + c, y);
    if (input_next) {
      Vec8<TS>::round(y);
      const float h = Hpre_next[t * N + rows[j]];
#pragma unroll
      for (int q = 0; q < 8; ++q) nxt[q] = fmaf(h, y[q], nxt[q]);
    }
  }
  if (input_next) Vec8<TS>::store(input_next + t * C + c, nxt);
}

hipError_t launch_post_apply(int state_dtype, void* X, const void* F, int64_t T, int64_t S, int N, int C, int k,
                             int Kr, const int32_t* kappa, const float* conv_w, const int32_t* idx, const float* p,
                             const float* Hres, const float* Hpost, const float* wb, const float* Hpre_next,
                             const void* base_next, void* input_next, void* Xact_save, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const dim3 grid((unsigned)(T * post_chunks(C)));
#define XHC_APPLY(TS, KR)                                                                                       \
  k_post_apply<TS, KR><<<grid, dim3(256), 0, s>>>(reinterpret_cast<TS*>(X), reinterpret_cast<const TS*>(F), T, S, \
                                                  N, C, k, kappa[0], kappa[1], kappa[2], conv_w, idx, p, Hres,   \
                                                  Hpost, wb, Hpre_next, reinterpret_cast<const TS*>(base_next),  \
                                                  reinterpret_cast<TS*>(input_next), reinterpret_cast<TS*>(Xact_save))
  if (state_dtype == XHC_BF16) {
    switch (Kr) {
      case 1: XHC_APPLY(uint16_t, 1); break;
      case 2: XHC_APPLY(uint16_t, 2); break;
      case 3: XHC_APPLY(uint16_t, 3); break;
      default: XHC_APPLY(uint16_t, 4); break;
    }
  } else {
    switch (Kr) {
      case 1: XHC_APPLY(float, 1); break;
      case 2: XHC_APPLY(float, 2); break;
      case 3: XHC_APPLY(float, 3); break;
      default: XHC_APPLY(float, 4); break;
    }
  }
#undef XHC_APPLY
  return hipGetLastError();
}

}  // namespace xhc

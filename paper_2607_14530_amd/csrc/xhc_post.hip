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


// ------------------------------------------------------------------ run-based MLP-type kernels
// For compile-time kernel sizes (K1, K2, K3) = (4, 8, 12): a thread owns 4
// channels and walks a run of kRun consecutive tokens, keeping the 24 conv taps
// of its channels and a sliding window of the last 12 outputs in registers,
// so F is read once per kernel and the taps once per run.

constexpr int kRun = 64;

template <typename TS> struct Vec4;
template <> struct Vec4<uint16_t> {
  static __device__ __forceinline__ void load(const uint16_t* p, float (&f)[4]) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    f[0] = bf_lo(v.x); f[1] = bf_hi(v.x); f[2] = bf_lo(v.y); f[3] = bf_hi(v.y);
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float (&f)[4]) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack2bf(f[0], f[1]), pack2bf(f[2], f[3]));
  }
  static __device__ __forceinline__ void round(float (&f)[4]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(f2bf(f[e]) << 16);
  }
};
template <> struct Vec4<float> {
  static __device__ __forceinline__ void load(const float* p, float (&f)[4]) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
  }
  static __device__ __forceinline__ void store(float* p, const float (&f)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
  }
  static __device__ __forceinline__ void round(float (&)[4]) {}
};

template <typename TS, int K1, int K2, int K3>
struct RunConv {
  static constexpr int KR = 1 + (K1 > 0) + (K2 > 0) + (K3 > 0);
  static constexpr int TAPS = K1 + K2 + K3;
  static constexpr int KW = (K1 > K2 ? (K1 > K3 ? K1 : K3) : (K2 > K3 ? K2 : K3));   // window length
  float w[TAPS][4];
  float win[KW][4];
  __device__ __forceinline__ void load_taps(const float* __restrict__ conv_w, int C, int c) {
#pragma unroll
    for (int r = 0; r < TAPS; ++r) {
      const float4 v = *reinterpret_cast<const float4*>(conv_w + (int64_t)r * C + c);
      w[r][0] = v.x; w[r][1] = v.y; w[r][2] = v.z; w[r][3] = v.w;
    }
  }
  // window before token t0: win[i] = F[t0 - 1 - i] inside t0's sequence, else 0
  __device__ __forceinline__ void init(const TS* __restrict__ F, int64_t t0, int64_t S, int C, int c) {
    const int64_t pos = t0 % S;
#pragma unroll
    for (int i = 0; i < KW; ++i) {
      if (i < KW - 1 && i + 1 <= pos) Vec4<TS>::load(F + (t0 - 1 - i) * C + c, win[i]);
      else {
#pragma unroll
        for (int q = 0; q < 4; ++q) win[i][q] = 0.f;
      }
    }
  }
  // shift in F[t]; clears the history at a sequence start
  __device__ __forceinline__ void push(const float (&f)[4], bool seq_start) {
#pragma unroll
    for (int i = KW - 1; i > 0; --i)
#pragma unroll
      for (int q = 0; q < 4; ++q) win[i][q] = seq_start ? 0.f : win[i - 1][q];
#pragma unroll
    for (int q = 0; q < 4; ++q) win[0][q] = f[q];
  }
  // components e_0 = F[t], e_j = sum_{i < kappa_j} w_j[i] F[t - i]
  __device__ __forceinline__ void components(float (&e)[KR][4]) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) e[0][q] = win[0][q];
    int b = 1, row = 0;
    auto branch = [&](int K) {
#pragma unroll
      for (int q = 0; q < 4; ++q) e[b][q] = 0.f;
#pragma unroll
      for (int i = 0; i < KW; ++i)
        if (i < K)
#pragma unroll
          for (int q = 0; q < 4; ++q) e[b][q] = fmaf(w[row + i][q], win[i][q], e[b][q]);
      row += K;
      ++b;
    };
    if (K1 > 0) branch(K1);
    if (K2 > 0) branch(K2);
    if (K3 > 0) branch(K3);
  }
};

template <typename TS, int K1, int K2, int K3>
__global__ __launch_bounds__(256) void k_post_gram_run(const TS* __restrict__ F, int64_t T, int64_t S, int C,
                                                       const float* __restrict__ conv_w,
                                                       float* __restrict__ gpart) {
  using RC = RunConv<TS, K1, K2, K3>;
  constexpr int KR = RC::KR, NP = KR * (KR + 1) / 2;
  __shared__ float red[kRun][4][NP];
  const int nw = blockDim.x / kWave;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t cb = blockIdx.y;
  const int c = (int)(cb * blockDim.x + threadIdx.x) * 4;
  const int64_t t0 = (int64_t)blockIdx.x * kRun;
  const int nt = (int)((T - t0 < kRun) ? T - t0 : kRun);
  RC rc;
  rc.load_taps(conv_w, C, c);
  rc.init(F, t0, S, C, c);
#pragma unroll 4
  for (int u = 0; u < nt; ++u) {
    const int64_t t = t0 + u;
    float f[4];
    Vec4<TS>::load(F + t * C + c, f);
    rc.push(f, (t % S) == 0);
    float e[KR][4];
    rc.components(e);
    int pi = 0;
#pragma unroll
    for (int a = 0; a < KR; ++a)
#pragma unroll
      for (int b = a; b < KR; ++b, ++pi) {
        float v = 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) v = fmaf(e[a][q], e[b][q], v);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
        if (lane == 0) red[u][wave][pi] = v;
      }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nt * NP; i += blockDim.x) {
    const int u = i / NP, pi = i % NP;
    float v = 0.f;
    for (int w = 0; w < nw; ++w) v += red[u][w][pi];
    gpart[(cb * NP + pi) * T + t0 + u] = v;
  }
}

template <typename TS, int K1, int K2, int K3, int KK>
__global__ __launch_bounds__(256) void k_post_apply_run(TS* __restrict__ X, const TS* __restrict__ F, int64_t T,
                                                        int64_t S, int N, int C, int k,
                                                        const float* __restrict__ conv_w,
                                                        const int32_t* __restrict__ idx,
                                                        const float* __restrict__ Hres,
                                                        const float* __restrict__ wb,
                                                        const float* __restrict__ Hpre_next,
                                                        const TS* __restrict__ base_next, TS* __restrict__ input_next,
                                                        TS* __restrict__ Xact_save) {
  using RC = RunConv<TS, K1, K2, K3>;
  constexpr int KR = RC::KR;
  constexpr int G = 2;   // tokens whose loads are issued together; KK >= k active rows
  const int c = (int)(blockIdx.y * blockDim.x + threadIdx.x) * 4;
  const int64_t t0 = (int64_t)blockIdx.x * kRun;
  const int nt = (int)((T - t0 < kRun) ? T - t0 : kRun);
  RC rc;
  rc.load_taps(conv_w, C, c);
  rc.init(F, t0, S, C, c);
  for (int u0 = 0; u0 < nt; u0 += G) {
    float f[G][4], a[G][KK][4], nxt[G][4];
    int32_t rows[G][KK];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (u0 + g < nt) {
        const int64_t t = t0 + u0 + g;
        Vec4<TS>::load(F + t * C + c, f[g]);
#pragma unroll
        for (int l = 0; l < KK; ++l) {
          if (l < k) {
            rows[g][l] = idx[t * k + l];
            Vec4<TS>::load(X + (t * N + rows[g][l]) * (int64_t)C + c, a[g][l]);
          }
        }
        if (input_next) Vec4<TS>::load(base_next + t * C + c, nxt[g]);
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (u0 + g >= nt) break;
      const int64_t t = t0 + u0 + g;
      rc.push(f[g], (t % S) == 0);
      float e[KR][4];
      rc.components(e);
      if (Xact_save) {
#pragma unroll
        for (int l = 0; l < KK; ++l)
          if (l < k) Vec4<TS>::store(Xact_save + (t * k + l) * (int64_t)C + c, a[g][l]);
      }
#pragma unroll
      for (int j = 0; j < KK; ++j) {
        if (j < k) {
          float y[4];
          if (Hres) {
#pragma unroll
            for (int q = 0; q < 4; ++q) y[q] = 0.f;
#pragma unroll
            for (int l = 0; l < KK; ++l) {
              if (l < k) {
                const float h = Hres[(t * k + j) * k + l];
#pragma unroll
                for (int q = 0; q < 4; ++q) y[q] = fmaf(h, a[g][l][q], y[q]);
              }
            }
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) y[q] = a[g][j][q];
          }
#pragma unroll
          for (int b = 0; b < KR; ++b) {
            const float wv = wb[(t * k + j) * KR + b];
#pragma unroll
            for (int q = 0; q < 4; ++q) y[q] = fmaf(wv, e[b][q], y[q]);
          }
          Vec4<TS>::store(X + (t * N + rows[g][j]) * (int64_t)C + c, y);
          if (input_next) {
            Vec4<TS>::round(y);
            const float h = Hpre_next[t * N + rows[g][j]];
#pragma unroll
            for (int q = 0; q < 4; ++q) nxt[g][q] = fmaf(h, y[q], nxt[g][q]);
          }
        }
      }
      if (input_next) Vec4<TS>::store(input_next + t * C + c, nxt[g]);
    }
  }
}

// threads per block of the run-based kernels for width C (4 channels each)
static inline int run_threads(int C) { return C >= 1024 ? 256 : C / 4; }
static inline bool run_ok(int C, int Kr, const int32_t* kappa) {
  if (Kr != 4 || kappa[0] != 4 || kappa[1] != 8 || kappa[2] != 12) return false;
  if (C % 4 != 0) return false;
  const int nthr = run_threads(C);
  return nthr % kWave == 0 && C % (nthr * 4) == 0;
}

int64_t gram_chunks(int C, int Kr, const int32_t* kappa) {
  if (run_ok(C, Kr, kappa)) return C / (run_threads(C) * 4);
  return post_chunks(C);
}

hipError_t launch_post_gram(int state_dtype, const void* F, int64_t T, int64_t S, int C, int Kr,
                            const int32_t* kappa, const float* conv_w, float* gpart, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (run_ok(C, Kr, kappa)) {
    const int nthr = run_threads(C);
    const dim3 grid((unsigned)((T + kRun - 1) / kRun), (unsigned)(C / (nthr * 4)));
    if (state_dtype == XHC_BF16)
      k_post_gram_run<uint16_t, 4, 8, 12><<<grid, dim3(nthr), 0, s>>>(reinterpret_cast<const uint16_t*>(F), T, S, C,
                                                                      conv_w, gpart);
    else
      k_post_gram_run<float, 4, 8, 12><<<grid, dim3(nthr), 0, s>>>(reinterpret_cast<const float*>(F), T, S, C,
                                                                   conv_w, gpart);
    return hipGetLastError();
  }
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
  if (wb && run_ok(C, Kr, kappa)) {
    const int nthr = run_threads(C);
    const dim3 grid((unsigned)((T + kRun - 1) / kRun), (unsigned)(C / (nthr * 4)));
#define XHC_APPLY_RUN(TS, KK)                                                                                     \
  k_post_apply_run<TS, 4, 8, 12, KK><<<grid, dim3(nthr), 0, s>>>(                                                \
      reinterpret_cast<TS*>(X), reinterpret_cast<const TS*>(F), T, S, N, C, k, conv_w, idx, Hres, wb, Hpre_next, \
      reinterpret_cast<const TS*>(base_next), reinterpret_cast<TS*>(input_next), reinterpret_cast<TS*>(Xact_save))
    if (state_dtype == XHC_BF16) {
      if (k <= 4) XHC_APPLY_RUN(uint16_t, 4); else XHC_APPLY_RUN(uint16_t, kMaxK);
    } else {
      if (k <= 4) XHC_APPLY_RUN(float, 4); else XHC_APPLY_RUN(float, kMaxK);
    }
#undef XHC_APPLY_RUN
    return hipGetLastError();
  }
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

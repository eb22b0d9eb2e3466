// Mapping generation of an xHC sublayer (multi-kernel path): packing and the
// per-token finalisation of the projections.
//
//  k_pack / k_colsum   fp32 weights -> bf16 MFMA fragments; column sums of bf16(W_r)
//  k_sum_chunks        per-token sums of the split-K partials
//  k_pre_route         per token: LayerNorm / RMSNorm corrections of the raw
//                      projection (eq:fused_normalized_projection), H^pre, routing
//  k_pre_coef          per token: RMS of the active state, H^post, H^res (Sinkhorn + clamp)
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {
// ----------------------------------------------------------------- packing

__global__ void k_pack(int64_t K, int nob, int ncols_a, const float* __restrict__ A, int ncols_b,
                       const float* __restrict__ B, int64_t b_count, int grouped, uint4* __restrict__ out) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nfrag = (K / 32) * nob;
  if (gid >= nfrag * kWave) return;
  const int lane = (int)(gid % kWave);
  const int64_t frag = gid / kWave;
  const int ob = (int)(frag % nob);
  const int64_t kb = frag / nob;
  const int col = ob * 16 + lane % 16;
  // grouped: fragment 4G + u, lane group g holds rows 128G + 32g + 8u .. +8
  const int64_t row0 = grouped ? (kb / 4) * 128 + (lane / 16) * 32 + (kb % 4) * 8 : kb * 32 + (lane / 16) * 8;
  const int64_t nb = (int64_t)ncols_b * b_count;
  float f[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int64_t row = row0 + e;
    float v = 0.f;
    if (col < ncols_a) {
      v = A[row * ncols_a + col];
    } else if (col - ncols_a < nb) {
      const int64_t q = (col - ncols_a) / ncols_b;
      const int cc = (col - ncols_a) % ncols_b;
      v = B[(q * K + row) * ncols_b + cc];
    }
    f[e] = v;
  }
  out[gid] = pack8(f);
}

__global__ void k_colsum(int64_t K, int ncols, const float* __restrict__ W, float* __restrict__ out) {
  __shared__ float red[256];
  const int col = blockIdx.x;
  float s = 0.f;
  for (int64_t r = threadIdx.x; r < K; r += 256) s += __uint_as_float(f2bf(W[r * ncols + col]) << 16);
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[col] = red[0];
}

hipError_t launch_pack(int64_t K, int64_t nout, int ncols_a, const float* A, int ncols_b, const float* B,
                       int64_t b_count, bool grouped, void* packed, hipStream_t s) {
  const int nob = (int)out_blocks(nout);
  const int64_t threads = (K / 32) * nob * kWave;
  if (threads == 0) return hipSuccess;
  k_pack<<<dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s>>>(K, nob, ncols_a, A, ncols_b, B, b_count,
                                                                       grouped ? 1 : 0,
                                                                       reinterpret_cast<uint4*>(packed));
  return hipGetLastError();
}

hipError_t launch_colsum(int64_t K, int ncols, const float* W, float* out, hipStream_t s) {
  k_colsum<<<dim3(ncols), dim3(256), 0, s>>>(K, ncols, W, out);
  return hipGetLastError();
}

// ----------------------------------------------------------------- per-token finalisation

// sums[o][t] = sum over chunks of part[chunk][o][t] (chunk order fixed), one
// thread per (o, t); the loads of all chunks are issued before the adds.
__global__ __launch_bounds__(256) void k_sum_chunks(const float* __restrict__ part, int64_t nchunk, int NO,
                                                    int64_t T, float* __restrict__ sums) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)NO * T) return;
  const int64_t stride = (int64_t)NO * T;
  float s = 0.f;
  for (int64_t c0 = 0; c0 < nchunk; c0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (c0 + u < nchunk) ? part[(c0 + u) * stride + i] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  sums[i] = s;
}

// Full-state projection sums -> router logits and npre pre-maps (one thread per token).
// z^r = (x W^r - mu colsum(W^r)) / sqrt(nu - mu^2 + eps),  z^pre = x W^pre / sqrt(nu + eps).
// NB: a bound of N (16, 32 or 64).  Each batch of a token's sums (the router
// logits, then each pre-map's logits) is loaded before any of it is used
// (clamped to row N - 1 past N), so a thread waits once per batch.
template <int NB>
__global__ __launch_bounds__(64) void k_pre_route(const float* __restrict__ sums, int NO, int64_t T, int N, int m,
                                                  int k, int npre, int64_t NC, const float* __restrict__ colsum,
                                                  const float* __restrict__ alpha_pre, int alpha_stride,
                                                  const float* __restrict__ b_pre, float eps,
                                                  int32_t* __restrict__ idx, float* __restrict__ p,
                                                  float* __restrict__ Hpre, float* __restrict__ saved,
                                                  int nsave, int save_stats_at, int softmax, int save_pre) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  float zr[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) zr[i] = sums[(int64_t)(i < N ? i : N - 1) * T + t];
  const float mu = sums[(int64_t)(NO - 2) * T + t] / (float)NC;
  const float nu = sums[(int64_t)(NO - 1) * T + t] / (float)NC;
  // save_pre < 0: one record per pre-map q at saved + q T nsave (router
  // logits and statistics in each)
  const int nrec = save_pre < 0 ? npre : 1;
  if (saved)
    for (int r = 0; r < nrec; ++r) {
      saved[(r * T + t) * nsave + save_stats_at] = mu;
      saved[(r * T + t) * nsave + save_stats_at + 1] = nu;
    }
  const float r_ln = 1.0f / sqrtf(ln_variance(mu, nu) + eps);
  const float r_rms = 1.0f / sqrtf(nu + eps);
  float z[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) z[i] = (i < N) ? (zr[i] - mu * colsum[i < N ? i : 0]) * r_ln : 0.f;
  int32_t id[kMaxK];
  float pp[kMaxK];
  route_token<NB>(z, N, m, k, id, pp, softmax != 0);
  for (int j = 0; j < k; ++j) {
    idx[t * k + j] = id[j];
    p[t * k + j] = pp[j];
  }
  if (saved)
    for (int r = 0; r < nrec; ++r)
      for (int i = 0; i < N; ++i) saved[(r * T + t) * nsave + i] = z[i];
  for (int q = 0; q < npre; ++q) {
    const float a = alpha_pre[q * alpha_stride];
#pragma unroll
    for (int i = 0; i < NB; ++i) zr[i] = sums[(int64_t)(N + q * N + (i < N ? i : N - 1)) * T + t];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      if (i >= N) break;
      const float zp = zr[i] * r_rms;
      if (saved && save_pre < 0) saved[((int64_t)q * T + t) * nsave + N + i] = zp;
      else if (saved && q == save_pre) saved[t * nsave + N + i] = zp;
      Hpre[((int64_t)q * T + t) * N + i] = sigmoidf(a * zp + b_pre[q * N + i]);
    }
  }
}

// Active projection sums -> H^post = 2 sigma(.) and (with_res) H^res = clamp(SK(exp(.))).
__global__ __launch_bounds__(128) void k_pre_coef(const float* __restrict__ sums, int NO, int64_t T, int k, int Kq,
                                                  int with_res, int64_t kC, const float* __restrict__ alpha_post,
                                                  const float* __restrict__ alpha_res,
                                                  const float* __restrict__ b_post,
                                                  const float* __restrict__ b_res, float eps, int iters,
                                                  float delta, float* __restrict__ Hpost,
                                                  float* __restrict__ Hres, float* __restrict__ saved, int nsave,
                                                  int save_z_at, int save_stats_at,
                                                  const int* __restrict__ err) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  if (err && *err != 0) {
    // the single-pass kernel gave up a wait: its partials are not valid
    const float nan = __uint_as_float(0x7fc00000u);
    for (int o = 0; o < k * Kq; ++o) Hpost[t * k * Kq + o] = nan;
    if (with_res)
      for (int o = 0; o < k * k; ++o) Hres[t * k * k + o] = nan;
    return;
  }
  const float nu_a = sums[(int64_t)(NO - 1) * T + t] / (float)kC;
  const float rstd = 1.0f / sqrtf(nu_a + eps);
  if (saved) {
    saved[t * nsave + save_stats_at] = nu_a;
    for (int o = 0; o < k * Kq + (with_res ? k * k : 0); ++o)
      saved[t * nsave + save_z_at + o] = sums[(int64_t)o * T + t] * rstd;
  }
  const float ap = alpha_post[0];
  for (int o = 0; o < k * Kq; ++o)
    Hpost[t * k * Kq + o] = 2.0f * sigmoidf(ap * (sums[(int64_t)o * T + t] * rstd) + b_post[o]);
  if (!with_res) return;
  const float ar = alpha_res[0];
  float M[kMaxK * kMaxK];
#pragma unroll
  for (int j = 0; j < kMaxK; ++j)
#pragma unroll
    for (int l = 0; l < kMaxK; ++l)
      M[j * kMaxK + l] = (j < k && l < k)
          ? ar * (sums[(int64_t)(k * Kq + j * k + l) * T + t] * rstd) + b_res[j * k + l] : 0.f;
  sinkhorn_clamp(M, k, iters, delta);
  for (int j = 0; j < k; ++j)
    for (int l = 0; l < k; ++l) Hres[(t * k + j) * k + l] = M[j * kMaxK + l];
}

// k = 4: the chunk sums of the active projection and the coefficients in one
// launch.  A block takes 32 tokens; thread (part h, token u) sums chunk range
// h of token u (8 ranges), the ranges are added in order through LDS, and one
// thread per token forms the coefficients.
constexpr int kCoefTok = 64, kCoefParts = 4;   // tokens per workgroup, member-chunk parts per token
template <int K>
__global__ __launch_bounds__(kCoefTok * kCoefParts) void k_pre_coef_sum(
    const float* __restrict__ part, int64_t nchunk, int NO, int64_t T, int Kq, int with_res, int64_t kC,
    const float* __restrict__ alpha_post, const float* __restrict__ alpha_res, const float* __restrict__ b_post,
    const float* __restrict__ b_res, float eps, int iters, float delta, float* __restrict__ Hpost,
    float* __restrict__ Hres, float* __restrict__ saved, int nsave, int save_z_at, int save_stats_at,
    const int* __restrict__ err) {
  constexpr int NA = K * kMaxKr + K * K;   // outputs kept (at most)
  __shared__ float red[kCoefParts][NA + 1][kCoefTok];
  const int u = threadIdx.x % kCoefTok, h = threadIdx.x / kCoefTok;
  const int64_t t = (int64_t)blockIdx.x * kCoefTok + u;
  const int nproj = K * Kq + (with_res ? K * K : 0);
  {
    float acc[NA + 1];
#pragma unroll
    for (int o = 0; o <= NA; ++o) acc[o] = 0.f;
    const int64_t per = (nchunk + kCoefParts - 1) / kCoefParts;
    const int64_t c0 = h * per, c1 = (c0 + per < nchunk) ? c0 + per : nchunk;
    if (t < T) {
      const int64_t stride = (int64_t)NO * T;
      for (int64_t c = c0; c < c1; ++c) {
        const float* pc = part + c * stride + t;
        float v[NA + 1];
#pragma unroll
        for (int o = 0; o < NA; ++o) v[o] = o < nproj ? pc[(int64_t)o * T] : 0.f;
        v[NA] = pc[(int64_t)(NO - 1) * T];
#pragma unroll
        for (int o = 0; o <= NA; ++o) acc[o] += v[o];
      }
    }
#pragma unroll
    for (int o = 0; o <= NA; ++o) red[h][o][u] = acc[o];
  }
  __syncthreads();
  if (h != 0 || t >= T) return;
  float acc[NA + 1];
#pragma unroll
  for (int o = 0; o <= NA; ++o) {
    float v = red[0][o][u];
#pragma unroll
    for (int q = 1; q < kCoefParts; ++q) v += red[q][o][u];
    acc[o] = v;
  }
  if (err && *err != 0) {
    // the single-pass kernel gave up a wait: its partials are not valid
    const float nan = __uint_as_float(0x7fc00000u);
    for (int o = 0; o < K * Kq; ++o) Hpost[t * K * Kq + o] = nan;
    if (with_res)
      for (int o = 0; o < K * K; ++o) Hres[t * K * K + o] = nan;
    return;
  }
  const float nu_a = acc[NA] / (float)kC;
  const float rstd = 1.0f / sqrtf(nu_a + eps);
  if (saved) {
    saved[t * nsave + save_stats_at] = nu_a;
#pragma unroll
    for (int o = 0; o < NA; ++o)
      if (o < nproj) saved[t * nsave + save_z_at + o] = acc[o] * rstd;
  }
  const float ap = alpha_post[0];
#pragma unroll
  for (int o = 0; o < K * kMaxKr; ++o)
    if (o < K * Kq) Hpost[t * K * Kq + o] = 2.0f * sigmoidf(ap * (acc[o] * rstd) + b_post[o]);
  if (!with_res) return;
  const float ar = alpha_res[0];
  float M[K * K];
#pragma unroll
  for (int o = 0; o < K * K; ++o) {
    // the W_res outputs follow the K Kq W_post outputs
    float z = 0.f;
#pragma unroll
    for (int q = 1; q <= kMaxKr; ++q)
      if (q == Kq) z = acc[K * q + o];
    M[o] = ar * (z * rstd) + b_res[o];
  }
  sinkhorn_clamp_k<K>(M, iters, delta);
#pragma unroll
  for (int o = 0; o < K * K; ++o) Hres[t * K * K + o] = M[o];
}

static hipError_t sum_chunks(const float* part, int64_t nchunk, int NO, int64_t T, float* sums, hipStream_t s) {
  const int64_t n = (int64_t)NO * T;
  k_sum_chunks<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s>>>(part, nchunk, NO, T, sums);
  return hipGetLastError();
}

hipError_t launch_pre_route(const float* part, int64_t nchunk, int64_t nout, int64_t T, int N, int m, int k,
                            int npre, int64_t C, const float* colsum, const float* alpha_pre, int alpha_stride,
                            const float* b_pre, float eps, int32_t* idx, float* p, float* Hpre, float* sums,
                            float* saved, int nsave, int save_stats_at, int router, hipStream_t s, int save_pre) {
  if (T == 0) return hipSuccess;
  const int NO = (int)out_blocks(nout) * 16 + 2;
  hipError_t e = sum_chunks(part, nchunk, NO, T, sums, s);
  if (e != hipSuccess) return e;
#define XHC_ROUTE(NBV)                                                                                      \
  k_pre_route<NBV><<<dim3((unsigned)((T + 63) / 64)), dim3(64), 0, s>>>(                                     \
      sums, NO, T, N, m, k, npre, (int64_t)N * C, colsum, alpha_pre, alpha_stride, b_pre, eps, idx, p, Hpre, \
      saved, nsave, save_stats_at, router == XHC_ROUTER_SOFTMAX ? 1 : 0, save_pre)
  if (N <= 16) XHC_ROUTE(16);
  else if (N <= 32) XHC_ROUTE(32);
  else XHC_ROUTE(kMaxN);
#undef XHC_ROUTE
  return hipGetLastError();
}

hipError_t launch_pre_coef(const float* part, int64_t nchunk, int64_t nout, int64_t T, int k, int Kq,
                           int with_res, int64_t C, const float* alpha_post, const float* alpha_res,
                           const float* b_post, const float* b_res, float eps, int iters, float delta,
                           float* Hpost, float* Hres, float* sums, float* saved, int nsave, int save_z_at,
                           int save_stats_at, hipStream_t s, const int* err) {
  if (T == 0) return hipSuccess;
  const int NO = (int)out_blocks(nout) * 16 + 2;
  if (k == 4 && Kq <= kMaxKr) {
    k_pre_coef_sum<4><<<dim3((unsigned)((T + kCoefTok - 1) / kCoefTok)), dim3(kCoefTok * kCoefParts), 0, s>>>(
        part, nchunk, NO, T, Kq, with_res, (int64_t)k * C, alpha_post, alpha_res, b_post, b_res, eps, iters, delta,
        Hpost, Hres, saved, nsave, save_z_at, save_stats_at, err);
    return hipGetLastError();
  }
  hipError_t e = sum_chunks(part, nchunk, NO, T, sums, s);
  if (e != hipSuccess) return e;
  k_pre_coef<<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(
      sums, NO, T, k, Kq, with_res, (int64_t)k * C, alpha_post, alpha_res, b_post, b_res, eps, iters, delta,
      Hpost, Hres, saved, nsave, save_z_at, save_stats_at, err);
  return hipGetLastError();
}

}  // namespace xhc

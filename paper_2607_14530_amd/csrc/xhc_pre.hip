// Mapping generation and dense read of an xHC sublayer (multi-kernel path).
//
//  k_pack / k_colsum   fp32 weights -> bf16 MFMA fragments; column sums of bf16(W_r)
//  k_proj_partial      split-K MFMA projection of 16-token tiles (full state,
//                      or the gathered active rows), plus the norm moments
//  k_pre_route         per token: LayerNorm / RMSNorm corrections of the raw
//                      projection (eq:fused_normalized_projection), H^pre, routing
//  k_pre_coef          per token: RMS of the active state, H^post, H^res (Sinkhorn + clamp)
//  k_dense_read        input = sum_i H^pre_i x_i (eq:dense_read); xHC-Flash bases
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {

// ----------------------------------------------------------------- packing

__global__ void k_pack(int64_t K, int nob, int ncols_a, const float* __restrict__ A, int ncols_b,
                       const float* __restrict__ B, int64_t b_count, uint4* __restrict__ out) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nfrag = (K / 32) * nob;
  if (gid >= nfrag * kWave) return;
  const int lane = (int)(gid % kWave);
  const int64_t frag = gid / kWave;
  const int ob = (int)(frag % nob);
  const int64_t kb = frag / nob;
  const int col = ob * 16 + lane % 16;
  const int64_t row0 = kb * 32 + (lane / 16) * 8;
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
                       int64_t b_count, void* packed, hipStream_t s) {
  const int nob = (int)out_blocks(nout);
  const int64_t threads = (K / 32) * nob * kWave;
  if (threads == 0) return hipSuccess;
  k_pack<<<dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s>>>(K, nob, ncols_a, A, ncols_b, B, b_count,
                                                                       reinterpret_cast<uint4*>(packed));
  return hipGetLastError();
}

hipError_t launch_colsum(int64_t K, int ncols, const float* W, float* out, hipStream_t s) {
  k_colsum<<<dim3(ncols), dim3(256), 0, s>>>(K, ncols, W, out);
  return hipGetLastError();
}

// ----------------------------------------------------------------- projection
// One workgroup = 4 waves = one 16-token tile x one chunk of kProjChunkBlocks
// 32-row blocks of K.  MFMA operands: A = packed weight fragment (outputs x K),
// B = 8 state elements per lane (K x tokens).  With GATHER, K runs over the
// active rows: row j of K is X[t, idx[t, j], :].
// Output part[chunk][o][t] for o < 16*NOB, then sum x and sum x^2 at
// o = 16*NOB and 16*NOB + 1.

template <typename TS, int NOB, bool GATHER>
__global__ __launch_bounds__(256) void k_proj_partial(const TS* __restrict__ X, int64_t T, int N, int C,
                                                      int64_t K, const uint4* __restrict__ wpk,
                                                      const int32_t* __restrict__ idx, int k,
                                                      float* __restrict__ part) {
  constexpr int NO = NOB * 16 + 2;
  __shared__ float red[4][NO][kProjTile];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int64_t tile = blockIdx.x, chunk = blockIdx.y;
  const int64_t t = tile * kProjTile + tl;
  const bool valid = t < T;
  const int64_t nblk = K / 32;
  f32x4 acc[NOB];
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  float s1 = 0.f, s2 = 0.f;
  // The state loads of UNR blocks are issued before any is used, so each wave
  // keeps UNR loads in flight instead of one.
  constexpr int UNR = Vec8<TS>::kSplit ? 4 : 16;
  constexpr int BPW = kProjChunkBlocks / 4;   // blocks per wave
  static_assert(BPW % UNR == 0, "unroll must divide the blocks per wave");
  for (int b0 = 0; b0 < BPW; b0 += UNR) {
    uint4 xb[UNR], xl[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int64_t kb = chunk * kProjChunkBlocks + (b0 + u) * 4 + wave;
      xb[u] = make_uint4(0, 0, 0, 0);
      xl[u] = make_uint4(0, 0, 0, 0);
      if (valid && kb < nblk) {
        const int64_t kk = kb * 32 + grp * 8;
        const TS* src;
        if (GATHER) {
          const int row = (int)(kk / C);
          const int c = (int)(kk % C);
          src = X + ((t * N + idx[t * k + row]) * (int64_t)C + c);
        } else {
          src = X + (t * (int64_t)N * C + kk);
        }
        float f[8];
        xb[u] = Vec8<TS>::operand(src, f, xl[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int64_t kb = chunk * kProjChunkBlocks + (b0 + u) * 4 + wave;
      if (kb < nblk) {
      // moments from the operand registers (hi + lo for an fp32 state, to 2^-16)
      float f[8], g[8];
      unpack8(xb[u], f);
      unpack8(xl[u], g);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = f[e] + g[e];
        s1 += x;
        s2 += x * x;
      }
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob) {
        const uint4 wa = wpk[(kb * NOB + ob) * kWave + lane];
        acc[ob] = mfma_16x16x32(wa, xb[u], acc[ob]);
        if (Vec8<TS>::kSplit) acc[ob] = mfma_16x16x32(wa, xl[u], acc[ob]);
      }
      }
    }
  }
  s1 += __shfl_xor(s1, 16);
  s1 += __shfl_xor(s1, 32);
  s2 += __shfl_xor(s2, 16);
  s2 += __shfl_xor(s2, 32);
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
    for (int v = 0; v < 4; ++v) red[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
  if (grp == 0) {
    red[wave][NO - 2][tl] = s1;
    red[wave][NO - 1][tl] = s2;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < NO * kProjTile; i += 256) {
    const int o = i / kProjTile, tt = i % kProjTile;
    const int64_t tg = tile * kProjTile + tt;
    if (tg < T) part[(chunk * NO + o) * T + tg] = red[0][o][tt] + red[1][o][tt] + red[2][o][tt] + red[3][o][tt];
  }
}

template <typename TS, bool GATHER>
static hipError_t proj_dispatch(const TS* X, int64_t T, int N, int C, int64_t K, const void* packed, int nob,
                                const int32_t* idx, int k, float* part, hipStream_t s) {
  const dim3 grid((unsigned)((T + kProjTile - 1) / kProjTile), (unsigned)proj_chunks(K));
  const uint4* w = reinterpret_cast<const uint4*>(packed);
#define XHC_PROJ_CASE(NB) \
  case NB: k_proj_partial<TS, NB, GATHER><<<grid, dim3(256), 0, s>>>(X, T, N, C, K, w, idx, k, part); break;
  switch (nob) {
    XHC_PROJ_CASE(1) XHC_PROJ_CASE(2) XHC_PROJ_CASE(3) XHC_PROJ_CASE(4)
    XHC_PROJ_CASE(5) XHC_PROJ_CASE(6) XHC_PROJ_CASE(7) XHC_PROJ_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef XHC_PROJ_CASE
  return hipGetLastError();
}

hipError_t launch_proj_partial(int state_dtype, const void* X, int64_t T, int N, int C, int64_t K,
                               const void* packed, int64_t nout, const int32_t* idx, int k, float* part,
                               hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int nob = (int)out_blocks(nout);
  if (state_dtype == XHC_BF16) {
    const uint16_t* x = reinterpret_cast<const uint16_t*>(X);
    return idx ? proj_dispatch<uint16_t, true>(x, T, N, C, K, packed, nob, idx, k, part, s)
               : proj_dispatch<uint16_t, false>(x, T, N, C, K, packed, nob, idx, k, part, s);
  }
  const float* x = reinterpret_cast<const float*>(X);
  return idx ? proj_dispatch<float, true>(x, T, N, C, K, packed, nob, idx, k, part, s)
             : proj_dispatch<float, false>(x, T, N, C, K, packed, nob, idx, k, part, s);
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
__global__ __launch_bounds__(128) void k_pre_route(const float* __restrict__ sums, int NO, int64_t T, int N, int m,
                                                   int k, int npre, int64_t NC, const float* __restrict__ colsum,
                                                   const float* __restrict__ alpha_pre, int alpha_stride,
                                                   const float* __restrict__ b_pre, float eps,
                                                   int32_t* __restrict__ idx, float* __restrict__ p,
                                                   float* __restrict__ Hpre, float* __restrict__ saved,
                                                   int nsave, int save_stats_at) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const float mu = sums[(int64_t)(NO - 2) * T + t] / (float)NC;
  const float nu = sums[(int64_t)(NO - 1) * T + t] / (float)NC;
  if (saved) {
    saved[t * nsave + save_stats_at] = mu;
    saved[t * nsave + save_stats_at + 1] = nu;
  }
  const float r_ln = 1.0f / sqrtf(fmaxf(nu - mu * mu, 0.f) + eps);
  const float r_rms = 1.0f / sqrtf(nu + eps);
  float z[kMaxN];
#pragma unroll
  for (int i = 0; i < kMaxN; ++i) z[i] = (i < N) ? (sums[(int64_t)i * T + t] - mu * colsum[i]) * r_ln : 0.f;
  int32_t id[kMaxK];
  float pp[kMaxK];
  route_token<kMaxN>(z, N, m, k, id, pp);
  for (int j = 0; j < k; ++j) {
    idx[t * k + j] = id[j];
    p[t * k + j] = pp[j];
  }
  if (saved)
    for (int i = 0; i < N; ++i) saved[t * nsave + i] = z[i];
  for (int q = 0; q < npre; ++q) {
    const float a = alpha_pre[q * alpha_stride];
    for (int i = 0; i < N; ++i) {
      const float zp = sums[(int64_t)(N + q * N + i) * T + t] * r_rms;
      if (saved && q == 0) saved[t * nsave + N + i] = zp;
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
                                                  int save_z_at, int save_stats_at) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
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

static hipError_t sum_chunks(const float* part, int64_t nchunk, int NO, int64_t T, float* sums, hipStream_t s) {
  const int64_t n = (int64_t)NO * T;
  k_sum_chunks<<<dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s>>>(part, nchunk, NO, T, sums);
  return hipGetLastError();
}

hipError_t launch_pre_route(const float* part, int64_t nchunk, int64_t nout, int64_t T, int N, int m, int k,
                            int npre, int64_t C, const float* colsum, const float* alpha_pre, int alpha_stride,
                            const float* b_pre, float eps, int32_t* idx, float* p, float* Hpre, float* sums,
                            float* saved, int nsave, int save_stats_at, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int NO = (int)out_blocks(nout) * 16 + 2;
  hipError_t e = sum_chunks(part, nchunk, NO, T, sums, s);
  if (e != hipSuccess) return e;
  k_pre_route<<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(
      sums, NO, T, N, m, k, npre, (int64_t)N * C, colsum, alpha_pre, alpha_stride, b_pre, eps, idx, p, Hpre,
      saved, nsave, save_stats_at);
  return hipGetLastError();
}

hipError_t launch_pre_coef(const float* part, int64_t nchunk, int64_t nout, int64_t T, int k, int Kq,
                           int with_res, int64_t C, const float* alpha_post, const float* alpha_res,
                           const float* b_post, const float* b_res, float eps, int iters, float delta,
                           float* Hpost, float* Hres, float* sums, float* saved, int nsave, int save_z_at,
                           int save_stats_at, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int NO = (int)out_blocks(nout) * 16 + 2;
  hipError_t e = sum_chunks(part, nchunk, NO, T, sums, s);
  if (e != hipSuccess) return e;
  k_pre_coef<<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(
      sums, NO, T, k, Kq, with_res, (int64_t)k * C, alpha_post, alpha_res, b_post, b_res, eps, iters, delta,
      Hpost, Hres, saved, nsave, save_z_at, save_stats_at);
  return hipGetLastError();
}

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
  constexpr int UNR = 8;   // stream rows loaded before use
  for (int i0 = 0; i0 < N; i0 += UNR) {
    float f[UNR][8];
#pragma unroll
    for (int u = 0; u < UNR; ++u)
      if (i0 + u < N) Vec8<TS>::load(xt + (int64_t)(i0 + u) * C, f[u]);
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int i = i0 + u;
      if (i >= N) break;
#pragma unroll
      for (int q = 0; q < NMAP; ++q) {
        float w = Hpre[((int64_t)q * T + t) * N + i];
        if (q > 0 && ((act >> i) & 1ull)) w = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[q][e] = fmaf(w, f[u][e], acc[q][e]);
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

}  // namespace xhc

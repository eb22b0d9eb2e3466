// Sparse write-back of an xHC sublayer (eq:aug, eq:gs, eq:sparse_write_delta,
// eq:sparse_write).
//
//  k_post_gram   MLP-type only: per token and channel chunk, the Gram matrix of
//                the components e_0 = out, e_j = DWConv_kappa_j(out) (fp32)
//  k_post_coef   per token: Gram-Schmidt in the component basis folded with p
//                and H^post into write-back weights wb[t][j][b]
//  k_post_apply  X[t, I_j, :] <- sum_l H^res[j,l] X[t, I_l, :] + sum_b wb[j][b] e_b;
//                the other N - k rows are never touched
#include "xhc_conv.h"
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


// Per token: G = sum over chunks; v_r = sum_b V[r][b] e_b (Gram-Schmidt, eq:gs);
// wb[j][b] = p_j sum_r H^post[j][r] V[r][b]  (p gates only the write-back term).
// out[j * Kr + b] receives token t's weights.
__device__ __forceinline__ void post_coef_token(const float* __restrict__ gpart, int64_t nchunk, int64_t T, int64_t t,
                                                int k, int Kr, int gram_schmidt, const float* __restrict__ p,
                                                const float* __restrict__ Hpost, float* __restrict__ out) {
  const int NP = Kr * (Kr + 1) / 2;
  // the chunk sums of every pair (a <= b < Kr: pair a Kr - a (a - 1) / 2 +
  // b - a in row-major upper order), each chunk's pairs loaded together (an
  // unused pair reads pair 0), summed in the order chunk 0, 1, ...
  float gs[kMaxKr][kMaxKr];
#pragma unroll
  for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
    for (int b = 0; b < kMaxKr; ++b) gs[a][b] = 0.f;
  for (int64_t c = 0; c < nchunk; ++c) {
    float v[kMaxKr][kMaxKr];
#pragma unroll
    for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
      for (int b = a; b < kMaxKr; ++b) {
        const int pab = (a < Kr && b < Kr) ? a * Kr - a * (a - 1) / 2 + (b - a) : 0;
        v[a][b] = gpart[(c * NP + pab) * T + t];
      }
#pragma unroll
    for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
      for (int b = a; b < kMaxKr; ++b) gs[a][b] += v[a][b];
  }
  double G[kMaxKr][kMaxKr];
#pragma unroll
  for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
    for (int b = a; b < kMaxKr; ++b) G[a][b] = G[b][a] = (a < Kr && b < Kr) ? (double)gs[a][b] : 0.0;
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
      out[j * Kr + b] = (float)(pj * s);
    }
  }
}

__global__ __launch_bounds__(128) void k_post_coef(const float* __restrict__ gpart, int64_t nchunk, int64_t T,
                                                   int k, int Kr, int gram_schmidt, const float* __restrict__ p,
                                                   const float* __restrict__ Hpost, float* __restrict__ wb) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  post_coef_token(gpart, nchunk, T, t, k, Kr, gram_schmidt, p, Hpost, wb + t * k * Kr);
}

// ------------------------------------------------------------------ run-based MLP-type kernels
// For compile-time kernel sizes (K1, K2, K3) = (4, 8, 12): a thread owns 4
// channels and walks a run of kRun consecutive tokens in groups of G, keeping
// the conv taps of its channels and the last 12 values of F in registers, so F
// is read once per kernel and the taps once per run.  Sequence starts fall on
// group starts (S % G == 0), where the history is cleared.

constexpr int kRun = 64;

// Gram partials per 1024-channel chunk.  Each lane forms its 4-channel
// products for G tokens; a wave sums them over its 64 lanes through an LDS
// transpose (lane v adds column v), and the waves' sums are added at the end.
template <typename TS, int K1, int K2, int K3>
__global__ __launch_bounds__(256) void k_post_gram_run(const TS* __restrict__ F, int64_t T, int64_t S, int C,
                                                       const float* __restrict__ conv_w,
                                                       float* __restrict__ gpart) {
  using CG = ConvGroup<K1, K2, K3>;
  constexpr int KR = CG::KR, NP = KR * (KR + 1) / 2;
  constexpr int G = 4, NV = G * NP, LD = (NV + 3) / 4 * 4 + 4;
  static_assert(NV <= kWave, "one column per lane");
  __shared__ __align__(16) float xpose[4][kWave][LD];
  __shared__ float red[kRun][4][NP];
  const int nw = blockDim.x / kWave;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t cb = blockIdx.y;
  const int c = (int)(cb * blockDim.x + threadIdx.x) * 4;
  const int64_t t0 = (int64_t)blockIdx.x * kRun;
  const int nt = (int)((T - t0 < kRun) ? T - t0 : kRun);
  CG cg;
  cg.load_taps(conv_w, C, c);
  cg.init(F, t0, S, C, c);
  float* mine = &xpose[wave][lane][0];
  // F rows are loaded PF groups ahead (a lane requests 8 bytes per token of a
  // bf16 state, so one group in flight would leave the memory system mostly
  // idle)
  constexpr int PF = sizeof(TS) == 2 ? 4 : 2;
  typename Row4<TS>::raw ring[PF][G];
#pragma unroll
  for (int f = 0; f < PF; ++f)
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int u = f * G + g;
      ring[f][g] = u < nt ? Row4<TS>::load(F + (t0 + u) * C + c) : Row4<TS>::zero();
    }
  for (int u1 = 0; u1 < nt; u1 += PF * G) {
#pragma unroll
    for (int f = 0; f < PF; ++f) {
      const int u0 = u1 + f * G;
      if (u0 >= nt) break;
      const int64_t t = t0 + u0;
      if (t % S == 0) cg.reset();
      float cur[G][4];
#pragma unroll
      for (int g = 0; g < G; ++g) Row4<TS>::unpack(ring[f][g], cur[g]);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int u = u0 + PF * G + g;
        ring[f][g] = u < nt ? Row4<TS>::load(F + (t0 + u) * C + c) : Row4<TS>::zero();
      }
      float part[NV];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float e[KR][4];
        cg.components(cur, g, e);
        int pi = 0;
#pragma unroll
        for (int a = 0; a < KR; ++a)
#pragma unroll
          for (int b = a; b < KR; ++b, ++pi) {
            float v = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q) v = fmaf(e[a][q], e[b][q], v);
            part[g * NP + pi] = v;
          }
      }
      cg.advance(cur);
#pragma unroll
      for (int v = 0; v < NV; v += 4)
        *reinterpret_cast<float4*>(mine + v) =
            make_float4(part[v], v + 1 < NV ? part[v + 1 < NV ? v + 1 : 0] : 0.f,
                        v + 2 < NV ? part[v + 2 < NV ? v + 2 : 0] : 0.f,
                        v + 3 < NV ? part[v + 3 < NV ? v + 3 : 0] : 0.f);
      // LDS operations of one wave complete in issue order; the fences keep the
      // compiler from moving the column reads above the row writes (or the next
      // group's writes above these reads).
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
      if (lane < NV) {
        float sum = 0.f;
#pragma unroll 16
        for (int r = 0; r < kWave; ++r) sum += xpose[wave][r][lane];
        const int g = lane / NP, pi = lane % NP;
        if (u0 + g < nt) red[u0 + g][wave][pi] = sum;
      }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      __builtin_amdgcn_wave_barrier();
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

// Write-back Y_j = sum_l H^res_jl a_l + sum_b wb_jb e_b for the KK active rows
// (without H^res: Y_j = a_j + ...); SAVE keeps the rows read, NEXT forms the
// next sublayer's input.  The run's indices and coefficients are staged in LDS
// once, the write-back weights wb formed there from the Gram partials; the
// loads of a group of G tokens are issued together.  T is a multiple of G.
template <typename TS, int KK, int G, bool RES, bool SAVE, bool NEXT>
__global__ __launch_bounds__(256) void k_post_apply_run(TS* __restrict__ X, const TS* __restrict__ F, int64_t T,
                                                        int64_t S, int N, int C,
                                                        const float* __restrict__ conv_w,
                                                        const int32_t* __restrict__ idx,
                                                        const float* __restrict__ Hres,
                                                        const float* __restrict__ gpart, int64_t nchunk,
                                                        int gram_schmidt, const float* __restrict__ p,
                                                        const float* __restrict__ Hpost,
                                                        const float* __restrict__ Hpre_next,
                                                        const TS* __restrict__ base_next, TS* __restrict__ input_next,
                                                        TS* __restrict__ Xact_save) {
  using CG = ConvGroup<4, 8, 12>;
  using R = Row4<TS>;
  constexpr int KR = CG::KR;
  __shared__ __align__(16) float s_hr[RES ? kRun * KK * KK : 4];
  __shared__ __align__(16) float s_wb[kRun * KK * KR];
  __shared__ int32_t s_idx[kRun * KK];
  __shared__ float s_hn[NEXT ? kRun * kMaxN : 1];
  const int c = (int)(blockIdx.y * blockDim.x + threadIdx.x) * 4;
  const int64_t t0 = (int64_t)blockIdx.x * kRun;
  const int nt = (int)((T - t0 < kRun) ? T - t0 : kRun);
  for (int i = threadIdx.x; i < nt * KK; i += blockDim.x) s_idx[i] = idx[t0 * KK + i];
  // write-back weights of the run's tokens from their Gram partials (the same
  // per-token arithmetic as k_post_coef; every channel chunk of a run forms them)
  for (int u = threadIdx.x; u < nt; u += blockDim.x)
    post_coef_token(gpart, nchunk, T, t0 + u, KK, KR, gram_schmidt, p, Hpost, s_wb + u * KK * KR);
  if (RES)
    for (int i = threadIdx.x; i < nt * KK * KK; i += blockDim.x) s_hr[i] = Hres[t0 * KK * KK + i];
  if (NEXT)
    for (int i = threadIdx.x; i < nt * N; i += blockDim.x) s_hn[i] = Hpre_next[t0 * N + i];
  CG cg;
  cg.load_taps(conv_w, C, c);
  cg.init(F, t0, S, C, c);
  __syncthreads();
  for (int u0 = 0; u0 < nt; u0 += G) {
    const int64_t t = t0 + u0;
    if (t % S == 0) cg.reset();
    int32_t rows[G][KK];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int l = 0; l < KK; ++l) rows[g][l] = __builtin_amdgcn_readfirstlane(s_idx[(u0 + g) * KK + l]);
    float cur[G][4];
    typename R::raw a[G][KK], nb[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      R::unpack(R::load(F + (t + g) * C + c), cur[g]);
#pragma unroll
      for (int l = 0; l < KK; ++l) a[g][l] = R::load(X + ((t + g) * N + rows[g][l]) * (int64_t)C + c);
      if (NEXT) nb[g] = R::load(base_next + (t + g) * C + c);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int u = u0 + g;
      const int64_t tg = t + g;
      float e[KR][4];
      cg.components(cur, g, e);
      if (SAVE) {
#pragma unroll
        for (int l = 0; l < KK; ++l) R::store_raw(Xact_save + (tg * KK + l) * (int64_t)C + c, a[g][l]);
      }
      float af[KK][4];
#pragma unroll
      for (int l = 0; l < KK; ++l) R::unpack(a[g][l], af[l]);
      float nxt[4];
      if (NEXT) R::unpack(nb[g], nxt);
      const float* hr = s_hr + (RES ? u * KK * KK : 0);
      const float* wv = s_wb + u * KK * KR;
#pragma unroll
      for (int j = 0; j < KK; ++j) {
        float y[4];
        if (RES) {
#pragma unroll
          for (int q = 0; q < 4; ++q) y[q] = 0.f;
#pragma unroll
          for (int l = 0; l < KK; ++l) {
            const float h = hr[j * KK + l];
#pragma unroll
            for (int q = 0; q < 4; ++q) y[q] = fmaf(h, af[l][q], y[q]);
          }
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) y[q] = af[j][q];
        }
#pragma unroll
        for (int b = 0; b < KR; ++b) {
          const float w = wv[j * KR + b];
#pragma unroll
          for (int q = 0; q < 4; ++q) y[q] = fmaf(w, e[b][q], y[q]);
        }
        R::store(X + (tg * N + rows[g][j]) * (int64_t)C + c, y);
        if (NEXT) {
          R::round(y);
          const float h = s_hn[u * N + rows[g][j]];
#pragma unroll
          for (int q = 0; q < 4; ++q) nxt[q] = fmaf(h, y[q], nxt[q]);
        }
      }
      if (NEXT) R::store(input_next + tg * C + c, nxt);
    }
    cg.advance(cur);
  }
}

// threads per block of the run-based kernels for width C (4 channels each)
static inline int run_threads(int C) { return C >= 1024 ? 256 : C / 4; }
static inline bool run_ok(int C, int64_t S, int Kr, const int32_t* kappa) {
  if (Kr != 4 || kappa[0] != 4 || kappa[1] != 8 || kappa[2] != 12) return false;
  if (C % 4 != 0 || S % 4 != 0) return false;
  const int nthr = run_threads(C);
  return nthr % kWave == 0 && C % (nthr * 4) == 0;
}

int64_t gram_chunks(int C, int64_t S, int Kr, const int32_t* kappa) {
  if (run_ok(C, S, Kr, kappa)) return C / (run_threads(C) * 4);
  return post_chunks(C);
}

hipError_t launch_post_gram(int state_dtype, const void* F, int64_t T, int64_t S, int C, int Kr,
                            const int32_t* kappa, const float* conv_w, float* gpart, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (run_ok(C, S, Kr, kappa)) {
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

static hipError_t launch_post_coef(const float* gpart, int64_t nchunk, int64_t T, int k, int Kr, int gram_schmidt,
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
  // the token's routed rows (the same in every lane), then every row load,
  // issued before anything waits for one: the rows stay raw until used, and
  // the components (F) are formed while they are in flight
  int32_t rows[kMaxK];
#pragma unroll
  for (int l = 0; l < kMaxK; ++l) rows[l] = idx[t * k + (l < k ? l : 0)];
  typename Raw8<TS>::raw ar[kMaxK] = {}, nr = {};
#pragma unroll
  for (int l = 0; l < kMaxK; ++l)
    if (l < k) ar[l] = Raw8<TS>::load(X + (t * N + rows[l]) * (int64_t)C + c);
  if (input_next) nr = Raw8<TS>::load(base_next + t * C + c);
  float e[KR][8];
  components<TS, KR>(F, conv_w, t, t % S, C, c, kap, e);
  float a[kMaxK][8];
#pragma unroll
  for (int l = 0; l < kMaxK; ++l) {
    if (l < k) {
      Raw8<TS>::unpack(ar[l], a[l]);
      if (Xact_save) Raw8<TS>::store(Xact_save + (t * k + l) * (int64_t)C + c, ar[l]);
    }
  }
  float nxt[8];
  if (input_next) Raw8<TS>::unpack(nr, nxt);
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
                             const float* Hres, const float* Hpost, const float* gpart, int64_t nchunk,
                             int gram_schmidt, float* wb, const float* Hpre_next, const void* base_next,
                             void* input_next, void* Xact_save, hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (gpart && run_ok(C, S, Kr, kappa) && T % 4 == 0 && (k == 4 || k == 8) &&
      !(Hres && input_next) && !(Xact_save && (input_next || !Hres))) {
    const int nthr = run_threads(C);
    const dim3 grid((unsigned)((T + kRun - 1) / kRun), (unsigned)(C / (nthr * 4)));
#define XHC_APPLY_RUN(TS, KK, G, RES, SAVE, NEXT)                                                                  \
  k_post_apply_run<TS, KK, G, RES, SAVE, NEXT><<<grid, dim3(nthr), 0, s>>>(                                      \
      reinterpret_cast<TS*>(X), reinterpret_cast<const TS*>(F), T, S, N, C, conv_w, idx, Hres, gpart, nchunk,    \
      gram_schmidt, p, Hpost, Hpre_next,                                                                         \
      reinterpret_cast<const TS*>(base_next), reinterpret_cast<TS*>(input_next), reinterpret_cast<TS*>(Xact_save))
#define XHC_APPLY_MODES(TS, KK, G)                                              \
  do {                                                                          \
    if (input_next) XHC_APPLY_RUN(TS, KK, G, false, false, true);               \
    else if (Xact_save) XHC_APPLY_RUN(TS, KK, G, true, true, false);            \
    else XHC_APPLY_RUN(TS, KK, G, true, false, false);                          \
  } while (0)
    if (state_dtype == XHC_BF16) {
      if (k == 4) XHC_APPLY_MODES(uint16_t, 4, 4); else XHC_APPLY_MODES(uint16_t, 8, 2);
    } else {
      if (k == 4) XHC_APPLY_MODES(float, 4, 2); else XHC_APPLY_MODES(float, 8, 1);
    }
#undef XHC_APPLY_MODES
#undef XHC_APPLY_RUN
    return hipGetLastError();
  }
  if (gpart) {
    const hipError_t e = launch_post_coef(gpart, nchunk, T, k, Kr, gram_schmidt, p, Hpost, wb, s);
    if (e != hipSuccess) return e;
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

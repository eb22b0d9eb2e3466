// Backward of a full xHC sublayer (reverse mode of xhc_pre + xhc_post).
//
// post backward
//  k_bwd_post_dots    per token and channel chunk: <dY_j, a_l>, <dY_j, e_b> and the
//                     Gram matrix of the components e_b (partials)
//  k_bwd_post_token   per token: dH^res, dH^post, dp; reverse of the Gram-Schmidt
//                     coefficients; coefficients of de_b in terms of dY_j and e_b'
//  k_bwd_post_elem    per element: gradient pass-through of the untouched rows,
//                     mixing gradient of the active rows, restore of the active rows,
//                     de_b (component gradients)
//  k_bwd_conv         dF = de_0 + anti-causal convolution of de_j;  k_bwd_convw: kernel
//                     gradient partials over token chunks
// pre backward
//  k_bwd_dhpre        per token and chunk: <d input, x_i> partials
//  k_bwd_pre_token    per token: sigmoid / Sinkhorn / routing reverses, norm-correction
//                     scalars, per-token gating and bias gradients
//  k_bwd_full_rows    weight-stationary over rows of [W_r | W_pre]: dX of every row,
//                     dW_r and dW_pre
//  k_bwd_act_rows     weight-stationary over rows of [W_post | W_res]: dX of the active
//                     rows, dW_post and dW_res partials
//  k_colsum_rows      deterministic column sums (token reductions)
#include "xhc_conv.h"
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {

// ------------------------------------------------------------ small-matrix reverses

// Reverse of gram_schmidt_basis: given G, V = GS(G) and the cotangent dV,
// return dG (G's entries taken as independent).
__device__ inline void gram_schmidt_basis_reverse(const double (&G)[kMaxKr][kMaxKr], int Kr,
                                                  const double (&dV_in)[kMaxKr][kMaxKr],
                                                  double (&dG)[kMaxKr][kMaxKr]) {
  // recompute the forward quantities
  double V[kMaxKr][kMaxKr], nrm[kMaxKr], dot[kMaxKr][kMaxKr], c[kMaxKr][kMaxKr];
  bool zero[kMaxKr];
  for (int i = 0; i < kMaxKr; ++i)
    for (int b = 0; b < kMaxKr; ++b) { V[i][b] = (i == b) ? 1.0 : 0.0; dot[i][b] = 0.0; c[i][b] = 0.0; dG[i][b] = 0.0; }
  for (int j = 0; j < Kr; ++j) {
    for (int i = 0; i < j; ++i) {
      if (zero[i]) continue;
      double d = 0.0;
      for (int b = 0; b < kMaxKr; ++b) d += V[i][b] * G[j][b];
      dot[j][i] = d;
      c[j][i] = d / nrm[i];
      for (int b = 0; b < kMaxKr; ++b) V[j][b] -= c[j][i] * V[i][b];
    }
    double n = 0.0;
    for (int a = 0; a < kMaxKr; ++a)
      for (int b = 0; b < kMaxKr; ++b) n += V[j][a] * G[a][b] * V[j][b];
    nrm[j] = n;
    zero[j] = n <= 1e-6 * G[j][j];   // a NaN norm is not "vanishing": it propagates
  }
  double dV[kMaxKr][kMaxKr], dnrm[kMaxKr];
  for (int i = 0; i < kMaxKr; ++i) {
    dnrm[i] = 0.0;
    for (int b = 0; b < kMaxKr; ++b) dV[i][b] = dV_in[i][b];
  }
  for (int j = Kr - 1; j >= 0; --j) {
    // nrm[j] = V_j^T G V_j (the zero decision is piecewise constant)
    if (dnrm[j] != 0.0) {
      for (int a = 0; a < kMaxKr; ++a) {
        double gv = 0.0;
        for (int b = 0; b < kMaxKr; ++b) gv += G[a][b] * V[j][b];
        dV[j][a] += 2.0 * gv * dnrm[j];
        for (int b = 0; b < kMaxKr; ++b) dG[a][b] += dnrm[j] * V[j][a] * V[j][b];
      }
    }
    // V_j = e_j - sum_i c_ji V_i with c_ji = <e_j, v_i> / nrm_i
    for (int i = j - 1; i >= 0; --i) {
      if (zero[i]) continue;
      double dc = 0.0;
      for (int b = 0; b < kMaxKr; ++b) dc -= dV[j][b] * V[i][b];
      for (int b = 0; b < kMaxKr; ++b) dV[i][b] -= c[j][i] * dV[j][b];
      const double ddot = dc / nrm[i];
      dnrm[i] -= dc * dot[j][i] / (nrm[i] * nrm[i]);
      for (int b = 0; b < kMaxKr; ++b) {
        dV[i][b] += ddot * G[j][b];
        dG[j][b] += ddot * V[i][b];
      }
    }
  }
}

// Forward Sinkhorn state after `steps` normalisations (rows first) of exp(L - rowmax).
__device__ inline void sinkhorn_steps(const float (&L)[kMaxK * kMaxK], int k, int steps, float (&M)[kMaxK * kMaxK]) {
  for (int j = 0; j < k; ++j) {
    float mx = L[j * kMaxK];
    for (int l = 1; l < k; ++l) mx = fmaxf(mx, L[j * kMaxK + l]);
    for (int l = 0; l < k; ++l) M[j * kMaxK + l] = __expf(L[j * kMaxK + l] - mx);
  }
  for (int s = 0; s < steps; ++s) {
    if ((s & 1) == 0) {
      for (int j = 0; j < k; ++j) {
        float sum = 0.f;
        for (int l = 0; l < k; ++l) sum += M[j * kMaxK + l];
        const float r = 1.0f / sum;
        for (int l = 0; l < k; ++l) M[j * kMaxK + l] *= r;
      }
    } else {
      for (int l = 0; l < k; ++l) {
        float sum = 0.f;
        for (int j = 0; j < k; ++j) sum += M[j * kMaxK + l];
        const float r = 1.0f / sum;
        for (int j = 0; j < k; ++j) M[j * kMaxK + l] *= r;
      }
    }
  }
}

// dL of H = clamp(SK_iters(exp(L))) given dH; the forward iterates are recomputed.
__device__ inline void sinkhorn_clamp_reverse(const float (&L)[kMaxK * kMaxK], int k, int iters, float delta,
                                              const float (&dH)[kMaxK * kMaxK], float (&dL)[kMaxK * kMaxK]) {
  float M[kMaxK * kMaxK], g[kMaxK * kMaxK];
  const int steps = 2 * iters;
  sinkhorn_steps(L, k, steps, M);
  // row clamp
  for (int j = 0; j < k; ++j) {
    float s = 0.f;
    for (int l = 0; l < k; ++l) s += M[j * kMaxK + l];
    if (s > 1.0f + delta) {
      float dot = 0.f;
      for (int l = 0; l < k; ++l) dot += dH[j * kMaxK + l] * (M[j * kMaxK + l] / s);
      for (int l = 0; l < k; ++l) g[j * kMaxK + l] = (dH[j * kMaxK + l] - dot) / s;
    } else {
      for (int l = 0; l < k; ++l) g[j * kMaxK + l] = dH[j * kMaxK + l];
    }
  }
  for (int s = steps - 1; s >= 0; --s) {
    sinkhorn_steps(L, k, s, M);   // input of normalisation step s
    if ((s & 1) == 0) {           // row normalisation: y = m / sum_l m
      for (int j = 0; j < k; ++j) {
        float sum = 0.f;
        for (int l = 0; l < k; ++l) sum += M[j * kMaxK + l];
        float dot = 0.f;
        for (int l = 0; l < k; ++l) dot += g[j * kMaxK + l] * (M[j * kMaxK + l] / sum);
        for (int l = 0; l < k; ++l) g[j * kMaxK + l] = (g[j * kMaxK + l] - dot) / sum;
      }
    } else {                      // column normalisation
      for (int l = 0; l < k; ++l) {
        float sum = 0.f;
        for (int j = 0; j < k; ++j) sum += M[j * kMaxK + l];
        float dot = 0.f;
        for (int j = 0; j < k; ++j) dot += g[j * kMaxK + l] * (M[j * kMaxK + l] / sum);
        for (int j = 0; j < k; ++j) g[j * kMaxK + l] = (g[j * kMaxK + l] - dot) / sum;
      }
    }
  }
  sinkhorn_steps(L, k, 0, M);     // exp(L - rowmax); the shift does not change H
  for (int j = 0; j < k; ++j)
    for (int l = 0; l < k; ++l) dL[j * kMaxK + l] = g[j * kMaxK + l] * M[j * kMaxK + l];
}

// The same for a compile-time k: the forward normaliser of every step is kept
// (sk[step][j] at sk[(step * K + j) * stride], LDS), so the reverse walks back
// step by step, undoing each normalisation on the iterate instead of
// recomputing it from the start.
constexpr int kSkMaxSteps = 64;   // 2 x sinkhorn_iters handled by the fast reverse
template <int K>
__device__ inline void sinkhorn_clamp_reverse_fast(const float (&L)[K * K], int iters, float delta,
                                                   const float (&dH)[K * K], float (&dL)[K * K], float* sk,
                                                   int stride) {
  float E[K * K], M[K * K], g[K * K];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    float mx = L[j * K];
#pragma unroll
    for (int l = 1; l < K; ++l) mx = fmaxf(mx, L[j * K + l]);
#pragma unroll
    for (int l = 0; l < K; ++l) M[j * K + l] = E[j * K + l] = __expf(L[j * K + l] - mx);
  }
  const int steps = 2 * iters;
  for (int st = 0; st < steps; ++st) {
    if ((st & 1) == 0) {
#pragma unroll
      for (int j = 0; j < K; ++j) {
        float sum = 0.f;
#pragma unroll
        for (int l = 0; l < K; ++l) sum += M[j * K + l];
        sk[(st * K + j) * stride] = sum;
        const float r = 1.0f / sum;
#pragma unroll
        for (int l = 0; l < K; ++l) M[j * K + l] *= r;
      }
    } else {
#pragma unroll
      for (int l = 0; l < K; ++l) {
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) sum += M[j * K + l];
        sk[(st * K + l) * stride] = sum;
        const float r = 1.0f / sum;
#pragma unroll
        for (int j = 0; j < K; ++j) M[j * K + l] *= r;
      }
    }
  }
  // row clamp
#pragma unroll
  for (int j = 0; j < K; ++j) {
    float sum = 0.f;
#pragma unroll
    for (int l = 0; l < K; ++l) sum += M[j * K + l];
    if (sum > 1.0f + delta) {
      float dot = 0.f;
#pragma unroll
      for (int l = 0; l < K; ++l) dot += dH[j * K + l] * (M[j * K + l] / sum);
#pragma unroll
      for (int l = 0; l < K; ++l) g[j * K + l] = (dH[j * K + l] - dot) / sum;
    } else {
#pragma unroll
      for (int l = 0; l < K; ++l) g[j * K + l] = dH[j * K + l];
    }
  }
  // M holds the output of step st; its input is M times the step's normaliser
  for (int st = steps - 1; st >= 0; --st) {
    if ((st & 1) == 0) {
#pragma unroll
      for (int j = 0; j < K; ++j) {
        const float sum = sk[(st * K + j) * stride];
        float dot = 0.f;
#pragma unroll
        for (int l = 0; l < K; ++l) dot += g[j * K + l] * M[j * K + l];
#pragma unroll
        for (int l = 0; l < K; ++l) {
          g[j * K + l] = (g[j * K + l] - dot) / sum;
          M[j * K + l] *= sum;
        }
      }
    } else {
#pragma unroll
      for (int l = 0; l < K; ++l) {
        const float sum = sk[(st * K + l) * stride];
        float dot = 0.f;
#pragma unroll
        for (int j = 0; j < K; ++j) dot += g[j * K + l] * M[j * K + l];
#pragma unroll
        for (int j = 0; j < K; ++j) {
          g[j * K + l] = (g[j * K + l] - dot) / sum;
          M[j * K + l] *= sum;
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < K * K; ++i) dL[i] = g[i] * E[i];
}

// ------------------------------------------------------------ post backward

// Layout of the per-token dot products (compile-time strides, KM >= k):
// [<dY_j, a_l> (KM x KM) | <dY_j, e_b> (KM x KR) | Gram of e (upper triangle)]
template <int KR, int KM>
struct PostDots {
  static constexpr int NG = KR * (KR + 1) / 2;
  static constexpr int ND = KM * KM + KM * KR + NG;
  static __host__ __device__ constexpr int ya(int j, int l) { return j * KM + l; }
  static __host__ __device__ constexpr int ye(int j, int b) { return KM * KM + j * KR + b; }
  static __host__ __device__ constexpr int gram(int p) { return KM * KM + KM * KR + p; }
};

// TS: element type of the state tensors (Xact, F); TG: of the state
// gradient (dXn), fp32 for the xHC-Flash active-row gradient.  ELEM (K_r = 1
// only, where the element pass needs no dot product: its weights are
// p_j H^post_j): the same thread also writes the element pass from the rows it
// has loaded, the mixing gradient into the active rows of dX (which may be dXn
// itself: every row is read before any is written), the restored rows into X
// (when given) and dF, so the gradient rows are read once.
template <typename TS, typename TG, int KR, int KM, bool ELEM = false>
__global__ __launch_bounds__(256) void k_bwd_post_dots(const TG* dXn, const TS* __restrict__ Xact,
                                                       const TS* __restrict__ F, int64_t T, int64_t S, int N, int C,
                                                       int k, int kap0, int kap1, int kap2,
                                                       const float* __restrict__ conv_w,
                                                       const int32_t* __restrict__ idx, float* __restrict__ part,
                                                       const float* __restrict__ Hres = nullptr,
                                                       const float* __restrict__ p = nullptr,
                                                       const float* __restrict__ Hpost = nullptr,
                                                       TS* __restrict__ X = nullptr, TG* dX = nullptr,
                                                       TS* __restrict__ dF = nullptr) {
  static_assert(!ELEM || KR == 1, "the element pass needs the dot products when K_r > 1");
  using PD = PostDots<KR, KM>;
  constexpr int MAXD = PD::ND;
  __shared__ float red[4][MAXD];
  const int nd = MAXD;
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb, cb = blockIdx.x % ncb;
  const int c = (int)(cb * 256 + threadIdx.x) * 8;
  float acc[MAXD];
#pragma unroll
  for (int i = 0; i < MAXD; ++i) acc[i] = 0.f;
  if (c < C) {
    const int kap[3] = {kap0, kap1, kap2};
    // the routed rows, then every row load, issued before any is used (raw
    // until then); the components (F) are formed while they are in flight
    int32_t rows[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) rows[j] = idx[t * k + (j < k ? j : 0)];
    typename Raw8<TG>::raw dyr[KM] = {};
    typename Raw8<TS>::raw ar[KM] = {};
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if (j < k) {
        dyr[j] = Raw8<TG>::load(dXn + (t * N + rows[j]) * (int64_t)C + c);
        ar[j] = Raw8<TS>::load(Xact + (t * k + j) * (int64_t)C + c);
      }
    float e[KR][8];
    components<TS, KR>(F, conv_w, t, t % S, C, c, kap, e);
    float dy[KM][8], a[KM][8];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
#pragma unroll
      for (int q = 0; q < 8; ++q) { dy[j][q] = 0.f; a[j][q] = 0.f; }
      if (j < k) {
        Raw8<TG>::unpack(dyr[j], dy[j]);
        Raw8<TS>::unpack(ar[j], a[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < KM; ++j)
#pragma unroll
      for (int l = 0; l < KM; ++l)
        if (j < k && l < k)
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[PD::ya(j, l)] = fmaf(dy[j][q], a[l][q], acc[PD::ya(j, l)]);
#pragma unroll
    for (int j = 0; j < KM; ++j)
#pragma unroll
      for (int b = 0; b < KR; ++b)
        if (j < k)
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[PD::ye(j, b)] = fmaf(dy[j][q], e[b][q], acc[PD::ye(j, b)]);
    int pi = PD::gram(0);
#pragma unroll
    for (int a0 = 0; a0 < KR; ++a0)
#pragma unroll
      for (int b = a0; b < KR; ++b, ++pi)
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[pi] = fmaf(e[a0][q], e[b][q], acc[pi]);
    if constexpr (ELEM) {
      // the element pass (the arithmetic of k_bwd_post_elem at K_r = 1)
#pragma unroll
      for (int l = 0; l < KM; ++l) {
        if (l >= k) break;
        float g[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) g[q] = 0.f;
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          if (j < k) {
            const float h = Hres[(t * k + j) * k + l];
#pragma unroll
            for (int q = 0; q < 8; ++q) g[q] = fmaf(h, dy[j][q], g[q]);
          }
        }
        Vec8<TG>::store(dX + (t * N + rows[l]) * (int64_t)C + c, g);
        if (X) Raw8<TS>::store(X + (t * N + rows[l]) * (int64_t)C + c, ar[l]);
      }
      float g[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) g[q] = 0.f;
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        if (j < k) {
          const float w = (float)((double)p[t * k + j] * (double)Hpost[t * k + j]);   // the coefficient pass's cf
#pragma unroll
          for (int q = 0; q < 8; ++q) g[q] = fmaf(w, dy[j][q], g[q]);
        }
      }
      Vec8<TS>::store(dF + t * C + c, g);
    }
  }
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
#pragma unroll
  for (int i = 0; i < MAXD; ++i) {
    float v = acc[i];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) red[wave][i] = v;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nd; i += 256) part[(cb * nd + i) * T + t] = red[0][i] + red[1][i] + red[2][i] + red[3][i];
}

// The dot products of k_bwd_post_dots for the paper's branches (K_r = 4,
// kappa = 4, 8, 12) and k <= 4, run-based: a thread owns 4 channels and walks
// a run of kDotRun tokens, keeping the conv taps and the last 11 values of F
// in registers (F read once), with the loads of the next PF tokens in
// flight.  Per token a wave sums its lanes' products through an LDS transpose
// (lane i adds column i) and lanes i < ND write them: part[w][t][i] with w the
// wave's 256-channel slice of C (workgroups of 256 or 64 threads).
constexpr int kDotRun = 64;
template <typename TS, typename TG>
__global__ __launch_bounds__(256) void k_bwd_post_dots_run(const TG* dXn, const TS* __restrict__ Xact,
                                                           const TS* __restrict__ F, int64_t T, int64_t S, int N,
                                                           int C, int k, const float* __restrict__ conv_w,
                                                           const int32_t* __restrict__ idx, float* __restrict__ part) {
  using CG = ConvGroup<4, 8, 12>;
  using PD = PostDots<4, 4>;
  constexpr int KM = 4, ND = PD::ND, LD = (ND + 3) / 4 * 4 + 4, PF = 1;
  static_assert(ND <= kWave, "one column per lane");
  __shared__ __align__(16) float xpose[4][kWave][LD];
  __shared__ int32_t s_idx[kDotRun][KM];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int g = (int)(blockIdx.y * blockDim.x + threadIdx.x);   // C % (4 blockDim.x) == 0
  const int c = g * 4, slice = g / kWave;
  const int64_t t0 = (int64_t)blockIdx.x * kDotRun;
  const int nt = (int)((T - t0 < kDotRun) ? T - t0 : kDotRun);
  for (int i = threadIdx.x; i < nt * KM; i += blockDim.x) {   // (workgroups of 64 or 256 threads)
    const int j = i % KM < k ? i % KM : k - 1;   // unused slots repeat the last one (in bounds)
    s_idx[i / KM][i % KM] = idx[(t0 + i / KM) * k + j];
  }
  CG cg;
  cg.load_taps(conv_w, C, c);
  cg.init(F, t0, S, C, c);
  __syncthreads();
  struct Tok {
    typename Row4<TS>::raw f, a[KM];
    typename Row4<TG>::raw y[KM];
  };
  // every load is issued (past the run from the last token: in bounds)
  auto load = [&](int u, Tok& b) {
    const int uc = u < nt ? u : nt - 1;
    const int64_t t = t0 + uc;
    b.f = Row4<TS>::load(F + t * C + c);
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      b.y[j] = Row4<TG>::load(dXn + (t * N + s_idx[uc][j]) * (int64_t)C + c);
      b.a[j] = Row4<TS>::load(Xact + (t * k + (j < k ? j : k - 1)) * (int64_t)C + c);
    }
  };
  float* mine = &xpose[wave][lane][0];
  Tok ring[PF];
#pragma unroll
  for (int f = 0; f < PF; ++f) load(f, ring[f]);
  for (int u1 = 0; u1 < nt; u1 += PF) {
#pragma unroll
    for (int f = 0; f < PF; ++f) {
      const int u = u1 + f;
      if (u < nt) {   // (no early exit: the loop unrolls and the ring stays in registers)
        const int64_t t = t0 + u;
        if (t % S == 0) cg.reset();
        float cur[1][4], dy[KM][4], a[KM][4];
        Row4<TS>::unpack(ring[f].f, cur[0]);
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          Row4<TG>::unpack(ring[f].y[j], dy[j]);
          Row4<TS>::unpack(ring[f].a[j], a[j]);
          if (j >= k) {
#pragma unroll
            for (int q = 0; q < 4; ++q) { dy[j][q] = 0.f; a[j][q] = 0.f; }
          }
        }
        load(u + PF, ring[f]);
        float e[4][4];
        cg.components(cur, 0, e);
        cg.advance(cur);
        // the lane's products, written to its LDS row in groups of 4 as formed
        // (ya row j, then ye row j, then the Gram)
        auto dot4 = [&](const float (&x)[4], const float (&y)[4]) {
          float v = 0.f;
#pragma unroll
          for (int q = 0; q < 4; ++q) v = fmaf(x[q], y[q], v);
          return v;
        };
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          *reinterpret_cast<float4*>(mine + PD::ya(j, 0)) =
              make_float4(dot4(dy[j], a[0]), dot4(dy[j], a[1]), dot4(dy[j], a[2]), dot4(dy[j], a[3]));
          *reinterpret_cast<float4*>(mine + PD::ye(j, 0)) =
              make_float4(dot4(dy[j], e[0]), dot4(dy[j], e[1]), dot4(dy[j], e[2]), dot4(dy[j], e[3]));
        }
        static_assert(PD::gram(0) % 4 == 0 && ND - PD::gram(0) == 10, "Gram block: 10 values after 32");
        *reinterpret_cast<float4*>(mine + PD::gram(0)) =
            make_float4(dot4(e[0], e[0]), dot4(e[0], e[1]), dot4(e[0], e[2]), dot4(e[0], e[3]));
        *reinterpret_cast<float4*>(mine + PD::gram(4)) =
            make_float4(dot4(e[1], e[1]), dot4(e[1], e[2]), dot4(e[1], e[3]), dot4(e[2], e[2]));
        *reinterpret_cast<float2*>(mine + PD::gram(8)) = make_float2(dot4(e[2], e[3]), dot4(e[3], e[3]));
        // LDS operations of one wave complete in issue order; the fences keep
        // the compiler from moving the column reads above the row writes (or
        // the next token's writes above these reads)
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
        if (lane < ND) {
          float sum = 0.f;
#pragma unroll 16
          for (int r = 0; r < kWave; ++r) sum += xpose[wave][r][lane];
          part[((int64_t)slice * T + t) * ND + lane] = sum;
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
      }
    }
  }
}

// Per token: dH^res, dH^post, dp and the coefficients of the component
// gradients: de_b = sum_j CY[b][j] dY_j + sum_b' CE[b][b'] e_b'.
// part: value i of chunk c for token t at c cs + i is + t ts.
template <int KR, int KM>
__global__ __launch_bounds__(128) void k_bwd_post_token(const float* __restrict__ part, int64_t nchunk, int64_t cs,
                                                        int64_t is, int64_t ts, int64_t T, int k, int gram_schmidt,
                                                        const float* __restrict__ p, const float* __restrict__ Hpost,
                                                        float* __restrict__ dHres, float* __restrict__ dHpost,
                                                        float* __restrict__ dp, float* __restrict__ coef) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  using PD = PostDots<KR, KM>;
  // the chunk sums of all PD::ND values, each chunk's values loaded together
  // (summed in the order chunk 0, 1, ...); every index below is a constant
  float ds[PD::ND];
#pragma unroll
  for (int i = 0; i < PD::ND; ++i) ds[i] = 0.f;
  for (int64_t c = 0; c < nchunk; ++c) {
    float v[PD::ND];
#pragma unroll
    for (int i = 0; i < PD::ND; ++i) v[i] = part[c * cs + i * is + t * ts];
#pragma unroll
    for (int i = 0; i < PD::ND; ++i) ds[i] += v[i];
  }
#pragma unroll
  for (int j = 0; j < KM; ++j)
#pragma unroll
    for (int l = 0; l < KM; ++l)
      if (j < k && l < k) dHres[(t * k + j) * k + l] = ds[PD::ya(j, l)];
  double D2[kMaxK][kMaxKr];   // <dY_j, e_b>
#pragma unroll
  for (int j = 0; j < kMaxK; ++j)
#pragma unroll
    for (int b = 0; b < kMaxKr; ++b) D2[j][b] = (j < KM && j < k && b < KR) ? (double)ds[PD::ye(j < KM ? j : 0, b < KR ? b : 0)] : 0.0;
  double G[kMaxKr][kMaxKr];
  int pi = PD::gram(0);
#pragma unroll
  for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
    for (int b = a; b < kMaxKr; ++b) {
      if (a < KR && b < KR) {
        G[a][b] = G[b][a] = ds[pi];
        ++pi;
      } else {
        G[a][b] = G[b][a] = 0.0;
      }
    }
  double V[kMaxKr][kMaxKr];
  if (gram_schmidt && KR > 1) {
    gram_schmidt_basis(G, KR, V);
  } else {
    for (int i = 0; i < kMaxKr; ++i)
      for (int b = 0; b < kMaxKr; ++b) V[i][b] = (i == b) ? 1.0 : 0.0;
  }
  // <dY_j, v_r> = sum_b V[r][b] <dY_j, e_b>
  double P[kMaxKr][kMaxKr];   // P[r][b] = <dv_r, e_b>, dv_r = sum_j p_j H^post[j][r] dY_j
  for (int r = 0; r < kMaxKr; ++r)
    for (int b = 0; b < kMaxKr; ++b) P[r][b] = 0.0;
  for (int j = 0; j < k; ++j) {
    const double pj = p[t * k + j];
    double dpj = 0.0;
    for (int r = 0; r < KR; ++r) {
      double yv = 0.0;
      for (int b = 0; b < KR; ++b) yv += V[r][b] * D2[j][b];
      const double h = Hpost[(t * k + j) * KR + r];
      dHpost[(t * k + j) * KR + r] = (float)(pj * yv);
      dpj += h * yv;
      for (int b = 0; b < KR; ++b) P[r][b] += pj * h * D2[j][b];
    }
    dp[t * k + j] = (float)dpj;
  }
  double dG[kMaxKr][kMaxKr];
  for (int a = 0; a < kMaxKr; ++a)
    for (int b = 0; b < kMaxKr; ++b) dG[a][b] = 0.0;
  if (gram_schmidt && KR > 1) gram_schmidt_basis_reverse(G, KR, P, dG);
  // coef layout per token: CY [KR][k] then CE [KR][KR]
  float* cf = coef + t * (KR * kMaxK + KR * KR);
  for (int b = 0; b < KR; ++b) {
    for (int j = 0; j < k; ++j) {
      double s = 0.0;
      for (int r = 0; r < KR; ++r) s += V[r][b] * (double)Hpost[(t * k + j) * KR + r];
      cf[b * kMaxK + j] = (float)((double)p[t * k + j] * s);
    }
    for (int b2 = 0; b2 < KR; ++b2) cf[KR * kMaxK + b * KR + b2] = (float)(dG[b][b2] + dG[b2][b]);
  }
}

// Element pass of the post backward (8 channels of one token per thread).
// dX may be dXn itself (in place): a thread reads the k active rows of its
// chunk before it writes any, and the untouched rows then already hold their
// gradient, so they are not copied.  TS: state tensors (X, Xact, F, dF);
// TG: the state gradient (dXn, dX).
template <typename TS, typename TG, int KR, int KM>
__global__ __launch_bounds__(256) void k_bwd_post_elem(const TG* dXn, TS* __restrict__ X,
                                                       const TS* __restrict__ Xact, const TS* __restrict__ F,
                                                       int64_t T, int64_t S, int N, int C, int k, int kap0, int kap1,
                                                       int kap2, const float* __restrict__ conv_w,
                                                       const int32_t* __restrict__ idx,
                                                       const float* __restrict__ Hres,
                                                       const float* __restrict__ coef, TG* dX,
                                                       TS* __restrict__ dF, float* __restrict__ de) {
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb;
  const int c = (int)((blockIdx.x % ncb) * 256 + threadIdx.x) * 8;
  if (c >= C) return;
  // the token's routed rows (the same in every lane; slots past k repeat
  // slot 0 and are not used)
  int32_t rows[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) rows[j] = idx[t * k + (j < k ? j : 0)];
  uint64_t act = 0;
#pragma unroll
  for (int j = 0; j < KM; ++j)
    if (j < k) act |= 1ull << rows[j];
  // untouched rows pass their gradient through (nothing to do in place)
  for (int i = 0; i < N && dX != dXn; ++i) {
    if ((act >> i) & 1ull) continue;
    float g[8];
    Vec8<TG>::load(dXn + (t * N + i) * (int64_t)C + c, g);
    Vec8<TG>::store(dX + (t * N + i) * (int64_t)C + c, g);
  }
  // every row load is issued before any is used (raw until then)
  typename Raw8<TG>::raw dyr[KM] = {};
  typename Raw8<TS>::raw ar[KM] = {};
#pragma unroll
  for (int j = 0; j < KM; ++j)
    if (j < k) {
      dyr[j] = Raw8<TG>::load(dXn + (t * N + rows[j]) * (int64_t)C + c);
      if (X) ar[j] = Raw8<TS>::load(Xact + (t * k + j) * (int64_t)C + c);
    }
  float dy[KM][8];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
#pragma unroll
    for (int q = 0; q < 8; ++q) dy[j][q] = 0.f;
    if (j < k) Raw8<TG>::unpack(dyr[j], dy[j]);
  }
  // active rows: mixing gradient sum_j H^res[j][l] dY_j; restore the pre-update rows
#pragma unroll
  for (int l = 0; l < KM; ++l) {
    if (l >= k) break;
    float g[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) g[q] = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (j < k) {
        const float h = Hres[(t * k + j) * k + l];
#pragma unroll
        for (int q = 0; q < 8; ++q) g[q] = fmaf(h, dy[j][q], g[q]);
      }
    }
    Vec8<TG>::store(dX + (t * N + rows[l]) * (int64_t)C + c, g);
    if (X) Raw8<TS>::store(X + (t * N + rows[l]) * (int64_t)C + c, ar[l]);   // restore (left out when X is null)
  }
  const int kap[3] = {kap0, kap1, kap2};
  float e[KR][8];
  if (KR > 1) components<TS, KR>(F, conv_w, t, t % S, C, c, kap, e);
  const float* cf = coef + t * (KR * kMaxK + KR * KR);
#pragma unroll
  for (int b = 0; b < KR; ++b) {
    float g[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) g[q] = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (j < k) {
        const float w = cf[b * kMaxK + j];
#pragma unroll
        for (int q = 0; q < 8; ++q) g[q] = fmaf(w, dy[j][q], g[q]);
      }
    }
    if (KR > 1) {
#pragma unroll
      for (int b2 = 0; b2 < KR; ++b2) {
        const float w = cf[KR * kMaxK + b * KR + b2];
#pragma unroll
        for (int q = 0; q < 8; ++q) g[q] = fmaf(w, e[b2][q], g[q]);
      }
      float* dst = de + ((int64_t)b * T + t) * C + c;
      reinterpret_cast<float4*>(dst)[0] = make_float4(g[0], g[1], g[2], g[3]);
      reinterpret_cast<float4*>(dst)[1] = make_float4(g[4], g[5], g[6], g[7]);
    } else {
      Vec8<TS>::store(dF + t * C + c, g);
    }
  }
}

// dF[t] = de_0[t] + sum_j sum_{i < kappa_j} w_j[i] de_j[t + i] over the part of the
// window inside t's sequence (the reverse of the causal convolution).
template <typename TS>
__global__ __launch_bounds__(256) void k_bwd_conv(const float* __restrict__ de, int64_t T, int64_t S, int C, int Kr,
                                                  int kap0, int kap1, int kap2, const float* __restrict__ conv_w,
                                                  TS* __restrict__ dF) {
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb;
  const int c = (int)((blockIdx.x % ncb) * 256 + threadIdx.x) * 8;
  if (c >= C) return;
  const int kap[3] = {kap0, kap1, kap2};
  const int64_t room = S - 1 - (t % S);   // tokens after t in its sequence
  float g[8];
  {
    const float4* p4 = reinterpret_cast<const float4*>(de + t * C + c);
    const float4 u = p4[0], v = p4[1];
    g[0] = u.x; g[1] = u.y; g[2] = u.z; g[3] = u.w; g[4] = v.x; g[5] = v.y; g[6] = v.z; g[7] = v.w;
  }
  int row = 0;
  for (int j = 1; j < Kr; ++j) {
    const int kj = kap[j - 1];
    for (int i = 0; i < kj && i <= room; ++i) {
      const float4* w4 = reinterpret_cast<const float4*>(conv_w + (int64_t)(row + i) * C + c);
      const float4* d4 = reinterpret_cast<const float4*>(de + ((int64_t)j * T + t + i) * C + c);
      const float4 wa = w4[0], wb = w4[1], da = d4[0], db = d4[1];
      g[0] = fmaf(wa.x, da.x, g[0]); g[1] = fmaf(wa.y, da.y, g[1]);
      g[2] = fmaf(wa.z, da.z, g[2]); g[3] = fmaf(wa.w, da.w, g[3]);
      g[4] = fmaf(wb.x, db.x, g[4]); g[5] = fmaf(wb.y, db.y, g[5]);
      g[6] = fmaf(wb.z, db.z, g[6]); g[7] = fmaf(wb.w, db.w, g[7]);
    }
    row += kj;
  }
  Vec8<TS>::store(dF + t * C + c, g);
}

// Kernel-gradient partials: part[chunk][row][c] = sum_{t in chunk} F[t - i][c] de_j[t][c]
// for row = (branch j, tap i), only where t - i lies in t's sequence.
constexpr int kConvChunk = 256;   // tokens per partial
template <typename TS>
__global__ __launch_bounds__(256) void k_bwd_convw(const float* __restrict__ de, const TS* __restrict__ F, int64_t T,
                                                   int64_t S, int C, int Kr, int kap0, int kap1, int kap2,
                                                   float* __restrict__ part) {
  // grid: (channel blocks of 2048) x (conv rows) x (token chunks)
  const int c = (int)(blockIdx.x * 256 + threadIdx.x) * 8;
  const int row = blockIdx.y;
  const int64_t chunk = blockIdx.z;
  if (c >= C) return;
  const int kap[3] = {kap0, kap1, kap2};
  int j = 1, base = 0;
  while (j < Kr && row >= base + kap[j - 1]) { base += kap[j - 1]; ++j; }
  const int i = row - base;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const int64_t t0 = chunk * kConvChunk, t1 = (t0 + kConvChunk < T) ? t0 + kConvChunk : T;
  for (int64_t t = t0; t < t1; ++t) {
    if ((t % S) < i) continue;
    float f[8];
    Vec8<TS>::load(F + (t - i) * C + c, f);
    const float4* d4 = reinterpret_cast<const float4*>(de + ((int64_t)j * T + t) * C + c);
    const float4 da = d4[0], db = d4[1];
    acc[0] = fmaf(f[0], da.x, acc[0]); acc[1] = fmaf(f[1], da.y, acc[1]);
    acc[2] = fmaf(f[2], da.z, acc[2]); acc[3] = fmaf(f[3], da.w, acc[3]);
    acc[4] = fmaf(f[4], db.x, acc[4]); acc[5] = fmaf(f[5], db.y, acc[5]);
    acc[6] = fmaf(f[6], db.z, acc[6]); acc[7] = fmaf(f[7], db.w, acc[7]);
  }
  float* dst = part + ((int64_t)chunk * gridDim.y + row) * C + c;
  reinterpret_cast<float4*>(dst)[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  reinterpret_cast<float4*>(dst)[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

// The conv reverse for the paper's branches (kappa = 4, 8, 12; K_r = 4) in
// one pass over a run of kConvRun tokens, one channel per thread:
//   dF[v] = de_0[v] + sum_j sum_{i < kappa_j} w_j[i] de_j[v + i]   (inside v's sequence)
//   part[run][row (j, i)][c] = sum_{u in run} F[u - i] de_j[u]     (F = 0 before the sequence start)
// Registers keep the last 12 F values of the channel (for the tap
// gradients) and the pending dF of the last 12 tokens, into which de_j[u]
// is scattered (the anti-causal sum in scatter form); a token's dF is stored
// once the window has moved 12 past it, or at a sequence start, or at the
// end.  The run reads 11 tokens of de past its end (the last tokens' dF
// needs them).  Loads of the next 4 tokens are in flight while 4 are used.
constexpr int kConvRun = 128;
constexpr int kConvRows = 24;   // 4 + 8 + 12 taps
template <typename TS>
__device__ __forceinline__ float ld_scalar(const TS* p);
template <> __device__ __forceinline__ float ld_scalar<uint16_t>(const uint16_t* p) { return __uint_as_float((uint32_t)*p << 16); }
template <> __device__ __forceinline__ float ld_scalar<float>(const float* p) { return *p; }
// an element's bits as loaded (bf16 zero-extended), converted where it is used:
// a conversion next to the load would make the compiler wait for it there
template <typename TS>
__device__ __forceinline__ uint32_t ld_raw(const TS* p);
template <> __device__ __forceinline__ uint32_t ld_raw<uint16_t>(const uint16_t* p) { return *p; }
template <> __device__ __forceinline__ uint32_t ld_raw<float>(const float* p) { return __float_as_uint(*p); }
template <typename TS>
__device__ __forceinline__ float from_raw(uint32_t r);
template <> __device__ __forceinline__ float from_raw<uint16_t>(uint32_t r) { return __uint_as_float(r << 16); }
template <> __device__ __forceinline__ float from_raw<float>(uint32_t r) { return __uint_as_float(r); }
template <typename TS>
__device__ __forceinline__ void st_scalar(TS* p, float v);
// (the hardware conversion: the bits of f2bf except the payload of a NaN)
template <> __device__ __forceinline__ void st_scalar<uint16_t>(uint16_t* p, float v) { *p = (uint16_t)pack2bf(v, 0.f); }
template <> __device__ __forceinline__ void st_scalar<float>(float* p, float v) { *p = v; }

template <typename TS>
__global__ __launch_bounds__(256) void k_bwd_conv_run(const float* __restrict__ de, const TS* __restrict__ F, int64_t T,
                                                      int64_t S, int C, const float* __restrict__ conv_w,
                                                      TS* __restrict__ dF, float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  const int64_t t0 = (int64_t)blockIdx.y * kConvRun;
  const int64_t t1 = t0 + kConvRun < T ? t0 + kConvRun : T;
  const int64_t uend = t1 + 11 < T ? t1 + 11 : T;
  float w[kConvRows];
#pragma unroll
  for (int r = 0; r < kConvRows; ++r) w[r] = conv_w[(int64_t)r * C + c];
  float fw[12], acc[kConvRows], P[12];
  int64_t seq0 = t0 - t0 % S;   // start of the current sequence
#pragma unroll
  for (int i = 0; i < 12; ++i) {
    const int64_t t = t0 - i;   // fw[i] = F[u - i] for u = t0 - 1 + 1 after the first shift
    fw[i] = (i > 0 && t >= seq0) ? ld_scalar<TS>(F + t * C + c) : 0.f;
    P[i] = 0.f;
  }
#pragma unroll
  for (int r = 0; r < kConvRows; ++r) acc[r] = 0.f;
  // fw holds F[t0 - 1 - i] at index i + 1 for the first token: shift it down once
#pragma unroll
  for (int i = 0; i < 11; ++i) fw[i] = fw[i + 1];
  fw[11] = 0.f;
  auto store = [&](int64_t v, float x) {
    if (v >= t0 && v < t1 && v >= seq0) st_scalar<TS>(dF + v * C + c, x);
  };
  // loads of one token: de_0..3 and F
  auto load = [&](int64_t u, float (&d)[4], float& f) {
    if (u < uend) {
#pragma unroll
      for (int j = 0; j < 4; ++j) d[j] = de[((int64_t)j * T + u) * C + c];
      f = u < t1 ? ld_scalar<TS>(F + u * C + c) : 0.f;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) d[j] = 0.f;
      f = 0.f;
    }
  };
  float bd[2][4][4], bf[2][4];
#pragma unroll
  for (int k = 0; k < 4; ++k) load(t0 + k, bd[0][k], bf[0][k]);
  bool done = false;
  for (int64_t ub = t0; ub < uend && !done; ub += 8) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int cur = half, nxt = half ^ 1;
      const int64_t u4 = ub + 4 * half;
#pragma unroll
      for (int k = 0; k < 4; ++k) load(u4 + 4 + k, bd[nxt][k], bf[nxt][k]);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t u = u4 + k;
        if (done || u >= uend) break;
        if (u % S == 0 && u > t0) {
          // a sequence starts at u: the tokens before it are complete
#pragma unroll
          for (int i = 0; i < 12; ++i) store(u - 1 - i, P[i]);
          if (u >= t1) { done = true; break; }
          seq0 = u;
#pragma unroll
          for (int i = 0; i < 12; ++i) { P[i] = 0.f; fw[i] = 0.f; }
        }
        // token u - 12 has all its contributions
        store(u - 12, P[11]);
#pragma unroll
        for (int i = 11; i > 0; --i) { P[i] = P[i - 1]; fw[i] = fw[i - 1]; }
        fw[0] = bf[cur][k];
        const float* d = bd[cur][k];
        P[0] = d[0];
        int r = 0;
#pragma unroll
        for (int j = 1; j < 4; ++j) {
          const int kap = j == 1 ? 4 : (j == 2 ? 8 : 12);
#pragma unroll
          for (int i = 0; i < kap; ++i, ++r) {
            P[i] = fmaf(w[r], d[j], P[i]);
            if (u < t1) acc[r] = fmaf(fw[i], d[j], acc[r]);
          }
        }
      }
    }
  }
  if (!done) {
    // the tokens still pending: u - 1 - i for the last u + 1 = uend
#pragma unroll
    for (int i = 0; i < 12; ++i) store(uend - 1 - i, P[i]);
  }
  float* dst = part + (int64_t)blockIdx.y * kConvRows * C + c;
#pragma unroll
  for (int r = 0; r < kConvRows; ++r) dst[(int64_t)r * C] = acc[r];
}

// The element pass and the conv reverse of the post backward fused, for the
// paper's branches (kappa = 4, 8, 12; K_r = 4) and k <= 4: one channel per
// thread over a run of kConvRun tokens, nothing but the gradients leaving
// registers.  Per token u of the run:
//   dX[u, I_l] = sum_j H^res[j][l] dY_j          (mixing gradient of the active rows)
//   X[u, I_l]  = Xact[u, l]                        (restore, when X is given)
//   de_b[u]    = sum_j CY[b][j] dY_j + sum_b' CE[b][b'] e_b'[u]   (e from the F history)
//   dF[v]     += de_0 at v = u and w_j[i] de_j[u] at v = u - i      (the reverse of the causal conv)
//   part[run][row (j, i)][c] += F[u - i] de_j[u]
// The runs are disjoint, so an in-place dX never meets a token another run
// still reads.  A token's dF is stored once complete; the last 11 tokens of a
// run (later runs still add to them) go to rb[run][i] (token t1 - 11 + i)
// and a run's additions to the 11 tokens before it to lb[run][i] (token
// t0 - 11 + i, zero where they are in an earlier sequence); k_bwd_post_fix
// stores their sums.  The loads of the next 4 tokens are in flight while 4
// are used.  RESTORE: X is given (the saved rows are read and written back).
template <typename TS, typename TG, bool RESTORE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_bwd_post_run(const TG* dXn, TS* __restrict__ X, const TS* __restrict__ Xact,
                                                      const TS* __restrict__ F, int64_t T, int64_t S, int N, int C,
                                                      int k, const float* __restrict__ conv_w,
                                                      const int32_t* __restrict__ idx, const float* __restrict__ Hres,
                                                      const float* __restrict__ coef, TG* dX, TS* __restrict__ dF,
                                                      float* __restrict__ part, float* __restrict__ rb,
                                                      float* __restrict__ lb) {
  constexpr int KM = 4, NCF = 4 * kMaxK + 16;   // slots; coefficients a token
  // the run's per-token values, staged once: element offsets of the slot rows
  // from the run's first state row (32-bit: the launcher keeps kConvRun N C
  // below 2^31), H^res, the component-gradient coefficients
  __shared__ int32_t s_row[kConvRun][KM];
  __shared__ float s_hr[kConvRun][KM * KM];
  __shared__ float s_cf[kConvRun][NCF];
  const int c = blockIdx.x * 256 + threadIdx.x;   // C % 256 == 0: every thread has a channel
  const int64_t run = blockIdx.y;
  const int64_t t0 = run * kConvRun;
  const int64_t t1 = t0 + kConvRun < T ? t0 + kConvRun : T;
  const int nt = (int)(t1 - t0);
  const bool last = t1 == T;
  for (int i = threadIdx.x; i < nt * KM; i += 256) {
    const int64_t u = t0 + i / KM;
    const int j = i % KM < k ? i % KM : k - 1;   // unused slots repeat the last one (in bounds)
    s_row[i / KM][i % KM] = (int32_t)(((u - t0) * N + idx[u * k + j]) * (int64_t)C);
  }
  for (int i = threadIdx.x; i < nt * KM * KM; i += 256) {
    const int64_t u = t0 + i / (KM * KM);
    const int j = (i % (KM * KM)) / KM, l = i % KM;
    s_hr[i / (KM * KM)][i % (KM * KM)] = (j < k && l < k) ? Hres[(u * k + j) * k + l] : 0.f;
  }
  for (int i = threadIdx.x; i < nt * NCF; i += 256) s_cf[i / NCF][i % NCF] = coef[t0 * NCF + i];
  __syncthreads();
  float w[kConvRows];
#pragma unroll
  for (int r = 0; r < kConvRows; ++r) w[r] = conv_w[(int64_t)r * C + c];
  float fw[12], acc[kConvRows], P[12];
  int64_t seq0 = t0 - t0 % S;   // start of the current sequence
  // fw[i] = F[u - i] (zero before the sequence start); before the first token
  // it holds F[t0 - 1 - i] at index i.  The 11 loads are issued together (a
  // token before the sequence start reads the run's first token instead and
  // is zeroed), so the run start waits for one round trip, not eleven.
#pragma unroll
  for (int i = 0; i < 12; ++i) {
    const int64_t t = t0 - 1 - i;
    const bool in = i < 11 && t >= seq0;
    const float v = ld_scalar<TS>(F + (in ? t : t0) * C + c);
    fw[i] = in ? v : 0.f;
    P[i] = 0.f;
  }
#pragma unroll
  for (int r = 0; r < kConvRows; ++r) acc[r] = 0.f;
  float* const lbr = lb + run * 11 * (int64_t)C + c;
  if (run > 0)
#pragma unroll
    for (int i = 0; i < 11; ++i) lbr[(int64_t)i * C] = 0.f;
  // Per-run bases and per-token offsets that are the same in every lane
  // (32-bit), so an access is a scalar address plus the lane's channel.
  const uint32_t cu = (uint32_t)c;
  const int64_t sbase = t0 * N * (int64_t)C;
  const TG* const dXn_r = dXn + sbase;
  TG* const dX_r = dX + sbase;
  const TS* const Xact_r = Xact + t0 * k * (int64_t)C;
  const TS* const F_r = F + t0 * (int64_t)C;
  TS* const dF_r = dF + t0 * (int64_t)C;
  auto row_at = [&](int ul, int j) { return __builtin_amdgcn_readfirstlane(s_row[ul][j]); };
  // a token's dF, complete (or this run's additions to an earlier run's token)
  auto emit = [&](int64_t v, float x) {
    if (v < seq0) return;
    if (v >= t0) st_scalar<TS>(&(dF_r + (int32_t)(v - t0) * C)[cu], x);
    else if (v >= t0 - 11) lbr[(v - (t0 - 11)) * C] = x;
  };
  // loads of one token: dY of the k slots, the saved rows, F, as raw bits.
  // Every load is issued (past the run or the k slots from a clamped,
  // in-bounds address), so the buffers stay in registers and the loads stay
  // in flight together; the values are converted, and those of unused slots
  // replaced by zero, where the token is processed (tokens past the run never
  // are).
  auto load = [&](int64_t u, uint32_t (&dy)[KM], uint32_t (&a)[KM], uint32_t& f) {
    const int ul = (int)((u < t1 ? u : t1 - 1) - t0);
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      const int jc = j < k ? j : k - 1;
      dy[j] = ld_raw<TG>(&(dXn_r + row_at(ul, j))[cu]);
      a[j] = 0u;
      if (RESTORE) a[j] = ld_raw<TS>(&(Xact_r + (ul * k + jc) * C)[cu]);
    }
    f = ld_raw<TS>(&(F_r + ul * C)[cu]);
  };
  uint32_t bdy[2][4][KM], ba[2][4][KM], bf[2][4];
#pragma unroll
  for (int q = 0; q < 4; ++q) load(t0 + q, bdy[0][q], ba[0][q], bf[0][q]);
  int64_t pos = t0 % S;   // position of token u in its sequence
  for (int64_t ub = t0; ub < t1; ub += 8) {
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int cur = half, nxt = half ^ 1;
      const int64_t u4 = ub + 4 * half;
#pragma unroll
      for (int q = 0; q < 4; ++q) load(u4 + 4 + q, bdy[nxt][q], ba[nxt][q], bf[nxt][q]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t u = u4 + q;
        if (u < t1) {   // (no early exit: the loop unrolls and the buffers stay in registers)
        if (pos == 0 && u > t0) {
          // a sequence starts at u: the tokens before it are complete
#pragma unroll
          for (int i = 0; i < 12; ++i) emit(u - 1 - i, P[i]);
          seq0 = u;
#pragma unroll
          for (int i = 0; i < 12; ++i) { P[i] = 0.f; fw[i] = 0.f; }
        }
        // token u - 12 has all its contributions
        emit(u - 12, P[11]);
#pragma unroll
        for (int i = 11; i > 0; --i) { P[i] = P[i - 1]; fw[i] = fw[i - 1]; }
        fw[0] = from_raw<TS>(bf[cur][q]);
        float dy[KM], av[KM];
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          dy[j] = j < k ? from_raw<TG>(bdy[cur][q][j]) : 0.f;
          av[j] = (RESTORE && j < k) ? from_raw<TS>(ba[cur][q][j]) : 0.f;
        }
        // the components at u (eq:aug): F[u] and the three causal convolutions
        float e[4];
        e[0] = fw[0];
        {
          int r = 0;
#pragma unroll
          for (int j = 1; j < 4; ++j) {
            const int kap = j == 1 ? 4 : (j == 2 ? 8 : 12);
            float v = 0.f;
#pragma unroll
            for (int i = 0; i < kap; ++i, ++r) v = fmaf(w[r], fw[i], v);
            e[j] = v;
          }
        }
        const int ul = (int)(u - t0);
        const float* cf = s_cf[ul];
        float d[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          float g = 0.f;
#pragma unroll
          for (int j = 0; j < KM; ++j)
            if (j < k) g = fmaf(cf[b * kMaxK + j], dy[j], g);
#pragma unroll
          for (int b2 = 0; b2 < 4; ++b2) g = fmaf(cf[4 * kMaxK + b * 4 + b2], e[b2], g);
          d[b] = g;
        }
        // the active rows: mixing gradient, and the pre-update rows back in X
#pragma unroll
        for (int l = 0; l < KM; ++l) {
          if (l < k) {
            float g = 0.f;
#pragma unroll
            for (int j = 0; j < KM; ++j) g = fmaf(s_hr[ul][j * KM + l], dy[j], g);
            const int32_t ro = row_at(ul, l);
            st_scalar<TG>(&(dX_r + ro)[cu], g);
            if (RESTORE) st_scalar<TS>(&(X + sbase + ro)[cu], av[l]);
          }
        }
        P[0] = d[0];
        int r = 0;
#pragma unroll
        for (int j = 1; j < 4; ++j) {
          const int kap = j == 1 ? 4 : (j == 2 ? 8 : 12);
#pragma unroll
          for (int i = 0; i < kap; ++i, ++r) {
            P[i] = fmaf(w[r], d[j], P[i]);
            acc[r] = fmaf(fw[i], d[j], acc[r]);
          }
        }
        pos = pos + 1 == S ? 0 : pos + 1;
        }
      }
    }
  }
  // the tokens still pending: t1 - 1 - i.  The last run completes them; any
  // other run leaves t1 - 11 .. t1 - 1 (same sequence as t1 - 1) to the fix-up.
#pragma unroll
  for (int i = 0; i < 12; ++i) {
    const int64_t v = t1 - 1 - i;
    if (last || i == 11) emit(v, P[i]);
    else if (v >= seq0) rb[(run * 11 + (v - (t1 - 11))) * (int64_t)C + c] = P[i];
  }
  float* dst = part + run * kConvRows * (int64_t)C + c;
#pragma unroll
  for (int r = 0; r < kConvRows; ++r) dst[(int64_t)r * C] = acc[r];
}

// dF of the 11 tokens before each run boundary t1 = b kConvRun (b = 1 ..
// nruns - 1): the earlier run's part (rb) plus the later run's (lb), for the
// tokens in the sequence of t1 - 1 (the others were stored complete).
template <typename TS>
__global__ __launch_bounds__(256) void k_bwd_post_fix(const float* __restrict__ rb, const float* __restrict__ lb,
                                                      int64_t T, int64_t S, int C, TS* __restrict__ dF) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  const int64_t b = blockIdx.y + 1;
  const int i = blockIdx.z;
  const int64_t t1 = b * kConvRun;
  const int64_t v = t1 - 11 + i;
  const int64_t s_end = (t1 - 1) - (t1 - 1) % S;
  if (t1 >= T || v < s_end) return;
  st_scalar<TS>(dF + v * C + c, rb[((b - 1) * 11 + i) * (int64_t)C + c] + lb[(b * 11 + i) * (int64_t)C + c]);
}

// out[col] = sum_r in[r][col] over nrows rows (row stride = ncols), fixed order.
__global__ __launch_bounds__(256) void k_colsum_rows(const float* __restrict__ in, int64_t nrows, int64_t ncols,
                                                     float* __restrict__ out) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= ncols) return;
  float s = 0.f;
  for (int64_t r0 = 0; r0 < nrows; r0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (r0 + u < nrows) ? in[(r0 + u) * ncols + col] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  out[col] = s;
}

// out[col] = sum over T of in[t][col], for few columns: one block per column,
// threads stride the tokens, tree reduction in a fixed order.
__global__ __launch_bounds__(256) void k_sum_tokens(const float* __restrict__ in, int64_t T, int ncols,
                                                    float* __restrict__ out) {
  __shared__ float red[256];
  const int col = blockIdx.x;
  float s = 0.f;
  for (int64_t t = threadIdx.x; t < T; t += 256) s += in[t * ncols + col];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[col] = red[0];
}

// ------------------------------------------------------------ pre backward

// <d input, x_i> partials: part[chunk][i][t]
template <typename TS>
__global__ __launch_bounds__(256) void k_bwd_dhpre(const TS* __restrict__ X, const TS* __restrict__ din, int64_t T,
                                                   int N, int C, float* __restrict__ part) {
  __shared__ float red[4][kMaxN];
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb, cb = blockIdx.x % ncb;
  const int c = (int)(cb * 256 + threadIdx.x) * 8;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  float g[8];
  if (c < C) Vec8<TS>::load(din + t * C + c, g);
  for (int i = 0; i < N; ++i) {
    float v = 0.f;
    if (c < C) {
      float x[8];
      Vec8<TS>::load(X + (t * N + i) * (int64_t)C + c, x);
#pragma unroll
      for (int q = 0; q < 8; ++q) v = fmaf(g[q], x[q], v);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if (lane == 0) red[wave][i] = v;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < N; i += 256) part[(cb * N + i) * T + t] = red[0][i] + red[1][i] + red[2][i] + red[3][i];
}

// The same partials for NQ input gradients din + q T C at once (one read of
// the state): part[q][chunk][i][t]
struct MultiParts {
  float* part[4];
};
template <typename TS, int NQ>
__global__ __launch_bounds__(256) void k_bwd_dhpre_multi(const TS* __restrict__ X, const TS* __restrict__ din,
                                                         int64_t T, int N, int C, MultiParts mp) {
  __shared__ float red[NQ][4][kMaxN];
  const int64_t ncb = post_chunks(C);
  const int64_t t = blockIdx.x / ncb, cb = blockIdx.x % ncb;
  const int c = (int)(cb * 256 + threadIdx.x) * 8;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  float g[NQ][8];
#pragma unroll
  for (int q = 0; q < NQ; ++q)
    if (c < C) Vec8<TS>::load(din + ((int64_t)q * T + t) * C + c, g[q]);
  for (int i = 0; i < N; ++i) {
    float v[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) v[q] = 0.f;
    if (c < C) {
      float x[8];
      Vec8<TS>::load(X + (t * N + i) * (int64_t)C + c, x);
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[q] = fmaf(g[q][e], x[e], v[q]);
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) v[q] += __shfl_xor(v[q], off);
      if (lane == 0) red[q][wave][i] = v[q];
    }
  }
  __syncthreads();
  for (int u = threadIdx.x; u < NQ * N; u += 256) {
    const int q = u / N, i = u % N;
    mp.part[q][(cb * N + i) * T + t] = red[q][0][i] + red[q][1][i] + red[q][2][i] + red[q][3][i];
  }
}

// Per-token record written by k_bwd_pre_token (floats):
//   [dz_r (N) | dz_pre (N) | dz_act (NA) | r | r_ln | mu | beta_pre | m1 | m2 | r_a | beta_a]
// and per-token gating/bias gradients pg: [dalpha_pre, dalpha_res, dalpha_post | db_pre (N) |
// db_res (k*k) | db_post (k*Kr)].
// dL/dH^pre of the active streams given per slot: the chunk partials of
// <d input, x_i> at i = idx[t, j] become dhact[t, j] (first chunk) and 0.
__global__ __launch_bounds__(256) void k_bwd_dhpre_override(const float* __restrict__ dhact,
                                                            const int32_t* __restrict__ idx, int64_t T, int N, int k,
                                                            int64_t nchunk, float* __restrict__ part) {
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= T * k) return;
  const int64_t t = u / k;
  const int i = idx[u];
  for (int64_t c = 0; c < nchunk; ++c) part[(c * N + i) * T + t] = c == 0 ? dhact[u] : 0.0f;
}

__host__ __device__ inline int tok_floats(int N, int NA) { return 2 * N + NA + 8; }
__host__ __device__ inline int pg_floats(int N, int k, int Kr) { return 3 + N + k * k + k * Kr; }

// KC > 0: k == KC at compile time, Sinkhorn reversed with kept normalisers;
// KC == 0: any k, Sinkhorn reversed by recomputing the forward iterates.
constexpr int kPreTokThreads = 64;
template <int KC>
__global__ __launch_bounds__(kPreTokThreads) void k_bwd_pre_token(
    const float* __restrict__ part, int64_t nchunk, int64_t T, int N, int m, int k_rt, int Kr, int C,
    const float* __restrict__ saved, const float* __restrict__ colsum, const float* __restrict__ alpha,
    const float* __restrict__ b_res, const int32_t* __restrict__ idx, const float* __restrict__ p,
    const float* __restrict__ Hpre, const float* __restrict__ Hpost, const float* __restrict__ dHres,
    const float* __restrict__ dHpost, const float* __restrict__ dp, float eps, int iters, float delta,
    float* __restrict__ tok, float* __restrict__ pg, int softmax) {
  __shared__ float sk[KC > 0 ? kSkMaxSteps * KC * kPreTokThreads : 1];
  const int k = KC > 0 ? KC : k_rt;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  const int NA = k * Kr + k * k, ns = saved_floats(N, k, Kr);
  const float* sv = saved + t * ns;
  float* tk = tok + t * tok_floats(N, NA);
  float* g = pg + t * pg_floats(N, k, Kr);
  const float mu = sv[ns - 4], nu = sv[ns - 3], nu_a = sv[ns - 2];
  const float NC = (float)N * (float)C, kC = (float)k * (float)C;
  const float r = 1.0f / sqrtf(nu + eps), r_ln = 1.0f / sqrtf(ln_variance(mu, nu) + eps);
  const float r_a = 1.0f / sqrtf(nu_a + eps);
  const float a_pre = alpha[0], a_res = alpha[1], a_post = alpha[2];
  // pre-map: H = sigma(a z + b)
  float da_pre = 0.f, bp = 0.f;
  for (int i0 = 0; i0 < N; i0 += 16) {
    // 16 streams at a time: each chunk's 16 partials loaded together (streams
    // past N read stream i0 and are not used), summed in the order chunk 0, 1, ...
    float dh[16], hv[16], zv[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) dh[u] = 0.f;
    for (int64_t c = 0; c < nchunk; ++c) {
      float v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = part[(c * N + (i0 + u < N ? i0 + u : i0)) * T + t];
#pragma unroll
      for (int u = 0; u < 16; ++u) dh[u] += v[u];
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = i0 + u < N ? i0 + u : i0;
      hv[u] = Hpre[t * N + i];
      zv[u] = sv[N + i];
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = i0 + u;
      if (i >= N) break;
      const float ds = dh[u] * hv[u] * (1.0f - hv[u]);
      tk[N + i] = a_pre * ds;
      da_pre += ds * zv[u];
      g[3 + i] = ds;
      bp += a_pre * ds * zv[u];
    }
  }
  const float beta_pre = r * r * bp / NC;
  // router: only routed slots carry gradient, through p = sigma(z_r); with the
  // softmax router p = s_i of s = softmax(z_r) over the N streams, so every
  // logit gets dz_i = s_i (g_i - sum_l s_l g_l), g_i = dp of the slot of i
  for (int i = 0; i < N; ++i) tk[i] = 0.f;
  float m1 = 0.f, m2 = 0.f;
  if (!softmax) {
    for (int j = m; j < k; ++j) {
      const int i = idx[t * k + j];
      const float pj = p[t * k + j];
      const float dz = dp[t * k + j] * pj * (1.0f - pj);
      tk[i] = dz;
      m1 += colsum[i] * dz;
      m2 += sv[i] * dz;
    }
  } else if (k > m) {
    float mx = sv[0];
    for (int i = 1; i < N; ++i) mx = fmaxf(mx, sv[i]);
    float den = 0.f;
    for (int i = 0; i < N; ++i) den += __expf(sv[i] - mx);
    float dot = 0.f;
    for (int j = m; j < k; ++j) dot += p[t * k + j] * dp[t * k + j];
    for (int i = 0; i < N; ++i) tk[i] = -(__expf(sv[i] - mx) / den) * dot;
    for (int j = m; j < k; ++j) tk[idx[t * k + j]] += p[t * k + j] * dp[t * k + j];
    for (int i = 0; i < N; ++i) {
      m1 += colsum[i] * tk[i];
      m2 += sv[i] * tk[i];
    }
  }
  m1 /= NC;
  m2 /= NC;
  // post-map: H = 2 sigma(a z + b)
  float da_post = 0.f, ba = 0.f;
  for (int o = 0; o < k * Kr; ++o) {
    const float h = Hpost[t * k * Kr + o];
    const float du = dHpost[t * k * Kr + o] * h * (1.0f - 0.5f * h);
    const float z = sv[2 * N + o];
    tk[2 * N + o] = a_post * du;
    da_post += du * z;
    g[3 + N + k * k + o] = du;
    ba += a_post * du * z;
  }
  // residual map: H = clamp(SK(exp(a z + b)))
  constexpr int KS = KC > 0 ? KC : kMaxK;   // row stride of the matrices below
  float dL[KS * KS];
  if constexpr (KC > 0) {
    float L[KC * KC], dH[KC * KC];
#pragma unroll
    for (int j = 0; j < KC; ++j)
#pragma unroll
      for (int l = 0; l < KC; ++l) {
        L[j * KC + l] = a_res * sv[2 * N + KC * Kr + j * KC + l] + b_res[j * KC + l];
        dH[j * KC + l] = dHres[(t * KC + j) * KC + l];
      }
    sinkhorn_clamp_reverse_fast<KC>(L, iters, delta, dH, dL, &sk[threadIdx.x], kPreTokThreads);
  } else {
    float L[kMaxK * kMaxK], dH[kMaxK * kMaxK];
    for (int j = 0; j < kMaxK; ++j)
      for (int l = 0; l < kMaxK; ++l) {
        const bool in = j < k && l < k;
        L[j * kMaxK + l] = in ? a_res * sv[2 * N + k * Kr + j * k + l] + b_res[j * k + l] : 0.f;
        dH[j * kMaxK + l] = in ? dHres[(t * k + j) * k + l] : 0.f;
        dL[j * kMaxK + l] = 0.f;
      }
    sinkhorn_clamp_reverse(L, k, iters, delta, dH, dL);
  }
  float da_res = 0.f;
  for (int j = 0; j < k; ++j)
    for (int l = 0; l < k; ++l) {
      const float z = sv[2 * N + k * Kr + j * k + l];
      const float d = dL[j * KS + l];
      tk[2 * N + k * Kr + j * k + l] = a_res * d;
      da_res += d * z;
      g[3 + N + j * k + l] = d;
      ba += a_res * d * z;
    }
  g[0] = da_pre;
  g[1] = da_res;
  g[2] = da_post;
  float* sc = tk + 2 * N + NA;
  sc[0] = r;
  sc[1] = r_ln;
  sc[2] = mu;
  sc[3] = beta_pre;
  sc[4] = m1;
  sc[5] = m2;
  sc[6] = r_a;
  sc[7] = r_a * r_a * ba / kC;
}

// Weight-stationary pass over rows K = i*C + c of [W_r | W_pre] (one row per
// thread) and a chunk of tokens.  Per token:
//   dX[t,i,c] += H^pre_i d_in[c] + r (W_pre dz_pre) - beta_pre x
//               + r_ln ((W_r dz_r) - m1 - r_ln (x - mu) m2)
// and the row's weight gradients accumulate x r dz_pre and r_ln (x - mu) dz_r.
constexpr int kRowTok = 32;   // tokens staged in LDS per step
constexpr int kRowBatch = 8;  // tokens whose elements one thread loads together
static_assert(kRowTok % kRowBatch == 0, "whole batches per staged step");

__device__ __forceinline__ float ld_elem(const uint16_t* p, int64_t i) { return __uint_as_float((uint32_t)p[i] << 16); }
__device__ __forceinline__ float ld_elem(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ void st_elem(uint16_t* p, int64_t i, float v) { p[i] = (uint16_t)f2bf(v); }
__device__ __forceinline__ void st_elem(float* p, int64_t i, float v) { p[i] = v; }
template <typename TS, int NN>
__global__ __launch_bounds__(256) void k_bwd_full_rows(const TS* __restrict__ X, const TS* __restrict__ din,
                                                       TS* __restrict__ dX, const float* __restrict__ W_r,
                                                       const float* __restrict__ W_pre, const float* __restrict__ Hpre,
                                                       const float* __restrict__ tok, int64_t T, int C, int NA,
                                                       int64_t tchunk, float* __restrict__ dWr_part,
                                                       float* __restrict__ dWp_part) {
  __shared__ float sdz[kRowTok][2 * NN + 8];
  __shared__ float shp[kRowTok];
  const int64_t NC = (int64_t)NN * C;
  const int64_t K = (int64_t)blockIdx.x * 256 + threadIdx.x;   // row of the weights
  const bool valid = K < NC;
  const int i = valid ? (int)(K / C) : 0, c = valid ? (int)(K % C) : 0;
  const int istream = (int)(((int64_t)blockIdx.x * 256) / C);  // one stream per block (C % 256 == 0)
  float wr[NN], wp[NN], gr[NN], gp[NN];
#pragma unroll
  for (int o = 0; o < NN; ++o) {
    wr[o] = valid ? __uint_as_float(f2bf(W_r[K * NN + o]) << 16) : 0.f;
    wp[o] = valid ? __uint_as_float(f2bf(W_pre[K * NN + o]) << 16) : 0.f;
    gr[o] = 0.f;
    gp[o] = 0.f;
  }
  const int TF = tok_floats(NN, NA);
  const int64_t t0 = (int64_t)blockIdx.y * tchunk, t1 = (t0 + tchunk < T) ? t0 + tchunk : T;
  for (int64_t tb = t0; tb < t1; tb += kRowTok) {
    const int nt = (int)((t1 - tb < kRowTok) ? t1 - tb : kRowTok);
    __syncthreads();
    for (int q = threadIdx.x; q < nt * (2 * NN + 8); q += 256) {
      const int u = q / (2 * NN + 8), f = q % (2 * NN + 8);
      const float* tk = tok + (tb + u) * TF;
      sdz[u][f] = (f < 2 * NN) ? tk[f] : tk[2 * NN + NA + (f - 2 * NN)];
    }
    for (int u = threadIdx.x; u < nt; u += 256) shp[u] = Hpre[(tb + u) * NN + istream];
    __syncthreads();
    if (!valid) continue;
    // the elements of kRowBatch tokens are loaded before any is written back:
    // the accumulator rows are read and written in place, so a load after a
    // store of the same array would wait for it
    for (int u0 = 0; u0 < nt; u0 += kRowBatch) {
      float xb[kRowBatch], gb[kRowBatch], db[kRowBatch];
#pragma unroll
      for (int e = 0; e < kRowBatch; ++e) {
        xb[e] = gb[e] = db[e] = 0.f;
        if (u0 + e < nt) {
          const int64_t t = tb + u0 + e, off = t * NC + K;
          xb[e] = ld_elem(X, off);
          gb[e] = ld_elem(din, t * C + c);
          db[e] = ld_elem(dX, off);
        }
      }
#pragma unroll
      for (int e = 0; e < kRowBatch; ++e) {
        if (u0 + e >= nt) break;
        const int u = u0 + e;
        const float* z = sdz[u];
        const float r = z[2 * NN + 0], r_ln = z[2 * NN + 1], mu = z[2 * NN + 2], bpre = z[2 * NN + 3];
        const float m1 = z[2 * NN + 4], m2 = z[2 * NN + 5];
        const float x = xb[e];
        float sr = 0.f, sp = 0.f;
        const float xh = (x - mu) * r_ln, xr = x * r;
#pragma unroll
        for (int o = 0; o < NN; ++o) {
          sr = fmaf(wr[o], z[o], sr);
          sp = fmaf(wp[o], z[NN + o], sp);
          gr[o] = fmaf(xh, z[o], gr[o]);
          gp[o] = fmaf(xr, z[NN + o], gp[o]);
        }
        const float g = shp[u] * gb[e] + r * sp - bpre * x + r_ln * (sr - m1) - r_ln * (x - mu) * r_ln * m2;
        st_elem(dX, (tb + u) * NC + K, db[e] + g);
      }
    }
  }
  if (!valid) return;
  float* dr = dWr_part + ((int64_t)blockIdx.y * NC + K) * NN;
  float* dp = dWp_part + ((int64_t)blockIdx.y * NC + K) * NN;
#pragma unroll
  for (int o = 0; o < NN; ++o) { dr[o] = gr[o]; dp[o] = gp[o]; }
}

// Weight-stationary pass over rows K = j*C + c of [W_post | W_res] (slot j):
//   dX[t, I_j, c] += r_a (W_act dz_act) - beta_a a,   dW_act[K] += r_a a dz_act.
// The NA outputs are padded with zeros to NAMAX (zero weights and logit
// gradients), so every row runs the same branch-free contraction.
template <typename TS, int NAMAX>
__global__ __launch_bounds__(256) void k_bwd_act_rows(const TS* __restrict__ X, TS* __restrict__ dX,
                                                      const float* __restrict__ W_post,
                                                      const float* __restrict__ W_res,
                                                      const int32_t* __restrict__ idx,
                                                      const float* __restrict__ tok, int64_t T, int N, int k, int C,
                                                      int Kr, int64_t tchunk, float* __restrict__ dWa_part) {
  static_assert(NAMAX % 4 == 0, "float4 rows");
  constexpr int ZP = NAMAX + 4;   // per token: dz_act (zero past NA), r_a, beta_a, 2 pad
  const int NA = k * Kr + k * k, NP = k * Kr;
  __shared__ __align__(16) float sdz[kRowTok][ZP];
  __shared__ int64_t sbase[kRowTok];
  const int64_t kC = (int64_t)k * C;
  const int64_t K = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool valid = K < kC;
  const int j = (int)(((int64_t)blockIdx.x * 256) / C);   // one slot per block (C % 256 == 0)
  const int c = valid ? (int)(K % C) : 0;
  float w[NAMAX], ga[NAMAX];
#pragma unroll
  for (int o = 0; o < NAMAX; ++o) {
    float v = 0.f;
    if (valid && o < NA)
      v = (o < NP) ? W_post[K * NP + o] : W_res[K * (k * k) + (o - NP)];
    w[o] = __uint_as_float(f2bf(v) << 16);
    ga[o] = 0.f;
  }
  const int TF = 2 * N + NA + 8;
  const int64_t t0 = (int64_t)blockIdx.y * tchunk, t1 = (t0 + tchunk < T) ? t0 + tchunk : T;
  for (int64_t tb = t0; tb < t1; tb += kRowTok) {
    const int nt = (int)((t1 - tb < kRowTok) ? t1 - tb : kRowTok);
    __syncthreads();
    for (int q = threadIdx.x; q < kRowTok * ZP; q += 256) {
      const int u = q / ZP, f = q % ZP;
      float v = 0.f;
      if (u < nt) {
        const float* tk = tok + (tb + u) * TF;
        if (f < NA) v = tk[2 * N + f];
        else if (f == NAMAX) v = tk[2 * N + NA + 6];
        else if (f == NAMAX + 1) v = tk[2 * N + NA + 7];
      }
      sdz[u][f] = v;
    }
    if (threadIdx.x < kRowTok) {
      const int u = threadIdx.x < nt ? threadIdx.x : nt - 1;
      sbase[threadIdx.x] = ((tb + u) * N + idx[(tb + u) * k + j]) * (int64_t)C;
    }
    __syncthreads();
    if (!valid) continue;
    // the elements of kRowBatch tokens are loaded before any is written back
    // (a load after a store of the same array waits for it); tokens past nt
    // repeat the last one with zero gradients and are not stored
    for (int u0 = 0; u0 < nt; u0 += kRowBatch) {
      float ab[kRowBatch], db[kRowBatch];
#pragma unroll
      for (int e = 0; e < kRowBatch; ++e) {
        const int64_t off = sbase[u0 + e] + c;
        ab[e] = ld_elem(X, off);
        db[e] = ld_elem(dX, off);
      }
      // the logit gradients of the next token are read while this one is used;
      // the scheduling barrier keeps the compiler from reading all of them
      // ahead (register pressure)
      float zc[ZP], zn[ZP];
#pragma unroll
      for (int o = 0; o < ZP; o += 4) *reinterpret_cast<float4*>(&zc[o]) = *reinterpret_cast<const float4*>(&sdz[u0][o]);
#pragma unroll
      for (int e = 0; e < kRowBatch; ++e) {
        if (e + 1 < kRowBatch) {
#pragma unroll
          for (int o = 0; o < ZP; o += 4)
            *reinterpret_cast<float4*>(&zn[o]) = *reinterpret_cast<const float4*>(&sdz[u0 + e + 1][o]);
        }
        const float* z = zc;
        const float r_a = z[NAMAX], beta_a = z[NAMAX + 1];
        const float a = ab[e], ar = a * r_a;
        float sacc = 0.f;
#pragma unroll
        for (int o = 0; o < NAMAX; ++o) {
          sacc = fmaf(w[o], z[o], sacc);
          ga[o] = fmaf(ar, z[o], ga[o]);
        }
        if (u0 + e < nt) st_elem(dX, sbase[u0 + e] + c, db[e] + (r_a * sacc - beta_a * a));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int o = 0; o < ZP; ++o) zc[o] = zn[o];
      }
    }
  }
  if (!valid) return;
  float* dst = dWa_part + ((int64_t)blockIdx.y * kC + K) * NAMAX;
#pragma unroll
  for (int o = 0; o < NAMAX; ++o) dst[o] = ga[o];
}

// MFMA form of the two row passes above for a bf16 state: a workgroup takes
// consecutive weight rows K (wave w: rows 16w .. 16w + 15, inside one stream /
// slot) and a chunk of tokens, in steps of 32 tokens staged in LDS:
//   dX[t, K] += sum_o W[K, o] dz'[t, o] + (row terms)   MFMA D[16 K x 16 t], contraction over 32 outputs a block
//   dW[K, o] += sum_t x[t, K] dz'[t, o]                 MFMA D[16 o x 16 K], contraction over 32 tokens
// with dz' the per-token scaled logit gradients (full rows: r_ln dz_r | r
// dz_pre; active rows: r_a dz_act), entered as a bf16 pair hi + lo (2^-16
// relative).  The pairs are formed once per token by k_dz_pack, in the two
// layouts the MFMA operands read (token rows for dX, 32-token transposes for
// dW).  The full rows take the ring pass of xhc_bwd_rows.hip (whose dW_r
// misses the token sum of mu dz'_r, which the reduction removes); the active
// rows of a routed state, gathered through idx, take k_bwd_act_rows_mfma.
constexpr int kMfRows = 64;    // weight rows per workgroup
constexpr int kDzBlock = 32;   // tokens per transposed block of the packed dz' (= kMfStep)
constexpr int kMfStep = 32;    // tokens per step
constexpr int kMfXPitch = kMfRows + 8;   // bf16 per staged token row (pad: fewer LDS bank conflicts)

// dz' of the MFMA row passes as bf16 pairs hi + lo (hi the round-to-nearest-
// even bf16 of the value, lo that of the rest; the packed hardware
// conversion), NO outputs a token (zero past the used ones and past T):
//   rows[t][0 .. NO)   hi,  rows[t][NO .. 2 NO)  lo
//   tr[b][o][u]        the same values of token 32 b + u, row o of 2 NO
// full rows (act = 0): r_ln dz_r | r dz_pre; active rows: r_a dz_act.
// srec (or null): [Tp][8] per-token scalars of the ring pass.
__global__ __launch_bounds__(256) void k_dz_pack(const float* __restrict__ tok, int64_t T, int N, int NA, int act,
                                                 int NO, uint16_t* __restrict__ rows, uint16_t* __restrict__ tr,
                                                 float* __restrict__ srec) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t Tp = (T + kDzBlock - 1) / kDzBlock * kDzBlock;
  if (i >= Tp * NO) return;
  const int64_t t = i / NO;
  const int o = (int)(i % NO);
  float v = 0.f;
  if (t < T) {
    const float* tk = tok + t * tok_floats(N, NA);
    if (act) v = o < NA ? tk[2 * N + NA + 6] * tk[2 * N + o] : 0.f;
    else if (o < N) v = tk[2 * N + NA + 1] * tk[o];
    else if (o < 2 * N) v = tk[2 * N + NA + 0] * tk[o];
  }
  const uint32_t hb = pack2bf(v, 0.f) & 0xFFFFu;
  const uint32_t lb = pack2bf(v - __uint_as_float(hb << 16), 0.f) & 0xFFFFu;
  rows[t * 2 * NO + o] = (uint16_t)hb;
  rows[t * 2 * NO + NO + o] = (uint16_t)lb;
  uint16_t* blk = tr + (t / kDzBlock) * 2 * NO * kDzBlock;
  blk[o * kDzBlock + t % kDzBlock] = (uint16_t)hb;
  blk[(NO + o) * kDzBlock + t % kDzBlock] = (uint16_t)lb;
  // the token's scalars as the ring pass reads them: r_ln, mu, m1, m2, beta,
  // then zero (full rows: beta_pre; active rows: beta_a, the others zero)
  if (srec && o < 8) {
    const int src[5] = {1, 2, 4, 5, 3};
    float sv = 0.f;
    if (t < T && o < 5 && (!act || o == 4)) sv = tok[t * tok_floats(N, NA) + 2 * N + NA + (act ? 7 : src[o])];
    srec[t * 8 + o] = sv;
  }
}

// 4 consecutive bf16 gradient elements from floats
__device__ __forceinline__ void st4(uint16_t* p, const float (&d)[4]) {
  *reinterpret_cast<uint2*>(p) = make_uint2(pack2bf(d[0], d[1]), pack2bf(d[2], d[3]));
}

// Active rows of a routed bf16 state (k * Kr + k * k <= 32 outputs, bf16
// gradient rows updated in place at the routed rows): 128 weight rows (128
// channels of one slot) per workgroup of 512 threads.  The inputs of step
// tb + 64 are fetched into registers while step tb is computed: this thread's
// pieces of the packed dz', one per-token scalar and 16 bytes of the state
// rows, and its gradient elements.  Every load is issued without a branch (a
// token past the chunk reads the chunk's last token; its dz' row and state row
// are zeroed where they are staged, its gradient row is not stored) and the
// barriers wait for LDS traffic only, so a step waits for nothing but its own
// prefetched loads.  The routed row of each token is loaded one step earlier
// still (rid), so the state and gradient loads do not wait on it.  A gradient
// row is read two steps before its token's step writes it, and no step in
// between writes that token.
constexpr int kActRows = 2 * kMfRows;   // weight rows per workgroup
__global__ __launch_bounds__(4 * kActRows) __attribute__((amdgpu_waves_per_eu(4))) void k_bwd_act_rows_mfma(const uint16_t* __restrict__ X,
                                                                uint16_t* __restrict__ dX,
                                                                const float* __restrict__ W_post,
                                                                const float* __restrict__ W_res,
                                                                const int32_t* __restrict__ idx,
                                                                const float* __restrict__ tok, int64_t T, int N, int k,
                                                                int C, int Kr, int NA, int64_t tchunk,
                                                                const uint16_t* __restrict__ dzp,
                                                                float* __restrict__ wpa) {
  constexpr int RW = kActRows, NT = RW * 4, PIECES = RW / 8;   // threads; 16-byte pieces of a staged token row
  constexpr int NO = 32, NOH = 2;                              // outputs (padded); 16-output tiles of dW
  constexpr int DZP = 512 / NT;                                // 16-byte pieces of packed dz' per thread and step
  static_assert(kMfStep == kDzBlock && DZP * NT == 16 * NO, "a step copies its packed dz' in whole pieces");
  __shared__ __align__(16) uint16_t xs[kMfStep][RW + 8];
  // packed dz' of the step: token rows (hi | lo) and the transpose; the row
  // pitches (2 NO + 8 and 40 elements) keep the 16-byte operand reads of a
  // 16-lane group on distinct banks
  __shared__ __align__(16) uint16_t dzr[kMfStep][2 * NO + 8];
  __shared__ __align__(16) uint16_t dzt[2 * NO][kMfStep + 8];
  __shared__ float beta_s[kMfStep];
  const int lane = threadIdx.x % kWave;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));   // uniform: its branches are scalar
  const int l16 = lane % 16, g4 = lane / 16;
  const int64_t K0 = (int64_t)blockIdx.x * RW;   // first weight row of the workgroup
  const int part = (int)(K0 / C);                 // slot
  const int c0 = (int)(K0 % C);
  const int64_t NK = (int64_t)k * C;              // weight rows
  const int NP = k * Kr;                          // W_post columns
  const int TF = tok_floats(N, NA);
  // A operand of the dX product: rows K0 + 16 wave + l16, outputs 8 g4 .. + 7, as bf16
  uint4 wfrag;
  {
    float f[8];
    const int64_t K = K0 + 16 * wave + l16;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int o = 8 * g4 + e;
      float v = 0.f;
      if (o < NP) v = W_post[K * NP + o];
      else if (o < NA) v = W_res[K * (k * k) + (o - NP)];
      f[e] = __uint_as_float(f2bf(v) << 16);
    }
    wfrag = pack8(f);
  }
  f32x4 dw[NOH];
#pragma unroll
  for (int oh = 0; oh < NOH; ++oh) dw[oh] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int64_t t0 = (int64_t)blockIdx.y * tchunk, t1 = (t0 + tchunk < T) ? t0 + tchunk : T;
  const uint16_t* const dzrows = dzp;
  const uint16_t* const dztr = dzp + (T + kDzBlock - 1) / kDzBlock * kDzBlock * 2 * NO;
  struct Stage {
    uint4 dz[DZP];
    float beta;     // beta_a of token threadIdx.x (threads < 32)
    int rowd[2];    // routed rows of the lane's two gradient tokens
    uint4 x;
    uint2 dx[2];    // the lane's gradient elements (two token halves), as loaded
  };
  auto tok_at = [&](int64_t tb, int u) -> int64_t { return tb + u < t1 ? tb + u : t1 - 1; };
  int rid[3];   // routed rows of the next fetch: state token, gradient tokens 0 and 1
  auto fetch_rows = [&](int64_t tb) {
    rid[0] = idx[tok_at(tb, threadIdx.x / PIECES) * k + part];
    rid[1] = idx[tok_at(tb, l16) * k + part];
    rid[2] = idx[tok_at(tb, 16 + l16) * k + part];
  };
  // pieces q of the packed dz': [0, 8 NO) token rows (NO / 4 pieces a token),
  // [8 NO, 16 NO) the transposed block (4 pieces a row); 8 NO is a multiple
  // of 64, so the choice is the same across a wave
  auto dz_rows = [&](int r) { return wave * kWave + r * NT < 8 * NO; };
  auto fetch = [&](Stage& st, int64_t tb) {
#pragma unroll
    for (int r = 0; r < DZP; ++r) {
      const int q = threadIdx.x + r * NT;
      if (dz_rows(r)) {
        st.dz[r] = *reinterpret_cast<const uint4*>(dzrows + tok_at(tb, q / (NO / 4)) * 2 * NO + (q % (NO / 4)) * 8);
      } else {
        const int qq = q - 8 * NO;
        st.dz[r] = *reinterpret_cast<const uint4*>(dztr + (tok_at(tb, 0) / kDzBlock) * 2 * NO * kDzBlock +
                                                   (qq / 4) * kDzBlock + (qq % 4) * 8);
      }
    }
    st.x = *reinterpret_cast<const uint4*>(X + (tok_at(tb, threadIdx.x / PIECES) * N + rid[0]) * (int64_t)C + c0 +
                                           (threadIdx.x % PIECES) * 8);
    // the gradient rows of the step (other tokens than the steps being
    // computed before it, so reading them two steps ahead is safe)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t t = tok_at(tb, 16 * h + l16);
      st.rowd[h] = rid[1 + h];
      st.dx[h] = *reinterpret_cast<const uint2*>(dX + (t * N + rid[1 + h]) * (int64_t)C + c0 + 16 * wave + 4 * g4);
    }
    // beta_a of token threadIdx.x % 32, loaded by every thread (the same
    // loads on every wave)
    st.beta = tok[tok_at(tb, threadIdx.x % kMfStep) * TF + 2 * N + NA + 7];
  };
  // One step of 32 tokens.  FULL: all 32 tokens exist, so the step has no
  // per-token predicates; the last, partial step of the chunk (T % 32 tokens)
  // is a separate instance.  The next step's loads are issued unconditionally
  // (past the chunk they read its last token again), so every path through
  // the loop has the same memory operations.
  auto step = [&](auto full, Stage& cur, int64_t tb) {
    constexpr bool FULL = decltype(full)::value;
    const int nt = FULL ? kMfStep : (int)(t1 - tb);
    lds_barrier();   // the previous step's LDS reads are done
#pragma unroll
    for (int r = 0; r < DZP; ++r) {
      const int q = threadIdx.x + r * NT;
      if (dz_rows(r)) {
        const int u = q / (NO / 4), off = (q % (NO / 4)) * 8;
        *reinterpret_cast<uint4*>(&dzr[u][off]) = (FULL || u < nt) ? cur.dz[r] : make_uint4(0, 0, 0, 0);
      } else {
        const int qq = q - 8 * NO, row = qq / 4, off = (qq % 4) * 8;
        *reinterpret_cast<uint4*>(&dzt[row][off]) = cur.dz[r];
      }
    }
    if (threadIdx.x < kMfStep) beta_s[threadIdx.x] = cur.beta;
    *reinterpret_cast<uint4*>(&xs[threadIdx.x / PIECES][(threadIdx.x % PIECES) * 8]) =
        (FULL || (int)(threadIdx.x / PIECES) < nt) ? cur.x : make_uint4(0, 0, 0, 0);
    const int rowd[2] = {cur.rowd[0], cur.rowd[1]};
    const uint2 dxr[2] = {cur.dx[0], cur.dx[1]};
    lds_barrier();
    fetch(cur, tb + 2 * kMfStep);
    fetch_rows(tb + 3 * kMfStep);
    // ---- dX: two token halves; the gradient rows were read a step ahead
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int u = 16 * h + l16;   // B operand token of this lane
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      acc = mfma_16x16x32(wfrag, *reinterpret_cast<const uint4*>(&dzr[u][8 * g4]), acc);
      acc = mfma_16x16x32(wfrag, *reinterpret_cast<const uint4*>(&dzr[u][NO + 8 * g4]), acc);
      // lane holds rows 16 wave + 4 g4 + v of token u
      if (FULL || u < nt) {
        const int kr = 16 * wave + 4 * g4;
        const uint2 xv = *reinterpret_cast<const uint2*>(&xs[u][kr]);
        const float x[4] = {bf_lo(xv.x), bf_hi(xv.x), bf_lo(xv.y), bf_hi(xv.y)};
        const float beta_a = beta_s[u];
        const float dxv[4] = {bf_lo(dxr[h].x), bf_hi(dxr[h].x), bf_lo(dxr[h].y), bf_hi(dxr[h].y)};
        float d[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) d[v] = dxv[v] + (acc[v] - beta_a * x[v]);
        st4(dX + ((tb + u) * N + rowd[h]) * (int64_t)C + c0 + kr, d);
      }
    }
    // ---- dW: contraction over the 32 staged tokens (rows past nt are zero)
    {
      uint16_t xb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) xb[e] = xs[8 * g4 + e][16 * wave + l16];
      const uint4 bx = make_uint4(xb[0] | ((uint32_t)xb[1] << 16), xb[2] | ((uint32_t)xb[3] << 16),
                                  xb[4] | ((uint32_t)xb[5] << 16), xb[6] | ((uint32_t)xb[7] << 16));
#pragma unroll
      for (int oh = 0; oh < NOH; ++oh) {
        const uint4 ah = *reinterpret_cast<const uint4*>(&dzt[16 * oh + l16][8 * g4]);
        const uint4 al = *reinterpret_cast<const uint4*>(&dzt[NO + 16 * oh + l16][8 * g4]);
        dw[oh] = mfma_16x16x32(ah, bx, dw[oh]);
        dw[oh] = mfma_16x16x32(al, bx, dw[oh]);
      }
    }
  };
  if (t0 < t1) {
    // two stages alternate, so the inputs of a step are fetched two steps
    // before it is computed (a step's own arithmetic is short)
    Stage sa, sb;
    fetch_rows(t0);
    fetch(sa, t0);
    fetch_rows(t0 + kMfStep);
    fetch(sb, t0 + kMfStep);
    fetch_rows(t0 + 2 * kMfStep);
    // the loop is entered with no load in flight, so the compiler's wait
    // counts inside it follow the loop's own order of loads and stores
    __builtin_amdgcn_s_waitcnt(0);
    int64_t tb = t0;
    for (; tb + 2 * kMfStep <= t1; tb += 2 * kMfStep) {
      step(std::true_type{}, sa, tb);
      step(std::true_type{}, sb, tb + kMfStep);
    }
    if (tb + kMfStep <= t1) {
      step(std::true_type{}, sa, tb);
      tb += kMfStep;
      if (tb < t1) step(std::false_type{}, sb, tb);
    } else if (tb < t1) {
      step(std::false_type{}, sa, tb);
    }
  }
  // lane holds dW[row K0 + 16 wave + l16][output 16 oh + 4 g4 + v]
  float* dst = wpa + ((int64_t)blockIdx.y * NK + K0 + 16 * wave + l16) * 32;
#pragma unroll
  for (int oh = 0; oh < NOH; ++oh)
    *reinterpret_cast<float4*>(dst + 16 * oh + 4 * g4) = make_float4(dw[oh][0], dw[oh][1], dw[oh][2], dw[oh][3]);
}

// corr[o] = sum_t mu_t r_ln,t dz_r[t, o] (the part of dW_r the MFMA full-row
// pass leaves out), one workgroup per output, fixed order
__global__ __launch_bounds__(256) void k_mu_dz_sum(const float* __restrict__ tok, int64_t T, int N, int NA,
                                                   float* __restrict__ corr) {
  __shared__ float red[256];
  const int o = blockIdx.x, TF = tok_floats(N, NA);
  float s = 0.f;
  for (int64_t t = threadIdx.x; t < T; t += 256) {
    const float* tk = tok + t * TF;
    s += tk[2 * N + NA + 2] * tk[2 * N + NA + 1] * tk[o];
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) corr[o] = red[0];
}

// out[col] = sum over rows of in[row][col] - corr[col % ncorr] (corr may be null)
__global__ __launch_bounds__(256) void k_colsum_rows_corr(const float* __restrict__ in, int64_t nrows, int64_t ncols,
                                                          const float* __restrict__ corr, int ncorr,
                                                          float* __restrict__ out) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= ncols) return;
  float s = 0.f;
  for (int64_t r0 = 0; r0 < nrows; r0 += 8) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = (r0 + u < nrows) ? in[(r0 + u) * ncols + col] : 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  out[col] = corr ? s - corr[col % ncorr] : s;
}

// ------------------------------------------------------------ launchers

// the one-pass conv reverse applies to the paper's branches
static bool conv_run_ok(const xhc_dims* d) {
  return d->Kr == 4 && d->kappa[0] == 4 && d->kappa[1] == 8 && d->kappa[2] == 12;
}
// the fused element pass + conv reverse (k_bwd_post_run)
static bool post_run_ok(const xhc_dims* d) {
  return conv_run_ok(d) && d->k <= 4 && d->C % 256 == 0 &&
         (int64_t)kConvRun * d->N * d->C < ((int64_t)1 << 31);   // 32-bit row offsets within a run
}

#define XHC_TS_DISPATCH(dt, ...) \
  if ((dt) == XHC_BF16) { using TS = uint16_t; __VA_ARGS__; } else { using TS = float; __VA_ARGS__; }

hipError_t launch_bwd_post(const xhc_dims* d, const void* dXn, void* X, const void* Xact, const void* F,
                           const float* conv_w, const int32_t* idx, const float* p, const float* Hres,
                           const float* Hpost, void* dX, void* dF, float* dHres, float* dHpost, float* dp,
                           float* dconv_w, char* ws, hipStream_t s, bool grad_f32) {
  const int64_t T = d->T, S = d->S;
  const int N = d->N, C = d->C, k = d->k, Kr = d->Kr;
  const int64_t ncb = post_chunks(C);
  const dim3 grid((unsigned)(T * ncb));
  // workspace: dots partials | coef | de (Kr planes, fp32; or, fused, the run
  // boundary parts rb and lb) | conv partials
  const int km = k <= 4 ? 4 : 8;
  const int nd = km * km + km * Kr + Kr * (Kr + 1) / 2;
  const bool fused = post_run_ok(d);
  const int64_t nruns = (T + kConvRun - 1) / kConvRun;
  float* part = reinterpret_cast<float*>(ws);
  // dots partials: [post_chunks(C)][nd][T], or, fused, [C / 256][T][nd]
  float* coef = part + (fused ? (int64_t)(C / 256) : ncb) * nd * T;
  float* de = coef + T * (Kr * kMaxK + Kr * Kr);
  float* rb = de;
  float* lb = rb + nruns * 11 * (int64_t)C;
  float* dsum = lb + nruns * 11 * (int64_t)C;   // fused: the dots partials summed over the C / 256 slices
  float* cpart = de + (fused ? 2 * nruns * 11 * (int64_t)C + (int64_t)nd * T : (Kr > 1 ? (int64_t)Kr * T * C : 0));
  const int* kap = d->kappa;
#define XHC_BWD_POST_TG(KRV, KMV)                                                                                \
    if (fused) {                                                                                                 \
      const int nthr = C % 1024 == 0 ? 256 : 64;                                                                 \
      k_bwd_post_dots_run<TS, TG><<<dim3((unsigned)((T + kDotRun - 1) / kDotRun), (unsigned)(C / (4 * nthr))),  \
                                    dim3(nthr), 0, s>>>(reinterpret_cast<const TG*>(dXn),                        \
          reinterpret_cast<const TS*>(Xact), reinterpret_cast<const TS*>(F), T, S, N, C, k, conv_w, idx, part);   \
      k_colsum_rows<<<dim3((unsigned)((T * nd + 255) / 256)), dim3(256), 0, s>>>(part, C / 256, T * nd, dsum);     \
      k_bwd_post_token<KRV, KMV><<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(dsum, 1, T * nd, 1, nd,    \
          T, k, d->gram_schmidt, p, Hpost, dHres, dHpost, dp, coef);                                              \
    } else if constexpr (KRV == 1) {                                                                             \
      /* one pass over the rows: the dot products and the element pass */                                      \
      if (dX != dXn && N > k) {                                                                                  \
        /* the untouched rows keep their gradient; the pass writes the active ones */                           \
        const hipError_t ec = hipMemcpyAsync(dX, dXn, (size_t)T * N * C * sizeof(TG), hipMemcpyDeviceToDevice, s); \
        if (ec != hipSuccess) return ec;                                                                         \
      }                                                                                                          \
      k_bwd_post_dots<TS, TG, KRV, KMV, true><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const TG*>(dXn),      \
          reinterpret_cast<const TS*>(Xact), reinterpret_cast<const TS*>(F), T, S, N, C, k, kap[0], kap[1],       \
          kap[2], conv_w, idx, part, Hres, p, Hpost, reinterpret_cast<TS*>(X), reinterpret_cast<TG*>(dX),        \
          reinterpret_cast<TS*>(dF));                                                                            \
      k_bwd_post_token<KRV, KMV><<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(part, ncb, nd * T, T,      \
          1, T, k, d->gram_schmidt, p, Hpost, dHres, dHpost, dp, coef);                                           \
    } else {                                                                                                     \
      k_bwd_post_dots<TS, TG, KRV, KMV><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const TG*>(dXn),            \
          reinterpret_cast<const TS*>(Xact), reinterpret_cast<const TS*>(F), T, S, N, C, k, kap[0], kap[1],       \
          kap[2], conv_w, idx, part);                                                                            \
      k_bwd_post_token<KRV, KMV><<<dim3((unsigned)((T + 127) / 128)), dim3(128), 0, s>>>(part, ncb, nd * T, T,      \
          1, T, k, d->gram_schmidt, p, Hpost, dHres, dHpost, dp, coef);                                           \
    }                                                                                                            \
    if (fused) {                                                                                                 \
      if (dX != dXn && N > k) {                                                                                  \
        /* the untouched rows keep their gradient; the fused pass writes the active ones */                     \
        const hipError_t ec = hipMemcpyAsync(dX, dXn, (size_t)T * N * C * sizeof(TG), hipMemcpyDeviceToDevice, s); \
        if (ec != hipSuccess) return ec;                                                                         \
      }                                                                                                          \
      if (X)                                                                                                     \
        k_bwd_post_run<TS, TG, true><<<dim3((unsigned)((C + 255) / 256), (unsigned)nruns), dim3(256), 0, s>>>(   \
            reinterpret_cast<const TG*>(dXn), reinterpret_cast<TS*>(X), reinterpret_cast<const TS*>(Xact),        \
            reinterpret_cast<const TS*>(F), T, S, N, C, k, conv_w, idx, Hres, coef, reinterpret_cast<TG*>(dX),   \
            reinterpret_cast<TS*>(dF), cpart, rb, lb);                                                            \
      else                                                                                                       \
        k_bwd_post_run<TS, TG, false><<<dim3((unsigned)((C + 255) / 256), (unsigned)nruns), dim3(256), 0, s>>>(  \
            reinterpret_cast<const TG*>(dXn), nullptr, reinterpret_cast<const TS*>(Xact),                         \
            reinterpret_cast<const TS*>(F), T, S, N, C, k, conv_w, idx, Hres, coef, reinterpret_cast<TG*>(dX),   \
            reinterpret_cast<TS*>(dF), cpart, rb, lb);                                                            \
      if (nruns > 1)                                                                                             \
        k_bwd_post_fix<TS><<<dim3((unsigned)((C + 255) / 256), (unsigned)(nruns - 1), 11u), dim3(256), 0, s>>>(   \
            rb, lb, T, S, C, reinterpret_cast<TS*>(dF));                                                         \
    } else if constexpr (KRV != 1)                                                                              \
    k_bwd_post_elem<TS, TG, KRV, KMV><<<grid, dim3(256), 0, s>>>(reinterpret_cast<const TG*>(dXn),              \
        reinterpret_cast<TS*>(X), reinterpret_cast<const TS*>(Xact), reinterpret_cast<const TS*>(F), T, S, N, C, \
        k, kap[0], kap[1], kap[2], conv_w, idx, Hres, coef, reinterpret_cast<TG*>(dX), reinterpret_cast<TS*>(dF), \
        de)
#define XHC_BWD_POST(KRV, KMV)                                                                                   \
  XHC_TS_DISPATCH(d->state_dtype,                                                                                \
    if (grad_f32) { using TG = float; XHC_BWD_POST_TG(KRV, KMV); } else { using TG = TS; XHC_BWD_POST_TG(KRV, KMV); })
#define XHC_BWD_POST_K(KRV) if (k <= 4) { XHC_BWD_POST(KRV, 4); } else { XHC_BWD_POST(KRV, 8); }
  switch (Kr) {
    case 1: XHC_BWD_POST_K(1); break;
    case 2: XHC_BWD_POST_K(2); break;
    case 3: XHC_BWD_POST_K(3); break;
    default: XHC_BWD_POST_K(4); break;
  }
#undef XHC_BWD_POST_K
#undef XHC_BWD_POST
#undef XHC_BWD_POST_TG
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || Kr == 1) return e;
  if (fused) {
    const int64_t ncols = (int64_t)kConvRows * C;
    k_colsum_rows<<<dim3((unsigned)((ncols + 255) / 256)), dim3(256), 0, s>>>(cpart, nruns, ncols, dconv_w);
    return hipGetLastError();
  }
  if (conv_run_ok(d)) {
    // dF and the tap gradients in one pass over de (the paper's branches)
    const int64_t nruns = (T + kConvRun - 1) / kConvRun;
    XHC_TS_DISPATCH(d->state_dtype,
      k_bwd_conv_run<TS><<<dim3((unsigned)((C + 255) / 256), (unsigned)nruns), dim3(256), 0, s>>>(
          de, reinterpret_cast<const TS*>(F), T, S, C, conv_w, reinterpret_cast<TS*>(dF), cpart));
    const int64_t ncols = (int64_t)kConvRows * C;
    k_colsum_rows<<<dim3((unsigned)((ncols + 255) / 256)), dim3(256), 0, s>>>(cpart, nruns, ncols, dconv_w);
    return hipGetLastError();
  }
  XHC_TS_DISPATCH(d->state_dtype,
    k_bwd_conv<TS><<<grid, dim3(256), 0, s>>>(de, T, S, C, Kr, kap[0], kap[1], kap[2], conv_w,
                                              reinterpret_cast<TS*>(dF)));
  int nrows = 0;
  for (int j = 0; j < Kr - 1; ++j) nrows += kap[j];
  const int64_t nchunks = (T + kConvChunk - 1) / kConvChunk;
  XHC_TS_DISPATCH(d->state_dtype,
    k_bwd_convw<TS><<<dim3((unsigned)((C / 8 + 255) / 256), (unsigned)nrows, (unsigned)nchunks), dim3(256), 0, s>>>(
        de, reinterpret_cast<const TS*>(F), T, S, C, Kr, kap[0], kap[1], kap[2], cpart));
  const int64_t ncols = (int64_t)nrows * C;
  k_colsum_rows<<<dim3((unsigned)((ncols + 255) / 256)), dim3(256), 0, s>>>(cpart, nchunks, ncols, dconv_w);
  return hipGetLastError();
}

size_t bwd_post_ws_bytes(const xhc_dims* d) {
  const int64_t T = d->T;
  const int C = d->C, k = d->k, Kr = d->Kr;
  const int km = k <= 4 ? 4 : 8;
  const int nd = km * km + km * Kr + Kr * (Kr + 1) / 2;
  const size_t nchunks = post_run_ok(d) ? (size_t)(C / 256) : (size_t)post_chunks(C);
  size_t n = nchunks * nd * T + (size_t)T * (Kr * kMaxK + Kr * Kr);
  if (Kr > 1) {
    int nrows = 0;
    for (int j = 0; j < Kr - 1; ++j) nrows += d->kappa[j];
    const size_t chunked = (size_t)((T + kConvChunk - 1) / kConvChunk) * nrows * C;
    const size_t nruns = (size_t)((T + kConvRun - 1) / kConvRun);
    const size_t runs = conv_run_ok(d) ? nruns * kConvRows * C : 0;
    // fused: only the run boundary parts instead of de
    n += (post_run_ok(d) ? 2 * nruns * 11 * (size_t)C + (size_t)nd * T : (size_t)Kr * T * C) +
         (chunked > runs ? chunked : runs);
  }
  return n * sizeof(float) + 256;
}


// The full-row pass of NQ pre-map reverses over one state in a single pass
// (the entry state of an xHC-Flash group: the router with the first pre-map,
// then one pre-map per sublayer; bf16 state, N = 16), run by the ring pass
// of xhc_bwd_rows.hip; the contraction of the dX product runs over the 16
// router and 16 NQ pre-map outputs, each pass's per-token record (tok) giving its
// own dz'.  The per-token terms add up over the passes: the dense reads
// sum_q H^pre,q_i d input_q, the pre-map norm terms sum_q beta_pre,q x, and
// the router's LayerNorm terms of the first pass (later passes have no router
// gradient, so theirs are zero).  The weight partials of output block ob go
// to wout[ob] ([chunk][N C][16]: the router, then pre-map q).
constexpr int kMultiMaxQ = 4;
struct MultiRows {
  const float* tok[kMultiMaxQ];   // per pass: the token records
  const float* hrd[kMultiMaxQ];   // per pass: weights of the dense read [T, N]
  const uint16_t* din[kMultiMaxQ];
  const float* w[kMultiMaxQ + 1];  // W_r, then W_pre of pass q ([N C][16] each)
  float* wout[kMultiMaxQ + 1];
};
// Per token, the inputs of the multi-map ring pass gathered from the passes' token
// records: [r_ln dz_r (16) | r dz_pre,q (16 each) | r_ln, mu, m1, m2,
// sum_q beta_pre,q, pad], pitch 16 (NQ + 1) + 8 floats.
template <int NQ>
__global__ __launch_bounds__(256) void k_multi_prep(MultiRows m, int64_t T, int N, int NA, float* __restrict__ out) {
  constexpr int NO = 16 * (NQ + 1), PITCH = NO + 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= T * PITCH) return;
  const int64_t t = i / PITCH;
  const int o = (int)(i % PITCH);
  const int TF = tok_floats(N, NA);
  float v = 0.f;
  if (o < NO) {
    const float* tk = m.tok[o < 16 ? 0 : o / 16 - 1] + t * TF;
    v = o < 16 ? tk[2 * N + NA + 1] * tk[o] : tk[2 * N + NA + 0] * tk[N + o % 16];   // r_ln dz_r | r dz_pre,q
  } else if (o < NO + 4) {
    const int map[4] = {1, 2, 4, 5};   // r_ln, mu, m1, m2 of the first pass
    v = m.tok[0][t * TF + 2 * N + NA + map[o - NO]];
  } else if (o == NO + 4) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) v += m.tok[q][t * TF + 2 * N + NA + 3];   // beta_pre, passes in order
  }
  out[i] = v;
}

// The dz' of k_multi_prep as bf16 pairs hi + lo in the layouts of
// k_dz_pack (token rows [t][2 NOP], 32-token transposes [b][2 NOP][32]),
// NOP = the NO outputs padded to whole 32-blocks (zero past NO and past T).
template <int NQ>
__global__ __launch_bounds__(256) void k_dz_pack_multi(const float* __restrict__ prep, int64_t T,
                                                       uint16_t* __restrict__ rows, uint16_t* __restrict__ tr) {
  constexpr int NO = 16 * (NQ + 1), NOP = (NO + 31) / 32 * 32, PITCH = NO + 8;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t Tp = (T + kDzBlock - 1) / kDzBlock * kDzBlock;
  if (i >= Tp * NOP) return;
  const int64_t t = i / NOP;
  const int o = (int)(i % NOP);
  const float v = (t < T && o < NO) ? prep[t * PITCH + o] : 0.f;
  const uint32_t hb = pack2bf(v, 0.f) & 0xFFFFu;
  const uint32_t lb = pack2bf(v - __uint_as_float(hb << 16), 0.f) & 0xFFFFu;
  rows[t * 2 * NOP + o] = (uint16_t)hb;
  rows[t * 2 * NOP + NOP + o] = (uint16_t)lb;
  uint16_t* blk = tr + (t / kDzBlock) * 2 * NOP * kDzBlock;
  blk[o * kDzBlock + t % kDzBlock] = (uint16_t)hb;
  blk[(NOP + o) * kDzBlock + t % kDzBlock] = (uint16_t)lb;
}

constexpr int64_t kRowChunk = 1024;   // tokens per weight-gradient partial

BwdPreWs bwd_pre_ws(const xhc_dims* d, char* ws) {
  const int64_t T = d->T;
  const int N = d->N, k = d->k, Kr = d->Kr, C = d->C;
  const int NA = k * Kr + k * k;
  const int64_t ncb = post_chunks(C);
  const int64_t nchunk = (T + kRowChunk - 1) / kRowChunk;
  BwdPreWs w;
  w.part = reinterpret_cast<float*>(ws);
  w.tok = w.part + ncb * N * T;
  w.pg = w.tok + T * tok_floats(N, NA);
  w.wpart_r = w.pg + T * pg_floats(N, k, Kr);
  w.wpart_p = w.wpart_r + nchunk * (int64_t)N * C * N;
  w.wpart_a = w.wpart_p + nchunk * (int64_t)N * C * N;
  w.red_a = w.wpart_a + nchunk * (int64_t)k * C * 32;           // [kC][32]
  w.pgsum = w.red_a + (int64_t)k * C * 32;
  // packed dz' (16-byte aligned): full rows 2 NO_f, active rows 2 x 32 bf16 a
  // token, in token rows and in transposed 32-token blocks
  const int64_t Tp = (T + kDzBlock - 1) / kDzBlock * kDzBlock;
  const uintptr_t a = reinterpret_cast<uintptr_t>(w.pgsum + pg_floats(N, k, Kr) + N);
  w.dzf = reinterpret_cast<uint16_t*>((a + 15) / 16 * 16);
  w.dza = w.dzf + Tp * 2 * (2 * N <= 32 ? 32 : 64) * 2;
  w.srec = reinterpret_cast<float*>(w.dza + Tp * 2 * 32 * 2);   // 16-byte aligned: Tp % 32 == 0
  w.sreca = w.srec + Tp * 8;
  return w;
}

bool bwd_rows_multi_supported(const xhc_dims* d, int Q) {
  return d->state_dtype == XHC_BF16 && d->N == 16 && bwd_rows_ring_supported((int64_t)d->N * d->C, d->C, kRowChunk) &&
         (Q == 2 || Q == 4);
}

hipError_t launch_bwd_dhpre_multi(const xhc_dims* d, int Q, const void* X, const void* d_input, char* const* ws,
                                  hipStream_t s) {
  if (!bwd_rows_multi_supported(d, Q)) return hipErrorInvalidValue;
  MultiParts mp{};
  for (int q = 0; q < Q; ++q) mp.part[q] = bwd_pre_ws(d, ws[q]).part;
  const dim3 g((unsigned)(d->T * post_chunks(d->C)));
  const uint16_t* x = reinterpret_cast<const uint16_t*>(X);
  const uint16_t* din = reinterpret_cast<const uint16_t*>(d_input);
  if (Q == 4) k_bwd_dhpre_multi<uint16_t, 4><<<g, dim3(256), 0, s>>>(x, din, d->T, d->N, d->C, mp);
  else k_bwd_dhpre_multi<uint16_t, 2><<<g, dim3(256), 0, s>>>(x, din, d->T, d->N, d->C, mp);
  return hipGetLastError();
}

// prep [T][16 (Q + 1) + 8] floats, then (16-byte aligned) the packed dz'
static size_t multi_prep_floats(int64_t T, int Q) { return (size_t)T * (16 * (Q + 1) + 8); }
static int64_t multi_nop(int Q) { return (16 * (Q + 1) + 31) / 32 * 32; }
size_t bwd_rows_multi_ws_bytes(const xhc_dims* d, int Q) {
  const size_t Tp = (size_t)((d->T + kDzBlock - 1) / kDzBlock * kDzBlock);
  return multi_prep_floats(d->T, Q) * sizeof(float) + 16 + Tp * 2 * multi_nop(Q) * 2 * sizeof(uint16_t);
}

hipError_t launch_bwd_rows_multi(const xhc_dims* d, int Q, const void* X, void* dX, const float* W_r,
                                 const float* W_pre, const void* d_input, const float* const* hrd, char* const* ws,
                                 float* prep, hipStream_t s) {
  if (!bwd_rows_multi_supported(d, Q)) return hipErrorInvalidValue;
  const int64_t T = d->T;
  const int N = d->N, C = d->C, NA = d->k * d->Kr + d->k * d->k;
  const int64_t NC = (int64_t)N * C;
  MultiRows m{};
  m.w[0] = W_r;
  m.wout[0] = bwd_pre_ws(d, ws[0]).wpart_r;
  for (int q = 0; q < Q; ++q) {
    const BwdPreWs w = bwd_pre_ws(d, ws[q]);
    m.tok[q] = w.tok;
    m.hrd[q] = hrd[q];
    m.din[q] = reinterpret_cast<const uint16_t*>(d_input) + (int64_t)q * T * C;
    m.w[q + 1] = W_pre + (int64_t)q * NC * N;
    m.wout[q + 1] = w.wpart_p;
  }
  const int64_t np = T * (16 * (Q + 1) + 8);
  const dim3 gp((unsigned)((np + 255) / 256));
  const int64_t Tp = (T + kDzBlock - 1) / kDzBlock * kDzBlock, nop = multi_nop(Q);
  const uintptr_t a = reinterpret_cast<uintptr_t>(prep + multi_prep_floats(T, Q));
  uint16_t* dzp = reinterpret_cast<uint16_t*>((a + 15) / 16 * 16);
  const dim3 gk((unsigned)((Tp * nop + 255) / 256));
  if (Q == 4) {
    k_multi_prep<4><<<gp, dim3(256), 0, s>>>(m, T, N, NA, prep);
    k_dz_pack_multi<4><<<gk, dim3(256), 0, s>>>(prep, T, dzp, dzp + Tp * 2 * nop);
  } else {
    k_multi_prep<2><<<gp, dim3(256), 0, s>>>(m, T, N, NA, prep);
    k_dz_pack_multi<2><<<gk, dim3(256), 0, s>>>(prep, T, dzp, dzp + Tp * 2 * nop);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // the ring pass reads the prep rows' scalars (r_ln, mu, m1, m2, sum beta_pre)
  // at offset 16 (Q + 1) of each row
  const int no = 16 * (Q + 1);
  RowRingDesc rd{};
  rd.X = X;
  rd.dX = dX;
  rd.nq = Q;
  for (int q = 0; q < Q; ++q) {
    rd.din[q] = m.din[q];
    rd.hp[q] = m.hrd[q];
  }
  rd.hp_stride = N;
  for (int b = 0; b <= Q; ++b) {
    rd.w[b] = m.w[b];
    rd.win[b] = 16;
    rd.wout[b] = m.wout[b];
  }
  rd.nwin = Q + 1;
  rd.wout_w = 16;
  rd.nout = no;
  rd.dzp = dzp;
  rd.nop = (int)nop;
  rd.srec = prep + no;
  rd.srec_stride = no + 8;
  rd.T = T;
  rd.tchunk = kRowChunk;
  rd.N = N;
  rd.C = C;
  return launch_bwd_rows_ring(rd, (int64_t)N * C, s);
}

size_t bwd_pre_ws_bytes(const xhc_dims* d) {
  const int64_t T = d->T;
  const int N = d->N, k = d->k, Kr = d->Kr, C = d->C;
  const int NA = k * Kr + k * k;
  const int64_t nchunk = (T + kRowChunk - 1) / kRowChunk;
  size_t n = (size_t)post_chunks(C) * N * T;                    // dH^pre partials
  n += (size_t)T * tok_floats(N, NA) + (size_t)T * pg_floats(N, k, Kr);
  n += (size_t)nchunk * N * C * N * 2;                           // dW_r, dW_pre partials
  n += (size_t)nchunk * k * C * 32;                              // dW_act partials (<= 32 columns)
  n += (size_t)k * C * 32 + (size_t)pg_floats(N, k, Kr);          // reduced dW_act, reduced gradients
  n += (size_t)N;                                                // token sum of mu dz'_r
  const size_t Tp = (size_t)((T + kDzBlock - 1) / kDzBlock * kDzBlock);
  const size_t dz = Tp * 2 * ((2 * N <= 32 ? 32 : 64) + 32) * 2 * sizeof(uint16_t);   // packed dz'
  return n * sizeof(float) + 16 + dz + 2 * Tp * 8 * sizeof(float) + 1024;             // + scalar rows
}

bool bwd_pre_supported(const xhc_dims* d) {
  return (d->N == 4 || d->N == 8 || d->N == 16 || d->N == 32) && d->C % 256 == 0 &&
         d->k * d->Kr + d->k * d->k <= 32;
}

hipError_t launch_bwd_pre(const xhc_dims* d, const void* X, const float* colsum, const float* W_r,
                          const float* W_pre, const float* W_res, const float* W_post, const float* alpha,
                          const float* b_res, const float* saved, const int32_t* idx, const float* p,
                          const float* Hpre, const float* Hpost, const void* d_input, const float* dHres,
                          const float* dHpost, const float* dp, void* dX, float* dW_r, float* dW_pre, float* dW_res,
                          float* dW_post, float* dalpha, float* db_pre, float* db_res, float* db_post, char* ws,
                          hipStream_t s, const float* dhpre_act, const float* Hpre_read, bool dense_rows,
                          const void* X_bf16, bool act_rows, int phase, const void* act_din) {
  const float* Hrd = Hpre_read ? Hpre_read : Hpre;   // weights of the dense-read term
  const int64_t T = d->T;
  const int N = d->N, k = d->k, Kr = d->Kr, C = d->C;
  const int NA = k * Kr + k * k;
  const int64_t ncb = post_chunks(C);
  const int64_t nchunk = (T + kRowChunk - 1) / kRowChunk;
  const BwdPreWs w = bwd_pre_ws(d, ws);
  float* const part = w.part;
  float* const tok = w.tok;
  float* const pg = w.pg;
  float* const wpart_r = w.wpart_r;
  float* const wpart_p = w.wpart_p;
  float* const wpart_a = w.wpart_a;
  float* const red_a = w.red_a;
  float* const pgsum = w.pgsum;
  const bool mf = d->state_dtype == XHC_BF16 && (N == 4 || N == 8 || N == 16 || N == 32) && NA <= 32 &&
                  C % (2 * kMfRows) == 0;
  hipError_t e = hipSuccess;
  if (phase == kBwdPreReduce) {
    // the row passes ran elsewhere (their partials are in this workspace)
    if (mf) k_mu_dz_sum<<<dim3((unsigned)N), dim3(256), 0, s>>>(tok, T, N, NA, pgsum + pg_floats(N, k, Kr));
  } else {
    if (phase == kBwdPreTokensGiven) {
      // the dH^pre partials are already in the workspace
    } else if (!dense_rows) {
      hipError_t e0 = launch_fill0(part, (size_t)ncb * N * T * sizeof(float), s);
      if (e0 != hipSuccess) return e0;
    } else {
      XHC_TS_DISPATCH(d->state_dtype,
        k_bwd_dhpre<TS><<<dim3((unsigned)(T * ncb)), dim3(256), 0, s>>>(reinterpret_cast<const TS*>(X),
            reinterpret_cast<const TS*>(d_input), T, N, C, part));
    }
    if (dhpre_act) {
      k_bwd_dhpre_override<<<dim3((unsigned)((T * k + 255) / 256)), dim3(256), 0, s>>>(dhpre_act, idx, T, N, k, ncb,
                                                                                      part);
    }
    {
      const dim3 gt((unsigned)((T + kPreTokThreads - 1) / kPreTokThreads)), bt(kPreTokThreads);
      if (k == 4 && 2 * d->sinkhorn_iters <= kSkMaxSteps)
        k_bwd_pre_token<4><<<gt, bt, 0, s>>>(part, ncb, T, N, d->m, k, Kr, C, saved, colsum, alpha, b_res, idx, p,
                                            Hpre, Hpost, dHres, dHpost, dp, d->eps, d->sinkhorn_iters,
                                            d->clamp_delta, tok, pg,
                                            d->router == XHC_ROUTER_SOFTMAX ? 1 : 0);
      else
        k_bwd_pre_token<0><<<gt, bt, 0, s>>>(part, ncb, T, N, d->m, k, Kr, C, saved, colsum, alpha, b_res, idx, p,
                                            Hpre, Hpost, dHres, dHpost, dp, d->eps, d->sinkhorn_iters,
                                            d->clamp_delta, tok, pg,
                                            d->router == XHC_ROUTER_SOFTMAX ? 1 : 0);
    }
    e = hipGetLastError();
    if (e != hipSuccess || phase == kBwdPreTokens || phase == kBwdPreTokensGiven) return e;
    if (mf) {
      // 128 rows per workgroup (256 contiguous bytes of each state row per
      // token); C % 256 == 0 is part of the backward's supported shapes
      const int64_t Tp = (T + kDzBlock - 1) / kDzBlock * kDzBlock;
      const int NOf = 2 * N <= 32 ? 32 : 64;
      if (dense_rows)
        k_dz_pack<<<dim3((unsigned)((Tp * NOf + 255) / 256)), dim3(256), 0, s>>>(tok, T, N, NA, 0, NOf, w.dzf,
                                                                                 w.dzf + Tp * 2 * NOf, w.srec);
      if (act_rows)
        k_dz_pack<<<dim3((unsigned)((Tp * 32 + 255) / 256)), dim3(256), 0, s>>>(tok, T, N, NA, 1, 32, w.dza,
                                                                                w.dza + Tp * 2 * 32, nullptr);
      if (dense_rows) {
        // 2N outputs padded to one block of 32 (N <= 16) or two (N = 32)
        RowRingDesc rd{};
        rd.X = X;
        rd.dX = dX;
        rd.nq = 1;
        rd.din[0] = d_input;
        rd.hp[0] = Hrd;
        rd.hp_stride = N;
        rd.w[0] = W_r;
        rd.w[1] = W_pre;
        rd.win[0] = rd.win[1] = N;
        rd.nwin = 2;
        rd.wout[0] = wpart_r;
        rd.wout[1] = wpart_p;
        rd.wout_w = N;
        rd.nout = 2 * N;
        rd.dzp = w.dzf;
        rd.nop = NOf;
        rd.srec = w.srec;
        rd.srec_stride = 8;
        rd.T = T;
        rd.tchunk = kRowChunk;
        rd.N = N;
        rd.C = C;
        e = launch_bwd_rows_ring(rd, (int64_t)N * C, s);
        if (e != hipSuccess) return e;
      }
      // 128 rows per workgroup (C % 256 == 0); the dense read of the active
      // rows is in the full-row pass
      const dim3 ga((unsigned)((int64_t)k * C / kActRows), (unsigned)nchunk);
      if (act_rows)
        k_bwd_act_rows_mfma<<<ga, dim3(4 * kActRows), 0, s>>>(reinterpret_cast<const uint16_t*>(X),
            reinterpret_cast<uint16_t*>(dX), W_post, W_res, idx, tok, T, N, k, C, Kr, NA, kRowChunk, w.dza, wpart_a);
      k_mu_dz_sum<<<dim3((unsigned)N), dim3(256), 0, s>>>(tok, T, N, NA, pgsum + pg_floats(N, k, Kr));
    }
    // an fp32 state given with its exact bf16 copy (the k-row view of an
    // xHC-Flash sublayer, N = k, whose slot j is row j): the active rows take
    // the ring pass with fp32 gradient rows
    const bool mfa32 = !mf && X_bf16 && d->state_dtype == XHC_F32 && NA <= 32 && C % (2 * kMfRows) == 0;
    if (mfa32 && act_rows) {
      if (N != k) return hipErrorInvalidValue;
      const int64_t Tp = (T + kDzBlock - 1) / kDzBlock * kDzBlock;
      k_dz_pack<<<dim3((unsigned)((Tp * 32 + 255) / 256)), dim3(256), 0, s>>>(tok, T, N, NA, 1, 32, w.dza,
                                                                              w.dza + Tp * 2 * 32, w.sreca);
      RowRingDesc rd{};
      rd.X = X_bf16;
      rd.dX = dX;
      rd.dx_f32 = true;
      rd.nq = act_din ? 1 : 0;
      rd.din[0] = act_din;
      rd.hp[0] = Hpre;   // [T, k]: the weight of each slot's read of d input
      rd.hp_stride = k;
      rd.w[0] = W_post;
      rd.w[1] = W_res;
      rd.win[0] = k * Kr;
      rd.win[1] = k * k;
      rd.nwin = 2;
      rd.wout[0] = wpart_a;
      rd.wout_w = 32;
      rd.nout = NA;
      rd.dzp = w.dza;
      rd.nop = 32;
      rd.srec = w.sreca;
      rd.srec_stride = 8;
      rd.T = T;
      rd.tchunk = kRowChunk;
      rd.N = N;
      rd.C = C;
      e = launch_bwd_rows_ring(rd, (int64_t)k * C, s);
      if (e != hipSuccess) return e;
    }
    const dim3 gfull((unsigned)(((int64_t)N * C + 255) / 256), (unsigned)nchunk);
#define XHC_FULL_ROWS(NNV)                                                                                       \
    XHC_TS_DISPATCH(d->state_dtype,                                                                                \
      k_bwd_full_rows<TS, NNV><<<gfull, dim3(256), 0, s>>>(reinterpret_cast<const TS*>(X),                        \
          reinterpret_cast<const TS*>(d_input), reinterpret_cast<TS*>(dX), W_r, W_pre, Hrd, tok, T, C, NA,         \
          kRowChunk, wpart_r, wpart_p))
    if (!mf) {
      if (dense_rows) {
        switch (N) {
          case 4: XHC_FULL_ROWS(4); break;
          case 8: XHC_FULL_ROWS(8); break;
          case 16: XHC_FULL_ROWS(16); break;
          default: XHC_FULL_ROWS(32); break;
        }
      }
      if (!mfa32 && act_rows) {
        const dim3 gact((unsigned)(((int64_t)k * C + 255) / 256), (unsigned)nchunk);
        XHC_TS_DISPATCH(d->state_dtype,
          k_bwd_act_rows<TS, 32><<<gact, dim3(256), 0, s>>>(reinterpret_cast<const TS*>(X), reinterpret_cast<TS*>(dX),
              W_post, W_res, idx, tok, T, N, k, C, Kr, kRowChunk, wpart_a));
      }
    }
#undef XHC_FULL_ROWS
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // token reductions (fixed order)
  const int64_t nfull = (int64_t)N * C * N;
  if (dense_rows) {
    k_colsum_rows_corr<<<dim3((unsigned)((nfull + 255) / 256)), dim3(256), 0, s>>>(
        wpart_r, nchunk, nfull, mf ? pgsum + pg_floats(N, k, Kr) : nullptr, N, dW_r);
    k_colsum_rows<<<dim3((unsigned)((nfull + 255) / 256)), dim3(256), 0, s>>>(wpart_p, nchunk, nfull, dW_pre);
  }
  // active partials are [chunk][kC][32]: split columns into W_post and W_res
  if (act_rows) {
    const int64_t nact = (int64_t)k * C * 32;
    k_colsum_rows<<<dim3((unsigned)((nact + 255) / 256)), dim3(256), 0, s>>>(wpart_a, nchunk, nact, red_a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = hipMemcpy2DAsync(dW_post, (size_t)k * Kr * sizeof(float), red_a, 32 * sizeof(float),
                         (size_t)k * Kr * sizeof(float), (size_t)k * C, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
    e = hipMemcpy2DAsync(dW_res, (size_t)k * k * sizeof(float), red_a + k * Kr, 32 * sizeof(float),
                         (size_t)k * k * sizeof(float), (size_t)k * C, hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
  }
  const int npg = pg_floats(N, k, Kr);
  k_sum_tokens<<<dim3((unsigned)npg), dim3(256), 0, s>>>(pg, T, npg, pgsum);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = hipMemcpyAsync(dalpha, pgsum, 3 * sizeof(float), hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess) e = hipMemcpyAsync(db_pre, pgsum + 3, N * sizeof(float), hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(db_res, pgsum + 3 + N, (size_t)k * k * sizeof(float), hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(db_post, pgsum + 3 + N + k * k, (size_t)k * Kr * sizeof(float), hipMemcpyDeviceToDevice, s);
  return e;
}

#undef XHC_TS_DISPATCH

}  // namespace xhc

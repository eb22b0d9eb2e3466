// Dense read (eq:dense_read, and the xHC-Flash non-active bases) fused with
// the projection of the routed rows onto the active-state weights.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {
// ----------------------------------------------------------------- dense read + active projection
// One pass over the state after routing: for a 16-token tile and a chunk of
// 32-channel slices, each lane (token tl = lane % 16, 8 channels at grp * 8)
// forms the dense read(s) of eq:dense_read from all N rows, and feeds the k
// routed rows of the same slice to the split-K MFMA projection onto the
// active-state weights (K index j * C + c, as packed by xhc_pack_active),
// with the active moments.  Partials as k_proj_partial, one per chunk.

// EXACT: N == NB and k == KK, so the row and slot loops carry no guards.  NOB
// is an upper bound of the nob output blocks.
template <typename TS, int NOB, int NMAP, int NB, int KK, bool EXACT>
__global__ __launch_bounds__(256) void k_read_active(const TS* __restrict__ X, int64_t T, int N, int C,
                                                     const float* __restrict__ Hpre,
                                                     const int32_t* __restrict__ idx, int k,
                                                     const uint4* __restrict__ wpk, int nob, TS* __restrict__ out0,
                                                     TS* __restrict__ outr, float* __restrict__ part) {
  using R8 = Raw8<TS>;
  constexpr int NO = NOB * 16 + 2;   // LDS rows: outputs, then the two moments
  const int NOr = nob * 16 + 2;      // rows of the partials
  constexpr int RB = (NMAP > 1 || Vec8<TS>::kSplit) ? 8 : 16;   // rows loaded before use
  __shared__ float red[4][NO][kProjTile];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int64_t tile = blockIdx.x, chunk = blockIdx.y;
  const int64_t t = tile * kProjTile + tl;
  const bool valid = t < T;
  if (EXACT) {
    N = NB;
    k = KK;
  }
  const int64_t tc = valid ? t : T - 1;   // loads stay in bounds; results of t >= T are dropped
  int32_t rows[KK];
  uint64_t act = 0;
#pragma unroll
  for (int j = 0; j < KK; ++j) {
    rows[j] = j < k ? idx[tc * k + j] : 0;
    if (j < k) act |= 1ull << rows[j];
  }
  float h[NMAP][NB];
#pragma unroll
  for (int q = 0; q < NMAP; ++q)
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      float w = i < N ? Hpre[((int64_t)q * T + tc) * N + i] : 0.f;
      if (q > 0 && ((act >> i) & 1ull)) w = 0.f;
      h[q][i] = w;
    }
  f32x4 acc[NOB];
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  float s1 = 0.f, s2 = 0.f;
  const int64_t nsl = C / 32;
  const int64_t kbr = C / 32;   // k-blocks per gathered row
  for (int r = 0; r < kReadSlices / 4; ++r) {
    const int64_t sl = chunk * kReadSlices + r * 4 + wave;
    if (sl >= nsl) break;
    const int c = (int)(sl * 32) + grp * 8;
    const TS* xt = X + tc * (int64_t)N * C + c;
    // routed rows and their weight fragments first, so their loads overlap the dense read's
    uint4 xb[KK], xl[KK], wa[KK][NOB];
#pragma unroll
    for (int j = 0; j < KK; ++j) {
      if (j < k) {
        float f[8];
        xb[j] = Vec8<TS>::operand(xt + (int64_t)rows[j] * C, f, xl[j]);
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
          if (ob < nob) wa[j][ob] = wpk[((j * kbr + sl) * nob + ob) * kWave + lane];
      }
    }
    float o[NMAP][8];
#pragma unroll
    for (int q = 0; q < NMAP; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) o[q][e] = 0.f;
#pragma unroll
    for (int i0 = 0; i0 < NB; i0 += RB) {
      if (i0 >= N) break;
      typename R8::raw rr[RB];
#pragma unroll
      for (int u = 0; u < RB; ++u)
        if (i0 + u < N) rr[u] = R8::load(xt + (int64_t)(i0 + u) * C);
#pragma unroll
      for (int u = 0; u < RB; ++u) {
        if (i0 + u < N) {
          float f[8];
          R8::unpack(rr[u], f);
#pragma unroll
          for (int q = 0; q < NMAP; ++q)
#pragma unroll
            for (int e = 0; e < 8; ++e) o[q][e] = fmaf(h[q][i0 + u], f[e], o[q][e]);
        }
      }
    }
    if (valid) {
      Vec8<TS>::store(out0 + t * C + c, o[0]);
#pragma unroll
      for (int q = 1; q < NMAP; ++q) Vec8<TS>::store(outr + ((int64_t)(q - 1) * T + t) * C + c, o[q]);
    }
#pragma unroll
    for (int j = 0; j < KK; ++j) {
      if (j < k) {
        float f[8], g[8];
        unpack8(xb[j], f);
        unpack8(xl[j], g);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = f[e] + g[e];
          s1 += x;
          s2 += x * x;
        }
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) {
          if (ob < nob) {
            acc[ob] = mfma_16x16x32(wa[j][ob], xb[j], acc[ob]);
            if (Vec8<TS>::kSplit) acc[ob] = mfma_16x16x32(wa[j][ob], xl[j], acc[ob]);
          }
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
  for (int i = threadIdx.x; i < NOr * kProjTile; i += 256) {
    const int o = i / kProjTile, tt = i % kProjTile;
    const int r = o < nob * 16 ? o : o - nob * 16 + NOB * 16;
    const int64_t tg = tile * kProjTile + tt;
    if (tg < T) part[(chunk * NOr + o) * T + tg] = red[0][r][tt] + red[1][r][tt] + red[2][r][tt] + red[3][r][tt];
  }
}

template <typename TS, int NOB, int NB, int KK, bool EXACT>
static hipError_t read_active_launch(const TS* X, int64_t T, int N, int C, const float* Hpre, int nmap,
                                     const int32_t* idx, int k, const uint4* w, int nob, TS* out0, TS* outr,
                                     float* part, hipStream_t s) {
  const dim3 grid((unsigned)((T + kProjTile - 1) / kProjTile), (unsigned)read_chunks(C));
#define XHC_RA(NM)                                                                                        \
  k_read_active<TS, NOB, NM, NB, KK, EXACT><<<grid, dim3(256), 0, s>>>(X, T, N, C, Hpre, idx, k, w, nob, \
                                                                       out0, outr, part)
  switch (nmap) {
    case 1: XHC_RA(1); break;
    case 2: XHC_RA(2); break;
    case 4: XHC_RA(4); break;
    default: return hipErrorInvalidValue;
  }
#undef XHC_RA
  return hipGetLastError();
}

// bf16 state with N = 16, k = 4: exact instances; otherwise row bound 16 or 64,
// slot bound kMaxK and output-block bound 2 or 6.
template <typename TS>
static hipError_t read_active_dispatch(const TS* X, int64_t T, int N, int C, const float* Hpre, int nmap,
                                       const int32_t* idx, int k, const void* packed, int nob, TS* out0, TS* outr,
                                       float* part, hipStream_t s) {
  const uint4* w = reinterpret_cast<const uint4*>(packed);
  if (nob > 6) return hipErrorInvalidValue;
  if (!Vec8<TS>::kSplit && N == 16 && k == 4 && nob <= 2) {
    if (nob == 1) return read_active_launch<TS, 1, 16, 4, true>(X, T, N, C, Hpre, nmap, idx, k, w, nob, out0, outr, part, s);
    return read_active_launch<TS, 2, 16, 4, true>(X, T, N, C, Hpre, nmap, idx, k, w, nob, out0, outr, part, s);
  }
  if (N <= 16) {
    if (nob <= 2) return read_active_launch<TS, 2, 16, kMaxK, false>(X, T, N, C, Hpre, nmap, idx, k, w, nob, out0, outr, part, s);
    return read_active_launch<TS, 6, 16, kMaxK, false>(X, T, N, C, Hpre, nmap, idx, k, w, nob, out0, outr, part, s);
  }
  if (nob <= 2) return read_active_launch<TS, 2, 64, kMaxK, false>(X, T, N, C, Hpre, nmap, idx, k, w, nob, out0, outr, part, s);
  return read_active_launch<TS, 6, 64, kMaxK, false>(X, T, N, C, Hpre, nmap, idx, k, w, nob, out0, outr, part, s);
}

hipError_t launch_read_active(int state_dtype, const void* X, int64_t T, int N, int C, const float* Hpre, int nmap,
                              const int32_t* idx, int k, const void* packed_act, int64_t nout_act, void* out0,
                              void* outr, float* part, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const int nob = (int)out_blocks(nout_act);
  if (state_dtype == XHC_BF16)
    return read_active_dispatch<uint16_t>(reinterpret_cast<const uint16_t*>(X), T, N, C, Hpre, nmap, idx, k,
                                          packed_act, nob, reinterpret_cast<uint16_t*>(out0),
                                          reinterpret_cast<uint16_t*>(outr), part, s);
  return read_active_dispatch<float>(reinterpret_cast<const float*>(X), T, N, C, Hpre, nmap, idx, k, packed_act,
                                     nob, reinterpret_cast<float*>(out0), reinterpret_cast<float*>(outr), part, s);
}

}  // namespace xhc

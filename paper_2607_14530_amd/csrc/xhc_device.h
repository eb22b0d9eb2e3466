// Device-side building blocks shared by the xHC kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "xhc.h"
#include "xhc_launch.h"

namespace xhc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- bf16 <-> f32

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
// Two fp32 -> packed bf16 (a in the low half), round to nearest even, by the
// gfx950 packed conversion (one instruction; the same bits as f2bf except the
// payload of a NaN).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2bf(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

__device__ __forceinline__ void unpack8(const uint4 v, float (&f)[8]) {
  f[0] = bf_lo(v.x); f[1] = bf_hi(v.x); f[2] = bf_lo(v.y); f[3] = bf_hi(v.y);
  f[4] = bf_lo(v.z); f[5] = bf_hi(v.z); f[6] = bf_lo(v.w); f[7] = bf_hi(v.w);
}
__device__ __forceinline__ uint4 pack8(const float (&f)[8]) {
  return make_uint4(pack2bf(f[0], f[1]), pack2bf(f[2], f[3]), pack2bf(f[4], f[5]), pack2bf(f[6], f[7]));
}

// Eight consecutive state elements <-> fp32, for bf16 (uint16_t) and fp32 states.
// kSplit: the state needs a second (lo) bf16 operand to enter the projection exactly.
template <typename TS> struct Vec8;
template <> struct Vec8<uint16_t> {
  static constexpr bool kSplit = false;
  static __device__ __forceinline__ void load(const uint16_t* p, float (&f)[8]) {
    unpack8(*reinterpret_cast<const uint4*>(p), f);
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float (&f)[8]) {
    *reinterpret_cast<uint4*>(p) = pack8(f);
  }
  // values as the state stores them (bf16, nearest even)
  static __device__ __forceinline__ void round(float (&f)[8]) {
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = __uint_as_float(f2bf(f[e]) << 16);
  }
  // bf16 operand bits of the same eight elements (exact for a bf16 state)
  static __device__ __forceinline__ uint4 operand(const uint16_t* p, float (&f)[8], uint4& lo) {
    uint4 v = *reinterpret_cast<const uint4*>(p);
    unpack8(v, f);
    lo = make_uint4(0, 0, 0, 0);
    return v;
  }
};
template <> struct Vec8<float> {
  static constexpr bool kSplit = true;
  static __device__ __forceinline__ void load(const float* p, float (&f)[8]) {
    float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  static __device__ __forceinline__ void store(float* p, const float (&f)[8]) {
    reinterpret_cast<float4*>(p)[0] = make_float4(f[0], f[1], f[2], f[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
  static __device__ __forceinline__ void round(float (&)[8]) {}
  // an fp32 state enters the projection as a bf16 pair hi + lo (hi = bf16(x),
  // lo = bf16(x - hi)), which represents x to about 2^-16 relative
  static __device__ __forceinline__ uint4 operand(const float* p, float (&f)[8], uint4& lo) {
    load(p, f);
    float h[8], l[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      h[e] = __uint_as_float(f2bf(f[e]) << 16);
      l[e] = f[e] - h[e];
    }
    lo = pack8(l);
    return pack8(h);
  }
};

// Eight consecutive state elements kept in their storage format until used.
template <typename TS> struct Raw8;
template <> struct Raw8<uint16_t> {
  using raw = uint4;
  static __device__ __forceinline__ raw load(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  static __device__ __forceinline__ void store(uint16_t* p, const raw& v) { *reinterpret_cast<uint4*>(p) = v; }
  static __device__ __forceinline__ void unpack(const raw& v, float (&f)[8]) { unpack8(v, f); }
};
template <> struct Raw8<float> {
  struct raw { float4 a, b; };
  static __device__ __forceinline__ raw load(const float* p) {
    return raw{reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
  }
  static __device__ __forceinline__ void store(float* p, const raw& v) {
    reinterpret_cast<float4*>(p)[0] = v.a;
    reinterpret_cast<float4*>(p)[1] = v.b;
  }
  static __device__ __forceinline__ void unpack(const raw& v, float (&f)[8]) {
    f[0] = v.a.x; f[1] = v.a.y; f[2] = v.a.z; f[3] = v.a.w; f[4] = v.b.x; f[5] = v.b.y; f[6] = v.b.z; f[7] = v.b.w;
  }
};

// ---------------------------------------------------------------- MFMA
// v_mfma_f32_16x16x32_bf16: D[16x16] += A[16x32] * B[32x16].
// Lane l holds A[l%16][8*(l/16) .. +8], B[8*(l/16) .. +8][l%16] and
// D[4*(l/16) + v][l%16], v = 0..3.
__device__ __forceinline__ f32x4 mfma_16x16x32(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------- wave reduction

// Sum of v over the 64 lanes of the wave, returned in every lane: pairs and
// quads by DPP quad permutes, half rows and rows by DPP mirrors (the values
// are uniform within the smaller group by then, so a mirror adds the other
// half), then row pairs and wave halves by the gfx950 permlane swaps.  Fixed
// order, so the result is deterministic.
__device__ __forceinline__ float dpp_add(float v, int ctrl_sel) {
  int o = 0;
  switch (ctrl_sel) {
    case 0: o = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false); break;   // quad_perm 1,0,3,2
    case 1: o = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false); break;   // quad_perm 2,3,0,1
    case 2: o = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false); break;  // row_half_mirror
    default: o = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false); break; // row_mirror
  }
  return v + __int_as_float(o);
}
__device__ __forceinline__ float wave_sum(float v) {
  v = dpp_add(v, 0);
  v = dpp_add(v, 1);
  v = dpp_add(v, 2);
  v = dpp_add(v, 3);
  const auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
  const auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

// ---------------------------------------------------------------- math

// Workgroup barrier for LDS traffic only: this wave's LDS accesses are
// complete (lgkmcnt(0)), then s_barrier; the compiler fences keep memory
// accesses on their side.  Unlike __syncthreads() it does not wait for the
// wave's outstanding global loads and stores (a release fence would), so
// loads issued ahead of their use stay in flight across it.  Only for
// kernels whose waves exchange data through LDS alone.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);   // vmcnt = 63, expcnt = 7 (no wait), lgkmcnt = 0
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// 16 (4) bytes per lane from global memory straight into LDS at lds_addr +
// 16 lane (4 lane): a wave's 1 KiB (256 B) lands contiguously; lds_addr is
// the same in every lane.  Issued as inline assembly so that the compiler
// does not track the copy (it would otherwise make every later LDS access of
// the wave wait for it: it cannot tell which LDS a copy writes); the caller
// waits for it explicitly (s_waitcnt vmcnt) before the data is read, and
// before the wave ends.
__device__ __forceinline__ void lds_dma16(const void* src, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(src), "s"(lds_addr) : "memory", "m0");
}
__device__ __forceinline__ void lds_dma4(const void* src, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" : : "v"(src), "s"(lds_addr) : "memory", "m0");
}

__device__ __forceinline__ float sigmoidf(float z) { return 1.0f / (1.0f + __expf(-z)); }

// Biased variance nu - mu^2 of the LayerNorm (eq:router), with a negative
// rounding residue taken as 0.  A NaN (an infinite or NaN state gives
// Inf - Inf) stays NaN, so the logits become NaN as the plain definition
// makes them (fmaxf would turn it into 0).
__device__ __forceinline__ float ln_variance(float mu, float nu) {
  const float v = nu - mu * mu;
  return v < 0.f ? 0.f : v;
}

// Order of router logits used by TopK, as a signed integer key: key order is
// the order of the floats (-0 and +0 tie), with NaN below every number (so a
// NaN never displaces a number; NaNs tie with each other).  Together with
// "ties to the lower index" this is a total order on (logit, stream), so every
// routed slot gets exactly one distinct stream whatever the logits hold.
// Host-callable so that the order can be checked on the CPU.
__host__ __device__ __forceinline__ int32_t logit_key(float z) {
  if (z != z) return INT32_MIN;
  uint32_t u;
  __builtin_memcpy(&u, &z, 4);
  if ((u & 0x7fffffffu) == 0) u = 0;   // -0 ties with +0
  return (u & 0x80000000u) ? (int32_t)(u ^ 0x7fffffffu) : (int32_t)u;
}

// Rank of stream `lane` among the routing candidates m..15 of one token: the
// number of candidates i whose (key, index) comes before (key, lane), key =
// logit_key.  The other 15 streams are visited in rotation order: keyrot(r),
// r = 1 .. 15, is the key of stream (lane - r) mod 16 (in the single-pass
// kernel a rotation of the 16-lane row, so no lane index is ever compared
// with a loop constant and nothing is hoisted into per-lane masks).  The ranks
// of the 16 - m candidates are 0 .. 15 - m, each once; slot m + rank takes the
// stream when rank < k - m.
template <class KeyRot>
__host__ __device__ __forceinline__ int route_rank16(KeyRot keyrot, int32_t key, int lane, int m) {
  int rank = 0;
#pragma unroll
  for (int r = 1; r < 16; ++r) {
    const int i = (lane - r) & 15;
    const int32_t ki = keyrot(r);
    const int before = (int)(ki > key) | ((int)(ki == key) & (int)(i < lane));
    rank += before & -(int)(i >= m);
  }
  return rank;
}

// Fixed-plus-TopK selection of one token (eq:router_topk): slots 0..m-1 take
// streams 0..m-1; slot j >= m takes the first remaining stream among m..N-1
// in the order of logit_key, ties to the lower index.  Writes the k stream
// indices and returns their logits in zsel (slots >= m).
template <int NMAX>
__host__ __device__ __forceinline__ void route_select(const float (&z)[NMAX], int N, int m, int k, int32_t* idx_out,
                                                      float* zsel) {
  uint64_t used = 0;
  for (int j = 0; j < m; ++j) idx_out[j] = j;
  for (int j = m; j < k; ++j) {
    int best = -1;
    int32_t bk = 0;
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
      if (i >= m && i < N && !((used >> i) & 1ull)) {
        const int32_t ki = logit_key(z[i]);
        if (best < 0 || ki > bk) { best = i; bk = ki; }
      }
    }
    used |= 1ull << best;
    idx_out[j] = best;
    zsel[j] = z[best];
  }
}

// Fixed-plus-TopK routing of one token: route_select, then p = 1 for fixed
// slots and, for a routed slot, sigma(z) (eq:router) or, with `softmax`,
// exp(z - max) / sum over the N streams of exp(z - max) (the softmax-router
// ablation); a NaN logit gives a NaN p.
template <int NMAX>
__device__ __forceinline__ void route_token(const float (&z)[NMAX], int N, int m, int k,
                                            int32_t* idx_out, float* p_out, bool softmax = false) {
  float zsel[kMaxK];
  route_select<NMAX>(z, N, m, k, idx_out, zsel);
  for (int j = 0; j < m; ++j) p_out[j] = 1.0f;
  for (int j = m; j < k; ++j) p_out[j] = softmax ? zsel[j] : sigmoidf(zsel[j]);   // softmax: the logit until the sum is known
  if (softmax && k > m) {
    float mx = z[0];
#pragma unroll
    for (int i = 1; i < NMAX; ++i)
      if (i < N) mx = fmaxf(mx, z[i]);
    float den = 0.f;
#pragma unroll
    for (int i = 0; i < NMAX; ++i)
      if (i < N) den += __expf(z[i] - mx);
    for (int j = m; j < k; ++j) p_out[j] = __expf(p_out[j] - mx) / den;
  }
}

// Sinkhorn-Knopp (rows, then columns, per iteration) of exp(L) followed by
// the row clamp, in place on a k x k row-major matrix holding L on entry.
// The row maximum is subtracted before exp: exactly invariant because the
// first operation of each iteration normalises rows.
__device__ __forceinline__ void sinkhorn_clamp(float (&M)[kMaxK * kMaxK], int k, int iters, float delta) {
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j >= k) break;
    float mx = M[j * kMaxK];
#pragma unroll
    for (int l = 1; l < kMaxK; ++l) if (l < k) mx = fmaxf(mx, M[j * kMaxK + l]);
#pragma unroll
    for (int l = 0; l < kMaxK; ++l) if (l < k) M[j * kMaxK + l] = __expf(M[j * kMaxK + l] - mx);
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < kMaxK; ++j) {
      if (j < k) {
        float s = 0.f;
#pragma unroll
        for (int l = 0; l < kMaxK; ++l) if (l < k) s += M[j * kMaxK + l];
        float r = 1.0f / s;
#pragma unroll
        for (int l = 0; l < kMaxK; ++l) if (l < k) M[j * kMaxK + l] *= r;
      }
    }
#pragma unroll
    for (int l = 0; l < kMaxK; ++l) {
      if (l < k) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) if (j < k) s += M[j * kMaxK + l];
        float r = 1.0f / s;
#pragma unroll
        for (int j = 0; j < kMaxK; ++j) if (j < k) M[j * kMaxK + l] *= r;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kMaxK; ++j) {
    if (j < k) {
      float s = 0.f;
#pragma unroll
      for (int l = 0; l < kMaxK; ++l) if (l < k) s += M[j * kMaxK + l];
      if (s > 1.0f + delta) {
        float r = 1.0f / s;
#pragma unroll
        for (int l = 0; l < kMaxK; ++l) if (l < k) M[j * kMaxK + l] *= r;
      }
    }
  }
}

// The same for a compile-time k (no padded rows or columns); identical
// arithmetic and order.
template <int K>
__device__ __forceinline__ void sinkhorn_clamp_k(float (&M)[K * K], int iters, float delta) {
#pragma unroll
  for (int j = 0; j < K; ++j) {
    float mx = M[j * K];
#pragma unroll
    for (int l = 1; l < K; ++l) mx = fmaxf(mx, M[j * K + l]);
#pragma unroll
    for (int l = 0; l < K; ++l) M[j * K + l] = __expf(M[j * K + l] - mx);
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
      float s = 0.f;
#pragma unroll
      for (int l = 0; l < K; ++l) s += M[j * K + l];
      const float r = 1.0f / s;
#pragma unroll
      for (int l = 0; l < K; ++l) M[j * K + l] *= r;
    }
#pragma unroll
    for (int l = 0; l < K; ++l) {
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < K; ++j) s += M[j * K + l];
      const float r = 1.0f / s;
#pragma unroll
      for (int j = 0; j < K; ++j) M[j * K + l] *= r;
    }
  }
#pragma unroll
  for (int j = 0; j < K; ++j) {
    float s = 0.f;
#pragma unroll
    for (int l = 0; l < K; ++l) s += M[j * K + l];
    if (s > 1.0f + delta) {
      const float r = 1.0f / s;
#pragma unroll
      for (int l = 0; l < K; ++l) M[j * K + l] *= r;
    }
  }
}

// Gram-Schmidt of the components e_0 = out, e_1..e_r = conv branches, in the
// basis {e_b}: given the Gram matrix G[a][b] = <e_a, e_b> of one token, returns
// V with v_{i+1} = sum_b V[i][b] e_b following eq:gs (each coefficient uses the
// raw g_j, as printed).  A component whose squared norm is at or below
// 1e-6 of its raw squared norm is taken as zero: a Gram matrix summed in fp32
// cannot resolve it, and its coefficient is then 0 as for an exact zero.
__device__ __forceinline__ void gram_schmidt_basis(const double (&G)[kMaxKr][kMaxKr], int Kr,
                                                   double (&V)[kMaxKr][kMaxKr]) {
#pragma unroll
  for (int i = 0; i < kMaxKr; ++i)
#pragma unroll
    for (int b = 0; b < kMaxKr; ++b) V[i][b] = (i == b) ? 1.0 : 0.0;
  double nrm[kMaxKr];
  bool zero[kMaxKr];
#pragma unroll
  for (int j = 0; j < kMaxKr; ++j) {
    if (j >= Kr) break;
    // v_{j+1} = e_j - sum_{i<j} <e_j, v_i> / <v_i, v_i> v_i
#pragma unroll
    for (int i = 0; i < kMaxKr; ++i) {
      if (i >= j) break;
      if (zero[i]) continue;
      double dot = 0.0;
#pragma unroll
      for (int b = 0; b < kMaxKr; ++b) dot += V[i][b] * G[j][b];
      double c = dot / nrm[i];
#pragma unroll
      for (int b = 0; b < kMaxKr; ++b) V[j][b] -= c * V[i][b];
    }
    double n = 0.0;
#pragma unroll
    for (int a = 0; a < kMaxKr; ++a)
#pragma unroll
      for (int b = 0; b < kMaxKr; ++b) n += V[j][a] * G[a][b] * V[j][b];
    nrm[j] = n;
    zero[j] = n <= 1e-6 * G[j][j];   // a NaN norm is not "vanishing": it propagates
  }
}

// Components e_0..e_{Kr-1} of token t at channels c..c+7: e_0 = F[t], e_j =
// sum_{i < kappa_j} w_j[i] F[t - i] over the part of the window inside t's
// sequence (zero padding before the sequence start).
template <typename TS, int KR>
__device__ __forceinline__ void components(const TS* __restrict__ F, const float* __restrict__ conv_w, int64_t t,
                                           int64_t pos, int C, int c, const int (&kap)[3], float (&e)[KR][8]) {
  float f0[8];
  Vec8<TS>::load(F + t * C + c, f0);
#pragma unroll
  for (int q = 0; q < 8; ++q) e[0][q] = f0[q];
  if (KR == 1) return;
  int row = 0;
#pragma unroll
  for (int j = 1; j < KR; ++j) {
#pragma unroll
    for (int q = 0; q < 8; ++q) e[j][q] = 0.f;
    const int kj = kap[j - 1];
    for (int i = 0; i < kj; ++i) {
      if (i > pos) break;
      float f[8];
      if (i == 0) {
#pragma unroll
        for (int q = 0; q < 8; ++q) f[q] = f0[q];
      } else {
        Vec8<TS>::load(F + (t - i) * C + c, f);
      }
      const float4* w4 = reinterpret_cast<const float4*>(conv_w + (int64_t)(row + i) * C + c);
      const float4 wa = w4[0], wb = w4[1];
      const float w[8] = {wa.x, wa.y, wa.z, wa.w, wb.x, wb.y, wb.z, wb.w};
#pragma unroll
      for (int q = 0; q < 8; ++q) e[j][q] = fmaf(w[q], f[q], e[j][q]);
    }
    row += kj;
  }
}

}  // namespace xhc

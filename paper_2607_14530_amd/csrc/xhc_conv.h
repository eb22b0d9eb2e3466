// Run-based causal depthwise convolution of the paper's branches (eq:aug)
// for kernels that walk consecutive tokens: a thread owns 4 channels and
// keeps the conv taps and the last values of F in registers.
#pragma once
#include "xhc_device.h"

namespace xhc {

// four channels of one row, held in the storage format until used
template <typename TS> struct Row4;
template <> struct Row4<uint16_t> {
  using raw = uint2;
  static __device__ __forceinline__ raw load(const uint16_t* p) { return *reinterpret_cast<const uint2*>(p); }
  static __device__ __forceinline__ raw zero() { return make_uint2(0u, 0u); }
  static __device__ __forceinline__ void unpack(raw v, float (&f)[4]) {
    f[0] = bf_lo(v.x); f[1] = bf_hi(v.x); f[2] = bf_lo(v.y); f[3] = bf_hi(v.y);
  }
  static __device__ __forceinline__ void store(uint16_t* p, const float (&f)[4]) {
    *reinterpret_cast<uint2*>(p) = make_uint2(pack2bf(f[0], f[1]), pack2bf(f[2], f[3]));
  }
  static __device__ __forceinline__ void store_raw(uint16_t* p, raw v) { *reinterpret_cast<uint2*>(p) = v; }
  static __device__ __forceinline__ void round(float (&f)[4]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(f2bf(f[e]) << 16);
  }
};
template <> struct Row4<float> {
  using raw = float4;
  static __device__ __forceinline__ raw load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  static __device__ __forceinline__ raw zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  static __device__ __forceinline__ void unpack(raw v, float (&f)[4]) { f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w; }
  static __device__ __forceinline__ void store(float* p, const float (&f)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
  }
  static __device__ __forceinline__ void store_raw(float* p, raw v) { *reinterpret_cast<float4*>(p) = v; }
  static __device__ __forceinline__ void round(float (&)[4]) {}
};

template <int K1, int K2, int K3>
struct ConvGroup {
  static constexpr int KR = 1 + (K1 > 0) + (K2 > 0) + (K3 > 0);
  static constexpr int TAPS = K1 + K2 + K3;
  static constexpr int KW = (K1 > K2 ? (K1 > K3 ? K1 : K3) : (K2 > K3 ? K2 : K3));
  float w[TAPS][4];
  float hist[KW][4];   // hist[KW - 1 - i] = F[t - 1 - i] before the current group's first token t

  __device__ __forceinline__ void load_taps(const float* __restrict__ conv_w, int C, int c) {
#pragma unroll
    for (int r = 0; r < TAPS; ++r) {
      const float4 v = *reinterpret_cast<const float4*>(conv_w + (int64_t)r * C + c);
      w[r][0] = v.x; w[r][1] = v.y; w[r][2] = v.z; w[r][3] = v.w;
    }
  }
  __device__ __forceinline__ void reset() {
#pragma unroll
    for (int i = 0; i < KW; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) hist[i][q] = 0.f;
  }
  // history before token t0, zero before the start of t0's sequence (the
  // loads are issued unconditionally and all before the first is used)
  template <typename TS>
  __device__ __forceinline__ void init(const TS* __restrict__ F, int64_t t0, int64_t S, int C, int c) {
    const int64_t pos = t0 % S;
    typename Row4<TS>::raw r[KW];
#pragma unroll
    for (int i = 0; i < KW; ++i) {
      const int lag = KW - i;   // hist[i] = F[t0 - lag]
      const int64_t src = t0 >= lag ? t0 - lag : 0;
      r[i] = Row4<TS>::load(F + src * C + c);
    }
#pragma unroll
    for (int i = 0; i < KW; ++i) {
      Row4<TS>::unpack(r[i], hist[i]);
      if (KW - i > pos) {
#pragma unroll
        for (int q = 0; q < 4; ++q) hist[i][q] = 0.f;
      }
    }
  }
  // e_0 = F[t], e_j = sum_{i < kappa_j} w_j[i] F[t - i] for token g of the group (cur[g] = F[t])
  template <int G>
  __device__ __forceinline__ void components(const float (&cur)[G][4], int g, float (&e)[KR][4]) const {
#pragma unroll
    for (int q = 0; q < 4; ++q) e[0][q] = cur[g][q];
    int b = 1, row = 0;
    auto branch = [&](int K) {
#pragma unroll
      for (int q = 0; q < 4; ++q) e[b][q] = 0.f;
#pragma unroll
      for (int i = 0; i < KW; ++i) {
        if (i < K) {
          const int x = g - i;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            e[b][q] = fmaf(w[row + i][q], x >= 0 ? cur[x >= 0 ? x : 0][q] : hist[KW + (x < 0 ? x : -1)][q], e[b][q]);
        }
      }
      row += K;
      ++b;
    };
    if (K1 > 0) branch(K1);
    if (K2 > 0) branch(K2);
    if (K3 > 0) branch(K3);
  }
  template <int G>
  __device__ __forceinline__ void advance(const float (&cur)[G][4]) {
#pragma unroll
    for (int i = 0; i < KW; ++i) {
      const int j = i + G;
#pragma unroll
      for (int q = 0; q < 4; ++q) hist[i][q] = j < KW ? hist[j < KW ? j : 0][q] : cur[j >= KW ? j - KW : 0][q];
    }
  }
};

}  // namespace xhc

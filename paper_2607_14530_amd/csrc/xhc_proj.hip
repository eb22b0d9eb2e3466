// Split-K MFMA projection of token tiles onto packed weights (full state, or
// the gathered active rows), plus the norm moments of each token.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ----------------------------------------------------------------- projection
// One workgroup = 4 waves = TG token groups of 16 x one chunk of cb 32-row
// blocks of K; wave w takes blocks w, w + 4, ... of the chunk for all TG
// groups, so each weight fragment it loads serves TG MFMAs.  MFMA operands:
// A = packed weight fragment (outputs x K), B = 8 state elements per lane
// (K x tokens).  With GATHER, K runs over the active rows: row j of K is
// X[t, idx[t, j], :].  Output part[chunk][o][t] for o < 16*NOB, then sum x and
// sum x^2 at o = NO-2, NO-1 (the moments of eq:router_ln / eq:rmsnorm).
// EXACT: cb divides the k-blocks, so no block needs a bound check.  NOB is an
// upper bound of the nob output blocks.
template <typename TS, int NOB, bool GATHER, bool EXACT, int TG>
__global__ __launch_bounds__(256) void k_proj_partial(const TS* __restrict__ X, int64_t T, int N, int C,
                                                      int64_t K, int64_t cb, const uint4* __restrict__ wpk,
                                                      int nob, const int32_t* __restrict__ idx, int k,
                                                      float* __restrict__ part) {
  constexpr int NO = NOB * 16 + 2;   // LDS rows: outputs, then the two moments
  const int NOr = nob * 16 + 2;      // rows of the partials
  constexpr int TT = kProjTile * TG;   // tokens per workgroup
  constexpr int UNR0 = 16 / TG < 8 ? 16 / TG : 8;
  constexpr int UNR = Vec8<TS>::kSplit ? (UNR0 > 1 ? UNR0 / 2 : 1) : UNR0;   // blocks loaded before use
  __shared__ float red[2][NO][TT];
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int64_t tile = blockIdx.x, chunk = blockIdx.y;
  int64_t tc[TG];
#pragma unroll
  for (int g = 0; g < TG; ++g) {
    const int64_t t = tile * TT + g * kProjTile + tl;
    tc[g] = t < T ? t : T - 1;   // loads stay in bounds; results of t >= T are dropped
  }
  const int64_t nblk = K / 32;
  f32x4 acc[TG][NOB];
  float s1[TG], s2[TG];
#pragma unroll
  for (int g = 0; g < TG; ++g) {
    s1[g] = s2[g] = 0.f;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) acc[g][ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const int64_t bpw = cb / 4;   // blocks per wave, a multiple of 8
  for (int64_t b0 = 0; b0 < bpw; b0 += UNR) {
    uint4 xb[UNR][TG], xl[UNR][TG], wa[UNR][NOB];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int64_t kb = chunk * cb + (b0 + u) * 4 + wave;
      if (EXACT || kb < nblk) {
        const int64_t kk = kb * 32 + grp * 8;
#pragma unroll
        for (int g = 0; g < TG; ++g) {
          const TS* src;
          if (GATHER) {
            const int row = (int)(kk / C);
            const int c = (int)(kk % C);
            src = X + ((tc[g] * N + idx[tc[g] * k + row]) * (int64_t)C + c);
          } else {
            src = X + (tc[g] * (int64_t)N * C + kk);
          }
          float f[8];
          xb[u][g] = Vec8<TS>::operand(src, f, xl[u][g]);
        }
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
          if (ob < nob) wa[u][ob] = wpk[(kb * nob + ob) * kWave + lane];
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int64_t kb = chunk * cb + (b0 + u) * 4 + wave;
      if (EXACT || kb < nblk) {
#pragma unroll
        for (int g = 0; g < TG; ++g) {
          // moments from the operand registers (hi + lo for an fp32 state, to 2^-16)
          float f[8], h[8];
          unpack8(xb[u][g], f);
          unpack8(xl[u][g], h);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float x = f[e] + h[e];
            s1[g] += x;
            s2[g] += x * x;
          }
#pragma unroll
          for (int ob = 0; ob < NOB; ++ob) {
            if (ob < nob) {
              acc[g][ob] = mfma_16x16x32(wa[u][ob], xb[u][g], acc[g][ob]);
              if (Vec8<TS>::kSplit) acc[g][ob] = mfma_16x16x32(wa[u][ob], xl[u][g], acc[g][ob]);
            }
          }
        }
      }
    }
  }
#pragma unroll
  for (int g = 0; g < TG; ++g) {
    s1[g] += __shfl_xor(s1[g], 16);
    s1[g] += __shfl_xor(s1[g], 32);
    s2[g] += __shfl_xor(s2[g], 16);
    s2[g] += __shfl_xor(s2[g], 32);
  }
  // waves 0, 1 write; waves 2, 3 add theirs; the two halves are added on the way out
  for (int step = 0; step < 2; ++step) {
    if ((wave >> 1) == step) {
      float(*r)[TT] = red[wave & 1];
#pragma unroll
      for (int g = 0; g < TG; ++g) {
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            float& dst = r[ob * 16 + grp * 4 + v][g * kProjTile + tl];
            dst = step ? dst + acc[g][ob][v] : acc[g][ob][v];
          }
        if (grp == 0) {
          float& d1 = r[NO - 2][g * kProjTile + tl];
          float& d2 = r[NO - 1][g * kProjTile + tl];
          d1 = step ? d1 + s1[g] : s1[g];
          d2 = step ? d2 + s2[g] : s2[g];
        }
      }
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; i < NOr * TT; i += 256) {
    const int o = i / TT, tt = i % TT;
    const int r = o < nob * 16 ? o : o - nob * 16 + NOB * 16;
    const int64_t tg = tile * TT + tt;
    if (tg < T) part[(chunk * NOr + o) * T + tg] = red[0][r][tt] + red[1][r][tt];
  }
}

// Wide path (bf16 state, full rows, grouped weight layout).  A workgroup
// takes 64 TG tokens (wave w: TG groups of 16, TG = 4, or 2 for five or more
// output blocks) and a chunk
// of cb k-blocks, walked in steps of one group of 4 k-blocks (128 elements):
// each lane loads 64 contiguous bytes of its token per step, so a wave
// requests 256 contiguous bytes of each of its 64 token rows together.  The
// weight fragments of SS steps (a segment) are copied once per workgroup into
// LDS, straight from global memory, and serve the token groups of the four
// waves.  Two LDS buffers alternate: the copy of segment g + 1 is issued when
// segment g starts and has landed by its end, so the only wait per segment
// is one LDS barrier.  Each wave owns its tokens, so partials go out without a
// cross-wave reduction.  EXACT: cb divides the k-blocks.
template <int NOB, bool EXACT, bool GATHER>
__global__ __launch_bounds__(256) void k_proj_wide(const uint16_t* __restrict__ X, int64_t T, int N, int C, int64_t K,
                                                   int64_t cb, const uint4* __restrict__ wpk,
                                                   const int32_t* __restrict__ idx, int k, float* __restrict__ part) {
  constexpr int TG = wide_tg(NOB), KS = kWideStep, NOr = NOB * 16 + 2;
  constexpr int SS = wide_seg_steps(NOB);   // steps whose fragments share one LDS fill
  constexpr int FILL = SS * KS * NOB;       // fragments per segment
  static_assert(FILL % 4 == 0, "every wave copies the same number of fragments");
  extern __shared__ uint4 wl[];             // [2][SS][KS][NOB][64 lanes]; dynamic, as the LDS copy needs it
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int64_t tile = blockIdx.x, chunk = blockIdx.y;
  const int64_t nblk = K / 32, kb0 = chunk * cb;
  const uint16_t* xr[TG];   // the token's state (GATHER: its first row)
  int64_t tok[TG];
  // GATHER: the routed rows of the wave's tokens, read per step from LDS (a
  // private array indexed by the step's row would live in scratch memory)
  __shared__ int32_t s_rows[GATHER ? 4 : 1][GATHER ? TG : 1][16][kMaxK];
  int32_t rid[GATHER ? TG : 1][kMaxK];
#pragma unroll
  for (int g = 0; g < TG; ++g) {
    tok[g] = tile * wide_tokens(NOB) + wave * (16 * TG) + g * 16 + tl;
    const int64_t tc = tok[g] < T ? tok[g] : T - 1;   // loads stay in bounds; results of t >= T are dropped
    if (GATHER) {
      xr[g] = X + tc * N * (int64_t)C + grp * 32;
      // all indices are loaded before any is stored (a store next to its load
      // would wait for it); slots j >= k are never read
#pragma unroll
      for (int j = 0; j < kMaxK; ++j) rid[g][j] = idx[tc * k + (j < k ? j : 0)];
    } else {
      xr[g] = X + tc * K + grp * 32;
    }
  }
  if (GATHER && grp == 0)
#pragma unroll
    for (int g = 0; g < TG; ++g)
#pragma unroll
      for (int j = 0; j < kMaxK; ++j) s_rows[wave][g][tl][j] = rid[g][j];
  if (GATHER) {
    // the rows are read by all lanes of the wave that wrote them: LDS
    // accesses of a wave complete in order once issued in this order
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
  f32x4 acc[TG][NOB];
  float s1[TG], s2[TG];
#pragma unroll
  for (int g = 0; g < TG; ++g) {
    s1[g] = s2[g] = 0.f;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob) acc[g][ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  struct Step {
    uint4 x[KS][TG];
  };
  // grouped layout: step u of the group at kbs takes 8 elements at 32 grp + 8 u
  // GATHER: K index j C + c is channel c of routed row j; a group of 128 never
  // straddles two rows (C % 128 == 0)
  auto load = [&](Step& b, int64_t kbs) {
    const int64_t ko = kbs * 32;
    const int j = GATHER ? (int)(ko / C) : 0;
    const int64_t c = GATHER ? ko % C : ko;
#pragma unroll
    for (int g = 0; g < TG; ++g) {
      const uint16_t* p = xr[g] + c;
      if (GATHER) p += (int64_t)s_rows[wave][g][tl][j] * C;
#pragma unroll
      for (int u = 0; u < KS; ++u) {
        b.x[u][g] = make_uint4(0, 0, 0, 0);
        if (EXACT || kbs + u < nblk) b.x[u][g] = *reinterpret_cast<const uint4*>(p + u * 8);
      }
    }
  };
  auto compute = [&](const Step& b, int64_t kbs, int sj) {
#pragma unroll
    for (int u = 0; u < KS; ++u) {
      if (EXACT || kbs + u < nblk) {
        uint4 wa[NOB];
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) wa[ob] = wl[((sj * KS + u) * NOB + ob) * kWave + lane];
#pragma unroll
        for (int g = 0; g < TG; ++g) {
          float f[8];
          unpack8(b.x[u][g], f);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            s1[g] += f[e];
            s2[g] += f[e] * f[e];
          }
#pragma unroll
          for (int ob = 0; ob < NOB; ++ob) acc[g][ob] = mfma_16x16x32(wa[ob], b.x[u][g], acc[g][ob]);
        }
      }
    }
  };
  const int64_t nsteps = cb / KS;
  const uint32_t wl_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint4*)wl;
  // fragments of segment g -> LDS buffer g % 2, one 1 KiB fragment per wave
  // instruction (a block past the end of K copies the last block; unused)
  auto fill = [&](int64_t g) {
    for (int fi = wave; fi < FILL; fi += 4) {
      int64_t kb = kb0 + g * SS * KS + fi / NOB;
      if (!EXACT && kb >= nblk) kb = nblk - 1;
      lds_dma16(wpk + (kb * NOB + fi % NOB) * kWave + lane,
                __builtin_amdgcn_readfirstlane(wl_base + (uint32_t)(((g & 1) * FILL + fi) * kWave * 16)));
    }
  };
  Step A, B;
  fill(0);
  load(A, kb0);
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  // step s: the next segment's copy goes out at a segment start and the state
  // loads of step s + 1 right after it; both are in flight while step s is
  // computed.  Each step starts with a full wait: then only its own state
  // (and, at a segment's second step, the copy issued one step earlier) is
  // outstanding, so with two or more steps per segment the copy has landed
  // long before the barrier that ends the segment (with one, that barrier
  // waits for it).  The barrier also frees the buffer just read.
  auto step = [&](int64_t s, Step& cur, Step& nxt) __attribute__((always_inline)) {
    const int64_t g = s / SS;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    // the empty asm pins the compiler's own wait for this step's state here,
    // before the copy and the next loads below (it does not count the copy)
#pragma unroll
    for (int u = 0; u < KS; ++u)
#pragma unroll
      for (int gg = 0; gg < TG; ++gg) {
        u32x4 t = {cur.x[u][gg].x, cur.x[u][gg].y, cur.x[u][gg].z, cur.x[u][gg].w};
        asm volatile("" : "+v"(t));
        cur.x[u][gg] = make_uint4(t[0], t[1], t[2], t[3]);
      }
    if (s % SS == 0 && (g + 1) * SS < nsteps) fill(g + 1);
    if (s + 1 < nsteps) load(nxt, kb0 + (s + 1) * KS);
    __builtin_amdgcn_sched_barrier(0);
    compute(cur, kb0 + s * KS, (int)((g & 1) * SS + s % SS));
    __builtin_amdgcn_sched_barrier(0);
    if ((s + 1) % SS == 0 && s + 1 < nsteps) {
      if (SS == 1) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      lds_barrier();
    }
  };
  // (the scheduling barriers keep each phase's loads from being hoisted into
  // the previous one, which would need a third register buffer)
#pragma nounroll
  for (int64_t s = 0; s < nsteps; s += 2) {
    step(s, A, B);
    step(s + 1, B, A);
  }
#pragma unroll
  for (int g = 0; g < TG; ++g) {
    s1[g] += __shfl_xor(s1[g], 16);
    s1[g] += __shfl_xor(s1[g], 32);
    s2[g] += __shfl_xor(s2[g], 16);
    s2[g] += __shfl_xor(s2[g], 32);
    if (tok[g] < T) {
      float* pc = part + chunk * NOr * T + tok[g];
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) pc[(int64_t)(ob * 16 + grp * 4 + v) * T] = acc[g][ob][v];
      if (grp == 0) {
        pc[(int64_t)(NOr - 2) * T] = s1[g];
        pc[(int64_t)(NOr - 1) * T] = s2[g];
      }
    }
  }
}


// output-block bound of a kernel instance: 1, 2, 3, 5 or 8
static inline int nob_bucket(int nob) { return nob <= 3 ? nob : (nob <= 5 ? 5 : 8); }

template <typename TS, bool GATHER, bool EXACT, int TG>
static hipError_t proj_launch(const TS* X, int64_t T, int N, int C, int64_t K, const ProjPlan& pl, const uint4* w,
                              int nob, const int32_t* idx, int k, float* part, hipStream_t s) {
  const dim3 grid((unsigned)((T + kProjTile * TG - 1) / (kProjTile * TG)), (unsigned)pl.nchunk);
#define XHC_PROJ_CASE(NB)                                                                           \
  case NB:                                                                                          \
    k_proj_partial<TS, NB, GATHER, EXACT, TG>                                                       \
        <<<grid, dim3(256), 0, s>>>(X, T, N, C, K, pl.chunk_blocks, w, nob, idx, k, part);          \
    break;
  switch (nob_bucket(nob)) {
    XHC_PROJ_CASE(1) XHC_PROJ_CASE(2) XHC_PROJ_CASE(3) XHC_PROJ_CASE(5) XHC_PROJ_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef XHC_PROJ_CASE
  return hipGetLastError();
}


// dynamic LDS of the wide path: two segment buffers
static inline size_t wide_lds_bytes(int nob) { return (size_t)2 * wide_seg_steps(nob) * kWideStep * nob * 1024; }

// every instance may use its LDS size (above 64 KiB for five or more output
// blocks); set once per device and thread
template <bool GATHER>
static bool wide_attrs_set() {
  static thread_local int dev_done = -1;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  if (dev == dev_done) return true;
  const void* fs[8] = {reinterpret_cast<const void*>(&k_proj_wide<1, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<2, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<3, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<4, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<5, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<6, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<7, false, GATHER>),
                       reinterpret_cast<const void*>(&k_proj_wide<8, false, GATHER>)};
  for (int nb = 1; nb <= 8; ++nb)
    if (hipFuncSetAttribute(fs[nb - 1], hipFuncAttributeMaxDynamicSharedMemorySize, (int)wide_lds_bytes(nb)) !=
        hipSuccess)
      return false;
  dev_done = dev;
  return true;
}

template <bool GATHER>
static hipError_t proj_wide_launch(const uint16_t* X, int64_t T, int N, int C, int64_t K, const ProjPlan& pl,
                                   const uint4* w, int nob, const int32_t* idx, int k, float* part, hipStream_t s) {
  // (the unguarded instance for chunks that divide K needs more registers
  // than two waves per SIMD allow, so the guarded one serves both)
  const dim3 grid((unsigned)((T + wide_tokens(nob) - 1) / wide_tokens(nob)), (unsigned)pl.nchunk);
  const size_t lds = wide_lds_bytes(nob);
  if (!wide_attrs_set<GATHER>()) return hipErrorInvalidConfiguration;
#define XHC_WIDE_CASE(NB)                                                                                      \
  case NB:                                                                                                     \
    k_proj_wide<NB, false, GATHER><<<grid, dim3(256), lds, s>>>(X, T, N, C, K, pl.chunk_blocks, w, idx, k, part); \
    break;
  switch (nob) {
    XHC_WIDE_CASE(1) XHC_WIDE_CASE(2) XHC_WIDE_CASE(3) XHC_WIDE_CASE(4)
    XHC_WIDE_CASE(5) XHC_WIDE_CASE(6) XHC_WIDE_CASE(7) XHC_WIDE_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef XHC_WIDE_CASE
  return hipGetLastError();
}

template <typename TS, bool GATHER>
static hipError_t proj_dispatch(const TS* X, int64_t T, int N, int C, int64_t K, const void* packed, int64_t nout,
                                const int32_t* idx, int k, float* part, hipStream_t s) {
  const ProjPlan pl = proj_plan(Vec8<TS>::kSplit ? XHC_F32 : XHC_BF16, GATHER, K, C, nout, T);
  const uint4* w = reinterpret_cast<const uint4*>(packed);
  const int nob = (int)out_blocks(nout);
  if (nob > 8) return hipErrorInvalidValue;
  if constexpr (!Vec8<TS>::kSplit) {
    if (pl.wide) return proj_wide_launch<GATHER>(X, T, N, C, K, pl, w, nob, idx, k, part, s);
  }
  if (Vec8<TS>::kSplit) return proj_launch<TS, GATHER, false, 1>(X, T, N, C, K, pl, w, nob, idx, k, part, s);
  const bool exact = !GATHER && (K / 32) % pl.chunk_blocks == 0;
#define XHC_PROJ_TG(TGV)                                                                            \
  return exact ? proj_launch<TS, GATHER, !GATHER, TGV>(X, T, N, C, K, pl, w, nob, idx, k, part, s) \
               : proj_launch<TS, GATHER, false, TGV>(X, T, N, C, K, pl, w, nob, idx, k, part, s)
  switch (pl.tg) {
    case 4: XHC_PROJ_TG(4);
    case 2: XHC_PROJ_TG(2);
    default: XHC_PROJ_TG(1);
  }
#undef XHC_PROJ_TG
}

hipError_t launch_proj_partial(int state_dtype, const void* X, int64_t T, int N, int C, int64_t K,
                               const void* packed, int64_t nout, const int32_t* idx, int k, float* part,
                               hipStream_t s) {
  if (T == 0) return hipSuccess;
  if (state_dtype == XHC_BF16) {
    const uint16_t* x = reinterpret_cast<const uint16_t*>(X);
    return idx ? proj_dispatch<uint16_t, true>(x, T, N, C, K, packed, nout, idx, k, part, s)
               : proj_dispatch<uint16_t, false>(x, T, N, C, K, packed, nout, idx, k, part, s);
  }
  const float* x = reinterpret_cast<const float*>(X);
  return idx ? proj_dispatch<float, true>(x, T, N, C, K, packed, nout, idx, k, part, s)
             : proj_dispatch<float, false>(x, T, N, C, K, packed, nout, idx, k, part, s);
}

}  // namespace xhc

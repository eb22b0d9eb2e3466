// Single-pass mapping generation + dense read of a full xHC sublayer
// (bf16 state, N = 16, k = 4, K_r <= 4, C = 128 G with G <= 32).
//
// The state X is read from HBM exactly once.  A 16-token tile of X
// ([16 tokens, 16 streams, C] = 2 MiB at C = 4096) is split over a team of G
// workgroups; member s copies its [16, 16, 128] slice straight into LDS
// (double-buffered) and keeps the matching slices of the projection weights in
// registers for the whole kernel.  Per tile:
//
//  A. every member: MFMA partial of x [W^r, W^pre] over its slice and the
//     partial moments (eq:fused_normalized_projection), published as tagged
//     64-bit records (value, tile tag): a record is valid once its tag matches,
//     so no counter, fence or flag orders the stores;
//  B. per token two members sum the G partials in member order
//     (deterministic): one the router outputs and moments, giving the
//     LayerNorm-corrected logits and the routing (eq:router_topk), the other
//     the pre-map outputs, giving H^pre (RMSNorm correction); they write them
//     out and publish idx and H^pre as tagged records;
//  C. every member collects H^pre and idx of the 16 tokens;
//  D. the dense read input = sum_i H^pre_i x_i of its slice from LDS
//     (eq:dense_read);
//  E. the MFMA partial of the gathered active rows [W^post, W^res] and of
//     sum a^2 over its slice, written to the workspace; a per-token pass after
//     the kernel sums the G partials and forms H^post and H^res.
//
// The copy of tile q + 1 is in flight while tile q is synchronised.  The
// kernel is launched cooperatively, so every member of a team is resident;
// every wait is bounded, so every wave exits.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {
namespace {

constexpr int FN = 16;                        // streams
constexpr int FK = 4;                         // active streams
constexpr int FM = 16;                        // tokens per tile (MFMA columns)
constexpr int FCS = 128;                      // channels per member slice
constexpr int FNT = 512;                      // threads per workgroup
constexpr int FNW = FNT / kWave;              // 8 waves
constexpr int ROWB = FCS * 2;                 // bytes of one (token, stream) row slice
constexpr int TOKP = FN * ROWB + 16;          // token pitch in LDS (16 B pad: conflict-free MFMA reads)
constexpr int BUFB = FM * TOKP;               // one tile buffer
constexpr int NBUF = 2;
constexpr int KB1 = FN * FCS / 32;            // 64 k-blocks of the full projection per slice
constexpr int KB1W = KB1 / FNW;               // 8 per wave
constexpr int NOB1 = 2;                       // 2N = 32 outputs
constexpr int KBA = FK * FCS / 32;            // 16 k-blocks of the active projection per slice
constexpr int KBAW = KBA / FNW;               // 2 per wave
constexpr int NOBA = 2;                       // k*Kr + k*k <= 32 outputs
constexpr int NV1 = 34;                       // 32 outputs + sum x + sum x^2
constexpr int NV2 = FN + FK;                  // broadcast per token: H^pre, idx
constexpr int RING = 4;                       // record slots per team
constexpr int kMaxG = 32;
constexpr unsigned kSpinLimit = 1u << 16;     // polls of one record before the wait gives up

static_assert(KB1 % FNW == 0 && KBA % FNW == 0, "k-blocks must split evenly over waves");
static_assert(FM * FN * ROWB / 1024 % FNW == 0, "tile copies must split evenly over waves");

struct FusedArgs {
  const uint16_t* X;
  const uint4* wfull;     // packed [W_r | W_pre], grouped layout
  const float* colsum;    // column sums of bf16(W_r)
  const uint4* wact;      // packed [W_post | W_res], grouped layout
  const float* alpha;     // pre, res, post
  const float* b_pre;
  uint16_t* input;
  int32_t* idx;
  float* p;
  float* Hpre;
  uint64_t* rec1;         // [teams][RING][G][FM][NV1]
  uint64_t* rec2;         // [teams][RING][FM][NV2]
  int* err;
  float* part2;           // [G][NV1][T] active partials
  int64_t T;
  int C;
  int G;                  // members per team = C / FCS
  int teams;
  int m;
  float eps;
};

struct Smem {
  float red[FNW][NV1][FM];       // per-wave partials for the cross-wave sum
  float vals[kMaxG][NV1];        // a token's member partials (reducer)
  float hp[FM][FN];              // H^pre of the tile
  int id[FM][FK];                // idx of the tile
};

__device__ __forceinline__ uint4 lds_read16(const unsigned char* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ void st_rec(uint64_t* p, float v, uint32_t tag) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Bounded wait until the record carries `tag`; returns its value.  A wait that
// gives up counts in *err, and once *err is set every later wait gives up
// within a few polls, so a failed run still drains quickly.
__device__ __forceinline__ float ld_rec(const uint64_t* p, uint32_t tag, int* err) {
  unsigned n = 0;
  while (true) {
    const uint64_t v = __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((uint32_t)(v >> 32) == tag) return __uint_as_float((uint32_t)v);
    ++n;
    if (n > kSpinLimit ||
        ((n & 255) == 0 && __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
      __hip_atomic_fetch_add(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return 0.f;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// The same for up to two records at once (both loads in flight per poll).
__device__ __forceinline__ void ld_recs2(const uint64_t* const (&p)[2], const bool (&want)[2], uint32_t tag,
                                         int* err, float (&out)[2]) {
  bool need0 = want[0], need1 = want[1];
  unsigned n = 0;
  while (need0 || need1) {
    const uint64_t v0 = need0 ? __hip_atomic_load(const_cast<uint64_t*>(p[0]), __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT) : 0;
    const uint64_t v1 = need1 ? __hip_atomic_load(const_cast<uint64_t*>(p[1]), __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT) : 0;
    if (need0 && (uint32_t)(v0 >> 32) == tag) {
      out[0] = __uint_as_float((uint32_t)v0);
      need0 = false;
    }
    if (need1 && (uint32_t)(v1 >> 32) == tag) {
      out[1] = __uint_as_float((uint32_t)v1);
      need1 = false;
    }
    if (!(need0 || need1)) break;
    ++n;
    if (n > kSpinLimit ||
        ((n & 255) == 0 && __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
      __hip_atomic_fetch_add(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

__global__ __launch_bounds__(FNT, 1) void k_pre_fused(FusedArgs a) {
  extern __shared__ unsigned char tbuf[];   // [NBUF][BUFB]; dynamic, as the LDS copy needs it
  __shared__ Smem sm;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int G = a.G;
  const int team = blockIdx.x / G, s = blockIdx.x % G;
  if (team >= a.teams) return;
  const int C = a.C;
  const int64_t ntiles = (a.T + FM - 1) / FM;
  int64_t nq = 0;
  if (team < ntiles) nq = (ntiles - team + a.teams - 1) / a.teams;
  if (nq == 0) return;

  // ---- weight slices in registers for the whole kernel (grouped layout:
  // fragment cb of the 128-channel slice meets channels 32 grp + 8 cb)
  uint4 wf[KB1W][NOB1];
#pragma unroll
  for (int r = 0; r < KB1W; ++r) {
    const int q = wave * KB1W + r, i = q / (FCS / 32), cb = q % (FCS / 32);
    const int64_t kb = ((int64_t)i * C + (int64_t)s * FCS) / 32 + cb;
#pragma unroll
    for (int ob = 0; ob < NOB1; ++ob) wf[r][ob] = a.wfull[(kb * NOB1 + ob) * kWave + lane];
  }
  uint4 wa[KBAW][NOBA];
#pragma unroll
  for (int r = 0; r < KBAW; ++r) {
    const int q = wave * KBAW + r, j = q / (FCS / 32), cb = q % (FCS / 32);
    const int64_t kb = ((int64_t)j * C + (int64_t)s * FCS) / 32 + cb;
#pragma unroll
    for (int ob = 0; ob < NOBA; ++ob) wa[r][ob] = a.wact[(kb * NOBA + ob) * kWave + lane];
  }

  // ---- tile copy: 64 wave instructions of 1 KiB (4 streams of one token),
  // instruction n -> token n / 4, streams 4 (n % 4) .. + 3; lane -> stream
  // + lane / 16, bytes (lane % 16) * 16 of the row slice
  auto copy_tile = [&](int64_t tile, int b) {
    unsigned char* dst0 = tbuf + (size_t)b * BUFB;
    for (int n = wave; n < FM * FN / 4; n += FNW) {
      const int t = n / 4, i = (n % 4) * 4 + lane / 16;
      int64_t tg = tile * FM + t;
      if (tg >= a.T) tg = a.T - 1;   // in bounds; the token's results are dropped
      const uint16_t* src = a.X + (tg * FN + i) * (int64_t)C + (int64_t)s * FCS + (lane % 16) * 8;
      __builtin_amdgcn_global_load_lds(src, dst0 + t * TOKP + (n % 4) * 4 * ROWB, 16, 0, 0);
    }
  };

  copy_tile(team, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  const float NC = (float)FN * (float)C;
  for (int64_t q = 0; q < nq; ++q) {
    const int64_t tile = team + q * a.teams;
    const int b = (int)(q % NBUF);
    const unsigned char* buf = tbuf + (size_t)b * BUFB;
    const uint32_t tag = (uint32_t)(q + 1);
    const int slot = (int)(q % RING);
    uint64_t* r1 = a.rec1 + (((int64_t)team * RING + slot) * G) * FM * NV1;
    uint64_t* r2 = a.rec2 + ((int64_t)team * RING + slot) * FM * NV2;

    // ---- A: partial projection of the slice, published as tagged records
    {
      f32x4 acc[NOB1];
#pragma unroll
      for (int ob = 0; ob < NOB1; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int r = 0; r < KB1W; ++r) {
        const int qq = wave * KB1W + r, i = qq / (FCS / 32), cb = qq % (FCS / 32);
        const uint4 xb = lds_read16(buf + tl * TOKP + i * ROWB + (grp * 32 + cb * 8) * 2);
        float f[8];
        unpack8(xb, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          s1 += f[e];
          s2 += f[e] * f[e];
        }
#pragma unroll
        for (int ob = 0; ob < NOB1; ++ob) acc[ob] = mfma_16x16x32(wf[r][ob], xb, acc[ob]);
      }
      s1 += __shfl_xor(s1, 16);
      s1 += __shfl_xor(s1, 32);
      s2 += __shfl_xor(s2, 16);
      s2 += __shfl_xor(s2, 32);
#pragma unroll
      for (int ob = 0; ob < NOB1; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) sm.red[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
      if (grp == 0) {
        sm.red[wave][32][tl] = s1;
        sm.red[wave][33][tl] = s2;
      }
    }
    __syncthreads();   // also: every wave is done with the other buffer (tile q - 1)
    if (q + 1 < nq) copy_tile(tile + a.teams, (int)((q + 1) % NBUF));
    for (int u = tid; u < NV1 * FM; u += FNT) {
      const int o = u / FM, t = u % FM;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < FNW; ++w) v += sm.red[w][o][t];
      st_rec(r1 + ((int64_t)s * FM + t) * NV1 + o, v, tag);
    }

    // ---- B: 32 jobs per tile, job j = 2 t + h taken by member j % G: h = 0
    // sums token t's router outputs and moments and routes it, h = 1 sums its
    // pre-map outputs and forms H^pre; both publish their results as records
    for (int j = s; j < 2 * FM; j += G) {
      const int t = j / 2, h = j % 2;
      const int nv = h == 0 ? FN + 2 : FN + 1;   // router outputs + sum x + sum x^2 | pre outputs + sum x^2
      const int n = G * nv;
      // every thread waits on its (at most two) records together
      float val[2] = {0.f, 0.f};
      const uint64_t* src[2];
      bool want[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int u = tid + r * FNT;
        want[r] = u < n;
        const int g = want[r] ? u / nv : 0, vi = want[r] ? u % nv : 0;
        const int o = h == 0 ? (vi < FN ? vi : 32 + (vi - FN)) : (vi < FN ? FN + vi : 33);
        src[r] = r1 + ((int64_t)g * FM + t) * NV1 + o;
      }
      ld_recs2(src, want, tag, a.err, val);
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const int u = tid + r * FNT;
        if (want[r]) sm.vals[u / nv][u % nv] = val[r];
      }
      __syncthreads();
      if (tid < kWave) {
        // lanes 0..nv-1 sum their value over the members in member order
        float v = 0.f;
        if (tid < nv)
          for (int g = 0; g < G; ++g) v += sm.vals[g][tid];
        const int64_t tg = tile * FM + t;
        if (h == 0) {
          const float mu = __shfl(v, FN) / NC, nu = __shfl(v, FN + 1) / NC;
          const float r_ln = 1.0f / sqrtf(fmaxf(nu - mu * mu, 0.f) + a.eps);
          float zr[FN];
#pragma unroll
          for (int i = 0; i < FN; ++i) zr[i] = (__shfl(v, i) - mu * a.colsum[i]) * r_ln;
          if (tid == 0) {
            int32_t id[FK];
            float pp[FK];
            route_token<FN>(zr, FN, a.m, FK, id, pp);
#pragma unroll
            for (int q2 = 0; q2 < FK; ++q2) {
              st_rec(r2 + t * NV2 + FN + q2, __int_as_float(id[q2]), tag);
              if (tg < a.T) {
                a.idx[tg * FK + q2] = id[q2];
                a.p[tg * FK + q2] = pp[q2];
              }
            }
          }
        } else {
          const float nu = __shfl(v, FN) / NC;
          const float r_rms = 1.0f / sqrtf(nu + a.eps);
          if (tid < FN) {
            const float hpre = sigmoidf(a.alpha[0] * (v * r_rms) + a.b_pre[tid]);
            st_rec(r2 + t * NV2 + tid, hpre, tag);
            if (tg < a.T) a.Hpre[tg * FN + tid] = hpre;
          }
        }
      }
      __syncthreads();
    }

    // ---- C: H^pre and idx of the tile
    if (tid < FM * NV2) {
      const int t = tid / NV2, v = tid % NV2;
      const float x = ld_rec(r2 + t * NV2 + v, tag, a.err);
      if (v < FN) sm.hp[t][v] = x;
      else sm.id[t][v - FN] = __float_as_int(x) & (FN - 1);   // always a row of the tile
    }
    __syncthreads();

    // ---- D: dense read of the slice, thread -> token tid / 32, channels 4 (tid % 32) .. + 3
    {
      const int t = tid / 32, c4 = (tid % 32) * 4;
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        const uint2 v = *reinterpret_cast<const uint2*>(buf + t * TOKP + i * ROWB + c4 * 2);
        const float h = sm.hp[t][i];
        acc[0] = fmaf(h, bf_lo(v.x), acc[0]);
        acc[1] = fmaf(h, bf_hi(v.x), acc[1]);
        acc[2] = fmaf(h, bf_lo(v.y), acc[2]);
        acc[3] = fmaf(h, bf_hi(v.y), acc[3]);
      }
      const int64_t tg = tile * FM + t;
      if (tg < a.T)
        *reinterpret_cast<uint2*>(a.input + tg * C + (int64_t)s * FCS + c4) =
            make_uint2(pack2bf(acc[0], acc[1]), pack2bf(acc[2], acc[3]));
    }

    // ---- E: partial projection of the gathered active rows of the slice
    {
      f32x4 acc[NOBA];
#pragma unroll
      for (int ob = 0; ob < NOBA; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      float s2 = 0.f;
#pragma unroll
      for (int r = 0; r < KBAW; ++r) {
        const int qq = wave * KBAW + r, j = qq / (FCS / 32), cb = qq % (FCS / 32);
        const int row = sm.id[tl][j];
        const uint4 xb = lds_read16(buf + tl * TOKP + row * ROWB + (grp * 32 + cb * 8) * 2);
        float f[8];
        unpack8(xb, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) s2 += f[e] * f[e];
#pragma unroll
        for (int ob = 0; ob < NOBA; ++ob) acc[ob] = mfma_16x16x32(wa[r][ob], xb, acc[ob]);
      }
      s2 += __shfl_xor(s2, 16);
      s2 += __shfl_xor(s2, 32);
#pragma unroll
      for (int ob = 0; ob < NOBA; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) sm.red[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
      if (grp == 0) {
        sm.red[wave][32][tl] = 0.f;
        sm.red[wave][33][tl] = s2;
      }
    }
    __syncthreads();
    for (int u = tid; u < NV1 * FM; u += FNT) {
      const int o = u / FM, t = u % FM;
      const int64_t tg = tile * FM + t;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < FNW; ++w) v += sm.red[w][o][t];
      if (tg < a.T) a.part2[((int64_t)s * NV1 + o) * a.T + tg] = v;
    }
    // the next tile's copy has landed in every wave; sm.red is free again
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
}

__global__ void k_zero_ints(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

struct DeviceInfo {
  int cus = 0;
  int per_cu = 0;
};

constexpr size_t kTileLds = (size_t)NBUF * BUFB;

DeviceInfo device_info() {
  static thread_local int dev_cached = -1;
  static thread_local DeviceInfo info;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DeviceInfo{};
  if (dev != dev_cached) {
    DeviceInfo di;
    if (hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return DeviceInfo{};
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(k_pre_fused), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kTileLds) != hipSuccess)
      return DeviceInfo{};
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&di.per_cu, reinterpret_cast<const void*>(k_pre_fused), FNT,
                                                     kTileLds) != hipSuccess)
      return DeviceInfo{};
    info = di;
    dev_cached = dev;
  }
  return info;
}

}  // namespace

bool fused_pre_supported(const xhc_dims* d) {
  return d->state_dtype == XHC_BF16 && d->N == FN && d->k == FK && d->Kr >= 1 &&
         FK * d->Kr + FK * FK <= 16 * NOBA && d->C % FCS == 0 && d->C / FCS <= kMaxG;
}

// Workspace: error counter, records (sized for up to kMaxResident co-resident
// workgroups), active partials [G][34][T] and their per-token sums.
constexpr int kMaxResident = 1024;
size_t rec1_words(int G) { return (size_t)(kMaxResident / G) * RING * G * FM * NV1; }
size_t rec2_words(int G) { return (size_t)(kMaxResident / G) * RING * FM * NV2; }
size_t align256(size_t b) { return (b + 255) / 256 * 256; }

size_t fused_pre_ws_bytes(const xhc_dims* d) {
  const int G = d->C / FCS;
  return 256 + align256(rec1_words(G) * 8) + align256(rec2_words(G) * 8) +
         align256((size_t)G * NV1 * d->T * sizeof(float)) + align256((size_t)NV1 * d->T * sizeof(float));
}

hipError_t launch_pre_fused(const xhc_dims* d, const void* X, const void* packed_full, const float* colsum,
                            const void* packed_act, const float* alpha, const float* b_pre, const float* b_res,
                            const float* b_post, void* input, int32_t* idx, float* p, float* Hpre, float* Hres,
                            float* Hpost, void* ws, hipStream_t s) {
  const DeviceInfo di = device_info();
  if (di.cus <= 0 || di.per_cu <= 0) return hipErrorInvalidConfiguration;
  const int G = d->C / FCS;
  int teams = di.cus * di.per_cu / G;
  if (teams < 1) return hipErrorInvalidConfiguration;
  if (teams > kMaxResident / G) teams = kMaxResident / G;
  char* w = reinterpret_cast<char*>(ws);
  FusedArgs a{};
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.wfull = reinterpret_cast<const uint4*>(packed_full);
  a.colsum = colsum;
  a.wact = reinterpret_cast<const uint4*>(packed_act);
  a.alpha = alpha;
  a.b_pre = b_pre;
  a.input = reinterpret_cast<uint16_t*>(input);
  a.idx = idx;
  a.p = p;
  a.Hpre = Hpre;
  a.err = reinterpret_cast<int*>(w);
  a.rec1 = reinterpret_cast<uint64_t*>(w + 256);
  a.rec2 = reinterpret_cast<uint64_t*>(w + 256 + align256(rec1_words(G) * 8));
  a.part2 = reinterpret_cast<float*>(w + 256 + align256(rec1_words(G) * 8) + align256(rec2_words(G) * 8));
  float* sums = a.part2 + align256((size_t)G * NV1 * d->T * sizeof(float)) / sizeof(float);
  a.T = d->T;
  a.C = d->C;
  a.G = G;
  a.teams = teams;
  a.m = d->m;
  a.eps = d->eps;
  // records start untagged: clear the error counter and the slots in use
  const size_t used1 = (size_t)teams * RING * G * FM * NV1, used2 = (size_t)teams * RING * FM * NV2;
  k_zero_ints<<<dim3(1), dim3(64), 0, s>>>(a.err, 64);
  k_zero_ints<<<dim3((unsigned)((2 * used1 + 255) / 256)), dim3(256), 0, s>>>(reinterpret_cast<int*>(a.rec1),
                                                                           (int)(2 * used1));
  k_zero_ints<<<dim3((unsigned)((2 * used2 + 255) / 256)), dim3(256), 0, s>>>(reinterpret_cast<int*>(a.rec2),
                                                                           (int)(2 * used2));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  void* args[] = {&a};
  e = hipLaunchCooperativeKernel(reinterpret_cast<const void*>(k_pre_fused), dim3(teams * G), dim3(FNT), args,
                                 kTileLds, s);
  if (e != hipSuccess) return e;
  // active partials -> H^post, H^res (Sinkhorn + clamp)
  return launch_pre_coef(a.part2, G, (int64_t)FK * d->Kr + FK * FK, d->T, FK, d->Kr, 1, d->C, alpha + 2, alpha + 1,
                         b_post, b_res, d->eps, d->sinkhorn_iters, d->clamp_delta, Hpost, Hres, sums, nullptr, 0, 0,
                         0, s);
}

}  // namespace xhc

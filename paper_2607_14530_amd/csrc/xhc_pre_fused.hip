// Single-pass mapping generation + dense read of a full xHC sublayer
// (bf16 state, N = 16, k = 4, K_r <= 4, C % 128 == 0).
//
// The state X is read from HBM exactly once.  A 16-token tile of X
// ([16 tokens, 16 streams, C] = 2 MiB at C = 4096) is split over a team of
// G = C / 128 workgroups; each workgroup keeps its [16, 16, 128] slice in LDS
// (64 KiB, double-buffered) and the matching slices of the projection weights
// in registers for the whole kernel.  Per tile:
//
//  1. MFMA partial of x [W^r, W^pre] over the slice + partial moments, written
//     to a ring slot; the last workgroup of the team to arrive reduces the G
//     partials in slot order (deterministic), applies the LayerNorm / RMSNorm
//     corrections (eq:fused_normalized_projection), H^pre and the routing
//     (eq:router_topk), and raises the tile's flag.
//  2. After the flag: the dense read input = sum_i H^pre_i x_i of the slice
//     from LDS (eq:dense_read), then the MFMA partial of the gathered active
//     rows [W^post, W^res] + partial sum a^2; the last workgroup to arrive
//     reduces them and produces H^post and H^res (Sinkhorn + row clamp).
//
// Loads of tile q+1 are in flight while tile q waits for its flag.  The kernel
// is launched cooperatively so that every workgroup of a team is resident;
// waits are bounded so that every wave always exits.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {
namespace {

constexpr int FN = 16;                        // streams
constexpr int FK = 4;                         // active streams
constexpr int FM = 8;                         // tokens per tile (MFMA columns 8..15 idle)
constexpr int FCS = 128;                      // channels per workgroup slice
constexpr int FNT = 512;                      // threads per workgroup
constexpr int FNW = FNT / kWave;              // 8 waves
constexpr int ROWB = FCS * 2;                 // bytes of one (token, stream) row slice
constexpr int TOKP = FN * ROWB + 16;          // token pitch in LDS (16 B pad: conflict-free MFMA reads)
constexpr int BUFB = FM * TOKP;               // one tile buffer
constexpr int KB1 = FN * FCS / 32;            // 64 k-blocks of the full projection per slice
constexpr int KB1W = KB1 / FNW;               // 8 per wave
constexpr int NOB1 = 2;                       // 2N = 32 outputs
constexpr int KBA = FK * FCS / 32;            // 16 k-blocks of the active projection per slice
constexpr int KBAW = KBA / FNW;               // 2 per wave
constexpr int NOBA = 2;                       // k*Kr + k*k <= 32 outputs
constexpr int PST = 36;                       // floats per token in a partial record
constexpr int NBUF = 4;                       // LDS tile buffers: NBUF - 1 tiles wait on their flag
constexpr int DEPTH = NBUF - 1;               // tiles published ahead of the one being read
constexpr int RING = 8;                       // ring slots per team (>= DEPTH + 2)
constexpr int LOADS = FM * FN * ROWB / 16 / FNT;  // 16-byte loads per thread per tile (4)
constexpr int TSUM_UNROLL = 16;               // independent loads in flight per thread in a team sum
constexpr unsigned kSpinLimit = 1u << 22;

static_assert(KB1 % FNW == 0 && KBA % FNW == 0, "k-blocks must split evenly over waves");
static_assert(FM <= 16 && LOADS * FNT * 16 == FM * FN * ROWB, "tile must split evenly over threads");
static_assert(RING >= DEPTH + 2, "ring too shallow for the pipeline depth");

struct FusedArgs {
  const uint16_t* X;
  const uint4* wfull;     // packed [W_r | W_pre]
  const float* colsum;    // column sums of bf16(W_r)
  const uint4* wact;      // packed [W_post | W_res]
  const float* alpha;     // pre, res, post
  const float* b_pre;
  const float* b_res;
  const float* b_post;
  uint16_t* input;
  int32_t* idx;
  float* p;
  float* Hpre;
  float* Hres;
  float* Hpost;
  float* part1;           // [teams*RING][G][FM][PST]
  float* part2;
  int* cnt1;              // [teams*RING]
  int* cnt2;
  int* flag;
  int* err;
  int64_t T;
  int C;
  int G;                  // workgroups per team = C / FCS
  int teams;
  int m;
  int Kr;
  int iters;
  float eps;
  float delta;
};

struct Smem {
  unsigned char buf[NBUF][BUFB];
  float red[FNW][34][FM];        // per-wave partials (outputs + 2 moments) for the cross-wave sum
  float fin[34][FM];             // reduced team values of one tile
  float hp[FM][FN];              // H^pre of the tile
  int id[FM][FK];                // idx of the tile
  int last;
};

__device__ __forceinline__ uint4 lds_read16(const unsigned char* p) { return *reinterpret_cast<const uint4*>(p); }

// Cross-workgroup data (partials, the tile's H^pre / idx, counters, flags)
// moves only through device-coherent accesses: agent-scope relaxed atomic
// loads and stores bypass the XCD-local caches, so no full-cache
// write-back / invalidate is needed.  A producer drains its stores
// (s_waitcnt) before the counter or flag update that publishes them; a
// consumer reads them only after observing that update.
template <typename V> __device__ __forceinline__ void st_dev(V* p, V v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename V> __device__ __forceinline__ V ld_dev(const V* p) {
  return __hip_atomic_load(const_cast<V*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void drain() { __builtin_amdgcn_s_waitcnt(0); }

// Bounded wait (thread 0) until flag == want.
__device__ __forceinline__ void wait_flag(int* flag, int want, int* err) {
  unsigned n = 0;
  while (ld_dev(flag) != want) {
    __builtin_amdgcn_s_sleep(2);
    if (++n > kSpinLimit) {
      __hip_atomic_fetch_add(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
  }
}

// Publish this workgroup's partial (stored by every thread with st_dev) and
// report whether it was the last of the team for that slot.
__device__ __forceinline__ bool publish(int* cnt, int G, Smem& sm) {
  drain();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sm.last = (old == G - 1);
  }
  __syncthreads();
  return sm.last != 0;
}

// Sum the per-wave values red[w][o][t] and store the workgroup record to part.
__device__ __forceinline__ void store_partial(Smem& sm, int nvals, float* rec) {
  for (int i = threadIdx.x; i < nvals * FM; i += FNT) {
    const int o = i / FM, t = i % FM;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < FNW; ++w) s += sm.red[w][o][t];
    st_dev(&rec[t * PST + o], s);
  }
}

// Team sum (slot order g = 0..G-1) of records -> sm.fin[o][t].  The loads of
// TSUM_UNROLL team members are issued before any is added, so a sum costs
// about G / TSUM_UNROLL memory round trips instead of G.
__device__ __forceinline__ void team_sum(Smem& sm, const float* slot, int G, int nvals) {
  for (int i = threadIdx.x; i < nvals * FM; i += FNT) {
    const int o = i / FM, t = i % FM;
    float s = 0.f;
    for (int g0 = 0; g0 < G; g0 += TSUM_UNROLL) {
      float v[TSUM_UNROLL];
#pragma unroll
      for (int u = 0; u < TSUM_UNROLL; ++u)
        v[u] = (g0 + u < G) ? ld_dev(&slot[((int64_t)(g0 + u) * FM + t) * PST + o]) : 0.f;
#pragma unroll
      for (int u = 0; u < TSUM_UNROLL; ++u) s += v[u];
    }
    sm.fin[o][t] = s;
  }
  __syncthreads();
}

__global__ __launch_bounds__(FNT, 1) void k_pre_fused(FusedArgs a) {
  __shared__ Smem sm;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int team = blockIdx.x / a.G, s = blockIdx.x % a.G;
  if (team >= a.teams) return;
  const int C = a.C;
  const int64_t ntiles = (a.T + FM - 1) / FM;
  const int nact = FK * a.Kr + FK * FK;

  // ---- weight slices in registers for the whole kernel
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

  // ---- tile loader: 8 x 16 B per thread; chunk c = it*512 + tid covers
  // row (token it*2 + tid/256, stream (tid/16)%16), bytes (tid%16)*16
  uint4 ld[LOADS];
  auto issue_loads = [&](int64_t tile) {
#pragma unroll
    for (int it = 0; it < LOADS; ++it) {
      const int t = it * (FNT / (FN * 16)) + tid / (FN * 16);
      const int i = (tid / 16) % FN, cr = tid % 16;
      const int64_t tg = tile * FM + t;
      if (tg < a.T)
        ld[it] = *reinterpret_cast<const uint4*>(a.X + (tg * FN + i) * (int64_t)C + (int64_t)s * FCS + cr * 8);
      else
        ld[it] = make_uint4(0, 0, 0, 0);
    }
  };
  auto store_loads = [&](int b) {
#pragma unroll
    for (int it = 0; it < LOADS; ++it) {
      const int t = it * (FNT / (FN * 16)) + tid / (FN * 16);
      const int i = (tid / 16) % FN, cr = tid % 16;
      *reinterpret_cast<uint4*>(&sm.buf[b][t * TOKP + i * ROWB + cr * 16]) = ld[it];
    }
  };

  // ---- step 1: partial full projection of the tile in buffer b, publish, finalise if last
  auto step1 = [&](int64_t tile, int b, int slot) {
    f32x4 acc[NOB1];
#pragma unroll
    for (int ob = 0; ob < NOB1; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int r = 0; r < KB1W; ++r) {
      const int q = wave * KB1W + r, i = q / (FCS / 32), cb = q % (FCS / 32);
      // grouped weight layout: fragment cb of the 128-channel slice meets channels 32 grp + 8 cb
      const uint4 xb = (tl < FM) ? lds_read16(&sm.buf[b][tl * TOKP + i * ROWB + (grp * 32 + cb * 8) * 2])
                                 : make_uint4(0, 0, 0, 0);
      float f[8];
      unpack8(xb, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) { s1 += f[e]; s2 += f[e] * f[e]; }
#pragma unroll
      for (int ob = 0; ob < NOB1; ++ob) acc[ob] = mfma_16x16x32(wf[r][ob], xb, acc[ob]);
    }
    s1 += __shfl_xor(s1, 16); s1 += __shfl_xor(s1, 32);
    s2 += __shfl_xor(s2, 16); s2 += __shfl_xor(s2, 32);
    if (tl < FM) {
#pragma unroll
      for (int ob = 0; ob < NOB1; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) sm.red[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
      if (grp == 0) { sm.red[wave][32][tl] = s1; sm.red[wave][33][tl] = s2; }
    }
    __syncthreads();
    float* slotp = a.part1 + (int64_t)slot * a.G * FM * PST;
    store_partial(sm, 34, slotp + (int64_t)s * FM * PST);
    if (!publish(&a.cnt1[slot], a.G, sm)) return;
    // last arriver: team reduction, norms, H^pre, routing
    team_sum(sm, slotp, a.G, 34);
    const float NC = (float)FN * (float)C;
    if (tid < FM * FN) {
      const int t = tid / FN, i = tid % FN;
      const int64_t tg = tile * FM + t;
      const float mu = sm.fin[32][t] / NC, nu = sm.fin[33][t] / NC;
      const float r_ln = 1.0f / sqrtf(fmaxf(nu - mu * mu, 0.f) + a.eps);
      const float r_rms = 1.0f / sqrtf(nu + a.eps);
      const float zr = (sm.fin[i][t] - mu * a.colsum[i]) * r_ln;
      const float hpre = sigmoidf(a.alpha[0] * (sm.fin[FN + i][t] * r_rms) + a.b_pre[i]);
      sm.red[0][i][t] = zr;
      if (tg < a.T) st_dev(&a.Hpre[tg * FN + i], hpre);
    }
    __syncthreads();
    if (tid < FM) {
      const int64_t tg = tile * FM + tid;
      float z[FN];
#pragma unroll
      for (int i = 0; i < FN; ++i) z[i] = sm.red[0][i][tid];
      int32_t id[FK];
      float pp[FK];
      route_token<FN>(z, FN, a.m, FK, id, pp);
      if (tg < a.T)
#pragma unroll
        for (int j = 0; j < FK; ++j) { st_dev(&a.idx[tg * FK + j], id[j]); a.p[tg * FK + j] = pp[j]; }
    }
    drain();
    __syncthreads();
    if (tid == 0) {
      st_dev(&a.cnt1[slot], 0);
      st_dev(&a.flag[slot], (int)(tile + 1));
    }
  };

  // ---- step 2: dense read + partial active projection of the tile in buffer b
  auto step2 = [&](int64_t tile, int b, int slot) {
    if (tid == 0) wait_flag(&a.flag[slot], (int)(tile + 1), a.err);
    __syncthreads();
    if (tid < FM * FN) {
      const int t = tid / FN, i = tid % FN;
      const int64_t tg = tile * FM + t;
      sm.hp[t][i] = (tg < a.T) ? ld_dev(&a.Hpre[tg * FN + i]) : 0.f;
    } else if (tid < FM * FN + FM * FK) {
      const int t = (tid - FM * FN) / FK, j = (tid - FM * FN) % FK;
      const int64_t tg = tile * FM + t;
      sm.id[t][j] = (tg < a.T) ? ld_dev(&a.idx[tg * FK + j]) : j;
    }
    __syncthreads();
    // dense read: thread -> token tid / TPT, channels (tid % TPT) * CPT .. + CPT
    {
      constexpr int TPT = FNT / FM;            // threads per token (64)
      constexpr int CPT = FCS / TPT;           // channels per thread (2)
      static_assert(CPT == 2, "dense read is written for two channels per thread");
      const int t = tid / TPT, c2 = (tid % TPT) * CPT;
      const int64_t tg = tile * FM + t;
      float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
      for (int i = 0; i < FN; ++i) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(&sm.buf[b][t * TOKP + i * ROWB + c2 * 2]);
        const float h = sm.hp[t][i];
        acc0 = fmaf(h, bf_lo(v), acc0);
        acc1 = fmaf(h, bf_hi(v), acc1);
      }
      if (tg < a.T)
        *reinterpret_cast<uint32_t*>(a.input + tg * C + (int64_t)s * FCS + c2) = pack2bf(acc0, acc1);
    }
    // active projection partial
    f32x4 acc[NOBA];
#pragma unroll
    for (int ob = 0; ob < NOBA; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
    float s2 = 0.f;
#pragma unroll
    for (int r = 0; r < KBAW; ++r) {
      const int q = wave * KBAW + r, j = q / (FCS / 32), cb = q % (FCS / 32);
      const int row = sm.id[tl % FM][j] & (FN - 1);   // always inside the tile, whatever idx holds
      // grouped weight layout (C % 128 == 0): fragment cb meets channels 32 grp + 8 cb
      const uint4 xb = (tl < FM) ? lds_read16(&sm.buf[b][tl * TOKP + row * ROWB + (grp * 32 + cb * 8) * 2])
                                 : make_uint4(0, 0, 0, 0);
      float f[8];
      unpack8(xb, f);
#pragma unroll
      for (int e = 0; e < 8; ++e) s2 += f[e] * f[e];
#pragma unroll
      for (int ob = 0; ob < NOBA; ++ob) acc[ob] = mfma_16x16x32(wa[r][ob], xb, acc[ob]);
    }
    s2 += __shfl_xor(s2, 16); s2 += __shfl_xor(s2, 32);
    __syncthreads();   // sm.red is free again (step 1 of this tile finished with it)
    if (tl < FM) {
#pragma unroll
      for (int ob = 0; ob < NOBA; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) sm.red[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
      if (grp == 0) sm.red[wave][32][tl] = s2;
    }
    __syncthreads();
    float* slotp = a.part2 + (int64_t)slot * a.G * FM * PST;
    store_partial(sm, 33, slotp + (int64_t)s * FM * PST);
    if (!publish(&a.cnt2[slot], a.G, sm)) return;
    team_sum(sm, slotp, a.G, 33);
    if (tid < FM) {
      const int t = tid;
      const int64_t tg = tile * FM + t;
      const float rstd = 1.0f / sqrtf(sm.fin[32][t] / ((float)FK * (float)C) + a.eps);
      if (tg < a.T) {
        for (int o = 0; o < FK * a.Kr; ++o)
          a.Hpost[tg * FK * a.Kr + o] = 2.0f * sigmoidf(a.alpha[2] * (sm.fin[o][t] * rstd) + a.b_post[o]);
        float Mx[kMaxK * kMaxK];
#pragma unroll
        for (int j = 0; j < kMaxK; ++j)
#pragma unroll
          for (int l = 0; l < kMaxK; ++l)
            Mx[j * kMaxK + l] = (j < FK && l < FK)
                ? a.alpha[1] * (sm.fin[FK * a.Kr + j * FK + l][t] * rstd) + a.b_res[j * FK + l] : 0.f;
        sinkhorn_clamp(Mx, FK, a.iters, a.delta);
#pragma unroll
        for (int j = 0; j < FK; ++j)
#pragma unroll
          for (int l = 0; l < FK; ++l) a.Hres[(tg * FK + j) * FK + l] = Mx[j * kMaxK + l];
      }
    }
    __syncthreads();
    if (tid == 0) st_dev(&a.cnt2[slot], 0);
    (void)nact;
  };

  // ---- software pipeline over this team's tiles (team, team + teams, ...):
  // DEPTH tiles are published (step 1) ahead of the tile whose flag is awaited
  // (step 2); loads of the next tile are in flight during that wait.
  int64_t nq = 0;
  if (team < ntiles) nq = (ntiles - team + a.teams - 1) / a.teams;
  if (nq == 0) return;
  auto tile_of = [&](int64_t q) { return team + q * a.teams; };
  auto slot_of = [&](int64_t q) { return team * RING + (int)(q % RING); };
  for (int64_t q = 0; q < DEPTH && q < nq; ++q) {
    issue_loads(tile_of(q));
    store_loads((int)(q % NBUF));
    __syncthreads();
    step1(tile_of(q), (int)(q % NBUF), slot_of(q));
  }
  for (int64_t q = 0; q < nq; ++q) {
    const int64_t qn = q + DEPTH;
    const bool more = qn < nq;
    if (more) issue_loads(tile_of(qn));
    step2(tile_of(q), (int)(q % NBUF), slot_of(q));
    if (more) {
      __syncthreads();
      store_loads((int)(qn % NBUF));
      __syncthreads();
      step1(tile_of(qn), (int)(qn % NBUF), slot_of(qn));
    }
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

DeviceInfo device_info() {
  static thread_local int dev_cached = -1;
  static thread_local DeviceInfo info;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DeviceInfo{};
  if (dev != dev_cached) {
    DeviceInfo di;
    if (hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return DeviceInfo{};
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&di.per_cu, reinterpret_cast<const void*>(k_pre_fused), FNT,
                                                     0) != hipSuccess)
      return DeviceInfo{};
    info = di;
    dev_cached = dev;
  }
  return info;
}

}  // namespace

bool fused_pre_supported(const xhc_dims* d) {
  return d->state_dtype == XHC_BF16 && d->N == FN && d->k == FK && d->Kr >= 1 &&
         FK * d->Kr + FK * FK <= 16 * NOBA && d->C % FCS == 0 && d->C / FCS <= 256;
}

// Workspace: ints (cnt1, cnt2, flag: one per ring slot; err) then part1, part2.
// Sized for up to kMaxResident co-resident workgroups.
constexpr int kMaxResident = 1024;
int max_teams(int G) { return kMaxResident / G > 0 ? kMaxResident / G : 1; }
size_t hdr_ints(int G) { return (size_t)3 * max_teams(G) * RING + 64; }
size_t hdr_bytes(int G) { return (hdr_ints(G) * sizeof(int) + 255) / 256 * 256; }
size_t part_floats(int G) { return (size_t)max_teams(G) * RING * G * FM * PST; }

size_t fused_pre_ws_bytes(const xhc_dims* d) {
  const int G = d->C / FCS;
  return hdr_bytes(G) + 2 * part_floats(G) * sizeof(float);
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
  if (teams > max_teams(G)) teams = max_teams(G);
  FusedArgs a{};
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.wfull = reinterpret_cast<const uint4*>(packed_full);
  a.colsum = colsum;
  a.wact = reinterpret_cast<const uint4*>(packed_act);
  a.alpha = alpha; a.b_pre = b_pre; a.b_res = b_res; a.b_post = b_post;
  a.input = reinterpret_cast<uint16_t*>(input);
  a.idx = idx; a.p = p; a.Hpre = Hpre; a.Hres = Hres; a.Hpost = Hpost;
  const int slots = max_teams(G) * RING;
  int* ints = reinterpret_cast<int*>(ws);
  a.cnt1 = ints;
  a.cnt2 = ints + slots;
  a.flag = ints + 2 * slots;
  a.err = ints + 3 * slots;
  a.part1 = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + hdr_bytes(G));
  a.part2 = a.part1 + part_floats(G);
  a.T = d->T; a.C = d->C; a.G = G; a.teams = teams; a.m = d->m; a.Kr = d->Kr;
  a.iters = d->sinkhorn_iters; a.eps = d->eps; a.delta = d->clamp_delta;
  const int nint_hdr = (int)hdr_ints(G);
  k_zero_ints<<<dim3((unsigned)((nint_hdr + 255) / 256)), dim3(256), 0, s>>>(ints, nint_hdr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(k_pre_fused), dim3(teams * G), dim3(FNT), args, 0,
                                    s);
}

}  // namespace xhc

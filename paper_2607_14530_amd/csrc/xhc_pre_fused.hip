// Single-pass mapping generation + dense read of a full xHC sublayer
// (bf16 state, N = 16, k = 4, K_r <= 4, C = 128 G with G dividing 32).
//
// The state X is read from HBM exactly once.  A 16-token tile of X
// ([16 tokens, 16 streams, C] = 2 MiB at C = 4096) is split over a team of G
// workgroups; member s takes the 128-channel slice s of every (token, stream)
// row and keeps the matching slices of the projection weights in registers
// for the whole kernel.  Wave w of a member holds channels 16 w .. 16 w + 15
// of all 16 streams of the tile (4 KiB, 32 registers per lane), so the dense
// read of a channel is a sum inside one lane pair.  Per tile q:
//
//  A. every member: MFMA partial of x [W^r, W^pre] over its slice and the
//     partial moments (eq:fused_normalized_projection), published as tagged
//     64-bit records (value, tile tag): a record is valid once its tag matches,
//     so no counter, fence or flag orders the stores;
//  B. one iteration later, per token two members sum the G partials in member
//     order (deterministic): one the router outputs and moments, giving the
//     LayerNorm-corrected logits and the routing (eq:router_topk), the other
//     the pre-map outputs, giving H^pre (RMSNorm correction); both publish
//     their results as records;
//  C. two iterations later every member collects H^pre and idx of the tile,
//     then forms the dense read input = sum_i H^pre_i x_i of its slice
//     (eq:dense_read) and the MFMA partial of the gathered active rows
//     [W^post, W^res] with sum a^2; a per-token pass after the kernel sums the
//     G partials and forms H^post and H^res.
//
// So every wait on another member has a full iteration of slack, and each
// member keeps three tiles in registers (q, q - 1, q - 2).  A tile reaches the
// registers through one LDS buffer: waves 0-3 copy it there with direct
// global->LDS loads, issued as soon as the previous tile has left the buffer.
// Waves 4-7 do all waiting on records: a wave that waits on a load also waits
// on every earlier load of its own, so the copy waves must not poll.  The
// reducer jobs run on waves 4, 5, ...; a step ends when its slowest wave does,
// so when wave 4 is the only reducer it neither polls nor publishes the
// partials of A after S3 (it stores the active partials before S3, where it
// would otherwise wait), and wave 0, which shares its SIMD, does not publish
// either.  The kernel is launched
// cooperatively, so every member of a team is resident; every wait is
// bounded, so every wave exits.
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
constexpr int NCOPY = 4;                      // waves 0..3 issue the tile copies
constexpr int NPOLL = FNW - NCOPY;            // waves 4..7 wait on records
constexpr int ROWB = FCS * 2;                 // bytes of one (token, stream) row slice
constexpr int TOKP = FN * ROWB + 16;          // token pitch in LDS (16 B pad)
constexpr int BUFB = FM * TOKP;               // the tile buffer
constexpr int KB1W = FN / 2;                  // k-blocks per wave, full projection (stream pairs)
constexpr int KBAW = FK / 2;                  // k-blocks per wave, active projection (slot pairs)
constexpr int NOB1 = 2;                       // 2N = 32 outputs
constexpr int NOBA = 2;                       // k*Kr + k*k <= 32 outputs
constexpr int NV1 = 34;                       // 32 outputs + sum x + sum x^2
constexpr int NV2 = FN + FK;                  // broadcast per token: H^pre, idx
constexpr int RING = 8;                       // record slots per team
constexpr int kMaxG = 32;
constexpr int NJV = FN + 2;                   // values per reducer job and member (at most)
constexpr int BREC = (2 * FM * NJV + NPOLL * kWave - 1) / (NPOLL * kWave);   // reducer records per polling lane
constexpr int CREC = (FM * NV2 + NPOLL * kWave - 1) / (NPOLL * kWave);       // H^pre / idx records per polling lane
constexpr unsigned kSpinLimit = 1u << 16;     // polls of one record before the wait gives up

static_assert(FM * FN / 4 % NCOPY == 0, "tile copies must split evenly over the copy waves");
// with one reducer wave the other three polling waves take all records
static_assert(BREC * (NPOLL - 1) * kWave >= 2 * FM * NJV && CREC * (NPOLL - 1) * kWave >= FM * NV2,
              "three polling waves cover the records");
static_assert(FCS == 16 * FNW, "a wave holds 16 channels of the slice");

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
  float* saved;           // per-token values for the backward (or null), nsave floats per token
  int nsave;
  uint64_t* rec1;         // [teams][RING][G][FM][NV1]
  uint64_t* rec2;         // [teams][RING][FM][NV2]
  int* err;
  float* part2;           // [G][NV1][T] active partials
  int64_t T;
  int C;
  int teams;
  int m;
  float eps;
  int softmax;            // softmax router (ablation) instead of sigma
};

struct Smem {
  float red[FNW][NV1][FM];            // per-wave projection partials (A)
  float red2[FNW][NV1][FM];           // per-wave active partials
  float vals[2 * FM][NJV];            // reducer partials: [job jj * G + member g][value]
  // H^pre of the tile being read with the streams ordered by parity ([t][8 par
  // + r] = stream 2 r + par), then idx (as bits) of the 4 slots
  float hpid[FM][NV2];
  int poff[BREC][NPOLL * kWave];      // reducer record r of polling lane pl: offset in the slot, -1 unused
};

__device__ __forceinline__ void st_rec(uint64_t* p, float v, uint32_t tag) {
  __hip_atomic_store(p, ((uint64_t)tag << 32) | __float_as_uint(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait until every wanted record carries its tag: records 0..R1-1
// tag1, records R1.. tag2 (all loads of a round in flight together).  A wait
// that gives up counts in *err, and once *err is set every later wait gives
// up within a few polls, so a failed run still drains quickly.
template <int R1, int R2>
__device__ __forceinline__ void ld_recs2t(const uint64_t* const (&p)[R1 + R2], const bool (&want)[R1 + R2],
                                          uint32_t tag1, uint32_t tag2, int* err, float (&out)[R1 + R2]) {
  constexpr int R = R1 + R2;
  bool need[R];
#pragma unroll
  for (int r = 0; r < R; ++r) need[r] = want[r];
  unsigned n = 0;
  while (true) {
    uint64_t v[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
      v[r] = need[r] ? __hip_atomic_load(const_cast<uint64_t*>(p[r]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                     : 0;
    bool any = false;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (need[r] && (uint32_t)(v[r] >> 32) == (r < R1 ? tag1 : tag2)) {
        out[r] = __uint_as_float((uint32_t)v[r]);
        need[r] = false;
      }
      any = any || need[r];
    }
    if (!__any(any)) return;
    ++n;
    if (n > kSpinLimit ||
        ((n & 255) == 0 && __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0)) {
      __hip_atomic_fetch_add(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// v of lane l ^ 32 (v_permlane32_swap with v in both operands leaves the low
// half in the low lanes of the first result and the high half in the second)
__device__ __forceinline__ uint32_t from_lane_xor32(uint32_t v, int lane) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return lane < 32 ? r[1] : r[0];
}
__device__ __forceinline__ float from_lane_xor32f(float v, int lane) {
  return __uint_as_float(from_lane_xor32(__float_as_uint(v), lane));
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// 16-byte LDS read the compiler does not see as a read of the copy buffer, so
// it adds no wait for the wave's outstanding loads (the copy has landed: its
// waves waited for it before the barrier).  The caller waits for lgkmcnt.
__device__ __forceinline__ u32x4 lds_read16_raw(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}

// v plus its value in lane l ^ 16 / l ^ 32 (gfx950 permlane swaps; the two
// halves are added in the same order in every lane, so partners agree bitwise)
__device__ __forceinline__ float add_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float add_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// sum of v over aligned groups of g lanes (g a power of two up to 32), in
// every lane of the group: DPP pairs and quads, then half-row and row mirrors
// (the values are uniform within the smaller groups by then), then row pairs
__device__ __forceinline__ float group_sum(float v, int g) {
  if (g > 1) v = dpp_add(v, 0);
  if (g > 2) v = dpp_add(v, 1);
  if (g > 4) v = dpp_add(v, 2);
  if (g > 8) v = dpp_add(v, 3);
  if (g > 16) v = add_xor16(v);
  return v;
}

// This lane's index, opaque to the optimiser: predicates on it are then
// formed where they are used instead of being hoisted out of the step loop as
// per-lane masks (which live in scalar registers and spill).
__device__ __forceinline__ int lane_id_here() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// v of lane (l - r) mod 16 of this lane's 16-lane row (DPP row rotation; r
// is a constant once the caller's loop is unrolled)
__device__ __forceinline__ int32_t row_ror(int32_t v, int r) {
  switch (r) {
    case 1: return __builtin_amdgcn_update_dpp(0, v, 0x121, 0xF, 0xF, false);
    case 2: return __builtin_amdgcn_update_dpp(0, v, 0x122, 0xF, 0xF, false);
    case 3: return __builtin_amdgcn_update_dpp(0, v, 0x123, 0xF, 0xF, false);
    case 4: return __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false);
    case 5: return __builtin_amdgcn_update_dpp(0, v, 0x125, 0xF, 0xF, false);
    case 6: return __builtin_amdgcn_update_dpp(0, v, 0x126, 0xF, 0xF, false);
    case 7: return __builtin_amdgcn_update_dpp(0, v, 0x127, 0xF, 0xF, false);
    case 8: return __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);
    case 9: return __builtin_amdgcn_update_dpp(0, v, 0x129, 0xF, 0xF, false);
    case 10: return __builtin_amdgcn_update_dpp(0, v, 0x12A, 0xF, 0xF, false);
    case 11: return __builtin_amdgcn_update_dpp(0, v, 0x12B, 0xF, 0xF, false);
    case 12: return __builtin_amdgcn_update_dpp(0, v, 0x12C, 0xF, 0xF, false);
    case 13: return __builtin_amdgcn_update_dpp(0, v, 0x12D, 0xF, 0xF, false);
    case 14: return __builtin_amdgcn_update_dpp(0, v, 0x12E, 0xF, 0xF, false);
    default: return __builtin_amdgcn_update_dpp(0, v, 0x12F, 0xF, 0xF, false);
  }
}

// value of v in lane i (compile-time lane: a scalar read, no LDS crossbar)
__device__ __forceinline__ float lane_value(float v, int i) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), i));
}
template <int G>
__global__ __launch_bounds__(FNT, 1) void k_pre_fused(FusedArgs a) {
  extern __shared__ unsigned char tbuf[];   // [BUFB]; dynamic, as the LDS copy needs it
  __shared__ Smem sm;
  __shared__ uint4 wal[KBAW][NOBA][FNW][kWave];
  __shared__ uint4 stage[FNW][FM][FK][2];   // routed rows of a tile per wave: [token][slot][channel half]
  // wave index made visibly uniform: branches on it are scalar and values
  // derived from it stay in scalar registers
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid % kWave;
  const int tl = lane % 16, grp = lane / 16;
  const int par = grp >> 1, half = grp & 1;   // stream parity and channel half of this lane
  const int team = blockIdx.x / G, s = blockIdx.x % G;
  if (team >= a.teams) return;
  const int C = a.C;
  const int T = (int)a.T;   // the launcher keeps T G NV1 below 2^31
  const int ntiles = (T + FM - 1) / FM;
  int nq = 0;
  if (team < ntiles) nq = (ntiles - team + a.teams - 1) / a.teams;
  if (nq == 0) return;   // the same for every member of the team

  // ---- weight slices in registers for the whole kernel.  This lane's MFMA
  // operand rows are channels s*128 + 16 wave + 8 half + e of stream (slot)
  // 2r + par: in the grouped layout that is lane 16 (wave / 2) + tl of
  // fragment 4 ((i C) / 128 + s) + 2 (wave % 2) + half.
  const int u4 = 2 * (wave % 2) + half, gl = (wave / 2) * 16 + tl;
  uint4 wf[KB1W][NOB1];
#pragma unroll
  for (int r = 0; r < KB1W; ++r) {
    const int64_t kb = (((int64_t)(2 * r + par) * C) / 128 + s) * 4 + u4;
#pragma unroll
    for (int ob = 0; ob < NOB1; ++ob) wf[r][ob] = a.wfull[(kb * NOB1 + ob) * kWave + gl];
  }
  // the active-row weights are used once per tile: they wait in LDS (32 KiB),
  // one 16-byte fragment per lane, [k-block][out block][wave][lane]
#pragma unroll
  for (int r = 0; r < KBAW; ++r) {
    const int64_t kb = (((int64_t)(2 * r + par) * C) / 128 + s) * 4 + u4;
#pragma unroll
    for (int ob = 0; ob < NOBA; ++ob) wal[r][ob][wave][lane] = a.wact[(kb * NOBA + ob) * kWave + gl];
  }
  // per-lane constants of the reducers (lane i < 16: output i)
  const float cs_l = a.colsum[tl], bpre_l = a.b_pre[tl], alpha_pre = a.alpha[0];

  // This member's reducer jobs of a tile are j = s + jj G (jj = 0, 1, ...;
  // token j / 2, half j % 2), run by waves NCOPY .. NCOPY + nred - 1.  The
  // records are polled by waves pw0 .. 7: all of 4 .. 7, or 5 .. 7 when wave
  // 4 is the only reducer (its step is the longest).
  const int njobs = (2 * FM - s + G - 1) / G;
  const int nred = njobs < NPOLL ? njobs : NPOLL;
  const int pw0 = nred == 1 ? NCOPY + 1 : NCOPY;
  const int pstride = (FNW - pw0) * kWave;          // polling lanes
  const bool poller = wave >= pw0;
  // offsets of this member's reducer records, per polling lane (the same for
  // every tile): flat record u = jj G + g, value vi -> sm.vals[u]
  if (poller) {
    const int pl = (wave - pw0) * kWave + lane;
#pragma unroll
    for (int r = 0; r < BREC; ++r) {
      const int u = pl + r * pstride;
      const int jg = u / NJV, vi = u % NJV, jj = jg / G, g = jg % G;
      const int j = s + jj * G;
      const int o = vi < FN ? (j % 2 == 0 ? vi : FN + vi) : (j % 2 == 0 ? 32 + (vi - FN) : (vi == FN ? 33 : -1));
      sm.poff[r][pl] = (jg < 2 * FM && jj * G + s < 2 * FM && o >= 0) ? (g * FM + j / 2) * NV1 + o : -1;
    }
  }

  // ---- tile copy by the copy waves: 64 wave instructions of 1 KiB (4 streams
  // of one token), instruction n -> token n / 4, streams 4 (n % 4) .. + 3;
  // lane -> stream + lane / 16, bytes (lane % 16) * 16 of the row slice
  const uint32_t tbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)tbuf;
  const uint16_t* xlane = a.X + s * FCS + (lane % 16) * 8;   // this lane's 16 bytes of a row slice
  auto copy_tile = [&](int tile) {
    for (int n = wave; n < FM * FN / 4; n += NCOPY) {
      const int t = n / 4, i = (n % 4) * 4 + lane / 16;
      int tg = tile * FM + t;
      if (tg >= T) tg = T - 1;   // in bounds; the token's results are dropped
      const uint16_t* src = xlane + (int64_t)(tg * FN + i) * C;
      lds_dma16(src, __builtin_amdgcn_readfirstlane(tbase + t * TOKP + (n % 4) * 4 * ROWB));
    }
  };
  // every load of the set-up has landed before the pipeline starts: a load
  // left pending until its first use inside the loop (the last weight
  // fragments, the reducers' constants) makes the compiler wait there for all
  // memory operations in flight, tile copies included, in every step
  __builtin_amdgcn_s_waitcnt(0);
  if (wave < NCOPY) copy_tile(team);

  // 1 / (N C): N C = 2048 G is a power of two, so multiplying by it is exact
  const float inv_nc = 1.0f / ((float)FN * (float)C);
  const int coff = s * FCS + 16 * wave + 8 * half;   // first channel of this lane's 8
  uint64_t* const rec1t = a.rec1 + (size_t)team * RING * G * FM * NV1;   // this team's record slots
  uint64_t* const rec2t = a.rec2 + (size_t)team * RING * FM * NV2;

  // ---- reducers.  Their member partials are polled by the polling waves
  // together: flat record u -> job jj and member g (jj G + g = u / NJV), value
  // vi = u % NJV.
  // finish job jj of tile qt from sm.vals (one wave)
  auto finish_job = [&](int qt, int jj) {
    const int lane = lane_id_here();
    const int j = s + jj * G, t = j / 2, h = j % 2;
    const int nv = h == 0 ? FN + 2 : FN + 1;
    const uint32_t tag = (uint32_t)(qt + 1);
    // sums over the G members in a fixed order: lane l adds output l % 16 of
    // its share of the members (ascending), then a butterfly over the four
    // lane groups; the moments (values 16, 17) are one per lane (member l % G,
    // moment l / G) and a butterfly over G lanes.  Every lane holding a sum
    // holds the same bits.
    const float* vrow = &sm.vals[jj * G][0];
    const int per = G >= 4 ? G / 4 : 1, mg = lane >> 4;
    // every read is issued before the sum (a read of an unused member goes
    // to member 0 and is not added), so the LDS latency is paid once
    float vv[kMaxG / 4];
#pragma unroll
    for (int e = 0; e < kMaxG / 4; ++e) {
      const int g = mg * per + e;
      vv[e] = vrow[(e < per && g < G ? g : 0) * NJV + (lane & 15)];
    }
    float v = 0.f;
#pragma unroll
    for (int e = 0; e < kMaxG / 4; ++e) {
      const int g = mg * per + e;
      const float sum = v + vv[e];
      v = (e < per && g < G) ? sum : v;
    }
    v = add_xor32(add_xor16(v));
    const int mi = lane / G;
    const float mo = group_sum(mi < nv - FN ? vrow[(lane % G) * NJV + FN + mi] : 0.f, G);
    const int tg = (team + qt * a.teams) * FM + t;
    uint64_t* r2 = rec2t + (qt % RING) * FM * NV2 + t * NV2;
    if (h == 0) {
      const float mu = lane_value(mo, 0) * inv_nc, nu = lane_value(mo, G) * inv_nc;
      const float r_ln = __builtin_amdgcn_rsqf(ln_variance(mu, nu) + a.eps);
      const float z = (v - mu * cs_l) * r_ln;   // lanes 0..15: LayerNorm-corrected router logit
      // rank among the candidates i >= m (total order of logit_key, ties to
      // the lower index; the same order as the multi-kernel route_token)
      const int32_t key = logit_key(z);
      const int rank = route_rank16([&](int r) { return row_ror(key, r); }, key, lane_id_here() & 15, a.m);
      int slot = -1;
      float pv = 1.0f;
      float sc = sigmoidf(z);
      if (a.softmax) {
        // softmax over the 16 logits (lanes 0..15)
        float mx = lane_value(z, 0);
#pragma unroll
        for (int i = 1; i < FN; ++i) mx = fmaxf(mx, lane_value(z, i));
        const float ez = __expf(z - mx);
        float den = 0.f;
#pragma unroll
        for (int i = 0; i < FN; ++i) den += lane_value(ez, i);
        sc = ez / den;
      }
      if (lane < a.m) slot = lane;
      else if (lane < FN && rank < FK - a.m) {
        slot = a.m + rank;
        pv = sc;
      }
      if (a.saved && tg < T) {
        float* sv = a.saved + tg * a.nsave;
        if (lane < FN) sv[lane] = z;
        else if (lane == FN) sv[a.nsave - 4] = mu;
        else if (lane == FN + 1) sv[a.nsave - 3] = nu;
      }
      if (slot >= 0) {
        st_rec(r2 + FN + slot, __int_as_float(lane), tag);
        if (tg < T) {
          a.idx[tg * FK + slot] = lane;
          a.p[tg * FK + slot] = pv;
        }
      }
    } else {
      const float nu = lane_value(mo, 0) * inv_nc;
      const float r_rms = __builtin_amdgcn_rsqf(nu + a.eps);
      if (lane < FN) {
        if (a.saved && tg < T) a.saved[tg * a.nsave + FN + lane] = v * r_rms;
        const float hpre = sigmoidf(alpha_pre * (v * r_rms) + bpre_l);
        st_rec(r2 + lane, hpre, tag);
        if (tg < T) a.Hpre[tg * FN + lane] = hpre;
      }
    }
  };

  // record r of this polling lane: address and whether it is wanted
  auto poll_rec = [&](int q, int r, bool& wanted) -> const uint64_t* {
    const bool hasB = q >= 1 && q - 1 < nq, hasC = q >= 2 && q - 2 < nq;
    const int pl = (wave - pw0) * kWave + lane_id_here();
    if (r < BREC) {
      const uint64_t* r1 = rec1t + ((q - 1 + RING) % RING) * G * FM * NV1;
      const int off = sm.poff[r][pl];
      wanted = hasB && off >= 0;
      return r1 + (wanted ? off : 0);
    }
    const uint64_t* r2 = rec2t + ((q - 2 + RING) % RING) * FM * NV2;
    const int u = pl + (r - BREC) * pstride;
    wanted = hasC && u < FM * NV2;
    return r2 + (wanted ? u : 0);
  };
  // first loads of the records of step qs, issued at the end of step qs - 1
  // (polling waves) and checked after A of step qs
  // (every lane loads, an unwanted record from the slot base, which is in
  // bounds; its value is never used: a register cleared by a plain move while
  // an earlier load into it may be in flight would make the compiler wait for
  // every memory operation of the wave)
  auto issue_polls = [&](int qs, uint64_t (&first)[BREC + CREC]) {
#pragma unroll
    for (int r = 0; r < BREC + CREC; ++r) {
      bool w;
      const uint64_t* pr = poll_rec(qs, r, w);
      first[r] = __hip_atomic_load(const_cast<uint64_t*>(pr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  };
  uint64_t first[BREC + CREC];
#pragma unroll
  for (int r = 0; r < BREC + CREC; ++r) first[r] = 0;

  // ---- pipeline steps: A of tile q (registers XA), B of tile q - 1, C of
  // tile q - 2 (registers XC); the registers rotate at the end of a step
  // active partials of tile qc (the C phase of a step, left in red2) summed
  // over the waves into part2; runs in the next step, after its first barrier.
  // The A partials are published (after S3) by the waves that are neither
  // reducers nor, when there are at most two reducers, their SIMD partners
  // (waves 0 .. nred - 1), so that the SIMDs running a reducer job carry less
  // of the other work.
  const bool reducer = wave >= NCOPY && wave - NCOPY < nred;
  const int nfree = nred <= 2 ? nred : 0;           // partners left out
  const int npub = FNW - nred - nfree;              // publishing waves
  const int pslot = reducer || wave < nfree ? -1 : (wave < NCOPY ? wave - nfree : wave - nred - nfree);
  const int ptid = pslot * kWave + lane_id_here();  // index among the publishing threads
  // The active partials (publish2) are stored by the waves that do not poll
  // (0 .. pw0 - 1), before S3: the reducer wave is idle there.
  auto publish2 = [&](int qc) {
    const int tile = team + qc * a.teams;
    if (poller) return;
    for (int u = tid; u < NV1 * FM; u += pw0 * kWave) {
      const int o = u / FM, t = u % FM;
      const int tg = tile * FM + t;
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < FNW; ++w) v += sm.red2[w][o][t];
      if (tg < T) a.part2[(s * NV1 + o) * T + tg] = v;
    }
  };
  // one pipeline step: A of tile q into XA, B of tile q - 1, C of tile q - 2
  // from XC.  Tile q lives in register set q % 3, so the loop below runs three
  // steps with the roles of the sets permuted and no register moves.
  auto step = [&](const int q, uint4 (&XA)[KB1W], const uint4 (&XC)[KB1W]) __attribute__((always_inline)) {
    const bool hasA = q < nq, hasB = q >= 1 && q - 1 < nq, hasC = q >= 2 && q - 2 < nq;
    if (wave < NCOPY) {
      __builtin_amdgcn_s_waitcnt(0);   // this wave's part of the copy of tile q has landed
    }
    // polling waves check the records of this step after A: the member
    // partials of this member's jobs of tile q - 1 (BREC per lane) and H^pre /
    // idx of tile q - 2 (CREC per lane); their first loads went out at the
    // end of the previous step
    const bool polls = poller && (hasB || hasC);
    lds_barrier();   // S1: tile q in the buffer
    if (hasA) {
      const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)tbuf +
                            tl * TOKP + par * ROWB + (16 * wave + 8 * half) * 2;
      u32x4 xr[KB1W];
#pragma unroll
      for (int r = 0; r < KB1W; ++r) xr[r] = lds_read16_raw(base + 2 * r * ROWB);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int r = 0; r < KB1W; ++r) {
        asm volatile("" : "+v"(xr[r]));   // uses stay after the wait
        XA[r] = make_uint4(xr[r][0], xr[r][1], xr[r][2], xr[r][3]);
      }
    }
    lds_barrier();   // S2: the buffer is free
    if (hasA) {
      if (wave < NCOPY && q + 1 < nq) copy_tile(team + (q + 1) * a.teams);
      // ---- A: partial projection and moments of the slice, all on the matrix
      // cores: sum x is a product with an all-ones A operand (every row of D
      // holds the column sums), sum x^2 the diagonal of the product of the
      // tile with itself (the B fragment read as an A fragment is its
      // transpose)
      f32x4 acc[NOB1], mom1 = {0.f, 0.f, 0.f, 0.f}, mom2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ob = 0; ob < NOB1; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
      const uint4 ones = make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u);
#pragma unroll
      for (int r = 0; r < KB1W; ++r) {
#pragma unroll
        for (int ob = 0; ob < NOB1; ++ob) acc[ob] = mfma_16x16x32(wf[r][ob], XA[r], acc[ob]);
        mom1 = mfma_16x16x32(ones, XA[r], mom1);
        mom2 = mfma_16x16x32(XA[r], XA[r], mom2);
      }
#pragma unroll
      for (int ob = 0; ob < NOB1; ++ob)
#pragma unroll
        for (int v = 0; v < 4; ++v) sm.red[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
      if (grp == 0) sm.red[wave][32][tl] = mom1[0];
      // D[t][t] sits in lane group t / 4, component t % 4
      if (grp == tl / 4) {
        const int v = tl % 4;
        sm.red[wave][33][tl] = v == 0 ? mom2[0] : (v == 1 ? mom2[1] : (v == 2 ? mom2[2] : mom2[3]));
      }
    }
    // red2 of the previous step (its C of tile q - 3), by the non-polling waves
    if (!poller && q >= 3 && q - 3 < nq) publish2(q - 3);
    if (polls) {
      // tags: tile q - 1 for the partials, tile q - 2 for H^pre / idx
      const uint64_t* src[BREC + CREC];
      bool want[BREC + CREC], need[BREC + CREC];
      float val[BREC + CREC];
      bool any = false;
#pragma unroll
      for (int r = 0; r < BREC + CREC; ++r) {
        src[r] = poll_rec(q, r, want[r]);
        const uint32_t tag = r < BREC ? (uint32_t)q : (uint32_t)(q - 1);
        need[r] = want[r] && (uint32_t)(first[r] >> 32) != tag;
        val[r] = __uint_as_float((uint32_t)first[r]);
        any = any || need[r];
      }
      if (__any(any)) ld_recs2t<BREC, CREC>(src, need, (uint32_t)q, (uint32_t)(q - 1), a.err, val);
      const int pl = (wave - pw0) * kWave + lane_id_here();
#pragma unroll
      for (int r = 0; r < BREC; ++r)
        if (want[r]) (&sm.vals[0][0])[pl + r * pstride] = val[r];
#pragma unroll
      for (int r = 0; r < CREC; ++r)
        if (want[BREC + r]) {
          const int u = pl + r * pstride, t = u / NV2, e = u % NV2;
          sm.hpid[t][e < FN ? 8 * (e & 1) + (e >> 1) : e] = val[BREC + r];
        }
    }
    lds_barrier();   // S3: A partials, polled records in LDS
    // the reducer waves (4 .. 4 + min(njobs, 4) - 1) finish their jobs of tile
    // q - 1 while the other waves publish the partials of tile q
    if (hasB && reducer)
      for (int jj = wave - NCOPY; jj < njobs; jj += NPOLL) finish_job(q - 1, jj);
    if (hasA && pslot >= 0) {
      uint64_t* r1 = rec1t + (q % RING) * G * FM * NV1;
      for (int u = ptid; u < NV1 * FM; u += npub * kWave) {
        const int o = u / FM, t = u % FM;
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < FNW; ++w) v += sm.red[w][o][t];
        st_rec(r1 + (s * FM + t) * NV1 + o, v, (uint32_t)(q + 1));
      }
    }
    if (hasC) {
      const int tg = (team + (q - 2) * a.teams) * FM + tl;
      // ---- dense read of the lane's 8 channels: its 8 streams, then the
      // other parity from lane ^ 32
      {
        float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        const float4 h0 = *reinterpret_cast<const float4*>(&sm.hpid[tl][8 * par]);
        const float4 h1 = *reinterpret_cast<const float4*>(&sm.hpid[tl][8 * par + 4]);
        const float hvs[KB1W] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
        for (int r = 0; r < KB1W; ++r) {
          const float hv = hvs[r];   // H^pre of stream 2 r + par
          float f[8];
          unpack8(XC[r], f);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[e] = fmaf(hv, f[e], acc[e]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += from_lane_xor32f(acc[e], lane);
        if (par == 0 && tg < T) *reinterpret_cast<uint4*>(a.input + (int64_t)tg * C + coff) = pack8(acc);
      }
      // ---- active rows: each lane stores those of its 8 streams that are
      // routed into the wave's staging area at their slot, then reads back the
      // slot pair it feeds to the MFMA (slot 2r + par).  A wave's LDS accesses
      // complete in order, so no barrier is needed.
      {
        uint32_t mask = 0, codes = 0;   // routed streams; 2-bit slot of each stream
#pragma unroll
        for (int j = 0; j < FK; ++j) {
          const int id = __float_as_int(sm.hpid[tl][FN + j]) & (FN - 1);   // always a row of the tile
          mask |= 1u << id;
          codes |= (uint32_t)j << (2 * id);
        }
        mask >>= par;
        codes >>= 2 * par;
#pragma unroll
        for (int r = 0; r < KB1W; ++r)   // stream 2r + par
          if ((mask >> (2 * r)) & 1u) stage[wave][tl][(codes >> (4 * r)) & 3u][half] = XC[r];
        f32x4 acc[NOBA], mom2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ob = 0; ob < NOBA; ++ob) acc[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int r = 0; r < KBAW; ++r) {
          const uint4 xa = stage[wave][tl][2 * r + par][half];
#pragma unroll
          for (int ob = 0; ob < NOBA; ++ob) acc[ob] = mfma_16x16x32(wal[r][ob][wave][lane], xa, acc[ob]);
          mom2 = mfma_16x16x32(xa, xa, mom2);   // diagonal: sum a^2 per token
        }
#pragma unroll
        for (int ob = 0; ob < NOBA; ++ob)
#pragma unroll
          for (int v = 0; v < 4; ++v) sm.red2[wave][ob * 16 + grp * 4 + v][tl] = acc[ob][v];
        if (grp == 0) sm.red2[wave][32][tl] = 0.f;
        if (grp == tl / 4) {
          const int v = tl % 4;
          sm.red2[wave][33][tl] = v == 0 ? mom2[0] : (v == 1 ? mom2[1] : (v == 2 ? mom2[2] : mom2[3]));
        }
      }
    }
    if (poller) issue_polls(q + 1, first);
  };
  uint4 X0[KB1W], X1[KB1W], X2[KB1W];
  for (int q = 0; q < nq + 2; q += 3) {
    step(q, X0, X1);
    if (q + 1 < nq + 2) step(q + 1, X1, X2);
    if (q + 2 < nq + 2) step(q + 2, X2, X0);
  }
  lds_barrier();   // red2 of the last C phase (tile nq - 1)
  publish2(nq - 1);
}

// zero n1 and n2 16-byte words at p1 and p2 (one launch)
__global__ void k_zero2(uint4* __restrict__ p1, int64_t n1, uint4* __restrict__ p2, int64_t n2) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint4 z = make_uint4(0, 0, 0, 0);
  if (i < n1) p1[i] = z;
  else if (i - n1 < n2) p2[i - n1] = z;
}

struct DeviceInfo {
  int cus = 0;
  int per_cu = 0;
};

constexpr size_t kTileLds = (size_t)BUFB;

// the kernel instance of a team size (G = C / 128, a power of two up to 32)
const void* fused_kernel(int G) {
  switch (G) {
    case 1: return reinterpret_cast<const void*>(k_pre_fused<1>);
    case 2: return reinterpret_cast<const void*>(k_pre_fused<2>);
    case 4: return reinterpret_cast<const void*>(k_pre_fused<4>);
    case 8: return reinterpret_cast<const void*>(k_pre_fused<8>);
    case 16: return reinterpret_cast<const void*>(k_pre_fused<16>);
    case 32: return reinterpret_cast<const void*>(k_pre_fused<32>);
    default: return nullptr;
  }
}

// CU count and resident workgroups per CU of every instance (all instances
// have the same launch shape and LDS); the dynamic LDS limit is raised once
// per device
DeviceInfo device_info() {
  static thread_local int dev_cached = -1;
  static thread_local DeviceInfo info;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DeviceInfo{};
  if (dev != dev_cached) {
    DeviceInfo di;
    if (hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return DeviceInfo{};
    di.per_cu = 1 << 30;
    for (int G = 1; G <= kMaxG; G *= 2) {
      const void* f = fused_kernel(G);
      int per = 0;
      if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kTileLds) != hipSuccess)
        return DeviceInfo{};
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, f, FNT, kTileLds) != hipSuccess) return DeviceInfo{};
      if (per < di.per_cu) di.per_cu = per;
    }
    info = di;
    dev_cached = dev;
  }
  return info;
}

}  // namespace

bool fused_pre_supported(const xhc_dims* d) {
  return d->state_dtype == XHC_BF16 && d->N == FN && d->k == FK && d->Kr >= 1 &&
         FK * d->Kr + FK * FK <= 16 * NOBA && d->C % FCS == 0 && d->C / FCS <= kMaxG &&
         kMaxG % (d->C / FCS) == 0 &&   // every member takes 32 / G reducer jobs per tile
         d->T * (d->C / FCS) * NV1 < ((int64_t)1 << 31);   // 32-bit token and partial indices
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
                            float* Hpost, float* saved, void* ws, hipStream_t s) {
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
  a.saved = saved;
  a.nsave = saved_floats(FN, FK, d->Kr);
  a.err = reinterpret_cast<int*>(w);
  a.rec1 = reinterpret_cast<uint64_t*>(w + 256);
  a.rec2 = reinterpret_cast<uint64_t*>(w + 256 + align256(rec1_words(G) * 8));
  a.part2 = reinterpret_cast<float*>(w + 256 + align256(rec1_words(G) * 8) + align256(rec2_words(G) * 8));
  float* sums = a.part2 + align256((size_t)G * NV1 * d->T * sizeof(float)) / sizeof(float);
  a.T = d->T;
  a.C = d->C;
  a.teams = teams;
  a.m = d->m;
  a.eps = d->eps;
  a.softmax = d->router == XHC_ROUTER_SOFTMAX ? 1 : 0;
  // records start untagged: clear the error counter (with the first 256
  // bytes) and the record slots in use, both whole 16-byte words
  const size_t used1 = (size_t)teams * RING * G * FM * NV1, used2 = (size_t)teams * RING * FM * NV2;
  const int64_t n1 = (int64_t)((256 + used1 * 8) / 16), n2 = (int64_t)((used2 * 8 + 15) / 16);
  k_zero2<<<dim3((unsigned)((n1 + n2 + 255) / 256)), dim3(256), 0, s>>>(reinterpret_cast<uint4*>(w), n1,
                                                                        reinterpret_cast<uint4*>(a.rec2), n2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  void* args[] = {&a};
  e = hipLaunchCooperativeKernel(fused_kernel(G), dim3(teams * G), dim3(FNT), args,
                                 kTileLds, s);
  if (e != hipSuccess) return e;
  // active partials -> H^post, H^res (Sinkhorn + clamp)
  return launch_pre_coef(a.part2, G, (int64_t)FK * d->Kr + FK * FK, d->T, FK, d->Kr, 1, d->C, alpha + 2, alpha + 1,
                         b_post, b_res, d->eps, d->sinkhorn_iters, d->clamp_delta, Hpost, Hres, sums, saved, a.nsave,
                         2 * FN, a.nsave - 2, s, a.err);
}

}  // namespace xhc

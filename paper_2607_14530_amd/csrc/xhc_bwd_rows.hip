// Row passes of the pre-map reverse with their inputs staged through an LDS
// ring: dX over the rows of a state and the weight gradients of a projection
// read from those rows.  Three uses:
//  * the full rows of one pre-map (a full xHC sublayer): router and pre-map
//    outputs, one input gradient;
//  * the full rows of an xHC-Flash group's entry state: the router and the
//    Q pre-maps read from it, Q input gradients;
//  * the active rows of a Flash sublayer (the k-row state a^(q-1), slot j =
//    row j, fp32 gradient rows): H^post and H^res outputs, and the read of
//    d input_q by the active streams when that sublayer has one.
//
// Per token t and weight row K = (row i, channel c), with dz' the per-token
// scaled logit gradients of the outputs o and the LayerNorm / RMS statistics
// of the forward (eq:fused_normalized_projection reversed; the dense reads of
// eq:dense_read, and eq:app_active_state_correction for the active rows, give
// the H^pre terms):
//   dX[t, K] += sum_q H^pre,q_i[t] d input_q[t, c] + sum_o W[K, o] dz'[t, o]
//               - beta x[t, K] - r_ln m1 - r_ln^2 (x[t, K] - mu) m2
//   dW[K, o] += sum_t x[t, K] dz'[t, o]
// (full rows: beta the sum of the pre-maps' beta_pre, and the router's own mean
// term of dW_r is added by the reduction; active rows: beta = beta_a, r_ln = 0).
//
// A workgroup (512 threads, 8 waves) takes 128 weight rows (128 channels of
// one row) and a chunk of tokens, in steps of 32 tokens.  Every input of a
// step (state rows, gradient rows, the input gradients, packed dz' rows and
// transposes, per-token scalars, H^pre weights) is copied global -> LDS with
// direct loads into a ring of NS stages, NS - 1 steps ahead, so a step's
// loads are in flight while the steps before it compute; each wave waits
// only for its own copies (an s_waitcnt count fixed by the order of its
// copies and stores), then the workgroup meets at a barrier that waits for
// LDS traffic only.  The MFMA products (D[16 rows x 16 tokens] for dX,
// D[16 outputs x 16 rows] for dW, bf16 hi + lo pairs of dz') read the stage;
// the dX product goes through LDS to a per-token layout, where each thread
// forms 8 consecutive outputs and writes them with 16-byte stores (a wave
// writes whole rows of contiguous bytes).  The 16-byte pieces of the staged
// arrays read by 16 lanes in 16 consecutive rows are XOR-swizzled (the copy
// lane picks its global piece accordingly), so such reads meet 16 different
// bank groups.
#include "xhc_device.h"
#include "xhc_launch.h"

namespace xhc {
namespace {

constexpr int RT = 32;             // tokens per step
constexpr int RR = 128;            // weight rows per workgroup (channels of one row)
constexpr int RNT = 512;           // threads per workgroup
constexpr int RNW = RNT / kWave;   // waves; wave w takes rows 16 w .. 16 w + 15
constexpr int ACCP = RR + 4;       // fp32 pitch of the staged dX product

// slot of 16-byte piece p of row u of a staged array with RP pieces a row:
// p ^ row_swz(u).  The same piece of 16 consecutive rows then falls in 16
// different 16-byte groups of a 256-byte bank line.
template <int RP>
__device__ __forceinline__ int row_swz(int u) {
  static_assert(RP % 4 == 0, "rows of whole four-piece groups");
  constexpr int s = RP % 16 == 0 ? 4 : (RP % 8 == 0 ? 3 : 2);
  return (u >> (4 - s)) & ((1 << s) - 1);
}
// state rows (16 pieces of 8 channels): the column read of the dW operand
// takes tokens 8 g + e (g = 0..3) of two neighbouring pieces
__device__ __forceinline__ int x_swz(int u) { return ((u >> 3) & 3) << 1; }

template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}
// wait until at most (LA - 1) CW + k S of this wave's memory operations are
// in flight (k = K .. LA, a value the same in every lane)
template <int LA, int CW, int S, int K>
__device__ __forceinline__ void wait_ring(int k) {
  if constexpr (K >= LA) {
    vm_wait<(LA - 1) * CW + LA * S>();
  } else {
    if (k == K) vm_wait<(LA - 1) * CW + K * S>();
    else wait_ring<LA, CW, S, K + 1>(k);
  }
}

// byte layout of one ring stage: NQ input gradients, GB bytes per gradient
// element, NOR real dz' outputs (a multiple of 16) of the NOP in the packed rows
template <int NQ, int NOR, int GB>
struct RingStage {
  static constexpr int RP = NOR / 4;                 // pieces of a staged dz' row: NOR / 8 hi, NOR / 8 lo
  static constexpr int TILE = RT * RR * 2;           // [32 tokens][128 channels] bf16
  static constexpr int GTILE = RT * RR * GB;         // the gradient rows
  static constexpr int XO = 0;                       // state rows (swizzled)
  static constexpr int GO = XO + TILE;               // gradient rows as read
  static constexpr int DO = GO + GTILE;              // input gradients, NQ tiles
  static constexpr int ZRO = DO + NQ * TILE;         // dz' token rows [32][RP pieces] (swizzled)
  static constexpr int ZTO = ZRO + RT * RP * 16;     // dz' transposes [2 NOR rows][4 pieces of 8 tokens] (swizzled)
  static constexpr int SRO = ZTO + 2 * NOR * RT * 2; // scalars [32][8] floats: r_ln, mu, m1, m2, beta
  static constexpr int HPO = SRO + RT * 8 * 4;       // H^pre weights [2 NHP][32] floats
  static constexpr int NHP = (NQ + 1) / 2;
  static constexpr int BYTES = HPO + NHP * 256;
  // copies (wave instructions: 1 KiB, the H^pre ones 256 B), in this order
  static constexpr int NT = TILE / 1024, NG = GTILE / 1024;
  static constexpr int NZR = RT * RP * 16 / 1024;
  static constexpr int NZT = 2 * NOR * RT * 2 / 1024;
  static constexpr int C_G = NT, C_D = C_G + NG, C_ZR = C_D + NQ * NT, C_ZT = C_ZR + NZR, C_SR = C_ZT + NZT;
  static constexpr int C_HP = C_SR + 1, NCOPY = C_HP + NHP;
};

struct RingArgs {
  RowRingDesc d;
  int64_t NK;   // weight rows
};

template <int NQ, int NOP, int NOR, int NS, typename TD>
__global__ __launch_bounds__(RNT, 1) void k_bwd_rows_ring(RingArgs ra) {
  constexpr int GB = (int)sizeof(TD);
  using L = RingStage<NQ, NOR, GB>;
  constexpr int LA = NS - 1;                                  // steps loaded ahead
  constexpr int NKB = NOP / 32, NOH = NOR / 16;
  constexpr int S = GB / 2;                                   // 16-byte stores of a thread per step
  constexpr int PPT = RR * GB / 16;                           // 16-byte pieces of a gradient row
  constexpr int C0 = L::NCOPY / RNW, CX = L::NCOPY % RNW;   // copies per wave and stage: C0, C0 + 1 below wave CX
  static_assert(NOP % 32 == 0 && NOR % 16 == 0 && NOR <= NOP && NQ <= kRowRingMaxQ, "output blocks");
  static_assert(LA >= 1 && LA <= 3, "one to three steps ahead");
  static_assert(RT * RR * 2 / 16 == RNT, "one 8-channel piece of the dX tile per thread");
  extern __shared__ __align__(16) unsigned char ring[];
  const RowRingDesc& a = ra.d;
  const int tid = threadIdx.x, lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int l16 = lane % 16, g4 = lane / 16;
  const int64_t T = a.T;
  const int N = a.N, C = a.C;
  const int64_t K0 = (int64_t)blockIdx.x * RR;
  const int part = (int)(K0 / C), c0 = (int)(K0 % C);
  const int64_t t0 = (int64_t)blockIdx.y * a.tchunk;
  const int64_t t1 = t0 + a.tchunk < T ? t0 + a.tchunk : T;
  const int nsteps = (int)((t1 - t0 + RT - 1) / RT);
  const uint32_t lbase = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)ring;
  float* const accb = reinterpret_cast<float*>(ring + NS * L::BYTES);   // [32][ACCP]
  const uint16_t* const Xs = reinterpret_cast<const uint16_t*>(a.X);
  TD* const dX = reinterpret_cast<TD*>(a.dX);

  // dX-product A operand: rows K0 + 16 wave + l16, outputs 32 kb + 8 g4 + e,
  // as bf16 (output o of weight block b: columns win[0] + .. + win[b - 1] on)
  uint4 wfrag[NKB];
  {
    // every weight is loaded before any is converted (a conversion next to
    // its load would wait for it); an unused output reads column 0 of its
    // block, in bounds, and is zeroed
    const int64_t K = K0 + 16 * wave + l16;
    float r[NKB][8];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        int o = 32 * kb + 8 * g4 + e;
        const bool used = o < a.nout;
        const float* wp = a.w[0];
        int wd = a.win[0];
#pragma unroll
        for (int bb = 1; bb < kRowRingMaxQ + 1; ++bb)
          if (bb < a.nwin && o >= wd) {
            o -= wd;
            wp = a.w[bb];
            wd = a.win[bb];
          }
        r[kb][e] = wp[K * wd + (used ? o : 0)];
      }
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      float f[8];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        f[e] = 32 * kb + 8 * g4 + e < a.nout ? __uint_as_float(f2bf(r[kb][e]) << 16) : 0.f;
      wfrag[kb] = pack8(f);
    }
  }
  f32x4 dw[NOH];
#pragma unroll
  for (int ob = 0; ob < NOH; ++ob) dw[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  // the set-up loads have landed: inside the loop only the ring copies and
  // the dX stores are in flight, in the order the waits below count
  __builtin_amdgcn_s_waitcnt(0);

  const int64_t Tp = (T + RT - 1) / RT * RT;
  const uint16_t* const dzrows = a.dzp;
  const uint16_t* const dztr = a.dzp + Tp * 2 * NOP;
  // tokens past the chunk read its last token (their results are dropped)
  auto tok = [&](int64_t t) -> int64_t { return t < t1 ? t : t1 - 1; };
  // copy i (the same in every lane) of the stage of tokens tb .. tb + 31
  auto copy = [&](int i, int64_t tb, uint32_t sb) {
    if (i < L::C_G) {
      // state rows: 4 tokens of 256 B a copy
      const int u = 4 * i + lane / 16, sl = lane % 16;
      lds_dma16(Xs + (tok(tb + u) * N + part) * (int64_t)C + c0 + 8 * (sl ^ x_swz(u)), sb + L::XO + i * 1024);
    } else if (i < L::C_D) {
      // gradient rows: 1024 / (RR GB) tokens a copy
      const int j = i - L::C_G, u = j * (kWave / PPT) + lane / PPT, sl = lane % PPT;
      lds_dma16(dX + (tok(tb + u) * N + part) * (int64_t)C + c0 + sl * (16 / GB), sb + L::GO + j * 1024);
    } else if (i < L::C_ZR) {
      // input gradients: 4 tokens of 256 B a copy
      const int j = i - L::C_D, q = j / L::NT, jj = j % L::NT;
      const int u = 4 * jj + lane / 16, sl = lane % 16;
      const uint16_t* din = reinterpret_cast<const uint16_t*>(a.din[0]);
#pragma unroll
      for (int qq = 1; qq < NQ; ++qq)
        if (q == qq) din = reinterpret_cast<const uint16_t*>(a.din[qq]);
      lds_dma16(din + tok(tb + u) * C + c0 + 8 * sl, sb + L::DO + j * 1024);
    } else if (i < L::C_ZT) {
      // dz' token rows: RP pieces a token (hi outputs, then lo)
      const int j = i - L::C_ZR, f = j * kWave + lane;
      const int u = f / L::RP, p = (f % L::RP) ^ row_swz<L::RP>(u);
      const int off = p < NOR / 8 ? 8 * p : NOP + 8 * (p - NOR / 8);
      lds_dma16(dzrows + tok(tb + u) * 2 * NOP + off, sb + L::ZRO + j * 1024);
    } else if (i < L::C_SR) {
      // dz' transposes: rows (hi outputs 0 .. NOR - 1, then lo) of 4 pieces of 8 tokens
      const int j = i - L::C_ZT, f = j * kWave + lane;
      const int r = f / 4, p = (f % 4) ^ ((r >> 2) & 3);
      const int gr = r < NOR ? r : NOP + (r - NOR);
      lds_dma16(dztr + (tok(tb) / RT) * 2 * NOP * RT + gr * RT + 8 * p, sb + L::ZTO + j * 1024);
    } else if (i < L::C_HP) {
      // scalars: token lane / 2, four of them a lane
      lds_dma16(a.srec + tok(tb + lane / 2) * a.srec_stride + 4 * (lane % 2), sb + L::SRO);
    } else {
      // dense-read weights: weight 2 j + lane / 32 of token lane % 32 (both
      // candidate pointers chosen with uniform tests, then one per lane: a
      // per-lane index into the arguments would become a load)
      const int j = i - L::C_HP;
      const float* h0 = a.hp[0];
      const float* h1 = a.hp[0];
#pragma unroll
      for (int qq = 1; qq < NQ; ++qq) {
        if (2 * j == qq) h0 = a.hp[qq];
        if (2 * j + 1 == qq) h1 = a.hp[qq];
      }
      const float* hp = lane < 32 ? h0 : h1;
      lds_dma4(hp + tok(tb + lane % 32) * a.hp_stride + part, sb + L::HPO + j * 256);
    }
  };
  auto issue = [&](int64_t tb, int slot) {
    const uint32_t sb = lbase + slot * L::BYTES;
#pragma unroll
    for (int i0 = 0; i0 < L::NCOPY; i0 += RNW)
      if (i0 + wave < L::NCOPY) copy(i0 + wave, tb, sb);
  };
  // this wave's copies of step n have landed: after them it issued the
  // copies of the LA - 1 later stages and the stores of min(n, LA) steps
  // (S 16-byte store instructions a step)
  auto wait_stage = [&](int n) {
    const int k = n < LA ? n : LA;
    if (wave < CX) wait_ring<LA, C0 + 1, S, 0>(k);
    else wait_ring<LA, C0, S, 0>(k);
  };

#pragma unroll
  for (int n = 0; n < LA; ++n) issue(t0 + n * RT, n);
  for (int n = 0; n < nsteps; ++n) {
    const int64_t tb = t0 + (int64_t)n * RT;
    const int nt = (int)(t1 - tb < RT ? t1 - tb : RT);
    const unsigned char* const st = ring + (n % NS) * L::BYTES;
    wait_stage(n);
    lds_barrier();   // stage n is in LDS (every wave waited for its own copies)
    // the copies of step n + LA go to the slot of step n - 1, whose reads
    // ended before this barrier (past the chunk they read its last token)
    issue(tb + LA * RT, (n + LA) % NS);
    if (nt < RT) {
      // the chunk's last, partial step: state rows past it are zeroed, so
      // their dW terms vanish (the packed dz' is zero past T as well)
      if (tid / 16 >= nt)
        *reinterpret_cast<uint4*>(ring + (n % NS) * L::BYTES + L::XO + tid * 16) = make_uint4(0, 0, 0, 0);
      lds_barrier();
    }
    // ---- dX product of the two 16-token halves, to the staging buffer
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int u = 16 * h + l16;
      const int sw = row_swz<L::RP>(u);
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        const int p = 4 * kb + g4;   // hi piece of outputs 32 kb + 8 g4 .. + 7
        uint4 bh = make_uint4(0, 0, 0, 0), bl = make_uint4(0, 0, 0, 0);
        if (4 * kb + 4 <= NOR / 8 || p < NOR / 8) {
          bh = *reinterpret_cast<const uint4*>(st + L::ZRO + (u * L::RP + (p ^ sw)) * 16);
          bl = *reinterpret_cast<const uint4*>(st + L::ZRO + (u * L::RP + ((NOR / 8 + p) ^ sw)) * 16);
        }
        acc = mfma_16x16x32(wfrag[kb], bh, acc);
        acc = mfma_16x16x32(wfrag[kb], bl, acc);
      }
      // lane holds rows 16 wave + 4 g4 + v of token u
      *reinterpret_cast<float4*>(accb + u * ACCP + 16 * wave + 4 * g4) = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
    // ---- dW: contraction over the 32 staged tokens
    {
      const int kc = 16 * wave + l16, pk = kc / 8, ek = kc % 8;
      uint16_t xb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int u = 8 * g4 + e;
        xb[e] = *reinterpret_cast<const uint16_t*>(st + L::XO + u * (RR * 2) + (pk ^ x_swz(u)) * 16 + ek * 2);
      }
      const uint4 bx = make_uint4(xb[0] | ((uint32_t)xb[1] << 16), xb[2] | ((uint32_t)xb[3] << 16),
                                  xb[4] | ((uint32_t)xb[5] << 16), xb[6] | ((uint32_t)xb[7] << 16));
#pragma unroll
      for (int ob = 0; ob < NOH; ++ob) {
        const int rh = 16 * ob + l16, rl = NOR + rh;
        const uint4 ah = *reinterpret_cast<const uint4*>(st + L::ZTO + (rh * 4 + (g4 ^ ((rh >> 2) & 3))) * 16);
        const uint4 al = *reinterpret_cast<const uint4*>(st + L::ZTO + (rl * 4 + (g4 ^ ((rl >> 2) & 3))) * 16);
        dw[ob] = mfma_16x16x32(ah, bx, dw[ob]);
        dw[ob] = mfma_16x16x32(al, bx, dw[ob]);
      }
    }
    lds_barrier();   // the dX product of every wave is staged
    // ---- outputs: thread -> token tid / 16, channels 8 (tid % 16) .. + 7
    {
      const int u = tid / 16, p = tid % 16;
      if (u < nt) {
        const float4 a0 = *reinterpret_cast<const float4*>(accb + u * ACCP + 8 * p);
        const float4 a1 = *reinterpret_cast<const float4*>(accb + u * ACCP + 8 * p + 4);
        const uint4 xv = *reinterpret_cast<const uint4*>(st + L::XO + u * (RR * 2) + (p ^ x_swz(u)) * 16);
        const float* sr = reinterpret_cast<const float*>(st + L::SRO) + u * 8;
        const float r_ln = sr[0], mu = sr[1], m1 = sr[2], m2 = sr[3], beta = sr[4];
        const float* hpw = reinterpret_cast<const float*>(st + L::HPO);
        float x[8], g[8], rd[8];
        unpack8(xv, x);
        if (GB == 2) {
          unpack8(*reinterpret_cast<const uint4*>(st + L::GO + u * (RR * 2) + p * 16), g);
        } else {
          const float4 g0 = *reinterpret_cast<const float4*>(st + L::GO + u * (RR * 4) + p * 32);
          const float4 g1 = *reinterpret_cast<const float4*>(st + L::GO + u * (RR * 4) + p * 32 + 16);
          g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
          g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) rd[e] = 0.f;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {   // sum_q H^pre,q d input_q, in the order of the maps
          const float hq = hpw[q * RT + u];
          float dq[8];
          unpack8(*reinterpret_cast<const uint4*>(st + L::DO + q * L::TILE + u * (RR * 2) + p * 16), dq);
#pragma unroll
          for (int e = 0; e < 8; ++e) rd[e] = fmaf(hq, dq[e], rd[e]);
        }
        const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        float d[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          d[e] = g[e] + (rd[e] + av[e] - beta * x[e] - r_ln * m1 - r_ln * r_ln * (x[e] - mu) * m2);
        TD* const out = dX + ((tb + u) * N + part) * (int64_t)C + c0 + 8 * p;
        if (GB == 2) {
          *reinterpret_cast<uint4*>(out) = pack8(d);
        } else {
          *reinterpret_cast<float4*>(out) = make_float4(d[0], d[1], d[2], d[3]);
          *reinterpret_cast<float4*>(out + 4) = make_float4(d[4], d[5], d[6], d[7]);
        }
      }
    }
  }
  vm_wait<0>();   // the copies issued past the chunk land before the wave ends
  // lane holds dW[row K0 + 16 wave + l16][output 16 ob + 4 g4 + v]
  const int64_t K = K0 + 16 * wave + l16;
#pragma unroll
  for (int ob = 0; ob < NOH; ++ob) {
    const int o = 16 * ob + 4 * g4;
    if (o < a.nout) {   // four outputs inside one block (wout_w % 4 == 0)
      const int b = o / a.wout_w;
      float* wo = a.wout[0];
#pragma unroll
      for (int bb = 1; bb < kRowRingMaxQ + 1; ++bb)
        if (b == bb) wo = a.wout[bb];
      *reinterpret_cast<float4*>(wo + ((int64_t)blockIdx.y * ra.NK + K) * a.wout_w + o % a.wout_w) =
          make_float4(dw[ob][0], dw[ob][1], dw[ob][2], dw[ob][3]);
    }
  }
}

template <int NQ, int NOP, int NOR, int NS, typename TD>
hipError_t launch_ring(const RingArgs& a, dim3 grid, hipStream_t s) {
  constexpr size_t lds =
      (size_t)NS * RingStage<NQ, NOR, (int)sizeof(TD)>::BYTES + (size_t)RT * ACCP * sizeof(float);
  static_assert(lds <= 160 * 1024, "the ring fits the LDS of a CU");
  const void* fn = reinterpret_cast<const void*>(k_bwd_rows_ring<NQ, NOP, NOR, NS, TD>);
  static thread_local int dev_set = -1;   // the device whose LDS limit was raised
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev != dev_set) {
    e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    dev_set = dev;
  }
  k_bwd_rows_ring<NQ, NOP, NOR, NS, TD><<<grid, dim3(RNT), lds, s>>>(a);
  return hipGetLastError();
}

}  // namespace

bool bwd_rows_ring_supported(int64_t rows, int C, int64_t tchunk) {
  return rows % RR == 0 && C % RR == 0 && tchunk % RT == 0;
}

hipError_t launch_bwd_rows_ring(const RowRingDesc& d, int64_t rows, hipStream_t s) {
  if (!bwd_rows_ring_supported(rows, d.C, d.tchunk) || d.nq < 0 || d.nq > kRowRingMaxQ || d.nwin < 1 ||
      d.nwin > kRowRingMaxQ + 1 || d.wout_w % 4 != 0 || d.T <= 0)
    return hipErrorInvalidValue;
  RingArgs a{};
  a.d = d;
  a.NK = rows;
  const dim3 grid((unsigned)(rows / RR), (unsigned)((d.T + d.tchunk - 1) / d.tchunk));
  // one pre-map: 2N outputs padded to 32 (64 at N = 32); the Flash group's
  // router and Q pre-maps: 16 (Q + 1) outputs; a Flash sublayer's active
  // rows: up to 32 outputs, fp32 gradient rows
  if (!d.dx_f32) {
    if (d.nq == 1 && d.nop == 32 && d.nout <= 32) return launch_ring<1, 32, 32, 4, uint16_t>(a, grid, s);
    if (d.nq == 1 && d.nop == 64 && d.nout <= 64) return launch_ring<1, 64, 64, 3, uint16_t>(a, grid, s);
    if (d.nq == 2 && d.nop == 64 && d.nout == 48) return launch_ring<2, 64, 48, 3, uint16_t>(a, grid, s);
    if (d.nq == 4 && d.nop == 96 && d.nout == 80) return launch_ring<4, 96, 80, 2, uint16_t>(a, grid, s);
  } else if (d.nop == 32 && d.nout <= 32) {
    if (d.nq == 0) return launch_ring<0, 32, 32, 3, float>(a, grid, s);
    if (d.nq == 1) return launch_ring<1, 32, 32, 3, float>(a, grid, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace xhc

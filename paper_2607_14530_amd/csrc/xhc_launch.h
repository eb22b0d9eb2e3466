// Internal launchers of the xHC kernels (host side).  Every launcher enqueues
// on `stream` and returns hipSuccess or the first launch error.  Shapes have
// been validated by the C-ABI layer before any launcher is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "xhc.h"

namespace xhc {

constexpr int kWave = 64;
constexpr int kMaxN = 64;   // streams
constexpr int kMaxK = 8;    // active streams
constexpr int kMaxKr = 4;   // write-back components

// packed projection layout: fragments of 64 lanes x 8 bf16 (1 KiB), indexed
// [k_block (32 rows)][out_block (16 columns)][lane]; lane l of fragment
// (kb, ob) holds W[kb*32 + 8*(l/16) + e][ob*16 + l%16], e = 0..7.  Grouped
// layout (full-state weights of a bf16 state, K % 128 == 0): fragment
// 4G + u holds rows 128G + 32*(l/16) + 8u + e instead, so that a lane's four
// consecutive fragments of a group meet 64 contiguous state bytes.
inline bool full_grouped(int state_dtype, int64_t K) { return state_dtype == XHC_BF16 && K % 128 == 0; }
// the same for the active-state weights (K = k C, gathered rows): groups must
// not straddle two rows
inline bool act_grouped(int state_dtype, int C) { return state_dtype == XHC_BF16 && C % 128 == 0; }
__host__ __device__ inline int64_t out_blocks(int64_t nout) { return (nout + 15) / 16; }
inline size_t packed_frag_bytes(int64_t K, int64_t nout) { return (size_t)(K / 32) * out_blocks(nout) * 1024; }
constexpr size_t kColsumBytes = 64 * sizeof(float);

hipError_t launch_pack(int64_t K, int64_t nout, int ncols_a, const float* A, int ncols_b, const float* B,
                       int64_t b_count, bool grouped, void* packed, hipStream_t s);
hipError_t launch_colsum(int64_t K, int ncols, const float* W, float* out, hipStream_t s);

// ---- pre (multi-kernel path)
constexpr int kProjTile = 16;    // tokens per MFMA column group

// Launch plan of the split-K projection.  Wide path (bf16 state, grouped
// weight layout, full or gathered rows): 256-token workgroups, 4 consecutive
// k-blocks per step, weight fragments shared through LDS.  Other cases: each wave multiplies tg token groups of
// 16 by the same weight fragment.  A workgroup covers chunk_blocks 32-row
// blocks of K; nchunk partials are summed per token afterwards.
struct ProjPlan {
  bool wide;
  int tg;
  int64_t chunk_blocks;
  int64_t nchunk;
};
// token groups of 16 per wave of the wide path: four, or two for five and more
// output blocks (their accumulators would otherwise leave one wave per SIMD)
__host__ __device__ constexpr int wide_tg(int nob) { return nob >= 5 ? 2 : 4; }
__host__ __device__ constexpr int wide_tokens(int nob) { return 64 * wide_tg(nob); }   // per workgroup
constexpr int kWideStep = 4;   // k-blocks per step of the wide path
// steps whose weight fragments (kWideStep x nob KiB each) share one LDS fill;
// two fills alternate: four steps up to four output blocks (at most 128 KiB),
// one step from five blocks on (40 KiB at five, more workgroups per CU;
// measured faster for the router-plus-pre projection of the Flash group)
__host__ __device__ constexpr int wide_seg_steps(int nob) { return nob <= 4 ? 4 : 1; }
inline ProjPlan proj_plan(int state_dtype, bool gather, int64_t K, int C, int64_t nout, int64_t T) {
  const int64_t nblk = K / 32, NO = out_blocks(nout) * 16 + 2;
  const bool wide = (gather ? act_grouped(state_dtype, C) : full_grouped(state_dtype, K)) && out_blocks(nout) <= 8;
  int tg = 4;
  while (tg > 1 && ((T + 16 * tg - 1) / (16 * tg) < 128 || NO * tg > 160)) tg /= 2;
  const int64_t wt = wide_tokens((int)out_blocks(nout));
  const int64_t tiles = wide ? (T + wt - 1) / wt : (T + 16 * tg - 1) / (16 * tg);
  const int64_t gran = 32;                                      // chunk granularity in k-blocks
  // chunks for about 1024 workgroups, 512 for five or more output blocks and
  // 256 for the gathered active rows (longer chunks, fewer weight fills and
  // pipeline starts per byte: measured faster there)
  int64_t want = ((gather ? 256 : (out_blocks(nout) >= 5 ? 512 : 1024)) + tiles - 1) / tiles;
  const int64_t most = (nblk + gran - 1) / gran;
  if (want > most) want = most;
  if (want < 1) want = 1;
  int64_t cb = (nblk + want - 1) / want;
  cb = (cb + gran - 1) / gran * gran;
  return ProjPlan{wide, tg, cb, (nblk + cb - 1) / cb};
}
inline int64_t proj_chunks(int state_dtype, bool gather, int64_t K, int C, int64_t nout, int64_t T) {
  return proj_plan(state_dtype, gather, K, C, nout, T).nchunk;
}

hipError_t launch_proj_partial(int state_dtype, const void* X, int64_t T, int N, int C, int64_t K,
                               const void* packed, int64_t nout, const int32_t* idx, int k,
                               float* part, hipStream_t s);
hipError_t launch_pre_route(const float* part, int64_t nchunk, int64_t nout, int64_t T, int N, int m, int k,
                            int npre, int64_t C, const float* colsum, const float* alpha_pre, int alpha_stride,
                            const float* b_pre, float eps, int32_t* idx, float* p, float* Hpre, float* sums,
                            float* saved, int nsave, int save_stats_at, int router, hipStream_t s,
                            int save_pre = 0);   // which pre-map's z goes to saved[N .. 2N); -1: all, one record each
hipError_t launch_pre_coef(const float* part, int64_t nchunk, int64_t nout, int64_t T, int k, int Kq,
                           int with_res, int64_t C, const float* alpha_post, const float* alpha_res,
                           const float* b_post, const float* b_res, float eps, int iters, float delta,
                           float* Hpost, float* Hres, float* sums, float* saved, int nsave, int save_z_at,
                           int save_stats_at, hipStream_t s, const int* err = nullptr);
// out0 gets map 0 (full dense read); maps 1..nmap-1 leave out the active
// streams and go to outr + (q - 1) * T * C.
hipError_t launch_dense_read(int state_dtype, const void* X, int64_t T, int N, int C, const float* Hpre,
                             int nmap, const int32_t* idx, int k, void* out0, void* outr, hipStream_t s);

// final stream reduction and its backward (broadcast)
hipError_t launch_stream_sum(int state_dtype, const void* X, int64_t T, int N, int C, void* out, hipStream_t s);
hipError_t launch_stream_bcast(int state_dtype, const void* dout, int64_t T, int N, int C, int accumulate, void* dX,
                               hipStream_t s);

// ---- pre (fused single-pass path: bf16 state, N = 16, k = 4, C % 128 == 0)
bool fused_pre_supported(const xhc_dims* d);
size_t fused_pre_ws_bytes(const xhc_dims* d);
hipError_t launch_pre_fused(const xhc_dims* d, const void* X, const void* packed_full, const float* colsum,
                            const void* packed_act, const float* alpha, const float* b_pre, const float* b_res,
                            const float* b_post, void* input, int32_t* idx, float* p, float* Hpre, float* Hres,
                            float* Hpost, float* saved, void* ws, hipStream_t s);

// ---- post
__host__ __device__ inline int64_t post_chunks(int C) { return ((int64_t)C / 8 + 255) / 256; }
// Gram partial chunks written by launch_post_gram (run-based kernels use 1024-channel chunks)
int64_t gram_chunks(int C, int64_t S, int Kr, const int32_t* kappa);
hipError_t launch_post_gram(int state_dtype, const void* F, int64_t T, int64_t S, int C, int Kr,
                            const int32_t* kappa, const float* conv_w, float* gpart, hipStream_t s);
// The write-back of the k active rows.  For K_r > 1 gpart holds the Gram
// partials of launch_post_gram (nchunk chunks): the write-back weights are then
// formed from them (Gram-Schmidt, p, H^post) inside the run-based kernel, or
// into the workspace wb by a per-token pass before the generic one.  K_r = 1:
// gpart and wb are null.
hipError_t launch_post_apply(int state_dtype, void* X, const void* F, int64_t T, int64_t S, int N, int C,
                             int k, int Kr, const int32_t* kappa, const float* conv_w, const int32_t* idx,
                             const float* p, const float* Hres, const float* Hpost, const float* gpart,
                             int64_t nchunk, int gram_schmidt, float* wb, const float* Hpre_next,
                             const void* base_next, void* input_next, void* Xact_save, hipStream_t s);

// ---- backward
hipError_t launch_bwd_post(const xhc_dims* d, const void* dXn, void* X, const void* Xact, const void* F,
                           const float* conv_w, const int32_t* idx, const float* p, const float* Hres,
                           const float* Hpost, void* dX, void* dF, float* dHres, float* dHpost, float* dp,
                           float* dconv_w, char* ws, hipStream_t s, bool grad_f32);
// (X null: the saved rows are not written back into X; grad_f32: dXn and dX
// are fp32 whatever the state dtype, as the xHC-Flash active-row gradient)
size_t bwd_post_ws_bytes(const xhc_dims* d);
bool bwd_pre_supported(const xhc_dims* d);
size_t bwd_pre_ws_bytes(const xhc_dims* d);
// phases of launch_bwd_pre: kBwdPreAll everything; kBwdPreTokens the
// per-token part only (the <d input, x_i> partials and the token reverse:
// the records the row passes read); kBwdPreTokensGiven the same with those
// partials already in the workspace (launch_bwd_dhpre_multi); kBwdPreReduce
// the reductions only (the row passes' partials already in the workspace)
constexpr int kBwdPreAll = 0, kBwdPreTokens = 1, kBwdPreReduce = 2, kBwdPreTokensGiven = 3;
struct BwdPreWs {
  float *part, *tok, *pg, *wpart_r, *wpart_p, *wpart_a, *red_a, *pgsum;
  uint16_t *dzf, *dza;   // packed dz' of the full-row and active-row MFMA passes
  float *srec, *sreca;   // per-token scalars of the ring passes [Tp][8]: full rows, active rows
};
// Row pass of the pre-map reverse with its inputs staged through an LDS ring
// (xhc_bwd_rows.hip): dX += (input-gradient reads, projection and
// normalisation terms) over rows x 128-channel blocks of a bf16 state, and the
// weight-gradient partials of the projection.  Weight row K = i C + c is
// channel c of row i of every token; slot j of the k-row view is row j.
constexpr int kRowRingMaxQ = 4;
struct RowRingDesc {
  const void* X;                        // bf16 state [T][N][C]
  void* dX;                             // gradient rows [T][N][C], updated in place
  bool dx_f32;                          // fp32 gradient rows (else bf16)
  int nq;                               // input gradients, 0 .. kRowRingMaxQ
  const void* din[kRowRingMaxQ];        // bf16 [T][C]
  const float* hp[kRowRingMaxQ];        // their weights: row i of token t at t hp_stride + i
  int hp_stride;
  const float* w[kRowRingMaxQ + 1];     // weight blocks [rows][win[b]] (fp32), outputs in block order
  int win[kRowRingMaxQ + 1];
  int nwin;
  float* wout[kRowRingMaxQ + 1];        // partials [chunk][rows][wout_w], outputs in blocks of wout_w
  int wout_w;
  int nout;                             // outputs
  const uint16_t* dzp;                  // packed dz' of nop outputs (rows, then 32-token transposes)
  int nop;
  const float* srec;                    // per-token r_ln, mu, m1, m2, beta (16-byte aligned rows)
  int64_t srec_stride;                  // floats
  int64_t T, tchunk;                    // tokens; tokens per partial (a multiple of 32)
  int N, C;
};
bool bwd_rows_ring_supported(int64_t rows, int C, int64_t tchunk);
hipError_t launch_bwd_rows_ring(const RowRingDesc& d, int64_t rows, hipStream_t s);
BwdPreWs bwd_pre_ws(const xhc_dims* d, char* ws);   // layout of launch_bwd_pre's workspace
hipError_t launch_bwd_pre(const xhc_dims* d, const void* X, const float* colsum, const float* W_r,
                          const float* W_pre, const float* W_res, const float* W_post, const float* alpha,
                          const float* b_res, const float* saved, const int32_t* idx, const float* p,
                          const float* Hpre, const float* Hpost, const void* d_input, const float* dHres,
                          const float* dHpost, const float* dp, void* dX, float* dW_r, float* dW_pre, float* dW_res,
                          float* dW_post, float* dalpha, float* db_pre, float* db_res, float* db_post, char* ws,
                          hipStream_t s, const float* dhpre_act = nullptr, const float* Hpre_read = nullptr,
                          bool dense_rows = true, const void* X_bf16 = nullptr, bool act_rows = true,
                          int phase = kBwdPreAll, const void* act_din = nullptr);
// dhpre_act [T,k]: when given, dL/dH^pre of the active streams (slot order)
// replaces <d input, x_i> there; Hpre_read [T,N]: when given, the weights of
// the dense-read term dX_i += H^pre_i d input (Hpre otherwise).  dense_rows
// false leaves out every term of the dense rows (the read H^pre_i d input and
// the full-state projection through W_r, W_pre): for a caller whose router
// and pre-map weights are zero; d_input is then not read, H^pre enters as
// zero gradient, and dW_r, dW_pre are not written.  X_bf16: for an fp32
// state whose values are exactly bf16 and whose slot j is row j (N = k: the
// k-row view of an xHC-Flash sublayer), the same rows as bf16 (read by the
// ring form of the active-row pass; the gradient rows stay fp32), and then
// act_din (bf16 [T, C]), when given: that pass also adds Hpre[t, j] act_din[t]
// to active row j (Hpre then holds [T, k] slot weights).  act_rows
// false leaves out the active-row pass (for a caller whose W_post and W_res
// are zero): dW_post, dW_res are not written.
// The full-row pass of Q pre-map reverses of one bf16 state (N = 16, Q = 2 or
// 4) in one pass: pass q's token records and weight partials live in the
// launch_bwd_pre workspace ws[q] (after its kBwdPreTokens phase; the router's
// partials in ws[0]), hrd[q] are its dense-read weights [T, N], d_input is
// [Q, T, C]; dX accumulates every pass's row terms.
// prep: a scratch buffer of bwd_rows_multi_ws_bytes (per-token inputs of the
// fused pass).
bool bwd_rows_multi_supported(const xhc_dims* d, int Q);
size_t bwd_rows_multi_ws_bytes(const xhc_dims* d, int Q);
// the <d input_q, x_i> partials of the Q passes in one read of the state,
// into each pass's workspace ws[q]
hipError_t launch_bwd_dhpre_multi(const xhc_dims* d, int Q, const void* X, const void* d_input, char* const* ws,
                                  hipStream_t s);
hipError_t launch_bwd_rows_multi(const xhc_dims* d, int Q, const void* X, void* dX, const float* W_r,
                                 const float* W_pre, const void* d_input, const float* const* hrd, char* const* ws,
                                 float* prep, hipStream_t s);

// ---- xHC-Flash backward helpers
hipError_t launch_fill0(void* p, size_t bytes, hipStream_t s);
hipError_t launch_fbwd_token(int state_dtype, int64_t T, int N, int k, int C, const int32_t* idx,
                             const float* Hpre_q, const void* din, const void* Xact, int32_t* idx_id, float* Hres_id,
                             float* Hsel, float* dhact, hipStream_t s);
hipError_t launch_fbwd_gather(int state_dtype, int64_t T, int N, int k, int C, const int32_t* idx, const void* dXn,
                              float* da, hipStream_t s);
hipError_t launch_fbwd_scatter(int state_dtype, int64_t T, int N, int k, int C, const int32_t* idx, const void* GX,
                               const float* da0, void* dX, hipStream_t s);
hipError_t launch_fbwd_mask(int64_t T, int N, int k, const int32_t* idx, const float* Hpre, float* Hm, hipStream_t s);
hipError_t launch_fbwd_add(float* dst, const float* src, int64_t n, hipStream_t s);
hipError_t launch_fbwd_alpha(const float* a0, const float* a1, const float* a2, float* out, hipStream_t s);
hipError_t launch_fbwd_finish(int state_dtype, int64_t T, int k, int C, const float* da_rev, const float* Hsel,
                              const void* din, float* da, hipStream_t s);

// per-token values xhc_pre saves for the backward: [z_r (N) | z_pre (N) |
// z_post, z_res (k*Kr + k*k) | mu | nu | nu_a | pad], z = normalised logits
__host__ __device__ inline int saved_floats(int N, int k, int Kr) { return 2 * N + k * Kr + k * k + 4; }

}  // namespace xhc

// Internal launchers of the libexfold kernels.  Every launcher enqueues on
// `stream` and returns hipGetLastError() of its launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace exfold {

// ---- routing (k_route.hip) ----
hipError_t launch_router_logits(int dtype, const void *x, const void *w_router, int T, int N, int d,
                                int P, float *part, hipStream_t s);
// Number of d-slices (partial sums) the router uses for T tokens: [P, T, N] floats.
int router_splits(int dtype, int T, int N, int d);
// Per-token Top-K + softmax (if part != nullptr: logits = sum of the P partials
// + bias, written to logits_out if given), prefill selection (if keep or fold
// outputs are requested) and prefill fold (if fold_ids != nullptr).
// loss_cap/flags: the prefill fold safeguards (EXFOLD_FOLD_* bits).
hipError_t launch_route_tokens(const float *part, int P, const float *bias, float *logits_out, int T,
                               int N, int K, int k_pre, const float *h, const float *S, const float *L,
                               int32_t *topk_ids, float *topk_w, uint8_t *keep,
                               const uint8_t *keep_in, int32_t *fold_ids, float *fold_w,
                               hipStream_t s, float loss_cap = 0.f, int flags = 0,
                               int32_t *om_src = nullptr, float *om_w = nullptr,
                               int32_t *om_q = nullptr, float *wret = nullptr);
// Router logits and the per-token steps of launch_route_tokens in one kernel, for
// bf16 layers of at most 32 experts (route_small_fits): one workgroup per token
// up to 1024 tokens, one per 16 tokens beyond; x [T, d], w_router [N, d].
bool route_small_fits(int dtype, int N, int T);
hipError_t launch_route_small(const void *x, const void *w_router, int d, const float *bias,
                              float *logits_out, int T, int N, int K, int k_pre, const float *h,
                              const float *S, const float *L, int32_t *topk_ids, float *topk_w,
                              uint8_t *keep, int32_t *fold_ids, float *fold_w, hipStream_t s,
                              float loss_cap = 0.f, int flags = 0, int32_t *om_src = nullptr,
                              float *om_w = nullptr, int32_t *om_q = nullptr, float *wret = nullptr);
// Decode pool (if do_pool) and per-source tables + per-slot remap (if out_ids).
hipError_t launch_decode_pool_fold(const int32_t *ids, const float *w, int B, int N, int K, int D,
                                   const float *h, const float *S, const float *L, bool do_pool,
                                   int32_t *pool, int32_t *pool_size, int32_t *out_ids,
                                   float *out_w, int32_t *tgt, float *scl, hipStream_t s);

// ---- permutation (k_permute.hip) ----
constexpr int kPermSlotsPerBlock = 1024;
struct PermBuffers {
  int32_t *blk_counts;   // [nblk, N]
  int32_t *offsets;      // [N + 2]: routed groups, then the shared group
  int32_t *tile_start0;  // [N + 2]: m-tile prefix for tile height bm0
  int32_t *tile_start1;  // [N + 2]: m-tile prefix for tile height bm1
  int32_t *row_token;    // [R + T_shared]
  int32_t *row_slot;     // [R + T_shared] (-1 for shared rows)
  float *row_w;          // [R + T_shared]
  int32_t *slot_row;     // [R]
};
// Stable counting sort of R = T*k_out route slots by expert; the T_shared
// shared-expert rows are appended after the routed rows.
hipError_t launch_permute(const int32_t *route_ids, const float *route_w, int T, int k_out, int N,
                          int t_shared, int bm0, int bm1, const PermBuffers &pb, hipStream_t s);
// Decode front end in one workgroup, after Top-K: pool, tables, remap and the
// permutation of the remapped [B, K] slots (pb.blk_counts unused).  For
// B * K <= kDecodeFrontMaxSlots.  With static_tgt/static_scl (precomputed
// tables of a static pool) the pool and table steps are skipped; h, S, L,
// pool, pool_size, tgt and scl are then unused.
constexpr int kDecodeFrontMaxSlots = 8192;
// With part != nullptr the front end also takes the per-token Top-K and softmax
// from the P router partials (+ bias), writing ids_out/w_out [B, K] (and the
// logits when logits_out is given); ids and w are then unused.  For batches
// where decode_front_fuses_topk holds (at most one token per wave; one launch
// fewer).
struct FrontTopK {
  const float *part = nullptr;
  int P = 0;
  const float *bias = nullptr;
  float *logits_out = nullptr;
  int32_t *ids_out = nullptr;
  float *w_out = nullptr;
};
bool decode_front_fuses_topk(int B, int N);
hipError_t launch_decode_front(const int32_t *ids, const float *w, int B, int N, int K, int D,
                               const float *h, const float *S, const float *L, int32_t *pool,
                               int32_t *pool_size, int32_t *out_ids, float *out_w, int32_t *tgt,
                               float *scl, int t_shared, int bm0, int bm1, const PermBuffers &pb,
                               const int32_t *static_tgt, const float *static_scl, hipStream_t s,
                               const FrontTopK &fused = FrontTopK{});
// The stable permutation of launch_permute in one workgroup (the decode front
// end with every expert mapped to itself), for T * k_out <= kDecodeFrontMaxSlots:
// one launch instead of three.
hipError_t launch_permute_one_block(const int32_t *ids, const float *w, int T, int k_out, int N,
                                    int t_shared, int bm0, int bm1, const PermBuffers &pb,
                                    hipStream_t s);
// Per-slot remap of [slots] routes with static tables (grid-wide).
hipError_t launch_static_remap(const int32_t *ids, const float *w, int slots, int N,
                               const int32_t *tgt, const float *scl, int32_t *out_ids, float *out_w,
                               hipStream_t s);
// Static decode pool TopK(h, D) and its per-source tables (one workgroup).
hipError_t launch_static_pool(const float *h, int N, int D, const float *S, const float *L,
                              int32_t *pool, int32_t *pool_size, int32_t *tgt, float *scl,
                              hipStream_t s);

// ---- expert GEMMs and combine (k_gemm.hip) ----
// kGemmTile: 128x128 tiles; kGemmSkinny: 32x64 tiles for few rows per expert;
// kGemmWide: 256x256 tiles (eight waves, loads straight into LDS) in rounds of
// `wgs` workgroups, a short last round split along the reduction.
enum { kGemmSimt = 0, kGemmTile = 1, kGemmSkinny = 2, kGemmWide = 3 };
struct GemmPlan {
  int bm, bn;  // tile height (rows; kGemmWide: the 128-row unit of its tile list) and width
               // (output columns, or weight rows for gate/up)
  int ksplit;  // splits of the reduction (down projection only; partial outputs)
  int grid;    // workgroups launched (an upper bound on the device-side tile count)
  int kind;    // kGemmSimt (float32 layers), kGemmTile, kGemmSkinny or kGemmWide (bf16 MFMA tiles)
  int wgs;     // kGemmWide: workgroups per round (one per CU)
};
struct ExpertArgs {
  int dtype;
  int d, inter, n_experts, groups;  // groups = N (+1 with a shared expert)
  const void *x;                     // [T, d]
  const void *w_gate_up, *w_down;    // routed [N, 2I, d], [N, d, I]
  const void *ws_gate_up, *ws_down;  // shared or nullptr
  const int32_t *offsets, *tile_start_gu, *tile_start_dn;
  const int32_t *row_token;
  const float *row_w;
  int rows;     // R + T_shared
  void *H;      // [rows, I]
  float *Y;     // [ksplit, rows, d] per-row outputs (nullptr when direct)
  void *y;      // [T, d] direct output (each token owns exactly one row)
  bool direct;
  bool y_bf16;  // bf16 GEMMs, no split: Y holds [rows, d] unscaled bf16 rows instead
  float *wide_part;  // kGemmWide: split-remainder partial tiles, wide_partial_floats(wgs) floats
};
// Partial-tile scratch of a kGemmWide launch in rounds of `wgs` workgroups (the
// split remainder holds at most wgs partial 256x256 tiles).
inline size_t wide_partial_floats(int wgs) { return (size_t)wgs * 256 * 256; }
// active_groups: expected number of non-empty groups (sizes the down split).
void plan_expert_gemms(int dtype, int rows, int groups, int active_groups, int d, int inter,
                       int cu_count, GemmPlan *gate_up, GemmPlan *down);
// ev_mid (optional) is recorded between the gate_up and the down GEMM.
hipError_t launch_expert_gemms(const ExpertArgs &a, const GemmPlan &gu, const GemmPlan &dn,
                               hipStream_t s, hipEvent_t ev_mid = nullptr);
// Plain bf16 product part[P][M][N] = partial sums over P equal reduction
// ranges of A[M, K] W[N, K]^T (fp32, MFMA 128x128 tiles).  plain_gemm_splits
// gives P for the shape (0: N % 128 != 0 or K % 64 != 0, not supported).
int plain_gemm_splits(int M, int N, int K, int cu_count);
hipError_t launch_plain_gemm_nt(const void *A, const void *W, int M, int N, int K, int P, float *part,
                                hipStream_t s);
// row_w: the rows' routing weights, applied here to bf16 rows (y_bf16).
hipError_t launch_combine(int dtype, const float *Y, bool y_bf16, int ksplit, int rows,
                          const int32_t *slot_row, const float *row_w, int T, int k_out, int d,
                          int shared_base, void *y, hipStream_t s);

// ---- diagonal projectors (k_diag.hip) ----
// Per-pair per-dimension statistics -> Dg [N, N, d] and the diagonal loss Ld [N, N].
hipError_t launch_diag_stats(const float *Y, const int32_t *slot_row, const double *gram,
                             const int16_t *pos, int m, int N, int kr, int d, double lambda, float *Dg,
                             float *Ld, hipStream_t s);
// y from the unweighted expert rows and the diagonal fold lists.
hipError_t launch_diag_combine(int dtype, const float *Yr, const int32_t *slot_row, const int32_t *ids,
                               const float *wret, const int32_t *om_src, const float *om_w,
                               const int32_t *om_q, const float *Dg, int T, int N, int K, int k_out,
                               int d, int shared_base, void *y, hipStream_t s);

// ---- calibration (k_calib.hip) ----
hipError_t launch_calib_routes(const int32_t *topk_ids, int m, int N, int K, int mode,
                               int32_t *route_ids, float *route_w, int16_t *pos, hipStream_t s);
hipError_t launch_calib_gram(const float *Y, const int32_t *slot_row, int m, int kr, int d,
                             double *gram, hipStream_t s);
hipError_t launch_calib_finalize(const double *gram, const int16_t *pos, int m, int N, int kr,
                                 double lambda, double clip, float *S, float *L, float *h,
                                 double *pair_stats, hipStream_t s);

}  // namespace exfold

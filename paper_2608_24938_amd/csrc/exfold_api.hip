// C-ABI entry points of libexfold: argument validation (before any launch),
// workspace planning, and the launch sequence of each call on the caller's
// stream.  No host synchronisation, no device allocation.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.hpp"
#include "exfold.h"
#include "kernels.hpp"

using namespace exfold;

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kMaxTokens = int64_t(1) << 22;  // keeps T*N and T*K_out*d offsets in range
constexpr int64_t kMaxSlots = int64_t(1) << 28;

inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

struct Carver {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes);
    return o;
  }
};

// Read-only cache of the CU count per device (the only state the library keeps).
int cu_count() {
  static std::mutex mu;
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

// The kernels move tensors in 16-byte vectors (loads of x and the weights,
// stores of y).
inline bool misaligned(const void *ptr) { return reinterpret_cast<uintptr_t>(ptr) % 16 != 0; }

exfold_status check_layer(const exfold_layer *L) {
  if (!L) return EXFOLD_ERR_NULL;
  if (L->dtype != EXFOLD_F32 && L->dtype != EXFOLD_BF16) return EXFOLD_ERR_DTYPE;
  if (!L->w_router || !L->w_gate_up || !L->w_down) return EXFOLD_ERR_NULL;
  if (misaligned(L->w_router) || misaligned(L->w_gate_up) || misaligned(L->w_down) ||
      misaligned(L->ws_gate_up) || misaligned(L->ws_down))
    return EXFOLD_ERR_ALIGN;
  if (L->d <= 0 || L->inter <= 0 || L->n_experts <= 0 || L->top_k <= 0 || L->shared_inter < 0)
    return EXFOLD_ERR_SHAPE;
  if (L->top_k > L->n_experts) return EXFOLD_ERR_SHAPE;
  if (L->n_experts > kMaxExperts || L->top_k > kMaxTopK) return EXFOLD_ERR_UNSUPPORTED;
  if (L->d % 128 != 0 || L->inter % 64 != 0) return EXFOLD_ERR_UNSUPPORTED;
  if (L->d > (1 << 16) || L->inter > (1 << 17)) return EXFOLD_ERR_UNSUPPORTED;
  if (L->shared_inter > 0) {
    if (!L->ws_gate_up || !L->ws_down) return EXFOLD_ERR_NULL;
    if (L->shared_inter != L->inter) return EXFOLD_ERR_UNSUPPORTED;
  }
  return EXFOLD_OK;
}

exfold_status check_routing(int64_t T, int64_t N, int64_t K) {
  if (T < 0 || N <= 0 || K <= 0 || K > N) return EXFOLD_ERR_SHAPE;
  if (N > kMaxExperts || K > kMaxTopK) return EXFOLD_ERR_UNSUPPORTED;
  if (T > kMaxTokens || T * K > kMaxSlots) return EXFOLD_ERR_SHAPE;
  return EXFOLD_OK;
}

// Buffers of the expert stage (permutation, H, Y) for T tokens of k_out routes.
struct ExecPlan {
  int T = 0, k_out = 0, N = 0, d = 0, inter = 0, dtype = 0;
  int t_shared = 0, R = 0, rows = 0, groups = 0;
  bool direct = false;
  GemmPlan gu{}, dn{};
  size_t o_blk = 0, o_offsets = 0, o_ts0 = 0, o_ts1 = 0, o_row_token = 0, o_row_slot = 0,
         o_row_w = 0, o_slot_row = 0, o_H = 0, o_Y = 0, o_wpart = 0;
};

void plan_exec(const exfold_layer *L, int phase, int T, int k_out, bool with_shared,
               bool keep_rows, int active_groups, Carver &c, ExecPlan &p) {
  p.T = T;
  p.k_out = k_out;
  p.N = (int)L->n_experts;
  p.d = (int)L->d;
  p.inter = (int)L->inter;
  p.dtype = L->dtype;
  p.t_shared = (with_shared && L->shared_inter > 0) ? T : 0;
  p.R = T * k_out;
  p.rows = p.R + p.t_shared;
  p.groups = p.N + (p.t_shared > 0 ? 1 : 0);
  p.direct = !keep_rows && k_out == 1 && p.t_shared == 0;
  (void)phase;
  plan_expert_gemms(p.dtype, p.rows, p.groups, active_groups, p.d, p.inter, cu_count(), &p.gu,
                    &p.dn);
  const int nblk = (p.R + kPermSlotsPerBlock - 1) / kPermSlotsPerBlock;
  const size_t esz = (p.dtype == EXFOLD_BF16) ? 2 : 4;
  p.o_blk = c.take(sizeof(int32_t) * (size_t)(nblk > 0 ? nblk : 1) * p.N);
  p.o_offsets = c.take(sizeof(int32_t) * (p.N + 2));
  p.o_ts0 = c.take(sizeof(int32_t) * (p.N + 2));
  p.o_ts1 = c.take(sizeof(int32_t) * (p.N + 2));
  p.o_row_token = c.take(sizeof(int32_t) * (size_t)p.rows);
  p.o_row_slot = c.take(sizeof(int32_t) * (size_t)p.rows);
  p.o_row_w = c.take(sizeof(float) * (size_t)p.rows);
  p.o_slot_row = c.take(sizeof(int32_t) * (size_t)(p.R > 0 ? p.R : 1));
  p.o_H = c.take(esz * (size_t)p.rows * p.inter);
  if (p.direct || keep_rows) {  // one row per token, or per-row outputs kept: no split
    p.dn.grid /= p.dn.ksplit;
    p.dn.ksplit = 1;
  }
  p.o_Y = p.direct ? c.take(0) : c.take(sizeof(float) * (size_t)p.dn.ksplit * p.rows * p.d);
  {
    const int wg = p.gu.kind == kGemmWide ? p.gu.wgs : 0, wd = p.dn.kind == kGemmWide ? p.dn.wgs : 0;
    const int wgs = wg > wd ? wg : wd;
    p.o_wpart = c.take(sizeof(float) * wide_partial_floats(wgs));  // shared: the GEMMs run in order
  }
}

template <typename T> T *at(void *ws, size_t off) { return reinterpret_cast<T *>(static_cast<char *>(ws) + off); }

// Permutation, expert GEMMs and (unless keep_rows) the combine.
inline void record(void *const *events, int i, hipStream_t s) {
  if (events && events[i]) (void)hipEventRecord(static_cast<hipEvent_t>(events[i]), s);
}

PermBuffers perm_buffers(const ExecPlan &p, void *ws, int32_t *offsets_dbg, int32_t *row_slot_dbg) {
  PermBuffers pb;
  pb.blk_counts = at<int32_t>(ws, p.o_blk);
  pb.offsets = offsets_dbg ? offsets_dbg : at<int32_t>(ws, p.o_offsets);
  pb.tile_start0 = at<int32_t>(ws, p.o_ts0);
  pb.tile_start1 = at<int32_t>(ws, p.o_ts1);
  pb.row_token = at<int32_t>(ws, p.o_row_token);
  pb.row_slot = row_slot_dbg ? row_slot_dbg : at<int32_t>(ws, p.o_row_slot);
  pb.row_w = at<float>(ws, p.o_row_w);
  pb.slot_row = at<int32_t>(ws, p.o_slot_row);
  return pb;
}

// permuted: the routes were already permuted into pb (the decode front end).
exfold_status run_exec(const exfold_layer *L, const ExecPlan &p, const void *x,
                       const int32_t *route_ids, const float *route_w, void *y, void *ws,
                       int32_t *offsets_dbg, int32_t *row_slot_dbg, bool keep_rows,
                       hipStream_t s, void *const *events = nullptr, bool permuted = false) {
  const PermBuffers pb = perm_buffers(p, ws, offsets_dbg, row_slot_dbg);
  if (!permuted &&
      launch_permute(route_ids, route_w, p.T, p.k_out, p.N, p.t_shared, p.gu.bm, p.dn.bm, pb, s) !=
          hipSuccess)
    return EXFOLD_ERR_DEVICE;
  record(events, EXFOLD_EV_PERMUTE, s);
  ExpertArgs a{};
  a.dtype = p.dtype;
  a.d = p.d;
  a.inter = p.inter;
  a.n_experts = p.N;
  a.groups = p.groups;
  a.x = x;
  a.w_gate_up = L->w_gate_up;
  a.w_down = L->w_down;
  a.ws_gate_up = L->ws_gate_up;
  a.ws_down = L->ws_down;
  a.offsets = pb.offsets;
  a.tile_start_gu = pb.tile_start0;
  a.tile_start_dn = pb.tile_start1;
  a.row_token = pb.row_token;
  a.row_w = pb.row_w;
  a.rows = p.rows;
  a.H = at<char>(ws, p.o_H);
  a.Y = p.direct ? nullptr : at<float>(ws, p.o_Y);
  a.y = y;
  a.direct = p.direct;
  // Rows that only the combine reads travel as bf16, unscaled: each is
  // rounded once and the combine multiplies it by its routing weight before
  // the fp32 sum over the token's routes.  Kept rows and split partials stay
  // fp32 (scaled in the GEMM epilogue).
  a.y_bf16 = p.dtype == EXFOLD_BF16 && !p.direct && !keep_rows && p.dn.ksplit == 1;
  a.wide_part = at<float>(ws, p.o_wpart);
  hipEvent_t ev_mid = (events && events[EXFOLD_EV_GATE_UP])
                          ? static_cast<hipEvent_t>(events[EXFOLD_EV_GATE_UP]) : nullptr;
  if (launch_expert_gemms(a, p.gu, p.dn, s, ev_mid) != hipSuccess) return EXFOLD_ERR_DEVICE;
  record(events, EXFOLD_EV_DOWN, s);
  if (!p.direct && !keep_rows) {
    if (launch_combine(p.dtype, a.Y, a.y_bf16, p.dn.ksplit, p.rows, pb.slot_row, pb.row_w, p.T, p.k_out, p.d,
                       p.t_shared > 0 ? p.R : -1, y, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
  }
  record(events, EXFOLD_EV_END, s);
  return EXFOLD_OK;
}

struct ForwardPlan {
  int T = 0, N = 0, K = 0, k_out = 0, phase = 0, budget = 0, dcap = 0, P = 1;
  size_t o_logits = 0, o_topk_ids = 0, o_topk_w = 0, o_keep = 0, o_pool = 0, o_pool_size = 0,
         o_tgt = 0, o_scl = 0, o_fold_ids = 0, o_fold_w = 0, o_om_src = 0, o_om_w = 0, o_om_q = 0,
         o_wret = 0;
  ExecPlan ex;
  size_t total = 0;
};

exfold_status plan_forward(const exfold_layer *L, int64_t T, int32_t phase, int64_t budget,
                           ForwardPlan &p) {
  exfold_status st = check_layer(L);
  if (st != EXFOLD_OK) return st;
  if (phase != EXFOLD_PHASE_DENSE && phase != EXFOLD_PHASE_PREFILL && phase != EXFOLD_PHASE_DECODE &&
      phase != EXFOLD_PHASE_DECODE_STATIC && phase != EXFOLD_PHASE_PREFILL_DIAG)
    return EXFOLD_ERR_ARG;
  st = check_routing(T, L->n_experts, L->top_k);
  if (st != EXFOLD_OK) return st;
  if (phase != EXFOLD_PHASE_DENSE && budget < 1) return EXFOLD_ERR_BUDGET;
  p.T = (int)T;
  p.N = (int)L->n_experts;
  p.K = (int)L->top_k;
  p.phase = phase;
  p.budget = (int)(budget > (1 << 20) ? (1 << 20) : budget);
  const bool per_token = phase == EXFOLD_PHASE_PREFILL || phase == EXFOLD_PHASE_PREFILL_DIAG;
  p.k_out = per_token ? (p.budget < p.K ? p.budget : p.K) : p.K;
  p.dcap = (p.budget < p.N) ? p.budget : p.N;
  p.P = router_splits(L->dtype, p.T, p.N, (int)L->d);
  Carver c;
  p.o_logits = c.take(sizeof(float) * (size_t)p.P * p.T * p.N);  // router partial sums
  p.o_topk_ids = c.take(sizeof(int32_t) * (size_t)p.T * p.K);
  p.o_topk_w = c.take(sizeof(float) * (size_t)p.T * p.K);
  p.o_keep = c.take((size_t)p.T * p.K);
  p.o_pool = c.take(sizeof(int32_t) * p.N);
  p.o_pool_size = c.take(sizeof(int32_t));
  p.o_tgt = c.take(sizeof(int32_t) * p.N);
  p.o_scl = c.take(sizeof(float) * p.N);
  p.o_fold_ids = c.take(sizeof(int32_t) * (size_t)p.T * p.k_out);
  p.o_fold_w = c.take(sizeof(float) * (size_t)p.T * p.k_out);
  if (phase == EXFOLD_PHASE_PREFILL_DIAG) {
    p.o_om_src = c.take(sizeof(int32_t) * (size_t)p.T * p.K);
    p.o_om_w = c.take(sizeof(float) * (size_t)p.T * p.K);
    p.o_om_q = c.take(sizeof(int32_t) * (size_t)p.T * p.K);
    p.o_wret = c.take(sizeof(float) * (size_t)p.T * p.k_out);
  }
  int active = p.N;
  if (phase == EXFOLD_PHASE_DECODE || phase == EXFOLD_PHASE_DECODE_STATIC) active = p.dcap;
  if (p.T * p.k_out < active) active = p.T * p.k_out;
  if (L->shared_inter > 0) active += 1;
  plan_exec(L, phase, p.T, p.k_out, true, phase == EXFOLD_PHASE_PREFILL_DIAG, active, c, p.ex);
  p.total = c.off;
  return EXFOLD_OK;
}

exfold_status plan_execute(const exfold_layer *L, int64_t T, int64_t k_out, ExecPlan &p,
                           size_t &total) {
  exfold_status st = check_layer(L);
  if (st != EXFOLD_OK) return st;
  if (k_out < 1 || k_out > kMaxExperts * 4) return EXFOLD_ERR_SHAPE;
  if (T < 0 || T > kMaxTokens || T * k_out > kMaxSlots) return EXFOLD_ERR_SHAPE;
  Carver c;
  int active = (int)L->n_experts;
  if (T * k_out < active) active = (int)(T * k_out);
  if (L->shared_inter > 0) active += 1;
  plan_exec(L, EXFOLD_PHASE_DENSE, (int)T, (int)k_out, true, false, active, c, p);
  total = c.off;
  return EXFOLD_OK;
}

struct CalibPlan {
  int m = 0, N = 0, K = 0, kr = 0, P = 1;
  size_t o_logits = 0, o_topk_ids = 0, o_topk_w = 0, o_route_ids = 0, o_route_w = 0, o_pos = 0,
         o_gram = 0;
  ExecPlan ex;
  size_t total = 0;
};

exfold_status plan_calibrate(const exfold_layer *L, int64_t m, int32_t mode, CalibPlan &p) {
  exfold_status st = check_layer(L);
  if (st != EXFOLD_OK) return st;
  if (mode != EXFOLD_CAL_COROUTED && mode != EXFOLD_CAL_COMMON) return EXFOLD_ERR_ARG;
  st = check_routing(m, L->n_experts, L->top_k);
  if (st != EXFOLD_OK) return st;
  p.m = (int)m;
  p.N = (int)L->n_experts;
  p.K = (int)L->top_k;
  p.kr = (mode == EXFOLD_CAL_COMMON) ? p.N : p.K;
  if ((int64_t)p.m * p.kr > kMaxSlots) return EXFOLD_ERR_SHAPE;
  p.P = router_splits(L->dtype, p.m, p.N, (int)L->d);
  Carver c;
  p.o_logits = c.take(sizeof(float) * (size_t)p.P * p.m * p.N);  // router partial sums
  p.o_topk_ids = c.take(sizeof(int32_t) * (size_t)p.m * p.K);
  p.o_topk_w = c.take(sizeof(float) * (size_t)p.m * p.K);
  p.o_route_ids = c.take(sizeof(int32_t) * (size_t)p.m * p.kr);
  p.o_route_w = c.take(sizeof(float) * (size_t)p.m * p.kr);
  p.o_pos = c.take(sizeof(int16_t) * (size_t)p.m * p.N);
  p.o_gram = c.take(sizeof(double) * (size_t)p.m * p.kr * p.kr);
  plan_exec(L, EXFOLD_PHASE_PREFILL, p.m, p.kr, false, true, p.N, c, p.ex);
  p.total = c.off;
  return EXFOLD_OK;
}

bool valid_fold_opts(float loss_cap, int32_t flags) {
  constexpr int32_t kAll = EXFOLD_FOLD_LOSS_CAP | EXFOLD_FOLD_RENORM | EXFOLD_FOLD_CONFIDENCE;
  if (flags & ~kAll) return false;
  if ((flags & EXFOLD_FOLD_LOSS_CAP) && !(loss_cap == loss_cap)) return false;  // NaN cap
  return true;
}

exfold_status check_ws(void *ws, size_t ws_bytes, size_t need) {
  if (need > 0 && !ws) return EXFOLD_ERR_NULL;
  if (ws_bytes < need) return EXFOLD_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0) return EXFOLD_ERR_WORKSPACE;
  return EXFOLD_OK;
}

}  // namespace

extern "C" {

const char *exfold_status_str(exfold_status s) {
  switch (s) {
    case EXFOLD_OK: return "ok";
    case EXFOLD_ERR_NULL: return "required pointer is NULL";
    case EXFOLD_ERR_ALIGN: return "tensor pointer not 16-byte aligned";
    case EXFOLD_ERR_SHAPE: return "size out of range or inconsistent";
    case EXFOLD_ERR_BUDGET: return "budget must be >= 1";
    case EXFOLD_ERR_DTYPE: return "unknown dtype";
    case EXFOLD_ERR_WORKSPACE: return "workspace too small or misaligned";
    case EXFOLD_ERR_DEVICE: return "HIP launch failed";
    case EXFOLD_ERR_UNSUPPORTED: return "outside the kernels' limits";
    case EXFOLD_ERR_ARG: return "invalid phase, mode or scalar argument";
    case EXFOLD_ERR_SCRATCH: return "request needs more than the static scratch (EXFOLD_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

exfold_status exfold_select_prefill(const float *logits, int64_t T, int64_t N, int64_t K,
                                    int64_t k_pre, const float *h, int32_t *topk_ids,
                                    float *topk_w, uint8_t *keep, void *stream) {
  exfold_status st = check_routing(T, N, K);
  if (st != EXFOLD_OK) return st;
  if (k_pre < 1) return EXFOLD_ERR_BUDGET;
  if (T == 0) return EXFOLD_OK;
  if (!h || !topk_ids || !topk_w || !keep) return EXFOLD_ERR_NULL;
  const int kp = (int)(k_pre > K ? K : k_pre);
  if (launch_route_tokens(logits, 1, nullptr, nullptr, (int)T, (int)N, (int)K, kp, h, nullptr, nullptr,
                          topk_ids, topk_w, keep, nullptr, nullptr, nullptr,
                          static_cast<hipStream_t>(stream)) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  return EXFOLD_OK;
}

exfold_status exfold_select_decode_pool(const float *logits, int64_t B, int64_t N, int64_t K,
                                        int64_t D, const float *h, int32_t *topk_ids,
                                        float *topk_w, int32_t *pool, int32_t *pool_size,
                                        void *stream) {
  exfold_status st = check_routing(B, N, K);
  if (st != EXFOLD_OK) return st;
  if (D < 1) return EXFOLD_ERR_BUDGET;
  if (!h || !pool || !pool_size) return EXFOLD_ERR_NULL;
  if (B > 0 && (!topk_ids || !topk_w)) return EXFOLD_ERR_NULL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int dd = (int)(D > N ? N : D);
  if (logits && B > 0) {
    if (launch_route_tokens(logits, 1, nullptr, nullptr, (int)B, (int)N, (int)K, (int)K, nullptr,
                            nullptr, nullptr, topk_ids, topk_w, nullptr, nullptr, nullptr, nullptr,
                            s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
  }
  if (launch_decode_pool_fold(topk_ids, topk_w, (int)B, (int)N, (int)K, dd, h, nullptr, nullptr,
                              true, pool, pool_size, nullptr, nullptr, nullptr, nullptr,
                              s) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  return EXFOLD_OK;
}

exfold_status exfold_static_pool(const float *h, int64_t N, int64_t D, const float *S,
                                 const float *L, int32_t *pool, int32_t *pool_size, int32_t *tgt,
                                 float *scl, void *stream) {
  if (N <= 0) return EXFOLD_ERR_SHAPE;
  if (N > kMaxExperts) return EXFOLD_ERR_UNSUPPORTED;
  if (D < 1) return EXFOLD_ERR_BUDGET;
  if (!h || !S || !L || !pool || !pool_size || !tgt || !scl) return EXFOLD_ERR_NULL;
  const int dd = (int)(D > N ? N : D);
  if (launch_static_pool(h, (int)N, dd, S, L, pool, pool_size, tgt, scl,
                         static_cast<hipStream_t>(stream)) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  return EXFOLD_OK;
}

exfold_status exfold_fold_gates(int32_t phase, int64_t T, int64_t N, int64_t K, int64_t budget,
                                const int32_t *topk_ids, const float *topk_w,
                                const uint8_t *keep, const int32_t *pool,
                                const int32_t *pool_size, const float *S, const float *L,
                                int32_t *out_ids, float *out_w, int32_t *tgt_ids,
                                float *tgt_scale, float loss_cap, int32_t fold_flags,
                                void *stream) {
  if (!valid_fold_opts(loss_cap, fold_flags)) return EXFOLD_ERR_ARG;
  if (phase != EXFOLD_PHASE_PREFILL && phase != EXFOLD_PHASE_DECODE) return EXFOLD_ERR_ARG;
  exfold_status st = check_routing(T, N, K);
  if (st != EXFOLD_OK) return st;
  if (budget < 1) return EXFOLD_ERR_BUDGET;
  if (!S || !L) return EXFOLD_ERR_NULL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (phase == EXFOLD_PHASE_PREFILL) {
    if (T == 0) return EXFOLD_OK;
    if (!topk_ids || !topk_w || !keep || !out_ids || !out_w) return EXFOLD_ERR_NULL;
    const int kp = (int)(budget > K ? K : budget);
    if (launch_route_tokens(nullptr, 0, nullptr, nullptr, (int)T, (int)N, (int)K, kp, nullptr, S, L,
                            const_cast<int32_t *>(topk_ids), const_cast<float *>(topk_w), nullptr,
                            keep, out_ids, out_w, s, loss_cap, fold_flags) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    return EXFOLD_OK;
  }
  if (!pool || !pool_size) return EXFOLD_ERR_NULL;
  if (T > 0 && (!topk_ids || !topk_w || !out_ids || !out_w)) return EXFOLD_ERR_NULL;
  if (T == 0 && !tgt_ids && !tgt_scale) return EXFOLD_OK;
  const int dd = (int)(budget > N ? N : budget);
  if (launch_decode_pool_fold(topk_ids, topk_w, (int)T, (int)N, (int)K, dd, nullptr, S, L, false,
                              const_cast<int32_t *>(pool), const_cast<int32_t *>(pool_size),
                              T > 0 ? out_ids : nullptr, T > 0 ? out_w : nullptr, tgt_ids,
                              tgt_scale, s) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  return EXFOLD_OK;
}

size_t exfold_moe_workspace_size(const exfold_layer *layer, int64_t T, int32_t phase,
                                 int64_t budget) {
  ForwardPlan p;
  if (plan_forward(layer, T, phase, budget, p) != EXFOLD_OK) return 0;
  return p.total;
}

}  // extern "C"

namespace {

// Validation of a forward that needs no workspace (everything but the workspace checks).
exfold_status check_forward(const exfold_layer *layer, const exfold_tables *tables, const void *x,
                            int64_t T, int32_t phase, const void *y) {
  if (phase == EXFOLD_PHASE_DECODE_STATIC) {
    if (!tables || !tables->tgt || !tables->scl) return EXFOLD_ERR_NULL;
  } else if (phase == EXFOLD_PHASE_PREFILL_DIAG) {
    if (!tables || !tables->L || !tables->h || !tables->Dg) return EXFOLD_ERR_NULL;
  } else if (phase != EXFOLD_PHASE_DENSE && (!tables || !tables->S || !tables->L || !tables->h)) {
    return EXFOLD_ERR_NULL;
  }
  if (phase == EXFOLD_PHASE_PREFILL && !valid_fold_opts(tables->loss_cap, tables->fold_flags))
    return EXFOLD_ERR_ARG;
  if (T == 0) return EXFOLD_OK;
  if (!x || !y) return EXFOLD_ERR_NULL;
  if (misaligned(x) || misaligned(y)) return EXFOLD_ERR_ALIGN;
  (void)layer;
  return EXFOLD_OK;
}

exfold_status forward_impl(const exfold_layer *layer, const exfold_tables *tables, const void *x,
                           const ForwardPlan &p, int32_t phase, void *y, const exfold_debug *debug,
                           void *ws, hipStream_t s);

// Scratch of exfold_moe_forward_scratch: one copy per GPU, held until the
// process ends.  Host code never passes the array's name to a kernel (on the
// host it is only a stand-in for the symbol); it uses the device address that
// hipGetSymbolAddress returns for the current device.
__device__ __align__(256) unsigned char scratch[EXFOLD_SCRATCH_BYTES];

// Device address of `scratch` on the current device, queried once per device
// with that device current; nullptr if the query fails.
void *scratch_address() {
  static std::mutex mu;
  static void *cache[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!cache[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    cache[dev] = ptr;
  }
  return cache[dev];
}

}  // namespace

extern "C" {

exfold_status exfold_moe_forward_scratch(const exfold_layer *layer, const exfold_tables *tables,
                                         const void *x, int64_t T, int32_t phase, int64_t budget,
                                         void *y, const exfold_debug *debug, void *stream) {
  ForwardPlan p;
  exfold_status st = plan_forward(layer, T, phase, budget, p);
  if (st != EXFOLD_OK) return st;
  st = check_forward(layer, tables, x, T, phase, y);
  if (st != EXFOLD_OK || T == 0) return st;
  if (p.total > EXFOLD_SCRATCH_BYTES) return EXFOLD_ERR_SCRATCH;
  void *ws = scratch_address();
  if (!ws) return EXFOLD_ERR_DEVICE;
  return forward_impl(layer, tables, x, p, phase, y, debug, ws, static_cast<hipStream_t>(stream));
}

exfold_status exfold_moe_forward(const exfold_layer *layer, const exfold_tables *tables,
                                 const void *x, int64_t T, int32_t phase, int64_t budget,
                                 void *y, const exfold_debug *debug, void *ws, size_t ws_bytes,
                                 void *stream) {
  ForwardPlan p;
  exfold_status st = plan_forward(layer, T, phase, budget, p);
  if (st != EXFOLD_OK) return st;
  st = check_forward(layer, tables, x, T, phase, y);
  if (st != EXFOLD_OK || T == 0) return st;
  st = check_ws(ws, ws_bytes, p.total);
  if (st != EXFOLD_OK) return st;
  return forward_impl(layer, tables, x, p, phase, y, debug, ws, static_cast<hipStream_t>(stream));
}

}  // extern "C"

namespace {

exfold_status forward_impl(const exfold_layer *layer, const exfold_tables *tables, const void *x,
                           const ForwardPlan &p, int32_t phase, void *y, const exfold_debug *debug,
                           void *ws, hipStream_t s) {
  exfold_status st = EXFOLD_OK;
  const exfold_debug z{};
  const exfold_debug &dbg = debug ? *debug : z;
  float *part = at<float>(ws, p.o_logits);
  int32_t *topk_ids = dbg.topk_ids ? dbg.topk_ids : at<int32_t>(ws, p.o_topk_ids);
  float *topk_w = dbg.topk_w ? dbg.topk_w : at<float>(ws, p.o_topk_w);
  uint8_t *keep = dbg.keep ? dbg.keep : at<uint8_t>(ws, p.o_keep);
  int32_t *pool = dbg.pool ? dbg.pool : at<int32_t>(ws, p.o_pool);
  int32_t *pool_size = dbg.pool_size ? dbg.pool_size : at<int32_t>(ws, p.o_pool_size);
  int32_t *fold_ids = dbg.fold_ids ? dbg.fold_ids : at<int32_t>(ws, p.o_fold_ids);
  float *fold_w = dbg.fold_w ? dbg.fold_w : at<float>(ws, p.o_fold_w);

  record(dbg.events, EXFOLD_EV_START, s);
  // few experts (bf16): the router logits are computed inside the routing
  // kernel (one workgroup per token), so the router stage takes no launch
  const bool small = route_small_fits(layer->dtype, p.N, p.T);
  if (!small && launch_router_logits(layer->dtype, x, layer->w_router, p.T, p.N, (int)layer->d, p.P, part,
                                     s) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  record(dbg.events, EXFOLD_EV_ROUTER, s);
  const int32_t *exec_ids = fold_ids;
  const float *exec_w = fold_w;
  const float *bias = layer->router_bias;
  // Top-K + softmax of every token, then (kp < K or fold outputs given) the
  // prefill selection and fold
  auto route = [&](int kp, const float *h, const float *S, const float *L, uint8_t *keep_out, int32_t *fi,
                   float *fw, float cap, int flags, int32_t *oms = nullptr, float *omw = nullptr,
                   int32_t *omq = nullptr, float *wret = nullptr) {
    if (small)
      return launch_route_small(x, layer->w_router, (int)layer->d, bias, dbg.logits, p.T, p.N, p.K, kp, h, S, L,
                                topk_ids, topk_w, keep_out, fi, fw, s, cap, flags, oms, omw, omq, wret);
    return launch_route_tokens(part, p.P, bias, dbg.logits, p.T, p.N, p.K, kp, h, S, L, topk_ids, topk_w,
                               keep_out, nullptr, fi, fw, s, cap, flags, oms, omw, omq, wret);
  };
  bool permuted = false;
  hipError_t e = hipSuccess;
  if (phase == EXFOLD_PHASE_DENSE) {
    e = route(p.K, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0.f, 0);
    exec_ids = topk_ids;
    exec_w = topk_w;
  } else if (phase == EXFOLD_PHASE_PREFILL) {
    e = route(p.k_out, tables->h, tables->S, tables->L, keep, fold_ids, fold_w, tables->loss_cap,
              tables->fold_flags);
  } else if (phase == EXFOLD_PHASE_PREFILL_DIAG) {
    e = route(p.k_out, tables->h, nullptr, tables->L, keep, fold_ids, fold_w, 0.f, 0, at<int32_t>(ws, p.o_om_src),
              at<float>(ws, p.o_om_w), at<int32_t>(ws, p.o_om_q), at<float>(ws, p.o_wret));
  } else {
    const bool stat = phase == EXFOLD_PHASE_DECODE_STATIC;
    const bool front = (int64_t)p.T * p.K <= kDecodeFrontMaxSlots;
    FrontTopK fused;
    if (!small && front && decode_front_fuses_topk(p.T, p.N))
      fused = FrontTopK{part, p.P, bias, dbg.logits, topk_ids, topk_w};
    else
      e = route(p.K, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0.f, 0);
    if (e == hipSuccess && front) {
      // (Top-K,) pool, tables, remap and permutation in one workgroup
      const PermBuffers pb = perm_buffers(p.ex, ws, dbg.offsets, dbg.row_slot);
      e = launch_decode_front(topk_ids, topk_w, p.T, p.N, p.K, p.dcap, tables->h, tables->S, tables->L,
                              pool, pool_size, fold_ids, fold_w, dbg.tgt_ids, dbg.tgt_scale,
                              p.ex.t_shared, p.ex.gu.bm, p.ex.dn.bm, pb, stat ? tables->tgt : nullptr,
                              stat ? tables->scl : nullptr, s, fused);
      permuted = true;
    } else if (e == hipSuccess && stat) {
      e = launch_static_remap(topk_ids, topk_w, p.T * p.K, p.N, tables->tgt, tables->scl, fold_ids,
                              fold_w, s);
    } else if (e == hipSuccess) {
      e = launch_decode_pool_fold(topk_ids, topk_w, p.T, p.N, p.K, p.dcap, tables->h, tables->S,
                                  tables->L, true, pool, pool_size, fold_ids, fold_w, dbg.tgt_ids,
                                  dbg.tgt_scale, s);
    }
  }
  if (e != hipSuccess) return EXFOLD_ERR_DEVICE;
  record(dbg.events, EXFOLD_EV_FOLD, s);
  if (phase != EXFOLD_PHASE_PREFILL_DIAG)
    return run_exec(layer, p.ex, x, exec_ids, exec_w, y, ws, dbg.offsets, dbg.row_slot, false, s,
                    dbg.events, permuted);
  // diagonal projectors: unweighted expert rows, then the element-wise combine
  st = run_exec(layer, p.ex, x, exec_ids, exec_w, nullptr, ws, dbg.offsets, dbg.row_slot, true, s,
                dbg.events);
  if (st != EXFOLD_OK) return st;
  const PermBuffers pb = perm_buffers(p.ex, ws, dbg.offsets, dbg.row_slot);
  if (launch_diag_combine(layer->dtype, at<float>(ws, p.ex.o_Y), pb.slot_row, fold_ids,
                          at<float>(ws, p.o_wret), at<int32_t>(ws, p.o_om_src), at<float>(ws, p.o_om_w),
                          at<int32_t>(ws, p.o_om_q), tables->Dg, p.T, p.N, p.K, p.k_out,
                          (int)layer->d, p.ex.t_shared > 0 ? p.ex.R : -1, y, s) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  record(dbg.events, EXFOLD_EV_END, s);
  return EXFOLD_OK;
}

}  // namespace

extern "C" {

size_t exfold_execute_workspace_size(const exfold_layer *layer, int64_t T, int64_t k_out) {
  ExecPlan p;
  size_t total = 0;
  if (plan_execute(layer, T, k_out, p, total) != EXFOLD_OK) return 0;
  return total;
}

exfold_status exfold_moe_execute(const exfold_layer *layer, const void *x, int64_t T,
                                 int64_t k_out, const int32_t *route_ids, const float *route_w,
                                 void *y, const exfold_debug *debug, void *ws, size_t ws_bytes,
                                 void *stream) {
  ExecPlan p;
  size_t total = 0;
  exfold_status st = plan_execute(layer, T, k_out, p, total);
  if (st != EXFOLD_OK) return st;
  if (T == 0) return EXFOLD_OK;
  if (!x || !y || !route_ids || !route_w) return EXFOLD_ERR_NULL;
  if (misaligned(x) || misaligned(y)) return EXFOLD_ERR_ALIGN;
  st = check_ws(ws, ws_bytes, total);
  if (st != EXFOLD_OK) return st;
  return run_exec(layer, p, x, route_ids, route_w, y, ws, debug ? debug->offsets : nullptr,
                  debug ? debug->row_slot : nullptr, false, static_cast<hipStream_t>(stream));
}

size_t exfold_calibrate_workspace_size(const exfold_layer *layer, int64_t m, int32_t mode) {
  CalibPlan p;
  if (plan_calibrate(layer, m, mode, p) != EXFOLD_OK) return 0;
  return p.total;
}

exfold_status exfold_calibrate_projectors(const exfold_layer *layer, const void *x_cal, int64_t m,
                                          double lambda, double clip, int32_t mode, float *S,
                                          float *L, float *h, double *pair_stats, void *ws,
                                          size_t ws_bytes, void *stream) {
  CalibPlan p;
  exfold_status st = plan_calibrate(layer, m, mode, p);
  if (st != EXFOLD_OK) return st;
  if (!(lambda >= 0.0) || !(clip >= 0.0)) return EXFOLD_ERR_ARG;
  if (!S || !L || !h) return EXFOLD_ERR_NULL;
  if (m > 0 && !x_cal) return EXFOLD_ERR_NULL;
  if (misaligned(x_cal)) return EXFOLD_ERR_ALIGN;
  st = check_ws(ws, ws_bytes, p.total);
  if (st != EXFOLD_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  float *logits = at<float>(ws, p.o_logits);
  int32_t *topk_ids = at<int32_t>(ws, p.o_topk_ids);
  float *topk_w = at<float>(ws, p.o_topk_w);
  int32_t *route_ids = at<int32_t>(ws, p.o_route_ids);
  float *route_w = at<float>(ws, p.o_route_w);
  int16_t *pos = at<int16_t>(ws, p.o_pos);
  double *gram = at<double>(ws, p.o_gram);
  if (p.m > 0) {
    if (launch_router_logits(layer->dtype, x_cal, layer->w_router, p.m, p.N, (int)layer->d, p.P,
                             logits, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    if (launch_route_tokens(logits, p.P, layer->router_bias, nullptr, p.m, p.N, p.K, p.K, nullptr,
                            nullptr, nullptr, topk_ids, topk_w, nullptr, nullptr, nullptr, nullptr,
                            s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    if (launch_calib_routes(topk_ids, p.m, p.N, p.K, mode, route_ids, route_w, pos, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    st = run_exec(layer, p.ex, x_cal, route_ids, route_w, nullptr, ws, nullptr, nullptr, true, s);
    if (st != EXFOLD_OK) return st;
    if (launch_calib_gram(at<float>(ws, p.ex.o_Y), at<int32_t>(ws, p.ex.o_slot_row), p.m, p.kr,
                          (int)layer->d, gram, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
  }
  if (launch_calib_finalize(gram, pos, p.m, p.N, p.kr, lambda, clip, S, L, h, pair_stats, s) !=
      hipSuccess)
    return EXFOLD_ERR_DEVICE;
  return EXFOLD_OK;
}

exfold_status exfold_calibrate_diagonal(const exfold_layer *layer, const void *x_cal, int64_t m,
                                        double lambda, int32_t mode, float *Dg, float *Ld, void *ws,
                                        size_t ws_bytes, void *stream) {
  CalibPlan p;
  exfold_status st = plan_calibrate(layer, m, mode, p);
  if (st != EXFOLD_OK) return st;
  if (!(lambda >= 0.0)) return EXFOLD_ERR_ARG;
  if (!Dg || !Ld) return EXFOLD_ERR_NULL;
  if (m > 0 && !x_cal) return EXFOLD_ERR_NULL;
  if (misaligned(x_cal)) return EXFOLD_ERR_ALIGN;
  st = check_ws(ws, ws_bytes, p.total);
  if (st != EXFOLD_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  float *logits = at<float>(ws, p.o_logits);
  int32_t *topk_ids = at<int32_t>(ws, p.o_topk_ids);
  float *topk_w = at<float>(ws, p.o_topk_w);
  int32_t *route_ids = at<int32_t>(ws, p.o_route_ids);
  float *route_w = at<float>(ws, p.o_route_w);
  int16_t *pos = at<int16_t>(ws, p.o_pos);
  double *gram = at<double>(ws, p.o_gram);
  if (p.m > 0) {
    if (launch_router_logits(layer->dtype, x_cal, layer->w_router, p.m, p.N, (int)layer->d, p.P,
                             logits, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    if (launch_route_tokens(logits, p.P, layer->router_bias, nullptr, p.m, p.N, p.K, p.K, nullptr,
                            nullptr, nullptr, topk_ids, topk_w, nullptr, nullptr, nullptr, nullptr,
                            s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    if (launch_calib_routes(topk_ids, p.m, p.N, p.K, mode, route_ids, route_w, pos, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
    st = run_exec(layer, p.ex, x_cal, route_ids, route_w, nullptr, ws, nullptr, nullptr, true, s);
    if (st != EXFOLD_OK) return st;
    if (launch_calib_gram(at<float>(ws, p.ex.o_Y), at<int32_t>(ws, p.ex.o_slot_row), p.m, p.kr,
                          (int)layer->d, gram, s) != hipSuccess)
      return EXFOLD_ERR_DEVICE;
  }
  if (launch_diag_stats(at<float>(ws, p.ex.o_Y), at<int32_t>(ws, p.ex.o_slot_row), gram, pos, p.m, p.N,
                        p.kr, (int)layer->d, lambda, Dg, Ld, s) != hipSuccess)
    return EXFOLD_ERR_DEVICE;
  return EXFOLD_OK;
}

static_assert(EXFOLD_GEMM_SIMT == kGemmSimt && EXFOLD_GEMM_TILE == kGemmTile &&
                  EXFOLD_GEMM_SKINNY == kGemmSkinny && EXFOLD_GEMM_WIDE == kGemmWide,
              "the header's GEMM kinds are the planner's");

exfold_status exfold_gemm_plan(const exfold_layer *L, int64_t rows, int64_t active_groups,
                               int32_t cu_count, int32_t *out) {
  exfold_status st = check_layer(L);
  if (st != EXFOLD_OK) return st;
  if (!out) return EXFOLD_ERR_NULL;
  if (rows < 0 || rows > (int64_t)kMaxSlots + kMaxTokens || active_groups < 1 || cu_count < 1)
    return EXFOLD_ERR_SHAPE;
  const int groups = (int)L->n_experts + (L->shared_inter > 0 ? 1 : 0);
  GemmPlan gu, dn;
  plan_expert_gemms(L->dtype, (int)rows, groups, (int)(active_groups < groups ? active_groups : groups),
                    (int)L->d, (int)L->inter, cu_count, &gu, &dn);
  const GemmPlan *pl[2] = {&gu, &dn};
  for (int i = 0; i < 2; ++i) {
    out[5 * i + 0] = pl[i]->kind;
    out[5 * i + 1] = pl[i]->bm;
    out[5 * i + 2] = pl[i]->bn;
    out[5 * i + 3] = pl[i]->ksplit;
    out[5 * i + 4] = pl[i]->grid;
  }
  return EXFOLD_OK;
}

}  // extern "C"

// Router logits, Top-K softmax, phase selection and folding of route metadata.
//
//   router logits    r = W_r x (+ bias)                   Sec. 2.1 (before Eq. topk_gate)
//   Top-K softmax    alpha_e = exp r_e / sum_{S_K} exp r   Eq. topk_gate
//   prefill select   TopK_{e in S_K}(w h_e, K')            Eq. prefill_budget (Eq. A6)
//   prefill fold     w~_t = w_t + sum w_s S_{s->t}         Eq. minimum_loss_assignment, Eq. prefill_fold
//   decode pool      TopK_{e in union S_K}(sum w h_e, D)   Eq. decode_budget (Eq. A7)
//   decode remap     (E_s, w_s) -> (E_pi(s), w_s S)        Eq. decode_remap (Eq. A11)
//
// Discrete decisions are taken on exact values: keys of float32 logits, exact
// float64 products of two float32 values, exact integer fixed-point weight sums.
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

// ---------------------------------------------------------------------------
// Router logits.  bf16: a workgroup of KS waves takes 16 tokens; wave w reduces
// its slice of d with 16x16x32 bf16 MFMA against all NT*16 (padded) experts, and
// the KS partial sums are added in a fixed order through LDS.  W_r stays in L2.
// f32: one thread per logit.
// ---------------------------------------------------------------------------
template <int NT, int KS>
__global__ __launch_bounds__(64 * KS) void router_logits_bf16(const bf16_t *__restrict__ x,
                                                              const bf16_t *__restrict__ wr,
                                                              const float *__restrict__ bias,
                                                              int T, int N, int d,
                                                              float *__restrict__ logits) {
  __shared__ float red[KS][NT * 4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t0 = blockIdx.x * 16;
  const int row = min(t0 + (lane & 15), T - 1);
  const int kq = (lane >> 4) * 8;
  f32x4 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16_t *wrow[NT];
  bool live[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int e = j * 16 + (lane & 15);
    live[j] = e < N;
    wrow[j] = wr + (size_t)(live[j] ? e : 0) * d + kq;
  }
  const bf16_t *xa = x + (size_t)row * d + kq;
  const int steps = d / 32;
  const int s0 = wave * steps / KS, s1 = (wave + 1) * steps / KS;
  bf16x8 zero;
#pragma unroll
  for (int q = 0; q < 8; ++q) zero[q] = (__bf16)0.0f;
  int st = s0;
  for (; st + 2 <= s1; st += 2) {
    const int k = st * 32;
    const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(xa + k);
    const bf16x8 a1 = *reinterpret_cast<const bf16x8 *>(xa + k + 32);
    bf16x8 b0[NT], b1[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      b0[j] = *reinterpret_cast<const bf16x8 *>(wrow[j] + k);
      b1[j] = *reinterpret_cast<const bf16x8 *>(wrow[j] + k + 32);
    }
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, live[j] ? b0[j] : zero, acc[j], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, live[j] ? b1[j] : zero, acc[j], 0, 0, 0);
    }
  }
  if (st < s1) {
    const int k = st * 32;
    const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(xa + k);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(wrow[j] + k);
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, live[j] ? b0 : zero, acc[j], 0, 0, 0);
    }
  }
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][j * 4 + i][lane] = acc[j][i];
  __syncthreads();
  // entry (j, i, l): expert j*16 + l%16, token t0 + (l/16)*4 + i
  for (int idx = threadIdx.x; idx < NT * 4 * 64; idx += 64 * KS) {
    const int ji = idx >> 6, l = idx & 63;
    const int j = ji >> 2, i = ji & 3;
    float v = red[0][ji][l];
#pragma unroll
    for (int w = 1; w < KS; ++w) v += red[w][ji][l];
    const int t = t0 + (l >> 4) * 4 + i;
    const int e = j * 16 + (l & 15);
    if (t < T && e < N) logits[(size_t)t * N + e] = v + (bias ? bias[e] : 0.0f);
  }
}

template <int NT>
static void launch_router_nt(const bf16_t *x, const bf16_t *wr, const float *bias, int T, int N, int d,
                             float *logits, hipStream_t s) {
  const int blocks = (T + 15) / 16;
  if (blocks < 512)
    router_logits_bf16<NT, 8><<<blocks, 512, 0, s>>>(x, wr, bias, T, N, d, logits);
  else
    router_logits_bf16<NT, 4><<<blocks, 256, 0, s>>>(x, wr, bias, T, N, d, logits);
}

__global__ __launch_bounds__(256) void router_logits_f32(const float *__restrict__ x,
                                                         const float *__restrict__ wr,
                                                         const float *__restrict__ bias, int T,
                                                         int N, int d, float *__restrict__ logits) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= T * N) return;
  const int t = idx / N, e = idx % N;
  const float *xr = x + (size_t)t * d;
  const float *wrow = wr + (size_t)e * d;
  float acc = 0.f;
  for (int k = 0; k < d; ++k) acc = fmaf(xr[k], wrow[k], acc);
  logits[idx] = acc + (bias ? bias[e] : 0.0f);
}

hipError_t launch_router_logits(int dtype, const void *x, const void *w_router, const float *bias,
                                int T, int N, int d, float *logits, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (dtype == EXFOLD_BF16) {
    const bf16_t *xb = static_cast<const bf16_t *>(x);
    const bf16_t *wb = static_cast<const bf16_t *>(w_router);
    const int nt = (N + 15) / 16;
    if (nt <= 1) launch_router_nt<1>(xb, wb, bias, T, N, d, logits, s);
    else if (nt <= 2) launch_router_nt<2>(xb, wb, bias, T, N, d, logits, s);
    else if (nt <= 4) launch_router_nt<4>(xb, wb, bias, T, N, d, logits, s);
    else if (nt <= 8) launch_router_nt<8>(xb, wb, bias, T, N, d, logits, s);
    else launch_router_nt<16>(xb, wb, bias, T, N, d, logits, s);
  } else {
    router_logits_f32<<<(T * N + 255) / 256, 256, 0, s>>>(
        static_cast<const float *>(x), static_cast<const float *>(w_router), bias, T, N, d, logits);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// One wave per token: Top-K, softmax, prefill selection, prefill fold.
// Lane k (< K) owns route k of the token.
// ---------------------------------------------------------------------------

// Top-K by (logit desc, id asc) over a row of N <= 256 logits; the softmax over
// the selected logits is evaluated in float64 and rounded once to float32.
__device__ __forceinline__ void wave_topk_softmax(const float *__restrict__ row, int N, int K,
                                                  int lane, int &my_id, float &my_w) {
  uint64_t key[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    key[j] = (e < N) ? ((uint64_t(float_key(row[e])) << 32) | uint64_t(0xffffffffu - uint32_t(e))) : 0ull;
  }
  my_id = 0;
  for (int k = 0; k < K; ++k) {
    uint64_t best = key[0];
#pragma unroll
    for (int j = 1; j < 4; ++j) best = key[j] > best ? key[j] : best;
    best = wave_max_u64(best);
    const int id = int(0xffffffffu - uint32_t(best & 0xffffffffu));
    if (lane == k) my_id = id;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane + 64 * j == id) key[j] = 0ull;
  }
  my_id = clamp_id(my_id, N);
  const double r = (double)row[my_id];
  const double r0 = shfl_f64(r, 0);  // route 0 holds the largest logit
  double z = (lane < K) ? exp(r - r0) : 0.0;
  double sum = z;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) sum += __shfl_xor(sum, m, kWave);
  my_w = (float)(z / sum);
}

__global__ __launch_bounds__(256) void route_tokens_kernel(
    const float *__restrict__ logits, int T, int N, int K, int k_pre, const float *__restrict__ h,
    const float *__restrict__ S, const float *__restrict__ L, int32_t *__restrict__ topk_ids,
    float *__restrict__ topk_w, uint8_t *__restrict__ keep, const uint8_t *__restrict__ keep_in,
    int32_t *__restrict__ fold_ids, float *__restrict__ fold_w) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;  // uniform per wave
  int my_id = 0;
  float my_w = 0.f;
  if (logits) {
    wave_topk_softmax(logits + (size_t)t * N, N, K, lane, my_id, my_w);
    if (lane < K) {
      topk_ids[(size_t)t * K + lane] = my_id;
      topk_w[(size_t)t * K + lane] = my_w;
    }
  } else if (lane < K) {
    my_id = clamp_id(topk_ids[(size_t)t * K + lane], N);
    my_w = topk_w[(size_t)t * K + lane];
  }
  if (!keep && !fold_ids) return;

  // Retained set: K' largest exact products w*h, ties to the smaller route position.
  bool kept;
  if (keep_in) {
    kept = (lane < K) && keep_in[(size_t)t * K + lane] != 0;
  } else {
    const double score = (lane < K) ? (double)my_w * (double)h[my_id] : 0.0;
    int rank = 0;
    for (int j = 0; j < K; ++j) {
      const double sj = shfl_f64(score, j);
      rank += (j != lane) && (sj > score || (sj == score && j < lane));
    }
    kept = (lane < K) && rank < k_pre;
    if (keep && lane < K) keep[(size_t)t * K + lane] = kept ? 1 : 0;
  }
  if (!fold_ids) return;

  // Broadcast the token's routes to every lane.
  const uint64_t kmask = __ballot(kept);
  int ids[kMaxTopK];
#pragma unroll
  for (int j = 0; j < kMaxTopK; ++j) ids[j] = __shfl(my_id, j < K ? j : 0, kWave);

  // Omitted route: first minimum of L[s, t] over the retained routes in route order.
  int tgt_lane = -1;
  double contrib = 0.0;
  if (lane < K && !kept) {
    const float *lrow = L + (size_t)my_id * N;
    float lv[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) lv[j] = (j < K && ((kmask >> j) & 1ull)) ? lrow[ids[j]] : 0.f;
    float best = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (j < K && ((kmask >> j) & 1ull)) {
        if (tgt_lane < 0 || lv[j] < best) {
          best = lv[j];
          tgt_lane = j;
        }
      }
    }
    if (tgt_lane >= 0) contrib = (double)my_w * (double)S[(size_t)my_id * N + ids[tgt_lane]];
  }
  // Coalesce onto each retained route, omitted routes in route order.
  double acc = (double)my_w;
  for (int j = 0; j < K; ++j) {
    const int tl = __shfl(tgt_lane, j, kWave);
    const double c = shfl_f64(contrib, j);
    if (tl == lane) acc += c;
  }
  // Retained routes in route order; a caller-supplied keep row with more than
  // k_out ones has its extra routes dropped (never written out of bounds).
  const int k_out = min(k_pre, K);
  const int p = __popcll(kmask & lanemask_lt(lane));
  if (kept && p < k_out) {
    fold_ids[(size_t)t * k_out + p] = my_id;
    fold_w[(size_t)t * k_out + p] = (float)acc;
  }
}

hipError_t launch_route_tokens(const float *logits, int T, int N, int K, int k_pre, const float *h,
                               const float *S, const float *L, int32_t *topk_ids, float *topk_w,
                               uint8_t *keep, const uint8_t *keep_in, int32_t *fold_ids,
                               float *fold_w, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  route_tokens_kernel<<<(T + 3) / 4, 256, 0, s>>>(logits, T, N, K, k_pre, h, S, L, topk_ids, topk_w,
                                                  keep, keep_in, fold_ids, fold_w);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Decode: batch pool (one workgroup) and per-source tables + per-slot remap.
// ---------------------------------------------------------------------------
constexpr int kPoolThreads = 1024;

__global__ __launch_bounds__(kPoolThreads) void decode_pool_fold_kernel(
    const int32_t *__restrict__ ids, const float *__restrict__ w, int B, int N, int K, int D,
    const float *__restrict__ h, const float *__restrict__ S, const float *__restrict__ L,
    int do_pool, int32_t *__restrict__ pool_g, int32_t *__restrict__ pool_size_g,
    int32_t *__restrict__ out_ids, float *__restrict__ out_w, int32_t *__restrict__ tgt_g,
    float *__restrict__ scl_g) {
  __shared__ unsigned long long wsum[kMaxExperts];
  __shared__ int cnt[kMaxExperts];
  __shared__ double score[kMaxExperts];
  __shared__ int pool[kMaxExperts];
  __shared__ int in_pool[kMaxExperts];
  __shared__ int tgt[kMaxExperts];
  __shared__ float scl[kMaxExperts];
  __shared__ int n_pool;
  const int tid = threadIdx.x;
  const int slots = B * K;
  const int dcap = min(D, N);

  if (tid < N) in_pool[tid] = 0;
  if (do_pool) {
    if (tid < N) {
      wsum[tid] = 0ull;
      cnt[tid] = 0;
    }
    __syncthreads();
    // W_e = sum of rint(w * 2^40) as an exact two's-complement integer.
    for (int j = tid; j < slots; j += kPoolThreads) {
      const int e = clamp_id(ids[j], N);
      const long long q = __double2ll_rn((double)w[j] * 1099511627776.0);  // 2^40
      atomicAdd(&wsum[e], (unsigned long long)q);
      atomicAdd(&cnt[e], 1);
    }
    __syncthreads();
    if (tid < N) score[tid] = (double)(long long)wsum[tid] * (double)h[tid];
    __syncthreads();
    int n_cand = 0;
    if (tid < N) {
      // rank among candidates by (score desc, id asc)
      int rank = 0;
      const bool cand = cnt[tid] > 0;
      const double sc = score[tid];
      for (int e = 0; e < N; ++e) {
        if (cnt[e] > 0) {
          ++n_cand;
          rank += (score[e] > sc) || (score[e] == sc && e < tid);
        }
      }
      if (cand && rank < dcap) {
        pool[rank] = tid;
        in_pool[tid] = 1;
      }
      if (tid == 0) n_pool = min(dcap, n_cand);
    }
    __syncthreads();
    if (tid < dcap) pool_g[tid] = (tid < n_pool) ? pool[tid] : -1;
    if (tid == 0) *pool_size_g = n_pool;
  } else {
    if (tid == 0) n_pool = max(0, min(*pool_size_g, dcap));
    __syncthreads();
    if (tid < n_pool) pool[tid] = clamp_id(pool_g[tid], N);
    __syncthreads();
    if (tid < n_pool) in_pool[pool[tid]] = 1;
  }
  __syncthreads();
  if (!out_ids && !tgt_g && !scl_g) return;

  // Per-source target: first minimum of L[s, t] over the pool in pool order.
  if (tid < N) {
    int t_best = tid;
    float s_best = 1.0f;
    if (!in_pool[tid] && n_pool > 0) {
      const float *lrow = L + (size_t)tid * N;
      t_best = pool[0];
      float best = lrow[t_best];
      for (int j = 1; j < n_pool; ++j) {
        const float v = lrow[pool[j]];
        if (v < best) {
          best = v;
          t_best = pool[j];
        }
      }
      s_best = S[(size_t)tid * N + t_best];
    }
    tgt[tid] = t_best;
    scl[tid] = s_best;
    if (tgt_g) tgt_g[tid] = t_best;
    if (scl_g) scl_g[tid] = s_best;
  }
  __syncthreads();
  // Per-slot remap; retained slots copied.
  if (!out_ids) return;
  for (int j = tid; j < slots; j += kPoolThreads) {
    const int e = clamp_id(ids[j], N);
    const float wv = w[j];
    out_ids[j] = tgt[e];
    out_w[j] = in_pool[e] ? wv : wv * scl[e];
  }
}

hipError_t launch_decode_pool_fold(const int32_t *ids, const float *w, int B, int N, int K, int D,
                                   const float *h, const float *S, const float *L, bool do_pool,
                                   int32_t *pool, int32_t *pool_size, int32_t *out_ids,
                                   float *out_w, int32_t *tgt, float *scl, hipStream_t s) {
  decode_pool_fold_kernel<<<1, kPoolThreads, 0, s>>>(ids, w, B, N, K, D, h, S, L, do_pool ? 1 : 0,
                                                     pool, pool_size, out_ids, out_w, tgt, scl);
  return hipGetLastError();
}

}  // namespace exfold

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
// Router logits, as P partial sums over slices of d (the bias and the sum of the
// partials are taken by the Top-K kernel, in a fixed order).  bf16: workgroup
// (bx, by, bz) takes 16*TT tokens x NT*16 experts x one d-slice; its KS waves
// split the slice, reduce with 16x16x32 bf16 MFMA (each weight fragment feeds TT
// token groups) and add their partial sums in a fixed order through LDS.  Many
// tokens: one block covers every expert (W_r is read once per 16*TT tokens); few tokens: 16 experts per block and the d axis split
// over the grid, so the small GEMM still spreads over the CUs.
// f32: one thread per logit.
// ---------------------------------------------------------------------------
template <int NT, int KS, int TT = 1>
__global__ __launch_bounds__(64 * KS) void router_logits_bf16(const bf16_t *__restrict__ x,
                                                              const bf16_t *__restrict__ wr,
                                                              int T, int N, int d, int d_slice,
                                                              float *__restrict__ part) {
  __shared__ float red[KS][TT * NT * 4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int t0 = blockIdx.x * 16 * TT;
  const int e0 = blockIdx.y * NT * 16;
  const int kq = (lane >> 4) * 8 + blockIdx.z * d_slice;
  f32x4 acc[TT][NT];
#pragma unroll
  for (int u = 0; u < TT; ++u)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[u][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16_t *wrow[NT];
  bool live[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int e = e0 + j * 16 + (lane & 15);
    live[j] = e < N;
    wrow[j] = wr + (size_t)(live[j] ? e : 0) * d + kq;
  }
  const bf16_t *xa[TT];
#pragma unroll
  for (int u = 0; u < TT; ++u) xa[u] = x + (size_t)min(t0 + u * 16 + (lane & 15), T - 1) * d + kq;
  const int steps = d_slice / 32;
  const int s0 = wave * steps / KS, s1 = (wave + 1) * steps / KS;
  const int npair = (s1 - s0) / 2;
  bf16x8 zero;
#pragma unroll
  for (int q = 0; q < 8; ++q) zero[q] = (__bf16)0.0f;
  for (int i = 0; i < npair; ++i) {
    const int k = (s0 + 2 * i) * 32;
    bf16x8 a0[TT], a1[TT], b0[NT], b1[NT];
#pragma unroll
    for (int u = 0; u < TT; ++u) {
      a0[u] = *reinterpret_cast<const bf16x8 *>(xa[u] + k);
      a1[u] = *reinterpret_cast<const bf16x8 *>(xa[u] + k + 32);
    }
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      b0[j] = *reinterpret_cast<const bf16x8 *>(wrow[j] + k);
      b1[j] = *reinterpret_cast<const bf16x8 *>(wrow[j] + k + 32);
    }
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int u = 0; u < TT; ++u) {
        acc[u][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], live[j] ? b0[j] : zero, acc[u][j], 0, 0, 0);
        acc[u][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[u], live[j] ? b1[j] : zero, acc[u][j], 0, 0, 0);
      }
  }
  if ((s1 - s0) & 1) {
    const int k = (s1 - 1) * 32;
    bf16x8 a0[TT];
#pragma unroll
    for (int u = 0; u < TT; ++u) a0[u] = *reinterpret_cast<const bf16x8 *>(xa[u] + k);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(wrow[j] + k);
#pragma unroll
      for (int u = 0; u < TT; ++u)
        acc[u][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], live[j] ? b0 : zero, acc[u][j], 0, 0, 0);
    }
  }
#pragma unroll
  for (int u = 0; u < TT; ++u)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][(u * NT + j) * 4 + i][lane] = acc[u][j][i];
  __syncthreads();
  float *out = part + (size_t)blockIdx.z * T * N;
  for (int idx = threadIdx.x; idx < TT * NT * 4 * 64; idx += 64 * KS) {
    const int ji = idx >> 6, l = idx & 63;
    const int u = ji / (NT * 4), j = (ji >> 2) % NT, i = ji & 3;
    float v = red[0][ji][l];
#pragma unroll
    for (int w = 1; w < KS; ++w) v += red[w][ji][l];
    const int t = t0 + u * 16 + (l >> 4) * 4 + i;
    const int e = e0 + j * 16 + (l & 15);
    if (t < T && e < N) out[(size_t)t * N + e] = v;
  }
}

// Many tokens and many experts: 32 tokens per workgroup, one wave per 16
// experts owning its experts over the whole of d (no cross-wave reduction).
// The tokens' x rows pass through LDS in chunks of 256 along d (double
// buffered, loaded one chunk ahead through registers); each wave streams its
// W_r rows from global (L2-resident), the next chunk's fragments in flight
// during the current chunk's MFMAs.  One pass writes the logits (P = 1).
constexpr int kRlTok = 32, kRlChunk = 256, kRlPad = 8;
constexpr int kRlRow = kRlChunk + kRlPad;  // LDS row stride (bf16): 16 rows of one read spread over the banks

template <int NW>
__global__ __launch_bounds__(64 * NW) void router_logits_lds(const bf16_t *__restrict__ x,
                                                            const bf16_t *__restrict__ wr, int T, int N,
                                                            int d, float *__restrict__ out) {
  __shared__ __attribute__((aligned(16))) bf16_t xs[2][kRlTok * kRlRow];
  constexpr int kThreads = 64 * NW;
  constexpr int kChunks16 = kRlTok * kRlChunk / 8;           // 16-byte pieces of one x chunk
  constexpr int kPer = (kChunks16 + kThreads - 1) / kThreads;  // per thread
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int t0 = blockIdx.x * kRlTok;
  const int e = wave * 16 + (lane & 15);
  const bool live = e < N;
  const bf16_t *wrow = wr + (size_t)(live ? e : 0) * d + (lane >> 4) * 8;
  const int nch = d / kRlChunk;

  u32x4 xr[kPer];
  auto load_x = [&](int ch) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = i * kThreads + tid;
      if (c < kChunks16) {
        const int r = c / (kRlChunk / 8), q = c % (kRlChunk / 8);
        const int t = min(t0 + r, T - 1);
        xr[i] = *reinterpret_cast<const u32x4 *>(x + (size_t)t * d + ch * kRlChunk + q * 8);
      }
    }
  };
  auto store_x = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = i * kThreads + tid;
      if (c < kChunks16) {
        const int r = c / (kRlChunk / 8), q = c % (kRlChunk / 8);
        *reinterpret_cast<u32x4 *>(&xs[buf][r * kRlRow + q * 8]) = xr[i];
      }
    }
  };
  constexpr int kSteps = kRlChunk / 32;
  auto load_w = [&](int ch, bf16x8 (&dst)[kSteps]) {
#pragma unroll
    for (int k = 0; k < kSteps; ++k)
      dst[k] = *reinterpret_cast<const bf16x8 *>(wrow + ch * kRlChunk + k * 32);
  };
  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  bf16x8 zero;
#pragma unroll
  for (int q = 0; q < 8; ++q) zero[q] = (__bf16)0.0f;
  auto compute = [&](int buf, const bf16x8 (&wb)[kSteps]) {
    const bf16_t *xa = &xs[buf][(lane & 15) * kRlRow + (lane >> 4) * 8];
#pragma unroll
    for (int k = 0; k < kSteps; ++k) {
      const bf16x8 b = live ? wb[k] : zero;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(xa + u * 16 * kRlRow + k * 32);
        acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[u], 0, 0, 0);
      }
    }
  };
  // chunk ch: its W_r fragments were loaded one chunk ahead (wb0 for even
  // chunks, wb1 for odd), its x rows stored to LDS buffer ch & 1 before the
  // barrier that ends chunk ch - 1
  bf16x8 wb0[kSteps], wb1[kSteps];
  load_x(0);
  load_w(0, wb0);
  store_x(0);
  if (nch > 1) load_x(1);
  __syncthreads();
  for (int ch = 0; ch < nch; ch += 2) {
    if (ch + 1 < nch) load_w(ch + 1, wb1);
    compute(0, wb0);
    if (ch + 1 < nch) {
      store_x(1);
      if (ch + 2 < nch) load_x(ch + 2);
    }
    __syncthreads();
    if (ch + 1 >= nch) break;
    if (ch + 2 < nch) load_w(ch + 2, wb0);
    compute(1, wb1);
    if (ch + 2 < nch) {
      store_x(0);
      if (ch + 3 < nch) load_x(ch + 3);
    }
    __syncthreads();
  }
  // acc[u][i]: token t0 + 16 u + 4 (lane / 16) + i, expert e
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = t0 + u * 16 + (lane >> 4) * 4 + i;
      if (t < T && live) out[(size_t)t * N + e] = acc[u][i];
    }
}

// Blocks of the all-experts layout at or above which the d axis is not split.
constexpr int kRouterWideBlocks = 64;

// Many tokens and a multiple of 128 experts: the router is a plain MFMA GEMM
// on 128 x 128 tiles with its reduction split so the tiles cover the CUs
// (8192 tokens x 128 experts x 2048: 256 tiles of 512-deep reductions).
static bool router_tiled(int T, int N, int d) {
  return (T + 15) / 16 >= kRouterWideBlocks && plain_gemm_splits(T, N, d, 256) > 0;
}

int router_splits(int dtype, int T, int N, int d) {
  if (dtype != EXFOLD_BF16 || T <= 0) return 1;
  if (router_tiled(T, N, d)) return plain_gemm_splits(T, N, d, 256);
  const int tb = (T + 15) / 16;
  if (tb >= kRouterWideBlocks) return 1;
  const int nb = (N + 15) / 16;
  int P = 1;
  // split d (slices of >= 256, multiples of 32) until the grid covers ~256 CUs
  while (tb * nb * P < 256 && d % (64 * P) == 0 && d / (2 * P) >= 256) P *= 2;
  return P;
}

template <int NT>
static void launch_router_wide(const bf16_t *x, const bf16_t *wr, int T, int N, int d, float *part,
                               hipStream_t s) {
  if constexpr (NT >= 4 && NT <= 8) {
    // 32 tokens per workgroup: each weight row piece is fetched once per 32
    // tokens; 8192 tokens x 128 experts x 2048 took 43 us with 16 tokens and
    // four waves, 29 us like this (64 tokens per workgroup: 48 us)
    router_logits_bf16<NT, 8, 2><<<dim3((T + 31) / 32, 1, 1), 512, 0, s>>>(x, wr, T, N, d, d, part);
    return;
  }
  const int blocks = (T + 15) / 16;
  if (blocks < 512)
    router_logits_bf16<NT, 8><<<dim3(blocks, 1, 1), 512, 0, s>>>(x, wr, T, N, d, d, part);
  else
    router_logits_bf16<NT, 4><<<dim3(blocks, 1, 1), 256, 0, s>>>(x, wr, T, N, d, d, part);
}

__global__ __launch_bounds__(256) void router_logits_f32(const float *__restrict__ x,
                                                         const float *__restrict__ wr, int T,
                                                         int N, int d, float *__restrict__ part) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= T * N) return;
  const int t = idx / N, e = idx % N;
  const float *xr = x + (size_t)t * d;
  const float *wrow = wr + (size_t)e * d;
  float acc = 0.f;
  for (int k = 0; k < d; ++k) acc = fmaf(xr[k], wrow[k], acc);
  part[idx] = acc;
}

hipError_t launch_router_logits(int dtype, const void *x, const void *w_router, int T, int N, int d,
                                int P, float *part, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (dtype == EXFOLD_BF16) {
    const bf16_t *xb = static_cast<const bf16_t *>(x);
    const bf16_t *wb = static_cast<const bf16_t *>(w_router);
    const int tb = (T + 15) / 16;
    if (router_tiled(T, N, d)) {
      if (P != plain_gemm_splits(T, N, d, 256)) return hipErrorInvalidValue;
      return launch_plain_gemm_nt(xb, wb, T, N, d, P, part, s);
    }
    if (tb < kRouterWideBlocks) {
      // 16 tokens x 16 experts x d/P per block
      const dim3 grid(tb, (N + 15) / 16, P);
      router_logits_bf16<1, 4><<<grid, 256, 0, s>>>(xb, wb, T, N, d, d / P, part);
    } else if (N > 32 && d % kRlChunk == 0) {
      // one wave per 16 experts over the whole of d
      const int nt = (N + 15) / 16, grid = (T + kRlTok - 1) / kRlTok;
      if (nt <= 4) router_logits_lds<4><<<grid, 256, 0, s>>>(xb, wb, T, N, d, part);
      else if (nt <= 8) router_logits_lds<8><<<grid, 512, 0, s>>>(xb, wb, T, N, d, part);
      else router_logits_lds<16><<<grid, 1024, 0, s>>>(xb, wb, T, N, d, part);
    } else {
      const int nt = (N + 15) / 16;
      if (nt <= 1) launch_router_wide<1>(xb, wb, T, N, d, part, s);
      else if (nt <= 2) launch_router_wide<2>(xb, wb, T, N, d, part, s);
      else if (nt <= 4) launch_router_wide<4>(xb, wb, T, N, d, part, s);
      else if (nt <= 8) launch_router_wide<8>(xb, wb, T, N, d, part, s);
      else launch_router_wide<16>(xb, wb, T, N, d, part, s);
    }
  } else {
    router_logits_f32<<<(T * N + 255) / 256, 256, 0, s>>>(
        static_cast<const float *>(x), static_cast<const float *>(w_router), T, N, d, part);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// One wave per token: Top-K, softmax, prefill selection, prefill fold.
// Lane k (< K) owns route k of the token.
// ---------------------------------------------------------------------------

// Logit row of token t: the P partial sums in order, then the bias; lane holds
// experts lane + 64 j.  The row is also written to `out` when given.
__device__ __forceinline__ void wave_logit_row(const float *__restrict__ part, int P, int T, int N,
                                               const float *__restrict__ bias, int t, int lane,
                                               float *__restrict__ out, float v[4]) {
  // the slices are loaded eight at a time (one latency per eight) and added in order
  constexpr int kBatch = 8;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int e = lane + 64 * j;
    float a = 0.f;
    if (e < N) {
      const float *col = part + (size_t)t * N + e;
      const size_t zs = (size_t)T * N;
      for (int z0 = 0; z0 < P; z0 += kBatch) {
        float pv[kBatch];
#pragma unroll
        for (int b = 0; b < kBatch; ++b) pv[b] = (z0 + b < P) ? col[(size_t)(z0 + b) * zs] : 0.f;
#pragma unroll
        for (int b = 0; b < kBatch; ++b)
          if (z0 + b < P) a = (z0 + b == 0) ? pv[b] : a + pv[b];
      }
      if (bias) a += bias[e];
      if (out) out[(size_t)t * N + e] = a;
    }
    v[j] = a;
  }
}

// Top-K by (logit desc, id asc) over a row of N <= 256 logits (lane holds
// experts lane + 64 j); the softmax over the selected logits is evaluated in
// float64 and rounded once to float32.
__device__ __forceinline__ void wave_topk_softmax(const float v[4], int N, int K, int lane,
                                                  int &my_id, float &my_w) {
  // 32-bit order keys (0 marks a taken or absent expert); each round takes the
  // wave maximum with DPP, then the smallest expert id holding it from ballots
  // (ids lane + 64 j grow with j, then with the lane)
  uint32_t key[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) key[j] = (lane + 64 * j < N) ? float_key(v[j]) : 0u;
  my_id = 0;
  for (int k = 0; k < K; ++k) {
    const uint32_t best = wave_max_u32(max(max(key[0], key[1]), max(key[2], key[3])));
    int id = 0;
    bool found = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint64_t m = __ballot(key[j] == best);
      if (!found && m != 0ull) {
        id = 64 * j + (int)__builtin_ctzll(m);
        found = true;
      }
    }
    if (lane == k) my_id = id;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane + 64 * j == id) key[j] = 0u;
  }
  my_id = clamp_id(my_id, N);
  // logit of my route: held by lane my_id % 64 in register my_id / 64
  const int src = my_id & 63, reg = my_id >> 6;
  const float c0 = __shfl(v[0], src, kWave), c1 = __shfl(v[1], src, kWave);
  const float c2 = __shfl(v[2], src, kWave), c3 = __shfl(v[3], src, kWave);
  const double r = (double)(reg == 0 ? c0 : reg == 1 ? c1 : reg == 2 ? c2 : c3);
  const double r0 = readlane_f64(r, 0);  // route 0 holds the largest logit
  const double z = (lane < K) ? exp(r - r0) : 0.0;
  const double sum = wave_sum_f64(z);
  my_w = (float)(z / sum);
}

// Per-token routing arguments (see launch_route_tokens).
struct RouteArgs {
  int T, N, K, k_pre;
  const float *h, *S, *L;
  int32_t *topk_ids;
  float *topk_w;
  uint8_t *keep;
  const uint8_t *keep_in;
  int32_t *fold_ids;
  float *fold_w;
  float loss_cap;
  int flags;
  int32_t *om_src;
  float *om_w;
  int32_t *om_q;
  float *wret;
};

// One wave routes token t: Top-K and softmax of its logit row v (lane holds
// experts lane + 64 j; have_v false: the routes are read from topk_ids/w),
// then the prefill selection and fold.  hv: h of experts lane + 64 j.
__device__ __forceinline__ void route_token_wave(const RouteArgs &a, int t, int lane, bool have_v,
                                                 const float (&v)[4], const float (&hv)[4]) {
  const int N = a.N, K = a.K, k_pre = a.k_pre;
  const float *__restrict__ S = a.S, *__restrict__ L = a.L;
  int32_t *__restrict__ topk_ids = a.topk_ids;
  float *__restrict__ topk_w = a.topk_w;
  uint8_t *__restrict__ keep = a.keep;
  const uint8_t *__restrict__ keep_in = a.keep_in;
  int32_t *__restrict__ fold_ids = a.fold_ids;
  float *__restrict__ fold_w = a.fold_w;
  const float loss_cap = a.loss_cap;
  const int flags = a.flags;
  int32_t *__restrict__ om_src = a.om_src;
  float *__restrict__ om_w = a.om_w;
  int32_t *__restrict__ om_q = a.om_q;
  float *__restrict__ wret = a.wret;
  int my_id = 0;
  float my_w = 0.f;
  if (have_v) {
    wave_topk_softmax(v, N, K, lane, my_id, my_w);
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
    // h of my route: held by lane my_id % 64 in register my_id / 64
    const int hs = my_id & 63, hr = my_id >> 6;
    const float h0 = __shfl(hv[0], hs, kWave), h1 = __shfl(hv[1], hs, kWave);
    const float h2 = __shfl(hv[2], hs, kWave), h3 = __shfl(hv[3], hs, kWave);
    const float h_my = hr == 0 ? h0 : hr == 1 ? h1 : hr == 2 ? h2 : h3;
    const double score = (lane < K) ? (double)my_w * (double)h_my : 0.0;
    int rank = 0;
    for (int j = 0; j < K; ++j) {
      const double sj = readlane_f64(score, j);
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
  for (int j = 0; j < kMaxTopK; ++j) ids[j] = (int)readlane_u32((uint32_t)my_id, j < K ? j : 0);

  // Omitted route: first minimum of L[s, t] over the retained routes in route
  // order (with the loss cap: over those with L[s, t] <= cap; none -> dropped).
  // Safeguard arithmetic is float64 with explicit roundings (no fused
  // multiply-add), in the order the fold is defined in.
  const bool capped = flags & EXFOLD_FOLD_LOSS_CAP, conf = flags & EXFOLD_FOLD_CONFIDENCE;
  int tgt_lane = -1;
  double contrib = 0.0, rest = 0.0;
  if (lane < K && !kept) {
    // L and S of every candidate target loaded together (one round trip)
    const float *lrow = L + (size_t)my_id * N;
    const float *srow = S ? S + (size_t)my_id * N : nullptr;
    float lv[kMaxTopK], sv[kMaxTopK];
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      const bool cand = j < K && ((kmask >> j) & 1ull);
      lv[j] = cand ? lrow[ids[j]] : 0.f;
      sv[j] = (cand && srow && !om_src) ? srow[ids[j]] : 0.f;
    }
    float best = 0.f, s_best = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxTopK; ++j) {
      if (j < K && ((kmask >> j) & 1ull) && (!capped || lv[j] <= loss_cap)) {
        if (tgt_lane < 0 || lv[j] < best) {
          best = lv[j];
          s_best = sv[j];
          tgt_lane = j;
        }
      }
    }
    if (tgt_lane >= 0 && !om_src) {
      double c = 1.0;
      if (conf) c = fmin(1.0, fmax(0.0, __dsub_rn(1.0, (double)best)));
      contrib = __dmul_rn(__dmul_rn((double)my_w, c), (double)s_best);
      if (conf) rest = __dmul_rn((double)my_w, __dsub_rn(1.0, c));
    }
  }
  // Diagonal projectors (unfused path): the retained routes execute with weight
  // 1 and keep their router weights aside; each omitted route records its
  // source, weight and the position of its target among the retained routes.
  if (om_src) {
    const int k_out = min(k_pre, K);
    const int p = __popcll(kmask & lanemask_lt(lane));
    if (kept && p < k_out) {
      fold_ids[(size_t)t * k_out + p] = my_id;
      fold_w[(size_t)t * k_out + p] = 1.0f;
      wret[(size_t)t * k_out + p] = my_w;
    }
    if (lane < K) {
      const int qpos = (!kept && tgt_lane >= 0) ? __popcll(kmask & lanemask_lt(tgt_lane)) : -1;
      om_src[(size_t)t * K + lane] = kept ? -1 : my_id;
      om_w[(size_t)t * K + lane] = my_w;
      om_q[(size_t)t * K + lane] = qpos;
    }
    return;
  }
  // Coalesce onto each retained route, omitted routes in route order: the
  // target's share, then (confidence split) the spread w_s (1 - c_s) w_t / W_ret.
  double w_ret = 0.0;
  if (conf)
    for (int j = 0; j < K; ++j)
      if ((kmask >> j) & 1ull) w_ret = __dadd_rn(w_ret, (double)readlane_f32(my_w, j));
  const double share = (conf && kept) ? __ddiv_rn((double)my_w, w_ret) : 0.0;
  double acc = (double)my_w;
  for (int j = 0; j < K; ++j) {
    const int tl = (int)readlane_u32((uint32_t)tgt_lane, j);
    const double c = readlane_f64(contrib, j);
    const double r = readlane_f64(rest, j);
    if (tl == lane) acc = __dadd_rn(acc, c);
    if (conf && tl >= 0 && kept) acc = __dadd_rn(acc, __dmul_rn(r, share));
  }
  // Renormalisation: scale the retained weights to the sum of the K router weights.
  if (flags & EXFOLD_FOLD_RENORM) {
    double w_all = 0.0, tot = 0.0;
    for (int j = 0; j < K; ++j) {
      w_all = __dadd_rn(w_all, (double)readlane_f32(my_w, j));
      const double a = readlane_f64(acc, j);
      if ((kmask >> j) & 1ull) tot = __dadd_rn(tot, a);
    }
    if (tot > 0.0) acc = __dmul_rn(acc, __ddiv_rn(w_all, tot));
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

__global__ __launch_bounds__(256) void route_tokens_kernel(const float *__restrict__ part, int P,
                                                          const float *__restrict__ bias,
                                                          float *__restrict__ logits_out, const RouteArgs a) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= a.T) return;  // uniform per wave
  // h of experts lane + 64 j, loaded with the logits (no load after Top-K)
  float hv[4] = {0.f, 0.f, 0.f, 0.f};
  if (a.h && !a.keep_in) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (lane + 64 * j < a.N) hv[j] = a.h[lane + 64 * j];
  }
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (part) wave_logit_row(part, P, a.T, a.N, bias, t, lane, logits_out, v);
  route_token_wave(a, t, lane, part != nullptr, v, hv);
}

// Routers of at most 32 experts (bf16): one workgroup per token computes its N
// logits (each thread a 16-byte slice of d per step against every expert,
// then a fixed-order tree: DPP inside each wave, the four waves in order)
// and wave 0 routes the token as route_tokens_kernel does.  One launch
// replaces the router and Top-K kernels; W_r (<= 32 d elements) stays in L2.
constexpr int kRouteSmallMaxT = 1024;  // route_small_kernel: one workgroup per token up to this batch

template <int NM>
__global__ __launch_bounds__(256) void route_small_kernel(const bf16_t *__restrict__ x,
                                                         const bf16_t *__restrict__ wr, int d,
                                                         const float *__restrict__ bias,
                                                         float *__restrict__ logits_out, const RouteArgs a) {
  __shared__ float red[4][NM];
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int N = a.N;
  float hv[4] = {0.f, 0.f, 0.f, 0.f};
  if (wave == 0 && a.h && !a.keep_in && lane < N) hv[0] = a.h[lane];
  float acc[NM];
#pragma unroll
  for (int e = 0; e < NM; ++e) acc[e] = 0.f;
  const bf16_t *xr = x + (size_t)t * d;
  // two 16-byte steps of d per round, every load of the round issued first
  constexpr int kU = NM <= 8 ? 2 : 1;
  for (int k0 = tid * 8; k0 < d; k0 += kU * 256 * 8) {
    u32x4 xu[kU], wu[kU][NM];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int k = k0 + u * 256 * 8;
      if (k < d) {
        xu[u] = *reinterpret_cast<const u32x4 *>(xr + k);
#pragma unroll
        for (int e = 0; e < NM; ++e)
          if (e < N) wu[u][e] = *reinterpret_cast<const u32x4 *>(wr + (size_t)e * d + k);
      }
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      if (k0 + u * 256 * 8 >= d) break;
      float xf[8];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        xf[2 * q] = __uint_as_float(xu[u][q] << 16);
        xf[2 * q + 1] = __uint_as_float(xu[u][q] & 0xffff0000u);
      }
#pragma unroll
      for (int e = 0; e < NM; ++e)
        if (e < N) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            acc[e] = fmaf(xf[2 * q], __uint_as_float(wu[u][e][q] << 16), acc[e]);
            acc[e] = fmaf(xf[2 * q + 1], __uint_as_float(wu[u][e][q] & 0xffff0000u), acc[e]);
          }
        }
    }
  }
#pragma unroll
  for (int e = 0; e < NM; ++e)
    if (e < N) {
      const float sum = wave_sum_f32(acc[e]);
      if (lane == 0) red[wave][e] = sum;
    }
  __syncthreads();
  if (wave != 0) return;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (lane < N) {
    float l = ((red[0][lane] + red[1][lane]) + red[2][lane]) + red[3][lane];
    if (bias) l += bias[lane];
    v[0] = l;
    if (logits_out) logits_out[(size_t)t * N + lane] = l;
  }
  route_token_wave(a, t, lane, true, v, hv);
}

// Up to about a thousand tokens: beyond that, the per-token reads of W_r cost
// more than the separate router kernel (4096 Mixtral-shaped tokens: 27 us
// against 11 + 9 us; 32 tokens: 6.8 us against 5.3 + 5.8 us).
// Beyond that batch size (few experts, many tokens): one workgroup per 16
// tokens takes their logits over the whole of d with 16x16x32 MFMAs (KS waves
// on consecutive ranges of d, the partial tiles added in wave order through
// LDS), adds the bias, and its waves then route the tokens (route_token_wave):
// no Top-K launch and no logit rows in memory.  Every workgroup reads all of W_r (64 KiB for the
// Mixtral-shaped layer), so this is for few experts only (at 128 experts the
// same kernel made decode layers 13-27 us slower than the d-split router).
template <int NT, int KS>
__global__ __launch_bounds__(64 * KS) void route_block_kernel(const bf16_t *__restrict__ x,
                                                              const bf16_t *__restrict__ wr, int d,
                                                              const float *__restrict__ bias,
                                                              float *__restrict__ logits_out, const RouteArgs a) {
  __shared__ float red[KS][NT * 4][64];
  __shared__ float lg[16][16 * NT];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int T = a.T, N = a.N;
  const int t0 = blockIdx.x * 16;
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
  const bf16_t *xa = x + (size_t)min(t0 + (lane & 15), T - 1) * d + kq;
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
  // accumulator i of lane l: token (l / 16) * 4 + i, expert 16 j + l % 16
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][j * 4 + i][lane] = acc[j][i];
  __syncthreads();
  for (int idx = threadIdx.x; idx < NT * 4 * 64; idx += 64 * KS) {
    const int ji = idx >> 6, l = idx & 63;
    float v = red[0][ji][l];
#pragma unroll
    for (int w = 1; w < KS; ++w) v += red[w][ji][l];
    const int tl = (l >> 4) * 4 + (ji & 3), e = (ji >> 2) * 16 + (l & 15);
    if (e < N) {
      if (bias) v += bias[e];
      lg[tl][e] = v;
      if (logits_out && t0 + tl < T) logits_out[(size_t)(t0 + tl) * N + e] = v;
    }
  }
  __syncthreads();
  float hv[4] = {0.f, 0.f, 0.f, 0.f};
  if (a.h && !a.keep_in && lane < N) hv[0] = a.h[lane];
  for (int tl = wave; tl < 16 && t0 + tl < T; tl += KS) {
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (lane < N) v[0] = lg[tl][lane];
    route_token_wave(a, t0 + tl, lane, true, v, hv);
  }
}

bool route_small_fits(int dtype, int N, int T) { return dtype == EXFOLD_BF16 && N <= 32; }

hipError_t launch_route_small(const void *x, const void *w_router, int d, const float *bias,
                              float *logits_out, int T, int N, int K, int k_pre, const float *h,
                              const float *S, const float *L, int32_t *topk_ids, float *topk_w,
                              uint8_t *keep, int32_t *fold_ids, float *fold_w, hipStream_t s,
                              float loss_cap, int flags, int32_t *om_src, float *om_w, int32_t *om_q,
                              float *wret) {
  if (T <= 0) return hipSuccess;
  const RouteArgs a{T, N, K, k_pre, h, S, L, topk_ids, topk_w, keep, nullptr, fold_ids, fold_w,
                    loss_cap, flags, om_src, om_w, om_q, wret};
  const bf16_t *xb = static_cast<const bf16_t *>(x), *wb = static_cast<const bf16_t *>(w_router);
  if (T > kRouteSmallMaxT) {
    const int blocks = (T + 15) / 16;
    // sixteen waves: one token each to route (eight waves routing two each: 19.4 against 16.0 us
    // for the Mixtral-shaped prefill's 4096 tokens)
    if (N <= 16) route_block_kernel<1, 16><<<blocks, 1024, 0, s>>>(xb, wb, d, bias, logits_out, a);
    else route_block_kernel<2, 16><<<blocks, 1024, 0, s>>>(xb, wb, d, bias, logits_out, a);
  } else if (N <= 8) route_small_kernel<8><<<T, 256, 0, s>>>(xb, wb, d, bias, logits_out, a);
  else if (N <= 16) route_small_kernel<16><<<T, 256, 0, s>>>(xb, wb, d, bias, logits_out, a);
  else route_small_kernel<32><<<T, 256, 0, s>>>(xb, wb, d, bias, logits_out, a);
  return hipGetLastError();
}

hipError_t launch_route_tokens(const float *part, int P, const float *bias, float *logits_out, int T,
                               int N, int K, int k_pre, const float *h, const float *S, const float *L,
                               int32_t *topk_ids, float *topk_w, uint8_t *keep,
                               const uint8_t *keep_in, int32_t *fold_ids, float *fold_w,
                               hipStream_t s, float loss_cap, int flags, int32_t *om_src,
                               float *om_w, int32_t *om_q, float *wret) {
  if (T <= 0) return hipSuccess;
  const RouteArgs a{T, N, K, k_pre, h, S, L, topk_ids, topk_w, keep, keep_in, fold_ids, fold_w,
                    loss_cap, flags, om_src, om_w, om_q, wret};
  route_tokens_kernel<<<(T + 3) / 4, 256, 0, s>>>(part, P, bias, logits_out, a);
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

// Per-source tables of a decode pool (Eq. minimum_loss_assignment over the
// pool): a source in the pool maps to itself with scale 1, any other source to
// the first minimum of L[s, t] over the pool in pool order, with scale S[s, t].
// Thread (s, p) = (tid / P, tid % P) reads L and S at the pool members
// p, p + P, ... (P = threads per source, all its loads in flight together) and
// keeps its first minimum as a 64-bit key (value, pool position); an LDS
// atomic min per source combines the threads, and the one thread whose key won
// writes the target and its scale.  Called by the whole workgroup (it holds
// two barriers); pool/in_pool/n_pool in LDS; writes tgt/scl (LDS) and
// tgt_g/scl_g (either may be NULL).  need (LDS, or NULL for every source):
// only sources with need[s] > 0 get tables (the routed ones, when no table
// output is asked for: no other entry is read).
__device__ void pool_tables(int N, const float *__restrict__ S, const float *__restrict__ L,
                            const int *pool, const int *in_pool, int n_pool, int *tgt, float *scl,
                            int32_t *__restrict__ tgt_g, float *__restrict__ scl_g,
                            const int *need = nullptr) {
  constexpr int kBatch = 8;  // loads in flight per thread
  __shared__ unsigned long long best[kMaxExperts];
  const int tid = threadIdx.x;
  const int P = kPoolThreads / N;  // N <= kMaxExperts <= kPoolThreads / 4
  // the P threads of one source are adjacent, so a wave's loads stay within a
  // few rows of L and S (few cache lines per load instruction)
  const int src = tid / P, part = tid % P;
  const bool mine = src < N && (need == nullptr || need[src] > 0);
  if (tid < N) best[tid] = ~0ull;
  __syncthreads();
  uint64_t key = ~0ull;
  float s_key = 1.0f;
  if (mine && !in_pool[src]) {
    const float *lrow = L + (size_t)src * N, *srow = S + (size_t)src * N;
    for (int j0 = part; j0 < n_pool; j0 += kBatch * P) {
      float lv[kBatch], sv[kBatch];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int j = j0 + b * P;
        lv[b] = 0.f;
        sv[b] = 0.f;
        if (j < n_pool) {
          const int t = pool[j];
          lv[b] = lrow[t];
          sv[b] = srow[t];
        }
      }
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const int j = j0 + b * P;
        const uint64_t k = (uint64_t(float_key(lv[b])) << 32) | uint64_t(uint32_t(j));
        if (j < n_pool && k < key) {
          key = k;
          s_key = sv[b];
        }
      }
    }
    if (key != ~0ull) atomicMin(&best[src], (unsigned long long)key);
  }
  __syncthreads();
  if (!mine) return;
  int t_out = -1;
  float s_out = 1.0f;
  if (in_pool[src] || n_pool == 0) {
    if (part == 0) t_out = src;  // maps to itself
  } else if (key != ~0ull && key == best[src]) {
    t_out = pool[(int)(key & 0xffffffffu)];
    s_out = s_key;
  }
  if (t_out >= 0) {
    tgt[src] = t_out;
    scl[src] = s_out;
    if (tgt_g) tgt_g[src] = t_out;
    if (scl_g) scl_g[src] = s_out;
  }
}

// Static decode pool (Appendix B, Eq. appendix_decode_static_budget): the D
// experts of largest h (ties to the lower id) and its per-source tables, formed
// once; a decode step then only gathers (Eq. appendix_decode_remap).
__global__ __launch_bounds__(kPoolThreads) void static_pool_kernel(
    const float *__restrict__ h, int N, int D, const float *__restrict__ S,
    const float *__restrict__ L, int32_t *__restrict__ pool_g, int32_t *__restrict__ pool_size_g,
    int32_t *__restrict__ tgt_g, float *__restrict__ scl_g) {
  __shared__ float hv[kMaxExperts];
  __shared__ int pool[kMaxExperts];
  __shared__ int in_pool[kMaxExperts];
  __shared__ int tgt[kMaxExperts];
  __shared__ float scl[kMaxExperts];
  const int tid = threadIdx.x;
  const int dcap = min(D, N);
  if (tid < N) {
    hv[tid] = h[tid];
    in_pool[tid] = 0;
  }
  __syncthreads();
  if (tid < N) {
    const float v = hv[tid];
    int rank = 0;
    for (int e = 0; e < N; ++e) rank += (hv[e] > v) || (hv[e] == v && e < tid);
    if (rank < dcap) {
      pool[rank] = tid;
      in_pool[tid] = 1;
    }
  }
  __syncthreads();
  if (tid < dcap) pool_g[tid] = pool[tid];
  if (tid == 0) *pool_size_g = dcap;
  pool_tables(N, S, L, pool, in_pool, dcap, tgt, scl, tgt_g, scl_g);
}

// Per-slot remap with precomputed static tables (Eq. appendix_decode_remap):
// the grid-wide form for batches beyond the one-workgroup front end.
__global__ __launch_bounds__(256) void static_remap_kernel(const int32_t *__restrict__ ids,
                                                           const float *__restrict__ w, int slots,
                                                           int N, const int32_t *__restrict__ tgt,
                                                           const float *__restrict__ scl,
                                                           int32_t *__restrict__ out_ids,
                                                           float *__restrict__ out_w) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= slots) return;
  const int e = clamp_id(ids[j], N);
  const int te = clamp_id(tgt[e], N);
  out_ids[j] = te;
  out_w[j] = (te == e) ? w[j] : w[j] * scl[e];
}

hipError_t launch_static_remap(const int32_t *ids, const float *w, int slots, int N,
                               const int32_t *tgt, const float *scl, int32_t *out_ids, float *out_w,
                               hipStream_t s) {
  if (slots <= 0) return hipSuccess;
  static_remap_kernel<<<(slots + 255) / 256, 256, 0, s>>>(ids, w, slots, N, tgt, scl, out_ids, out_w);
  return hipGetLastError();
}

hipError_t launch_static_pool(const float *h, int N, int D, const float *S, const float *L,
                              int32_t *pool, int32_t *pool_size, int32_t *tgt, float *scl,
                              hipStream_t s) {
  static_pool_kernel<<<1, kPoolThreads, 0, s>>>(h, N, D, S, L, pool, pool_size, tgt, scl);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Decode front end in one workgroup, after the per-token Top-K: the batch pool,
// the per-source tables, the remap of every slot and the stable permutation of
// the remapped slots by expert (the same outputs as the separate pool/fold and
// permutation kernels), so a decode step launches one kernel between Top-K and
// the expert GEMMs.  The [B, K] slots stay in LDS after one read.
// ---------------------------------------------------------------------------
constexpr int kFrontWaves = kPoolThreads / kWave;
// Up to this many experts the front end loads each thread's share of L and S
// with the slots (at most kFrontPfCols entries of each per thread), so the
// table step does not wait for a load that depends on the pool.  Larger
// tables load only the pool's columns, after the pool step (prefetching all
// 128 x 128 entries measured about 2 us slower).
constexpr int kFrontPfN = 32;
constexpr int kFrontPfCols = (kFrontPfN * kFrontPfN + kPoolThreads - 1) / kPoolThreads;
constexpr int kFrontScanWaves = (kMaxExperts + 2 + kWave - 1) / kWave;

__global__ __launch_bounds__(kPoolThreads) void decode_front_kernel(
    const int32_t *__restrict__ ids, const float *__restrict__ w, int B, int N, int K, int D,
    const float *__restrict__ h, const float *__restrict__ S, const float *__restrict__ L,
    int32_t *__restrict__ pool_g, int32_t *__restrict__ pool_size_g, int32_t *__restrict__ out_ids,
    float *__restrict__ out_w, int32_t *__restrict__ tgt_g, float *__restrict__ scl_g, int t_shared,
    int bm0, int bm1, int32_t *__restrict__ offsets, int32_t *__restrict__ tile_start0,
    int32_t *__restrict__ tile_start1, int32_t *__restrict__ row_token,
    int32_t *__restrict__ row_slot, float *__restrict__ row_w, int32_t *__restrict__ slot_row,
    const int32_t *__restrict__ static_tgt, const float *__restrict__ static_scl, int identity,
    const float *__restrict__ lpart, int lP, const float *__restrict__ bias,
    float *__restrict__ logits_out, int32_t *__restrict__ ids_out, float *__restrict__ w_out) {
  __shared__ uint8_t sid[kDecodeFrontMaxSlots];   // expert of each slot (N <= 256)
  __shared__ float sw[kDecodeFrontMaxSlots];      // its weight
  __shared__ unsigned long long wsum[kMaxExperts];
  __shared__ int cnt[kMaxExperts];
  __shared__ double score[kMaxExperts];
  __shared__ int pool[kMaxExperts];
  __shared__ int in_pool[kMaxExperts];
  __shared__ int tgt[kMaxExperts];
  __shared__ float scl[kMaxExperts];
  __shared__ int rows_of[kMaxExperts];  // executed rows per routed expert
  __shared__ int rank_sh[kMaxExperts];
  __shared__ int cur[kMaxExperts];
  __shared__ int wcnt[kFrontWaves][kMaxExperts];
  __shared__ unsigned long long best[kMaxExperts];
  __shared__ int scan_part[3 * kFrontScanWaves];
  __shared__ int cand[kMaxExperts];
  __shared__ int n_cand_sh;
  __shared__ int n_pool;
  // Threads hand data to each other through LDS only, and no global output is
  // read back here, so the phase barriers order LDS alone.
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int slots = B * K;
  const int dcap = min(D, N);
  const int groups = N + (t_shared > 0 ? 1 : 0);

  const float h_e = (tid < N && h) ? h[tid] : 0.f;
  // identity: the permutation alone (every expert maps to itself; out_ids and
  // out_w unused); else precomputed static tables, else the batch pool
  const bool dynamic = !identity && static_tgt == nullptr;  // uniform over the workgroup
  // Table entries of thread (src, part): L[src, t] and S[src, t] for
  // t = part, part + P, ... (N <= kFrontPfN, so at most kFrontPfCols of each),
  // loaded once the slots are in (loads complete in issue order, so loading
  // them first would hold up the slots) and used after the pool step.
  const bool pf = dynamic && N <= kFrontPfN;
  const int P = kPoolThreads / N;
  const int src = tid / P, part = tid % P;
  float lv[kFrontPfCols], sv[kFrontPfCols];
  if (tid == 0) n_cand_sh = 0;
  if (tid < N) {
    best[tid] = ~0ull;
    wsum[tid] = 0ull;
    cnt[tid] = 0;
    in_pool[tid] = 0;
    rows_of[tid] = 0;
    rank_sh[tid] = 0;
    if (identity) {
      tgt[tid] = tid;
      scl[tid] = 1.0f;
      in_pool[tid] = 1;
    } else if (!dynamic) {
      // precomputed static tables: a source is in the pool iff it maps to itself
      const int te = clamp_id(static_tgt[tid], N);
      tgt[tid] = te;
      scl[tid] = static_scl[tid];
      in_pool[tid] = te == tid;
    }
  }
  lds_barrier();

  // ---- pool (Eq. decode_budget): exact fixed-point weight sums ----
  auto add_slot = [&](int j, int e, float wv) {
    sid[j] = (uint8_t)e;
    sw[j] = wv;
    atomicAdd(&cnt[e], 1);
    if (dynamic) {
      const long long q = __double2ll_rn((double)wv * 1099511627776.0);  // 2^40
      atomicAdd(&wsum[e], (unsigned long long)q);
    }
  };
  if (lpart) {
    // Top-K and softmax of the batch here (small batches): wave w takes tokens
    // w, w + kFrontWaves, ... with the per-token steps of route_tokens_kernel
    for (int t = wave; t < B; t += kFrontWaves) {
      float v[4];
      wave_logit_row(lpart, lP, B, N, bias, t, lane, logits_out, v);
      int my_id = 0;
      float my_w = 0.f;
      wave_topk_softmax(v, N, K, lane, my_id, my_w);
      if (lane < K) {
        const int j = t * K + lane;
        ids_out[j] = my_id;
        w_out[j] = my_w;
        add_slot(j, my_id, my_w);
      }
    }
  } else {
    for (int j = tid; j < slots; j += kPoolThreads) add_slot(j, clamp_id(ids[j], N), w[j]);
  }
#pragma unroll
  for (int b = 0; b < kFrontPfCols; ++b) {
    const int t = part + b * P;
    const bool ok = pf && src < N && t < N;
    lv[b] = ok ? L[(size_t)src * N + t] : 0.f;
    sv[b] = ok ? S[(size_t)src * N + t] : 0.f;
  }
  lds_barrier();
  if (dynamic) {
  // candidates (experts with a routed slot) gathered in any order: their ranks
  // come from comparisons, not from list positions
  if (tid < N) {
    score[tid] = (double)(long long)wsum[tid] * (double)h_e;
    if (cnt[tid] > 0) cand[atomicAdd(&n_cand_sh, 1)] = tid;
  }
  lds_barrier();
  const int n_cand = n_cand_sh;
  // rank of each candidate by (score desc, id asc): the P = threads / n_cand
  // threads of a candidate compare it with one slice of the candidate list
  // each; the integer partial ranks add in any order
  if (n_cand > 0) {
    const int parts = kPoolThreads / n_cand;
    const int ci = tid % n_cand, pt = tid / n_cand;
    if (pt < parts) {
      const int e = cand[ci];
      const int chunk = (n_cand + parts - 1) / parts;
      const int lo = pt * chunk, hi = min(n_cand, lo + chunk);
      const double sc = score[e];
      int my = 0;
#pragma unroll 4
      for (int q = lo; q < hi; ++q) {
        const int o = cand[q];
        my += (score[o] > sc) || (score[o] == sc && o < e);
      }
      if (hi > lo) atomicAdd(&rank_sh[e], my);
    }
  }
  lds_barrier();
  if (tid < N && cnt[tid] > 0 && rank_sh[tid] < dcap) {
    pool[rank_sh[tid]] = tid;
    in_pool[tid] = 1;
  }
  if (tid == 0) n_pool = min(dcap, n_cand);
  lds_barrier();
  if (tid < dcap) pool_g[tid] = (tid < n_pool) ? pool[tid] : -1;
  if (tid == 0) *pool_size_g = n_pool;

  // ---- per-source tables (Eq. minimum_loss_assignment over the pool) ----
  if (pf) {
    // the same first minimum in pool order as pool_tables, on the entries
    // loaded at the start: key (L value, pool position), the pool position of
    // a member t being its rank
    uint64_t key = ~0ull;
    float s_key = 1.0f;
    if (src < N && !in_pool[src]) {
#pragma unroll
      for (int b = 0; b < kFrontPfCols; ++b) {
        const int t = part + b * P;
        if (t < N && in_pool[t]) {
          const uint64_t k = (uint64_t(float_key(lv[b])) << 32) | uint64_t(uint32_t(rank_sh[t]));
          if (k < key) {
            key = k;
            s_key = sv[b];
          }
        }
      }
      if (key != ~0ull) atomicMin(&best[src], (unsigned long long)key);
    }
    lds_barrier();
    if (src < N) {
      int t_out = -1;
      float s_out = 1.0f;
      if (in_pool[src] || n_pool == 0) {
        if (part == 0) t_out = src;  // maps to itself
      } else if (key != ~0ull && key == best[src]) {
        t_out = pool[(int)(key & 0xffffffffu)];
        s_out = s_key;
      }
      if (t_out >= 0) {
        tgt[src] = t_out;
        scl[src] = s_out;
        if (tgt_g) tgt_g[src] = t_out;
        if (scl_g) scl_g[src] = s_out;
      }
    }
  } else {
    // without table outputs, only the routed sources need a target: none when
    // every candidate is in the pool
    pool_tables(N, S, L, pool, in_pool, n_pool, tgt, scl, tgt_g, scl_g, (tgt_g || scl_g) ? nullptr : cnt);
  }
  }  // dynamic
  lds_barrier();

  // executed rows per target: the slots of its sources
  if (tid < N && cnt[tid] > 0) atomicAdd(&rows_of[tgt[tid]], cnt[tid]);
  // ---- remap every slot (Eq. decode_remap); retained slots copied ----
  for (int j = tid; j < slots; j += kPoolThreads) {
    const int e = sid[j];
    const float wv = sw[j];
    const int te = tgt[e];
    const float wn = in_pool[e] ? wv : wv * scl[e];
    if (!identity) {
      out_ids[j] = te;
      out_w[j] = wn;
    }
    sid[j] = (uint8_t)te;
    sw[j] = wn;
  }
  lds_barrier();

  // ---- group offsets and GEMM m-tile lists: one group per thread ----
  {
    int v[3] = {0, 0, 0};
    if (tid < groups) {
      const int r = tid < N ? rows_of[tid] : t_shared;
      v[0] = r;
      v[1] = (r + bm0 - 1) / bm0;
      v[2] = (r + bm1 - 1) / bm1;
    }
    for (int e = tid; e < N; e += kPoolThreads) {
#pragma unroll
      for (int q = 0; q < kFrontWaves; ++q) wcnt[q][e] = 0;
    }
    int ex[3], tot[3];
    block_scan3<kFrontScanWaves>(v, ex, tot, scan_part);
    if (tid < N) cur[tid] = ex[0];  // group start (routed experts)
    if (tid < N + 2) {
      offsets[tid] = (tid < N) ? ex[0] : (tid == N) ? slots : slots + t_shared;
      tile_start0[tid] = (tid < groups) ? ex[1] : tot[1];
      tile_start1[tid] = (tid < groups) ? ex[2] : tot[2];
    }
  }
  lds_barrier();

  // ---- stable scatter: rounds of kPoolThreads slots in slot order ----
  for (int base = 0; base < slots; base += kPoolThreads) {
    const int j = base + tid;
    const bool valid = j < slots;
    const int e = valid ? (int)sid[j] : 0;
    // lanes of this wave with the same expert (8 ballots: N <= 256)
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool set = (e >> bit) & 1;
      const uint64_t bal = __ballot(set);
      m &= set ? bal : ~bal;
    }
    const int rank = __popcll(m & lanemask_lt(lane));
    if (valid && rank == 0) wcnt[wave][e] = __popcll(m);
    lds_barrier();
    if (valid) {
      int pos = cur[e] + rank;
      for (int q = 0; q < wave; ++q) pos += wcnt[q][e];
      row_slot[pos] = j;
      row_token[pos] = j / K;
      row_w[pos] = sw[j];
      slot_row[j] = pos;
    }
    lds_barrier();
    for (int x = tid; x < N; x += kPoolThreads) {
      int add = 0;
#pragma unroll
      for (int q = 0; q < kFrontWaves; ++q) {
        add += wcnt[q][x];
        wcnt[q][x] = 0;
      }
      cur[x] += add;
    }
    lds_barrier();
  }
  // Shared-expert rows follow the routed rows, one per token, weight 1.
  for (int i = tid; i < t_shared; i += kPoolThreads) {
    row_token[slots + i] = i;
    row_slot[slots + i] = -1;
    row_w[slots + i] = 1.0f;
  }
}

hipError_t launch_decode_front(const int32_t *ids, const float *w, int B, int N, int K, int D,
                               const float *h, const float *S, const float *L, int32_t *pool,
                               int32_t *pool_size, int32_t *out_ids, float *out_w, int32_t *tgt,
                               float *scl, int t_shared, int bm0, int bm1, const PermBuffers &pb,
                               const int32_t *static_tgt, const float *static_scl, hipStream_t s,
                               const FrontTopK &fused) {
  decode_front_kernel<<<1, kPoolThreads, 0, s>>>(ids, w, B, N, K, D, h, S, L, pool, pool_size, out_ids,
                                                 out_w, tgt, scl, t_shared, bm0, bm1, pb.offsets,
                                                 pb.tile_start0, pb.tile_start1, pb.row_token,
                                                 pb.row_slot, pb.row_w, pb.slot_row, static_tgt,
                                                 static_scl, 0, fused.part, fused.P, fused.bias,
                                                 fused.logits_out, fused.ids_out, fused.w_out);
  return hipGetLastError();
}

// One token per wave: with two, the second token's partial-logit loads wait
// behind the first (32 tokens of the Mixtral-shaped layer: 16.7 us fused
// against 5.2 + 8.4 us in two launches; one token of the Qwen3-shaped layer:
// 12.5 us against 4.8 + 9.1 us).
bool decode_front_fuses_topk(int B, int N) {
  (void)N;
  return B <= kFrontWaves;
}

hipError_t launch_permute_one_block(const int32_t *ids, const float *w, int T, int k_out, int N,
                                    int t_shared, int bm0, int bm1, const PermBuffers &pb,
                                    hipStream_t s) {
  decode_front_kernel<<<1, kPoolThreads, 0, s>>>(ids, w, T, N, k_out, N, nullptr, nullptr, nullptr,
                                                 nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                                 t_shared, bm0, bm1, pb.offsets, pb.tile_start0,
                                                 pb.tile_start1, pb.row_token, pb.row_slot, pb.row_w,
                                                 pb.slot_row, nullptr, nullptr, 1, nullptr, 0,
                                                 nullptr, nullptr, nullptr, nullptr);
  return hipGetLastError();
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

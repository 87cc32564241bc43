// Grouped SwiGLU expert GEMMs over the permuted route rows and the weighted
// combine (Eq. gated_expert, Eq. moe_output / Eq. folded_moe).
//
// gate_up:  H[r, :] = SiLU(X[tok(r)] W_gate[e]^T) * (X[tok(r)] W_up[e]^T)     (bf16 H)
// down:     Y[r, :] = w(r) * (H[r] W_down[e]^T)                                (fp32 Y)
//           or, when every token owns exactly one row, y[tok(r)] = Y[r] directly
// combine:  y_i = sum over the token's routes (slot order) of Y[row], + shared row
//
// bf16 path: MFMA (v_mfma_f32_32x32x16_bf16 / v_mfma_f32_16x16x32_bf16), LDS
// double-buffered BK=64 tiles with an XOR swizzle of 16-byte chunks, device-
// side tile lists (no host synchronisation on group sizes), XCD-aware tile
// order.  Weights are [rows, K] with K contiguous, so both operands load along K.
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

template <int MF> struct Mfma;
template <> struct Mfma<32> {
  typedef f32x16 acc_t;
  static constexpr int kRegs = 16;
  static constexpr int kSteps = 4;  // BK=64 / 16
  __device__ static __forceinline__ acc_t mma(bf16x8 a, bf16x8 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ int frag_row(int lane) { return lane & 31; }
  __device__ static __forceinline__ int frag_chunk(int ks, int lane) { return ks * 2 + (lane >> 5); }
  __device__ static __forceinline__ int out_row(int lane, int r) { return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3); }
  __device__ static __forceinline__ int out_col(int lane) { return lane & 31; }
};
template <> struct Mfma<16> {
  typedef f32x4 acc_t;
  static constexpr int kRegs = 4;
  static constexpr int kSteps = 2;  // BK=64 / 32
  __device__ static __forceinline__ acc_t mma(bf16x8 a, bf16x8 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ int frag_row(int lane) { return lane & 15; }
  __device__ static __forceinline__ int frag_chunk(int ks, int lane) { return ks * 4 + (lane >> 4); }
  __device__ static __forceinline__ int out_row(int lane, int r) { return (lane >> 4) * 4 + r; }
  __device__ static __forceinline__ int out_col(int lane) { return lane & 15; }
};

struct GemmKArgs {
  const bf16_t *A;  // gate_up: x [T, d] gathered by row_token; down: H [rows, I]
  int lda;
  const int32_t *row_token;
  const int32_t *offsets;
  const int32_t *tile_start;
  int groups, n_experts, n_tiles, ksplit, kc;
  const bf16_t *W, *Ws;  // routed base and shared expert
  long long w_stride;    // elements per routed expert
  int ldw;               // K extent of a weight row
  int inter;             // gate_up: intermediate size (up-row offset, H width)
  int d;                 // down: output width
  int rows;
  bf16_t *H;
  float *Y;
  bf16_t *y;
  const float *row_w;
};

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

constexpr int kBK = 64;

// LDS element offset of 16-byte chunk q of tile row r (8 chunks per 128-byte row).
__device__ __forceinline__ int swz(int r, int q) { return (r * 8 + (q ^ (r & 7))) * 8; }

template <int BM, int BN, int WM, int WN, int MF, bool GATE_UP, bool DIRECT>
__global__ __launch_bounds__(256) void expert_gemm_bf16(const GemmKArgs p) {
  typedef Mfma<MF> M;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / MF, TN = WTN / MF;
  constexpr int PA = BM * 8 / 256, PB = BN * 8 / 256;
  static_assert(WM * WN == 4, "4 waves");
  static_assert(TM >= 1 && TN >= 1 && PA >= 1 && PB >= 1, "tile shape");
  static_assert(!GATE_UP || (TN % 2 == 0), "gate/up pairs");

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM * kBK];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN * kBK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  // ---- tile decode: (group, n-tile, k-split) outer, m-tile inner ----
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int units = p.n_tiles * p.ksplit;
  const int total = p.tile_start[p.groups] * units;
  if (L >= total) return;
  int lo = 0, hi = p.groups;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (p.tile_start[mid] * units <= L) lo = mid; else hi = mid;
  }
  const int g = lo;
  const int mt_g = p.tile_start[g + 1] - p.tile_start[g];
  const int local = L - p.tile_start[g] * units;
  const int mt = local % mt_g;
  const int rest = local / mt_g;
  const int ks = rest % p.ksplit;
  const int nt = rest / p.ksplit;
  const int row0 = p.offsets[g] + mt * BM;
  const int valid = min(BM, p.offsets[g + 1] - row0);
  const bf16_t *Wg = (g < p.n_experts) ? p.W + (long long)g * p.w_stride : p.Ws;
  const int k_begin = ks * p.kc;

  // ---- per-thread global source rows ----
  const bf16_t *a_src[PA];
  const bf16_t *b_src[PB];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int c = i * 256 + tid;
    const int r = c >> 3, q = c & 7;
    const int rr = row0 + (r < valid ? r : 0);
    const long long arow = GATE_UP ? (long long)p.row_token[rr] : (long long)rr;
    a_src[i] = p.A + arow * p.lda + k_begin + q * 8;
  }
#pragma unroll
  for (int i = 0; i < PB; ++i) {
    const int c = i * 256 + tid;
    const int r = c >> 3, q = c & 7;
    int wrow;
    if (GATE_UP)
      wrow = (r < BN / 2) ? nt * (BN / 2) + r : p.inter + nt * (BN / 2) + (r - BN / 2);
    else
      wrow = nt * BN + r;
    b_src[i] = Wg + (long long)wrow * p.ldw + k_begin + q * 8;
  }

  uint4 ra[PA], rb[PB];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < PA; ++i) ra[i] = *reinterpret_cast<const uint4 *>(a_src[i] + k0);
#pragma unroll
    for (int i = 0; i < PB; ++i) rb[i] = *reinterpret_cast<const uint4 *>(b_src[i] + k0);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PA; ++i) {
      const int c = i * 256 + tid;
      *reinterpret_cast<uint4 *>(&As[buf][swz(c >> 3, c & 7)]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      const int c = i * 256 + tid;
      *reinterpret_cast<uint4 *>(&Bs[buf][swz(c >> 3, c & 7)]) = rb[i];
    }
  };

  typename M::acc_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < M::kRegs; ++r) acc[i][j][r] = 0.f;

  // B-tile row of wave subtile j (gate/up pairs for GATE_UP)
  auto b_row0 = [&](int j) {
    if (GATE_UP)
      return (j < TN / 2) ? wn * (WTN / 2) + j * MF : BN / 2 + wn * (WTN / 2) + (j - TN / 2) * MF;
    return wn * WTN + j * MF;
  };

  const int KT = p.kc / kBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * kBK);
#pragma unroll
    for (int s = 0; s < M::kSteps; ++s) {
      bf16x8 a[TM], b[TN];
      const int ch = M::frag_chunk(s, lane);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int m = wm * WTM + i * MF + M::frag_row(lane);
        a[i] = *reinterpret_cast<const bf16x8 *>(&As[cur][swz(m, ch)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = b_row0(j) + M::frag_row(lane);
        b[j] = *reinterpret_cast<const bf16x8 *>(&Bs[cur][swz(n, ch)]);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = M::mma(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < KT) lstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue ----
  if (GATE_UP) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN / 2; ++j)
#pragma unroll
        for (int r = 0; r < M::kRegs; ++r) {
          const int ml = wm * WTM + i * MF + M::out_row(lane, r);
          if (ml < valid) {
            const int n = nt * (BN / 2) + wn * (WTN / 2) + j * MF + M::out_col(lane);
            const float hv = silu(acc[i][j][r]) * acc[i][j + TN / 2][r];
            p.H[(long long)(row0 + ml) * p.inter + n] = f32_to_bf16(hv);
          }
        }
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < M::kRegs; ++r) {
          const int ml = wm * WTM + i * MF + M::out_row(lane, r);
          if (ml < valid) {
            const int row = row0 + ml;
            const int n = nt * BN + wn * WTN + j * MF + M::out_col(lane);
            const float v = acc[i][j][r] * p.row_w[row];
            if (DIRECT)
              p.y[(long long)p.row_token[row] * p.d + n] = f32_to_bf16(v);
            else
              p.Y[((long long)ks * p.rows + row) * p.d + n] = v;
          }
        }
  }
}

// ---------------------------------------------------------------------------
// float32 path (SIMT, one thread per output element): the fp32 layer is small.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int find_group(const int32_t *offsets, int groups, int row) {
  int lo = 0, hi = groups;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (offsets[mid] <= row) lo = mid; else hi = mid;
  }
  return lo;
}

__global__ __launch_bounds__(256) void expert_gate_up_f32(const float *__restrict__ x,
                                                          const int32_t *__restrict__ row_token,
                                                          const int32_t *__restrict__ offsets,
                                                          int groups, int n_experts,
                                                          const float *__restrict__ W,
                                                          const float *__restrict__ Ws, int d,
                                                          int inter, int rows,
                                                          float *__restrict__ H) {
  const int n = blockIdx.x * 64 + (threadIdx.x & 63);
  const int row = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (row >= rows || n >= inter) return;
  const int g = find_group(offsets, groups, row);
  const float *Wg = (g < n_experts) ? W + (long long)g * 2 * inter * d : Ws;
  const float *xr = x + (long long)row_token[row] * d;
  const float *wg = Wg + (long long)n * d;
  const float *wu = Wg + (long long)(inter + n) * d;
  float ga = 0.f, ua = 0.f;
  for (int k = 0; k < d; ++k) {
    ga = fmaf(xr[k], wg[k], ga);
    ua = fmaf(xr[k], wu[k], ua);
  }
  H[(long long)row * inter + n] = silu(ga) * ua;
}

__global__ __launch_bounds__(256) void expert_down_f32(const float *__restrict__ H,
                                                       const int32_t *__restrict__ row_token,
                                                       const int32_t *__restrict__ offsets,
                                                       int groups, int n_experts,
                                                       const float *__restrict__ W,
                                                       const float *__restrict__ Ws, int d,
                                                       int inter, int rows,
                                                       const float *__restrict__ row_w,
                                                       float *__restrict__ Y,
                                                       float *__restrict__ y) {
  const int n = blockIdx.x * 64 + (threadIdx.x & 63);
  const int row = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (row >= rows || n >= d) return;
  const int g = find_group(offsets, groups, row);
  const float *Wg = (g < n_experts) ? W + (long long)g * d * inter : Ws;
  const float *hr = H + (long long)row * inter;
  const float *wr = Wg + (long long)n * inter;
  float acc = 0.f;
  for (int k = 0; k < inter; ++k) acc = fmaf(hr[k], wr[k], acc);
  const float v = acc * row_w[row];
  if (y)
    y[(long long)row_token[row] * d + n] = v;
  else
    Y[(long long)row * d + n] = v;
}

// ---------------------------------------------------------------------------
// Planning and launch.
// ---------------------------------------------------------------------------
static int largest_divisor_at_most(int n, int cap) {
  for (int v = cap < n ? cap : n; v > 1; --v)
    if (n % v == 0) return v;
  return 1;
}

void plan_expert_gemms(int dtype, int rows, int groups, int active_groups, int d, int inter,
                       int cu_count, GemmPlan *gu, GemmPlan *dn) {
  if (dtype != EXFOLD_BF16) {
    *gu = GemmPlan{4, 64, 1, 0};
    *dn = GemmPlan{4, 64, 1, 0};
    return;
  }
  // Tile height from the rows each active group is expected to hold (not from
  // the phase), so equal problems get equal plans whatever the phase.
  const int active = active_groups < 1 ? 1 : active_groups;
  const bool small = rows <= 48 * active;
  if (small) {
    *gu = GemmPlan{32, 128, 1, 0};
    *dn = GemmPlan{32, 128, 1, 0};
  } else {
    *gu = GemmPlan{128, 128, 1, 0};
    *dn = GemmPlan{128, 128, 1, 0};
  }
  const int mt_gu = rows / gu->bm + groups;
  const int mt_dn = rows / dn->bm + groups;
  gu->grid = mt_gu * (inter / (gu->bn / 2));
  const int nt_dn = d / dn->bn;
  if (small) {
    // Split the down projection's reduction so that the few retained groups
    // still spread over every CU.
    const int want = (2 * cu_count + active * nt_dn - 1) / (active * nt_dn);
    dn->ksplit = largest_divisor_at_most(inter / kBK, want < 1 ? 1 : want);
  }
  dn->grid = mt_dn * nt_dn * dn->ksplit;
}

template <int BM, int BN, int WM, int WN, int MF>
static void launch_pair(const GemmKArgs &gu_args, const GemmKArgs &dn_args, int gu_grid, int dn_grid,
                        bool direct, hipStream_t s, hipEvent_t ev_mid) {
  if (gu_grid > 0) expert_gemm_bf16<BM, BN, WM, WN, MF, true, false><<<gu_grid, 256, 0, s>>>(gu_args);
  if (ev_mid) (void)hipEventRecord(ev_mid, s);
  if (dn_grid > 0) {
    if (direct)
      expert_gemm_bf16<BM, BN, WM, WN, MF, false, true><<<dn_grid, 256, 0, s>>>(dn_args);
    else
      expert_gemm_bf16<BM, BN, WM, WN, MF, false, false><<<dn_grid, 256, 0, s>>>(dn_args);
  }
}

hipError_t launch_expert_gemms(const ExpertArgs &a, const GemmPlan &gu, const GemmPlan &dn,
                               hipStream_t s, hipEvent_t ev_mid) {
  if (a.rows <= 0) return hipSuccess;
  if (a.dtype != EXFOLD_BF16) {
    dim3 g1((a.inter + 63) / 64, (a.rows + 3) / 4);
    expert_gate_up_f32<<<g1, 256, 0, s>>>(
        static_cast<const float *>(a.x), a.row_token, a.offsets, a.groups, a.n_experts,
        static_cast<const float *>(a.w_gate_up), static_cast<const float *>(a.ws_gate_up), a.d,
        a.inter, a.rows, static_cast<float *>(a.H));
    if (ev_mid) (void)hipEventRecord(ev_mid, s);
    dim3 g2((a.d + 63) / 64, (a.rows + 3) / 4);
    expert_down_f32<<<g2, 256, 0, s>>>(
        static_cast<const float *>(a.H), a.row_token, a.offsets, a.groups, a.n_experts,
        static_cast<const float *>(a.w_down), static_cast<const float *>(a.ws_down), a.d, a.inter,
        a.rows, a.row_w, a.Y, a.direct ? static_cast<float *>(a.y) : nullptr);
    return hipGetLastError();
  }
  GemmKArgs ga{};
  ga.A = static_cast<const bf16_t *>(a.x);
  ga.lda = a.d;
  ga.row_token = a.row_token;
  ga.offsets = a.offsets;
  ga.tile_start = a.tile_start_gu;
  ga.groups = a.groups;
  ga.n_experts = a.n_experts;
  ga.n_tiles = a.inter / (gu.bn / 2);
  ga.ksplit = 1;
  ga.kc = a.d;
  ga.W = static_cast<const bf16_t *>(a.w_gate_up);
  ga.Ws = static_cast<const bf16_t *>(a.ws_gate_up);
  ga.w_stride = 2LL * a.inter * a.d;
  ga.ldw = a.d;
  ga.inter = a.inter;
  ga.d = a.d;
  ga.rows = a.rows;
  ga.H = static_cast<bf16_t *>(a.H);

  GemmKArgs da{};
  da.A = static_cast<const bf16_t *>(a.H);
  da.lda = a.inter;
  da.row_token = a.row_token;
  da.offsets = a.offsets;
  da.tile_start = a.tile_start_dn;
  da.groups = a.groups;
  da.n_experts = a.n_experts;
  da.n_tiles = a.d / dn.bn;
  da.ksplit = dn.ksplit;
  da.kc = a.inter / dn.ksplit;
  da.W = static_cast<const bf16_t *>(a.w_down);
  da.Ws = static_cast<const bf16_t *>(a.ws_down);
  da.w_stride = (long long)a.d * a.inter;
  da.ldw = a.inter;
  da.inter = a.inter;
  da.d = a.d;
  da.rows = a.rows;
  da.Y = a.Y;
  da.y = static_cast<bf16_t *>(a.y);
  da.row_w = a.row_w;

  if (gu.bm == 32)
    launch_pair<32, 128, 1, 4, 16>(ga, da, gu.grid, dn.grid, a.direct, s, ev_mid);
  else
    launch_pair<128, 128, 2, 2, 32>(ga, da, gu.grid, dn.grid, a.direct, s, ev_mid);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weighted combine: y_i = sum_k sum_split Y[split][row(i,k)] (+ shared row),
// in slot order; float32 accumulation, one rounding to the output dtype.
// ---------------------------------------------------------------------------
template <typename OutT>
__global__ __launch_bounds__(256) void combine_kernel(const float *__restrict__ Y, int ksplit,
                                                     int rows, const int32_t *__restrict__ slot_row,
                                                     int k_out, int d, int shared_base,
                                                     OutT *__restrict__ y) {
  const int i = blockIdx.x;
  for (int c = threadIdx.x * 4; c < d; c += 256 * 4) {
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int k = 0; k < k_out; ++k) {
      const int r = slot_row[(long long)i * k_out + k];
      for (int sp = 0; sp < ksplit; ++sp) {
        const float4 v = *reinterpret_cast<const float4 *>(Y + ((long long)sp * rows + r) * d + c);
        acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
      }
    }
    if (shared_base >= 0) {
      for (int sp = 0; sp < ksplit; ++sp) {
        const float4 v = *reinterpret_cast<const float4 *>(Y + ((long long)sp * rows + shared_base + i) * d + c);
        acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
      }
    }
    OutT *o = y + (long long)i * d + c;
    o[0] = store_cvt<OutT>(acc.x);
    o[1] = store_cvt<OutT>(acc.y);
    o[2] = store_cvt<OutT>(acc.z);
    o[3] = store_cvt<OutT>(acc.w);
  }
}

hipError_t launch_combine(int dtype, const float *Y, int ksplit, int rows, const int32_t *slot_row,
                          int T, int k_out, int d, int shared_base, void *y, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (dtype == EXFOLD_BF16)
    combine_kernel<bf16_t><<<T, 256, 0, s>>>(Y, ksplit, rows, slot_row, k_out, d, shared_base,
                                             static_cast<bf16_t *>(y));
  else
    combine_kernel<float><<<T, 256, 0, s>>>(Y, ksplit, rows, slot_row, k_out, d, shared_base,
                                            static_cast<float *>(y));
  return hipGetLastError();
}

}  // namespace exfold

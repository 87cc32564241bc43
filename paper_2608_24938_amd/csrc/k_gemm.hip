// Grouped SwiGLU expert GEMMs over the permuted route rows and the weighted
// combine (Eq. gated_expert, Eq. moe_output / Eq. folded_moe).
//
// gate_up:  H[r, :] = SiLU(X[tok(r)] W_gate[e]^T) * (X[tok(r)] W_up[e]^T)     (bf16 H)
// down:     Y[r, :] = w(r) * (H[r] W_down[e]^T)                                (fp32 Y)
//           or, when every token owns exactly one row, y[tok(r)] = Y[r] directly
// combine:  y_i = sum over the token's routes (slot order) of Y[row], + shared row
//
// Weights are [rows, K] with K contiguous, so both operands load along K.  Group
// sizes are device data: each kernel walks a device-side tile list built by the
// permutation (no host synchronisation), in an XCD-aware order that keeps the
// tiles sharing one weight tile on one XCD's L2.
//
// expert_gemm_tile: 128x128 macro tile, 4 waves of 32x32x16 bf16 MFMA, BK=64 LDS
// double buffer with an XOR swizzle of 16-byte chunks, two tiles of global loads
// in flight through registers.  The down projection may split its reduction
// (few rows per retained expert): split s writes its own partial Y[s], and the
// combine adds the splits in a fixed order.
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

struct GemmKArgs {
  const bf16_t *A;  // gate_up: x [T, d] gathered by row_token; down: H [rows, I]
  int lda;
  const int32_t *row_token;
  const int32_t *offsets;
  const int32_t *tile_start;
  int groups, n_experts, n_tiles, ksplit, kc, rows;
  const bf16_t *W, *Ws;  // routed base and shared expert
  long long w_stride;    // elements per routed expert
  int ldw;               // K extent of a weight row
  int inter;             // gate_up: intermediate size (up-row offset, H width)
  int d;                 // down: output width
  bf16_t *H;
  float *Y;
  bf16_t *Yh;  // down, when set: bf16 per-row outputs instead of Y (no split)
  float *P;    // wide tiles: split-remainder partial tiles [workgroups][256 * 256]
  bf16_t *y;
  const float *row_w;
};

// g * sigmoid(g) with the hardware reciprocal (one rounding step instead of
// the IEEE division sequence; the result is rounded to bf16 or kept fp32
// within 1 ulp).
__device__ __forceinline__ float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

constexpr int kBK = 64;

// LDS element offset of 16-byte chunk q of tile row r (8 chunks per 128-byte row).
// The slot is q XOR gray(r): one chunk column of any 8 or 16 consecutive rows
// (the lanes of one LDS cycle of ds_read_b128) then spans distinct banks.
__device__ __forceinline__ int swz(int r, int q) { return (r * 8 + (q ^ ((r ^ (r >> 1)) & 7))) * 8; }

// Tile of workgroup `wg`: group g, n-tile nt, split ks, m-tile mt (m-tile
// fastest, so the m-tiles sharing one weight tile run together).  The grid is an
// upper bound of the tile count; workgroups past the device-side count exit, and
// the XCD-aware remap is taken over the actual count so that every XCD gets an
// equal, contiguous share of the real tiles.
struct TileId {
  int g, nt, ks, mt;
  int dbl;  // wide tiles: a 128-row tail spanning n-tiles nt and nt + 1
};
// Tile of logical id L (m-tile fastest within a group and n-tile).
__device__ __forceinline__ void tile_at(const GemmKArgs &p, int L, TileId &t) {
  const int units = p.n_tiles * p.ksplit;
  int lo = 0, hi = p.groups;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (p.tile_start[mid] * units <= L) lo = mid; else hi = mid;
  }
  const int mt_g = p.tile_start[lo + 1] - p.tile_start[lo];
  const int local = L - p.tile_start[lo] * units;
  t.g = lo;
  t.mt = local % mt_g;
  const int u = local / mt_g;
  t.ks = u % p.ksplit;
  t.nt = u / p.ksplit;
}

__device__ __forceinline__ bool decode_tile(const GemmKArgs &p, int wg, TileId &t) {
  const int units = p.n_tiles * p.ksplit;
  const int total = p.tile_start[p.groups] * units;
  if (wg >= total) return false;
  tile_at(p, xcd_remap(wg, total), t);
  return true;
}

// ---------------------------------------------------------------------------
// Macro-tile kernel.
// ---------------------------------------------------------------------------
// PLAIN: one group of p.rows rows read in order (no offsets, tile list or
// gather), partial sums of split ks written unscaled to Y[ks] (a plain
// x W^T with a split reduction: the router logits of large batches).
template <int BM, int BN, int STAGES, bool GATE_UP, bool DIRECT, bool PLAIN = false>
__global__ __launch_bounds__(256, 1) void expert_gemm_tile(const GemmKArgs p) {
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int PA = BM / 32, PB = BN / 32;  // 16-byte chunks per thread per stage
  static_assert(!GATE_UP || (TN % 2 == 0), "gate/up pairs");

  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (BM + BN) * kBK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  TileId t;
  int row0, valid;
  const bf16_t *Wg;
  if constexpr (PLAIN) {
    const int mt_n = (p.rows + BM - 1) / BM, total = mt_n * p.n_tiles * p.ksplit;
    if ((int)blockIdx.x >= total) return;
    const int L = xcd_remap(blockIdx.x, total);
    t.g = 0;
    t.mt = L % mt_n;
    t.ks = (L / mt_n) % p.ksplit;
    t.nt = L / mt_n / p.ksplit;
    row0 = t.mt * BM;
    valid = min(BM, p.rows - row0);
    Wg = p.W;
  } else {
    if (!decode_tile(p, blockIdx.x, t)) return;
    row0 = p.offsets[t.g] + t.mt * BM;
    valid = min(BM, p.offsets[t.g + 1] - row0);
    Wg = (t.g < p.n_experts) ? p.W + (long long)t.g * p.w_stride : p.Ws;
  }

  // global source of this thread's 16-byte chunks (row r = c / 8, chunk q = c % 8)
  // A rows past the group's end are not loaded (their outputs are never stored):
  // a tile with few rows (decode) then reads only its live rows.
  const bf16_t *a_src[PA];
  const bf16_t *b_src[PB];
  bool a_live[PA];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int c = i * 256 + tid;
    const int r = c >> 3;
    a_live[i] = r < valid;
    const int rr = row0 + (r < valid ? r : 0);
    const long long arow = GATE_UP ? (long long)p.row_token[rr] : (long long)rr;
    a_src[i] = p.A + arow * p.lda + t.ks * p.kc + (c & 7) * 8;
  }
#pragma unroll
  for (int i = 0; i < PB; ++i) {
    const int c = i * 256 + tid;
    const int r = c >> 3;
    int wrow;
    if (GATE_UP)
      wrow = (r < BN / 2) ? t.nt * (BN / 2) + r : p.inter + t.nt * (BN / 2) + (r - BN / 2);
    else
      wrow = t.nt * BN + r;
    b_src[i] = Wg + (long long)wrow * p.ldw + t.ks * p.kc + (c & 7) * 8;
  }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // LDS row of wave subtile j of B (gate/up pairs for GATE_UP)
  int b_row[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j)
    b_row[j] = GATE_UP ? ((j < TN / 2) ? wn * (WTN / 2) + j * 32 : BN / 2 + wn * (WTN / 2) + (j - TN / 2) * 32)
                       : wn * WTN + j * 32;

  // The prefetch registers are plain arrays indexed only by unrolled constants
  // (macros, not lambdas taking their address), so they stay in VGPRs.
#define EXF_GLOAD(RA, RB, K0)                                                                \
  do {                                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < PA; ++i_) if (a_live[i_]) RA[i_] =               \
        *reinterpret_cast<const u32x4 *>(a_src[i_] + (K0));                                  \
    _Pragma("unroll") for (int i_ = 0; i_ < PB; ++i_) RB[i_] =                               \
        *reinterpret_cast<const u32x4 *>(b_src[i_] + (K0));                                  \
  } while (0)
#define EXF_LSTORE(RA, RB, BUF)                                                              \
  do {                                                                                       \
    bf16_t *As_ = smem + (BUF) * BM * kBK;                                                   \
    bf16_t *Bs_ = smem + 2 * BM * kBK + (BUF) * BN * kBK;                                    \
    _Pragma("unroll") for (int i_ = 0; i_ < PA; ++i_) {                                      \
      const int c_ = i_ * 256 + tid;                                                         \
      *reinterpret_cast<u32x4 *>(&As_[swz(c_ >> 3, c_ & 7)]) = RA[i_];                        \
    }                                                                                        \
    _Pragma("unroll") for (int i_ = 0; i_ < PB; ++i_) {                                      \
      const int c_ = i_ * 256 + tid;                                                         \
      *reinterpret_cast<u32x4 *>(&Bs_[swz(c_ >> 3, c_ & 7)]) = RB[i_];                        \
    }                                                                                        \
  } while (0)
// Fragments of k-step s+1 are read while the MFMAs of step s run.
#define EXF_FRAGS(A_, B_, S_)                                                                \
  do {                                                                                       \
    const int ch_ = (S_) * 2 + (lane >> 5);                                                  \
    _Pragma("unroll") for (int i_ = 0; i_ < TM; ++i_) A_[i_] =                               \
        *reinterpret_cast<const bf16x8 *>(&As_[swz(wm * WTM + i_ * 32 + (lane & 31), ch_)]); \
    _Pragma("unroll") for (int j_ = 0; j_ < TN; ++j_) B_[j_] =                               \
        *reinterpret_cast<const bf16x8 *>(&Bs_[swz(b_row[j_] + (lane & 31), ch_)]);           \
  } while (0)
#define EXF_MMA(A_, B_)                                                                      \
  do {                                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < TM; ++i_)                                        \
        _Pragma("unroll") for (int j_ = 0; j_ < TN; ++j_) acc[i_][j_] =                      \
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(A_[i_], B_[j_], acc[i_][j_], 0, 0, 0);   \
  } while (0)
#define EXF_COMPUTE(BUF)                                                                     \
  do {                                                                                       \
    const bf16_t *As_ = smem + (BUF) * BM * kBK;                                             \
    const bf16_t *Bs_ = smem + 2 * BM * kBK + (BUF) * BN * kBK;                              \
    bf16x8 a0_[TM], b0_[TN], a1_[TM], b1_[TN];                                               \
    EXF_FRAGS(a0_, b0_, 0);                                                                  \
    EXF_FRAGS(a1_, b1_, 1);                                                                  \
    EXF_MMA(a0_, b0_);                                                                       \
    EXF_FRAGS(a0_, b0_, 2);                                                                  \
    EXF_MMA(a1_, b1_);                                                                       \
    EXF_FRAGS(a1_, b1_, 3);                                                                  \
    EXF_MMA(a0_, b0_);                                                                       \
    EXF_MMA(a1_, b1_);                                                                       \
  } while (0)

  // Schedule of one phase: the next tile's global loads first, fragments of
  // k-step s+1 read while the MFMAs of step s run, and the staged tile written to
  // the other LDS buffer before the last MFMA group.
#define EXF_SCHEDULE()                                                               \
  do {                                                                               \
    __builtin_amdgcn_sched_group_barrier(0x020, PA + PB, 0); /* VMEM read */         \
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * (TM + TN), 0); /* DS read */     \
    __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0); /* MFMA */              \
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);                          \
    __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);                          \
    __builtin_amdgcn_sched_group_barrier(0x100, TM + TN, 0);                          \
    __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);                          \
    __builtin_amdgcn_sched_group_barrier(0x200, PA + PB, 0); /* DS write */           \
    __builtin_amdgcn_sched_group_barrier(0x008, TM * TN, 0);                          \
  } while (0)

  // Pairs of phases over the two LDS buffers, no early exit (one loop exit keeps
  // the accumulators in one register set); an odd tile count ends with buffer 0.
  // Loads past the last tile re-read the last tile (k clamped) and land in a
  // buffer that is never read again, so each phase is one straight-line block.
  const int KT = p.kc / kBK;
  const int k_last = (KT - 1) * kBK;
  if (STAGES == 2) {
    // LDS buffer (kt & 1) holds tile kt; the other register set holds tile kt + 1,
    // so each tile's loads are covered by two compute phases.
    u32x4 ra0[PA], rb0[PB], ra1[PA], rb1[PB];
    _Pragma("unroll") for (int i_ = 0; i_ < PA; ++i_) ra0[i_] = ra1[i_] = u32x4{0u, 0u, 0u, 0u};
    EXF_GLOAD(ra0, rb0, 0);
    EXF_LSTORE(ra0, rb0, 0);
    EXF_GLOAD(ra1, rb1, min(kBK, k_last));
    __syncthreads();
    int kt = 0;
    for (; kt + 2 <= KT; kt += 2) {
      EXF_GLOAD(ra0, rb0, min((kt + 2) * kBK, k_last));
      EXF_COMPUTE(0);
      EXF_LSTORE(ra1, rb1, 1);
      EXF_SCHEDULE();
      __syncthreads();
      EXF_GLOAD(ra1, rb1, min((kt + 3) * kBK, k_last));
      EXF_COMPUTE(1);
      EXF_LSTORE(ra0, rb0, 0);
      EXF_SCHEDULE();
      __syncthreads();
    }
    if (kt < KT) EXF_COMPUTE(0);
  } else {
    // One tile of loads in flight, covered by one compute phase.
    u32x4 ra[PA], rb[PB];
    _Pragma("unroll") for (int i_ = 0; i_ < PA; ++i_) ra[i_] = u32x4{0u, 0u, 0u, 0u};
    EXF_GLOAD(ra, rb, 0);
    EXF_LSTORE(ra, rb, 0);
    __syncthreads();
    int kt = 0;
    for (; kt + 2 <= KT; kt += 2) {
      EXF_GLOAD(ra, rb, (kt + 1) * kBK);
      EXF_COMPUTE(0);
      EXF_LSTORE(ra, rb, 1);
      EXF_SCHEDULE();
      __syncthreads();
      EXF_GLOAD(ra, rb, min((kt + 2) * kBK, k_last));
      EXF_COMPUTE(1);
      EXF_LSTORE(ra, rb, 0);
      EXF_SCHEDULE();
      __syncthreads();
    }
    if (kt < KT) EXF_COMPUTE(0);
  }
#undef EXF_GLOAD
#undef EXF_LSTORE
#undef EXF_COMPUTE
#undef EXF_FRAGS
#undef EXF_MMA
#undef EXF_SCHEDULE

  // ---- epilogue ----
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < (GATE_UP ? TN / 2 : TN); ++j) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ml = wm * WTM + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        if (ml < valid) {
          const int row = row0 + ml;
          if (GATE_UP) {
            const int n = t.nt * (BN / 2) + wn * (WTN / 2) + j * 32 + (lane & 31);
            p.H[(long long)row * p.inter + n] = f32_to_bf16(silu(acc[i][j][r]) * acc[i][j + TN / 2][r]);
          } else {
            const int n = t.nt * BN + wn * WTN + j * 32 + (lane & 31);
            if (PLAIN)
              p.Y[((long long)t.ks * p.rows + row) * p.d + n] = acc[i][j][r];
            else if (DIRECT)
              p.y[(long long)p.row_token[row] * p.d + n] = f32_to_bf16(acc[i][j][r] * p.row_w[row]);
            else if (p.Yh)
              p.Yh[(long long)row * p.d + n] = f32_to_bf16(acc[i][j][r]);
            else
              p.Y[((long long)t.ks * p.rows + row) * p.d + n] = acc[i][j][r] * p.row_w[row];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Wide tile for the prefill GEMMs (many rows per retained expert): 256x256
// macro tile, eight waves (two per SIMD), wave (wm, wn) owning tile rows
// 128 wm .. 128 wm + 127 and 64 columns (gate/up: gate columns 32 wn .. 32 wn +
// 31 with the matching up columns; 4x2 MFMA tiles); a group's last rows, when
// at most 128, form a 128x512 tile over two n-tiles (the waves in one row).
// Four waves of 128x128 each (one per SIMD, accumulators in AGPRs) measured
// 7-11% slower.  The operands go from global memory
// straight into LDS (global_load_lds_dwordx4) through a ring of reduction
// stages: no staging registers and no LDS write instructions.  Against 128x128
// tiles the bytes loaded per flop halve, and the weight panel a tile shares
// with the other m-tiles of its expert is fetched from HBM about once (2.4 GB
// per Mixtral-shaped launch against 3.8-5 GB).  Measured on that launch, the
// 64-wide stages with two ring buffers beat 32-wide stages with four or five
// buffers (more bytes in flight, but 64-byte row pieces and twice the barriers).
// ---------------------------------------------------------------------------
constexpr int kWide = 256, kWideWaves = 8, kWideBK = 64, kWideStages = 2;

// LDS byte address of a shared-memory pointer (for M0).
__device__ __forceinline__ uint32_t lds_addr(const void *ptr) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)ptr;
}

// One 16-byte chunk per lane from global g into the 1 KiB LDS block at byte
// address lds (wave-uniform): lane l lands at lds + 16 l.  M0 holds the block
// address; one wait state separates its write from the load.  The statement
// clobbers M0, which the compiler does not save around it: the kernels that
// use it must give the compiler no reason to hold a value in M0 (register
// arrays indexed by compile-time constants only, no indirect register moves).
// The compiler's own LDS-DMA builtin keeps M0 safe but schedules the main loop
// 2% slower (its conservative waits).
__device__ __forceinline__ void lds_dma16(const void *g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(lds)
               : "memory", "m0");
}

// Wide tile of logical id L.  The tile list counts rows of a group in
// 128-row units (u_g = ceil(rows_g / 128), prefix tile_start); per group and
// per pair j of n-tiles (2j, 2j + 1) there are u_g tiles: the M = u_g / 2
// full-height m-tiles of n-tile 2j, then those of n-tile 2j + 1 (m-tile
// fastest: the tiles that share a weight panel run side by side), then, for
// odd u_g, one tail tile of at most 128 rows that spans both n-tiles.  The
// tail costs half a tile and starts and ends with its neighbours, so the tiles
// that share a panel stay in step (a half-height tile on one n-tile would run
// ahead of its siblings and fetch the panel a second time).
__device__ __forceinline__ void wide_tile_at(const GemmKArgs &p, int L, TileId &t) {
  const int pairs = p.n_tiles / 2;
  int lo = 0, hi = p.groups;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (p.tile_start[mid] * pairs <= L) lo = mid; else hi = mid;
  }
  const int u_g = p.tile_start[lo + 1] - p.tile_start[lo];
  const int local = L - p.tile_start[lo] * pairs;
  const int j = local / u_g, u = local % u_g, M = u_g >> 1;
  t.g = lo;
  t.ks = 0;
  if (u < 2 * M) {
    t.nt = 2 * j + u / M;
    t.mt = u % M;
    t.dbl = 0;
  } else {
    t.nt = 2 * j;
    t.mt = M;
    t.dbl = 1;
  }
}

// Slot of 16-byte chunk q in a tile row of BK bf16 (an involution in q): the
// chunk columns that one ds_read_b128 takes from consecutive rows land in
// distinct LDS banks.  64-byte rows: q ^ bits 2..3 of r; 128-byte rows: the
// Gray-code swizzle of the register-staged tiles.
template <int BK>
__device__ __forceinline__ int wide_slot(int r, int q) {
  if (BK == 32) return q ^ ((r >> 2) & 3);
  return q ^ ((r ^ (r >> 1)) & 7);
}

// 32x32 MFMA tiles per wave: the waves form two rows of kWideWaves / 2, each
// wave owning 128 tile rows and 32 kWideTN of the 256 tile columns
constexpr int kWideTM = 4, kWideTN = 16 / kWideWaves;
constexpr int kWideBN = 32 * kWideTN * (kWideWaves / 2);  // tile columns (gate/up: weight rows)
static_assert(kWideBN == kWide, "square wide tile");
// LDS ring: two stages of the 256 x 256 tile (128 KiB) or of the 128 x 512 tail (160 KiB)
constexpr int kWideSmemElems = kWideStages * (kWide / 2 + 2 * kWideBN) * kWideBK;

// Main loop of one wide tile over the reduction stages [k0, k1): zeroes acc,
// streams the stages through the LDS ring and leaves the products in acc.
// All waves of the workgroup call it; it ends with every load landed and a
// barrier, so the ring may be refilled right after.  DBL: the 128 x 512 tail
// tile (one row of NW waves) instead of 256 x 256 (two rows of NW / 2).
// TMV: the calling wave's 32-row blocks that hold rows of the group (the
// others are padding: their fragments are not read and their MFMAs not
// issued, so their accumulators stay zero); the wave still loads its share of
// every stage and takes every barrier.
template <bool GATE_UP, int BK, int STAGES, int NW, bool DBL, int TMV>
__device__ __forceinline__ void wide_tile_mma(const GemmKArgs &p, const TileId &t, int row0, int valid,
                                              int k0, int k1, bf16_t *smem,
                                              f32x16 (&acc)[kWideTM][kWideTN]) {
  // NW waves in WM rows of WN; each wave owns 128 rows and 32 TN columns
  // (gate/up: 16 TN gate + the matching 16 TN up columns)
  constexpr int WM = DBL ? 1 : 2, WN = NW / WM;
  constexpr int BM = 128 * WM, TM = kWideTM, TN = kWideTN, BN = 32 * TN * WN;
  static_assert(NW == kWideWaves, "accumulator shape");
  static_assert(TMV >= 0 && TMV <= TM, "valid row blocks");
  constexpr int STAGE = (BM + BN) * BK;          // elements of one stage (A rows, then B rows)
  constexpr int CPR = BK / 8;                    // 16-byte chunks per row
  constexpr int RPB = 64 / CPR;                  // rows per 1 KiB block
  constexpr int BLOCKS = (BM + BN) / RPB;        // blocks per stage
  constexpr int PW = BLOCKS / NW;                // DMA loads per wave per stage
  constexpr int AHEAD = STAGES - 1;              // stages in flight while one is computed
  constexpr int VMC = (AHEAD - 1) * PW;          // loads allowed in flight at a stage's wait
  static_assert(VMC == 0 || VMC == 6 || VMC == 8 || VMC == 10 || VMC == 12 || VMC == 16, "vmcnt immediates below");
  static_assert(BLOCKS % NW == 0, "blocks per wave");
  static_assert(STAGES * STAGE <= kWideSmemElems, "LDS ring");

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const bf16_t *Wg = (t.g < p.n_experts) ? p.W + (long long)t.g * p.w_stride : p.Ws;

  // Wave w fills blocks w, w + NW, ...; lane l fills row RPB b + l / CPR of its
  // block at slot l % CPR, i.e. it fetches the chunk that the swizzle puts
  // there.  Rows past the group's end re-read its first row (in bounds, never
  // stored).
  const bf16_t *src[PW];
#pragma unroll
  for (int i = 0; i < PW; ++i) {
    const int blk = i * NW + wave;
    const int r = blk * RPB + lane / CPR;  // stage row: A rows 0..255, then B rows
    if (r < BM) {
      const int q = wide_slot<BK>(r, lane % CPR);
      const int rr = row0 + (r < valid ? r : 0);
      const long long arow = GATE_UP ? (long long)p.row_token[rr] : (long long)rr;
      src[i] = p.A + arow * p.lda + (long long)t.ks * p.kc + q * 8;
    } else {
      const int rb = r - BM;
      const int q = wide_slot<BK>(rb, lane % CPR);
      int wrow;
      if (GATE_UP)
        wrow = (rb < BN / 2) ? t.nt * (kWideBN / 2) + rb : p.inter + t.nt * (kWideBN / 2) + (rb - BN / 2);
      else
        wrow = t.nt * kWideBN + rb;
      src[i] = Wg + (long long)wrow * p.ldw + (long long)t.ks * p.kc + q * 8;
    }
  }
  const uint32_t lds0 = lds_addr(smem);

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  int a_row[TM], b_row[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) a_row[i] = wm * 128 + i * 32 + (lane & 31);
#pragma unroll
  for (int j = 0; j < TN; ++j)
    b_row[j] = (GATE_UP ? (j < TN / 2 ? 0 : BN / 2) + (j % (TN / 2)) * 32 + wn * 16 * TN : wn * 32 * TN + j * 32) +
               (lane & 31);

  // Stage kt (clamped to the last of the range: loads past it refill a buffer
  // that is never read again) into ring buffer BUF.
#define EXF_W_ISSUE(BUF, KT_)                                                                  \
  do {                                                                                         \
    const int k0_ = min((KT_), k1 - 1) * BK;                                                   \
    const uint32_t base_ = lds0 + (uint32_t)(BUF) * (STAGE * 2);                               \
    _Pragma("unroll") for (int i_ = 0; i_ < PW; ++i_)                                          \
        lds_dma16(src[i_] + k0_, base_ + (i_ * NW + wave) * 1024);                             \
  } while (0)
#define EXF_W_FRAGS(A_, B_, BUF, S_)                                                           \
  do {                                                                                         \
    const bf16_t *As_ = smem + (BUF) * STAGE;                                                  \
    const bf16_t *Bs_ = As_ + BM * BK;                                                         \
    const int ch_ = (S_) * 2 + (lane >> 5);                                                    \
    _Pragma("unroll") for (int i_ = 0; i_ < TMV; ++i_) A_[i_] = *reinterpret_cast<const bf16x8 *>( \
        As_ + a_row[i_] * BK + wide_slot<BK>(a_row[i_], ch_) * 8);                             \
    if (TMV > 0)                                                                               \
      _Pragma("unroll") for (int j_ = 0; j_ < TN; ++j_) B_[j_] = *reinterpret_cast<const bf16x8 *>( \
          Bs_ + b_row[j_] * BK + wide_slot<BK>(b_row[j_], ch_) * 8);                           \
  } while (0)
#define EXF_W_MMA(A_, B_)                                                                      \
  do {                                                                                         \
    _Pragma("unroll") for (int i_ = 0; i_ < TMV; ++i_)                                         \
        _Pragma("unroll") for (int j_ = 0; j_ < TN; ++j_) acc[i_][j_] =                        \
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(B_[j_], A_[i_], acc[i_][j_], 0, 0, 0);     \
  } while (0)

  for (int q = 0; q < AHEAD; ++q) EXF_W_ISSUE(q, k0 + q);
  static_assert((BK / 16) % 2 == 0, "the last step of a stage uses fragment set 1");
  bf16x8 fa[2][TM], fb[2][TN];
  int buf = 0;  // ring buffer of stage kt (wave-uniform)
  for (int kt = k0; kt < k1; ++kt) {
    // Wait until this wave's loads of stage kt have landed (the later stages
    // stay in flight) and its LDS reads of the previous stage are done; after
    // the barrier every wave's part of stage kt is in LDS and nobody reads the
    // previous buffer any more, so it is refilled with stage kt + AHEAD; then
    // the k16 steps of stage kt, software-pipelined: the fragments of step s
    // are read while the MFMAs of step s - 1 run (the last step of a stage,
    // already in registers, runs after the next barrier).
    if (VMC == 0)
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else if (VMC == 6)
      asm volatile("s_waitcnt vmcnt(6) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else if (VMC == 8)
      asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else if (VMC == 10)
      asm volatile("s_waitcnt vmcnt(10) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else if (VMC == 12)
      asm volatile("s_waitcnt vmcnt(12) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(16) lgkmcnt(0)\n\ts_barrier" ::: "memory");
    const int prev = (buf == 0) ? STAGES - 1 : buf - 1;
    EXF_W_ISSUE(prev, kt + AHEAD);
    {
#pragma unroll
      for (int s_ = 0; s_ < BK / 16; ++s_) {
        EXF_W_FRAGS(fa[s_ & 1], fb[s_ & 1], buf, s_);
        if (s_ > 0) {
          EXF_W_MMA(fa[(s_ - 1) & 1], fb[(s_ - 1) & 1]);
          // one LDS read after each of the first MFMAs
          constexpr int MF = TMV * TN, RD = TMV > 0 ? TMV + TN : 0, PAIRS = MF < RD ? MF : RD;
#pragma unroll
          for (int g_ = 0; g_ < PAIRS; ++g_) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          if (MF > PAIRS) __builtin_amdgcn_sched_group_barrier(0x008, MF - PAIRS, 0);
          if (RD > PAIRS) __builtin_amdgcn_sched_group_barrier(0x100, RD - PAIRS, 0);
        } else if (kt > k0) {
          EXF_W_MMA(fa[1], fb[1]);
        }
      }
    }
    buf = (buf == STAGES - 1) ? 0 : buf + 1;
  }
  EXF_W_MMA(fa[1], fb[1]);
  // the clamped loads past the end land before the ring is refilled or released,
  // and no wave still reads it
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
#undef EXF_W_ISSUE
#undef EXF_W_FRAGS
#undef EXF_W_MMA
}

// Accumulator layout: the MFMAs take the weight fragment as their first
// operand, so register r of tile (i, j) of wave (wm, wn) holds tile row (token)
// 128 wm + 32 i + lane % 32 and tile column 32 TN wn + 32 j + 8 (r / 4) +
// 4 (lane / 32) + r % 4: each lane owns four runs of four consecutive columns of
// one row, stored 8 (bf16) or 16 (fp32) bytes at a time.
__device__ __forceinline__ void store4_bf16(bf16_t *dst, float a, float b, float c, float d) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};   // two v_cvt_pk_bf16_f32
  *reinterpret_cast<bf16x4 *>(dst) = v;
}
// The same as a non-temporal store, for the layer output y written by the wide
// down GEMM (nothing in the layer reads it back): its lines are not kept dirty
// in the caches, whose later write-back otherwise lands in the next kernels (a
// decode forward right after the Mixtral-shaped prefill: 265.0-265.2 against
// 268.9-270.1 us, the prefill unchanged).
__device__ __forceinline__ void store4_bf16_nt(bf16_t *dst, float a, float b, float c, float d) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  const bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
  __builtin_nontemporal_store(*reinterpret_cast<const u32x2 *>(&v), reinterpret_cast<u32x2 *>(dst));
}

// Finished tile: gate/up writes H = SiLU(gate) * up; down writes y (direct)
// or fp32 rows Y scaled by the row's routing weight, or unscaled bf16 rows Yh
// (the combine applies the weight).
template <bool GATE_UP, bool DIRECT, int NW, bool DBL>
__device__ __forceinline__ void wide_store(const GemmKArgs &p, const TileId &t, int row0, int valid,
                                           const f32x16 (&acc)[kWideTM][kWideTN]) {
  constexpr int WN = DBL ? NW : NW / 2, TN = kWideTN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int c4 = 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < kWideTM; ++i) {
    const int ml = wm * 128 + i * 32 + (lane & 31);
    if (ml >= valid) continue;
    const int row = row0 + ml;
    if (GATE_UP) {
      bf16_t *dst = p.H + (long long)row * p.inter + t.nt * (kWideBN / 2) + wn * 16 * TN + c4;
#pragma unroll
      for (int j = 0; j < TN / 2; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16 &gt = acc[i][j], &up = acc[i][j + TN / 2];
          store4_bf16(dst + j * 32 + 8 * g, silu(gt[4 * g]) * up[4 * g], silu(gt[4 * g + 1]) * up[4 * g + 1],
                      silu(gt[4 * g + 2]) * up[4 * g + 2], silu(gt[4 * g + 3]) * up[4 * g + 3]);
        }
    } else {
      const float w = p.Yh && !DIRECT ? 1.f : p.row_w[row];
      const int n0 = t.nt * kWideBN + wn * 32 * TN + c4;
      const long long base = DIRECT ? (long long)p.row_token[row] * p.d : (long long)row * p.d;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16 &c = acc[i][j];
          const int n = n0 + j * 32 + 8 * g;
          const float v0 = c[4 * g] * w, v1 = c[4 * g + 1] * w, v2 = c[4 * g + 2] * w, v3 = c[4 * g + 3] * w;
          if (DIRECT)
            store4_bf16_nt(p.y + base + n, v0, v1, v2, v3);
          else if (p.Yh)
            store4_bf16(p.Yh + base + n, v0, v1, v2, v3);
          else
            *reinterpret_cast<float4 *>(p.Y + ((long long)t.ks * p.rows + row) * p.d + n) =
                make_float4(v0, v1, v2, v3);
        }
    }
  }
}

// Finished bf16 tile through LDS (the ring is free after the main loop): each
// lane writes its runs of four columns (SiLU(gate) * up, or the down output,
// scaled by the row's routing weight only when it goes straight to y) into a
// row-major bf16 tile, and the
// workgroup then stores whole rows 16 bytes a lane, so one store instruction
// covers a few complete rows instead of 32 scattered 16-byte pieces.  Taken
// for the bf16 rows of the down projection (Qwen3-shaped prefill: down 200 ->
// 177 us); for H and the direct y it cost more than it saved (the extra path
// spills scalar registers in those kernels).
template <bool GATE_UP, bool DIRECT, int NW, bool DBL>
__device__ __forceinline__ void wide_store_lds(const GemmKArgs &p, const TileId &t, int row0, int valid,
                                               const f32x16 (&acc)[kWideTM][kWideTN], bf16_t *smem) {
  constexpr int WN = DBL ? NW : NW / 2, TN = kWideTN, BM = DBL ? kWide / 2 : kWide;
  constexpr int COLS = (GATE_UP ? 16 : 32) * TN * WN;        // output columns of the tile
  constexpr int PITCH = COLS * 2 + 16;                        // LDS bytes per row (padded)
  static_assert(BM * PITCH <= kWideSmemElems * 2, "staging tile fits the ring");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int c4 = 4 * (lane >> 5);
  char *lds = reinterpret_cast<char *>(smem);
#pragma unroll
  for (int i = 0; i < kWideTM; ++i) {
    const int ml = wm * 128 + i * 32 + (lane & 31);
    const float w = (!GATE_UP && DIRECT && ml < valid) ? p.row_w[row0 + ml] : 1.f;
    char *rowp = lds + ml * PITCH;
    if (GATE_UP) {
#pragma unroll
      for (int j = 0; j < TN / 2; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16 &gt = acc[i][j], &up = acc[i][j + TN / 2];
          store4_bf16(reinterpret_cast<bf16_t *>(rowp) + wn * 16 * TN + j * 32 + 8 * g + c4,
                      silu(gt[4 * g]) * up[4 * g], silu(gt[4 * g + 1]) * up[4 * g + 1],
                      silu(gt[4 * g + 2]) * up[4 * g + 2], silu(gt[4 * g + 3]) * up[4 * g + 3]);
        }
    } else {
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x16 &c = acc[i][j];
          store4_bf16(reinterpret_cast<bf16_t *>(rowp) + wn * 32 * TN + j * 32 + 8 * g + c4, c[4 * g] * w,
                      c[4 * g + 1] * w, c[4 * g + 2] * w, c[4 * g + 3] * w);
        }
    }
  }
  lds_barrier();
  constexpr int CPR = COLS / 8;                               // 16-byte chunks per row
  for (int q = threadIdx.x; q < BM * CPR; q += 64 * NW) {
    const int ml = q / CPR, ch = q % CPR;
    if (ml >= valid) continue;
    const int row = row0 + ml;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(lds + ml * PITCH + ch * 16);
    bf16_t *dst;
    if (GATE_UP)
      dst = p.H + (long long)row * p.inter + t.nt * (kWideBN / 2);
    else if (DIRECT)
      dst = p.y + (long long)p.row_token[row] * p.d + t.nt * kWideBN;
    else
      dst = p.Yh + (long long)row * p.d + t.nt * kWideBN;
    *reinterpret_cast<u32x4 *>(dst + ch * 8) = v;
  }
}


// ---------------------------------------------------------------------------
// Wide-tile launches: whole rounds of tiles plus a split remainder.  With one
// workgroup per CU (the ring takes 128 KiB of LDS), tiles run in rounds of G =
// CU count; the last, partial round would leave most CUs idle.  When it holds
// at most half a round, its rem tiles have their reductions cut into s equal
// ranges of stages (s = G / rem, at most kWideMaxSplit, at least four stages a
// range) on separate workgroups: range c of remainder tile r leaves its fp32
// partial tile in P[r s + c], and expert_wide_fixup adds the s partials in
// range order and applies the epilogue.  Whole tiles keep the lock-step order
// in which the m-tiles of one weight panel and the n-tiles of one row block
// share an XCD's L2 (dealing the stages of every tile out evenly instead
// breaks that sharing: measured slower).  The ranges of one remainder tile are
// disjoint in K, so the remainder is laid out range-major: neighbouring
// workgroups take neighbouring tiles over the same stages.  The sums depend on
// the problem and G only, so the result is deterministic.
// ---------------------------------------------------------------------------
constexpr int kWideTileElems = kWide * kWide;
constexpr int kWideMaxSplit = 16;

struct WideSplit {
  int ndp;  // tiles run whole: logical ids 0 .. ndp - 1
  int rem;  // tiles split s ways: logical ids ndp .. ndp + rem - 1
  int s;
};
__device__ __forceinline__ WideSplit wide_split(const GemmKArgs &p, int G) {
  const int total = p.tile_start[p.groups] * (p.n_tiles / 2);
  const int rem = total % G;
  const int s = rem > 0 ? min(G / rem, min(kWideMaxSplit, p.kc / kWideBK / 4)) : 1;
  if (rem > 0 && s >= 2) return WideSplit{total - rem, rem, s};
  return WideSplit{total, 0, 1};
}

// Partial tile in the accumulator layout: row-major, 256 (DBL: 512) columns.
template <bool DBL>
__device__ __forceinline__ void wide_store_partial(float *P, const f32x16 (&acc)[kWideTM][kWideTN]) {
  constexpr int WN = DBL ? kWideWaves : kWideWaves / 2, BN = 32 * kWideTN * WN;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
#pragma unroll
  for (int i = 0; i < kWideTM; ++i) {
    float *prow = P + (wm * 128 + i * 32 + (lane & 31)) * BN + wn * 32 * kWideTN + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < kWideTN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x16 &c = acc[i][j];
        *reinterpret_cast<float4 *>(prow + j * 32 + 8 * g) =
            make_float4(c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]);
      }
  }
}

// Workgroup blockIdx.x of a launch of ndp + rem s workgroups (more exit).
template <bool GATE_UP, bool DIRECT>
__device__ __forceinline__ void wide_gemm(const GemmKArgs &p, int G, bf16_t *smem) {
  constexpr int NW = kWideWaves;
  const WideSplit w = wide_split(p, G);
  const int KT = p.kc / kWideBK;
  const int b = blockIdx.x;
  TileId t;
  int k0 = 0, k1 = KT;
  float *part = nullptr;
  if (b < w.ndp) {
    wide_tile_at(p, xcd_remap(b, w.ndp), t);
  } else {
    const int j = b - w.ndp, n = w.rem * w.s;
    if (j >= n) return;
    const int lj = xcd_remap(j, n), c = lj / w.rem, r = lj % w.rem;
    wide_tile_at(p, w.ndp + r, t);
    k0 = c * KT / w.s;
    k1 = (c + 1) * KT / w.s;
    part = p.P + (size_t)(r * w.s + c) * kWideTileElems;
  }
  const int row0 = p.offsets[t.g] + t.mt * kWide;
  f32x16 acc[kWideTM][kWideTN];
  // the wave's 32-row blocks that hold rows of the group (wave-uniform)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  auto blocks = [&](int valid, int wm) { return max(0, min(kWideTM, (valid - wm * 128 + 31) >> 5)); };
#define EXF_W_MAIN(DBL_, TMV_) \
  wide_tile_mma<GATE_UP, kWideBK, kWideStages, NW, DBL_, TMV_>(p, t, row0, valid, k0, k1, smem, acc)
#define EXF_W_DISPATCH(DBL_, TMV_VAL)                                                          \
  switch (TMV_VAL) {                                                                           \
    case 4: EXF_W_MAIN(DBL_, 4); break;                                                        \
    case 3: EXF_W_MAIN(DBL_, 3); break;                                                        \
    case 2: EXF_W_MAIN(DBL_, 2); break;                                                        \
    case 1: EXF_W_MAIN(DBL_, 1); break;                                                        \
    default: EXF_W_MAIN(DBL_, 0); break;                                                       \
  }
  static_assert(kWideTM == 4, "the dispatch below covers 0 .. 4 valid row blocks");
  if (__builtin_amdgcn_readfirstlane(t.dbl)) {
    const int valid = min(kWide / 2, p.offsets[t.g + 1] - row0);
    EXF_W_DISPATCH(true, blocks(valid, 0))
    if (part)
      wide_store_partial<true>(part, acc);
    else if (!GATE_UP && !DIRECT && p.Yh)
      wide_store_lds<GATE_UP, DIRECT, NW, true>(p, t, row0, valid, acc, smem);
    else
      wide_store<GATE_UP, DIRECT, NW, true>(p, t, row0, valid, acc);
  } else {
    const int valid = min(kWide, p.offsets[t.g + 1] - row0);
    EXF_W_DISPATCH(false, blocks(valid, wave / (NW / 2)))
    if (part)
      wide_store_partial<false>(part, acc);
    else if (!GATE_UP && !DIRECT && p.Yh)
      wide_store_lds<GATE_UP, DIRECT, NW, false>(p, t, row0, valid, acc, smem);
    else
      wide_store<GATE_UP, DIRECT, NW, false>(p, t, row0, valid, acc);
  }
#undef EXF_W_MAIN
#undef EXF_W_DISPATCH
}


__global__ __launch_bounds__(64 * kWideWaves, 1) void expert_gate_up_wide(const GemmKArgs p, int G) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kWideSmemElems];
  wide_gemm<true, false>(p, G, smem);
}

template <bool DIRECT>
__global__ __launch_bounds__(64 * kWideWaves, 1) void expert_down_wide(const GemmKArgs p, int G) {
  __shared__ __attribute__((aligned(1024))) bf16_t smem[kWideSmemElems];
  wide_gemm<false, DIRECT>(p, G, smem);
}

// Block (r, c): remainder tile r, tile rows 16 c .. 16 c + 15, sixteen threads
// a row.  Gate/up: H columns 128 nt + col from the gate and up partials laid
// out as the accumulators of the waves (wide_store_partial); down: the 256
// (tail tile: 512) output columns scaled by the row's routing weight.
template <bool GATE_UP, bool DIRECT>
__global__ __launch_bounds__(256) void expert_wide_fixup(const GemmKArgs p, int G) {
  const WideSplit w = wide_split(p, G);
  const int r = blockIdx.x;
  if (r >= w.rem) return;
  TileId t;
  wide_tile_at(p, w.ndp + r, t);
  const int bm = t.dbl ? kWide / 2 : kWide, bn = t.dbl ? 2 * kWideBN : kWideBN;
  const int row0 = p.offsets[t.g] + t.mt * kWide;
  const int valid = min(bm, p.offsets[t.g + 1] - row0);
  const int ml = blockIdx.y * 16 + (threadIdx.x >> 4);
  if (ml >= valid) return;
  const int row = row0 + ml;
  const float *P0 = p.P + (size_t)r * w.s * kWideTileElems + (size_t)ml * bn;
  // all s partials of a column group are loaded before the in-order sum (the
  // loads do not wait on each other)
  auto sum4 = [&](int col) {
    float4 q[kWideMaxSplit];
#pragma unroll
    for (int k = 0; k < kWideMaxSplit; ++k)
      if (k < w.s) q[k] = *reinterpret_cast<const float4 *>(P0 + (size_t)k * kWideTileElems + col);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int k = 0; k < kWideMaxSplit; ++k)
      if (k < w.s) {
        v.x += q[k].x;
        v.y += q[k].y;
        v.z += q[k].z;
        v.w += q[k].w;
      }
    return v;
  };
  if (GATE_UP) {
    for (int q = 0; q < bn / 128; ++q) {
      const int col = q * 64 + (threadIdx.x & 15) * 4;
      // gate tile (col / 32) % (TN / 2) of wave col / (16 TN); its up tile TN / 2 further
      const int pc = (col / (16 * kWideTN)) * 32 * kWideTN + ((col >> 5) % (kWideTN / 2)) * 32 + (col & 31);
      const float4 g = sum4(pc), u = sum4(pc + 16 * kWideTN);
      const float h[4] = {silu(g.x) * u.x, silu(g.y) * u.y, silu(g.z) * u.z, silu(g.w) * u.w};
      bf16_t *dst = p.H + (long long)row * p.inter + t.nt * (kWideBN / 2) + col;
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[e] = f32_to_bf16(h[e]);
    }
  } else {
    const float rw = p.Yh && !DIRECT ? 1.f : p.row_w[row];
    for (int q = 0; q < bn / 64; ++q) {
      const int col = q * 64 + (threadIdx.x & 15) * 4;
      const float4 a = sum4(col);
      const float v[4] = {a.x * rw, a.y * rw, a.z * rw, a.w * rw};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int n = t.nt * kWideBN + col + e;
        if (DIRECT)
          __builtin_nontemporal_store(f32_to_bf16(v[e]), &p.y[(long long)p.row_token[row] * p.d + n]);
        else if (p.Yh)
          p.Yh[(long long)row * p.d + n] = f32_to_bf16(v[e]);
        else
          p.Y[(long long)row * p.d + n] = v[e];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Skinny tile for decode (few rows per retained expert): 32 rows x 64 output
// columns (gate/up: 32 gate + 32 up columns), BK = 128 per stage (256 contiguous
// bytes of every weight row per load step), and the four waves split each
// stage's reduction (wave w takes k16 steps w and w + 4) instead of the tile, so
// the weights stream through many small workgroups (three per CU by LDS).  The
// four partial tiles are added in wave order through LDS at the end.
// ---------------------------------------------------------------------------
constexpr int kSkM = 32, kSkN = 64, kSkK = 128;

// LDS element offset of 16-byte chunk q of row r in a 256-byte row (16 chunks):
// q XOR (r mod 16) spreads one chunk column of 16 consecutive rows over all banks.
__device__ __forceinline__ int swz16(int r, int q) { return (r * 16 + (q ^ (r & 15))) * 8; }

template <bool GATE_UP, bool DIRECT>
__global__ __launch_bounds__(256) void expert_gemm_skinny(const GemmKArgs p) {
  constexpr int PA = kSkM * 16 / 256, PB = kSkN * 16 / 256;  // 16-byte chunks per thread per stage
  constexpr int STAGE = (kSkM + kSkN) * kSkK;                  // elements per LDS stage
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * STAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  TileId t;
  if (!decode_tile(p, blockIdx.x, t)) return;
  const int row0 = p.offsets[t.g] + t.mt * kSkM;
  const int valid = min(kSkM, p.offsets[t.g + 1] - row0);
  const bf16_t *Wg = (t.g < p.n_experts) ? p.W + (long long)t.g * p.w_stride : p.Ws;

  // chunk c = i * 256 + tid: row c / 16, 16-byte column c % 16
  const bf16_t *a_src[PA];
  const bf16_t *b_src[PB];
#pragma unroll
  for (int i = 0; i < PA; ++i) {
    const int c = i * 256 + tid, r = c >> 4;
    const int rr = row0 + (r < valid ? r : 0);
    const long long arow = GATE_UP ? (long long)p.row_token[rr] : (long long)rr;
    a_src[i] = p.A + arow * p.lda + (long long)t.ks * p.kc + (c & 15) * 8;
  }
#pragma unroll
  for (int i = 0; i < PB; ++i) {
    const int c = i * 256 + tid, r = c >> 4;
    int wrow;
    if (GATE_UP)
      wrow = (r < kSkN / 2) ? t.nt * (kSkN / 2) + r : p.inter + t.nt * (kSkN / 2) + (r - kSkN / 2);
    else
      wrow = t.nt * kSkN + r;
    b_src[i] = Wg + (long long)wrow * p.ldw + (long long)t.ks * p.kc + (c & 15) * 8;
  }

  f32x16 acc[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;

#define EXF_SK_GLOAD(RA, RB, K0)                                                            \
  do {                                                                                      \
    _Pragma("unroll") for (int i_ = 0; i_ < PA; ++i_) RA[i_] =                              \
        *reinterpret_cast<const u32x4 *>(a_src[i_] + (K0));                                 \
    _Pragma("unroll") for (int i_ = 0; i_ < PB; ++i_) RB[i_] =                              \
        *reinterpret_cast<const u32x4 *>(b_src[i_] + (K0));                                 \
  } while (0)
#define EXF_SK_LSTORE(RA, RB, BUF)                                                          \
  do {                                                                                      \
    bf16_t *As_ = smem + (BUF) * STAGE;                                                     \
    bf16_t *Bs_ = As_ + kSkM * kSkK;                                                        \
    _Pragma("unroll") for (int i_ = 0; i_ < PA; ++i_) {                                     \
      const int c_ = i_ * 256 + tid;                                                        \
      *reinterpret_cast<u32x4 *>(&As_[swz16(c_ >> 4, c_ & 15)]) = RA[i_];                   \
    }                                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < PB; ++i_) {                                     \
      const int c_ = i_ * 256 + tid;                                                        \
      *reinterpret_cast<u32x4 *>(&Bs_[swz16(c_ >> 4, c_ & 15)]) = RB[i_];                   \
    }                                                                                       \
  } while (0)
  // wave w: k16 steps w and w + 4 of the stage; lane l reads row l % 32, 8 k at (l / 32) * 8
#define EXF_SK_COMPUTE(BUF)                                                                 \
  do {                                                                                      \
    const bf16_t *As_ = smem + (BUF) * STAGE;                                               \
    const bf16_t *Bs_ = As_ + kSkM * kSkK;                                                  \
    _Pragma("unroll") for (int h_ = 0; h_ < 2; ++h_) {                                      \
      const int ch_ = (wave + 4 * h_) * 2 + (lane >> 5);                                    \
      const bf16x8 a_ = *reinterpret_cast<const bf16x8 *>(&As_[swz16(lane & 31, ch_)]);     \
      const bf16x8 b0_ = *reinterpret_cast<const bf16x8 *>(&Bs_[swz16(lane & 31, ch_)]);    \
      const bf16x8 b1_ = *reinterpret_cast<const bf16x8 *>(&Bs_[swz16(32 + (lane & 31), ch_)]); \
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_, b0_, acc[0], 0, 0, 0);           \
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_, b1_, acc[1], 0, 0, 0);           \
    }                                                                                       \
  } while (0)

  // Two register sets: the loads of stage kt + 2 fly during the MFMAs of stage kt.
  const int KT = p.kc / kSkK;
  const int k_last = (KT - 1) * kSkK;
  u32x4 ra0[PA], rb0[PB], ra1[PA], rb1[PB];
  EXF_SK_GLOAD(ra0, rb0, 0);
  EXF_SK_LSTORE(ra0, rb0, 0);
  EXF_SK_GLOAD(ra1, rb1, min(kSkK, k_last));
  __syncthreads();
  int kt = 0;
  for (; kt + 2 <= KT; kt += 2) {
    EXF_SK_GLOAD(ra0, rb0, min((kt + 2) * kSkK, k_last));
    EXF_SK_COMPUTE(0);
    EXF_SK_LSTORE(ra1, rb1, 1);
    __syncthreads();
    EXF_SK_GLOAD(ra1, rb1, min((kt + 3) * kSkK, k_last));
    EXF_SK_COMPUTE(1);
    EXF_SK_LSTORE(ra0, rb0, 0);
    __syncthreads();
  }
  if (kt < KT) EXF_SK_COMPUTE(0);
#undef EXF_SK_GLOAD
#undef EXF_SK_LSTORE
#undef EXF_SK_COMPUTE

  // Partial tiles of the four waves, added in wave order (LDS reused).
  __syncthreads();
  float *red = reinterpret_cast<float *>(smem);  // [4][2][16][64] floats = 32 KB
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) red[((wave * 2 + j) * 16 + r) * 64 + lane] = acc[j][r];
  __syncthreads();
  // wave w finishes accumulator registers r in [4 w, 4 w + 4) of both column halves
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r = wave * 4 + q;
      float v = red[((0 * 2 + j) * 16 + r) * 64 + lane];
#pragma unroll
      for (int w = 1; w < 4; ++w) v += red[((w * 2 + j) * 16 + r) * 64 + lane];
      acc[j][q] = v;
    }

  // ---- epilogue: rows (r / 4) * 8 + (lane / 32) * 4 + r % 4 of the 32x32 MFMA layout ----
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int r = wave * 4 + q;
    const int ml = (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
    if (ml < valid) {
      const int row = row0 + ml;
      if (GATE_UP) {
        const int n = t.nt * (kSkN / 2) + (lane & 31);
        p.H[(long long)row * p.inter + n] = f32_to_bf16(silu(acc[0][q]) * acc[1][q]);
      } else {
        const float w = p.row_w[row];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int n = t.nt * kSkN + j * 32 + (lane & 31);
          if (DIRECT)
            p.y[(long long)p.row_token[row] * p.d + n] = f32_to_bf16(acc[j][q] * w);
          else if (p.Yh)
            p.Yh[(long long)row * p.d + n] = f32_to_bf16(acc[j][q]);
          else
            p.Y[((long long)t.ks * p.rows + row) * p.d + n] = acc[j][q] * w;
        }
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
    *gu = GemmPlan{4, 64, 1, 0, kGemmSimt};
    *dn = GemmPlan{4, 64, 1, 0, kGemmSimt};
    return;
  }
  // The plan depends on the problem only (rows, groups, sizes), never on the
  // phase, so equal problems get equal plans.
  const int active = active_groups < 1 ? 1 : active_groups;
  // Few rows per retained expert (decode): skinny 32x64 tiles stream the weights
  // through many small workgroups; otherwise 128x128 tiles.  The gate/up
  // projection takes 128-row tiles once the experts hold more than about 24
  // rows each, even where those tiles do not cover the CUs: skinny tiles then
  // read the weights of a busy expert more than once (Qwen3-shaped decode, 128
  // tokens on a pool of 16: 80.8 against 85.6 us per layer).
  const bool sk_shapes = inter % 128 == 0 && d % 64 == 0;
  const bool gu_skinny = sk_shapes && rows <= 24 * active;
  // Many rows per retained expert (prefill, at least 128 on average): wide
  // tiles.  With the 128-row tail tiles a skewed load pays at most half a tile
  // per group: the Qwen3-shaped prefill (8192 tokens, K' = 4, 98 of 128 experts
  // busy, 334 rows on average, 3974 at most) runs 19% faster than on 128x128.
  // Fewer than a quarter round of wide tiles (then split four ways or more)
  // loses to 128x128 tiles (Qwen3-shaped decode, 256 tokens on a pool of 16,
  // 48 wide tiles: 130.8 against 103.8 us per layer).
  const bool gu_wide = !gu_skinny && inter % kWideBN == 0 && d % 128 == 0 && 2 * rows >= kWide * active &&
                       (long long)(rows / 128) * (inter / kWideBN) * 4 >= cu_count;
  // The down projection keeps skinny tiles up to about 48 rows per expert (at
  // 64, 128x128 tiles: Qwen3-shaped decode, 256 tokens on a pool of 32, 115
  // against 125 us per layer).
  const bool dn_skinny = sk_shapes && rows <= 48 * active;
  if (gu_skinny) {
    *gu = GemmPlan{kSkM, kSkN, 1, 0, kGemmSkinny};
    gu->grid = (rows / kSkM + groups) * (inter / (kSkN / 2));  // >= sum of ceil(rows_g / 32) tiles
  } else if (gu_wide) {
    // tile list in 128-row units, one tile per unit and pair of 128-column
    // n-tiles; whole rounds plus the split remainder: at most that + one round
    *gu = GemmPlan{kWide / 2, kWideBN, 1, 0, kGemmWide, cu_count};
    gu->grid = (rows / 128 + groups) * (inter / kWideBN) + cu_count;
  } else {
    *gu = GemmPlan{128, 128, 1, 0, kGemmTile};
    gu->grid = (rows / 128 + groups) * (inter / 64);
  }
  // Down projection on the wide tile where the gate/up projection takes it,
  // also when its tiles do not fill one round (they then all run split along
  // the reduction: Qwen3-shaped decode, 512 tokens on a pool of 32, 150.7
  // against 160.0 us per layer with 128x128 tiles).
  if (!dn_skinny && gu_wide && d % (2 * kWideBN) == 0) {
    *dn = GemmPlan{kWide / 2, kWideBN, 1, 0, kGemmWide, cu_count};
    dn->grid = (rows / 128 + groups) * (d / (2 * kWideBN)) + cu_count;
    return;
  }
  // Few expected tiles: split the down projection's reduction so the workgroups
  // still cover every CU.  Partial sums land in separate buffers and are added
  // in a fixed order by the combine.  Only long reductions are split: every
  // range keeps at least kMinSplitStages stages (an intermediate size of 768
  // split three ways ran 3 us slower per decode layer than unsplit, a 14336
  // one split in two 20 us faster).
  const int bm = dn_skinny ? kSkM : 128;
  const int bn = dn_skinny ? kSkN : 128;
  const int kk = dn_skinny ? kSkK : kBK, fill = dn_skinny ? 3 : 2;
  *dn = GemmPlan{bm, bn, 1, 0, dn_skinny ? kGemmSkinny : kGemmTile};
  const int mt_expect = (rows + bm - 1) / bm > active ? (rows + bm - 1) / bm : active;
  const int dn_tiles = mt_expect * (d / bn);
  constexpr int kMinSplitStages = 8;
  const int max_split = (inter / kk) / kMinSplitStages;
  if (dn_tiles < fill * cu_count && max_split >= 2) {
    const int want = (fill * cu_count + dn_tiles - 1) / dn_tiles;
    const int cap = want < max_split ? want : max_split;
    dn->ksplit = largest_divisor_at_most(inter / kk, cap > 8 ? 8 : cap);
  }
  dn->grid = (rows / bm + groups) * (d / bn) * dn->ksplit;
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
  ga.rows = a.rows;
  ga.W = static_cast<const bf16_t *>(a.w_gate_up);
  ga.Ws = static_cast<const bf16_t *>(a.ws_gate_up);
  ga.w_stride = 2LL * a.inter * a.d;
  ga.ldw = a.d;
  ga.inter = a.inter;
  ga.d = a.d;
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
  da.rows = a.rows;
  da.W = static_cast<const bf16_t *>(a.w_down);
  da.Ws = static_cast<const bf16_t *>(a.ws_down);
  da.w_stride = (long long)a.d * a.inter;
  da.ldw = a.inter;
  da.inter = a.inter;
  da.d = a.d;
  da.Y = a.y_bf16 ? nullptr : a.Y;
  da.Yh = a.y_bf16 ? reinterpret_cast<bf16_t *>(a.Y) : nullptr;
  da.y = static_cast<bf16_t *>(a.y);
  da.row_w = a.row_w;

  if (gu.grid > 0) {
    if (gu.kind == kGemmSkinny) {
      expert_gemm_skinny<true, false><<<gu.grid, 256, 0, s>>>(ga);
    } else if (gu.kind == kGemmWide) {
      ga.P = a.wide_part;
      expert_gate_up_wide<<<gu.grid, 64 * kWideWaves, 0, s>>>(ga, gu.wgs);
      expert_wide_fixup<true, false><<<dim3(gu.wgs / 2, kWide / 16), 256, 0, s>>>(ga, gu.wgs);
    } else {
      expert_gemm_tile<128, 128, 2, true, false><<<gu.grid, 256, 0, s>>>(ga);
    }
  }
  if (ev_mid) (void)hipEventRecord(ev_mid, s);
  if (dn.grid > 0) {
    if (dn.kind == kGemmWide) {
      da.P = a.wide_part;
      const dim3 fg(dn.wgs / 2, kWide / 16);
      if (a.direct) {
        expert_down_wide<true><<<dn.grid, 64 * kWideWaves, 0, s>>>(da, dn.wgs);
        expert_wide_fixup<false, true><<<fg, 256, 0, s>>>(da, dn.wgs);
      } else {
        expert_down_wide<false><<<dn.grid, 64 * kWideWaves, 0, s>>>(da, dn.wgs);
        expert_wide_fixup<false, false><<<fg, 256, 0, s>>>(da, dn.wgs);
      }
    } else if (dn.kind == kGemmSkinny) {
      if (a.direct)
        expert_gemm_skinny<false, true><<<dn.grid, 256, 0, s>>>(da);
      else
        expert_gemm_skinny<false, false><<<dn.grid, 256, 0, s>>>(da);
    } else {
      if (a.direct)
        expert_gemm_tile<128, 128, 2, false, true><<<dn.grid, 256, 0, s>>>(da);
      else
        expert_gemm_tile<128, 128, 2, false, false><<<dn.grid, 256, 0, s>>>(da);
    }
  }
  return hipGetLastError();
}

int plain_gemm_splits(int M, int N, int K, int cu_count) {
  if (M <= 0 || N % 128 != 0 || K % kBK != 0) return 0;
  const int tiles = (M + 127) / 128 * (N / 128);
  int P = 1;
  // split the reduction until the tiles cover the CUs, every range at least
  // four stages of kBK
  while (tiles * P < cu_count && P < 8 && K % (2 * P * kBK) == 0 && K / (2 * P) >= 4 * kBK) P *= 2;
  return P;
}

hipError_t launch_plain_gemm_nt(const void *A, const void *W, int M, int N, int K, int P, float *part,
                                hipStream_t s) {
  GemmKArgs g{};
  g.A = static_cast<const bf16_t *>(A);
  g.lda = K;
  g.W = static_cast<const bf16_t *>(W);
  g.ldw = K;
  g.rows = M;
  g.d = N;
  g.n_tiles = N / 128;
  g.ksplit = P;
  g.kc = K / P;
  g.Y = part;
  const int grid = (M + 127) / 128 * g.n_tiles * P;
  expert_gemm_tile<128, 128, 2, false, false, true><<<grid, 256, 0, s>>>(g);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weighted combine: y_i = sum_k Y[row(i,k)] (+ shared row), in slot order;
// float32 accumulation, one rounding to the output dtype.
// ---------------------------------------------------------------------------
template <typename InT>
__device__ __forceinline__ float4 load4(const InT *p);
template <>
__device__ __forceinline__ float4 load4<float>(const float *p) {
  return *reinterpret_cast<const float4 *>(p);
}
template <>
__device__ __forceinline__ float4 load4<bf16_t>(const bf16_t *p) {
  const uint2 u = *reinterpret_cast<const uint2 *>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

template <typename InT, int C>
__device__ __forceinline__ void load_cols(const InT *p, float (&v)[C]) {
#pragma unroll
  for (int q = 0; q < C; q += 4) {
    const float4 f = load4<InT>(p + q);
    v[q] = f.x;
    v[q + 1] = f.y;
    v[q + 2] = f.z;
    v[q + 3] = f.w;
  }
}

template <typename InT, typename OutT, int C, bool PAIRS>
__global__ __launch_bounds__(256) void combine_kernel(const InT *__restrict__ Y, int ksplit,
                                                     int rows, const int32_t *__restrict__ slot_row,
                                                     const float *__restrict__ row_w,
                                                     int k_out, int d, int shared_base,
                                                     OutT *__restrict__ y) {
  // block (i, c): token i, columns [256 C c, 256 C (c + 1)), C per thread.  The
  // token's row indices are loaded first (one round trip), then the rows are
  // loaded four at a time and added in slot order, split partials in order.
  // bf16 rows arrive unscaled: each is multiplied by its routing weight here,
  // in fp32, so two routes of one token to the same expert share one rounded
  // row and their weights add exactly as in the unrounded sum.
  const int i = blockIdx.x;
  const int c = (blockIdx.y * 256 + threadIdx.x) * C;
  if (c >= d) return;
  const long long split = (long long)rows * d;
  const int nr = k_out + (shared_base >= 0 ? 1 : 0);
  int r[kMaxTopK + 1];
#pragma unroll
  for (int k = 0; k <= kMaxTopK; ++k)
    r[k] = (k < k_out) ? slot_row[(long long)i * k_out + k] : (k == k_out && shared_base >= 0) ? shared_base + i : 0;
  constexpr bool kScale = sizeof(InT) == 2;
  float rw[kMaxTopK + 1];
#pragma unroll
  for (int k = 0; k <= kMaxTopK; ++k) rw[k] = (kScale && k < nr) ? row_w[r[k]] : 1.f;
  float acc[C];
#pragma unroll
  for (int q = 0; q < C; ++q) acc[q] = 0.f;
  for (int sp = 0; sp < ksplit; sp += 2) {
    // splits sp and sp + 1 of four rows at a time, all loaded before the adds
    // (rows in slot order, the two splits in order); with one split this is
    // the whole sum in slot order
    const InT *base = Y + sp * split + c;
    const bool two = PAIRS && sp + 1 < ksplit;
#pragma unroll
    for (int k0 = 0; k0 <= kMaxTopK; k0 += 4) {
      if (k0 >= nr) break;
      float v[2][4][C];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (k0 + u < nr) {
          load_cols<InT, C>(base + (long long)r[k0 + u] * d, v[0][u]);
          if (two) load_cols<InT, C>(base + split + (long long)r[k0 + u] * d, v[1][u]);
        }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (k0 + u < nr && (h == 0 || two)) {
#pragma unroll
            for (int q = 0; q < C; ++q) acc[q] = kScale ? fmaf(rw[k0 + u], v[h][u][q], acc[q]) : acc[q] + v[h][u][q];
          }
    }
  }
  OutT *o = y + (long long)i * d + c;
#pragma unroll
  for (int q = 0; q < C; q += 4) {
    if constexpr (sizeof(OutT) == 2)
      store4_bf16(reinterpret_cast<bf16_t *>(o) + q, acc[q], acc[q + 1], acc[q + 2], acc[q + 3]);
    else
      *reinterpret_cast<float4 *>(o + q) = make_float4(acc[q], acc[q + 1], acc[q + 2], acc[q + 3]);
  }
}

template <typename InT, typename OutT>
static void launch_combine_t(const InT *Y, int ksplit, int rows, const int32_t *slot_row, const float *row_w,
                             int T, int k_out, int d, int shared_base, OutT *y, hipStream_t s) {
  // eight columns a thread once the grid covers the CUs a few times over; four below
  if ((long long)T * d >= 256LL * 256 * 8 * 4) {
    const dim3 grid(T, (d + 2047) / 2048);
    if (ksplit > 1)
      combine_kernel<InT, OutT, 8, true><<<grid, 256, 0, s>>>(Y, ksplit, rows, slot_row, row_w, k_out, d,
                                                                   shared_base, y);
    else
      combine_kernel<InT, OutT, 8, false><<<grid, 256, 0, s>>>(Y, ksplit, rows, slot_row, row_w, k_out, d,
                                                                   shared_base, y);
  } else {
    const dim3 grid(T, (d + 1023) / 1024);
    if (ksplit > 1)
      combine_kernel<InT, OutT, 4, true><<<grid, 256, 0, s>>>(Y, ksplit, rows, slot_row, row_w, k_out, d,
                                                                   shared_base, y);
    else
      combine_kernel<InT, OutT, 4, false><<<grid, 256, 0, s>>>(Y, ksplit, rows, slot_row, row_w, k_out, d,
                                                                   shared_base, y);
  }
}

hipError_t launch_combine(int dtype, const float *Y, bool y_bf16, int ksplit, int rows,
                          const int32_t *slot_row, const float *row_w, int T, int k_out, int d,
                          int shared_base, void *y, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  if (dtype == EXFOLD_BF16 && y_bf16)
    launch_combine_t<bf16_t, bf16_t>(reinterpret_cast<const bf16_t *>(Y), ksplit, rows, slot_row, row_w, T, k_out,
                                     d, shared_base, static_cast<bf16_t *>(y), s);
  else if (dtype == EXFOLD_BF16)
    launch_combine_t<float, bf16_t>(Y, ksplit, rows, slot_row, nullptr, T, k_out, d, shared_base,
                                    static_cast<bf16_t *>(y), s);
  else
    launch_combine_t<float, float>(Y, ksplit, rows, slot_row, nullptr, T, k_out, d, shared_base,
                                   static_cast<float *>(y), s);
  return hipGetLastError();
}

}  // namespace exfold

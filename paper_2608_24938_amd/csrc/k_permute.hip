// Stable permutation of the executed route slots by expert id.  Folded routes
// are grouped per retained expert before the expert computation (Sec. 4.1:
// routes folded onto one target are coalesced before expert computation, so
// each retained expert runs once over its rows).
//
// count:   per-block expert histograms (LDS integer atomics; order-free)
// scan:    exclusive scans -> group offsets, per-block bases, GEMM m-tile lists
// scatter: per-block stable ranks (wave match by ballots + cross-wave prefix)
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

constexpr int kPermThreads = 256;
constexpr int kScanLdsInts = 16384;  // per-block counts scanned in LDS up to 64 KiB
constexpr int kPermRounds = kPermSlotsPerBlock / kPermThreads;
constexpr int kPermOneBlockSlots = 4096;
static_assert(kPermOneBlockSlots <= kDecodeFrontMaxSlots, "one-workgroup permutation capacity");

__global__ __launch_bounds__(kPermThreads) void perm_count_kernel(const int32_t *__restrict__ ids,
                                                                  int R, int N,
                                                                  int32_t *__restrict__ blk_counts) {
  __shared__ int cnt[kMaxExperts];
  for (int e = threadIdx.x; e < N; e += kPermThreads) cnt[e] = 0;
  __syncthreads();
  const int lo = blockIdx.x * kPermSlotsPerBlock;
  const int hi = min(R, lo + kPermSlotsPerBlock);
  for (int j = lo + threadIdx.x; j < hi; j += kPermThreads) atomicAdd(&cnt[clamp_id(ids[j], N)], 1);
  __syncthreads();
  for (int e = threadIdx.x; e < N; e += kPermThreads) blk_counts[(size_t)blockIdx.x * N + e] = cnt[e];
}

// One thread per group in the scan kernel: kScanWaves waves cover the
// kMaxExperts + 1 groups (routed experts, shared expert).
constexpr int kScanWaves = (kMaxExperts + 1 + kWave - 1) / kWave;
constexpr int kScanThreads = kScanWaves * kWave;

__global__ __launch_bounds__(kScanThreads) void perm_scan_kernel(
    int32_t *__restrict__ blk_counts, int nblk, int N, int R, int t_shared, int bm0, int bm1,
    int32_t *__restrict__ offsets, int32_t *__restrict__ tile_start0,
    int32_t *__restrict__ tile_start1) {
  __shared__ int part[3 * kScanWaves];
  __shared__ int off_sh[kMaxExperts];
  // The per-block counts are scanned in LDS when they fit (one coalesced read
  // and one write): a per-expert walk over the blocks in global memory is a
  // chain of nblk dependent load/store round trips (32 blocks: about 20 us).
  __shared__ int cl[kScanLdsInts];
  const int tid = threadIdx.x;
  const bool in_lds = (long long)nblk * N <= kScanLdsInts;
  const int groups = N + (t_shared > 0 ? 1 : 0);
  if (in_lds) {
    for (int i = tid; i < nblk * N; i += kScanThreads) cl[i] = blk_counts[i];
    lds_barrier();
  }
  // Thread e: exclusive scan of expert e's counts over the blocks, in block
  // order; the counts are read eight blocks at a time.
  int total = 0;
  if (tid < N) {
    constexpr int kB = 8;
    int *base = in_lds ? cl : blk_counts;
    int b = 0;
    for (; b + kB <= nblk; b += kB) {
      int c[kB];
#pragma unroll
      for (int q = 0; q < kB; ++q) c[q] = base[(size_t)(b + q) * N + tid];
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        base[(size_t)(b + q) * N + tid] = total;
        total += c[q];
      }
    }
    for (; b < nblk; ++b) {
      const int c = base[(size_t)b * N + tid];
      base[(size_t)b * N + tid] = total;
      total += c;
    }
  }
  // Group g: rows, m-tiles of height bm0 and bm1; exclusive scans over groups.
  int v[3] = {0, 0, 0};
  if (tid < groups) {
    const int r = tid < N ? total : t_shared;
    v[0] = r;
    v[1] = (r + bm0 - 1) / bm0;
    v[2] = (r + bm1 - 1) / bm1;
  }
  int ex[3], tot[3];
  block_scan3<kScanWaves>(v, ex, tot, part);
  if (tid < N) {
    offsets[tid] = ex[0];
    off_sh[tid] = ex[0];
  }
  if (tid == N) offsets[N] = R;
  if (tid == N + 1) offsets[N + 1] = R + t_shared;
  if (tid < N + 2) {
    tile_start0[tid] = tid < groups ? ex[1] : tot[1];
    tile_start1[tid] = tid < groups ? ex[2] : tot[2];
  }
  // Per-block bases: the block's exclusive prefix plus the group offset.
  if (in_lds) {
    lds_barrier();
    for (int i = tid; i < nblk * N; i += kScanThreads) blk_counts[i] = cl[i] + off_sh[i % N];
  } else if (tid < N) {
    for (int b = 0; b < nblk; ++b) blk_counts[(size_t)b * N + tid] += ex[0];
  }
}

__global__ __launch_bounds__(kPermThreads) void perm_scatter_kernel(
    const int32_t *__restrict__ ids, const float *__restrict__ route_w, int R, int k_out, int N,
    int t_shared, const int32_t *__restrict__ blk_base, int32_t *__restrict__ row_token,
    int32_t *__restrict__ row_slot, float *__restrict__ row_w, int32_t *__restrict__ slot_row) {
  __shared__ int cur[kMaxExperts];
  __shared__ int wcnt[kPermThreads / kWave][kMaxExperts];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int e = tid; e < N; e += kPermThreads) {
    cur[e] = blk_base[(size_t)blockIdx.x * N + e];
#pragma unroll
    for (int w = 0; w < kPermThreads / kWave; ++w) wcnt[w][e] = 0;
  }
  __syncthreads();
  const int lo = blockIdx.x * kPermSlotsPerBlock;
  for (int round = 0; round < kPermRounds; ++round) {
    const int j = lo + round * kPermThreads + tid;
    const bool valid = j < R;
    const int e = valid ? clamp_id(ids[j], N) : 0;
    // lanes of this wave holding the same expert id
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool set = (e >> bit) & 1;
      const uint64_t bal = __ballot(set);
      m &= set ? bal : ~bal;
    }
    const int rank = __popcll(m & lanemask_lt(lane));
    if (valid && rank == 0) wcnt[wave][e] = __popcll(m);
    __syncthreads();
    if (valid) {
      int pos = cur[e] + rank;
      for (int w = 0; w < wave; ++w) pos += wcnt[w][e];
      row_slot[pos] = j;
      row_token[pos] = j / k_out;
      row_w[pos] = route_w[j];
      slot_row[j] = pos;
    }
    __syncthreads();
    for (int x = tid; x < N; x += kPermThreads) {
      int add = 0;
#pragma unroll
      for (int w = 0; w < kPermThreads / kWave; ++w) {
        add += wcnt[w][x];
        wcnt[w][x] = 0;
      }
      cur[x] += add;
    }
    __syncthreads();
  }
  // Shared-expert rows follow the routed rows, one per token, weight 1.
  const int s_hi = min(t_shared, lo + kPermSlotsPerBlock);
  for (int i = lo + tid; i < s_hi; i += kPermThreads) {
    row_token[R + i] = i;
    row_slot[R + i] = -1;
    row_w[R + i] = 1.0f;
  }
}

hipError_t launch_permute(const int32_t *route_ids, const float *route_w, int T, int k_out, int N,
                          int t_shared, int bm0, int bm1, const PermBuffers &pb, hipStream_t s) {
  const int R = T * k_out;
  // Up to 4096 slots one workgroup is faster (Mixtral-shaped prefill, 4096
  // slots: 14.2 us against 15.1 us for the three kernels; 64 tokens of the tiny
  // layer: 4.6 us against about 13 us); beyond that its rounds cost more.
  if (R <= kPermOneBlockSlots && N <= kMaxExperts)
    return launch_permute_one_block(route_ids, route_w, T, k_out, N, t_shared, bm0, bm1, pb, s);
  const int nblk = (R + kPermSlotsPerBlock - 1) / kPermSlotsPerBlock;
  if (nblk > 0) perm_count_kernel<<<nblk, kPermThreads, 0, s>>>(route_ids, R, N, pb.blk_counts);
  perm_scan_kernel<<<1, kScanThreads, 0, s>>>(pb.blk_counts, nblk, N, R, t_shared, bm0, bm1,
                                              pb.offsets, pb.tile_start0, pb.tile_start1);
  if (nblk > 0)
    perm_scatter_kernel<<<nblk, kPermThreads, 0, s>>>(route_ids, route_w, R, k_out, N, t_shared,
                                                      pb.blk_counts, pb.row_token, pb.row_slot,
                                                      pb.row_w, pb.slot_row);
  return hipGetLastError();
}

}  // namespace exfold

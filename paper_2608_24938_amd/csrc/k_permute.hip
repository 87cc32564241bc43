// Stable permutation of the executed route slots by expert id.  Folded routes
// are grouped per retained expert before the expert computation (Sec. 4.1:
// routes folded onto one target are coalesced before expert computation, so
// each retained expert runs once over its rows).
//
// count:        per-block expert histograms (LDS integer atomics; order-free)
// scan+scatter: every block scans the counts itself (group offsets, its own
//               per-expert bases, GEMM m-tile lists), then ranks its slots
//               stably (wave match by ballots + cross-wave prefix)
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

constexpr int kPermThreads = 256;
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

// Scatter with its own scan: block b reads every block's counts (nblk * N
// ints, L2-resident), thread e forms expert e's total and its prefix over the
// blocks before b, and a workgroup scan over the experts gives the group
// offsets and m-tile lists (written by block 0).  One launch fewer than a
// separate scan kernel, whose one workgroup was a chain of dependent steps.
__global__ __launch_bounds__(kPermThreads) void perm_scan_scatter_kernel(
    const int32_t *__restrict__ ids, const float *__restrict__ route_w, int R, int k_out, int N,
    int t_shared, int bm0, int bm1, int nblk, const int32_t *__restrict__ blk_counts,
    int32_t *__restrict__ offsets, int32_t *__restrict__ tile_start0, int32_t *__restrict__ tile_start1,
    int32_t *__restrict__ row_token, int32_t *__restrict__ row_slot, float *__restrict__ row_w,
    int32_t *__restrict__ slot_row) {
  static_assert(kPermThreads >= kMaxExperts, "one thread per routed expert");
  constexpr int kW = kPermThreads / kWave;
  __shared__ int cur[kMaxExperts];
  __shared__ int wcnt[kW][kMaxExperts];
  __shared__ int part[3 * kW];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // expert tid: total over all blocks and prefix over the blocks before this one
  int total = 0, pre = 0;
  if (tid < N) {
    constexpr int kB = 8;
    int b = 0;
    for (; b + kB <= nblk; b += kB) {
      int c[kB];
#pragma unroll
      for (int q = 0; q < kB; ++q) c[q] = blk_counts[(size_t)(b + q) * N + tid];
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        pre += (b + q < (int)blockIdx.x) ? c[q] : 0;
        total += c[q];
      }
    }
    for (; b < nblk; ++b) {
      const int c = blk_counts[(size_t)b * N + tid];
      pre += (b < (int)blockIdx.x) ? c : 0;
      total += c;
    }
  }
  // routed groups: rows and m-tiles of either height; the shared group follows them
  int v[3] = {0, 0, 0};
  if (tid < N) {
    v[0] = total;
    v[1] = (total + bm0 - 1) / bm0;
    v[2] = (total + bm1 - 1) / bm1;
  }
  int ex[3], tot[3];
  block_scan3<kW>(v, ex, tot, part);
  if (tid < N) {
    cur[tid] = ex[0] + pre;
#pragma unroll
    for (int w = 0; w < kW; ++w) wcnt[w][tid] = 0;
  }
  if (blockIdx.x == 0) {
    const int s0 = t_shared > 0 ? (t_shared + bm0 - 1) / bm0 : 0;
    const int s1 = t_shared > 0 ? (t_shared + bm1 - 1) / bm1 : 0;
    if (tid < N) {
      offsets[tid] = ex[0];
      tile_start0[tid] = ex[1];
      tile_start1[tid] = ex[2];
    }
    if (tid == 0) {
      offsets[N] = R;
      offsets[N + 1] = R + t_shared;
      tile_start0[N] = tot[1];
      tile_start1[N] = tot[2];
      tile_start0[N + 1] = tot[1] + s0;
      tile_start1[N + 1] = tot[2] + s1;
    }
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
      for (int w = 0; w < kW; ++w) {
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
  // blocks cover the routed slots and the shared rows (t_shared <= T <= R)
  const int nblk = (R + kPermSlotsPerBlock - 1) / kPermSlotsPerBlock;
  perm_count_kernel<<<nblk, kPermThreads, 0, s>>>(route_ids, R, N, pb.blk_counts);
  perm_scan_scatter_kernel<<<nblk, kPermThreads, 0, s>>>(route_ids, route_w, R, k_out, N, t_shared, bm0, bm1,
                                                         nblk, pb.blk_counts, pb.offsets, pb.tile_start0,
                                                         pb.tile_start1, pb.row_token, pb.row_slot, pb.row_w,
                                                         pb.slot_row);
  return hipGetLastError();
}

}  // namespace exfold

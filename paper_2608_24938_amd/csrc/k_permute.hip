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

// Exclusive scan of buf[0..n) (n <= 2 * kPermThreads) in LDS; returns the total.
__device__ int block_exclusive_scan(int *buf, int n, int *tmp) {
  const int t = threadIdx.x;
  const int a = (2 * t < n) ? buf[2 * t] : 0;
  const int b = (2 * t + 1 < n) ? buf[2 * t + 1] : 0;
  tmp[t] = a + b;
  __syncthreads();
  for (int off = 1; off < kPermThreads; off <<= 1) {
    const int v = (t >= off) ? tmp[t - off] : 0;
    __syncthreads();
    tmp[t] += v;
    __syncthreads();
  }
  const int excl = tmp[t] - (a + b);
  const int total = tmp[kPermThreads - 1];
  __syncthreads();
  if (2 * t < n) buf[2 * t] = excl;
  if (2 * t + 1 < n) buf[2 * t + 1] = excl + a;
  __syncthreads();
  return total;
}

__global__ __launch_bounds__(kPermThreads) void perm_scan_kernel(
    int32_t *__restrict__ blk_counts, int nblk, int N, int R, int t_shared, int bm0, int bm1,
    int32_t *__restrict__ offsets, int32_t *__restrict__ tile_start0,
    int32_t *__restrict__ tile_start1) {
  __shared__ int tot[kMaxExperts + 2];
  __shared__ int t0[kMaxExperts + 2];
  __shared__ int t1[kMaxExperts + 2];
  __shared__ int tmp[kPermThreads];
  // The per-block counts are scanned in LDS when they fit (one coalesced read
  // and one write): a per-expert walk over the blocks in global memory is a
  // chain of nblk dependent load/store round trips (32 blocks: about 20 us).
  __shared__ int cl[kScanLdsInts];
  const bool in_lds = (long long)nblk * N <= kScanLdsInts;
  const int groups = N + (t_shared > 0 ? 1 : 0);
  if (in_lds) {
    for (int i = threadIdx.x; i < nblk * N; i += kPermThreads) cl[i] = blk_counts[i];
    __syncthreads();
  }
  for (int e = threadIdx.x; e < N; e += kPermThreads) {
    int running = 0;
    for (int b = 0; b < nblk; ++b) {
      int *slot = in_lds ? &cl[b * N + e] : &blk_counts[(size_t)b * N + e];
      const int c = *slot;
      *slot = running;
      running += c;
    }
    tot[e] = running;
  }
  if (threadIdx.x == 0) tot[N] = t_shared;
  __syncthreads();
  for (int g = threadIdx.x; g < groups; g += kPermThreads) {
    t0[g] = (tot[g] + bm0 - 1) / bm0;
    t1[g] = (tot[g] + bm1 - 1) / bm1;
  }
  __syncthreads();
  const int n_t0 = block_exclusive_scan(t0, groups, tmp);
  const int n_t1 = block_exclusive_scan(t1, groups, tmp);
  block_exclusive_scan(tot, N, tmp);
  for (int e = threadIdx.x; e < N; e += kPermThreads) offsets[e] = tot[e];
  if (in_lds) {
    for (int i = threadIdx.x; i < nblk * N; i += kPermThreads) blk_counts[i] = cl[i] + tot[i % N];
  } else {
    for (int e = threadIdx.x; e < N; e += kPermThreads)
      for (int b = 0; b < nblk; ++b) blk_counts[(size_t)b * N + e] += tot[e];
  }
  for (int g = threadIdx.x; g < groups; g += kPermThreads) {
    tile_start0[g] = t0[g];
    tile_start1[g] = t1[g];
  }
  if (threadIdx.x == 0) {
    offsets[N] = R;
    offsets[N + 1] = R + t_shared;
    for (int g = groups; g < N + 2; ++g) {
      tile_start0[g] = n_t0;
      tile_start1[g] = n_t1;
    }
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
  const int nblk = (R + kPermSlotsPerBlock - 1) / kPermSlotsPerBlock;
  if (nblk > 0) perm_count_kernel<<<nblk, kPermThreads, 0, s>>>(route_ids, R, N, pb.blk_counts);
  perm_scan_kernel<<<1, kPermThreads, 0, s>>>(pb.blk_counts, nblk, N, R, t_shared, bm0, bm1,
                                              pb.offsets, pb.tile_start0, pb.tile_start1);
  if (nblk > 0)
    perm_scatter_kernel<<<nblk, kPermThreads, 0, s>>>(route_ids, route_w, R, k_out, N, t_shared,
                                                      pb.blk_counts, pb.row_token, pb.row_slot,
                                                      pb.row_w, pb.slot_row);
  return hipGetLastError();
}

}  // namespace exfold

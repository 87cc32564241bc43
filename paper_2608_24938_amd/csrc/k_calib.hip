// Projector calibration: per-pair sufficient statistics and the closed-form
// scalar projector and loss (Sec. 4.2, Eq. calibration_outputs,
// Eq. scalar_projector, Eq. projection_loss; Appendix A protocol; Appendix B,
// Eq. A1-A2).  The expert outputs u = E_e(x) come from the expert GEMMs run
// with weight 1 on every evaluated (token, expert) pair.
//
// gram:     G_i[a][b] = <u_{i,a}, u_{i,b}> in float64 for the evaluated experts of token i
// finalize: per ordered pair (s, t), in token order, with w = ||u_s||:
//           A += w G[s][t], V += w G[t][t], C += w G[s][s], n += 1;
//           S = A / (V + lambda) (clipped), L = max(0, C - 2 S A + S^2 V) / (C + eps);
//           h_e = mean ||u_e|| over the tokens that evaluated e.
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

__global__ __launch_bounds__(256) void calib_routes_kernel(const int32_t *__restrict__ topk_ids, int m,
                                                           int N, int K, int mode,
                                                           int32_t *__restrict__ route_ids,
                                                           float *__restrict__ route_w,
                                                           int16_t *__restrict__ pos) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= m) return;
  int16_t *pr = pos + (long long)i * N;
  for (int e = 0; e < N; ++e) pr[e] = -1;
  if (mode == EXFOLD_CAL_COMMON) {
    for (int e = 0; e < N; ++e) {
      route_ids[(long long)i * N + e] = e;
      route_w[(long long)i * N + e] = 1.0f;
      pr[e] = (int16_t)e;
    }
  } else {
    for (int k = 0; k < K; ++k) {
      const int e = clamp_id(topk_ids[(long long)i * K + k], N);
      route_ids[(long long)i * K + k] = e;
      route_w[(long long)i * K + k] = 1.0f;
      pr[e] = (int16_t)k;
    }
  }
}

hipError_t launch_calib_routes(const int32_t *topk_ids, int m, int N, int K, int mode,
                               int32_t *route_ids, float *route_w, int16_t *pos, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  calib_routes_kernel<<<(m + 255) / 256, 256, 0, s>>>(topk_ids, m, N, K, mode, route_ids, route_w, pos);
  return hipGetLastError();
}

// One workgroup per token; each wave takes pairs (a <= b) round-robin.
__global__ __launch_bounds__(256) void calib_gram_kernel(const float *__restrict__ Y,
                                                         const int32_t *__restrict__ slot_row, int kr,
                                                         int d, double *__restrict__ gram) {
  const int i = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_pairs = kr * (kr + 1) / 2;
  double *Gi = gram + (long long)i * kr * kr;
  for (int pidx = wave; pidx < n_pairs; pidx += 4) {
    // pidx -> (a, b), a <= b, row-major over the upper triangle
    int a = 0, rem = pidx;
    while (rem >= kr - a) {
      rem -= kr - a;
      ++a;
    }
    const int b = a + rem;
    const float *ya = Y + (long long)slot_row[(long long)i * kr + a] * d;
    const float *yb = Y + (long long)slot_row[(long long)i * kr + b] * d;
    double acc = 0.0;
    for (int c = lane; c < d; c += 64) acc += (double)ya[c] * (double)yb[c];
#pragma unroll
    for (int msk = 32; msk >= 1; msk >>= 1) acc += __shfl_xor(acc, msk, kWave);
    if (lane == 0) {
      Gi[a * kr + b] = acc;
      Gi[b * kr + a] = acc;
    }
  }
}

hipError_t launch_calib_gram(const float *Y, const int32_t *slot_row, int m, int kr, int d,
                             double *gram, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  calib_gram_kernel<<<m, 256, 0, s>>>(Y, slot_row, kr, d, gram);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void calib_pairs_kernel(const double *__restrict__ gram,
                                                          const int16_t *__restrict__ pos, int m,
                                                          int N, int kr, double lambda, double clip,
                                                          float *__restrict__ S, float *__restrict__ L,
                                                          double *__restrict__ stats) {
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= N * N) return;
  const int s = idx / N, t = idx % N;
  double A = 0.0, V = 0.0, C = 0.0;
  long long n = 0;
  if (s != t) {
    for (int i = 0; i < m; ++i) {
      const int a = pos[(long long)i * N + s];
      const int b = pos[(long long)i * N + t];
      if (a >= 0 && b >= 0) {
        const double *Gi = gram + (long long)i * kr * kr;
        const double uu = Gi[a * kr + a];
        const double w = sqrt(uu);
        A += w * Gi[a * kr + b];
        V += w * Gi[b * kr + b];
        C += w * uu;
        ++n;
      }
    }
  }
  double sc, lo;
  if (s == t) {
    sc = 1.0;
    lo = 0.0;
  } else if (n == 0) {
    sc = 0.0;
    lo = 1e30;
  } else {
    const double den = V + lambda;
    sc = (den != 0.0) ? A / den : 0.0;
    if (clip > 0.0) sc = fmin(fmax(sc, -clip), clip);
    const double resid = C - 2.0 * sc * A + sc * sc * V;
    lo = fmax(0.0, resid) / (C + 1e-12);
  }
  S[idx] = (float)sc;
  L[idx] = (float)lo;
  if (stats) {
    stats[4LL * idx + 0] = A;
    stats[4LL * idx + 1] = V;
    stats[4LL * idx + 2] = C;
    stats[4LL * idx + 3] = (double)n;
  }
}

__global__ __launch_bounds__(256) void calib_norms_kernel(const double *__restrict__ gram,
                                                          const int16_t *__restrict__ pos, int m,
                                                          int N, int kr, float *__restrict__ h) {
  __shared__ double hv[kMaxExperts];
  __shared__ int seen[kMaxExperts];
  __shared__ double fill;
  const int e = threadIdx.x;
  if (e < N) {
    double sum = 0.0;
    int cnt = 0;
    for (int i = 0; i < m; ++i) {
      const int a = pos[(long long)i * N + e];
      if (a >= 0) {
        sum += sqrt(gram[(long long)i * kr * kr + a * kr + a]);
        ++cnt;
      }
    }
    hv[e] = cnt ? sum / cnt : 0.0;
    seen[e] = cnt > 0;
  }
  __syncthreads();
  if (e == 0) {
    double sum = 0.0;
    int cnt = 0;
    for (int x = 0; x < N; ++x)
      if (seen[x]) {
        sum += hv[x];
        ++cnt;
      }
    fill = cnt ? sum / cnt : 0.0;
  }
  __syncthreads();
  if (e < N) h[e] = (float)(seen[e] ? hv[e] : fill);
}

hipError_t launch_calib_finalize(const double *gram, const int16_t *pos, int m, int N, int kr,
                                 double lambda, double clip, float *S, float *L, float *h,
                                 double *pair_stats, hipStream_t s) {
  calib_pairs_kernel<<<(N * N + 255) / 256, 256, 0, s>>>(gram, pos, m, N, kr, lambda, clip, S, L,
                                                         pair_stats);
  calib_norms_kernel<<<1, 256, 0, s>>>(gram, pos, m, N, kr, h);
  return hipGetLastError();
}

}  // namespace exfold

// Diagonal projector family (Appendix B, Eq. appendix_diagonal_projector): the
// unfused reconstruction path of the projector ablation.
//
// stats:   per ordered pair (s, t), in token order over the calibration tokens
//          that evaluated both, with w = ||u_s||:  A_n += w v_n u_n,
//          V_n += w v_n^2 (float64, per hidden dimension n), C += w ||u_s||^2;
//          d_n = A_n / (V_n + lambda), loss = max(0, C - 2 sum d.A + sum d^2 V) / (C + eps).
// combine: y_i = sum over retained routes t of (w_t + sum of w_s d_{s->t}) . Y_t(x_i),
//          where Y_t holds the target expert's unweighted output rows.
#include "common.hpp"
#include "kernels.hpp"

namespace exfold {

constexpr int kDiagThreads = 256;
constexpr int kDiagCols = 4;           // hidden dimensions per thread and pass
constexpr int kDiagChunk = 1024;       // calibration tokens per LDS chunk of positions
constexpr double kDiagEps = 1e-12;
constexpr double kUnobservedLoss = 1e30;

// One workgroup per ordered pair (s, t).
__global__ __launch_bounds__(kDiagThreads) void diag_stats_kernel(
    const float *__restrict__ Y, const int32_t *__restrict__ slot_row, const double *__restrict__ gram,
    const int16_t *__restrict__ pos, int m, int N, int kr, int d, double lambda,
    float *__restrict__ Dg, float *__restrict__ Ld) {
  __shared__ int16_t ps[kDiagChunk], pt[kDiagChunk];
  __shared__ double red[2][kDiagThreads];
  const int p = blockIdx.x, tid = threadIdx.x;
  const int s = p / N, t = p % N;
  float *dout = Dg + (size_t)p * d;
  if (s == t) {
    for (int n = tid; n < d; n += kDiagThreads) dout[n] = 1.0f;
    if (tid == 0) Ld[p] = 0.0f;
    return;
  }
  double C = 0.0, sA = 0.0, sV = 0.0;
  int cnt = 0;
  for (int n0 = 0; n0 < d; n0 += kDiagThreads * kDiagCols) {
    double A[kDiagCols], V[kDiagCols];
#pragma unroll
    for (int r = 0; r < kDiagCols; ++r) A[r] = V[r] = 0.0;
    double Cp = 0.0;
    int cp = 0;
    for (int c0 = 0; c0 < m; c0 += kDiagChunk) {
      const int cn = min(kDiagChunk, m - c0);
      __syncthreads();
      for (int i = tid; i < cn; i += kDiagThreads) {
        ps[i] = pos[(size_t)(c0 + i) * N + s];
        pt[i] = pos[(size_t)(c0 + i) * N + t];
      }
      __syncthreads();
      for (int i = 0; i < cn; ++i) {
        const int a = ps[i], b = pt[i];
        if (a < 0 || b < 0) continue;  // uniform over the workgroup
        const size_t tok = (size_t)(c0 + i);
        const double uu = gram[(tok * kr + a) * kr + a];
        const double w = sqrt(uu);
        const float *yu = Y + (size_t)slot_row[tok * kr + a] * d;
        const float *yv = Y + (size_t)slot_row[tok * kr + b] * d;
#pragma unroll
        for (int r = 0; r < kDiagCols; ++r) {
          const int n = n0 + r * kDiagThreads + tid;
          if (n < d) {
            const double u = yu[n], v = yv[n];
            A[r] += w * (v * u);
            V[r] += w * (v * v);
          }
        }
        Cp += w * uu;
        ++cp;
      }
    }
    C = Cp;
    cnt = cp;
#pragma unroll
    for (int r = 0; r < kDiagCols; ++r) {
      const int n = n0 + r * kDiagThreads + tid;
      if (n < d) {
        double dv = 0.0;
        if (cnt > 0) {
          const double den = V[r] + lambda;
          dv = (den != 0.0) ? A[r] / den : 0.0;
        }
        sA += dv * A[r];
        sV += dv * dv * V[r];
        dout[n] = (float)dv;
      }
    }
  }
  // fixed-order tree reduction of the loss terms
  red[0][tid] = sA;
  red[1][tid] = sV;
  __syncthreads();
  for (int off = kDiagThreads / 2; off > 0; off >>= 1) {
    if (tid < off) {
      red[0][tid] += red[0][tid + off];
      red[1][tid] += red[1][tid + off];
    }
    __syncthreads();
  }
  if (tid == 0) {
    if (cnt == 0) {
      Ld[p] = (float)kUnobservedLoss;
    } else {
      const double resid = C - 2.0 * red[0][0] + red[1][0];
      Ld[p] = (float)((resid > 0.0 ? resid : 0.0) / (C + kDiagEps));
    }
  }
}

hipError_t launch_diag_stats(const float *Y, const int32_t *slot_row, const double *gram,
                             const int16_t *pos, int m, int N, int kr, int d, double lambda, float *Dg,
                             float *Ld, hipStream_t s) {
  diag_stats_kernel<<<N * N, kDiagThreads, 0, s>>>(Y, slot_row, gram, pos, m, N, kr, d, lambda, Dg, Ld);
  return hipGetLastError();
}

// Block (i, c): token i, columns [1024 c, 1024 c + 1024), four per thread.
template <typename OutT>
__global__ __launch_bounds__(256) void diag_combine_kernel(
    const float *__restrict__ Yr, const int32_t *__restrict__ slot_row, const int32_t *__restrict__ ids,
    const float *__restrict__ wret, const int32_t *__restrict__ om_src, const float *__restrict__ om_w,
    const int32_t *__restrict__ om_q, const float *__restrict__ Dg, int N, int K, int k_out, int d,
    int shared_base, OutT *__restrict__ y) {
  const int i = blockIdx.x;
  for (int c = blockIdx.y * 1024 + threadIdx.x * 4; c < min(d, (int)(blockIdx.y + 1) * 1024); c += 1024) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int q = 0; q < k_out; ++q) {
      const long long r = slot_row[(long long)i * k_out + q];
      const int te = clamp_id(ids[(long long)i * k_out + q], N);
      const float wt = wret[(long long)i * k_out + q];
      float coef[4] = {wt, wt, wt, wt};
      for (int j = 0; j < K; ++j) {
        if (om_q[(long long)i * K + j] != q) continue;
        const int se = clamp_id(om_src[(long long)i * K + j], N);
        const float ws = om_w[(long long)i * K + j];
        const float *dr = Dg + ((size_t)se * N + te) * d + c;
#pragma unroll
        for (int u = 0; u < 4; ++u) coef[u] = fmaf(ws, dr[u], coef[u]);
      }
      const float4 v = *reinterpret_cast<const float4 *>(Yr + r * d + c);
      acc[0] = fmaf(coef[0], v.x, acc[0]);
      acc[1] = fmaf(coef[1], v.y, acc[1]);
      acc[2] = fmaf(coef[2], v.z, acc[2]);
      acc[3] = fmaf(coef[3], v.w, acc[3]);
    }
    if (shared_base >= 0) {
      const float4 v = *reinterpret_cast<const float4 *>(Yr + (long long)(shared_base + i) * d + c);
      acc[0] += v.x; acc[1] += v.y; acc[2] += v.z; acc[3] += v.w;
    }
    OutT *o = y + (long long)i * d + c;
#pragma unroll
    for (int u = 0; u < 4; ++u) o[u] = store_cvt<OutT>(acc[u]);
  }
}

hipError_t launch_diag_combine(int dtype, const float *Yr, const int32_t *slot_row, const int32_t *ids,
                               const float *wret, const int32_t *om_src, const float *om_w,
                               const int32_t *om_q, const float *Dg, int T, int N, int K, int k_out,
                               int d, int shared_base, void *y, hipStream_t s) {
  if (T <= 0) return hipSuccess;
  const dim3 grid(T, (d + 1023) / 1024);
  if (dtype == EXFOLD_BF16)
    diag_combine_kernel<bf16_t><<<grid, 256, 0, s>>>(Yr, slot_row, ids, wret, om_src, om_w, om_q, Dg, N, K,
                                                     k_out, d, shared_base, static_cast<bf16_t *>(y));
  else
    diag_combine_kernel<float><<<grid, 256, 0, s>>>(Yr, slot_row, ids, wret, om_src, om_w, om_q, Dg, N, K,
                                                    k_out, d, shared_base, static_cast<float *>(y));
  return hipGetLastError();
}

}  // namespace exfold

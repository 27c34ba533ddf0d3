// Statistics of repeated gradient estimates: per-element running mean and
// sum of squared deviations (Welford's update), and their summary over all
// elements (mean standard deviation across repeats, mean absolute deviation
// of the mean from a reference gradient), reduced in a fixed order.
#include <math.h>

#include "../../include/bgpo.h"
#include "../../include/bgpo_stats.h"
#include "common.hpp"

namespace bgpo {

// k = number of estimates already folded in: delta = g - mean,
// mean += delta / (k + 1), m2 += delta (g - mean_new).
__global__ __launch_bounds__(256) void k_moments_update(const float* __restrict__ g,
                                                        float* __restrict__ mean,
                                                        float* __restrict__ m2, int64_t n,
                                                        int k) {
  const float inv = 1.f / (float)(k + 1);
  const int64_t stride = (int64_t)gridDim.x * 256 * 4;
  for (int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; i < n; i += stride) {
    if (i + 4 <= n) {
      const float4 gv = *reinterpret_cast<const float4*>(g + i);
      float4 mv = *reinterpret_cast<float4*>(mean + i);
      float4 sv = *reinterpret_cast<float4*>(m2 + i);
      float dl;
      dl = gv.x - mv.x; mv.x += dl * inv; sv.x += dl * (gv.x - mv.x);
      dl = gv.y - mv.y; mv.y += dl * inv; sv.y += dl * (gv.y - mv.y);
      dl = gv.z - mv.z; mv.z += dl * inv; sv.z += dl * (gv.z - mv.z);
      dl = gv.w - mv.w; mv.w += dl * inv; sv.w += dl * (gv.w - mv.w);
      *reinterpret_cast<float4*>(mean + i) = mv;
      *reinterpret_cast<float4*>(m2 + i) = sv;
    } else {
      for (int64_t q = i; q < n; ++q) {
        const float dl = g[q] - mean[q];
        mean[q] += dl * inv;
        m2[q] += dl * (g[q] - mean[q]);
      }
    }
  }
}

constexpr int kSumBlocks = 1024;

// Per-block partial sums of (std_i, |mean_i - ref_i|, |ref_i|) over a fixed
// element range, in float64; std_i = sqrt(m2_i / (count - 1)).
__global__ __launch_bounds__(256) void k_moments_partial(const float* __restrict__ mean,
                                                         const float* __restrict__ m2,
                                                         const float* __restrict__ ref, int64_t n,
                                                         int count, double* __restrict__ part) {
  __shared__ double red[3][4];
  const int64_t per = (n + kSumBlocks - 1) / kSumBlocks;
  const int64_t lo = (int64_t)blockIdx.x * per, hi = lo + per < n ? lo + per : n;
  const double dof = count > 1 ? 1.0 / (double)(count - 1) : 0.0;
  double s0 = 0.0, s1 = 0.0, s2 = 0.0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += 256) {
    s0 += sqrt((double)m2[i] * dof);
    if (ref) {
      s1 += fabs((double)mean[i] - (double)ref[i]);
      s2 += fabs((double)ref[i]);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    s0 += __shfl_xor(s0, off, 64);
    s1 += __shfl_xor(s1, off, 64);
    s2 += __shfl_xor(s2, off, 64);
  }
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][wv] = s0;
    red[1][wv] = s1;
    red[2][wv] = s2;
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    const int c = threadIdx.x;
    part[(int64_t)blockIdx.x * 3 + c] = red[c][0] + red[c][1] + red[c][2] + red[c][3];
  }
}

__global__ void k_moments_final(const double* __restrict__ part, int64_t n,
                                double* __restrict__ out) {
  if (threadIdx.x >= 3) return;
  double s = 0.0;
  for (int b = 0; b < kSumBlocks; ++b) s += part[b * 3 + threadIdx.x];
  out[threadIdx.x] = s / (double)n;
}

}  // namespace bgpo

using namespace bgpo;

extern "C" {

int bgpo_moments_update(const float* g, float* mean, float* m2, int64_t n, int32_t count,
                        void* stream) {
  if (!g || !mean || !m2 || n < 0 || count < 0) return BGPO_ERR_INVALID_ARG;
  if (((uintptr_t)g | (uintptr_t)mean | (uintptr_t)m2) & 15) return BGPO_ERR_INVALID_ARG;
  if (n == 0) return BGPO_OK;
  const int64_t blocks = (n / 4 + 255) / 256;
  k_moments_update<<<(unsigned)(blocks < 4096 ? (blocks > 0 ? blocks : 1) : 4096), 256, 0,
                     (hipStream_t)stream>>>(g, mean, m2, n, count);
  return hipGetLastError() == hipSuccess ? BGPO_OK : BGPO_ERR_HIP;
}

size_t bgpo_moments_workspace_size(void) { return (size_t)kSumBlocks * 3 * sizeof(double); }

int bgpo_moments_summary(const float* mean, const float* m2, const float* ref, int64_t n,
                         int32_t count, double* out, void* workspace, size_t ws_bytes,
                         void* stream) {
  if (!mean || !m2 || !out || n <= 0 || count < 1) return BGPO_ERR_INVALID_ARG;
  if (!workspace || ((uintptr_t)workspace & 7) || ws_bytes < bgpo_moments_workspace_size())
    return BGPO_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  double* part = static_cast<double*>(workspace);
  k_moments_partial<<<kSumBlocks, 256, 0, s>>>(mean, m2, ref, n, count, part);
  if (hipGetLastError() != hipSuccess) return BGPO_ERR_HIP;
  k_moments_final<<<1, 64, 0, s>>>(part, n, out);
  return hipGetLastError() == hipSuccess ? BGPO_OK : BGPO_ERR_HIP;
}

}  // extern "C"

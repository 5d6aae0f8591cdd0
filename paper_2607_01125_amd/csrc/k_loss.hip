// Losses of the two perturbed halves, L+ and L- (Algorithm 2 evaluates the loss
// under each perturbation).  Both reductions are deterministic: a fixed grid of
// kLossBlocks blocks per half writes fp64 partial sums in a fixed assignment, and
// one block adds them in a fixed tree order.  No atomics.
//
//  * MSE (single-layer workload): mean over T*N of (y[h] - target)^2.
//  * Next-token cross entropy (decoder models): one block per (half, position)
//    row computes log-sum-exp over the vocabulary with an online max / sum of
//    exponentials (wave64 shuffles, then the block), minus the target logit.
// Both are HBM-bound single passes over y or the logits.
#include "common.hpp"

namespace zoact {

namespace {

__device__ __forceinline__ double block_sum_d(double v, double* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  if (l == 0) sh[w] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0) {
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += sh[i];
  }
  __syncthreads();
  return t;  // valid in thread 0
}

template <bool BF16>
__global__ void __launch_bounds__(256) mse_partial(const void* __restrict__ y, const void* __restrict__ tgt, int64_t n,
                                                   double* __restrict__ part) {
  __shared__ double sh[4];
  const int h = blockIdx.y;
  float acc = 0.f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
  for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; i < n; i += stride) {
    float a[4], b[4];
    if (i + 4 <= n && (n & 3) == 0) {  // vector path keeps the second half 8/16-byte aligned
      if (BF16) {
        const ushort4 u = *reinterpret_cast<const ushort4*>(reinterpret_cast<const uint16_t*>(y) + (int64_t)h * n + i);
        const ushort4 t = *reinterpret_cast<const ushort4*>(reinterpret_cast<const uint16_t*>(tgt) + i);
        a[0] = bf2f(u.x); a[1] = bf2f(u.y); a[2] = bf2f(u.z); a[3] = bf2f(u.w);
        b[0] = bf2f(t.x); b[1] = bf2f(t.y); b[2] = bf2f(t.z); b[3] = bf2f(t.w);
      } else {
        const float4 u = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(y) + (int64_t)h * n + i);
        const float4 t = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(tgt) + i);
        a[0] = u.x; a[1] = u.y; a[2] = u.z; a[3] = u.w;
        b[0] = t.x; b[1] = t.y; b[2] = t.z; b[3] = t.w;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float d = a[j] - b[j];
        acc += d * d;
      }
    } else {
      for (int64_t j = i; j < n && j < i + 4; ++j) {
        const float av = BF16 ? bf2f(reinterpret_cast<const uint16_t*>(y)[(int64_t)h * n + j])
                              : reinterpret_cast<const float*>(y)[(int64_t)h * n + j];
        const float bv = BF16 ? bf2f(reinterpret_cast<const uint16_t*>(tgt)[j]) : reinterpret_cast<const float*>(tgt)[j];
        const float d = av - bv;
        acc += d * d;
      }
    }
  }
  const double s = block_sum_d((double)acc, sh);
  if (threadIdx.x == 0) part[h * kLossBlocks + blockIdx.x] = s;
}

// Sum n partials per half ([2][n]) in a fixed order and scale: the per-tile squared errors
// of the fused regression-loss epilogue.  One block per half; each thread adds its
// partials i = t, t + 256, ... in index order, with the loads issued eight at a time (index
// clamped, value replaced by zero past n) so that they overlap.
__global__ void __launch_bounds__(256) sum_mean(const double* __restrict__ part, int64_t n, double count,
                                                float* loss_pm) {
  __shared__ double sh[4];
  const int h = blockIdx.x;
  const double* ph = part + (int64_t)h * n;
  double v = 0.0;
  for (int64_t i0 = threadIdx.x; i0 < n; i0 += 8 * (int64_t)blockDim.x) {
    double t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t i = i0 + u * (int64_t)blockDim.x;
      t[u] = ph[i < n ? i : n - 1];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) v += (i0 + u * (int64_t)blockDim.x < n) ? t[u] : 0.0;
  }
  const double s = block_sum_d(v, sh);
  if (threadIdx.x == 0) loss_pm[h] = (float)(s / count);
}

// Cross entropy from the fused LM-head epilogue's per-block (max, sum of exp): one wave per
// row merges its nblk blocks (lanes strided, then a butterfly, in the online-softmax rule of
// xent_partial), and lane 0 adds max + log(sum) - next-token logit; kLossBlocks fixed
// partial sums per half as in xent_partial.
__global__ void __launch_bounds__(256) xent_combine(const float2* __restrict__ xpart, const float* __restrict__ xtgt,
                                                    int64_t T, int64_t S, int nblk, double* __restrict__ part) {
  __shared__ double sh[4];
  const int h = blockIdx.y;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  double acc = 0.0;
  for (int64_t m = (int64_t)blockIdx.x * 4 + w; m < T; m += (int64_t)gridDim.x * 4) {
    if (m % S == S - 1) continue;              // the last position has no next token
    const float2* pr = xpart + ((int64_t)h * T + m) * nblk;
    float mm = -INFINITY, se = 0.f;
    for (int i = l; i < nblk; i += 64) {
      const float2 q = pr[i];
      const float m2 = fmaxf(mm, q.x);
      se = (m2 == -INFINITY) ? 0.f : se * __expf(mm - m2) + q.y * __expf(q.x - m2);
      mm = m2;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float m2 = __shfl_xor(mm, o, 64), s2 = __shfl_xor(se, o, 64);
      const float mx = fmaxf(mm, m2);
      se = (mx == -INFINITY) ? 0.f : se * __expf(mm - mx) + s2 * __expf(m2 - mx);
      mm = mx;
    }
    if (l == 0) acc += (double)mm + log((double)se) - (double)xtgt[(int64_t)h * T + m];
  }
  const double s = block_sum_d(l == 0 ? acc : 0.0, sh);
  if (threadIdx.x == 0) part[h * kLossBlocks + blockIdx.x] = s;
}

// Sum kLossBlocks partials per half in a fixed order and scale (one block per half).
__global__ void __launch_bounds__(256) finish_mean(const double* __restrict__ part, double count, float* loss_pm) {
  __shared__ double sh[4];
  const int h = blockIdx.x;
  double v = 0.0;
  for (int i = threadIdx.x; i < kLossBlocks; i += blockDim.x) v += part[h * kLossBlocks + i];
  const double s = block_sum_d(v, sh);
  if (threadIdx.x == 0) loss_pm[h] = (float)(s / count);
}

__global__ void __launch_bounds__(256) xent_partial(const float* __restrict__ logits, const int32_t* __restrict__ tokens,
                                                    int64_t B, int64_t S, int64_t V, double* __restrict__ part) {
  __shared__ float smax[4], ssum[4];
  __shared__ double sh[4];
  const int h = blockIdx.y;
  const int64_t rows = B * (S - 1);
  double acc = 0.0;
  for (int64_t rrow = blockIdx.x; rrow < rows; rrow += gridDim.x) {
    const int64_t b = rrow / (S - 1), s = rrow % (S - 1);
    const float* lg = logits + (((int64_t)h * B + b) * S + s) * V;
    float m = -INFINITY, se = 0.f;
    for (int64_t v = threadIdx.x; v < V; v += blockDim.x) {
      const float x = lg[v];
      if (x > m) {
        se = se * __expf(m - x) + 1.0f;
        m = x;
      } else {
        se += __expf(x - m);
      }
    }
    // wave reduction of (m, se)
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float m2 = __shfl_xor(m, o, 64), s2 = __shfl_xor(se, o, 64);
      const float mm = fmaxf(m, m2);
      se = (mm == -INFINITY) ? 0.f : se * __expf(m - mm) + s2 * __expf(m2 - mm);
      m = mm;
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      smax[w] = m;
      ssum[w] = se;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      float mm = smax[0], ss = ssum[0];
      for (int i = 1; i < (int)(blockDim.x >> 6); ++i) {
        const float m2 = fmaxf(mm, smax[i]);
        ss = ss * __expf(mm - m2) + ssum[i] * __expf(smax[i] - m2);
        mm = m2;
      }
      int64_t tok = tokens[b * S + s + 1];
      tok = tok < 0 ? 0 : (tok >= V ? V - 1 : tok);
      acc += (double)mm + log((double)ss) - (double)lg[tok];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) part[h * kLossBlocks + blockIdx.x] = acc;
  (void)sh;
}

}  // namespace

hipError_t launch_xent_combine(const float2* xpart, const float* xtgt, int64_t T, int64_t S, int nblk, int64_t B,
                               double* part, float* loss_pm, hipStream_t s) {
  xent_combine<<<dim3(kLossBlocks, 2), dim3(256), 0, s>>>(xpart, xtgt, T, S, nblk, part);
  finish_mean<<<dim3(2), dim3(256), 0, s>>>(part, (double)(B * (S - 1)), loss_pm);
  return hipGetLastError();
}

hipError_t launch_sum_mean(const double* part, int64_t n, double count, float* loss_pm, hipStream_t s) {
  sum_mean<<<dim3(2), dim3(256), 0, s>>>(part, n, count, loss_pm);
  return hipGetLastError();
}

hipError_t launch_mse_pm(const void* y, int32_t dtype, const void* target, int64_t T, int64_t N, float* loss_pm,
                         void* ws, hipStream_t s) {
  double* part = static_cast<double*>(ws);
  const int64_t n = T * N;
  if (dtype == ZOACT_BF16) mse_partial<true><<<dim3(kLossBlocks, 2), dim3(256), 0, s>>>(y, target, n, part);
  else mse_partial<false><<<dim3(kLossBlocks, 2), dim3(256), 0, s>>>(y, target, n, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  finish_mean<<<2, 256, 0, s>>>(part, (double)n, loss_pm);
  return hipGetLastError();
}

hipError_t launch_xent_pm(const float* logits, const int32_t* tokens, int64_t B, int64_t S, int64_t V, float* loss_pm,
                          void* ws, hipStream_t s) {
  double* part = static_cast<double*>(ws);
  xent_partial<<<dim3(kLossBlocks, 2), dim3(256), 0, s>>>(logits, tokens, B, S, V, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  finish_mean<<<2, 256, 0, s>>>(part, (double)(B * (S - 1)), loss_pm);
  return hipGetLastError();
}

}  // namespace zoact

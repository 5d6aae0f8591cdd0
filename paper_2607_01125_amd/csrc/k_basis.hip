// One-shot activation basis (Algorithm 1): top-r right singular vectors of the
// calibration activations X, computed as the top-r eigenvectors of the uncentred
// Gram G = X^T X (their eigenvalues are the squared singular values).
//
//  * Gram: for bf16 X a v_mfma_f32_16x16x32_bf16 kernel over 128 x 128 output
//    tiles of the upper triangle (mirrored on store), contraction over tokens in
//    steps of 32; the X tile is transposed through LDS so that each lane's
//    fragment holds 8 consecutive tokens of one feature.  Every output tile is
//    owned by one workgroup and summed in token order (deterministic).  fp32 X
//    uses a plain SIMT kernel (small models).
//  * Eigenvectors: randomised block subspace iteration (Halko, Martinsson, Tropp
//    2011) with block b = r + p: Q = orth(G Omega), then `iters` times
//    Q = orth(G Q); orth is Cholesky-QR applied twice; Rayleigh-Ritz H = Q^T G Q;
//    the b x b eigenproblem is solved by a parallel cyclic Jacobi method in one
//    workgroup (round-robin pairing, all disjoint rotations of a round at once);
//    U = Q S[:, top r].  The d x b blocks and all small matrices are fp64; G is
//    read as fp32 (the only large operand).
//  * Sign: each column is flipped so its largest-magnitude entry is positive,
//    lowest index on ties.
#include "common.hpp"
#include "rng.hpp"

namespace zoact {

namespace {

constexpr int GT = 128;  // Gram output tile

// --------------------------------------------------------------- Gram, bf16 MFMA
__global__ void __launch_bounds__(256) gram_bf16_kernel(const uint16_t* __restrict__ x, int64_t n_tok, int64_t d,
                                                        float* __restrict__ g, int accumulate, int ntile) {
  // upper-triangular tile index -> (ti, tj), ti <= tj
  int t = blockIdx.x, ti = 0;
  while (t >= ntile - ti) {
    t -= ntile - ti;
    ++ti;
  }
  const int tj = ti + t;
  __shared__ __align__(16) uint16_t sa[GT][40];  // [feature][token], padded
  __shared__ __align__(16) uint16_t sb[GT][40];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int wi = (wave >> 1) * 64, wj = (wave & 1) * 64;
  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int64_t fi0 = (int64_t)ti * GT, fj0 = (int64_t)tj * GT;
  for (int64_t k0 = 0; k0 < n_tok; k0 += 32) {
    // 32 tokens x 128 features per operand: 512 chunks of 8 features, 2 per thread
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int idx = threadIdx.x + 256 * c;
      const int tok = idx >> 4, fc = idx & 15;
      const int64_t tk = k0 + tok;
      uint4 va = make_uint4(0, 0, 0, 0), vb = make_uint4(0, 0, 0, 0);
      if (tk < n_tok) {
        if (fi0 + fc * 8 < d) va = *reinterpret_cast<const uint4*>(x + tk * d + fi0 + fc * 8);
        if (fj0 + fc * 8 < d) vb = *reinterpret_cast<const uint4*>(x + tk * d + fj0 + fc * 8);
      }
      const uint16_t* pa = reinterpret_cast<const uint16_t*>(&va);
      const uint16_t* pb = reinterpret_cast<const uint16_t*>(&vb);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sa[fc * 8 + e][tok] = pa[e];
        sb[fc * 8 + e][tok] = pb[e];
      }
    }
    __syncthreads();
    bf16x8 af[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8*>(&sa[wi + i * 16 + lr][lk * 8]);
#pragma unroll
    for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(&sb[wj + j * 16 + lr][lk * 8]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t r = fi0 + wi + i * 16 + lk * 4 + q;
        const int64_t c = fj0 + wj + j * 16 + lr;
        if (r < d && c < d) {
          float v = acc[i][j][q];
          if (accumulate) v += g[r * d + c];
          g[r * d + c] = v;
          if (ti != tj) g[c * d + r] = v;
        }
      }
}

__global__ void gram_f32_kernel(const float* __restrict__ x, int64_t n_tok, int64_t d, float* __restrict__ g,
                                int accumulate) {
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < d * d; o += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = o / d, j = o % d;
    double s = 0.0;
    for (int64_t t = 0; t < n_tok; ++t) s += (double)x[t * d + i] * (double)x[t * d + j];
    g[o] = accumulate ? g[o] + (float)s : (float)s;
  }
}

// --------------------------------------------------------------- subspace iteration
struct EigWs {
  double* q;      // [d][b]
  double* y;      // [d][b]
  double* m;      // [b][b]
  double* s;      // [b][b] eigenvectors of H (columns)
  double* theta;  // [b]
  int* order;     // [b]
  double* u;      // [d][r]
};

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

EigWs carve(void* ws, int64_t d, int b, int r) {
  char* p = static_cast<char*>(ws);
  EigWs w;
  w.q = reinterpret_cast<double*>(p); p += align256((size_t)d * b * 8);
  w.y = reinterpret_cast<double*>(p); p += align256((size_t)d * b * 8);
  w.m = reinterpret_cast<double*>(p); p += align256((size_t)b * b * 8);
  w.s = reinterpret_cast<double*>(p); p += align256((size_t)b * b * 8);
  w.theta = reinterpret_cast<double*>(p); p += align256((size_t)b * 8);
  w.order = reinterpret_cast<int*>(p); p += align256((size_t)b * 4);
  w.u = reinterpret_cast<double*>(p);
  return w;
}

__global__ void omega_kernel(double* q, int64_t d, int b, uint64_t seed) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < d * b; i += (int64_t)gridDim.x * blockDim.x)
    q[i] = (double)rng::gauss_at(seed, 0xFFFFFFFFu, 0xB0515u, (uint64_t)i);
}

// Y[d][nc] = G[d][d] (fp32) * Q[d][ldq] (fp64, first nc columns); 64 x 64 tiles.
__global__ void __launch_bounds__(256) gq_kernel(const float* __restrict__ g, const double* __restrict__ q, double* __restrict__ y,
                                                 int64_t d, int ldq, int nc) {
  __shared__ double gs[64][17];
  __shared__ double qs[16][65];
  const int64_t r0 = (int64_t)blockIdx.x * 64;
  const int c0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[4][4] = {};
  for (int64_t k0 = 0; k0 < d; k0 += 16) {
    for (int i = threadIdx.x; i < 64 * 16; i += 256) {
      const int rr = i >> 4, kk = i & 15;
      const int64_t row = r0 + rr, k = k0 + kk;
      gs[rr][kk] = (row < d && k < d) ? (double)g[row * d + k] : 0.0;
      const int kq = i >> 6, cc = i & 63;
      const int64_t k2 = k0 + kq;
      qs[kq][cc] = (k2 < d && c0 + cc < nc) ? q[k2 * ldq + c0 + cc] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      double a[4], bb[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        a[p] = gs[ty * 4 + p][kk];
        bb[p] = qs[kk][tx * 4 + p];
      }
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[p][s] += a[p] * bb[s];
    }
    __syncthreads();
  }
  for (int p = 0; p < 4; ++p)
    for (int s = 0; s < 4; ++s) {
      const int64_t row = r0 + ty * 4 + p;
      const int c = c0 + tx * 4 + s;
      if (row < d && c < nc) y[row * nc + c] = acc[p][s];
    }
}

// M[b][b] = A^T B for A, B [d][b] (fp64); one 16 x 16 output tile per block, rows in order.
__global__ void __launch_bounds__(256) atb_kernel(const double* __restrict__ a, const double* __restrict__ bm, double* __restrict__ m,
                                                  int64_t d, int b) {
  __shared__ double as[64][17];
  __shared__ double bs[64][17];
  const int i0 = blockIdx.x * 16, j0 = blockIdx.y * 16;
  const int ti = threadIdx.x >> 4, tj = threadIdx.x & 15;
  double acc = 0.0;
  for (int64_t k0 = 0; k0 < d; k0 += 64) {
    for (int e = threadIdx.x; e < 64 * 16; e += 256) {
      const int kk = e >> 4, cc = e & 15;
      const int64_t k = k0 + kk;
      as[kk][cc] = (k < d && i0 + cc < b) ? a[k * b + i0 + cc] : 0.0;
      bs[kk][cc] = (k < d && j0 + cc < b) ? bm[k * b + j0 + cc] : 0.0;
    }
    __syncthreads();
    for (int kk = 0; kk < 64; ++kk) acc += as[kk][ti] * bs[kk][tj];
    __syncthreads();
  }
  if (i0 + ti < b && j0 + tj < b) m[(i0 + ti) * b + j0 + tj] = acc;
}

// In-place upper Cholesky factor of M (M = R^T R), one workgroup.
__global__ void __launch_bounds__(256) chol_kernel(double* m, int b) {
  for (int j = 0; j < b; ++j) {
    __shared__ double piv;
    if (threadIdx.x == 0) {
      double s = m[j * b + j];
      for (int k = 0; k < j; ++k) s -= m[k * b + j] * m[k * b + j];
      piv = s > 1e-300 ? sqrt(s) : 1e-150;
      m[j * b + j] = piv;
    }
    __syncthreads();
    for (int i = j + 1 + threadIdx.x; i < b; i += blockDim.x) {
      double s = m[j * b + i];
      for (int k = 0; k < j; ++k) s -= m[k * b + j] * m[k * b + i];
      m[j * b + i] = s / piv;
    }
    __syncthreads();
  }
}

// Q = Y R^{-1} row by row (R upper triangular in m).
__global__ void trsm_rows_kernel(const double* __restrict__ y, const double* __restrict__ rmat, double* __restrict__ q,
                                 int64_t d, int b) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < d; i += (int64_t)gridDim.x * blockDim.x) {
    for (int j = 0; j < b; ++j) {
      double s = y[i * b + j];
      for (int k = 0; k < j; ++k) s -= q[i * b + k] * rmat[k * b + j];
      q[i * b + j] = s / rmat[j * b + j];
    }
  }
}

// Parallel cyclic Jacobi on the symmetric b x b matrix h (in place), eigenvectors in s.
// Round-robin pairing: in each of the n-1 rounds of a sweep, index 0 is fixed and
// the others rotate, giving n/2 disjoint pairs (n = b rounded up to even).
__global__ void __launch_bounds__(256) jacobi_kernel(double* h, double* s, double* theta, int* order, int b, int sweeps) {
  __shared__ double cs[256], sn[256];
  __shared__ int pp[256], qq[256];
  __shared__ double off_sh[256], tot_sh[256];
  const int n = (b + 1) & ~1;
  for (int e = threadIdx.x; e < b * b; e += blockDim.x) s[e] = (e / b == e % b) ? 1.0 : 0.0;
  __syncthreads();
  for (int sw = 0; sw < sweeps; ++sw) {
    // convergence test: off-diagonal mass against the total
    double off = 0.0, tot = 0.0;
    for (int e = threadIdx.x; e < b * b; e += blockDim.x) {
      const double v = h[e] * h[e];
      tot += v;
      if (e / b != e % b) off += v;
    }
    off_sh[threadIdx.x] = off;
    tot_sh[threadIdx.x] = tot;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if ((int)threadIdx.x < o) {
        off_sh[threadIdx.x] += off_sh[threadIdx.x + o];
        tot_sh[threadIdx.x] += tot_sh[threadIdx.x + o];
      }
      __syncthreads();
    }
    const bool done = off_sh[0] <= 1e-30 * tot_sh[0];
    __syncthreads();
    if (done) break;
    for (int round = 0; round < n - 1; ++round) {
      // pairs of this round
      for (int k = threadIdx.x; k < n / 2; k += blockDim.x) {
        int a, c;
        if (k == 0) {
          a = 0;
          c = 1 + (round % (n - 1));
        } else {
          a = 1 + ((round + k) % (n - 1));
          c = 1 + ((round + n - 1 - k) % (n - 1));
        }
        if (a > c) { const int t = a; a = c; c = t; }
        pp[k] = a;
        qq[k] = c;
        double cc = 1.0, ss = 0.0;
        if (c < b) {
          const double apq = h[a * b + c];
          if (fabs(apq) > 1e-300) {
            const double tau = (h[c * b + c] - h[a * b + a]) / (2.0 * apq);
            const double t = (tau >= 0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
            cc = 1.0 / sqrt(1.0 + t * t);
            ss = t * cc;
          }
        }
        cs[k] = cc;
        sn[k] = ss;
      }
      __syncthreads();
      // columns: H <- H J, S <- S J
      for (int e = threadIdx.x; e < (n / 2) * b; e += blockDim.x) {
        const int k = e / b, i = e % b;
        const int a = pp[k], c = qq[k];
        if (c >= b || sn[k] == 0.0) continue;
        const double hp = h[i * b + a], hq = h[i * b + c];
        h[i * b + a] = cs[k] * hp - sn[k] * hq;
        h[i * b + c] = sn[k] * hp + cs[k] * hq;
        const double vp = s[i * b + a], vq = s[i * b + c];
        s[i * b + a] = cs[k] * vp - sn[k] * vq;
        s[i * b + c] = sn[k] * vp + cs[k] * vq;
      }
      __syncthreads();
      // rows: H <- J^T H
      for (int e = threadIdx.x; e < (n / 2) * b; e += blockDim.x) {
        const int k = e / b, j = e % b;
        const int a = pp[k], c = qq[k];
        if (c >= b || sn[k] == 0.0) continue;
        const double hp = h[a * b + j], hq = h[c * b + j];
        h[a * b + j] = cs[k] * hp - sn[k] * hq;
        h[c * b + j] = sn[k] * hp + cs[k] * hq;
      }
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) {
    // descending order of the diagonal (selection; b <= 512)
    for (int i = 0; i < b; ++i) order[i] = i;
    for (int i = 0; i < b; ++i) {
      int best = i;
      for (int j = i + 1; j < b; ++j)
        if (h[order[j] * b + order[j]] > h[order[best] * b + order[best]]) best = j;
      const int t = order[i];
      order[i] = order[best];
      order[best] = t;
      theta[i] = h[order[i] * b + order[i]];
    }
  }
}

// u[d][r] = Q[d][b] S[:, order[:r]]
__global__ void ritz_vectors_kernel(const double* __restrict__ q, const double* __restrict__ s, const int* __restrict__ order,
                                    double* __restrict__ u, int64_t d, int b, int r) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < d * r; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / r;
    const int c = (int)(e % r);
    const int col = order[c];
    double acc = 0.0;
    for (int k = 0; k < b; ++k) acc += q[i * b + k] * s[k * b + col];
    u[e] = acc;
  }
}

// Per column: sign so that the largest-|.| entry (lowest index on ties) is positive;
// write U^T in the requested dtype, the fp32 master and the eigenvalues.
__global__ void __launch_bounds__(256) finish_basis_kernel(const double* __restrict__ u, const double* __restrict__ theta, int64_t d,
                                                           int r, void* ut, int ut_bf16, float* ut_master, float* eigvals) {
  __shared__ double bv[256];
  __shared__ int bi[256];
  const int c = blockIdx.x;
  double best = -1.0;
  int besti = 0x7fffffff;
  for (int64_t i = threadIdx.x; i < d; i += blockDim.x) {
    const double a = fabs(u[i * r + c]);
    if (a > best) {  // strided scan visits increasing i: first maximum kept
      best = a;
      besti = (int)i;
    }
  }
  bv[threadIdx.x] = best;
  bi[threadIdx.x] = besti;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      const double v2 = bv[threadIdx.x + o];
      const int i2 = bi[threadIdx.x + o];
      if (v2 > bv[threadIdx.x] || (v2 == bv[threadIdx.x] && i2 < bi[threadIdx.x])) {
        bv[threadIdx.x] = v2;
        bi[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  const double sgn = u[(int64_t)bi[0] * r + c] < 0 ? -1.0 : 1.0;
  for (int64_t i = threadIdx.x; i < d; i += blockDim.x) {
    const float v = (float)(sgn * u[i * r + c]);
    if (ut_bf16) reinterpret_cast<uint16_t*>(ut)[(int64_t)c * d + i] = f2bf(v);
    else reinterpret_cast<float*>(ut)[(int64_t)c * d + i] = v;
    if (ut_master) ut_master[(int64_t)c * d + i] = v;
  }
  if (threadIdx.x == 0 && eigvals) eigvals[c] = (float)theta[c];
}

// resid = max_c ||G u_c - theta_c u_c|| / theta_0, with y = G u already formed.
__global__ void __launch_bounds__(256) resid_kernel(const double* __restrict__ y, const double* __restrict__ u,
                                                    const double* __restrict__ theta, int64_t d, int r, float* resid) {
  __shared__ double sh[256];
  double worst = 0.0;
  for (int c = 0; c < r; ++c) {
    double s = 0.0;
    for (int64_t i = threadIdx.x; i < d; i += blockDim.x) {
      const double e = y[i * r + c] - theta[c] * u[i * r + c];
      s += e * e;
    }
    sh[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
      __syncthreads();
    }
    if (threadIdx.x == 0) worst = fmax(worst, sqrt(sh[0]));
    __syncthreads();
  }
  if (threadIdx.x == 0) *resid = (float)(worst / fmax(fabs(theta[0]), 1e-300));
}

hipError_t orth(EigWs& w, int64_t d, int b, hipStream_t s) {
  // Cholesky-QR twice: y holds the block to orthonormalise, result in q.
  for (int pass = 0; pass < 2; ++pass) {
    const double* src = pass == 0 ? w.y : w.q;
    atb_kernel<<<dim3((b + 15) / 16, (b + 15) / 16), 256, 0, s>>>(src, src, w.m, d, b);
    chol_kernel<<<1, 256, 0, s>>>(w.m, b);
    if (pass == 1) {
      // second pass works in place: copy q to y first (trsm reads y, writes q)
      hipError_t e = hipMemcpyAsync(w.y, w.q, (size_t)d * b * 8, hipMemcpyDeviceToDevice, s);
      if (e != hipSuccess) return e;
    }
    int64_t gb = (d + 255) / 256;
    trsm_rows_kernel<<<dim3((unsigned)gb), 256, 0, s>>>(w.y, w.m, w.q, d, b);
  }
  return hipGetLastError();
}

}  // namespace

size_t basis_ws_bytes(int64_t d, int32_t r, int32_t p) {
  const int b = r + p;
  return align256((size_t)d * b * 8) * 2 + align256((size_t)b * b * 8) * 2 + align256((size_t)b * 8) +
         align256((size_t)b * 4) + align256((size_t)d * b * 8);
}

hipError_t launch_gram(const void* x, int32_t dtype, int64_t n_tok, int64_t d, float* g, int accumulate, hipStream_t s) {
  if (dtype == ZOACT_BF16) {
    const int nt = (int)((d + GT - 1) / GT);
    gram_bf16_kernel<<<dim3((unsigned)(nt * (nt + 1) / 2)), 256, 0, s>>>(static_cast<const uint16_t*>(x), n_tok, d, g,
                                                                          accumulate, nt);
  } else {
    int64_t gb = (d * d + 255) / 256;
    if (gb > 65535) gb = 65535;
    gram_f32_kernel<<<dim3((unsigned)gb), 256, 0, s>>>(static_cast<const float*>(x), n_tok, d, g, accumulate);
  }
  return hipGetLastError();
}

hipError_t launch_basis_from_gram(const float* g, int64_t d, int32_t r, int32_t p, int32_t iters, uint64_t seed,
                                  void* ut, int32_t ut_dtype, float* ut_master, float* eigvals, float* resid, void* ws,
                                  hipStream_t s) {
  const int b = r + p;
  EigWs w = carve(ws, d, b, r);
  const dim3 gq_grid((unsigned)((d + 63) / 64), (unsigned)((b + 63) / 64));
  omega_kernel<<<dim3((unsigned)((d * b + 255) / 256 > 65535 ? 65535 : (d * b + 255) / 256)), 256, 0, s>>>(w.q, d, b, seed);
  for (int it = 0; it <= iters; ++it) {
    gq_kernel<<<gq_grid, 256, 0, s>>>(g, w.q, w.y, d, b, b);
    hipError_t e = orth(w, d, b, s);
    if (e != hipSuccess) return e;
  }
  // Rayleigh-Ritz: H = Q^T G Q
  gq_kernel<<<gq_grid, 256, 0, s>>>(g, w.q, w.y, d, b, b);
  atb_kernel<<<dim3((b + 15) / 16, (b + 15) / 16), 256, 0, s>>>(w.q, w.y, w.m, d, b);
  jacobi_kernel<<<1, 256, 0, s>>>(w.m, w.s, w.theta, w.order, b, 40);
  int64_t gb = (d * r + 255) / 256;
  if (gb > 65535) gb = 65535;
  ritz_vectors_kernel<<<dim3((unsigned)gb), 256, 0, s>>>(w.q, w.s, w.order, w.u, d, b, r);
  finish_basis_kernel<<<dim3((unsigned)r), 256, 0, s>>>(w.u, w.theta, d, r, ut, ut_dtype == ZOACT_BF16 ? 1 : 0,
                                                        ut_master, eigvals);
  if (resid) {
    // y = G u (u has r columns)
    gq_kernel<<<dim3((unsigned)((d + 63) / 64), (unsigned)((r + 63) / 64)), 256, 0, s>>>(g, w.u, w.y, d, r, r);
    resid_kernel<<<1, 256, 0, s>>>(w.y, w.u, w.theta, d, r, resid);
  }
  return hipGetLastError();
}

}  // namespace zoact

// One-shot activation basis (Algorithm 1): top-r right singular vectors of the
// calibration activations X, computed as the top-r eigenvectors of the uncentred
// Gram G = X^T X (their eigenvalues are the squared singular values).
//
//  * Gram: for bf16 X a v_mfma_f32_16x16x32_bf16 kernel over 128 x 128 output
//    tiles of the upper triangle (mirrored on store), contraction over tokens in
//    steps of 64; 8 x 8 blocks of X are transposed in registers so that each lane's
//    fragment holds 8 consecutive tokens of one feature.  Every output tile is owned
//    by one workgroup and summed in token order (deterministic).  fp32 X uses a plain
//    SIMT kernel (small models).
//  * Eigenvectors: randomised block subspace iteration (Halko, Martinsson, Tropp
//    2011) with block b = r + p: Q = orth(G Omega), then up to max_iter times
//    Q = orth(G Q); orth is Cholesky-QR (twice on the last block); Rayleigh-Ritz
//    H = Q^T G Q; the b x b eigenproblem is solved in one workgroup by a one-sided
//    Jacobi method (b <= 128) or a two-sided one (larger b), all disjoint rotations of
//    a round at once; U = Q S[:, top r].  The iteration's products G Q run on fp32
//    MFMA; the orthonormalisation, the Rayleigh-Ritz product and all small matrices
//    are fp64.  An adaptive mode stops once an estimate of the top-r residuals, formed
//    from the iteration's own products, meets the caller's bound.
//  * Sign: each column is flipped so its largest-magnitude entry is positive,
//    lowest index on ties.
//  * Fewer calibration rows n than features D (the wide inputs of the down
//    projections): the thin SVD X = U_x S V^T read from its left side.  The same
//    solver runs on the n x n token Gram X X^T, whose eigenvectors are U_x and whose
//    eigenvalues are those of X^T X; the basis is V_r = X^T U_x,r S_r^{-1}, formed as
//    X^T v with each column scaled to unit length in fp64.  Forming X X^T costs
//    n^2 D instead of D^2 n, and each iteration reads n^2 instead of D^2 values.
#include "common.hpp"
#include "rng.hpp"

#include <algorithm>
#include <climits>
#include <cmath>
#include <utility>

namespace zoact {

namespace {

constexpr int GT = 128;  // Gram output tile

// --------------------------------------------------------------- Gram, bf16 MFMA
// One workgroup per 128 x 128 tile of the upper triangle; four waves of 64 x 64
// (4 x 4 v_mfma_f32_16x16x32_bf16 tiles).  Tokens advance 64 at a time.  The MFMA wants
// each lane's 8 contraction values (tokens) consecutive, X has features consecutive, so
// each thread loads an 8 token x 8 feature block (eight 16-byte row loads, coalesced
// across the 16 lanes that cover 128 features), transposes it in registers with byte
// permutes and writes eight 16-byte feature rows into the LDS tile [feature][token].  The
// LDS tiles are double-buffered and the next block's loads are issued before the current
// block's MFMAs, one barrier per 64 tokens.  A diagonal tile loads its operand once.
constexpr int GK = 64;        // tokens per step
constexpr int GLD = GK + 8;   // LDS row pitch (elements): 144 bytes

// 8 x 8 transpose of 16-bit values: in[e] holds row e (8 values), out[j] column j.
__device__ __forceinline__ void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;   // high or low halves
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t* a = reinterpret_cast<const uint32_t*>(&in[2 * q]);
      const uint32_t* b = reinterpret_cast<const uint32_t*>(&in[2 * q + 1]);
      w[q] = __builtin_amdgcn_perm(b[j >> 1], a[j >> 1], sel);
    }
    out[j] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

__global__ void __launch_bounds__(256) gram_bf16_kernel(const uint16_t* __restrict__ x, int64_t n_tok, int64_t d,
                                                        int64_t ld, float* __restrict__ g, int accumulate, int ntile) {
  // upper-triangular tile index -> (ti, tj), ti <= tj
  int t = blockIdx.x, ti = 0;
  while (t >= ntile - ti) {
    t -= ntile - ti;
    ++ti;
  }
  const int tj = ti + t;
  const bool diag = ti == tj;
  __shared__ __align__(16) uint16_t sm[2][2][GT * GLD];   // [buffer][operand][feature][token]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int wi = (wave >> 1) * 64, wj = (wave & 1) * 64;
  const int64_t fi0 = (int64_t)ti * GT, fj0 = (int64_t)tj * GT;
  // this thread's load block: operand, token group (8 tokens), feature group (8 features)
  const int opnd = threadIdx.x >> 7, tg = (threadIdx.x >> 4) & 7, fg = threadIdx.x & 15;
  const bool loader = !(diag && opnd == 1);
  const int64_t feat = (opnd ? fj0 : fi0) + fg * 8;
  const bool fvalid = feat < d;
  uint4 rows[8];
  auto load = [&](int64_t k0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t tk = k0 + tg * 8 + e;
      rows[e] = (loader && fvalid && tk < n_tok) ? *reinterpret_cast<const uint4*>(x + tk * ld + feat)
                                                 : make_uint4(0u, 0u, 0u, 0u);
    }
  };
  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const int nsteps = (int)((n_tok + GK - 1) / GK);
  load(0);
  for (int step = 0; step < nsteps; ++step) {
    const int buf = step & 1;
    if (loader) {
      uint4 cols[8];
      transpose8x8(rows, cols);
      uint16_t* dst = &sm[buf][opnd][(fg * 8) * GLD + tg * 8];
#pragma unroll
      for (int j = 0; j < 8; ++j) *reinterpret_cast<uint4*>(dst + j * GLD) = cols[j];
    }
    __syncthreads();
    if (step + 1 < nsteps) load((int64_t)(step + 1) * GK);
    const uint16_t* sa = sm[buf][0];
    const uint16_t* sb = sm[buf][diag ? 0 : 1];
#pragma unroll
    for (int kh = 0; kh < GK / 32; ++kh) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(sa + (wi + i * 16 + lr) * GLD + kh * 32 + lk * 8);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(sb + (wj + j * 16 + lr) * GLD + kh * 32 + lk * 8);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
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
          if (!diag) g[c * d + r] = v;
        }
      }
}

// --------------------------------------------------------------- token-side Gram
// G' = X X^T [n][n] for bf16 X [n][ld] (d values per row, d % 64 == 0).  The contraction
// runs along X's rows, so each lane's MFMA operand (8 depth values of one row) comes
// straight from global memory with no transpose and no LDS.  One workgroup per 128 x 128
// tile of the upper triangle, four waves of 64 x 64 (4 x 4 blocks of
// v_mfma_f32_16x16x32_bf16); depth in 64-deep steps, the next step's operands loaded
// while the current step's MFMAs run.  A sum over the depth does not depend on which
// lane holds which depth value as long as both operands agree, so lane group lk takes
// the 16 consecutive values 16 lk .. 16 lk + 15 of each step (two 16-byte loads: the
// first half feeds the first MFMA, the second half the second) and a row's 64 values of
// a step are one 128-byte line.  Entries with row <= column are stored and mirrored, so
// G' is exactly symmetric; rows past n read zeros and store nothing.
__global__ void __launch_bounds__(256) gram_rows_bf16_kernel(const uint16_t* __restrict__ x, int64_t n, int64_t d,
                                                             int64_t ld, float* __restrict__ g, int ntile) {
  int t = blockIdx.x, ti = 0;
  while (t >= ntile - ti) {
    t -= ntile - ti;
    ++ti;
  }
  const int tj = ti + t;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t i0 = (int64_t)ti * GT + (wave >> 1) * 64, j0 = (int64_t)tj * GT + (wave & 1) * 64;
  const uint16_t* pa[4];
  const uint16_t* pb[4];
  bool va[4], vb[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t ra = i0 + q * 16 + lr, rb = j0 + q * 16 + lr;
    va[q] = ra < n;
    vb[q] = rb < n;
    pa[q] = x + (va[q] ? ra : 0) * ld + lk * 16;   // a row past n reads row 0, then zeros
    pb[q] = x + (vb[q] ? rb : 0) * ld + lk * 16;
  }
  const bf16x8 zero = {};
  auto load = [&](bf16x8 (&a)[4][2], bf16x8 (&b)[4][2], int64_t k) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16x8 av = *reinterpret_cast<const bf16x8*>(pa[q] + k + h * 8);
        const bf16x8 bv = *reinterpret_cast<const bf16x8*>(pb[q] + k + h * 8);
        a[q][h] = va[q] ? av : zero;
        b[q][h] = vb[q] ? bv : zero;
      }
  };
  floatx4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](const bf16x8 (&a)[4][2], const bf16x8 (&b)[4][2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i][h], b[j][h], acc[i][j], 0, 0, 0);
  };
  bf16x8 a0[4][2], b0[4][2], a1[4][2], b1[4][2];
  load(a0, b0, 0);
  int64_t k = 0;
  for (; k + 128 <= d; k += 128) {
    load(a1, b1, k + 64);
    mma(a0, b0);
    if (k + 128 < d) load(a0, b0, k + 128);
    mma(a1, b1);
  }
  if (k < d) mma(a0, b0);   // d % 128 == 64: the last step, loaded by the loop's last pass
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t r = i0 + i * 16 + lk * 4 + q;
        const int64_t c = j0 + j * 16 + lr;
        if (r <= c && c < n) {
          g[r * n + c] = acc[i][j][q];
          if (r < c) g[c * n + r] = acc[i][j][q];
        }
      }
}

// Lower triangle of g [n][n] replaced by the upper one (g[i][j] = g[j][i] for i > j),
// through 32 x 32 LDS tiles so both sides are read and written along rows.
__global__ void __launch_bounds__(256) mirror_upper_kernel(float* __restrict__ g, int64_t n, int nt) {
  __shared__ float tl[32][33];
  int t = blockIdx.x, bi = 0;   // tile (bi, bj), bi < bj: rows bi, columns bj are the source
  while (t >= nt - 1 - bi) {
    t -= nt - 1 - bi;
    ++bi;
  }
  const int bj = bi + 1 + t;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8) {
    const int64_t i = (int64_t)bi * 32 + k, j = (int64_t)bj * 32 + tx;
    tl[k][tx] = (i < n && j < n) ? g[i * n + j] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int64_t i = (int64_t)bj * 32 + k, j = (int64_t)bi * 32 + tx;   // lower-triangle entry (i, j)
    if (i < n && j < n) g[i * n + j] = tl[tx][k];
  }
}

// Diagonal 32 x 32 blocks: entries below the diagonal take their mirror.
__global__ void __launch_bounds__(256) mirror_diag_kernel(float* __restrict__ g, int64_t n) {
  __shared__ float tl[32][33];
  const int64_t b0 = (int64_t)blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8)
    tl[k][tx] = (b0 + k < n && b0 + tx < n) ? g[(b0 + k) * n + b0 + tx] : 0.f;
  __syncthreads();
  for (int k = ty; k < 32; k += 8)
    if (k > tx && b0 + k < n) g[(b0 + k) * n + b0 + tx] = tl[tx][k];
}

// part[z][D][r] (fp64) = X[rows of chunk z]^T V[rows of chunk z] for bf16 X [n][ld] (D
// values per row, D % 8 == 0) and V fp64 [n][r]; grid (D / 512 feature blocks, r / 32
// column blocks, depth chunks of `tchunk` rows).  32 rows of X (512 features) and of V
// (32 columns) are staged in LDS per step; each thread owns 8 features x 8 columns in
// fp64 registers and walks the rows in order.
constexpr int XV_J = 512, XV_C = 32, XV_T = 32;
__global__ void __launch_bounds__(256) xt_v_kernel(const uint16_t* __restrict__ x, int64_t n, int64_t D, int64_t ld,
                                                   const double* __restrict__ v, int r, int64_t tchunk,
                                                   double* __restrict__ part) {
  __shared__ __align__(16) uint16_t xs[XV_T][XV_J + 8];
  __shared__ __align__(16) double vs[XV_T][XV_C];
  const int tc = threadIdx.x & 3, tj = threadIdx.x >> 2;
  const int64_t j0 = (int64_t)blockIdx.x * XV_J;
  const int c0 = blockIdx.y * XV_C;
  const int64_t tb = (int64_t)blockIdx.z * tchunk;
  const int64_t te = tb + tchunk < n ? tb + tchunk : n;
  double acc[8][8];
#pragma unroll
  for (int a = 0; a < 8; ++a)
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[a][b] = 0.0;
  for (int64_t t0 = tb; t0 < te; t0 += XV_T) {
    __syncthreads();
    for (int e = threadIdx.x; e < XV_T * XV_J / 8; e += 256) {
      const int tt = e >> 6, jc = (e & 63) * 8;
      const int64_t t = t0 + tt, j = j0 + jc;
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (t < te && j < D) val = *reinterpret_cast<const uint4*>(x + t * ld + j);
      *reinterpret_cast<uint4*>(&xs[tt][jc]) = val;
    }
    for (int e = threadIdx.x; e < XV_T * XV_C; e += 256) {
      const int tt = e >> 5, c = e & 31;
      vs[tt][c] = (t0 + tt < te && c0 + c < r) ? v[(t0 + tt) * r + c0 + c] : 0.0;
    }
    __syncthreads();
    for (int tt = 0; tt < XV_T; ++tt) {
      const uint4 xq = *reinterpret_cast<const uint4*>(&xs[tt][tj * 8]);
      const uint32_t xw[4] = {xq.x, xq.y, xq.z, xq.w};
      double xv[8], vv[8];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        xv[2 * a] = (double)__uint_as_float(xw[a] << 16);
        xv[2 * a + 1] = (double)__uint_as_float(xw[a] & 0xFFFF0000u);
      }
#pragma unroll
      for (int b = 0; b < 8; ++b) vv[b] = vs[tt][tc * 8 + b];
#pragma unroll
      for (int a = 0; a < 8; ++a)
#pragma unroll
        for (int b = 0; b < 8; ++b) acc[a][b] = fma(xv[a], vv[b], acc[a][b]);
    }
  }
  double* out = part + (int64_t)blockIdx.z * D * r;
#pragma unroll
  for (int a = 0; a < 8; ++a) {
    const int64_t j = j0 + tj * 8 + a;
    if (j >= D) continue;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const int c = c0 + tc * 8 + b;
      if (c < r) out[j * r + c] = acc[a][b];
    }
  }
}

// out[e] = sum over z = 0 .. ks-1 of part[z][e], in that order.
__global__ void __launch_bounds__(256) sum_chunks_kernel(const double* __restrict__ part, int ks, int64_t m,
                                                         double* __restrict__ out) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < m; e += (int64_t)gridDim.x * 256) {
    double acc = part[e];
    for (int z = 1; z < ks; ++z) acc += part[(int64_t)z * m + e];
    out[e] = acc;
  }
}

// Columns of a [D][r] scaled to unit length: s[c] = ||a[:, c]|| (fixed-order reduction)
// and a[:, c] /= s[c]; with compute == 0 the s given is applied instead.  A zero column
// stays zero.
__global__ void __launch_bounds__(256) colscale_kernel(double* __restrict__ a, int64_t D, int r, double* __restrict__ s,
                                                       int compute) {
  __shared__ double sh[256];
  const int c = blockIdx.x;
  double nrm;
  if (compute) {
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < D; j += 256) acc += a[j * r + c] * a[j * r + c];
    sh[threadIdx.x] = acc;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if ((int)threadIdx.x < o) sh[threadIdx.x] += sh[threadIdx.x + o];
      __syncthreads();
    }
    nrm = sqrt(sh[0]);
    if (threadIdx.x == 0) s[c] = nrm;
  } else {
    nrm = s[c];
  }
  const double inv = nrm > 0.0 ? 1.0 / nrm : 0.0;
  for (int64_t j = threadIdx.x; j < D; j += 256) a[j * r + c] *= inv;
}

__global__ void gram_f32_kernel(const float* __restrict__ x, int64_t n_tok, int64_t d, int64_t ld,
                                float* __restrict__ g, int accumulate) {
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < d * d; o += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = o / d, j = o % d;
    double s = 0.0;
    for (int64_t t = 0; t < n_tok; ++t) s += (double)x[t * ld + i] * (double)x[t * ld + j];
    g[o] = accumulate ? g[o] + (float)s : (float)s;
  }
}

// --------------------------------------------------------------- subspace iteration
// Per iteration: Y = G Q on fp32 MFMA (fp32 copy of Q, K split across workgroups into
// fp32 partial products summed in a fixed order into fp64), then Q = orth(Y) by
// Cholesky-QR applied twice in fp64 (column Gram M = Y^T Y from fixed-order partial
// sums, M = L L^T in LDS, L^{-1} in place, Q = Y L^{-T}).  The fp32 products only
// steer the subspace; the Rayleigh-Ritz step that yields the eigenvectors forms G Q
// with fp64 accumulation, so the result carries the accuracy of the fp32 Gram.
constexpr int GQ_ROWS = 128;   // rows of G per workgroup of the products
constexpr int GQ_K = 32;       // contraction chunk staged in LDS
constexpr int NPART = 64;      // workgroups (partial sums) of the column-Gram pass

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// K split of the products for b columns: chunks a multiple of GQ_K and at least 256
// deep; the grid (row blocks x ks x column blocks of 64) a whole number of workgroups per
// CU where a split gives one (several workgroups of the products fit on a CU at once, and
// with a fractional count the CUs that get one more set the time), at least two per CU,
// else the most even split; at equal balance the fewest chunks (the partials are summed
// in a second pass).
void ksplit_for(int64_t d, int b, int& ks, int64_t& kchunk) {
  const int64_t nrb = (d + GQ_ROWS - 1) / GQ_ROWS, ncb = (b + 63) / 64;
  const int ncu = cu_count();
  const int64_t cu = ncu > 0 ? ncu : 256;
  double best = -1.0;
  ks = 1;
  kchunk = (d + GQ_K - 1) / GQ_K * GQ_K;
  for (int k = 1; k <= 32; ++k) {
    const int64_t chunk = ((d + k - 1) / k + GQ_K - 1) / GQ_K * GQ_K;
    if (k > 1 && chunk < 256) break;
    const int ke = (int)((d + chunk - 1) / chunk);
    const int64_t wgs = nrb * ke * ncb;
    double score = (double)wgs / (double)(((wgs + cu - 1) / cu) * cu);
    if (wgs < 2 * cu) score *= 0.5;
    if (score > best + 1e-9) {
      best = score;
      ks = ke;
      kchunk = chunk;
    }
  }
}

struct EigWs {
  double* q;      // [d][b] orthonormal block
  double* y;      // [d][b] work block
  float* q32;     // [d][b] fp32 copy of q
  double* part;   // [ks][d][b] partial products (fp32 or fp64 elements)
  int ks;         // the products' K split (ksplit_for) and its chunk
  int64_t kchunk;
  double* mp;     // [NPART][b][b] partial column Grams
  double* m;      // [b][b]
  double* linvt;  // [b][b] (L^{-1})^T
  double* chol;   // [b][b + 1] Cholesky / Jacobi work matrix (when it does not fit in LDS)
  double* jac;    // [b][b + 1] Jacobi rotations (when they do not fit in LDS)
  double* s;      // [b][b] eigenvectors of H (columns)
  double* theta;  // [b]
  int* order;     // [b]
  double* u;      // [d][r]
  double* h;      // [b][b] projected block Q^T Y of a convergence check
  double* info;   // [4]: estimated residual, final residual
  float* info32;  // [4]: the same in fp32, for the host to read
};

EigWs carve(void* ws, int64_t d, int b, int r, int ks) {
  char* p = static_cast<char*>(ws);
  EigWs w;
  w.q = reinterpret_cast<double*>(p); p += align256((size_t)d * b * 8);
  w.y = reinterpret_cast<double*>(p); p += align256((size_t)d * b * 8);
  w.q32 = reinterpret_cast<float*>(p); p += align256((size_t)d * b * 4);
  w.part = reinterpret_cast<double*>(p); p += align256((size_t)ks * d * b * 8);
  w.mp = reinterpret_cast<double*>(p); p += align256((size_t)NPART * b * b * 8);
  w.m = reinterpret_cast<double*>(p); p += align256((size_t)b * b * 8);
  w.linvt = reinterpret_cast<double*>(p); p += align256((size_t)b * b * 8);
  w.chol = reinterpret_cast<double*>(p); p += align256((size_t)b * (b + 1) * 8);
  w.jac = reinterpret_cast<double*>(p); p += align256((size_t)b * (b + 1) * 8);
  w.s = reinterpret_cast<double*>(p); p += align256((size_t)b * b * 8);
  w.theta = reinterpret_cast<double*>(p); p += align256((size_t)b * 8);
  w.order = reinterpret_cast<int*>(p); p += align256((size_t)b * 4);
  w.u = reinterpret_cast<double*>(p); p += align256((size_t)d * r * 8);
  w.h = reinterpret_cast<double*>(p); p += align256((size_t)b * b * 8);
  w.info = reinterpret_cast<double*>(p); p += 256;
  w.info32 = reinterpret_cast<float*>(p); p += 256;
  return w;
}

size_t carve_bytes(int64_t d, int b, int r, int ks) {
  return align256((size_t)d * b * 8) * 2 + align256((size_t)d * b * 4) + align256((size_t)ks * d * b * 8) +
         align256((size_t)NPART * b * b * 8) + align256((size_t)b * b * 8) * 3 + align256((size_t)b * (b + 1) * 8) * 2 +
         align256((size_t)b * 8) +
         align256((size_t)b * 4) + align256((size_t)d * r * 8) + align256((size_t)b * b * 8) + 512;
}

__global__ void omega_kernel(double* q, float* q32, int64_t d, int b, uint64_t seed) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < d * b; i += (int64_t)gridDim.x * blockDim.x) {
    const float z = rng::gauss_at(seed, 0xFFFFFFFFu, 0xB0515u, (uint64_t)i);
    q[i] = (double)z;
    q32[i] = z;
  }
}

// Stage G[r0 .. r0+127][k0 .. k0+31] (rows and columns past the range read as 0).
__device__ __forceinline__ void stage_g(const float* __restrict__ g, int64_t d, int64_t r0, int64_t k0, int64_t k_end,
                                        float (*gs)[GQ_K + 1]) {
  for (int e = threadIdx.x; e < GQ_ROWS * GQ_K / 4; e += 256) {
    const int row = e >> 3, kc = (e & 7) * 4;
    const int64_t gr = r0 + row, gk = k0 + kc;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (gr < d) {
      const float* src = g + gr * d + gk;
      if ((d & 3) == 0 && gk + 3 < k_end) {
        const float4 f = *reinterpret_cast<const float4*>(src);
        v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = (gk + t < k_end) ? src[t] : 0.f;
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) gs[row][kc + t] = v[t];
  }
}

// part[ks][d][b] (fp32) = G[:, K range ks] Q32[K range ks][:] on v_mfma_f32_16x16x4f32;
// grid (row blocks of 128, ks, column blocks of 64); four waves of 32 rows x 64 columns.
// The next 32-deep chunk of G and Q is loaded into registers while the current one is
// multiplied out of LDS.
__global__ void __launch_bounds__(256) gq32_kernel(const float* __restrict__ g, const float* __restrict__ q,
                                                   float* __restrict__ part, int64_t d, int b, int64_t kchunk) {
  __shared__ float gs[GQ_ROWS][GQ_K + 1];
  __shared__ float qs[GQ_K][80];
  const int64_t r0 = (int64_t)blockIdx.x * GQ_ROWS;
  const int64_t k_begin = (int64_t)blockIdx.y * kchunk;
  const int64_t k_end = k_begin + kchunk < d ? k_begin + kchunk : d;
  const int c0 = blockIdx.z * 64;
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const bool vec = (d & 3) == 0;
  float gv[4][4], qv[8];
  auto load = [&](int64_t k0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = t + 256 * u;
      const int row = e >> 3, kc = (e & 7) * 4;
      const int64_t gr = r0 + row, gk = k0 + kc;
      const float* src = g + gr * d + gk;
      if (gr < d && vec && gk + 3 < k_end) {
        const float4 f = *reinterpret_cast<const float4*>(src);
        gv[u][0] = f.x; gv[u][1] = f.y; gv[u][2] = f.z; gv[u][3] = f.w;
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) gv[u][c] = (gr < d && gk + c < k_end) ? src[c] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = t + 256 * u;
      const int kk = e >> 6, cc = e & 63;
      const int64_t gk = k0 + kk;
      qv[u] = (gk < k_end && c0 + cc < b) ? q[gk * b + c0 + cc] : 0.f;
    }
  };
  floatx4 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (k_begin < k_end) load(k_begin);
  for (int64_t k0 = k_begin; k0 < k_end; k0 += GQ_K) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = t + 256 * u;
      const int row = e >> 3, kc = (e & 7) * 4;
#pragma unroll
      for (int c = 0; c < 4; ++c) gs[row][kc + c] = gv[u][c];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = t + 256 * u;
      qs[e >> 6][e & 63] = qv[u];
    }
    __syncthreads();
    if (k0 + GQ_K < k_end) load(k0 + GQ_K);
#pragma unroll
    for (int kk = 0; kk < GQ_K; kk += 4) {
      float a[2], bq[4];
#pragma unroll
      for (int i = 0; i < 2; ++i) a[i] = gs[wave * 32 + i * 16 + lr][kk + lk];
#pragma unroll
      for (int j = 0; j < 4; ++j) bq[j] = qs[kk + lk][j * 16 + lr];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], bq[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  float* out = part + (int64_t)blockIdx.y * d * b;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = r0 + wave * 32 + i * 16 + lk * 4 + v;
        const int col = c0 + j * 16 + lr;
        if (row < d && col < b) out[row * b + col] = acc[i][j][v];
      }
}

// part[ks][d][nc] (fp64) = G[:, K range ks] Q[K range ks][:nc] with fp64 accumulation
// (G read as fp32); grid (row blocks of 128, ks, column blocks of 64); each thread 8 rows
// x 4 columns.
__global__ void __launch_bounds__(256) gq64_kernel(const float* __restrict__ g, const double* __restrict__ q,
                                                   double* __restrict__ part, int64_t d, int nc, int64_t kchunk) {
  __shared__ float gs[GQ_ROWS][GQ_K + 1];
  __shared__ double qs[GQ_K][64];
  const int64_t r0 = (int64_t)blockIdx.x * GQ_ROWS;
  const int64_t k_begin = (int64_t)blockIdx.y * kchunk;
  const int64_t k_end = k_begin + kchunk < d ? k_begin + kchunk : d;
  const int c0 = blockIdx.z * 64;
  const int tc = threadIdx.x & 15, tr = threadIdx.x >> 4;   // columns tc + 16 j, rows tr * 8 + i
  double acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int64_t k0 = k_begin; k0 < k_end; k0 += GQ_K) {
    stage_g(g, d, r0, k0, k_end, gs);
    for (int e = threadIdx.x; e < GQ_K * 64; e += 256) {
      const int kk = e >> 6, cc = e & 63;
      const int64_t gk = k0 + kk;
      qs[kk][cc] = (gk < k_end && c0 + cc < nc) ? q[gk * nc + c0 + cc] : 0.0;
    }
    __syncthreads();
    for (int kk = 0; kk < GQ_K; ++kk) {
      double a[8], bq[4];
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = (double)gs[tr * 8 + i][kk];
#pragma unroll
      for (int j = 0; j < 4; ++j) bq[j] = qs[kk][tc + 16 * j];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], bq[j], acc[i][j]);
    }
    __syncthreads();
  }
  double* out = part + (int64_t)blockIdx.y * d * nc;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t row = r0 + tr * 8 + i;
      const int col = c0 + tc + 16 * j;
      if (row < d && col < nc) out[row * nc + col] = acc[i][j];
    }
}

// y[n] = sum over ks of part[ks][n] in split order (fp32 or fp64 partials), fp64 result.
template <typename T>
__global__ void sum_parts_kernel(const T* __restrict__ part, int ks, int64_t n, double* __restrict__ y) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    double s = 0.0;
    for (int k = 0; k < ks; ++k) s += (double)part[(int64_t)k * n + i];
    y[i] = s;
  }
}

// mp[p][i][j] = sum over the rows assigned to workgroup p of a[row][i] * bm[row][j]
// (fp64), for the CTT x CTT output block (blockIdx.y / nbk, blockIdx.y % nbk), CTT = 16 TU;
// rows are dealt to the gridDim.x workgroups in chunks of 32, each summed in row order.
template <int TU>
__global__ void __launch_bounds__(256) cross_partial_kernel(const double* __restrict__ a, const double* __restrict__ bm,
                                                            int64_t d, int b, double* __restrict__ mp) {
  constexpr int CTT = 16 * TU;
  __shared__ double as[32][CTT + 1];
  __shared__ double bs[32][CTT + 1];
  const int nbk = (b + CTT - 1) / CTT;
  const int i0 = (blockIdx.y / nbk) * CTT, j0 = (blockIdx.y % nbk) * CTT;
  const int ti = threadIdx.x >> 4, tj = threadIdx.x & 15;  // outputs (ti + 16 u, tj + 16 v)
  double acc[TU][TU];
#pragma unroll
  for (int u = 0; u < TU; ++u)
#pragma unroll
    for (int v = 0; v < TU; ++v) acc[u][v] = 0.0;
  for (int64_t c = blockIdx.x; c * 32 < d; c += gridDim.x) {
    const int64_t row0 = c * 32;
    for (int e = threadIdx.x; e < 32 * CTT; e += 256) {
      const int rr = e / CTT, cc = e % CTT;
      const int64_t row = row0 + rr;
      as[rr][cc] = (row < d && i0 + cc < b) ? a[row * b + i0 + cc] : 0.0;
      bs[rr][cc] = (row < d && j0 + cc < b) ? bm[row * b + j0 + cc] : 0.0;
    }
    __syncthreads();
    for (int rr = 0; rr < 32; ++rr) {
      double av[TU], bv[TU];
#pragma unroll
      for (int u = 0; u < TU; ++u) av[u] = as[rr][ti + 16 * u];
#pragma unroll
      for (int v = 0; v < TU; ++v) bv[v] = bs[rr][tj + 16 * v];
#pragma unroll
      for (int u = 0; u < TU; ++u)
#pragma unroll
        for (int v = 0; v < TU; ++v) acc[u][v] = fma(av[u], bv[v], acc[u][v]);
    }
    __syncthreads();
  }
  double* out = mp + (int64_t)blockIdx.x * b * b;
#pragma unroll
  for (int u = 0; u < TU; ++u)
#pragma unroll
    for (int v = 0; v < TU; ++v) {
      const int i = i0 + ti + 16 * u, j = j0 + tj + 16 * v;
      if (i < b && j < b) out[i * b + j] = acc[u][v];
    }
}

// m[e] = sum over p of mp[p][e] in a fixed order: 64 entries per workgroup, each summed
// by 4 threads over interleaved quarters of the partials, then the 4 sums in order.
__global__ void __launch_bounds__(256) reduce_parts_kernel(const double* __restrict__ mp, int np, int64_t n,
                                                           double* __restrict__ m) {
  __shared__ double sh[4][64];
  const int64_t e = (int64_t)blockIdx.x * 64 + (threadIdx.x & 63);
  const int q = threadIdx.x >> 6;
  double s = 0.0;
  if (e < n)
    for (int p = q; p < np; p += 4) s += mp[(int64_t)p * n + e];
  sh[q][threadIdx.x & 63] = s;
  __syncthreads();
  if (q == 0 && e < n) m[e] = ((sh[0][threadIdx.x] + sh[1][threadIdx.x]) + sh[2][threadIdx.x]) + sh[3][threadIdx.x];
}

// M = A^T B for A, B [d][b] (fp64), deterministic: partial sums over row chunks, then
// their sum in partial order.
void cross(const double* a, const double* bm, int64_t d, int b, double* mp, double* m, hipStream_t s) {
  int np = (int)((d + 63) / 64);
  np = np < 1 ? 1 : (np > NPART ? NPART : np);
  if (b <= 64) {
    const int nbk = (b + 63) / 64;
    cross_partial_kernel<4><<<dim3((unsigned)np, (unsigned)(nbk * nbk)), 256, 0, s>>>(a, bm, d, b, mp);
  } else {
    const int nbk = (b + 127) / 128;
    cross_partial_kernel<8><<<dim3((unsigned)np, (unsigned)(nbk * nbk)), 256, 0, s>>>(a, bm, d, b, mp);
  }
  reduce_parts_kernel<<<(unsigned)(((int64_t)b * b + 63) / 64), 256, 0, s>>>(mp, np, (int64_t)b * b, m);
}

// M = L L^T (left-looking Cholesky), then X = L^{-1} by forward substitution, written
// out transposed: linvt[k][j] = X[j][k].  For blocks past the register-blocked kernel
// below (b > 128): one workgroup, one lane per row (or column), the matrix in `scratch`
// with row stride b + 1.  L occupies the lower triangle; column c of X is kept transposed
// in row c's upper part (A[c][i] = X[i][c], i > c) and its diagonal in `xd`.
__global__ void __launch_bounds__(256) chol_inv_kernel(const double* __restrict__ m, double* __restrict__ A,
                                                       double* __restrict__ linvt, int b) {
  __shared__ double xd[512];
  __shared__ double sq[512];   // running sum of squares of each row of L
  const int ld = b + 1;
  const int t = threadIdx.x;
  for (int i = t / 64; i < b; i += 4)
    for (int k = t % 64; k < b; k += 64) A[i * ld + k] = m[i * b + k];
  for (int i = t; i < b; i += 256) sq[i] = 0.0;
  __syncthreads();
  if (t == 0) {
    const double s00 = A[0];
    A[0] = s00 > 1e-300 ? sqrt(s00) : 1e-150;
  }
  __syncthreads();
  // step j: every row i > j forms L_ij = (M_ij - sum_{k<j} L_ik L_jk) / L_jj; row j + 1,
  // then complete up to column j, forms its diagonal from its running sum of squares
  for (int j = 0; j < b - 1; ++j) {
    const double* lj = A + j * ld;
    const double inv = 1.0 / lj[j];
    for (int i = j + 1 + t; i < b; i += 256) {
      double* li = A + i * ld;
      double s0 = 0.0, s1 = 0.0;
      int k = 0;
      for (; k + 1 < j; k += 2) {
        s0 = fma(li[k], lj[k], s0);
        s1 = fma(li[k + 1], lj[k + 1], s1);
      }
      if (k < j) s0 = fma(li[k], lj[k], s0);
      const double v = (li[j] - (s0 + s1)) * inv;
      li[j] = v;
      const double ss = sq[i] + v * v;
      sq[i] = ss;
      if (i == j + 1) {
        const double dd = li[i] - ss;
        li[i] = dd > 1e-300 ? sqrt(dd) : 1e-150;
      }
    }
    __syncthreads();
  }
  // forward substitution L x = e_c per column c: x_c = 1 / L_cc,
  // x_i = -(sum_{k=c}^{i-1} L_ik x_k) / L_ii, x_k (k > c) stored at A[c][k]
  for (int c = t; c < b; c += 256) xd[c] = 1.0 / A[c * ld + c];
  __syncthreads();
  for (int c = t; c < b; c += 256) {
    double* xr = A + c * ld;
    for (int i = c + 1; i < b; ++i) {
      const double* li = A + i * ld;
      double s0 = li[c] * xd[c], s1 = 0.0;
      int k = c + 1;
      for (; k + 1 < i; k += 2) {
        s0 = fma(li[k], xr[k], s0);
        s1 = fma(li[k + 1], xr[k + 1], s1);
      }
      if (k < i) s0 = fma(li[k], xr[k], s0);
      xr[i] = -(s0 + s1) * xd[i];
    }
  }
  __syncthreads();
  for (int k = t / 64; k < b; k += 4)
    for (int jj = t % 64; jj < b; jj += 64)
      linvt[k * b + jj] = jj > k ? A[k * ld + jj] : (jj == k ? xd[k] : 0.0);
}

// The same factorisation and inverse for b <= 32 BS (BS = 2, 4) with the matrix in
// registers: 1024 threads as a 32 x 32 grid, thread (ti, tk) holding the BS x BS block of
// rows ti BS .., columns tk BS .. (order padded with identity; four waves per SIMD hide
// each other's latency).  Elimination is
// right-looking in the unscaled (LDL^T) form: at step j the threads holding column j
// publish it through LDS and every element of the trailing part takes
// a_ik -= (a_ij / a_jj) a_kj, one barrier per step (the column buffer alternates between
// two slots; the upper triangle is updated too and ignored).  L_ik = a_ik / sqrt(a_kk)
// then goes to LDS, and L X = I is solved the same way, row k of X published at step k
// and subtracted from the rows below it.  Pivots at or below 1e-300 are replaced by
// 1e-300 (a rank-deficient block stays finite), as in chol_inv_kernel.
template <int BS>
__global__ void __launch_bounds__(1024) chol_inv_blk_kernel(const double* __restrict__ m, double* __restrict__ linvt,
                                                            int b) {
  constexpr int TG = 32, NT = TG * TG, BP = TG * BS, LD = BP + 1;
  __shared__ double A[BP * LD];
  __shared__ double col[2][BP];
  __shared__ double piv[BP];
  __shared__ double xd[BP];   // 1 / L_kk
  const int ti = threadIdx.x / TG, tk = threadIdx.x % TG;
  const int i0 = ti * BS, k0 = tk * BS;
  double a[BS][BS];
#pragma unroll
  for (int ii = 0; ii < BS; ++ii)
#pragma unroll
    for (int kk = 0; kk < BS; ++kk) {
      const int i = i0 + ii, k = k0 + kk;
      a[ii][kk] = (i < b && k < b) ? m[(int64_t)i * b + k] : (i == k ? 1.0 : 0.0);
    }
  for (int j = 0; j < b; ++j) {
    double* cj = col[j & 1];
    if (tk == j / BS) {
      const int jc = j % BS;
#pragma unroll
      for (int ii = 0; ii < BS; ++ii) {
        double v = a[ii][0];   // column jc of the block, by selects (registers stay static)
#pragma unroll
        for (int q = 1; q < BS; ++q) v = jc == q ? a[ii][q] : v;
        cj[i0 + ii] = v;
      }
    }
    __syncthreads();
    const double pv = cj[j] > 1e-300 ? cj[j] : 1e-300;
    const double ipv = 1.0 / pv;
    if (k0 + BS - 1 > j && i0 + BS - 1 > j) {   // block reaches past row and column j
      double ck[BS];
#pragma unroll
      for (int kk = 0; kk < BS; ++kk) ck[kk] = cj[k0 + kk];
#pragma unroll
      for (int ii = 0; ii < BS; ++ii) {
        const double f = cj[i0 + ii] * ipv;
#pragma unroll
        for (int kk = 0; kk < BS; ++kk)
          if (k0 + kk > j) a[ii][kk] = fma(-f, ck[kk], a[ii][kk]);
      }
    }
    if (threadIdx.x == 0) piv[j] = pv;
  }
  __syncthreads();
  for (int k = threadIdx.x; k < BP; k += NT) {
    const double l = k < b ? sqrt(piv[k]) : 1.0;
    piv[k] = l;
    xd[k] = 1.0 / l;
  }
  __syncthreads();
#pragma unroll
  for (int ii = 0; ii < BS; ++ii)
#pragma unroll
    for (int kk = 0; kk < BS; ++kk) {
      const int i = i0 + ii, k = k0 + kk;
      if (k < i) A[i * LD + k] = i < b ? a[ii][kk] * xd[k] : 0.0;
      else if (k == i) A[i * LD + k] = piv[k];
    }
  // X = L^{-1}: the block starts as I and row k is final at step k
#pragma unroll
  for (int ii = 0; ii < BS; ++ii)
#pragma unroll
    for (int kk = 0; kk < BS; ++kk) a[ii][kk] = (i0 + ii == k0 + kk) ? 1.0 : 0.0;
  __syncthreads();
  for (int k = 0; k < b; ++k) {
    double* xr = col[k & 1];
    if (ti == k / BS) {
      const int r = k % BS;
#pragma unroll
      for (int ii = 0; ii < BS; ++ii)
        if (ii == r) {
#pragma unroll
          for (int kk = 0; kk < BS; ++kk) {
            a[ii][kk] *= xd[k];
            xr[k0 + kk] = a[ii][kk];
          }
        }
    }
    __syncthreads();
    if (i0 + BS - 1 > k && k0 <= k) {   // rows below k; X is zero right of column k
      double xk[BS];
#pragma unroll
      for (int kk = 0; kk < BS; ++kk) xk[kk] = xr[k0 + kk];
#pragma unroll
      for (int ii = 0; ii < BS; ++ii) {
        const double l = A[(i0 + ii) * LD + k];
        if (i0 + ii > k) {
#pragma unroll
          for (int kk = 0; kk < BS; ++kk) a[ii][kk] = fma(-l, xk[kk], a[ii][kk]);
        }
      }
    }
  }
  // linvt[c][i] = X[i][c]
#pragma unroll
  for (int ii = 0; ii < BS; ++ii)
#pragma unroll
    for (int kk = 0; kk < BS; ++kk) {
      const int i = i0 + ii, c = k0 + kk;
      if (i < b && c < b) linvt[(int64_t)c * b + i] = i >= c ? a[ii][kk] : 0.0;
    }
}

// q[i][j] = sum over k <= j of y[i][k] linvt[k][j]  (Q = Y L^{-T}); also the fp32 copy.
// Rows are processed 256 / b at a time (b <= 256: one thread per output), staged in LDS.
__global__ void __launch_bounds__(256) apply_linv_kernel(const double* __restrict__ y, const double* __restrict__ linvt,
                                                         int64_t d, int b, double* __restrict__ q, float* __restrict__ q32) {
  __shared__ double lt[128 * 128];
  __shared__ double yr[256];
  const bool in_lds = b <= 128;
  if (in_lds) {
    for (int e = threadIdx.x; e < b * b; e += 256) lt[e] = linvt[e];
  }
  const double* L = in_lds ? lt : linvt;
  const int rows = b <= 256 ? 256 / b : 1;          // rows per pass
  const int t = threadIdx.x;
  for (int64_t r0 = (int64_t)blockIdx.x * rows; r0 < d; r0 += (int64_t)gridDim.x * rows) {
    __syncthreads();
    if (b <= 256) {
      const int64_t idx = r0 * b + t;
      if (t < rows * b && r0 + t / b < d) yr[t] = y[idx];
    }
    __syncthreads();
    if (b <= 256) {
      const int rr = t / b, j = t % b;
      const int64_t i = r0 + rr;
      if (rr < rows && i < d) {
        const double* yy = yr + rr * b;
        double s0 = 0.0, s1 = 0.0;
        int k = 0;
        for (; k + 1 <= j; k += 2) {
          s0 = fma(yy[k], L[k * b + j], s0);
          s1 = fma(yy[k + 1], L[(k + 1) * b + j], s1);
        }
        if (k == j) s0 = fma(yy[k], L[k * b + j], s0);
        const double sum = s0 + s1;
        q[i * b + j] = sum;
        if (q32) q32[i * b + j] = (float)sum;
      }
    } else {
      for (int j = t; j < b; j += 256) {
        const double* yy = y + r0 * b;
        double sum = 0.0;
        for (int k = 0; k <= j; ++k) sum = fma(yy[k], L[k * b + j], sum);
        q[r0 * b + j] = sum;
        if (q32) q32[r0 * b + j] = (float)sum;
      }
    }
  }
}

// Parallel cyclic Jacobi on the symmetric b x b matrix hg, eigenvectors in s (global,
// [b][b]), eigenvalues sorted descending into theta/order.  Round-robin pairing: in
// each of the n-1 rounds of a sweep, index 0 is fixed and the others rotate, giving
// n/2 disjoint pairs (n = b rounded up to even).  For blocks past the one-sided kernel
// below (b > 128): H and the rotations S are worked on in `work` and `swork` ([b][b + 1]
// each, row stride b + 1); S is written to s ([b][b]) at the end.
template <int PMAX>
__global__ void __launch_bounds__(256) jacobi_kernel(const double* __restrict__ hg, double* __restrict__ work,
                                                     double* __restrict__ swork, double* __restrict__ s_out,
                                                     double* theta, int* order, int b, int sweeps) {
  __shared__ double cs[256], sn[256];
  __shared__ int pp[256], qq[256];
  __shared__ double off_sh[256], tot_sh[256];
  double* h = work;
  double* s = swork;
  const int ld = b + 1;
  const int n = (b + 1) & ~1;
  const int t = threadIdx.x;
  const int wv = t >> 6, lane = t & 63;
  for (int i = t / 64; i < b; i += 4)
    for (int j = t % 64; j < b; j += 64) {
      s[i * ld + j] = (i == j) ? 1.0 : 0.0;
      h[i * ld + j] = hg[i * b + j];
    }
  __syncthreads();
  for (int sw = 0; sw < sweeps; ++sw) {
    double off = 0.0, tot = 0.0;
    for (int i = t / 64; i < b; i += 4)
      for (int j = t % 64; j < b; j += 64) {
        const double v = h[i * ld + j] * h[i * ld + j];
        tot += v;
        if (i != j) off += v;
      }
    off_sh[t] = off;
    tot_sh[t] = tot;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if (t < o) {
        off_sh[t] += off_sh[t + o];
        tot_sh[t] += tot_sh[t + o];
      }
      __syncthreads();
    }
    const bool done = off_sh[0] <= 1e-26 * tot_sh[0];   // off-diagonal norm <= 1e-13 of the whole
    __syncthreads();
    if (done) break;
    for (int round = 0; round < n - 1; ++round) {
      for (int k = t; k < n / 2; k += 256) {
        int a, c;
        if (k == 0) {
          a = 0;
          c = 1 + (round % (n - 1));
        } else {
          a = 1 + ((round + k) % (n - 1));
          c = 1 + ((round + n - 1 - k) % (n - 1));
        }
        if (a > c) { const int tt = a; a = c; c = tt; }
        pp[k] = a;
        qq[k] = c;
        double cc = 1.0, ss = 0.0;
        if (c < b) {
          const double apq = h[a * ld + c];
          if (fabs(apq) > 1e-300) {
            const double tau = (h[c * ld + c] - h[a * ld + a]) / (2.0 * apq);
            const double tq = (tau >= 0 ? 1.0 : -1.0) / (fabs(tau) + sqrt(1.0 + tau * tau));
            cc = 1.0 / sqrt(1.0 + tq * tq);
            ss = tq * cc;
          }
        }
        cs[k] = cc;
        sn[k] = ss;
      }
      __syncthreads();
      // columns: H <- H J, S <- S J.  Wave w takes pairs w, w + 4, ...; each lane one row.
      // All loads of a row are issued before its stores (the pairs are disjoint).
      for (int kb = 0; kb < n / 2; kb += 4 * PMAX)
      for (int i = lane; i < b; i += 64) {
        double hp[PMAX], hq[PMAX], vp[PMAX], vq[PMAX];
#pragma unroll
        for (int u = 0; u < PMAX; ++u) {
          const int k = kb + wv + 4 * u;
          if (k < n / 2 && qq[k] < b) {
            hp[u] = h[i * ld + pp[k]];
            hq[u] = h[i * ld + qq[k]];
            vp[u] = s[i * ld + pp[k]];
            vq[u] = s[i * ld + qq[k]];
          }
        }
#pragma unroll
        for (int u = 0; u < PMAX; ++u) {
          const int k = kb + wv + 4 * u;
          if (k < n / 2 && qq[k] < b) {
            const double ck = cs[k], sk = sn[k];
            h[i * ld + pp[k]] = ck * hp[u] - sk * hq[u];
            h[i * ld + qq[k]] = sk * hp[u] + ck * hq[u];
            s[i * ld + pp[k]] = ck * vp[u] - sk * vq[u];
            s[i * ld + qq[k]] = sk * vp[u] + ck * vq[u];
          }
        }
      }
      __syncthreads();
      // rows: H <- J^T H; each lane one column
      for (int kb = 0; kb < n / 2; kb += 4 * PMAX)
      for (int j = lane; j < b; j += 64) {
        double ha[PMAX], hc[PMAX];
#pragma unroll
        for (int u = 0; u < PMAX; ++u) {
          const int k = kb + wv + 4 * u;
          if (k < n / 2 && qq[k] < b) {
            ha[u] = h[pp[k] * ld + j];
            hc[u] = h[qq[k] * ld + j];
          }
        }
#pragma unroll
        for (int u = 0; u < PMAX; ++u) {
          const int k = kb + wv + 4 * u;
          if (k < n / 2 && qq[k] < b) {
            const double ck = cs[k], sk = sn[k];
            h[pp[k] * ld + j] = ck * ha[u] - sk * hc[u];
            h[qq[k] * ld + j] = sk * ha[u] + ck * hc[u];
          }
        }
      }
      __syncthreads();
    }
  }
  for (int i = t / 64; i < b; i += 4)
    for (int j = t % 64; j < b; j += 64) s_out[i * b + j] = s[i * ld + j];
  if (t == 0) {
    for (int i = 0; i < b; ++i) order[i] = i;
    for (int i = 0; i < b; ++i) {
      int best = i;
      for (int j = i + 1; j < b; ++j)
        if (h[order[j] * ld + order[j]] > h[order[best] * ld + order[best]]) best = j;
      const int tt = order[i];
      order[i] = order[best];
      order[best] = tt;
      theta[i] = h[order[i] * ld + order[i]];
    }
  }
}

// One-sided (Hestenes) Jacobi for b <= BP (BP = 64 or 128) on a symmetric positive
// semidefinite H: the columns a_p of A (A = H at the start) are rotated in disjoint pairs,
// round-robin as above, until every pair is orthogonal.  Then A = H V with V orthogonal
// and A^T A diagonal, so V diagonalises H^2 and hence H: a_p = theta_p v_p, the
// eigenvalue is the column norm and the eigenvector the normalised column (accurate for
// the large eigenvalues the basis keeps; no V is accumulated).  A sits in LDS column by
// column (stride BP + 1); each pair is worked on by 16 lanes, BP / 16 rows each, held in
// registers between the pair's dot products and its update (8 BP threads: several waves
// per SIMD hide each other's latency); one barrier per round.  A pair rotates when
// |a_p . a_q| > 1e-15 ||a_p|| ||a_q||; the sweeps stop once the largest such ratio of a
// sweep is at most 1e-13.  Outputs as jacobi_kernel.
template <int BP>
__global__ void __launch_bounds__(8 * BP) jacobi1s_kernel(const double* __restrict__ hg, double* __restrict__ s_out,
                                                          double* __restrict__ theta, int* __restrict__ order, int b,
                                                          int sweeps) {
  constexpr int LD = BP + 1, G = 16, RPL = BP / G, NT = 8 * BP, NW = NT / 64;
  __shared__ double A[BP * LD];
  __shared__ double nrm[BP];
  __shared__ double wmax[NW];
  const int t = threadIdx.x, grp = t / G, gl = t % G;
  const int n = (b + 1) & ~1;
  for (int e = t; e < BP * BP; e += NT) {
    const int c = e / BP, i = e % BP;
    A[c * LD + i] = (i < b && c < b) ? hg[c * b + i] : 0.0;   // column c of H (= row c)
  }
  __syncthreads();
  for (int sw = 0; sw < sweeps; ++sw) {
    double worst = 0.0;
    for (int round = 0; round < n - 1; ++round) {
      if (grp < n / 2) {
        int p, q;
        if (grp == 0) {
          p = 0;
          q = 1 + round;
        } else {
          int a1 = round + grp, a2 = round - grp;   // round +- grp modulo n - 1
          if (a1 >= n - 1) a1 -= n - 1;
          if (a2 < 0) a2 += n - 1;
          p = 1 + a1;
          q = 1 + a2;
        }
        if (p > q) { const int tt = p; p = q; q = tt; }
        if (q < b) {
          double ap[RPL], aq[RPL];
          double al0 = 0.0, al1 = 0.0, be0 = 0.0, be1 = 0.0, ga0 = 0.0, ga1 = 0.0;
#pragma unroll
          for (int k = 0; k < RPL; ++k) {
            ap[k] = A[p * LD + k * G + gl];
            aq[k] = A[q * LD + k * G + gl];
          }
#pragma unroll
          for (int k = 0; k < RPL; k += 2) {
            al0 = fma(ap[k], ap[k], al0);
            be0 = fma(aq[k], aq[k], be0);
            ga0 = fma(ap[k], aq[k], ga0);
            al1 = fma(ap[k + 1], ap[k + 1], al1);
            be1 = fma(aq[k + 1], aq[k + 1], be1);
            ga1 = fma(ap[k + 1], aq[k + 1], ga1);
          }
          double al = al0 + al1, be = be0 + be1, ga = ga0 + ga1;
#pragma unroll
          for (int o = 1; o < G; o <<= 1) {
            al += __shfl_xor(al, o, 64);
            be += __shfl_xor(be, o, 64);
            ga += __shfl_xor(ga, o, 64);
          }
          const double nn = sqrt(al * be);
          if (fabs(ga) > 1e-15 * nn && fabs(ga) > 1e-300) {
            worst = fmax(worst, fabs(ga) / nn);
            const double zeta = (be - al) / (2.0 * ga);
            const double tq = (zeta >= 0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
            const double cc = 1.0 / sqrt(1.0 + tq * tq), ss = tq * cc;
#pragma unroll
            for (int k = 0; k < RPL; ++k) {
              A[p * LD + k * G + gl] = cc * ap[k] - ss * aq[k];
              A[q * LD + k * G + gl] = ss * ap[k] + cc * aq[k];
            }
          }
        }
      }
      __syncthreads();
    }
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) worst = fmax(worst, __shfl_xor(worst, o, 64));
    if ((t & 63) == 0) wmax[t >> 6] = worst;
    __syncthreads();
    double w = 0.0;
#pragma unroll
    for (int q = 0; q < NW; ++q) w = fmax(w, wmax[q]);
    __syncthreads();
    if (w <= 1e-13) break;
  }
  if (t < b) {
    double s2 = 0.0;
    for (int i = 0; i < b; ++i) s2 = fma(A[t * LD + i], A[t * LD + i], s2);
    nrm[t] = sqrt(s2);
  }
  __syncthreads();
  if (t < b) {   // rank by value, descending, lower index first on ties
    const double v = nrm[t];
    int rank = 0;
    for (int j = 0; j < b; ++j) rank += (nrm[j] > v || (nrm[j] == v && j < t)) ? 1 : 0;
    order[rank] = t;
    theta[rank] = v;
  }
  for (int e = t; e < b * b; e += NT) {
    const int k = e / b, c = e % b;
    s_out[e] = A[c * LD + k] / fmax(nrm[c], 1e-300);
  }
}

// Symmetric eigenproblem of the b x b block: one-sided Jacobi up to b = 128, else the
// two-sided kernel with its matrices in global memory.
void eig_small(const double* h, EigWs& w, int b, hipStream_t s) {
  if (b <= 64) jacobi1s_kernel<64><<<1, 512, 0, s>>>(h, w.s, w.theta, w.order, b, 40);
  else if (b <= 128) jacobi1s_kernel<128><<<1, 1024, 0, s>>>(h, w.s, w.theta, w.order, b, 40);
  else jacobi_kernel<12><<<1, 256, 0, s>>>(h, w.chol, w.jac, w.s, w.theta, w.order, b, 40);
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

// resid = max_c ||G u_c - theta_c u_c|| / theta_0, with y = G u already formed: one
// workgroup per column writes its norm to cn[c] (fixed-order reduction), then
// resid_max_kernel takes the maximum and writes info[1] (fp64) and info32[1] (fp32).
__global__ void __launch_bounds__(256) resid_cols_kernel(const double* __restrict__ y, const double* __restrict__ u,
                                                         const double* __restrict__ theta, int64_t d, int r,
                                                         double* __restrict__ cn) {
  __shared__ double sh[256];
  const int c = blockIdx.x;
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
  if (threadIdx.x == 0) cn[c] = sqrt(sh[0]);
}

__global__ void resid_max_kernel(const double* __restrict__ cn, const double* __restrict__ theta, int r, double* info,
                                 float* info32) {
  if (threadIdx.x != 0) return;
  double worst = 0.0;
  for (int c = 0; c < r; ++c) worst = fmax(worst, cn[c]);
  const double v = worst / fmax(fabs(theta[0]), 1e-300);
  info[1] = v;
  info32[1] = (float)v;
}

// h <- (h + h^T) / 2 in place (b x b).  The check's projected block comes from the fp32
// products and is symmetric only to their rounding; the Jacobi solver needs it exact.
__global__ void sym_kernel(double* h, int b) {
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < b * b; e += gridDim.x * blockDim.x) {
    const int i = e / b, j = e % b;
    if (i < j) {
      const double v = 0.5 * (h[i * b + j] + h[j * b + i]);
      h[i * b + j] = v;
      h[j * b + i] = v;
    }
  }
}

// Convergence estimate of the current block without another product: with Q orthonormal,
// Y = G Q (the iteration's fp32 product), H = sym(Q^T Y) and M = Y^T Y, the Ritz pair
// (theta_c, Q s_c) of a unit eigenvector s_c of H has residual
//   ||Y s_c - theta_c Q s_c||^2 = s_c^T M s_c - theta_c^2,  theta_c = s_c^T H s_c.
// Workgroup c (one of the top r) forms both quadratic forms (thread k: (M s)_k and
// (H s)_k, coalesced over k since M and H are symmetric) into part[c], part[r + c].
__global__ void __launch_bounds__(256) est_cols_kernel(const double* __restrict__ m, const double* __restrict__ h,
                                                       const double* __restrict__ sv, const int* __restrict__ order,
                                                       int b, int r, double* __restrict__ part) {
  __shared__ double sc[512];
  __shared__ double rm[256], rh[256];
  const int c = blockIdx.x, t = threadIdx.x, col = order[c];
  for (int k = t; k < b; k += 256) sc[k] = sv[k * b + col];
  __syncthreads();
  double qm = 0.0, qh = 0.0;
  for (int k = t; k < b; k += 256) {
    double um = 0.0, uh = 0.0;
    for (int i = 0; i < b; ++i) {
      um = fma(m[i * b + k], sc[i], um);
      uh = fma(h[i * b + k], sc[i], uh);
    }
    qm = fma(sc[k], um, qm);
    qh = fma(sc[k], uh, qh);
  }
  rm[t] = qm;
  rh[t] = qh;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o) {
      rm[t] += rm[t + o];
      rh[t] += rh[t + o];
    }
    __syncthreads();
  }
  if (t == 0) {
    part[c] = rm[0];
    part[r + c] = rh[0];
  }
}

// max_c sqrt(max(s_c^T M s_c - theta_c^2, 0)) / theta_0 into info[0] and info32[0].
__global__ void est_final_kernel(const double* __restrict__ part, int r, double* info, float* info32) {
  if (threadIdx.x != 0) return;
  double worst = 0.0;
  for (int c = 0; c < r; ++c) {
    const double th = part[r + c];
    worst = fmax(worst, sqrt(fmax(part[c] - th * th, 0.0)));
  }
  const double v = worst / fmax(fabs(part[r]), 1e-300);
  info[0] = v;
  info32[0] = (float)v;
}

// The caller's convergence report: residual (info[1]), gap theta_{r-1} / theta_r of the
// final Ritz values (0-based: last kept over first discarded), iterations, and whether
// the residual meets tol (always 1 when tol == 0).
__global__ void report_kernel(zoact_eig_report* rep, const double* info, const double* theta, int r, int iters,
                              float tol) {
  const float res = (float)info[1];
  rep->resid = res;
  rep->gap = (float)(theta[r - 1] / fmax(fabs(theta[r]), 1e-300));
  rep->iters = iters;
  rep->converged = (tol <= 0.f || res <= tol) ? 1 : 0;
}

// (L^{-1})^T of the Cholesky factor of w.m into w.linvt.
void chol_inv(EigWs& w, int b, hipStream_t s) {
  if (b <= 64) chol_inv_blk_kernel<2><<<1, 1024, 0, s>>>(w.m, w.linvt, b);
  else if (b <= 128) chol_inv_blk_kernel<4><<<1, 1024, 0, s>>>(w.m, w.linvt, b);
  else chol_inv_kernel<<<1, 256, 0, s>>>(w.m, w.chol, w.linvt, b);
}

// Q = orth(Y) by Cholesky-QR (applied `passes` times).  Reads y, leaves the
// orthonormal block in q (and its fp32 copy in q32); y is overwritten.  Inside the
// iteration one pass keeps the block well conditioned; the block handed to
// Rayleigh-Ritz gets two, which makes it orthonormal to working precision.
hipError_t orth(EigWs& w, int64_t d, int b, int passes, hipStream_t s) {
  const unsigned gapp = (unsigned)((d * b + 255) / 256 > 256 ? 256 : (d * b + 255) / 256);
  double* src = w.y;
  double* dst = w.q;
  for (int pass = 0; pass < passes; ++pass) {
    cross(src, src, d, b, w.mp, w.m, s);
    chol_inv(w, b, s);
    apply_linv_kernel<<<gapp, 256, 0, s>>>(src, w.linvt, d, b, dst, pass == passes - 1 ? w.q32 : nullptr);
    double* t = src;
    src = dst;
    dst = t;
  }
  // the result is in src; make it w.q
  if (src != w.q) {
    w.y = w.q;
    w.q = src;
  }
  return hipGetLastError();
}

// G X with fp64 accumulation into y [d][nc] (X fp64 [d][nc], nc <= 512).
hipError_t gx64(const float* g, const double* x, int64_t d, int nc, EigWs& w, double* y, hipStream_t s) {
  const int ks = w.ks;
  const int64_t kchunk = w.kchunk;
  gq64_kernel<<<dim3((unsigned)((d + GQ_ROWS - 1) / GQ_ROWS), (unsigned)ks, (unsigned)((nc + 63) / 64)), 256, 0, s>>>(
      g, x, w.part, d, nc, kchunk);
  const int64_t n = d * nc;
  sum_parts_kernel<double><<<(unsigned)((n + 255) / 256 > 4096 ? 4096 : (n + 255) / 256), 256, 0, s>>>(w.part, ks, n, y);
  return hipGetLastError();
}

}  // namespace

size_t basis_ws_bytes(int64_t d, int32_t r, int32_t p) {
  int ks;
  int64_t kchunk;
  ksplit_for(d, r + p, ks, kchunk);
  return carve_bytes(d, r + p, r, ks);
}

hipError_t launch_gram(const void* x, int32_t dtype, int64_t n_tok, int64_t d, int64_t ld, float* g, int accumulate,
                       hipStream_t s) {
  if (dtype == ZOACT_BF16) {
    const int nt = (int)((d + GT - 1) / GT);
    gram_bf16_kernel<<<dim3((unsigned)(nt * (nt + 1) / 2)), 256, 0, s>>>(static_cast<const uint16_t*>(x), n_tok, d, ld,
                                                                          g, accumulate, nt);
  } else {
    int64_t gb = (d * d + 255) / 256;
    if (gb > 65535) gb = 65535;
    gram_f32_kernel<<<dim3((unsigned)gb), 256, 0, s>>>(static_cast<const float*>(x), n_tok, d, ld, g, accumulate);
  }
  return hipGetLastError();
}

// The token-side form: X (bf16 [n][ld], D values per row) whose Gram X X^T the solver
// ran on, and the buffers that carry its Ritz vectors back to the D features.
struct Rows {
  const uint16_t* x;
  int64_t D, ld;
  double* up;    // [D][r] basis
  double* yp;    // [D][r] X^T X times the basis (residual)
  double* sc;    // [r] column norms of X^T V
  double* part;  // [ks][D][r] depth-chunk partials of X^T V
  int ks;
  int64_t tchunk;
};

// Depth split of X^T V over n rows: about two workgroups per CU, chunks a multiple of 32
// rows (at least 64).
static void xv_split(int64_t n, int64_t D, int r, int& ks, int64_t& tchunk) {
  const int64_t blocks = ((D + XV_J - 1) / XV_J) * ((r + XV_C - 1) / XV_C);
  const int ncu = cu_count();
  const int64_t want = (2 * (int64_t)(ncu > 0 ? ncu : 256) + blocks - 1) / blocks;
  tchunk = ((n + want - 1) / want + XV_T - 1) / XV_T * XV_T;
  if (tchunk < 64) tchunk = 64;
  ks = (int)((n + tchunk - 1) / tchunk);
}

// out [D][r] = X^T v for v [n][r] (fp64), summed over the depth chunks in order.
static void xt_v(const Rows& rw, int64_t n, const double* v, int r, double* out, hipStream_t s) {
  const dim3 grid((unsigned)((rw.D + XV_J - 1) / XV_J), (unsigned)((r + XV_C - 1) / XV_C), (unsigned)rw.ks);
  xt_v_kernel<<<grid, 256, 0, s>>>(rw.x, n, rw.D, rw.ld, v, r, rw.tchunk, rw.part);
  const int64_t m = rw.D * r;
  sum_chunks_kernel<<<(unsigned)((m + 255) / 256 > 4096 ? 4096 : (m + 255) / 256), 256, 0, s>>>(rw.part, rw.ks, m, out);
}

// The residual of a finished basis into info[1] / info32[1]; the column norms go to w.mp
// (free once the Rayleigh-Ritz product is formed).
static void basis_resid(const double* y, const double* u, const double* theta, int64_t d, int r, EigWs& w, hipStream_t s) {
  resid_cols_kernel<<<dim3((unsigned)r), 256, 0, s>>>(y, u, theta, d, r, w.mp);
  resid_max_kernel<<<1, 64, 0, s>>>(w.mp, theta, r, w.info, w.info32);
}

// Rayleigh-Ritz of the orthonormal block w.q with fp64 accumulation, the basis outputs,
// and (when `resid` is set) the residual of the result into info[1] / info32[1].  With
// `rows`, g is X X^T and its Ritz vectors V are eigenvectors of that Gram (X's left
// singular vectors); the basis is then X^T V with unit columns, X^T X u = X^T (X X^T v) / s
// gives the residual against X^T X, and the Ritz values are the same eigenvalues.
static hipError_t finish(const float* g, int64_t d, int b, int r, EigWs& w, const Rows* rows, void* ut,
                         int32_t ut_dtype, float* ut_master, float* eigvals, bool resid, hipStream_t s) {
  hipError_t e = gx64(g, w.q, d, b, w, w.y, s);   // H = Q^T (G Q)
  if (e != hipSuccess) return e;
  cross(w.q, w.y, d, b, w.mp, w.m, s);
  eig_small(w.m, w, b, s);
  int64_t gb = (d * r + 255) / 256;
  if (gb > 65535) gb = 65535;
  ritz_vectors_kernel<<<dim3((unsigned)gb), 256, 0, s>>>(w.q, w.s, w.order, w.u, d, b, r);
  const int ubf = ut_dtype == ZOACT_BF16 ? 1 : 0;
  if (!rows) {
    finish_basis_kernel<<<dim3((unsigned)r), 256, 0, s>>>(w.u, w.theta, d, r, ut, ubf, ut_master, eigvals);
    if (resid) {
      e = gx64(g, w.u, d, r, w, w.y, s);   // y = G u
      if (e != hipSuccess) return e;
      basis_resid(w.y, w.u, w.theta, d, r, w, s);
    }
    return hipGetLastError();
  }
  xt_v(*rows, d, w.u, r, rows->up, s);
  colscale_kernel<<<dim3((unsigned)r), 256, 0, s>>>(rows->up, rows->D, r, rows->sc, 1);
  finish_basis_kernel<<<dim3((unsigned)r), 256, 0, s>>>(rows->up, w.theta, rows->D, r, ut, ubf, ut_master, eigvals);
  if (resid) {
    e = gx64(g, w.u, d, r, w, w.y, s);   // X X^T v
    if (e != hipSuccess) return e;
    xt_v(*rows, d, w.y, r, rows->yp, s);
    colscale_kernel<<<dim3((unsigned)r), 256, 0, s>>>(rows->yp, rows->D, r, rows->sc, 0);
    basis_resid(rows->yp, rows->up, w.theta, rows->D, r, w, s);
  }
  return hipGetLastError();
}

static hipError_t read_info(const EigWs& w, int k, float& v, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(&v, w.info32 + k, sizeof(float), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return e;
}

// Subspace iteration: product k (k = 0 .. max_iter) forms Y = G Q_{k-1} (Q_{-1} = Omega)
// and Q_k = orth(Y).  Fixed mode runs all max_iter + 1 products, the last with a second
// Cholesky-QR pass, with no host synchronisation unless tol > 0 (then the final residual
// is read back).  Adaptive mode estimates the residual of the top-r Ritz pairs at
// checks (est_cols_kernel, from the products already formed), reads it back, and when
// it is at or below tol finishes with Rayleigh-Ritz and the exact residual; if that is
// still above tol and products remain, the iteration continues from Q.
static hipError_t solve(const float* g, int64_t d, int32_t r, int32_t p, const zoact_eig_opts& o, const Rows* rows,
                        void* ut, int32_t ut_dtype, float* ut_master, float* eigvals, zoact_eig_report* report,
                        void* ws, hipStream_t s, bool& met) {
  const int b = r + p;
  int ks;
  int64_t kchunk;
  ksplit_for(d, b, ks, kchunk);
  EigWs w = carve(ws, d, b, r, ks);
  w.ks = ks;
  w.kchunk = kchunk;
  const int64_t n = d * b;
  const unsigned g1 = (unsigned)((n + 255) / 256 > 4096 ? 4096 : (n + 255) / 256);
  const dim3 gq_grid((unsigned)((d + GQ_ROWS - 1) / GQ_ROWS), (unsigned)ks, (unsigned)((b + 63) / 64));
  const bool adaptive = o.adaptive != 0;
  const bool want_resid = report != nullptr || o.tol > 0.f;
  met = true;
  omega_kernel<<<g1, 256, 0, s>>>(w.q, w.q32, d, b, o.seed);
  int k = 0;
  hipError_t e;
  // Checks: the first two check_every iterations apart; from then on at the iteration
  // where the estimates' geometric rate predicts tol, at least check_every later, and
  // none once the prediction lies past max_iter or the estimate stops falling (the run
  // then ends like the fixed mode, with the exact residual deciding).
  int next_check = adaptive ? o.check_every : INT32_MAX;
  int prev_k = -1;
  float prev_est = 0.f;
  for (;;) {
    bool final_product = k == o.max_iter;
    const bool check = !final_product && k == next_check;
    gq32_kernel<<<gq_grid, 256, 0, s>>>(g, w.q32, reinterpret_cast<float*>(w.part), d, b, kchunk);
    sum_parts_kernel<float><<<g1, 256, 0, s>>>(reinterpret_cast<const float*>(w.part), ks, n, w.y);
    if (check) {
      cross(w.q, w.y, d, b, w.mp, w.h, s);   // H = Q^T Y before Q is replaced
      sym_kernel<<<(unsigned)((b * b + 255) / 256), 256, 0, s>>>(w.h, b);
    }
    e = orth(w, d, b, final_product ? 2 : 1, s);   // leaves M = Y^T Y of the first pass in w.m
    if (e != hipSuccess) return e;
    if (check) {
      eig_small(w.h, w, b, s);
      est_cols_kernel<<<(unsigned)r, 256, 0, s>>>(w.m, w.h, w.s, w.order, b, r, w.mp);
      est_final_kernel<<<1, 64, 0, s>>>(w.mp, r, w.info, w.info32);
      float est = 0.f;
      if ((e = read_info(w, 0, est, s)) != hipSuccess) return e;
      next_check = k + o.check_every;
      if (prev_k >= 0 && est > o.tol) {
        if (!(est < prev_est) || !(est > 0.f)) {
          next_check = INT32_MAX;
        } else {
          const double rate = std::log((double)est / prev_est) / (k - prev_k);   // < 0
          const double need = std::log((double)o.tol / est) / rate;
          next_check = k + need > (double)o.max_iter ? INT32_MAX : k + std::max(o.check_every, (int)std::ceil(need));
        }
      }
      prev_k = k;
      prev_est = est;
      if (est <= o.tol) {
        // second Cholesky-QR pass of Q, as the last product of the fixed mode gets
        std::swap(w.y, w.q);
        if ((e = orth(w, d, b, 1, s)) != hipSuccess) return e;
        final_product = true;
      }
    }
    if (final_product) {
      if ((e = finish(g, d, b, r, w, rows, ut, ut_dtype, ut_master, eigvals, want_resid, s)) != hipSuccess)
        return e;
      if (o.tol > 0.f) {
        float res = 0.f;
        if ((e = read_info(w, 1, res, s)) != hipSuccess) return e;
        met = res <= o.tol;
        if (!met && adaptive && k < o.max_iter) {
          ++k;
          continue;   // Q (and its fp32 copy) are intact: keep iterating
        }
      }
      break;
    }
    ++k;
  }
  if (report) report_kernel<<<1, 1, 0, s>>>(report, w.info, w.theta, r, k, o.tol);
  return hipGetLastError();
}

hipError_t launch_basis_from_gram(const float* g, int64_t d, int32_t r, int32_t p, const zoact_eig_opts& o, void* ut,
                                  int32_t ut_dtype, float* ut_master, float* eigvals, zoact_eig_report* report, void* ws,
                                  hipStream_t s, bool& met) {
  return solve(g, d, r, p, o, nullptr, ut, ut_dtype, ut_master, eigvals, report, ws, s, met);
}

// Token-side workspace: X X^T [n][n] fp32, the solver's workspace for n rows, then the
// basis and residual blocks [D][r] fp64, the r column norms and the X^T V partials.
size_t basis_rows_ws_bytes(int64_t n, int64_t D, int32_t r, int32_t p) {
  int ks;
  int64_t tchunk;
  xv_split(n, D, r, ks, tchunk);
  return align256((size_t)n * n * 4) + basis_ws_bytes(n, r, p) + 2 * align256((size_t)D * r * 8) +
         align256((size_t)r * 8) + align256((size_t)ks * D * r * 8);
}

// X X^T: with dense rows and n a multiple of 32 (the GEMM's output rows are whole 16-value
// blocks) the plain bf16 GEMM (both halves of X against all of X: the full square), then
// the upper triangle mirrored onto the lower so the matrix is exactly symmetric; otherwise
// the triangle kernel.
hipError_t launch_basis_init_rows(const uint16_t* x, int64_t n, int64_t D, int64_t ld, int32_t r, int32_t p,
                                  const zoact_eig_opts& o, void* ut, int32_t ut_dtype, float* ut_master, float* eigvals,
                                  zoact_eig_report* report, void* ws, hipStream_t s, bool& met) {
  char* pw = static_cast<char*>(ws);
  float* g = reinterpret_cast<float*>(pw);
  pw += align256((size_t)n * n * 4);
  void* sws = pw;
  pw += basis_ws_bytes(n, r, p);
  Rows rows;
  rows.x = x;
  rows.D = D;
  rows.ld = ld;
  xv_split(n, D, r, rows.ks, rows.tchunk);
  rows.up = reinterpret_cast<double*>(pw);
  pw += align256((size_t)D * r * 8);
  rows.yp = reinterpret_cast<double*>(pw);
  pw += align256((size_t)D * r * 8);
  rows.sc = reinterpret_cast<double*>(pw);
  pw += align256((size_t)r * 8);
  rows.part = reinterpret_cast<double*>(pw);
  if (n % 32 == 0 && ld == D) {
    hipError_t e = launch_gemm_nt_f32(x, n / 2, x, n, D, g, s);
    if (e != hipSuccess) return e;
    const int nt = (int)((n + 31) / 32);
    if (nt > 1) mirror_upper_kernel<<<dim3((unsigned)((int64_t)nt * (nt - 1) / 2)), 256, 0, s>>>(g, n, nt);
    mirror_diag_kernel<<<dim3((unsigned)nt), 256, 0, s>>>(g, n);
  } else {
    const int nt = (int)((n + GT - 1) / GT);
    gram_rows_bf16_kernel<<<dim3((unsigned)(nt * (nt + 1) / 2)), 256, 0, s>>>(x, n, D, ld, g, nt);
  }
  return solve(g, n, r, p, o, &rows, ut, ut_dtype, ut_master, eigvals, report, sws, s, met);
}

}  // namespace zoact

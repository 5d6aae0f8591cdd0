// Fused +/- adapted linear and the X U projection prepass.
//
// Section 3 evaluates the perturbed layer without forming W_eff:
//   Y+ = X W + (X V_r)(B + mu Z).
// In the library orientation (W [d_out][d_in], U^T [r][d_in], C = B^T [d_out][r])
// both perturbation signs of a +/- step are computed by one GEMM over the stacked
// batch x [2][T][d_in]:
//   y[h] = x[h] W^T + b + p[h] (C + s_h eps Z)^T,   p[h] = x[h] U,  s = (+1, -1),
// i.e. a single contraction over the extended depth [x[h] | p[h]] . [W ; C_h]^T
// in which the last r columns of the depth belong to the rank-r correction.
//
// gfx950 design (bf16 / INT4 weights):
//  * Workgroup tile: 256 output features x 256 tokens, depth step 64, 512 threads
//    (8 wave64s as 2 along features x 4 along tokens, 128 x 64 per wave), fp32
//    accumulators in registers, v_mfma_f32_16x16x32_bf16.  The MFMA A operand is the
//    W tile (rows = features) and the B operand the x tile (columns = tokens), so
//    each lane ends up holding 4 consecutive features of one token: epilogue
//    stores are 8-byte (bf16) or 16-byte (fp32) vectors along the feature axis.
//  * Tiles live in LDS, double-buffered ([2] x (W tile + x tile) = 128 KB), rows of
//    64 bf16 with the 16-byte chunk index XOR-swizzled by (row & 7) so that the
//    16-byte fragment reads of 8 consecutive lanes hit distinct banks.  Global
//    loads for tile k+1 are issued before the MFMAs of tile k.
//  * A token tile never straddles the two halves: the grid has ceil(T/256) token
//    tiles per half, so each workgroup knows its sign s_h.
//  * The correction block is appended after the depth loop as ceil(r/64) extra
//    depth tiles: the W side is C_h = C + s_h eps Z, formed in fp32 from the arena
//    with Z regenerated from its counter (the same generator as the optimiser
//    step), rounded to bf16; the x side is p[h].  Nothing of Z is stored.
//  * INT4 weights: each thread fetches 16 bytes (32 nibbles of one row) per depth
//    tile and dequantises them in registers to bf16(q * s) before the LDS store.
//  * blockIdx -> tile: workgroups are dispatched round-robin over the 8 XCDs, so
//    the linear id is first regrouped so that each XCD receives a contiguous run of
//    tiles, and runs are ordered in groups of 4 token tiles x all feature tiles to
//    keep both operands L2-resident.
#include <stdlib.h>

#include <mutex>

#include "gemm_common.hpp"

namespace zoact {

namespace {

using namespace gemm;

constexpr int BN = 256;  // features per tile (MFMA rows)
constexpr int BM = 256;  // tokens per tile (MFMA columns)
constexpr int BK = 64;   // depth per tile
constexpr int NTHR = 512;
constexpr int WAVES_N = 2;
constexpr int WAVES_M = 4;
constexpr int WN = BN / WAVES_N;  // 128 features per wave
constexpr int WM = BM / WAVES_M;  // 64 tokens per wave
constexpr int FI = WN / 16;       // 8 MFMA blocks along features
constexpr int FJ = WM / 16;       // 4 MFMA blocks along tokens
constexpr int GROUP_M = 4;

template <bool INT4>
__device__ __forceinline__ void load_main(const GemmArgs& a, int64_t n0, const uint16_t* xh, int64_t m0, int64_t T,
                                          int kt, uint4 (&ws)[4], uint4 (&xs)[4]) {
  const int t = threadIdx.x;
  const int64_t k0 = (int64_t)kt * BK;
  if (INT4) {
    const int row = t >> 1, half = t & 1;
    int64_t n = n0 + row;
    if (n > a.N - 1) n = a.N - 1;
    const uint8_t* wq = reinterpret_cast<const uint8_t*>(a.w);
    const uint4 q = *reinterpret_cast<const uint4*>(wq + n * (a.K >> 1) + ((k0 + half * 32) >> 1));
    const float s = bf2f(a.wsc[n * (a.K >> 7) + ((k0 + half * 32) >> 7)]);
    ws[0] = dequant8(q.x, s);
    ws[1] = dequant8(q.y, s);
    ws[2] = dequant8(q.z, s);
    ws[3] = dequant8(q.w, s);
  } else {
    const uint16_t* w = reinterpret_cast<const uint16_t*>(a.w);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = t + NTHR * i;
      const int row = c >> 3, kc = c & 7;
      int64_t n = n0 + row;
      if (n > a.N - 1) n = a.N - 1;
      ws[i] = *reinterpret_cast<const uint4*>(w + n * a.K + k0 + kc * 8);
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = t + NTHR * i;
    const int row = c >> 3, kc = c & 7;
    int64_t m = m0 + row;
    if (m > T - 1) m = T - 1;
    xs[i] = *reinterpret_cast<const uint4*>(xh + m * a.K + k0 + kc * 8);
  }
}

template <bool INT4>
__device__ __forceinline__ void store_main(uint16_t* wl, uint16_t* xl, const uint4 (&ws)[4], const uint4 (&xs)[4]) {
  const int t = threadIdx.x;
  if (INT4) {
    const int row = t >> 1, half = t & 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) *reinterpret_cast<uint4*>(wl + swz(row, half * 4 + i)) = ws[i];
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = t + NTHR * i;
      *reinterpret_cast<uint4*>(wl + swz(c >> 3, c & 7)) = ws[i];
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = t + NTHR * i;
    *reinterpret_cast<uint4*>(xl + swz(c >> 3, c & 7)) = xs[i];
  }
}

// Correction-block tile `tt`: W side = bf16(C + s eps Z) for coefficient columns
// tt*64 .. tt*64+63 of each feature row, x side = p[h] for the same columns.
__device__ __forceinline__ void load_tail(const GemmArgs& a, int64_t n0, const uint16_t* ph, int64_t m0, int64_t T,
                                          int hf, int tt, uint4 (&ws)[4], uint4 (&xs)[4]) {
  const int t = threadIdx.x;
  const int row = t >> 1, half = t & 1;
  const int col0 = tt * 64 + half * 32;
  const int64_t n = n0 + row;
  const int64_t m = m0 + row;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint16_t wv[8], xv[8];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int col = col0 + i * 8 + g * 4;
      float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
      float cv[4] = {0.f, 0.f, 0.f, 0.f};
      const bool any = (n < a.N) && (col < a.r);
      if (any) {
        const uint64_t e = (uint64_t)(a.coef_offset + n * a.r + col);
        z = gauss4(a.seed, a.step, a.query_h[hf], e);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (col + j < a.r)
            cv[j] = a.c_bf16 ? bf2f(reinterpret_cast<const uint16_t*>(a.c)[e + j])
                             : reinterpret_cast<const float*>(a.c)[e + j];
        }
      }
      const float zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool ok = any && (col + j < a.r);
        wv[g * 4 + j] = ok ? perturbed_bf16(cv[j], zz[j], a.eps, a.sign_h[hf]) : (uint16_t)0;
        xv[g * 4 + j] = (col + j < a.r && m < T) ? ph[m * a.r + col + j] : (uint16_t)0;
      }
    }
    ws[i] = make_uint4(pack2(wv[0], wv[1]), pack2(wv[2], wv[3]), pack2(wv[4], wv[5]), pack2(wv[6], wv[7]));
    xs[i] = make_uint4(pack2(xv[0], xv[1]), pack2(xv[2], xv[3]), pack2(xv[4], xv[5]), pack2(xv[6], xv[7]));
  }
}

__device__ __forceinline__ void store_tail(uint16_t* wl, uint16_t* xl, const uint4 (&ws)[4], const uint4 (&xs)[4]) {
  const int t = threadIdx.x;
  const int row = t >> 1, half = t & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    *reinterpret_cast<uint4*>(wl + swz(row, half * 4 + i)) = ws[i];
    *reinterpret_cast<uint4*>(xl + swz(row, half * 4 + i)) = xs[i];
  }
}

__device__ __forceinline__ void mfma_tile(const uint16_t* wl, const uint16_t* xl, int wn0, int wm0, int ksteps,
                                          floatx4 (&acc)[FI][FJ]) {
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  for (int ks = 0; ks < ksteps; ++ks) {
    bf16x8 af[FI], bfr[FJ];
#pragma unroll
    for (int i = 0; i < FI; ++i) {
      const int row = wn0 + i * 16 + lr;
      af[i] = *reinterpret_cast<const bf16x8*>(wl + swz(row, ks * 4 + lk));
    }
#pragma unroll
    for (int j = 0; j < FJ; ++j) {
      const int row = wm0 + j * 16 + lr;
      bfr[j] = *reinterpret_cast<const bf16x8*>(xl + swz(row, ks * 4 + lk));
    }
#pragma unroll
    for (int i = 0; i < FI; ++i)
#pragma unroll
      for (int j = 0; j < FJ; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
  }
}


template <bool INT4, int EPI, bool OUT_F32>
__global__ void __launch_bounds__(NTHR, 1) gemm_pm_kernel(GemmArgs a) {
  extern __shared__ __align__(16) uint16_t lds[];
  // LDS: W tiles [2][BN][BK] then x tiles [2][BM][BK]
#define WL(buf) (lds + (buf) * (BN * BK))
#define XL(buf) (lds + 2 * BN * BK + (buf) * (BM * BK))

  // ---- tile assignment (XCD-contiguous runs, grouped token-major order)
  const int ntiles = gridDim.x;
  int lin = blockIdx.x;
  if ((ntiles & 7) == 0) lin = (blockIdx.x & 7) * (ntiles >> 3) + (blockIdx.x >> 3);
  const int tiles_m = 2 * a.tiles_m_half;
  const int per_group = GROUP_M * a.tiles_n;
  const int grp = lin / per_group;
  const int first_m = grp * GROUP_M;
  const int gsz = min(GROUP_M, tiles_m - first_m);
  const int tm = first_m + (lin % per_group) % gsz;
  const int tn = (lin % per_group) / gsz;
  const int half = tm / a.tiles_m_half;
  const int64_t m0 = (int64_t)(tm % a.tiles_m_half) * BM;
  const int64_t n0 = (int64_t)tn * BN;
  const uint16_t* xh = a.x + (int64_t)half * a.T * a.K;
  const uint16_t* ph = a.p ? a.p + (int64_t)half * a.T * a.r : nullptr;

  const int wave = threadIdx.x >> 6;
  const int wn0 = (wave % WAVES_N) * WN;
  const int wm0 = (wave / WAVES_N) * WM;

  floatx4 acc[FI][FJ];
#pragma unroll
  for (int i = 0; i < FI; ++i)
#pragma unroll
    for (int j = 0; j < FJ; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  const int nk = (int)(a.K / BK);
  uint4 ws[4], xs[4];
  load_main<INT4>(a, n0, xh, m0, a.T, 0, ws, xs);
  store_main<INT4>(WL(0), XL(0), ws, xs);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int nxt = kt + 1;
    if (nxt < nk) load_main<INT4>(a, n0, xh, m0, a.T, nxt, ws, xs);
    mfma_tile(WL(kt & 1), XL(kt & 1), wn0, wm0, 2, acc);
    if (nxt < nk) store_main<INT4>(WL(nxt & 1), XL(nxt & 1), ws, xs);
    __syncthreads();
  }
  // correction block: [p[h] | C + s eps Z], 64 coefficient columns per tile
  for (int tt = 0; tt < a.n_tail; ++tt) {
    load_tail(a, n0, ph, m0, a.T, half, tt, ws, xs);
    store_tail(WL(tt & 1), XL(tt & 1), ws, xs);
    __syncthreads();
    const int rem = a.r - tt * 64;
    mfma_tile(WL(tt & 1), XL(tt & 1), wn0, wm0, rem >= 64 ? 2 : (rem + 31) / 32, acc);
  }

#undef WL
#undef XL
  // ---- epilogue: bias, residual, activation, one rounding, vector stores
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t nout = (EPI == ZOACT_EPI_SWIGLU) ? a.N / 2 : a.N;
#pragma unroll
  for (int j = 0; j < FJ; ++j) {
    const int64_t m = m0 + wm0 + j * 16 + lr;
    if (m >= a.T) continue;
    const int64_t row = (int64_t)half * a.T + m;
    if (EPI == ZOACT_EPI_SWIGLU) {
#pragma unroll
      for (int i = 0; i < FI; i += 2) {
        const int64_t ng = n0 + wn0 + i * 16 + lk * 4;  // fused gate row
        if (ng >= a.N) continue;
        const int64_t f = (ng >> 5) * 16 + (ng & 31);  // output feature
        float o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float g = acc[i][j][q], u = acc[i + 1][j][q];
          if (a.bias) {
            g += bf2f(a.bias[ng + q]);
            u += bf2f(a.bias[ng + 16 + q]);
          }
          o[q] = silu(g) * u;
        }
        if (a.resid) {
          const ushort4 rv = *reinterpret_cast<const ushort4*>(a.resid + row * nout + f);
          o[0] += bf2f(rv.x); o[1] += bf2f(rv.y); o[2] += bf2f(rv.z); o[3] += bf2f(rv.w);
        }
        if (OUT_F32) *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.y) + row * nout + f) = make_float4(o[0], o[1], o[2], o[3]);
        else *reinterpret_cast<ushort4*>(reinterpret_cast<uint16_t*>(a.y) + row * nout + f) = make_ushort4(f2bf(o[0]), f2bf(o[1]), f2bf(o[2]), f2bf(o[3]));
      }
    } else {
#pragma unroll
      for (int i = 0; i < FI; ++i) {
        const int64_t n = n0 + wn0 + i * 16 + lk * 4;
        if (n >= a.N) continue;
        float o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          o[q] = acc[i][j][q];
          if (a.bias) o[q] += bf2f(a.bias[n + q]);
        }
        if (a.resid) {
          const ushort4 rv = *reinterpret_cast<const ushort4*>(a.resid + row * nout + n);
          o[0] += bf2f(rv.x); o[1] += bf2f(rv.y); o[2] += bf2f(rv.z); o[3] += bf2f(rv.w);
        }
        if (EPI == ZOACT_EPI_RELU) {
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = fmaxf(o[q], 0.0f);
        }
        if (OUT_F32) *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.y) + row * nout + n) = make_float4(o[0], o[1], o[2], o[3]);
        else *reinterpret_cast<ushort4*>(reinterpret_cast<uint16_t*>(a.y) + row * nout + n) = make_ushort4(f2bf(o[0]), f2bf(o[1]), f2bf(o[2]), f2bf(o[3]));
      }
    }
  }
}

// ------------------------------------------------------------------ fp32 path
// Plain fp32 SIMT tile (64 x 64 outputs, 256 threads, 4 x 4 per thread) for the
// fp32 mode of small models; the correction block is appended as extra depth.
struct GemmArgsF32 {
  const float* x;
  const float* w;
  const float* bias;
  const float* p;
  const float* c;
  const float* resid;
  float* y;
  int64_t T, N, K;
  int32_t r;
  int64_t coef_offset;
  uint64_t seed;
  uint32_t step;
  uint32_t query_h[2];
  int32_t sign_h[2];
  float eps;
  int32_t tiles_m_half;
};

// Column q of thread tx covers tile feature (tx/8)*32 + (tx%8)*2 + (q&1) + (q>>1)*16,
// so each thread holds a gate row (q = 0, 1) and the up row 16 later (q = 2, 3) of the
// interleaved gate|up layout.
__device__ __forceinline__ int f32_col(int tx, int q) { return (tx >> 3) * 32 + (tx & 7) * 2 + (q & 1) + (q >> 1) * 16; }

template <int EPI>
__global__ void __launch_bounds__(256) gemm_pm_f32_kernel(GemmArgsF32 a) {
  __shared__ float xs[16][65];
  __shared__ float wsh[16][65];
  const int tm = blockIdx.y;
  const int half = tm / a.tiles_m_half;
  const int64_t m0 = (int64_t)(tm % a.tiles_m_half) * 64;
  const int64_t n0 = (int64_t)blockIdx.x * 64;
  const float* xh = a.x + (int64_t)half * a.T * a.K;
  const float* ph = a.p ? a.p + (int64_t)half * a.T * a.r : nullptr;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  const int64_t ktot = a.K + a.r;
  for (int64_t k0 = 0; k0 < ktot; k0 += 16) {
    for (int i = threadIdx.x; i < 16 * 64; i += 256) {
      const int kk = i & 15, rr = i >> 4;
      const int64_t k = k0 + kk;
      const int64_t m = m0 + rr, n = n0 + rr;
      float xv = 0.f, wv = 0.f;
      if (k < a.K) {
        if (m < a.T) xv = xh[m * a.K + k];
        if (n < a.N) wv = a.w[n * a.K + k];
      } else if (k < ktot) {
        const int64_t i2 = k - a.K;
        if (m < a.T) xv = ph[m * a.r + i2];
        if (n < a.N) {
#pragma clang fp contract(off)
          const int64_t e = a.coef_offset + n * a.r + i2;
          const float z = rng::gauss_at(a.seed, a.step, a.query_h[half], (uint64_t)e);
          const float ez = a.eps * z;
          const int sg = a.sign_h[half];
          wv = sg > 0 ? a.c[e] + ez : (sg < 0 ? a.c[e] - ez : a.c[e]);
        }
      }
      xs[kk][rr] = xv;
      wsh[kk][rr] = wv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float xr[4], wr[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        xr[q] = xs[kk][ty * 4 + q];
        wr[q] = wsh[kk][f32_col(tx, q)];
      }
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[p][q] += xr[p] * wr[q];
    }
    __syncthreads();
  }
  const int64_t nout = (EPI == ZOACT_EPI_SWIGLU) ? a.N / 2 : a.N;
  for (int p = 0; p < 4; ++p) {
    const int64_t m = m0 + ty * 4 + p;
    if (m >= a.T) continue;
    const int64_t row = (int64_t)half * a.T + m;
    if (EPI == ZOACT_EPI_SWIGLU) {
      for (int q = 0; q < 2; ++q) {
        const int64_t ng = n0 + f32_col(tx, q);
        if (ng >= a.N) continue;
        const float g = acc[p][q] + (a.bias ? a.bias[ng] : 0.f);
        const float u = acc[p][q + 2] + (a.bias ? a.bias[ng + 16] : 0.f);
        const int64_t f = (ng >> 5) * 16 + (ng & 31);
        float o = (g / (1.0f + __expf(-g))) * u;
        if (a.resid) o += a.resid[row * nout + f];
        a.y[row * nout + f] = o;
      }
    } else {
      for (int q = 0; q < 4; ++q) {
        const int64_t n = n0 + f32_col(tx, q);
        if (n >= a.N) continue;
        float o = acc[p][q] + (a.bias ? a.bias[n] : 0.f);
        if (a.resid) o += a.resid[row * nout + n];
        if (EPI == ZOACT_EPI_RELU) o = fmaxf(o, 0.f);
        a.y[row * nout + n] = o;
      }
    }
  }
}

// ------------------------------------------------------------------ projection
// p = x U for x [n_tok][d_in], U^T [r][d_in]: HBM-bound (r FLOP per byte of x), so the
// design goal is to keep enough of x in flight.  A workgroup owns 16 TB tokens and splits
// the depth over its 4 waves; each wave reads its x fragments straight from global memory
// and its U^T fragments from L2 (16 bytes per lane per 32-deep step, the next 128-deep
// step's loads issued before this step's MFMAs), runs v_mfma_f32_16x16x32_bf16 into fp32
// partials, and the 4 partials are summed in a fixed order through LDS before the single
// rounding to bf16.

template <int RB, int TB>
__global__ void __launch_bounds__(256) project_bf16_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ ut,
                                                          uint16_t* __restrict__ p, int64_t n_tok, int64_t d, int r,
                                                          int64_t dq) {
  constexpr int PROJ_TOK = 16 * TB;
  __shared__ float part[4][PROJ_TOK][RB * 16 + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * PROJ_TOK;
  const int lr = lane & 15, lk = lane >> 4;
  floatx4 acc[TB][RB];
#pragma unroll
  for (int i = 0; i < TB; ++i)
#pragma unroll
    for (int j = 0; j < RB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* xr[TB];
#pragma unroll
  for (int i = 0; i < TB; ++i) {
    int64_t t = t0 + i * 16 + lr;
    t = t < n_tok ? t : n_tok - 1;
    xr[i] = x + t * d + lk * 8;
  }
  const bf16x8 zero8 = {};
  const int64_t k_begin = (int64_t)wave * dq, k_end = k_begin + dq < d ? k_begin + dq : d;
  // the x and U^T chunks of the next 128-deep step are loaded while this step's MFMAs run
  // (the pass is bound by the bytes each wave keeps in flight; U^T comes from L2); with
  // r > 64 the U^T chunks are loaded step by step instead
  constexpr bool PRE_B = RB <= 4;
  bf16x8 a[4][TB], an[4][TB];
  bf16x8 bq[PRE_B ? 4 : 1][PRE_B ? RB : 1], bn[PRE_B ? 4 : 1][PRE_B ? RB : 1];
  auto load_b = [&](int64_t k, int u, int j) -> bf16x8 {
    const int rc = j * 16 + lr;
    return (rc < r && k + u * 32 < k_end) ? *reinterpret_cast<const bf16x8*>(ut + (int64_t)rc * d + k + u * 32 + lk * 8)
                                         : zero8;
  };
  auto load_ab = [&](int64_t k) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int i = 0; i < TB; ++i)
        an[u][i] = (k + u * 32 < k_end) ? *reinterpret_cast<const bf16x8*>(xr[i] + k + u * 32) : zero8;
      if constexpr (PRE_B) {
#pragma unroll
        for (int j = 0; j < RB; ++j) bn[u][j] = load_b(k, u, j);
      }
    }
  };
  if (k_begin < k_end) load_ab(k_begin);
  for (int64_t k = k_begin; k < k_end; k += 128) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int i = 0; i < TB; ++i) a[u][i] = an[u][i];
      if constexpr (PRE_B) {
#pragma unroll
        for (int j = 0; j < RB; ++j) bq[u][j] = bn[u][j];
      }
    }
    if (k + 128 < k_end) load_ab(k + 128);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (k + u * 32 < k_end) {
        bf16x8 b[RB];
#pragma unroll
        for (int j = 0; j < RB; ++j) {
          if constexpr (PRE_B) b[j] = bq[u][j];
          else b[j] = load_b(k, u, j);
        }
#pragma unroll
        for (int i = 0; i < TB; ++i)
#pragma unroll
          for (int j = 0; j < RB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][i], b[j], acc[i][j], 0, 0, 0);
      }
    }
  }
  // D[token = 4*lk + q][col = lr] of each 16 x 16 block -> LDS partials
#pragma unroll
  for (int i = 0; i < TB; ++i)
#pragma unroll
    for (int j = 0; j < RB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) part[wave][i * 16 + lk * 4 + q][j * 16 + lr] = acc[i][j][q];
  __syncthreads();
  for (int e = threadIdx.x; e < PROJ_TOK * RB * 16; e += 256) {
    const int tl = e / (RB * 16), col = e % (RB * 16);
    const int64_t t = t0 + tl;
    if (t < n_tok && col < r) {
      const float v = ((part[0][tl][col] + part[1][tl][col]) + part[2][tl][col]) + part[3][tl][col];
      p[t * r + col] = f2bf(v);
    }
  }
}

// The same product as a software pipeline for a fixed depth share: each wave walks its NS
// 32-deep steps fully unrolled (straight-line code, so every wait on the loads is exact)
// with the loads of the next PF - 1 steps in flight, through buffer descriptors (U^T rows
// past r read 0 from the descriptor's bound; x rows past n_tok repeat the last row, not
// stored).  Same summation as project_bf16_kernel's: fp32 per wave in depth order, waves
// added in a fixed order.
template <int RB, int TB, int PF, int NS>
__global__ void __launch_bounds__(256) project_pipe_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ ut,
                                                           uint16_t* __restrict__ p, int64_t n_tok, int64_t d, int r) {
  constexpr int PROJ_TOK = 16 * TB;
  __shared__ float part[4][PROJ_TOK][RB * 16 + 1];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t t0 = (int64_t)blockIdx.x * PROJ_TOK;
  const int lr = lane & 15, lk = lane >> 4;
  const __amdgpu_buffer_rsrc_t xrs = gemm::buffer_rsrc(x, (uint32_t)(n_tok * d * 2));
  const __amdgpu_buffer_rsrc_t urs = gemm::buffer_rsrc(ut, (uint32_t)((int64_t)r * d * 2));
  int xo[TB], uo[RB];
#pragma unroll
  for (int i = 0; i < TB; ++i) {
    int64_t t = t0 + i * 16 + lr;
    t = t < n_tok ? t : n_tok - 1;
    xo[i] = (int)((t * d + lk * 8) * 2);
  }
#pragma unroll
  for (int j = 0; j < RB; ++j) uo[j] = (int)(((int64_t)(j * 16 + lr) * d + lk * 8) * 2);
  const int kb = wave * NS * 32 * 2;   // byte offset of this wave's share
  floatx4 acc[TB][RB];
#pragma unroll
  for (int i = 0; i < TB; ++i)
#pragma unroll
    for (int j = 0; j < RB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  bf16x8 xa[PF][TB], ub[PF][RB];
  auto load = [&](int st) {
    const int buf = st % PF, ko = kb + st * 64;
#pragma unroll
    for (int i = 0; i < TB; ++i)
      xa[buf][i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(xrs, xo[i], ko, 0));
#pragma unroll
    for (int j = 0; j < RB; ++j)
      ub[buf][j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(urs, uo[j], ko, 0));
  };
  // (scheduling barriers keep each step's loads PF - 1 steps ahead of its use: left alone,
  // the compiler moves them next to their use)
#pragma unroll
  for (int st = 0; st < PF - 1; ++st) load(st);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int st = 0; st < NS; ++st) {
    if (st + PF - 1 < NS) load(st + PF - 1);
#pragma unroll
    for (int i = 0; i < TB; ++i)
#pragma unroll
      for (int j = 0; j < RB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xa[st % PF][i], ub[st % PF][j], acc[i][j], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int i = 0; i < TB; ++i)
#pragma unroll
    for (int j = 0; j < RB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) part[wave][i * 16 + lk * 4 + q][j * 16 + lr] = acc[i][j][q];
  __syncthreads();
  for (int e = threadIdx.x; e < PROJ_TOK * RB * 16; e += 256) {
    const int tl = e / (RB * 16), col = e % (RB * 16);
    const int64_t t = t0 + tl;
    if (t < n_tok && col < r) {
      const float v = ((part[0][tl][col] + part[1][tl][col]) + part[2][tl][col]) + part[3][tl][col];
      p[t * r + col] = f2bf(v);
    }
  }
}

// The same product with the depth also split over workgroups (workspace form): workgroup
// (b, s) owns 16 TB tokens and depth chunk s of S, its 4 waves splitting the chunk further
// (64-deep steps, the next step's x and U^T fragments in flight).  More tokens per
// workgroup than above means fewer U^T bytes per x byte (r / (16 TB) instead of r / 32).
// Each workgroup writes its fp32 partial [16 TB][r] (waves summed in a fixed order) to
// part[s]; a second pass adds the S partials in the order s = 0 .. S - 1 and rounds once
// to bf16.  (Letting the last workgroup of a token block do the sum needs a device-scope
// release per workgroup, which on this GPU writes back the XCD's L2: it measured four
// times slower than the second launch.)
template <int RB, int TB>
__global__ void __launch_bounds__(256) project_split_kernel(const uint16_t* __restrict__ x,
                                                            const uint16_t* __restrict__ ut, uint16_t* __restrict__ p,
                                                            int64_t n_tok, int64_t d, int r, int64_t chunk,
                                                            float* __restrict__ part) {
  constexpr int TOK = 16 * TB, NC = RB * 16;
  __shared__ float red[4][TOK][NC + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t t0 = (int64_t)blockIdx.x * TOK;
  const int sp = blockIdx.y;
  floatx4 acc[TB][RB];
#pragma unroll
  for (int i = 0; i < TB; ++i)
#pragma unroll
    for (int j = 0; j < RB; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* xr[TB];
#pragma unroll
  for (int i = 0; i < TB; ++i) {
    int64_t t = t0 + i * 16 + lr;
    t = t < n_tok ? t : n_tok - 1;
    xr[i] = x + t * d + lk * 8;
  }
  const bf16x8 zero8 = {};
  // this wave's depth range: a quarter of the chunk, a multiple of 32
  const int64_t c0 = (int64_t)sp * chunk, c1 = c0 + chunk < d ? c0 + chunk : d;
  int64_t wq = (chunk + 3) / 4;
  wq = (wq + 31) / 32 * 32;
  const int64_t k_begin = c0 + wave * wq, k_end = k_begin + wq < c1 ? k_begin + wq : c1;
  bf16x8 a[2][TB], an[2][TB], bq[2][RB], bn[2][RB];
  auto load = [&](int64_t k) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const bool in = k + u * 32 < k_end;
#pragma unroll
      for (int i = 0; i < TB; ++i) an[u][i] = in ? *reinterpret_cast<const bf16x8*>(xr[i] + k + u * 32) : zero8;
#pragma unroll
      for (int j = 0; j < RB; ++j) {
        const int rc = j * 16 + lr;
        bn[u][j] = (in && rc < r) ? *reinterpret_cast<const bf16x8*>(ut + (int64_t)rc * d + k + u * 32 + lk * 8) : zero8;
      }
    }
  };
  if (k_begin < k_end) load(k_begin);
  for (int64_t k = k_begin; k < k_end; k += 64) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
#pragma unroll
      for (int i = 0; i < TB; ++i) a[u][i] = an[u][i];
#pragma unroll
      for (int j = 0; j < RB; ++j) bq[u][j] = bn[u][j];
    }
    if (k + 64 < k_end) load(k + 64);
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int i = 0; i < TB; ++i)
#pragma unroll
        for (int j = 0; j < RB; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][i], bq[u][j], acc[i][j], 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < TB; ++i)
#pragma unroll
    for (int j = 0; j < RB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) red[wave][i * 16 + lk * 4 + q][j * 16 + lr] = acc[i][j][q];
  __syncthreads();
  // this workgroup's partial: waves summed in order
  float* mine = part + ((int64_t)sp * n_tok + t0) * r;
  for (int e = threadIdx.x; e < TOK * NC; e += 256) {
    const int tl = e / NC, col = e % NC;
    if (t0 + tl < n_tok && col < r)
      mine[(int64_t)tl * r + col] = ((red[0][tl][col] + red[1][tl][col]) + red[2][tl][col]) + red[3][tl][col];
  }
}

// p = bf16(part[0] + part[1] + ... + part[S - 1]), in that order, 4 outputs per thread.
__global__ void __launch_bounds__(256) project_sum_kernel(const float* __restrict__ part, int nsplit, int64_t n,
                                                          uint16_t* __restrict__ p, int vec) {
  const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i >= n) return;
  if (vec) {   // n % 4 == 0, p 8-byte aligned
    float4 v = *reinterpret_cast<const float4*>(part + i);
    for (int q = 1; q < nsplit; ++q) {
      const float4 w = *reinterpret_cast<const float4*>(part + (int64_t)q * n + i);
      v.x += w.x, v.y += w.y, v.z += w.z, v.w += w.w;
    }
    *reinterpret_cast<uint2*>(p + i) = make_uint2(pack2(f2bf(v.x), f2bf(v.y)), pack2(f2bf(v.z), f2bf(v.w)));
  } else {
    for (int64_t e = i; e < i + 4 && e < n; ++e) {
      float v = part[e];
      for (int q = 1; q < nsplit; ++q) v += part[(int64_t)q * n + e];
      p[e] = f2bf(v);
    }
  }
}

__global__ void project_f32_kernel(const float* x, const float* ut, float* p, int64_t n_tok, int64_t d, int r) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_tok * r; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = i / r;
    const int c = (int)(i % r);
    float s = 0.f;
    for (int64_t k = 0; k < d; ++k) s += x[t * d + k] * ut[(int64_t)c * d + k];
    p[i] = s;
  }
}

template <bool INT4, int EPI, bool OUT_F32>
hipError_t launch_bf16(const GemmArgs& a, dim3 grid, hipStream_t s) {
  const size_t lds = (size_t)2 * (BN + BM) * BK * sizeof(uint16_t);
  static bool attr_set = false;  // benign race: every thread sets the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_pm_kernel<INT4, EPI, OUT_F32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  gemm_pm_kernel<INT4, EPI, OUT_F32><<<grid, dim3(NTHR), lds, s>>>(a);
  return hipGetLastError();
}

// INT4 weights to bf16 in one streaming pass (the values the INT4 GEMMs form in registers
// or LDS).
__global__ void __launch_bounds__(256) dequant_int4_kernel(const uint32_t* __restrict__ w, const uint16_t* __restrict__ sc,
                                                           int64_t n_units, int64_t units_per_row, int64_t groups,
                                                           uint4* __restrict__ out) {
  // unit = 8 weights of one row (4 packed bytes -> 16 bytes of bf16); consecutive lanes
  // take consecutive units, so every load and store instruction is contiguous, one unit per
  // thread and pass of the grid-stride loop (gate|up 4096 x 28672: 49 us; four units a
  // thread in flight: 57 us; 64 bytes per thread as four 16-byte stores 64 bytes apart:
  // 3.0-3.6 TB/s)
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < n_units; u += stride) {
    const int64_t row = u / units_per_row, cu = u % units_per_row;
    const uint32_t q = __builtin_nontemporal_load(w + u);
    out[u] = dequant8(q, bf2f(sc[row * groups + (cu >> 4)]));
  }
}

}  // namespace

hipError_t launch_linear_pm_4w(const gemm::GemmArgs& a, int w_dtype, int epi, bool out_f32, hipStream_t s);
hipError_t launch_linear_pm_4w64(const gemm::GemmArgs& a, int w_dtype, int epi, bool out_f32, bool shared,
                                 hipStream_t s);

// Arguments of the bf16-activation kernels for one call.
static GemmArgs bf16_args(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T, const void* p,
                   const void* residual, const zoact_pert_pair& pert, void* y) {
  GemmArgs a{};
  a.x = static_cast<const uint16_t*>(x);
  a.w = L.w;
  a.wsc = static_cast<const uint16_t*>(L.w_scales);
  a.bias = static_cast<const uint16_t*>(L.bias);
  a.p = static_cast<const uint16_t*>(p);
  a.c = (L.r > 0 && A) ? A->c : nullptr;
  a.resid = static_cast<const uint16_t*>(residual);
  a.y = y;
  a.T = T;
  a.N = L.d_out;
  a.K = L.d_in;
  a.r = L.r;
  a.c_bf16 = (A && A->c_dtype == ZOACT_BF16) ? 1 : 0;
  a.coef_offset = L.coef_offset;
  a.seed = pert.seed;
  a.step = pert.step;
  for (int h = 0; h < 2; ++h) a.query_h[h] = pert.query[h], a.sign_h[h] = pert.sign[h];
  a.eps = pert.eps;
  a.tiles_m_half = (int32_t)((T + BM - 1) / BM);
  a.tiles_n = (int32_t)((L.d_out + BN - 1) / BN);
  a.n_tail = (L.r + 63) / 64;
  a.ch = static_cast<const uint16_t*>(L.ch);
  a.ch_stride = L.ch_half_stride;
  if (L.r > 0) {
    a.plain_begin = L.plain_begin;
    a.plain_end = L.plain_end;
  }
  a.tail_ws = static_cast<float*>(L.ws);
  a.tail_ws_bytes = L.ws ? (int64_t)L.ws_bytes : 0;
  return a;
}

hipError_t launch_linear_pm(const zoact_linear& L, const zoact_arena* A, const void* x, int32_t x_dtype, int64_t T,
                            const void* p, const void* residual, uint32_t flags, const zoact_pert_pair& pert, void* y,
                            int32_t y_dtype, hipStream_t s) {
  const int epi = (flags & ZOACT_EPI_SWIGLU) ? ZOACT_EPI_SWIGLU : (flags & ZOACT_EPI_RELU) ? ZOACT_EPI_RELU : 0;
  if (x_dtype == ZOACT_F32) {
    if (L.r > 0 && L.plain_end > L.plain_begin) return hipErrorNotSupported;
    GemmArgsF32 a{};
    a.x = static_cast<const float*>(x);
    a.w = static_cast<const float*>(L.w);
    a.bias = static_cast<const float*>(L.bias);
    a.p = static_cast<const float*>(p);
    a.c = (L.r > 0) ? static_cast<const float*>(A->c) : nullptr;
    a.T = T;
    a.N = L.d_out;
    a.K = L.d_in;
    a.r = L.r;
    a.coef_offset = L.coef_offset;
    a.seed = pert.seed;
    a.step = pert.step;
    for (int h = 0; h < 2; ++h) a.query_h[h] = pert.query[h], a.sign_h[h] = pert.sign[h];
    a.eps = pert.eps;
    a.tiles_m_half = (int32_t)((T + 63) / 64);
    dim3 grid((unsigned)((L.d_out + 63) / 64), (unsigned)(2 * a.tiles_m_half));
    a.resid = static_cast<const float*>(residual);
    a.y = static_cast<float*>(y);
    if (epi == ZOACT_EPI_SWIGLU) gemm_pm_f32_kernel<ZOACT_EPI_SWIGLU><<<grid, dim3(256), 0, s>>>(a);
    else if (epi == ZOACT_EPI_RELU) gemm_pm_f32_kernel<ZOACT_EPI_RELU><<<grid, dim3(256), 0, s>>>(a);
    else gemm_pm_f32_kernel<0><<<grid, dim3(256), 0, s>>>(a);
    return hipGetLastError();
  }

  GemmArgs a = bf16_args(L, A, x, T, p, residual, pert, y);
  const dim3 grid((unsigned)(2 * a.tiles_m_half * a.tiles_n));
  const bool i4 = L.w_dtype == ZOACT_INT4_G128;
  const bool of = y_dtype == ZOACT_F32;
  // one half's x and p read by both halves: the 64-deep schedule's shared-input form only
  if (flags & ZOACT_SHARED_X) return launch_linear_pm_4w64(a, L.w_dtype, epi, of, true, s);
  // a plain feature range: the 64-deep schedule only
  if (a.plain_end > a.plain_begin) return launch_linear_pm_4w64(a, L.w_dtype, epi, of, false, s);
  // the 64-deep persistent schedule where it applies (bf16 weights, C_h precomputed or
  // r = 0), else the 32-deep one (C_h formed in its prologue; INT4 in registers), else the
  // generic kernel (shapes outside both)
  hipError_t e = launch_linear_pm_4w64(a, L.w_dtype, epi, of, false, s);
  if (e != hipErrorNotSupported) return e;
  e = launch_linear_pm_4w(a, L.w_dtype, epi, of, s);
  if (e != hipErrorNotSupported) return e;
#define ZO_DISPATCH(I4, EP, OF) \
  if (i4 == I4 && epi == EP && of == OF) return launch_bf16<I4, EP, OF>(a, grid, s);
  ZO_DISPATCH(false, 0, false)
  ZO_DISPATCH(false, 0, true)
  ZO_DISPATCH(false, ZOACT_EPI_SWIGLU, false)
  ZO_DISPATCH(false, ZOACT_EPI_RELU, false)
  ZO_DISPATCH(true, 0, false)
  ZO_DISPATCH(true, 0, true)
  ZO_DISPATCH(true, ZOACT_EPI_SWIGLU, false)
  ZO_DISPATCH(true, ZOACT_EPI_RELU, false)
#undef ZO_DISPATCH
  return hipErrorNotSupported;
}

// y [2 T][N] fp32 = x [2 T][K] w^T for bf16 x and w [N][K] (rows dense), through the
// adapted-linear launch with r = 0 and no perturbation: the library's plain bf16 GEMM.
hipError_t launch_gemm_nt_f32(const uint16_t* x, int64_t T, const uint16_t* w, int64_t N, int64_t K, float* y,
                              hipStream_t s) {
  zoact_linear L{};
  L.w_dtype = ZOACT_BF16;
  L.w = w;
  L.d_in = K;
  L.d_out = N;
  zoact_pert_pair pert{};
  return launch_linear_pm(L, nullptr, x, ZOACT_BF16, T, nullptr, nullptr, 0, pert, y, ZOACT_F32, s);
}

hipError_t launch_linear_mse(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T, uint32_t flags,
                             const void* p, const zoact_pert_pair& pert, const void* target, double* part,
                             float* loss_pm, hipStream_t s) {
  GemmArgs a = bf16_args(L, A, x, T, p, nullptr, pert, nullptr);
  a.tgt = static_cast<const uint16_t*>(target);
  a.part = part;
  const bool shared = (flags & ZOACT_SHARED_X) != 0;
  hipError_t e = launch_linear_pm_4w64(a, L.w_dtype, EPI_MSE, false, shared, s);
  if (e == hipErrorNotSupported && !shared && a.plain_end == a.plain_begin)
    e = launch_linear_pm_4w(a, L.w_dtype, EPI_MSE, false, s);
  if (e != hipSuccess) return e;
  return launch_sum_mean(part, (int64_t)a.tiles_m_half * a.tiles_n * 4, (double)T * (double)L.d_out, loss_pm, s);
}

// Partial sums of the no-allocation regression-loss call: one array per GPU the library
// runs on, kept until the process ends.  Host code never passes `scratch` itself to a
// kernel (on the host it is only a stand-in for the symbol); it uses the device address
// that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) double scratch[ZOACT_MSE_SCRATCH_BYTES / sizeof(double)];

// Device address of `scratch` on the current device, looked up once per device with that
// device current and kept; nullptr (and *err set) if the lookup fails.
static void* mse_scratch_ptr(hipError_t* err) {
  static std::mutex mu;
  static void* addr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= 64) {
    *err = e != hipSuccess ? e : hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr) {
      *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    addr[dev] = ptr;
  }
  *err = hipSuccess;
  return addr[dev];
}

hipError_t launch_linear_mse_noalloc(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T,
                                     uint32_t flags, const void* p, const zoact_pert_pair& pert, const void* target,
                                     float* loss_pm, hipStream_t s) {
  hipError_t e = hipSuccess;
  void* part = mse_scratch_ptr(&e);
  if (part == nullptr) return e;
  // every partial slot is written by the GEMM's epilogue before the sum reads it, so the
  // previous call's contents need no clearing
  return launch_linear_mse(L, A, x, T, flags, p, pert, target, static_cast<double*>(part), loss_pm, s);
}

size_t linear_xent_ws_bytes(int64_t T, int64_t d_out) {
  const int64_t nblk = (d_out + 127) / 128;
  const size_t a = (size_t)2 * T * nblk * sizeof(float2);
  const size_t b = ((size_t)2 * T * sizeof(float) + 255) / 256 * 256;
  return (a + 255) / 256 * 256 + b + (size_t)2 * kLossBlocks * sizeof(double);
}

hipError_t launch_linear_xent(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T, const void* p,
                              const zoact_pert_pair& pert, const int32_t* tokens, int64_t S, float* loss_pm, void* ws,
                              hipStream_t s) {
  GemmArgs a = bf16_args(L, A, x, T, p, nullptr, pert, nullptr);
  const int64_t nblk = (L.d_out + 127) / 128;
  char* w = static_cast<char*>(ws);
  a.xpart = reinterpret_cast<float2*>(w);
  w += ((size_t)2 * T * nblk * sizeof(float2) + 255) / 256 * 256;
  a.xtgt = reinterpret_cast<float*>(w);
  w += ((size_t)2 * T * sizeof(float) + 255) / 256 * 256;
  double* part = reinterpret_cast<double*>(w);
  a.tok = tokens;
  a.seq = S;
  a.xnblk = (int32_t)nblk;
  const hipError_t e = launch_linear_pm_4w64(a, L.w_dtype, EPI_XENT, false, false, s);
  if (e != hipSuccess) return e;
  return launch_xent_combine(a.xpart, a.xtgt, T, S, (int)nblk, T / S, part, loss_pm, s);
}

hipError_t launch_dequant_int4(const void* w, const void* scales, int64_t d_out, int64_t d_in, void* out,
                               hipStream_t s) {
  const int64_t units = d_out * (d_in / 8);
  int64_t g = (units + 1023) / 1024;
  g = g > (1 << 20) ? (1 << 20) : g;
  dequant_int4_kernel<<<dim3((unsigned)g), dim3(256), 0, s>>>(static_cast<const uint32_t*>(w),
                                                               static_cast<const uint16_t*>(scales), units, d_in / 8,
                                                               d_in / 128, static_cast<uint4*>(out));
  return hipGetLastError();
}

// Depth split of the workspace form: about four chunks of a multiple of 256, and at most
// as many as leave each wave 64 deep.
static int project_nsplit(int64_t d_in) {
  int ns = (int)(d_in / 1024);
  return ns < 1 ? 1 : (ns > 4 ? 4 : ns);
}
constexpr int PROJ_SPLIT_TB = 4;   // 64 tokens per workgroup

size_t project_ws_bytes(int64_t n_tok, int64_t d_in, int32_t r) {
  return (size_t)project_nsplit(d_in) * (size_t)n_tok * (size_t)r * 4;
}

hipError_t launch_project_split(const void* x, int64_t n_tok, int64_t d_in, const void* ut, int32_t r, void* p,
                                void* ws, hipStream_t s) {
  const int ns = project_nsplit(d_in);
  int64_t chunk = (d_in + ns - 1) / ns;
  chunk = (chunk + 255) / 256 * 256;
  const int64_t nb = (n_tok + 16 * PROJ_SPLIT_TB - 1) / (16 * PROJ_SPLIT_TB);
  float* part = static_cast<float*>(ws);
  const dim3 grid((unsigned)nb, (unsigned)ns);
  const auto* xx = static_cast<const uint16_t*>(x);
  const auto* uu = static_cast<const uint16_t*>(ut);
  auto* pp = static_cast<uint16_t*>(p);
  const int rb = (r + 15) / 16;
#define ZO_PS(RB) project_split_kernel<RB, PROJ_SPLIT_TB><<<grid, dim3(256), 0, s>>>(xx, uu, pp, n_tok, d_in, r, chunk, part)
  if (rb <= 1) ZO_PS(1);
  else if (rb <= 2) ZO_PS(2);
  else if (rb <= 4) ZO_PS(4);
  else return hipErrorNotSupported;
#undef ZO_PS
  const int64_t n = n_tok * r;
  const int vec = (n % 4 == 0) && (reinterpret_cast<uintptr_t>(p) % 8 == 0);
  project_sum_kernel<<<dim3((unsigned)((n + 1023) / 1024)), dim3(256), 0, s>>>(part, ns, n, pp, vec);
  return hipGetLastError();
}

hipError_t launch_project(const void* x, int32_t dtype, int64_t n_tok, int64_t d_in, const void* ut, int32_t r, void* p,
                          hipStream_t s) {
  if (dtype == ZOACT_F32) {
    int64_t g = (n_tok * r + 255) / 256;
    if (g > 65535) g = 65535;
    project_f32_kernel<<<dim3((unsigned)g), dim3(256), 0, s>>>(static_cast<const float*>(x),
                                                               static_cast<const float*>(ut), static_cast<float*>(p),
                                                               n_tok, d_in, r);
    return hipGetLastError();
  }
  // 32 tokens per workgroup (two 16-token blocks per wave): fewer would multiply the U^T
  // reads per token
  constexpr int TB = 2;
  const dim3 grid((unsigned)((n_tok + 16 * TB - 1) / (16 * TB)));
  // depth quarter per wave, a multiple of 32 (the last wave may get less or nothing)
  int64_t dq = (d_in + 3) / 4;
  dq = (dq + 31) / 32 * 32;
  const uint16_t* xx = static_cast<const uint16_t*>(x);
  const uint16_t* uu = static_cast<const uint16_t*>(ut);
  uint16_t* pp = static_cast<uint16_t*>(p);
  const int rb = (r + 15) / 16;
#ifndef ZOACT_PROJ_PIPE
#define ZOACT_PROJ_PIPE 1
#endif
  // d_in = 4096 (a 1024-deep share per wave, 32 steps): the fully unrolled pipeline (8192
  // tokens: 17.3 against 18.6 us for the loop below)
  if (ZOACT_PROJ_PIPE && d_in == 4096 && rb <= 2 && n_tok * d_in * 2 < (int64_t(1) << 31)) {
    if (rb <= 1) project_pipe_kernel<1, TB, 8, 32><<<grid, dim3(256), 0, s>>>(xx, uu, pp, n_tok, d_in, r);
    else project_pipe_kernel<2, TB, 8, 32><<<grid, dim3(256), 0, s>>>(xx, uu, pp, n_tok, d_in, r);
    return hipGetLastError();
  }
#define ZO_PROJ(RB) project_bf16_kernel<RB, TB><<<grid, dim3(256), 0, s>>>(xx, uu, pp, n_tok, d_in, r, dq)
  if (rb <= 1) ZO_PROJ(1);
  else if (rb <= 2) ZO_PROJ(2);
  else if (rb <= 4) ZO_PROJ(4);
  else if (rb <= 8) ZO_PROJ(8);
  else ZO_PROJ(16);
#undef ZO_PROJ
  return hipGetLastError();
}

}  // namespace zoact

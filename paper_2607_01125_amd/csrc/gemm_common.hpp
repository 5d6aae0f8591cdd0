// Argument block and small device helpers shared by the fused +/- GEMM kernels.
#pragma once
#include "common.hpp"
#include "rng.hpp"

namespace zoact {
namespace gemm {

struct GemmArgs {
  const uint16_t* x;      // [2][T][K]
  const void* w;          // [N][K] bf16 or packed int4 [N][K/2]
  const uint16_t* wsc;    // int4 scales [N][K/128]
  const uint16_t* bias;   // [N] or null
  const uint16_t* p;      // [2][T][r]
  const void* c;          // arena coefficients
  const uint16_t* resid;  // [2][T][Nout] or null
  void* y;                // [2][T][Nout]
  int64_t T, N, K;
  int32_t r;
  int32_t c_bf16;
  int64_t coef_offset;
  uint64_t seed;
  uint32_t step;
  uint32_t query_h[2];   // query index of half 0 / half 1
  int32_t sign_h[2];     // -1, 0 or +1: half h uses C + sign_h[h] eps Z(query_h[h])
  float eps;
  int32_t tiles_m_half;  // token tiles per half
  int32_t tiles_n;
  int32_t n_tail;        // depth tiles of the correction block
  const uint16_t* ch;    // precomputed bf16(C + sign_h eps Z), [2][N][r] with half stride ch_stride, or null
  int64_t ch_stride;
  const uint16_t* tgt;   // EPI_MSE: regression target [T][N] (bf16); y is not stored
  double* part;          // EPI_MSE: sums of squared errors per tile and wave [2][tiles_m_half * tiles_n][4]
  const int32_t* tok;    // EPI_XENT: token ids [T / seq][seq] shared by both halves
  int64_t seq;           // EPI_XENT: sequence length
  float2* xpart;         // EPI_XENT: (max, sum of exp) per row and 128-column block [2 T][xnblk]
  float* xtgt;           // EPI_XENT: the logit of each row's next token [2 T]
  int32_t xnblk;         // EPI_XENT: ceil(N / 128)
  int64_t plain_begin;   // output features [plain_begin, plain_end): no correction, no coefficient rows
  int64_t plain_end;
  float* tail_ws;        // split tail (64-deep schedule): the half tiles' fp32 accumulators
  int64_t tail_ws_bytes;
  int32_t tail_first;    // first virtual tile that is half a tile (= the tile count: none)
  int32_t tail_cols;     // feature tiles (the last ones, both halves' token tiles) of the split tail
};

// Buffer descriptor over [base, base + bytes): loads past the end read 0, stores past it are
// dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Internal epilogue selector (not a public flag): the tile's squared errors against tgt
// are summed instead of storing y.
constexpr int EPI_MSE = 1 << 8;
// Internal epilogue selector: per row and 128-column block, the maximum and the sum of
// exp(logit - maximum), plus the logit of the row's next token; logits are not stored.
constexpr int EPI_XENT = 1 << 9;

__device__ __forceinline__ int swz(int row, int kc) { return (row << 6) + ((kc ^ (row & 7)) << 3); }

// Four consecutive Z values starting at arena index e (any alignment).
__device__ __forceinline__ float4 gauss4(uint64_t seed, uint32_t step, uint32_t query, uint64_t e) {
  const float4 a = rng::gauss_block(seed, step, query, e >> 2);
  const int o = (int)(e & 3);
  if (o == 0) return a;
  const float4 b = rng::gauss_block(seed, step, query, (e >> 2) + 1);
  float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  return make_float4(v[o], v[o + 1], v[o + 2], v[o + 3]);
}

// fp32 (C + sign*eps*z) rounded to bf16; the product eps*z is rounded before the sum
// (sign 0: C itself).
__device__ __forceinline__ uint16_t perturbed_bf16(float c, float z, float eps, int sign) {
#pragma clang fp contract(off)
  const float ez = eps * z;
  return f2bf(sign > 0 ? c + ez : (sign < 0 ? c - ez : c));
}

__device__ __forceinline__ uint32_t pack2(uint16_t lo, uint16_t hi) { return (uint32_t)lo | ((uint32_t)hi << 16); }

// Dequantise 8 nibbles (one uint32, element 2j in the low nibble of byte j) with scale s.
__device__ __forceinline__ uint4 dequant8(uint32_t q, float s) {
  uint16_t o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int v = ((int)(q << (28 - 4 * j))) >> 28;  // sign-extend nibble j
    o[j] = f2bf((float)v * s);
  }
  return make_uint4(pack2(o[0], o[1]), pack2(o[2], o[3]), pack2(o[4], o[5]), pack2(o[6], o[7]));
}


// g * sigmoid(g) with the hardware reciprocal (1 ulp) in place of an IEEE divide: the
// result is rounded to bf16 (or carries fp32 GEMM rounding), far coarser than the
// reciprocal's error.
__device__ __forceinline__ float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

}  // namespace gemm
}  // namespace zoact

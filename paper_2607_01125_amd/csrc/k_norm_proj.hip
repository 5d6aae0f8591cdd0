// Normalisation fused with the rank-r projection of its output (Section 3: the X V_r
// factor of the perturbed forward, Y = X W + (X V_r)(B + mu Z), for the sites whose input
// is a norm's output: the attention input and the MLP input).
//
// The separate form writes the normalised rows and then reads them again to form
// P = X U.  Here one workgroup of NW waves owns 16 tokens and wave w the slice
// [w d/NW, (w + 1) d/NW) of their rows, read in the MFMA's A-fragment layout (lane
// (lr, lk): token lr, features c 32 + lk 8 .. +7 of the slice, chunk c).  The statistics
// (the mean for LayerNorm, then the sum of squares about it) are accumulated over the
// chunks, reduced over the four lanes of a token and then over the waves in a fixed
// order; a last pass reads each chunk again (from L2), normalises it (one rounding to
// bf16, the norm's output), stores it and multiplies it with the chunk's U^T rows on
// v_mfma_f32_16x16x32_bf16.  Keeping no row in registers between the passes leaves room
// for several workgroups per CU, whose passes overlap.  The waves' fp32 partial products
// are summed in a fixed order through LDS before P's single rounding to bf16.
#include "common.hpp"

namespace zoact {

namespace {

__device__ __forceinline__ float lo16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Sum over the four lanes that hold one token's chunks (lanes lr, lr + 16, lr + 32, lr + 48).
__device__ __forceinline__ float token_sum(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

template <bool LN, int NW, int NC, int RB>
__global__ void __launch_bounds__(NW * 64, 2) norm_project_kernel(const uint16_t* __restrict__ x,
                                                           const uint16_t* __restrict__ w,
                                                           const uint16_t* __restrict__ bias, int64_t n_tok,
                                                           int64_t d, float eps, const uint16_t* __restrict__ ut,
                                                           int r, uint16_t* __restrict__ y, uint16_t* __restrict__ p) {
  __shared__ float red[2][NW][16];
  __shared__ float part[NW][16][RB * 16 + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t t = (int64_t)blockIdx.x * 16 + lr;
  const bool valid = t < n_tok;
  const int64_t f0 = (int64_t)wave * (d / NW) + lk * 8;   // this lane's first feature
  const uint16_t* xr = x + (valid ? t : 0) * d + f0;

  auto chunk = [&](int c) -> uint4 {
    return valid ? *reinterpret_cast<const uint4*>(xr + c * 32) : make_uint4(0u, 0u, 0u, 0u);
  };

  // statistics of the token over its d features
  float mu = 0.f;
  if constexpr (LN) {
    float s = 0.f;
#pragma unroll 4
    for (int c = 0; c < NC; ++c) {
      const uint4 h = chunk(c);
      const uint32_t q[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        s += lo16(q[e]);
        s += hi16(q[e]);
      }
    }
    s = token_sum(s);
    if (lk == 0) red[0][wave][lr] = s;
    __syncthreads();
    float tot = 0.f;
#pragma unroll
    for (int q = 0; q < NW; ++q) tot += red[0][q][lr];
    mu = tot / (float)d;
  }
  float ss = 0.f;
#pragma unroll 4
  for (int c = 0; c < NC; ++c) {
    const uint4 h = chunk(c);
    const uint32_t q[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = LN ? lo16(q[e]) - mu : lo16(q[e]);
      const float b = LN ? hi16(q[e]) - mu : hi16(q[e]);
      ss += a * a;
      ss += b * b;
    }
  }
  ss = token_sum(ss);
  if (lk == 0) red[1][wave][lr] = ss;
  __syncthreads();
  float tss = 0.f;
#pragma unroll
  for (int q = 0; q < NW; ++q) tss += red[1][q][lr];
  const float inv = rsqrtf(tss / (float)d + eps);

  // normalise chunk by chunk: store the norm's output and multiply it with U^T
  floatx4 acc[RB];
#pragma unroll
  for (int j = 0; j < RB; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
  uint16_t* yr = y + (valid ? t : 0) * d + f0;
  const bf16x8 zero8 = {};
#pragma unroll 4
  for (int c = 0; c < NC; ++c) {
    const uint4 hc = chunk(c);
    const uint4 g = *reinterpret_cast<const uint4*>(w + f0 + c * 32);
    uint4 bb = make_uint4(0u, 0u, 0u, 0u);
    if constexpr (LN) bb = *reinterpret_cast<const uint4*>(bias + f0 + c * 32);
    const uint32_t q[4] = {hc.x, hc.y, hc.z, hc.w};
    const uint32_t gv[4] = {g.x, g.y, g.z, g.w}, bv[4] = {bb.x, bb.y, bb.z, bb.w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float a, b;
      if constexpr (LN) {
        a = ((lo16(q[e]) - mu) * inv) * lo16(gv[e]) + lo16(bv[e]);
        b = ((hi16(q[e]) - mu) * inv) * hi16(gv[e]) + hi16(bv[e]);
      } else {
        a = (lo16(q[e]) * inv) * lo16(gv[e]);
        b = (hi16(q[e]) * inv) * hi16(gv[e]);
      }
      o[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
    }
    const uint4 xo = make_uint4(o[0], o[1], o[2], o[3]);
    if (valid) *reinterpret_cast<uint4*>(yr + c * 32) = xo;
    const bf16x8 af = __builtin_bit_cast(bf16x8, xo);
#pragma unroll
    for (int j = 0; j < RB; ++j) {
      const int rc = j * 16 + lr;
      const bf16x8 bf = rc < r ? *reinterpret_cast<const bf16x8*>(ut + (int64_t)rc * d + f0 + c * 32) : zero8;
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf, acc[j], 0, 0, 0);
    }
  }
  // D[token = 4 lk + v][column = 16 j + lr] per wave, then the waves summed in order
#pragma unroll
  for (int j = 0; j < RB; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) part[wave][lk * 4 + v][j * 16 + lr] = acc[j][v];
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * r; e += NW * 64) {
    const int tok = e / r, col = e % r;
    const int64_t tt = (int64_t)blockIdx.x * 16 + tok;
    if (tt < n_tok) {
      float v = 0.f;
#pragma unroll
      for (int q = 0; q < NW; ++q) v += part[q][tok][col];
      p[tt * r + col] = f2bf(v);
    }
  }
}

template <bool LN, int NW, int NC>
hipError_t launch_np_r(const uint16_t* x, const uint16_t* w, const uint16_t* b, int64_t n_tok, int64_t d, float eps,
                       const uint16_t* ut, int r, uint16_t* y, uint16_t* p, hipStream_t s) {
  const dim3 grid((unsigned)((n_tok + 15) / 16)), block(NW * 64);
  if (r <= 16) norm_project_kernel<LN, NW, NC, 1><<<grid, block, 0, s>>>(x, w, b, n_tok, d, eps, ut, r, y, p);
  else if (r <= 32) norm_project_kernel<LN, NW, NC, 2><<<grid, block, 0, s>>>(x, w, b, n_tok, d, eps, ut, r, y, p);
  else if (r <= 64) norm_project_kernel<LN, NW, NC, 4><<<grid, block, 0, s>>>(x, w, b, n_tok, d, eps, ut, r, y, p);
  else norm_project_kernel<LN, NW, NC, 8><<<grid, block, 0, s>>>(x, w, b, n_tok, d, eps, ut, r, y, p);
  return hipGetLastError();
}

}  // namespace

// Shapes this fused form covers: d = 128 (four waves, one chunk each) or d a multiple of
// 256 with d / 256 chunks per wave in {1, 2, 4, 8, 16, 20} (eight waves; d = 256 .. 5120),
// 1 <= r <= 128.  Others: hipErrorNotSupported.
hipError_t launch_norm_project(bool layernorm, const void* x, const void* w, const void* b, int64_t n_tok, int64_t d,
                               float eps, const void* ut, int r, void* y, void* p, hipStream_t s) {
  if (d % 128 != 0 || r < 1 || r > 128 || n_tok < 1) return hipErrorNotSupported;
  const auto* xx = static_cast<const uint16_t*>(x);
  const auto* ww = static_cast<const uint16_t*>(w);
  const auto* bb = static_cast<const uint16_t*>(b);
  const auto* uu = static_cast<const uint16_t*>(ut);
  auto* yy = static_cast<uint16_t*>(y);
  auto* pp = static_cast<uint16_t*>(p);
#define ZO_NP(NW, NC)                                                                                  \
  if (d == (int64_t)NW * 32 * NC)                                                                      \
    return layernorm ? launch_np_r<true, NW, NC>(xx, ww, bb, n_tok, d, eps, uu, r, yy, pp, s)         \
                     : launch_np_r<false, NW, NC>(xx, ww, bb, n_tok, d, eps, uu, r, yy, pp, s);
  ZO_NP(4, 1)
  ZO_NP(8, 1)
  ZO_NP(8, 2)
  ZO_NP(8, 4)
  ZO_NP(8, 8)
  ZO_NP(8, 16)
  ZO_NP(8, 20)
#undef ZO_NP
  return hipErrorNotSupported;
}

}  // namespace zoact

// Support operations of the decoder forward (embeddings, RMSNorm, LayerNorm, rotary
// embedding, causal attention) and their extern "C" entry points (zoact_model.h).
//
// All are HBM-bound elementwise/row passes except attention, which is a small MFMA
// contraction (under 1% of a ZO step's FLOPs at the 8B/13B shapes): one workgroup per
// (64-query block, head, sequence), scores and P.V on v_mfma_f32_16x16x32_bf16, a
// two-pass softmax in fp32 with wave64 shuffles, K and V staged through LDS (V
// transposed so that each lane's fragment holds 8 consecutive keys).
#include <math.h>
#include <stdio.h>

#include <string>

#include "common.hpp"
#include "zoact_model.h"

namespace zoact {
namespace {

template <typename T>
__device__ __forceinline__ float ld_act(const T* p, int64_t i);
template <>
__device__ __forceinline__ float ld_act<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ld_act<uint16_t>(const uint16_t* p, int64_t i) { return bf2f(p[i]); }
template <typename T>
__device__ __forceinline__ void st_act(T* p, int64_t i, float v);
template <>
__device__ __forceinline__ void st_act<float>(float* p, int64_t i, float v) { p[i] = v; }
template <>
__device__ __forceinline__ void st_act<uint16_t>(uint16_t* p, int64_t i, float v) { p[i] = f2bf(v); }

template <typename T>
__global__ void embed_kernel(const int32_t* __restrict__ tok, int64_t n_tok, int distinct, int64_t vocab,
                             const T* __restrict__ table, const T* __restrict__ pos, int64_t max_pos, int pos_offset,
                             int64_t seq, int64_t d, T* __restrict__ out) {
  const int64_t half = n_tok * d;
  const int64_t total = distinct ? 2 * half : half;  // distinct: one element per output; else one per pair
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / d, c = i % d;   // row indexes tokens[] (the [2][n_tok] set when distinct)
    const int64_t t = row % n_tok;
    int64_t id = tok[row];
    id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
    float v = ld_act(table, id * d + c);
    if (pos) {
      int64_t pp = t % seq + pos_offset;
      pp = pp >= max_pos ? max_pos - 1 : pp;
      v += ld_act(pos, pp * d + c);
    }
    st_act(out, i, v);
    if (!distinct) st_act(out, half + i, v);
  }
}

__device__ __forceinline__ float block_sum(float v, float* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) t += sh[i];
  __syncthreads();
  return t;
}

template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const T* __restrict__ x, const T* __restrict__ w, int64_t d, float eps,
                                                      T* __restrict__ y) {
  __shared__ float sh[4];
  const T* xr = x + (int64_t)blockIdx.x * d;
  T* yr = y + (int64_t)blockIdx.x * d;
  float ss = 0.f;
  for (int64_t c = threadIdx.x; c < d; c += blockDim.x) {
    const float v = ld_act(xr, c);
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum(ss, sh) / (float)d + eps);
  for (int64_t c = threadIdx.x; c < d; c += blockDim.x) st_act(yr, c, (ld_act(xr, c) * inv) * ld_act(w, c));
}

template <typename T>
__global__ void __launch_bounds__(256) layernorm_kernel(const T* __restrict__ x, const T* __restrict__ w, const T* __restrict__ b,
                                                        int64_t d, float eps, T* __restrict__ y) {
  __shared__ float sh[4];
  const T* xr = x + (int64_t)blockIdx.x * d;
  T* yr = y + (int64_t)blockIdx.x * d;
  float s = 0.f;
  for (int64_t c = threadIdx.x; c < d; c += blockDim.x) s += ld_act(xr, c);
  const float mu = block_sum(s, sh) / (float)d;
  float ss = 0.f;
  for (int64_t c = threadIdx.x; c < d; c += blockDim.x) {
    const float v = ld_act(xr, c) - mu;
    ss += v * v;
  }
  const float inv = rsqrtf(block_sum(ss, sh) / (float)d + eps);
  for (int64_t c = threadIdx.x; c < d; c += blockDim.x)
    st_act(yr, c, ((ld_act(xr, c) - mu) * inv) * ld_act(w, c) + ld_act(b, c));
}

// bf16 RMSNorm with 16-byte accesses: each thread keeps its VPT values of the row in
// registers between the two passes (d = 256 * 8 * VPT8).
template <int VPT8>
__global__ void __launch_bounds__(256) rmsnorm_bf16_vec_kernel(const uint16_t* __restrict__ x,
                                                               const uint16_t* __restrict__ w, int64_t d, float eps,
                                                               uint16_t* __restrict__ y) {
  __shared__ float sh[4];
  const uint16_t* xr = x + (int64_t)blockIdx.x * d;
  uint16_t* yr = y + (int64_t)blockIdx.x * d;
  uint4 v[VPT8];
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < VPT8; ++u) {
    v[u] = *reinterpret_cast<const uint4*>(xr + (int64_t)(u * 256 + threadIdx.x) * 8);
    const uint32_t wv[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = bf2f((uint16_t)(wv[e] & 0xFFFF)), b = bf2f((uint16_t)(wv[e] >> 16));
      ss += a * a;
      ss += b * b;
    }
  }
  const float inv = rsqrtf(block_sum(ss, sh) / (float)d + eps);
#pragma unroll
  for (int u = 0; u < VPT8; ++u) {
    const int64_t c = (int64_t)(u * 256 + threadIdx.x) * 8;
    const uint4 g = *reinterpret_cast<const uint4*>(w + c);
    const uint32_t xv[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    const uint32_t gv[4] = {g.x, g.y, g.z, g.w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = (bf2f((uint16_t)(xv[e] & 0xFFFF)) * inv) * bf2f((uint16_t)(gv[e] & 0xFFFF));
      const float b = (bf2f((uint16_t)(xv[e] >> 16)) * inv) * bf2f((uint16_t)(gv[e] >> 16));
      o[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
    }
    *reinterpret_cast<uint4*>(yr + c) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// bf16 LayerNorm with 16-byte accesses, the same arrangement (row chunks of 8 in registers,
// chunk u * 256 + thread, d % 8 == 0, d <= 2048 * VPT8): mean, then the centred second
// moment, then ((x - mean) * inv) * w + b with one rounding.
template <int VPT8>
__global__ void __launch_bounds__(256) layernorm_bf16_vec_kernel(const uint16_t* __restrict__ x,
                                                                 const uint16_t* __restrict__ w,
                                                                 const uint16_t* __restrict__ bias, int64_t d,
                                                                 float eps, uint16_t* __restrict__ y) {
  __shared__ float sh[4];
  const uint16_t* xr = x + (int64_t)blockIdx.x * d;
  uint16_t* yr = y + (int64_t)blockIdx.x * d;
  const int nch = (int)(d / 8);
  float f[VPT8][8];
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < VPT8; ++u) {
    const int ch = u * 256 + threadIdx.x;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (ch < nch) v = *reinterpret_cast<const uint4*>(xr + (int64_t)ch * 8);
    const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[u][2 * e] = bf2f((uint16_t)(wv[e] & 0xFFFF));
      f[u][2 * e + 1] = bf2f((uint16_t)(wv[e] >> 16));
      s += f[u][2 * e];
      s += f[u][2 * e + 1];
    }
  }
  const float mu = block_sum(s, sh) / (float)d;
  float ss = 0.f;
#pragma unroll
  for (int u = 0; u < VPT8; ++u) {
    if (u * 256 + (int)threadIdx.x >= nch) continue;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float c = f[u][e] - mu;
      ss += c * c;
    }
  }
  const float inv = rsqrtf(block_sum(ss, sh) / (float)d + eps);
#pragma unroll
  for (int u = 0; u < VPT8; ++u) {
    const int ch = u * 256 + threadIdx.x;
    if (ch >= nch) continue;
    const uint4 g = *reinterpret_cast<const uint4*>(w + (int64_t)ch * 8);
    const uint4 bb = *reinterpret_cast<const uint4*>(bias + (int64_t)ch * 8);
    const uint32_t gv[4] = {g.x, g.y, g.z, g.w}, bv[4] = {bb.x, bb.y, bb.z, bb.w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = ((f[u][2 * e] - mu) * inv) * bf2f((uint16_t)(gv[e] & 0xFFFF)) + bf2f((uint16_t)(bv[e] & 0xFFFF));
      const float b = ((f[u][2 * e + 1] - mu) * inv) * bf2f((uint16_t)(gv[e] >> 16)) + bf2f((uint16_t)(bv[e] >> 16));
      o[e] = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
    }
    *reinterpret_cast<uint4*>(yr + (int64_t)ch * 8) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// One rotary pair: (lo, hi) -> (lo c - hi s, hi c + lo s), products rounded before the
// sum (no contraction), so that every kernel that rotates gives the same bits.
__device__ __forceinline__ float rot_lo(float lo, float hi, float c, float s) {
#pragma clang fp contract(off)
  return lo * c - hi * s;
}
__device__ __forceinline__ float rot_hi(float lo, float hi, float c, float s) {
#pragma clang fp contract(off)
  return hi * c + lo * s;
}

// bf16 rotary embedding with 16-byte accesses: one thread rotates 8 pairs (j .. j + 7 with
// their partners j + half .. j + half + 7) of one head of one row.
__global__ void rope_bf16_vec_kernel(uint16_t* __restrict__ x, int64_t rows, int64_t ld, int64_t col0, int heads,
                                     int hd, int64_t seq, const float* __restrict__ ct, const float* __restrict__ st) {
  const int half = hd / 2, g8 = half / 8;
  const int64_t total = rows * heads * g8;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(i % g8) * 8;
    const int h = (int)((i / g8) % heads);
    const int64_t r = i / ((int64_t)g8 * heads);
    const int64_t pos = r % seq;
    uint16_t* p = x + r * ld + col0 + (int64_t)h * hd;
    const uint4 lo4 = *reinterpret_cast<const uint4*>(p + j);
    const uint4 hi4 = *reinterpret_cast<const uint4*>(p + j + half);
    const float4 c0 = *reinterpret_cast<const float4*>(ct + pos * half + j);
    const float4 c1 = *reinterpret_cast<const float4*>(ct + pos * half + j + 4);
    const float4 s0 = *reinterpret_cast<const float4*>(st + pos * half + j);
    const float4 s1 = *reinterpret_cast<const float4*>(st + pos * half + j + 4);
    const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
    const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
    const uint32_t lw[4] = {lo4.x, lo4.y, lo4.z, lo4.w}, hw[4] = {hi4.x, hi4.y, hi4.z, hi4.w};
    uint32_t lo_o[4], hi_o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint16_t lo_r[2], hi_r[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const float lo = bf2f((uint16_t)(q ? lw[e] >> 16 : lw[e] & 0xFFFF));
        const float hi = bf2f((uint16_t)(q ? hw[e] >> 16 : hw[e] & 0xFFFF));
        const float c = cv[2 * e + q], sn = sv[2 * e + q];
        lo_r[q] = f2bf(rot_lo(lo, hi, c, sn));
        hi_r[q] = f2bf(rot_hi(lo, hi, c, sn));
      }
      lo_o[e] = (uint32_t)lo_r[0] | ((uint32_t)lo_r[1] << 16);
      hi_o[e] = (uint32_t)hi_r[0] | ((uint32_t)hi_r[1] << 16);
    }
    *reinterpret_cast<uint4*>(p + j) = make_uint4(lo_o[0], lo_o[1], lo_o[2], lo_o[3]);
    *reinterpret_cast<uint4*>(p + j + half) = make_uint4(hi_o[0], hi_o[1], hi_o[2], hi_o[3]);
  }
}

template <typename T>
__global__ void rope_kernel(T* __restrict__ x, int64_t rows, int64_t ld, int64_t col0, int heads, int hd, int64_t seq,
                            const float* __restrict__ ct, const float* __restrict__ st) {
  const int half = hd / 2;
  const int64_t total = rows * heads * half;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int j = (int)(i % half);
    const int h = (int)((i / half) % heads);
    const int64_t r = i / ((int64_t)half * heads);
    const int64_t pos = r % seq;
    T* p = x + r * ld + col0 + (int64_t)h * hd;
    const float c = ct[pos * half + j], s = st[pos * half + j];
    const float lo = ld_act(p, j), hi = ld_act(p, j + half);
    st_act(p, j, rot_lo(lo, hi, c, s));
    st_act(p, j + half, rot_hi(lo, hi, c, s));
  }
}

// ---------------------------------------------------------------- attention, fp32 (small)
// One workgroup per (sequence, head); K and V of the sequence in LDS; one thread per query.
__global__ void __launch_bounds__(256) attention_f32_kernel(const float* __restrict__ q, int64_t ldq, const float* __restrict__ k,
                                                            int64_t ldk, const float* __restrict__ v, int64_t ldv, int64_t seq,
                                                            int heads, int kv_heads, int hd, float scale,
                                                            float* __restrict__ out) {
  extern __shared__ float kv[];  // [seq][hd] K then [seq][hd] V
  const int h = blockIdx.x, b = blockIdx.y;
  const int hk = h / (heads / kv_heads);
  const int64_t r0 = (int64_t)b * seq;
  for (int64_t i = threadIdx.x; i < seq * hd; i += blockDim.x) {
    const int64_t s = i / hd, e = i % hd;
    kv[i] = k[(r0 + s) * ldk + (int64_t)hk * hd + e];
    kv[seq * hd + i] = v[(r0 + s) * ldv + (int64_t)hk * hd + e];
  }
  __syncthreads();
  for (int64_t sq = threadIdx.x; sq < seq; sq += blockDim.x) {
    const float* qr = q + (r0 + sq) * ldq + (int64_t)h * hd;
    float m = -INFINITY, l = 0.f;
    float acc[128];
    for (int e = 0; e < hd; ++e) acc[e] = 0.f;
    for (int64_t sk = 0; sk <= sq; ++sk) {
      float sc = 0.f;
      for (int e = 0; e < hd; ++e) sc += qr[e] * kv[sk * hd + e];
      sc *= scale;
      const float mn = fmaxf(m, sc);
      const float a = expf(m - mn), p = expf(sc - mn);
      l = l * a + p;
      for (int e = 0; e < hd; ++e) acc[e] = acc[e] * a + p * kv[seq * hd + sk * hd + e];
      m = mn;
    }
    float* o = out + (r0 + sq) * (int64_t)heads * hd + (int64_t)h * hd;
    for (int e = 0; e < hd; ++e) o[e] = acc[e] / l;
  }
}

// ---------------------------------------------------------------- attention, bf16 MFMA
// Two passes over the key blocks: the first finds each query row's maximum score, the
// second forms P = exp(s - max) against that final maximum, rounds P to bf16 and
// accumulates P.V on MFMA (normaliser summed from the unrounded P).  Forming P against
// the final maximum (instead of rescaling a running one) keeps each bf16 rounding of P
// the same as in the plain softmax definition; the extra Q.K^T pass costs little, as
// attention is a small share of a step's FLOPs.
template <int HD>
__device__ __forceinline__ void stage_k(const uint16_t* __restrict__ k, int64_t ldk, int64_t r0, int64_t seq, int hk,
                                        int kb, uint16_t* ks) {
  constexpr int KC = HD / 8;
  for (int cidx = threadIdx.x; cidx < 64 * KC; cidx += 256) {
    const int key = cidx / KC, ch = cidx % KC;
    int64_t kr = (int64_t)kb * 64 + key;
    kr = kr < seq ? kr : seq - 1;
    const uint4 kvv = *reinterpret_cast<const uint4*>(k + (r0 + kr) * ldk + (int64_t)hk * HD + ch * 8);
    *reinterpret_cast<uint4*>(ks + key * HD + ((ch ^ (key & 7)) * 8)) = kvv;
  }
}

// scores S[q = 4*lk + i][key = j*16 + lr] of this wave's 16 queries against key block kb
template <int HD>
__device__ __forceinline__ void scores(const bf16x8* qf, const uint16_t* ks, int lr, int lk, floatx4* s) {
  constexpr int KS = HD / 32;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    s[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const int key = j * 16 + lr;
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + key * HD + (((kk * 4 + lk) ^ (key & 7)) * 8));
      s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[kk], kf, s[j], 0, 0, 0);
    }
  }
}

template <int HD>
__global__ void __launch_bounds__(256) attention_bf16_kernel(const uint16_t* __restrict__ q, int64_t ldq,
                                                             const uint16_t* __restrict__ k, int64_t ldk,
                                                             const uint16_t* __restrict__ v, int64_t ldv, int64_t seq,
                                                             int heads, int kv_heads, float scale,
                                                             uint16_t* __restrict__ out) {
  constexpr int KC = HD / 8;         // 16-byte chunks per row
  constexpr int KS = HD / 32;        // 32-deep steps over the head dimension
  constexpr int NB = HD / 16;        // output column blocks
  __shared__ __align__(16) uint16_t ks[64 * HD];       // K block [key][hd], chunk-swizzled
  __shared__ __align__(16) uint16_t vt[HD * 72];       // V block transposed [hd][key], padded
  __shared__ __align__(16) uint16_t pw[4][16 * 72];    // per-wave probabilities [q][key], padded
  const int qb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int hk = h / (heads / kv_heads);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t r0 = (int64_t)b * seq;
  const int64_t q0 = (int64_t)qb * 64 + wave * 16;    // first query row of this wave

  // Q fragments (A operand): row lr, depth kk*32 + lk*8
  bf16x8 qf[KS];
  {
    int64_t qr = q0 + lr;
    qr = qr < seq ? qr : seq - 1;
    const uint16_t* qp = q + (r0 + qr) * ldq + (int64_t)h * HD;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 32 + lk * 8);
  }
  const int64_t qmax = (int64_t)qb * 64 + 63;
  const int nkb = (int)((qmax < seq - 1 ? qmax : seq - 1) / 64) + 1;

  // pass 1: row maxima of the scaled, masked scores
  float mrow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) mrow[i] = -INFINITY;
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    stage_k<HD>(k, ldk, r0, seq, hk, kb, ks);
    __syncthreads();
    floatx4 s[4];
    scores<HD>(qf, ks, lr, lk, s);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t qi = q0 + lk * 4 + i;
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t key = (int64_t)kb * 64 + j * 16 + lr;
        if (key <= qi && key < seq) mx = fmaxf(mx, s[j][i] * scale);
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      mrow[i] = fmaxf(mrow[i], mx);
    }
  }

  // pass 2: P = exp(s - max) rounded to bf16, O += P V, l += P (unrounded)
  floatx4 o[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) o[n] = floatx4{0.f, 0.f, 0.f, 0.f};
  float lrow[4] = {0.f, 0.f, 0.f, 0.f};
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    stage_k<HD>(k, ldk, r0, seq, hk, kb, ks);
    for (int cidx = threadIdx.x; cidx < 64 * KC; cidx += 256) {
      const int key = cidx / KC, ch = cidx % KC;
      int64_t kr = (int64_t)kb * 64 + key;
      kr = kr < seq ? kr : seq - 1;
      const uint4 vv = *reinterpret_cast<const uint4*>(v + (r0 + kr) * ldv + (int64_t)hk * HD + ch * 8);
      const uint16_t* ve = reinterpret_cast<const uint16_t*>(&vv);
#pragma unroll
      for (int e = 0; e < 8; ++e) vt[(ch * 8 + e) * 72 + key] = ve[e];
    }
    __syncthreads();
    floatx4 s[4];
    scores<HD>(qf, ks, lr, lk, s);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t qi = q0 + lk * 4 + i;
      float ps = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t key = (int64_t)kb * 64 + j * 16 + lr;
        const float p = (key <= qi && key < seq) ? expf(s[j][i] * scale - mrow[i]) : 0.f;
        s[j][i] = p;
        ps += p;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) ps += __shfl_xor(ps, off, 64);
      lrow[i] += ps;
    }
    // probabilities to bf16 through LDS, read back as A fragments (row lr, keys lk*8 ..)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) pw[wave][(lk * 4 + i) * 72 + j * 16 + lr] = f2bf(s[j][i]);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS writes done
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const bf16x8 pf = *reinterpret_cast<const bf16x8*>(&pw[wave][lr * 72 + kk * 32 + lk * 8]);
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&vt[(n * 16 + lr) * 72 + kk * 32 + lk * 8]);
        o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf, vf, o[n], 0, 0, 0);
      }
    }
  }
  // O[q = 4*lk + i][col = n*16 + lr] / l
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t qi = q0 + lk * 4 + i;
    if (qi >= seq) continue;
    const float inv = 1.f / lrow[i];
    uint16_t* op = out + (r0 + qi) * (int64_t)heads * HD + (int64_t)h * HD;
#pragma unroll
    for (int n = 0; n < NB; ++n) op[n * 16 + lr] = f2bf(o[n][i] * inv);
  }
}

// ---------------------------------------------------------------- attention, bf16 MFMA, shared K/V
// Same two-pass definition as attention_bf16_kernel (P = exp(s - final max) rounded to bf16,
// normaliser from the unrounded P), organised for grouped-query heads: a workgroup takes one
// key/value head of one sequence and HG = min(G, 4) of the G query heads that read it, each
// wave 16 * QB queries of one head (QT = 64 QB / HG queries per workgroup tile), so every
// K/V block staged in LDS serves four waves' worth of queries.  QB = 2 keeps a thread within
// 256 registers, two workgroups per CU.  Scores are formed transposed,
// S^T[key][query] (K as the MFMA A operand, Q as B): a lane then holds four keys of one
// query, its probabilities are already the B operand of O^T = V^T P^T, and V^T is read in
// the same key order (the order of the 32 keys inside one MFMA does not change the sum
// beyond rounding), so P never goes through LDS.
template <int HD, int QB>
__global__ void __launch_bounds__(256, 2) attention_gqa_kernel(const uint16_t* __restrict__ q, int64_t ldq,
                                                            const uint16_t* __restrict__ k, int64_t ldk,
                                                            const uint16_t* __restrict__ v, int64_t ldv, int64_t seq,
                                                            int heads, int kv_heads, float scale,
                                                            uint16_t* __restrict__ out) {
  constexpr int KC = HD / 8;   // 16-byte chunks per row
  constexpr int KS = HD / 32;  // 32-deep steps over the head dimension
  constexpr int ND = HD / 16;  // 16-row blocks of the head dimension
  // K chunks XOR-swizzled over 16 rows (8 when a row has only 8 chunks) and V^T rows of 34
  // words keep the fragment reads free of LDS bank conflicts
  constexpr int KSW = KC >= 16 ? 15 : 7;
  constexpr int VW = 34;
  __shared__ __align__(16) uint16_t ks[64 * HD];   // K block [key][hd], chunk-swizzled
  __shared__ __align__(16) uint32_t vt[HD * VW];   // V block transposed [d][key], key pairs per word, padded
  const int G = heads / kv_heads;
  const int HG = G < 4 ? G : 4;
  const int QT = 64 * QB / HG;                             // queries per workgroup tile
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int sub = G / HG;                                   // workgroups per key/value head
  const int hk = blockIdx.y / sub;
  const int h = hk * G + (blockIdx.y % sub) * HG + (wave % HG);
  const int64_t r0 = (int64_t)blockIdx.z * seq;
  const int64_t qt0 = (int64_t)blockIdx.x * QT;
  const int64_t q0 = qt0 + (int64_t)(wave / HG) * (16 * QB);   // this wave's first query
  const int64_t wq_last = q0 + 16 * QB - 1 < seq - 1 ? q0 + 16 * QB - 1 : seq - 1;
  const int64_t tq_last = qt0 + QT - 1 < seq - 1 ? qt0 + QT - 1 : seq - 1;
  const int nkb = (int)(tq_last / 64) + 1;

  // Q fragments (B operand): q-block b, row lr, depth kk*32 + lk*8
  bf16x8 qf[QB][KS];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    int64_t qr = q0 + b * 16 + lr;
    qr = qr < seq ? qr : seq - 1;
    const uint16_t* qp = q + (r0 + qr) * ldq + (int64_t)h * HD;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[b][kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 32 + lk * 8);
  }
  // S^T of key block kb against q-block b: lane holds S^T[key = j*16 + 4*lk + i][query = b*16 + lr]
  auto scores_t = [&](int b, floatx4 (&st)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      st[j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const int key = j * 16 + lr;
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + key * HD + (((kk * 4 + lk) ^ (key & KSW)) * 8));
        st[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[b][kk], st[j], 0, 0, 0);
      }
    }
  };

  // keys of block kb this lane's query of q-block b may see: key offset within the block
  // <= the returned limit (causal: key <= query; and key < seq)
  auto key_limit = [&](int b, int kb) -> int {
    int64_t last = q0 + b * 16 + lr;
    last = last < seq - 1 ? last : seq - 1;
    return (int)(last - (int64_t)kb * 64);
  };

  // a key block needs the causal mask only where it reaches past the q-block's first query
  // (or past the sequence); the test is uniform over the wave
  auto masked = [&](int b, int kb) {
    return (int64_t)kb * 64 + 63 > (q0 + b * 16 < seq - 1 ? q0 + b * 16 : seq - 1);
  };
  // pass 1: row maxima of the raw scores over visible keys (scaling by a positive constant
  // keeps the maximiser, so the scale is applied once, to the maximum)
  float mq[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) mq[b] = -INFINITY;
  // K and V blocks go global -> registers -> LDS between two barriers: all loads of a block
  // are issued before the first LDS write
  constexpr int KPT = 64 * KC / 256;   // 16-byte K chunks per thread and block
  constexpr int VPT = 32 * KC / 256;   // V items (key pair x 8 columns) per thread and block
  auto stage = [&](int kb, bool with_v) {
    uint4 kreg[KPT], vreg[VPT][2];
#pragma unroll
    for (int t = 0; t < KPT; ++t) {
      const int cidx = threadIdx.x + t * 256, key = cidx / KC, ch = cidx % KC;
      int64_t kr = (int64_t)kb * 64 + key;
      kr = kr < seq ? kr : seq - 1;
      kreg[t] = *reinterpret_cast<const uint4*>(k + (r0 + kr) * ldk + (int64_t)hk * HD + ch * 8);
    }
    if (with_v) {
#pragma unroll
      for (int t = 0; t < VPT; ++t) {
        const int it = threadIdx.x + t * 256, kp = it & 31, dc = it >> 5;
        int64_t k0r = (int64_t)kb * 64 + 2 * kp, k1r = k0r + 1;
        k0r = k0r < seq ? k0r : seq - 1;
        k1r = k1r < seq ? k1r : seq - 1;
        vreg[t][0] = *reinterpret_cast<const uint4*>(v + (r0 + k0r) * ldv + (int64_t)hk * HD + dc * 8);
        vreg[t][1] = *reinterpret_cast<const uint4*>(v + (r0 + k1r) * ldv + (int64_t)hk * HD + dc * 8);
      }
    }
#pragma unroll
    for (int t = 0; t < KPT; ++t) {
      const int cidx = threadIdx.x + t * 256, key = cidx / KC, ch = cidx % KC;
      *reinterpret_cast<uint4*>(ks + key * HD + ((ch ^ (key & KSW)) * 8)) = kreg[t];
    }
    if (with_v) {
      // V^T: item (key pair kp, 8-column chunk dc) -> eight words (V[2kp][d], V[2kp+1][d])
#pragma unroll
      for (int t = 0; t < VPT; ++t) {
        const int it = threadIdx.x + t * 256, kp = it & 31, dc = it >> 5;
        const uint32_t aw[4] = {vreg[t][0].x, vreg[t][0].y, vreg[t][0].z, vreg[t][0].w};
        const uint32_t cw[4] = {vreg[t][1].x, vreg[t][1].y, vreg[t][1].z, vreg[t][1].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vt[(dc * 8 + 2 * e) * VW + kp] = (aw[e] & 0xFFFFu) | (cw[e] << 16);
          vt[(dc * 8 + 2 * e + 1) * VW + kp] = (aw[e] >> 16) | (cw[e] & 0xFFFF0000u);
        }
      }
    }
  };

  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    stage(kb, false);
    __syncthreads();
    if ((int64_t)kb * 64 > wq_last) continue;   // wave-uniform: this block is masked for all its queries
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      floatx4 st[4];
      scores_t(b, st);
      if (masked(b, kb)) {
        const int lim = key_limit(b, kb);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (j * 16 + lk * 4 + i <= lim) mq[b] = fmaxf(mq[b], st[j][i]);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) mq[b] = fmaxf(mq[b], st[j][i]);
      }
    }
  }
  // exp(s * scale - max) = 2^(s * c - max * c) with c = scale * log2(e): one fma and the
  // hardware base-2 exponential per score; masked scores become -inf, whose 2^ is 0
  const float c2 = scale * 1.4426950408889634f;
  float mc[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    mq[b] = fmaxf(mq[b], __shfl_xor(mq[b], 16, 64));
    mq[b] = fmaxf(mq[b], __shfl_xor(mq[b], 32, 64));
    mc[b] = mq[b] * c2;
  }

  // pass 2: P = exp(s - max) rounded to bf16, O^T += V^T P^T, l += P (unrounded)
  floatx4 o[ND][QB];
#pragma unroll
  for (int n = 0; n < ND; ++n)
#pragma unroll
    for (int b = 0; b < QB; ++b) o[n][b] = floatx4{0.f, 0.f, 0.f, 0.f};
  float lq[QB];
#pragma unroll
  for (int b = 0; b < QB; ++b) lq[b] = 0.f;
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();
    stage(kb, true);
    __syncthreads();
    if ((int64_t)kb * 64 > wq_last) continue;
    // probabilities of the four q-blocks as B operands: 32-key step c holds keys
    // c*32 + 4*lk + i (block j = 2c) and c*32 + 16 + 4*lk + i (block j = 2c + 1)
    bf16x8 pb[QB][2];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      floatx4 st[4];
      scores_t(b, st);
      if (masked(b, kb)) {
        const int lim = key_limit(b, kb);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (j * 16 + lk * 4 + i > lim) st[j][i] = -INFINITY;
      }
      uint16_t pbits[4][4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float p = __builtin_amdgcn_exp2f(fmaf(st[j][i], c2, -mc[b]));
          lq[b] += p;
          pbits[j][i] = f2bf(p);
        }
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const uint4 u = make_uint4((uint32_t)pbits[2 * c][0] | ((uint32_t)pbits[2 * c][1] << 16),
                                   (uint32_t)pbits[2 * c][2] | ((uint32_t)pbits[2 * c][3] << 16),
                                   (uint32_t)pbits[2 * c + 1][0] | ((uint32_t)pbits[2 * c + 1][1] << 16),
                                   (uint32_t)pbits[2 * c + 1][2] | ((uint32_t)pbits[2 * c + 1][3] << 16));
        pb[b][c] = __builtin_bit_cast(bf16x8, u);
      }
    }
    // A operand: V^T rows d = n*16 + lr, the same keys (two 8-byte reads per step)
#pragma unroll
    for (int n = 0; n < ND; ++n)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const uint32_t* vr = vt + (n * 16 + lr) * VW + c * 16 + lk * 2;
        const uint2 lo = *reinterpret_cast<const uint2*>(vr);
        const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
        const bf16x8 va = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
        for (int b = 0; b < QB; ++b) o[n][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[b][c], o[n][b], 0, 0, 0);
      }
  }
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    lq[b] += __shfl_xor(lq[b], 16, 64);
    lq[b] += __shfl_xor(lq[b], 32, 64);
  }
  // O^T[d = n*16 + 4*lk + i][query = b*16 + lr] / l -> four consecutive columns per store
#pragma unroll
  for (int b = 0; b < QB; ++b) {
    const int64_t qi = q0 + b * 16 + lr;
    if (qi >= seq) continue;
    const float inv = 1.f / lq[b];
    uint16_t* op = out + (r0 + qi) * (int64_t)heads * HD + (int64_t)h * HD;
#pragma unroll
    for (int n = 0; n < ND; ++n) {
      const uint2 w2 = make_uint2((uint32_t)f2bf(o[n][b][0] * inv) | ((uint32_t)f2bf(o[n][b][1] * inv) << 16),
                                  (uint32_t)f2bf(o[n][b][2] * inv) | ((uint32_t)f2bf(o[n][b][3] * inv) << 16));
      *reinterpret_cast<uint2*>(op + n * 16 + lk * 4) = w2;
    }
  }
}

// Whole sequence resident (seq <= 256): one workgroup per (sequence, key/value head, group
// of up to four of its query heads), WPH = 4 / QB waves per query head.  K and V^T of the
// sequence go into LDS once (K rows chunk-swizzled, V^T as key-pair words, as above), and
// both passes of the softmax (row maxima, then P = bf16(exp(s - max)) with l summed
// unrounded and O^T += V^T P^T) read them from there: nothing is staged twice and no
// barrier is needed after the load.  A wave takes units of QB 16-query blocks (each K and
// V^T fragment read from LDS feeds QB MFMAs).  Units are dealt so that every wave of a head
// gets the same causal work: with QB = 2 the two waves take the units u with u mod 4 in
// {w, 3 - w}; with QB = 1 wave w takes the units with u mod 4 = w.  The launcher runs
// QB = 1 (sixteen waves), which measured faster than two blocks per wave.
// rc, rs (nullable): rotary tables [seq][HD / 2] fp32; when given, q and k are rotated as
// they are read (rotate-half, the arithmetic and bf16 rounding of the rotary pass).
template <int HD, int QB>
__global__ void __launch_bounds__(1024 / QB, 1) attention_res_kernel(const uint16_t* __restrict__ q, int64_t ldq,
                                                                   const uint16_t* __restrict__ k, int64_t ldk,
                                                                   const uint16_t* __restrict__ v, int64_t ldv,
                                                                   int64_t seq, int heads, int kv_heads, float scale,
                                                                   uint16_t* __restrict__ out, const float* __restrict__ rc,
                                                                   const float* __restrict__ rs) {
  constexpr int KC = HD / 8;    // 16-byte chunks per row
  constexpr int KS = HD / 32;   // 32-deep steps over the head dimension
  constexpr int ND = HD / 16;   // 16-row blocks of the head dimension
  constexpr int SMAX = 256;
  constexpr int WPH = 4 / QB;   // waves per query head
  // Padding and swizzle keep the fragment reads free of LDS bank conflicts: V^T rows of
  // 130 words, K chunks XOR-swizzled over 16 rows (8 when a row has only 8 chunks)
  constexpr int VW = SMAX / 2 + 2;
  constexpr int KSW = KC >= 16 ? 15 : 7;
  __shared__ __align__(16) uint16_t ks[SMAX * HD];   // K [key][hd], chunk-swizzled
  __shared__ __align__(16) uint32_t vt[HD * VW];     // V^T [d][key pair]
  const int G = heads / kv_heads;
  const int HG = G < 4 ? G : 4;
  const int sub = G / HG;
  const int nthr = 64 * WPH * HG;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int hk = blockIdx.y / sub;
  const int h = hk * G + (blockIdx.y % sub) * HG + (wave % HG);
  const int hv = wave / HG;   // which of the head's waves
  const int64_t r0 = (int64_t)blockIdx.x * seq;
  const int nk = (int)((seq + 63) / 64) * 64;   // keys held (whole 64-key blocks)

  // ---- K and V^T of the sequence into LDS; rows past seq are copies of the last row, so
  // masked probabilities (exactly zero) never meet non-finite values.  Loads go out in
  // batches (eight K chunks, then four V key pairs, per thread) before their LDS writes.
  const int nkc = nk * KC, nvi = (nk / 2) * KC;
  // with rotary tables (rc, rs: [seq][HD / 2] fp32) q and k are rotated as they are read,
  // rounded to bf16 as a separate rotary pass would store them: a thread takes chunk ch of a
  // key row with its partner ch + KC / 2
  constexpr int KH = KC / 2;
  if (rc != nullptr) {
    const int nkp = nk * KH;
    for (int c0 = threadIdx.x; c0 < nkp; c0 += 2 * nthr) {
      uint4 ka[2], kb[2];
      float4 cva[2][2], sva[2][2];   // the 8 cos / sin values of the chunk's pairs
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = c0 + u * nthr < nkp ? c0 + u * nthr : nkp - 1;
        const int key = c / KH, ch = c % KH;
        const int64_t row = key < seq ? key : seq - 1;
        const uint16_t* kr = k + (r0 + row) * ldk + (int64_t)hk * HD;
        ka[u] = *reinterpret_cast<const uint4*>(kr + ch * 8);
        kb[u] = *reinterpret_cast<const uint4*>(kr + (ch + KH) * 8);
        const float4* cp = reinterpret_cast<const float4*>(rc + row * (HD / 2) + ch * 8);
        const float4* sp = reinterpret_cast<const float4*>(rs + row * (HD / 2) + ch * 8);
        cva[u][0] = cp[0], cva[u][1] = cp[1], sva[u][0] = sp[0], sva[u][1] = sp[1];
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = c0 + u * nthr;
        if (c < nkp) {
          const int key = c / KH, ch = c % KH;
          const float cv[8] = {cva[u][0].x, cva[u][0].y, cva[u][0].z, cva[u][0].w,
                               cva[u][1].x, cva[u][1].y, cva[u][1].z, cva[u][1].w};
          const float sv[8] = {sva[u][0].x, sva[u][0].y, sva[u][0].z, sva[u][0].w,
                               sva[u][1].x, sva[u][1].y, sva[u][1].z, sva[u][1].w};
          const uint32_t aw[4] = {ka[u].x, ka[u].y, ka[u].z, ka[u].w}, bw[4] = {kb[u].x, kb[u].y, kb[u].z, kb[u].w};
          uint32_t ao[4], bo[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            uint16_t lo_r[2], hi_r[2];
#pragma unroll
            for (int q2 = 0; q2 < 2; ++q2) {
              const float lo = bf2f((uint16_t)(q2 ? aw[e] >> 16 : aw[e] & 0xFFFF));
              const float hi = bf2f((uint16_t)(q2 ? bw[e] >> 16 : bw[e] & 0xFFFF));
              lo_r[q2] = f2bf(rot_lo(lo, hi, cv[2 * e + q2], sv[2 * e + q2]));
              hi_r[q2] = f2bf(rot_hi(lo, hi, cv[2 * e + q2], sv[2 * e + q2]));
            }
            ao[e] = (uint32_t)lo_r[0] | ((uint32_t)lo_r[1] << 16);
            bo[e] = (uint32_t)hi_r[0] | ((uint32_t)hi_r[1] << 16);
          }
          *reinterpret_cast<uint4*>(ks + key * HD + ((ch ^ (key & KSW)) * 8)) = make_uint4(ao[0], ao[1], ao[2], ao[3]);
          *reinterpret_cast<uint4*>(ks + key * HD + (((ch + KH) ^ (key & KSW)) * 8)) =
              make_uint4(bo[0], bo[1], bo[2], bo[3]);
        }
      }
    }
  }
  for (int c0 = threadIdx.x; c0 < (rc != nullptr ? 0 : nkc); c0 += 8 * nthr) {
    uint4 kr[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = c0 + u * nthr < nkc ? c0 + u * nthr : nkc - 1;   // in range; written only below nkc
      const int key = c / KC, ch = c % KC;
      const int64_t row = key < seq ? key : seq - 1;
      kr[u] = *reinterpret_cast<const uint4*>(k + (r0 + row) * ldk + (int64_t)hk * HD + ch * 8);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = c0 + u * nthr;
      if (c < nkc) {
        const int key = c / KC, ch = c % KC;
        *reinterpret_cast<uint4*>(ks + key * HD + ((ch ^ (key & KSW)) * 8)) = kr[u];
      }
    }
  }
  for (int i0 = threadIdx.x; i0 < nvi; i0 += 4 * nthr) {
    uint4 va[4], vb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int it = i0 + u * nthr < nvi ? i0 + u * nthr : nvi - 1;
      const int kp = it % (nk / 2), dc = it / (nk / 2);
      int64_t k0r = 2 * kp, k1r = k0r + 1;
      k0r = k0r < seq ? k0r : seq - 1;
      k1r = k1r < seq ? k1r : seq - 1;
      va[u] = *reinterpret_cast<const uint4*>(v + (r0 + k0r) * ldv + (int64_t)hk * HD + dc * 8);
      vb[u] = *reinterpret_cast<const uint4*>(v + (r0 + k1r) * ldv + (int64_t)hk * HD + dc * 8);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int it = i0 + u * nthr;
      if (it < nvi) {
        const int kp = it % (nk / 2), dc = it / (nk / 2);
        const uint32_t aw[4] = {va[u].x, va[u].y, va[u].z, va[u].w};
        const uint32_t cw[4] = {vb[u].x, vb[u].y, vb[u].z, vb[u].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vt[(dc * 8 + 2 * e) * VW + kp] = (aw[e] & 0xFFFFu) | (cw[e] << 16);
          vt[(dc * 8 + 2 * e + 1) * VW + kp] = (aw[e] >> 16) | (cw[e] & 0xFFFF0000u);
        }
      }
    }
  }
  __syncthreads();

  const int nunit = (int)((seq + 16 * QB - 1) / (16 * QB));
  for (int un = 0; un < nunit; ++un) {
    if (QB == 2 ? ((un & 3) != hv && (un & 3) != 3 - hv) : ((un & 3) != hv)) continue;
    const int64_t q0 = (int64_t)un * 16 * QB;
    // Q fragments (B operand): q-block b, row lr, depth kk*32 + lk*8
    bf16x8 qf[QB][KS];
    int lastq[QB];   // this lane's query in q-block b, clamped to the sequence
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      int64_t qr = q0 + b * 16 + lr;
      qr = qr < seq ? qr : seq - 1;
      lastq[b] = (int)qr;
      const uint16_t* qp = q + (r0 + qr) * ldq + (int64_t)h * HD;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qf[b][kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 32 + lk * 8);
      if (rc != nullptr) {
        // depth kk*32 + lk*8 + e (kk < KS / 2) pairs with the same lane's kk + KS / 2; the
        // tables are read as aligned 16-byte vectors (rows of HD / 2 floats)
#pragma unroll
        for (int kk = 0; kk < KS / 2; ++kk) {
          const float4* cp = reinterpret_cast<const float4*>(rc + qr * (HD / 2) + kk * 32 + lk * 8);
          const float4* sp = reinterpret_cast<const float4*>(rs + qr * (HD / 2) + kk * 32 + lk * 8);
          const float4 c0 = cp[0], c1 = cp[1], s0 = sp[0], s1 = sp[1];
          const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
          const float sv[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
          bf16x8 lo8 = qf[b][kk], hi8 = qf[b][kk + KS / 2];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float lo = (float)lo8[e], hi = (float)hi8[e];
            lo8[e] = (__bf16)rot_lo(lo, hi, cv[e], sv[e]);
            hi8[e] = (__bf16)rot_hi(lo, hi, cv[e], sv[e]);
          }
          qf[b][kk] = lo8;
          qf[b][kk + KS / 2] = hi8;
        }
      }
    }
    const int64_t ulast = q0 + 16 * QB - 1 < seq - 1 ? q0 + 16 * QB - 1 : seq - 1;
    const int nkb = (int)(ulast / 64) + 1;
    // S^T of key block kb for the unit's q-blocks: st[b][j] holds S^T[key = j*16 + 4*lk + i][query lr]
    auto scores_t = [&](int kb, floatx4 (&st)[QB][4]) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int b = 0; b < QB; ++b) st[b][j] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const int key = kb * 64 + j * 16 + lr;
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(ks + key * HD + (((kk * 4 + lk) ^ (key & KSW)) * 8));
#pragma unroll
          for (int b = 0; b < QB; ++b)
            st[b][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[b][kk], st[b][j], 0, 0, 0);
        }
      }
    };
    // a key block needs the causal mask only where it reaches past the q-block's first
    // query (or past the sequence); the test is uniform over the wave
    auto masked = [&](int b, int kb) {
      return (int64_t)kb * 64 + 63 > (q0 + b * 16 < seq - 1 ? q0 + b * 16 : seq - 1);
    };
    // pass 1: the row maxima of the raw scores over visible keys (key <= query); scaling by
    // a positive constant keeps the maximiser, so the scale is applied once, to the maximum
    float mq[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) mq[b] = -INFINITY;
    for (int kb = 0; kb < nkb; ++kb) {
      floatx4 st[QB][4];
      scores_t(kb, st);
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        if (masked(b, kb)) {
          const int lim = lastq[b] - kb * 64;
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (j * 16 + lk * 4 + i <= lim) mq[b] = fmaxf(mq[b], st[b][j][i]);
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i) mq[b] = fmaxf(mq[b], st[b][j][i]);
        }
      }
    }
    // exp(s * scale - max) = 2^(s * c - max * c) with c = scale * log2(e): one fma and the
    // hardware base-2 exponential per score; masked scores become -inf, whose 2^ is 0
    const float c2 = scale * 1.4426950408889634f;
    float mc[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      mq[b] = fmaxf(mq[b], __shfl_xor(mq[b], 16, 64));
      mq[b] = fmaxf(mq[b], __shfl_xor(mq[b], 32, 64));
      mc[b] = mq[b] * c2;
    }
    // pass 2: P = exp(s - max) rounded to bf16, O^T += V^T P^T, l += P (unrounded)
    floatx4 o[ND][QB];
#pragma unroll
    for (int n = 0; n < ND; ++n)
#pragma unroll
      for (int b = 0; b < QB; ++b) o[n][b] = floatx4{0.f, 0.f, 0.f, 0.f};
    float lq[QB];
#pragma unroll
    for (int b = 0; b < QB; ++b) lq[b] = 0.f;
    for (int kb = 0; kb < nkb; ++kb) {
      floatx4 st[QB][4];
      scores_t(kb, st);
      // B operands: 32-key step c holds keys c*32 + 4*lk + i (j = 2c) and c*32 + 16 + 4*lk + i
      bf16x8 pb[QB][2];
#pragma unroll
      for (int b = 0; b < QB; ++b) {
        if (masked(b, kb)) {
          const int lim = lastq[b] - kb * 64;
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (j * 16 + lk * 4 + i > lim) st[b][j][i] = -INFINITY;
        }
        uint16_t pbits[4][4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float pv = __builtin_amdgcn_exp2f(fmaf(st[b][j][i], c2, -mc[b]));
            lq[b] += pv;
            pbits[j][i] = f2bf(pv);
          }
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const uint4 u = make_uint4((uint32_t)pbits[2 * c][0] | ((uint32_t)pbits[2 * c][1] << 16),
                                     (uint32_t)pbits[2 * c][2] | ((uint32_t)pbits[2 * c][3] << 16),
                                     (uint32_t)pbits[2 * c + 1][0] | ((uint32_t)pbits[2 * c + 1][1] << 16),
                                     (uint32_t)pbits[2 * c + 1][2] | ((uint32_t)pbits[2 * c + 1][3] << 16));
          pb[b][c] = __builtin_bit_cast(bf16x8, u);
        }
      }
      // A operand: V^T rows d = n*16 + lr, the same keys (two 8-byte reads per step)
#pragma unroll
      for (int n = 0; n < ND; ++n)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const uint32_t* vr = vt + (n * 16 + lr) * VW + kb * 32 + c * 16 + lk * 2;
          const uint2 lo = *reinterpret_cast<const uint2*>(vr);
          const uint2 hi = *reinterpret_cast<const uint2*>(vr + 8);
          const bf16x8 va = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
          for (int b = 0; b < QB; ++b) o[n][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb[b][c], o[n][b], 0, 0, 0);
        }
    }
    // O^T[d = n*16 + 4*lk + i][query lr] / l -> four consecutive columns per store
#pragma unroll
    for (int b = 0; b < QB; ++b) {
      lq[b] += __shfl_xor(lq[b], 16, 64);
      lq[b] += __shfl_xor(lq[b], 32, 64);
      const int64_t qi = q0 + b * 16 + lr;
      if (qi >= seq) continue;
      const float inv = 1.f / lq[b];
      uint16_t* op = out + (r0 + qi) * (int64_t)heads * HD + (int64_t)h * HD;
#pragma unroll
      for (int n = 0; n < ND; ++n) {
        const uint2 w2 = make_uint2((uint32_t)f2bf(o[n][b][0] * inv) | ((uint32_t)f2bf(o[n][b][1] * inv) << 16),
                                    (uint32_t)f2bf(o[n][b][2] * inv) | ((uint32_t)f2bf(o[n][b][3] * inv) << 16));
        *reinterpret_cast<uint2*>(op + n * 16 + lk * 4) = w2;
      }
    }
  }
}

unsigned grid1d(int64_t n) {
  int64_t g = (n + 255) / 256;
  return (unsigned)(g < 1 ? 1 : (g > 65535 ? 65535 : g));
}

}  // namespace
}  // namespace zoact

using namespace zoact;

#define ZO_CHECK(cond, msg)                                 \
  do {                                                      \
    if (!(cond)) return zoact::set_error(ZOACT_E_INVALID, msg); \
  } while (0)

static zoact_status launched(const char* who) {
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess) return ZOACT_OK;
  std::string m = std::string(who) + ": " + hipGetErrorString(e);
  return zoact::set_error(ZOACT_E_HIP, m.c_str());
}

extern "C" zoact_status zoact_embed(const int32_t* tokens, int64_t n_tok, int32_t distinct_halves, int64_t vocab,
                                    const void* table, const void* pos, int64_t max_pos, int32_t pos_offset,
                                    int64_t seq, int64_t d, int32_t dtype, void* out, zoact_stream stream) {
  ZO_CHECK(tokens && table && out, "embed: NULL pointer");
  ZO_CHECK(distinct_halves == 0 || distinct_halves == 1, "embed: distinct_halves must be 0 or 1");
  ZO_CHECK(n_tok >= 1 && vocab >= 1 && d >= 1 && seq >= 1, "embed: empty shape");
  ZO_CHECK(dtype == ZOACT_F32 || dtype == ZOACT_BF16, "embed: dtype must be F32 or BF16");
  ZO_CHECK(pos == nullptr || (max_pos >= 1 && pos_offset >= 0), "embed: bad position table");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int64_t work = n_tok * d * (distinct_halves ? 2 : 1);
  if (dtype == ZOACT_BF16)
    embed_kernel<uint16_t><<<grid1d(work), 256, 0, s>>>(tokens, n_tok, distinct_halves, vocab, (const uint16_t*)table,
                                                        (const uint16_t*)pos, max_pos, pos_offset, seq, d,
                                                        (uint16_t*)out);
  else
    embed_kernel<float><<<grid1d(work), 256, 0, s>>>(tokens, n_tok, distinct_halves, vocab, (const float*)table,
                                                     (const float*)pos, max_pos, pos_offset, seq, d, (float*)out);
  return launched("embed");
}

extern "C" zoact_status zoact_rmsnorm(const void* x, const void* w, int64_t rows, int64_t d, float eps, int32_t dtype,
                                      void* y, zoact_stream stream) {
  ZO_CHECK(x && w && y, "rmsnorm: NULL pointer");
  ZO_CHECK(rows >= 1 && d >= 1 && rows <= 0x7FFFFFFF, "rmsnorm: bad shape");
  ZO_CHECK(dtype == ZOACT_F32 || dtype == ZOACT_BF16, "rmsnorm: dtype must be F32 or BF16");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool vec = dtype == ZOACT_BF16 && ((uintptr_t)x % 16) == 0 && ((uintptr_t)w % 16) == 0 && ((uintptr_t)y % 16) == 0;
  if (vec && d == 2048)
    rmsnorm_bf16_vec_kernel<1><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w, d, eps, (uint16_t*)y);
  else if (vec && d == 4096)
    rmsnorm_bf16_vec_kernel<2><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w, d, eps, (uint16_t*)y);
  else if (vec && d == 6144)
    rmsnorm_bf16_vec_kernel<3><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w, d, eps, (uint16_t*)y);
  else if (vec && d == 8192)
    rmsnorm_bf16_vec_kernel<4><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w, d, eps, (uint16_t*)y);
  else if (dtype == ZOACT_BF16)
    rmsnorm_kernel<uint16_t><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w, d, eps, (uint16_t*)y);
  else
    rmsnorm_kernel<float><<<(unsigned)rows, 256, 0, s>>>((const float*)x, (const float*)w, d, eps, (float*)y);
  return launched("rmsnorm");
}

extern "C" zoact_status zoact_layernorm(const void* x, const void* w, const void* b, int64_t rows, int64_t d, float eps,
                                        int32_t dtype, void* y, zoact_stream stream) {
  ZO_CHECK(x && w && b && y, "layernorm: NULL pointer");
  ZO_CHECK(rows >= 1 && d >= 1 && rows <= 0x7FFFFFFF, "layernorm: bad shape");
  ZO_CHECK(dtype == ZOACT_F32 || dtype == ZOACT_BF16, "layernorm: dtype must be F32 or BF16");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool vec = dtype == ZOACT_BF16 && d % 8 == 0 && d <= 8192 && ((uintptr_t)x % 16) == 0 &&
                   ((uintptr_t)w % 16) == 0 && ((uintptr_t)b % 16) == 0 && ((uintptr_t)y % 16) == 0;
  const int vpt = (int)((d / 8 + 255) / 256);
#define ZO_LN(V)                                                                                     \
  layernorm_bf16_vec_kernel<V><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w, \
                                                               (const uint16_t*)b, d, eps, (uint16_t*)y)
  if (vec && vpt <= 1) ZO_LN(1);
  else if (vec && vpt == 2) ZO_LN(2);
  else if (vec && vpt == 3) ZO_LN(3);
  else if (vec) ZO_LN(4);
#undef ZO_LN
  else if (dtype == ZOACT_BF16)
    layernorm_kernel<uint16_t><<<(unsigned)rows, 256, 0, s>>>((const uint16_t*)x, (const uint16_t*)w,
                                                              (const uint16_t*)b, d, eps, (uint16_t*)y);
  else
    layernorm_kernel<float><<<(unsigned)rows, 256, 0, s>>>((const float*)x, (const float*)w, (const float*)b, d, eps,
                                                           (float*)y);
  return launched("layernorm");
}

extern "C" zoact_status zoact_rope(void* x, int32_t dtype, int64_t rows, int64_t ld, int64_t col0, int32_t n_heads,
                                   int32_t head_dim, int64_t seq, const float* cos_t, const float* sin_t,
                                   zoact_stream stream) {
  ZO_CHECK(x && cos_t && sin_t, "rope: NULL pointer");
  ZO_CHECK(rows >= 1 && seq >= 1 && n_heads >= 1 && head_dim >= 2 && head_dim % 2 == 0, "rope: bad shape");
  ZO_CHECK(col0 >= 0 && col0 + (int64_t)n_heads * head_dim <= ld, "rope: heads exceed the row");
  ZO_CHECK(dtype == ZOACT_F32 || dtype == ZOACT_BF16, "rope: dtype must be F32 or BF16");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const int64_t total = rows * n_heads * (head_dim / 2);
  const bool vec = dtype == ZOACT_BF16 && (head_dim / 2) % 8 == 0 && ld % 8 == 0 && col0 % 8 == 0 &&
                   ((uintptr_t)x % 16) == 0 && ((uintptr_t)cos_t % 16) == 0 && ((uintptr_t)sin_t % 16) == 0;
  if (vec)
    rope_bf16_vec_kernel<<<grid1d(total / 8), 256, 0, s>>>((uint16_t*)x, rows, ld, col0, n_heads, head_dim, seq, cos_t,
                                                           sin_t);
  else if (dtype == ZOACT_BF16)
    rope_kernel<uint16_t><<<grid1d(total), 256, 0, s>>>((uint16_t*)x, rows, ld, col0, n_heads, head_dim, seq, cos_t, sin_t);
  else
    rope_kernel<float><<<grid1d(total), 256, 0, s>>>((float*)x, rows, ld, col0, n_heads, head_dim, seq, cos_t, sin_t);
  return launched("rope");
}

// Whole sequence resident in LDS: bf16, groups of four or more query heads per key/value
// head (sixteen waves per workgroup), seq <= 256, and a grid of one workgroup per
// (sequence, key/value head, four query heads) that covers every compute unit; smaller
// grids run the staged kernel, which splits the queries over more workgroups.
static bool attention_resident(int32_t dtype, int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads,
                               int32_t head_dim) {
  if (dtype != ZOACT_BF16 || (head_dim != 64 && head_dim != 128) || n_kv_heads < 1 || n_heads % n_kv_heads) return false;
  const int G = n_heads / n_kv_heads;
  const int ncu = cu_count();
  return ncu > 0 && G % 4 == 0 && seq <= 256 && (int64_t)n_kv_heads * (G / 4) <= 65535 &&
         n_seq * n_kv_heads * (G / 4) >= ncu;
}

// Argument checks of the attention entry points (before anything is enqueued).
static zoact_status attention_check(const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv,
                                    int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                    int32_t dtype, const void* out) {
  ZO_CHECK(q && k && v && out, "attention: NULL pointer");
  ZO_CHECK(n_seq >= 1 && seq >= 1 && n_heads >= 1 && n_kv_heads >= 1 && n_heads % n_kv_heads == 0,
           "attention: bad shape or head grouping");
  ZO_CHECK(ldq >= (int64_t)n_heads * head_dim && ldk >= (int64_t)n_kv_heads * head_dim &&
               ldv >= (int64_t)n_kv_heads * head_dim,
           "attention: row strides smaller than the heads");
  ZO_CHECK(n_seq <= 65535 && n_heads <= 65535, "attention: grid too large");
  if (dtype == ZOACT_BF16) {
    ZO_CHECK(head_dim == 64 || head_dim == 128, "attention: bf16 head_dim must be 64 or 128");
    ZO_CHECK(ldq % 8 == 0 && ldk % 8 == 0 && ldv % 8 == 0, "attention: bf16 strides must be multiples of 8");
  } else if (dtype == ZOACT_F32) {
    ZO_CHECK(head_dim <= 128 && seq * head_dim <= 4096, "attention: fp32 path needs head_dim <= 128, seq*hd <= 4096");
  } else {
    return zoact::set_error(ZOACT_E_INVALID, "attention: dtype must be F32 or BF16");
  }
  return ZOACT_OK;
}

static zoact_status attention_impl(const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv,
                                   int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                                   float scale, int32_t dtype, void* out, const float* rc, const float* rs,
                                   zoact_stream stream) {
  const zoact_status chk = attention_check(q, ldq, k, ldk, v, ldv, n_seq, seq, n_heads, n_kv_heads, head_dim, dtype,
                                           out);
  if (chk != ZOACT_OK) return chk;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (dtype == ZOACT_BF16) {
    const int G = n_heads / n_kv_heads;
    if (attention_resident(dtype, n_seq, seq, n_heads, n_kv_heads, head_dim)) {
      const dim3 g1((unsigned)n_seq, (unsigned)(n_kv_heads * (G / 4)));
      if (head_dim == 128)
        attention_res_kernel<128, 1><<<g1, 1024, 0, s>>>((const uint16_t*)q, ldq, (const uint16_t*)k, ldk,
                                                         (const uint16_t*)v, ldv, seq, n_heads, n_kv_heads, scale,
                                                         (uint16_t*)out, rc, rs);
      else
        attention_res_kernel<64, 1><<<g1, 1024, 0, s>>>((const uint16_t*)q, ldq, (const uint16_t*)k, ldk,
                                                        (const uint16_t*)v, ldv, seq, n_heads, n_kv_heads, scale,
                                                        (uint16_t*)out, rc, rs);
      return launched("attention");
    }
    ZO_CHECK(rc == nullptr, "attention: rotary tables reach only the resident kernel");
    if ((G == 1 || G == 2 || G % 4 == 0) && (int64_t)n_kv_heads * (G < 4 ? 1 : G / 4) <= 65535) {
      constexpr int QB = 2;                     // 16-query blocks per wave
      const int HG = G < 4 ? G : 4;
      const int QT = 64 * QB / HG;
      const dim3 g2((unsigned)((seq + QT - 1) / QT), (unsigned)(n_kv_heads * (G / HG)), (unsigned)n_seq);
      if (head_dim == 128)
        attention_gqa_kernel<128, QB><<<g2, 256, 0, s>>>((const uint16_t*)q, ldq, (const uint16_t*)k, ldk,
                                                         (const uint16_t*)v, ldv, seq, n_heads, n_kv_heads, scale,
                                                         (uint16_t*)out);
      else
        attention_gqa_kernel<64, QB><<<g2, 256, 0, s>>>((const uint16_t*)q, ldq, (const uint16_t*)k, ldk,
                                                        (const uint16_t*)v, ldv, seq, n_heads, n_kv_heads, scale,
                                                        (uint16_t*)out);
      return launched("attention");
    }
    const dim3 grid((unsigned)((seq + 63) / 64), (unsigned)n_heads, (unsigned)n_seq);
    if (head_dim == 128)
      attention_bf16_kernel<128><<<grid, 256, 0, s>>>((const uint16_t*)q, ldq, (const uint16_t*)k, ldk,
                                                      (const uint16_t*)v, ldv, seq, n_heads, n_kv_heads, scale,
                                                      (uint16_t*)out);
    else
      attention_bf16_kernel<64><<<grid, 256, 0, s>>>((const uint16_t*)q, ldq, (const uint16_t*)k, ldk,
                                                     (const uint16_t*)v, ldv, seq, n_heads, n_kv_heads, scale,
                                                     (uint16_t*)out);
  } else if (dtype == ZOACT_F32) {
    ZO_CHECK(head_dim <= 128 && seq * head_dim <= 4096, "attention: fp32 path needs head_dim <= 128, seq*hd <= 4096");
    const dim3 grid((unsigned)n_heads, (unsigned)n_seq);
    attention_f32_kernel<<<grid, 256, (size_t)2 * seq * head_dim * sizeof(float), s>>>(
        (const float*)q, ldq, (const float*)k, ldk, (const float*)v, ldv, seq, n_heads, n_kv_heads, head_dim, scale,
        (float*)out);
  } else {
    return zoact::set_error(ZOACT_E_INVALID, "attention: dtype must be F32 or BF16");
  }
  return launched("attention");
}

extern "C" zoact_status zoact_attention(const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v,
                                        int64_t ldv, int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads,
                                        int32_t head_dim, float scale, int32_t dtype, void* out, zoact_stream stream) {
  return attention_impl(q, ldq, k, ldk, v, ldv, n_seq, seq, n_heads, n_kv_heads, head_dim, scale, dtype, out, nullptr,
                        nullptr, stream);
}

extern "C" int32_t zoact_attention_rope_in_place(int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads,
                                                 int32_t head_dim, int32_t dtype) {
  if ((dtype != ZOACT_F32 && dtype != ZOACT_BF16) || n_seq < 1 || seq < 1 || n_heads < 1 || n_kv_heads < 1 ||
      head_dim < 1 || n_heads % n_kv_heads != 0)
    return -1;
  return attention_resident(dtype, n_seq, seq, n_heads, n_kv_heads, head_dim) ? 0 : 1;
}

extern "C" zoact_status zoact_attention_rope(void* q, int64_t ldq, void* k, int64_t ldk, const void* v, int64_t ldv,
                                             int64_t n_seq, int64_t seq, int32_t n_heads, int32_t n_kv_heads,
                                             int32_t head_dim, float scale, int32_t dtype, const float* cos_t,
                                             const float* sin_t, void* out, zoact_stream stream) {
  const zoact_status chk = attention_check(q, ldq, k, ldk, v, ldv, n_seq, seq, n_heads, n_kv_heads, head_dim, dtype,
                                           out);
  if (chk != ZOACT_OK) return chk;
  ZO_CHECK(cos_t && sin_t, "attention_rope: NULL rotary table");
  ZO_CHECK(((uintptr_t)cos_t % 16) == 0 && ((uintptr_t)sin_t % 16) == 0, "attention_rope: tables must be 16-byte aligned");
  if (attention_resident(dtype, n_seq, seq, n_heads, n_kv_heads, head_dim))
    return attention_impl(q, ldq, k, ldk, v, ldv, n_seq, seq, n_heads, n_kv_heads, head_dim, scale, dtype, out, cos_t,
                          sin_t, stream);
  // other shapes: the rotary pass in place, then attention
  zoact_status st = zoact_rope(q, dtype, n_seq * seq, ldq, 0, n_heads, head_dim, seq, cos_t, sin_t, stream);
  if (st != ZOACT_OK) return st;
  st = zoact_rope(k, dtype, n_seq * seq, ldk, 0, n_kv_heads, head_dim, seq, cos_t, sin_t, stream);
  if (st != ZOACT_OK) return st;
  return attention_impl(q, ldq, k, ldk, v, ldv, n_seq, seq, n_heads, n_kv_heads, head_dim, scale, dtype, out, nullptr,
                        nullptr, stream);
}

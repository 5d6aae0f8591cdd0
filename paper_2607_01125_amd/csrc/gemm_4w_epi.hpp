// Pieces shared by the four-wave fused GEMM schedules (32-deep and 64-deep stages): wait
// counts, the workgroup barrier, buffer descriptors, and the epilogue that stages each
// wave's 128 x 128 accumulator tile through LDS and applies bias, residual, activation
// (or the fused regression loss) with one rounding.
#pragma once
#include <math.h>

#include "gemm_common.hpp"

namespace zoact {
namespace gemm {

typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0,15:14], expcnt[6:4], lgkmcnt[11:8])
constexpr int WAIT_VM0 = 0x0F70;
constexpr int WAIT_VM8 = 0x0F78;
constexpr int WAIT_VM12 = 0x0F7C;
constexpr int WAIT_VM16 = 0x4F70;
constexpr int WAIT_LGKM0 = 0xC07F;
constexpr int WAIT_ALL0 = 0x0070;

__device__ __forceinline__ void barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

template <int EPI, bool OUT_F32>
__device__ __forceinline__ void epilogue_4w(const GemmArgs& a, floatx4 (&acc)[8][8], uint16_t* lds, int wave,
                                            int lane, int64_t m0, int64_t n0, int half, int tm, int tn) {
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128;   // features of this wave
  const int wm0 = (wave >> 1) * 128;  // tokens of this wave
  // ---- epilogue through LDS: each wave stages its 128 x 128 tile as fp32 in its own 32 KB
  // slice of the (now idle) stage area, 64 tokens at a time, then applies bias, residual and
  // activation on rows and stores 16 bytes per lane along the feature axis (one rounding).
  __builtin_amdgcn_s_waitcnt(WAIT_ALL0);
  barrier();
  float* ep = reinterpret_cast<float*>(lds) + wave * (64 * 132);
  constexpr int LDR = 132;  // padded fp32 row
  float sq_acc = 0.f;       // EPI_MSE: this lane's sum of squared errors
  // EPI_MSE: the target rows this lane meets in both passes, loaded up front so their
  // latency overlaps the staging instead of stalling every row (clamped in bounds; rows
  // past the ends are skipped below)
  uint4 tpre[2][16];
  if constexpr (EPI == EPI_MSE) {
    const int64_t nc = min((int64_t)(n0 + wn0 + (lane & 15) * 8), a.N - 8);
#pragma unroll
    for (int ps = 0; ps < 2; ++ps)
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int64_t m = min((int64_t)(m0 + wm0 + ps * 64 + (lane >> 4) + 4 * it), a.T - 1);
        tpre[ps][it] = *reinterpret_cast<const uint4*>(a.tgt + m * a.N + nc);
      }
  }
  const int64_t nout = (EPI == ZOACT_EPI_SWIGLU) ? a.N / 2 : a.N;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const int j = pass * 4 + jj;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<floatx4*>(ep + (jj * 16 + lr) * LDR + i * 16 + lk * 4) = acc[i][j];
    }
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    if (EPI == ZOACT_EPI_SWIGLU) {
      // 64 output features per wave: lane -> chunk c = lane & 7 (8 outputs), rows lane >> 3 + 8 it
      const int c = lane & 7;
      const int g0 = (c >> 1) * 32 + (c & 1) * 8;           // fused gate index inside the wave
      const int64_t ng = n0 + wn0 + g0;
      const int64_t fo = (n0 + wn0) / 2 + c * 8;           // output feature
      float bg[8], bu[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bg[e] = (a.bias && ng < a.N) ? bf2f(a.bias[ng + e]) : 0.f;
        bu[e] = (a.bias && ng < a.N) ? bf2f(a.bias[ng + 16 + e]) : 0.f;
      }
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const int tl = (lane >> 3) + 8 * it;
        const int64_t m = m0 + wm0 + pass * 64 + tl;
        if (m >= a.T || ng >= a.N) continue;
        const int64_t row = (int64_t)half * a.T + m;
        const floatx4 g_lo = *reinterpret_cast<const floatx4*>(ep + tl * LDR + g0);
        const floatx4 g_hi = *reinterpret_cast<const floatx4*>(ep + tl * LDR + g0 + 4);
        const floatx4 u_lo = *reinterpret_cast<const floatx4*>(ep + tl * LDR + g0 + 16);
        const floatx4 u_hi = *reinterpret_cast<const floatx4*>(ep + tl * LDR + g0 + 20);
        float o[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = silu(g_lo[e] + bg[e]) * (u_lo[e] + bu[e]);
          o[e + 4] = silu(g_hi[e] + bg[e + 4]) * (u_hi[e] + bu[e + 4]);
        }
        if (a.resid) {
          const uint4 rv = *reinterpret_cast<const uint4*>(a.resid + row * nout + fo);
          const uint32_t rw[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            o[2 * e] += bf2f((uint16_t)(rw[e] & 0xFFFF));
            o[2 * e + 1] += bf2f((uint16_t)(rw[e] >> 16));
          }
        }
        if (OUT_F32) {
          float* yp = reinterpret_cast<float*>(a.y) + row * nout + fo;
          *reinterpret_cast<float4*>(yp) = make_float4(o[0], o[1], o[2], o[3]);
          *reinterpret_cast<float4*>(yp + 4) = make_float4(o[4], o[5], o[6], o[7]);
        } else {
          *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.y) + row * nout + fo) =
              make_uint4(pack2(f2bf(o[0]), f2bf(o[1])), pack2(f2bf(o[2]), f2bf(o[3])), pack2(f2bf(o[4]), f2bf(o[5])),
                         pack2(f2bf(o[6]), f2bf(o[7])));
        }
      }
    } else {
      // 128 features per wave: lane -> chunk c = lane & 15 (8 features), rows lane >> 4 + 4 it
      const int c = lane & 15;
      const int64_t n = n0 + wn0 + c * 8;
      float bb[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) bb[e] = (a.bias && n < a.N) ? bf2f(a.bias[n + e]) : 0.f;
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int tl = (lane >> 4) + 4 * it;
        const int64_t m = m0 + wm0 + pass * 64 + tl;
        // (the cross-entropy reduction runs over the 16 lanes of a row: they skip together)
        if (m >= a.T || (EPI != EPI_XENT && n >= a.N)) continue;
        const int64_t row = (int64_t)half * a.T + m;
        const floatx4 v_lo = *reinterpret_cast<const floatx4*>(ep + tl * LDR + c * 8);
        const floatx4 v_hi = *reinterpret_cast<const floatx4*>(ep + tl * LDR + c * 8 + 4);
        float o[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = v_lo[e] + bb[e];
          o[e + 4] = v_hi[e] + bb[e + 4];
        }
        if constexpr (EPI == EPI_XENT) {
          // this row's 128 columns: maximum and sum of exp over the 16 lanes (8 each), then
          // the next token's logit from the lane that holds it
          float mx = -INFINITY;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (n + e < a.N) mx = fmaxf(mx, o[e]);
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
          float se = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (n + e < a.N) se += __expf(o[e] - mx);
#pragma unroll
          for (int off = 1; off < 16; off <<= 1) se += __shfl_xor(se, off, 64);
          if (c == 0) a.xpart[row * a.xnblk + (n0 + wn0) / 128] = make_float2(mx, se);
          const int64_t pos = m % a.seq;
          if (pos < a.seq - 1) {
            int64_t t = a.tok[m + 1];
            t = t < 0 ? 0 : (t >= a.N ? a.N - 1 : t);
            if (t >= n && t < n + 8) {
              float tv = o[0];
#pragma unroll
              for (int e = 1; e < 8; ++e)
                if (t - n == e) tv = o[e];
              a.xtgt[row] = tv;
            }
          }
          continue;
        }
        if (EPI != EPI_MSE && a.resid) {
          const uint4 rv = *reinterpret_cast<const uint4*>(a.resid + row * nout + n);
          const uint32_t rw[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            o[2 * e] += bf2f((uint16_t)(rw[e] & 0xFFFF));
            o[2 * e + 1] += bf2f((uint16_t)(rw[e] >> 16));
          }
        }
        if (EPI == ZOACT_EPI_RELU) {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = fmaxf(o[e], 0.0f);
        }
        if constexpr (EPI == EPI_MSE) {
          // squared error of the bf16-rounded output against the target, summed in fp32
          const uint4 tv = tpre[pass][it];
          const uint32_t tw[4] = {tv.x, tv.y, tv.z, tv.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d0 = bf2f(f2bf(o[2 * e])) - bf2f((uint16_t)(tw[e] & 0xFFFF));
            const float d1 = bf2f(f2bf(o[2 * e + 1])) - bf2f((uint16_t)(tw[e] >> 16));
            sq_acc += d0 * d0;
            sq_acc += d1 * d1;
          }
          continue;
        }
        if (OUT_F32) {
          float* yp = reinterpret_cast<float*>(a.y) + row * nout + n;
          *reinterpret_cast<float4*>(yp) = make_float4(o[0], o[1], o[2], o[3]);
          *reinterpret_cast<float4*>(yp + 4) = make_float4(o[4], o[5], o[6], o[7]);
        } else {
          *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.y) + row * nout + n) =
              make_uint4(pack2(f2bf(o[0]), f2bf(o[1])), pack2(f2bf(o[2]), f2bf(o[3])), pack2(f2bf(o[4]), f2bf(o[5])),
                         pack2(f2bf(o[6]), f2bf(o[7])));
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
  }
  if constexpr (EPI == EPI_MSE) {
    // tile sum in a fixed order: lanes (fp64 butterfly), then the four waves in order
    double v = (double)sq_acc;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    double* red = reinterpret_cast<double*>(reinterpret_cast<char*>(lds) + 4 * 64 * LDR * 4);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0)
      a.part[(int64_t)half * a.tiles_m_half * a.tiles_n + (int64_t)(tm % a.tiles_m_half) * a.tiles_n + tn] =
          ((red[0] + red[1]) + red[2]) + red[3];
  }
}

}  // namespace gemm
}  // namespace zoact

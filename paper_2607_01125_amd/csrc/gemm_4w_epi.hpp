// Pieces shared by the four-wave fused GEMM schedules (32-deep and 64-deep stages): wait
// counts, the workgroup barrier, buffer descriptors, and the epilogue that stages each
// wave's 128 x 128 accumulator tile through LDS and applies bias, residual, activation
// (or the fused regression loss) with one rounding, and the same operations straight from
// the accumulators.
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


// Tile index of the regression loss's partial sums (four per tile, one per wave):
// half-major, then token tile, then feature tile.
__device__ __forceinline__ int64_t mse_slot(const GemmArgs& a, int half, int tm, int tn) {
  return (int64_t)half * a.tiles_m_half * a.tiles_n + (int64_t)(tm % a.tiles_m_half) * a.tiles_n + tn;
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
          if (c == 0 && n0 + wn0 < a.N) a.xpart[row * a.xnblk + (n0 + wn0) / 128] = make_float2(mx, se);
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
    // this wave's sum (fp64 butterfly over lanes) into its own slot: four per tile
    double v = (double)sq_acc;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) a.part[mse_slot(a, half, tm, tn) * 4 + wave] = v;
  }
}

// Epilogue straight from the accumulators, for the persistent schedule whose operand ring
// stays busy with the next tile's first stages: no LDS.  Lane (lr, lk) holds, for every
// 16 x 16 block (i, j), features i*16 + lk*4 .. +3 of token j*16 + lr (the MFMA output
// layout), so each store writes 4 consecutive features of one row; the row reductions of
// the cross entropy run over the 4 lanes that share lr.  Rows go through buffer
// descriptors based at the wave's first token and feature, sized to its tokens below T:
// the per-lane part of an address is one register, the block's part is scalar, and rows
// past T fall outside the range (loads read zeros, stores are dropped).  N is a multiple
// of 16, so a 16-feature block lies wholly below N or past it: those tests are uniform.

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Descriptor over `rows` rows of `ld` elements of `esz` bytes from element `first` (all
// wave-uniform: read from the first lane so that the compiler keeps the descriptor in
// scalar registers rather than looping over lanes at every access).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, int64_t first, int64_t ld, int rows,
                                                           int esz) {
  const uint64_t p = reinterpret_cast<uint64_t>(base) + (uint64_t)(first * esz);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(p >> 32));
  const uint32_t n = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(rows * ld * esz));
  return buffer_rsrc(reinterpret_cast<const void*>(((uint64_t)hi << 32) | lo), n);
}

// Tokens of this wave below T (0 .. 128).
__device__ __forceinline__ int wave_rows(const GemmArgs& a, int64_t mw) {
  const int64_t r = a.T - mw;
  return r <= 0 ? 0 : (r >= 128 ? 128 : (int)r);
}

// One accumulator element read into a VGPR where it is used: kept in order with the block
// fences, so a block's values are read with the block instead of all 256 at once.
__device__ __forceinline__ float acc_read(float x) {
  float r;
  asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(r) : "a"(x));
  return r;
}

// Per-lane byte offset past any descriptor's range: a store through it is dropped.
constexpr int OFF_NONE = (int)0x80000000u;

// Operand rows the epilogue reads, for this lane's blocks in token blocks J0 .. J0 + 3:
// the regression target (EPI_MSE) or the residual (stored outputs with a residual; block b
// is output block b).  Rows past T read zeros; blocks past N are not read (a descriptor
// starts at the wave's first feature, so in its last row such a block would still be in
// its range but past the end of the tensor).
template <int EPI, int J0>
__device__ __forceinline__ void epi_prefetch(const GemmArgs& a, uint2 (&tv)[8][8], int wave, int lane, int64_t m0,
                                             int64_t n0, int half) {
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t nw = n0 + (wave & 1) * 128, mw = m0 + (wave >> 1) * 128;
  if constexpr (EPI == EPI_MSE) {
    const __amdgpu_buffer_rsrc_t rs = rows_rsrc(a.tgt, mw * a.N + nw, a.N, wave_rows(a, mw), 2);
    const int vo = (int)((lr * a.N + lk * 4) * 2);
#pragma unroll
    for (int j = J0; j < J0 + 4; ++j)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        u32x2_t u = {0u, 0u};
        if (nw + i * 16 < a.N) u = __builtin_amdgcn_raw_buffer_load_b64(rs, vo, (int)(j * 16 * a.N * 2) + i * 32, 0);
        tv[j][i] = make_uint2(u.x, u.y);
      }
  } else if constexpr (EPI != EPI_XENT) {
    if (a.resid == nullptr) return;
    constexpr bool SW = EPI == ZOACT_EPI_SWIGLU;
    constexpr int NB = SW ? 4 : 8;
    const int64_t nout = SW ? a.N / 2 : a.N;
    const int64_t first = ((int64_t)half * a.T + mw) * nout + (SW ? nw / 2 : nw);
    const __amdgpu_buffer_rsrc_t rs = rows_rsrc(a.resid, first, nout, wave_rows(a, mw), 2);
    const int vo = (int)((lr * nout + lk * 4) * 2);
#pragma unroll
    for (int j = J0; j < J0 + 4; ++j)
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        u32x2_t u = {0u, 0u};
        if (nw + b * (SW ? 32 : 16) < a.N)
          u = __builtin_amdgcn_raw_buffer_load_b64(rs, vo, (int)(j * 16 * nout * 2) + b * 32, 0);
        tv[j][b] = make_uint2(u.x, u.y);
      }
  }
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to bf16 (round to nearest even) in one conversion, lo in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Epilogues that use the interleaved W-row order of the 64-deep schedule, in which lane
// (lr, lk) holds features q * 32 + lk * 8 .. +7 of block pair q (blocks 2q, 2q + 1): those
// with one output per feature, whose rows are then read and written 16 bytes per lane.
// (SwiGLU needs gate and up in one lane; the cross entropy reduces over whole rows.)
constexpr bool epi_perm(int epi) { return epi == 0 || epi == ZOACT_EPI_RELU || epi == EPI_MSE; }

// Per-lane offset of a lane's 8 features of block pair q, or an offset past the range where
// they lie past N (N is a multiple of 8, so 8 features lie wholly on one side).
__device__ __forceinline__ int pair_off(const GemmArgs& a, int64_t nw, int q, int lk, int vo) {
  return nw + q * 32 + lk * 8 < a.N ? vo : OFF_NONE;
}

// Interleaved order: the 8 bf16 values of each lane's block pair q in token blocks 0 .. 7 of
// `src` (the regression target, or the residual), 16 bytes per lane; rows past T and
// features past N read zeros.
__device__ __forceinline__ void epi_prefetch8(const GemmArgs& a, const uint16_t* src, int64_t ld, uint4 (&tq)[8][4],
                                              int wave, int lane, int64_t m0, int64_t n0, int half) {
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t nw = n0 + (wave & 1) * 128, mw = m0 + (wave >> 1) * 128;
  const __amdgpu_buffer_rsrc_t rs = rows_rsrc(src, ((int64_t)half * a.T + mw) * ld + nw, ld, wave_rows(a, mw), 2);
  const int vo = (int)((lr * ld + lk * 8) * 2);
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const u32x4_t u = __builtin_amdgcn_raw_buffer_load_b128(rs, pair_off(a, nw, q, lk, vo),
                                                              (int)((j * 16 * ld + q * 32) * 2), 0);
      tq[j][q] = make_uint4(u.x, u.y, u.z, u.w);
    }
}

// EPI_MSE: the regression target's rows, requested before the rank correction so that
// their latency overlaps it.  (A residual is requested in the epilogue: beside the
// correction's operands it would not fit in registers with the stores' working set.)
template <int EPI>
__device__ __forceinline__ void epi_rows_early(const GemmArgs& a, uint4 (&tq)[8][4], int wave, int lane, int64_t m0,
                                               int64_t n0) {
  if constexpr (EPI == EPI_MSE) epi_prefetch8(a, a.tgt, a.N, tq, wave, lane, m0, n0, 0);
}

// CORR (shared input, half 0): the accumulators hold the base x W^T only, and each block's
// value is the rank-r correction MFMA of C_0's and p's slices with that base block as its
// accumulator input (r <= 32, one slice): the stacked form's correction step, the base left
// in place for the other half.  The MFMAs are issued in their VGPR form (inline assembly):
// in the accumulator form they would need free accumulator registers, and every one holds
// the tile.  The assembly carries its own wait states, as the compiler does not look inside
// it: 2 before (a VALU result read as MFMA input) and 20 after (an 8-pass MFMA result read
// by a VALU or memory instruction needs fewer).
template <int EPI, bool OUT_F32, bool BIAS, bool CORR>
__device__ __forceinline__ void epilogue_regs_impl(const GemmArgs& a, floatx4 (&acc)[8][8], uint4 (&tq)[8][4],
                                                   int wave, int lane, int64_t m0, int64_t n0, int half, int tm,
                                                   int tn) {
  const int lr = lane & 15, lk = lane >> 4;
  const int64_t nw = n0 + (wave & 1) * 128;   // first feature of this wave
  const int64_t mw = m0 + (wave >> 1) * 128;  // first token of this wave
  const int rows = wave_rows(a, mw);
  constexpr bool PERM = epi_perm(EPI);
  // the rows this epilogue reads: in the interleaved order 16 bytes per lane and block pair
  // (the regression target was requested before the rank correction, a residual is now),
  // else 8 bytes per block
  uint2 tv[8][8];
  uint4 tr[8][4];   // a residual in the interleaved order
  if constexpr (PERM && EPI != EPI_MSE) {
    if (a.resid) epi_prefetch8(a, a.resid, a.N, tr, wave, lane, m0, n0, half);
  } else if constexpr (!PERM) {
    epi_prefetch<EPI, 0>(a, tv, wave, lane, m0, n0, half);
    epi_prefetch<EPI, 4>(a, tv, wave, lane, m0, n0, half);
  }
  // bias of the lane's 32 features as bf16 pairs (per block pair, or per block), zero past N
  uint32_t bw[16];
  if constexpr (BIAS) {
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(a.bias, (uint32_t)(a.N * 2));
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (PERM) {
        const u32x4_t u = __builtin_amdgcn_raw_buffer_load_b128(rs, pair_off(a, nw, q, lk, lk * 16),
                                                                (int)((nw + q * 32) * 2), 0);
        bw[4 * q] = u.x, bw[4 * q + 1] = u.y, bw[4 * q + 2] = u.z, bw[4 * q + 3] = u.w;
      } else {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const u32x2_t u = __builtin_amdgcn_raw_buffer_load_b64(rs, lk * 8, (int)((nw + (2 * q + h) * 16) * 2), 0);
          bw[4 * q + 2 * h] = u.x, bw[4 * q + 2 * h + 1] = u.y;
        }
      }
    }
  }
  // accumulator element e of block (i, j), plus the bias (none added without one).  Either
  // order keeps block i's 4 bias values in words 2i, 2i + 1.
  auto val = [&](int i, int j, int e) -> float {
    const float v = acc_read(acc[i][j][e]);
    if constexpr (BIAS) {
      const uint32_t w = bw[2 * i + (e >> 1)];
      return v + (e & 1 ? bf_hi(w) : bf_lo(w));
    }
    return v;
  };
  // CORR: correction operands (p [T][r] shared by both halves, C_0 in the interleaved row
  // order), their slices read one pair / one token block ahead of use
  [[maybe_unused]] const int r = a.r;
  [[maybe_unused]] const int lrow = (lr >> 2) * 8 + (lr & 3);
  [[maybe_unused]] const __amdgpu_buffer_rsrc_t prs = buffer_rsrc(a.p, (uint32_t)(a.T * a.r * 2));
  [[maybe_unused]] const __amdgpu_buffer_rsrc_t crs = buffer_rsrc(a.ch, (uint32_t)(a.N * a.r * 2));
  [[maybe_unused]] const int pvo = (int)(((mw - m0) + lr) * a.r + lk * 8) * 2;
  [[maybe_unused]] const int cvo = (int)(((nw - n0) + lrow) * a.r + lk * 8) * 2;
  auto cfrag = [&](__amdgpu_buffer_rsrc_t rs, int vo, int so) -> bf16x8 {
    const u32x4_t u = __builtin_amdgcn_raw_buffer_load_b128(rs, vo, so, 0);
    return __builtin_bit_cast(bf16x8, lk * 8 < r ? u : u32x4_t{0u, 0u, 0u, 0u});   // columns past r: zero
  };
  auto cblk = [&](int i) -> bf16x8 { return cfrag(crs, cvo, (int)((n0 + (i >> 1) * 32 + (i & 1) * 4) * r * 2)); };
  auto pblk = [&](int j) -> bf16x8 { return cfrag(prs, pvo, (int)((m0 + j * 16) * r * 2)); };
  bf16x8 cn0 = {}, cn1 = {}, pn = {};
  if constexpr (CORR) {
    cn0 = cblk(0), cn1 = cblk(1), pn = pblk(0);
  }
  // values of block pair q in token block j (features lk*8 .. +7, blocks 2q and 2q + 1), bias
  // added; pairs are visited in the order j, q
  auto pair_vals = [&](int q, int j, float (&v)[8]) {
    if constexpr (CORR) {
      const bf16x8 c0 = cn0, c1 = cn1, pf = pn;
      const int k = 4 * j + q + 1;   // the next pair
      if (k < 32) {
        cn0 = cblk(2 * (k & 3)), cn1 = cblk(2 * (k & 3) + 1);
        if ((k & 3) == 0) pn = pblk(k >> 2);
      }
      floatx4 b0, b1, y0, y1;
#pragma unroll
      for (int e = 0; e < 4; ++e) b0[e] = acc_read(acc[2 * q][j][e]);
#pragma unroll
      for (int e = 0; e < 4; ++e) b1[e] = acc_read(acc[2 * q + 1][j][e]);
      asm volatile(
          "s_nop 1\n\t"
          "v_mfma_f32_16x16x32_bf16 %0, %2, %4, %5\n\t"
          "v_mfma_f32_16x16x32_bf16 %1, %3, %4, %6\n\t"
          "s_nop 15\n\t"
          "s_nop 3"
          : "=&v"(y0), "=&v"(y1)
          : "v"(c0), "v"(c1), "v"(pf), "v"(b0), "v"(b1));
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = y0[e], v[4 + e] = y1[e];
      if constexpr (BIAS) {
#pragma unroll
        for (int f = 0; f < 8; ++f) {
          const uint32_t w = bw[4 * q + (f >> 1)];
          v[f] += f & 1 ? bf_hi(w) : bf_lo(w);
        }
      }
    } else {
#pragma unroll
      for (int f = 0; f < 8; ++f) v[f] = val(2 * q + (f >> 2), j, f & 3);
    }
  };
  // the values of token block j's four pairs: without the in-epilogue correction all 32
  // accumulator elements are read first (in block order), so that the arithmetic of the
  // block's outputs is independent work the scheduler can interleave; with it, pair by pair
  float vj[4][8];
  auto block_vals = [&](int j) {
    if constexpr (!CORR) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int f = 0; f < 8; ++f) vj[q][f] = val(2 * q + (f >> 2), j, f & 3);
    }
  };
  auto pair_of = [&](int q, int j, float (&v)[8]) {
    if constexpr (CORR) {
      pair_vals(q, j, v);
    } else {
#pragma unroll
      for (int f = 0; f < 8; ++f) v[f] = vj[q][f];
    }
  };
  if constexpr (EPI == EPI_MSE) {
    float sq = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float sj = 0.f;
      block_vals(j);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // squared error of the bf16-rounded outputs (features lk*8 .. +7) against the target;
        // a pair past N is computed too and its terms dropped
        float v[8];
        pair_of(q, j, v);
        const uint32_t t[4] = {tq[j][q].x, tq[j][q].y, tq[j][q].z, tq[j][q].w};
        float sp = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t o = pack_bf16x2(v[2 * w], v[2 * w + 1]);
          const float d0 = bf_lo(o) - bf_lo(t[w]), d1 = bf_hi(o) - bf_hi(t[w]);
          sp = fmaf(d0, d0, sp);
          sp = fmaf(d1, d1, sp);
        }
        sj += nw + q * 32 + lk * 8 < a.N ? sp : 0.f;
      }
      sq += j * 16 + lr < rows ? sj : 0.f;   // rows past T add nothing
      __builtin_amdgcn_sched_barrier(0);     // one token block at a time: bounded registers
    }
    double v = (double)sq;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) a.part[mse_slot(a, half, tm, tn) * 4 + wave] = v;
  } else if constexpr (EPI == EPI_XENT) {
    // branch-free per token block (stores through an offset outside the range where a lane
    // must not write) so that the block's values stay the only ones in registers
    const __amdgpu_buffer_rsrc_t trs = buffer_rsrc(a.tok, (uint32_t)(a.T * 4));
    const __amdgpu_buffer_rsrc_t xps = buffer_rsrc(a.xpart, (uint32_t)(2 * a.T * a.xnblk * 8));
    const __amdgpu_buffer_rsrc_t xts = buffer_rsrc(a.xtgt, (uint32_t)(2 * a.T * 4));
    const int seq = (int)a.seq;
    int nxt[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int m = (int)mw + j * 16 + lr;
      const bool has = j * 16 + lr < rows && m % seq < seq - 1;
      // (m + 1 = T reads zero: past the range)
      const int t = (int)__builtin_amdgcn_raw_buffer_load_b32(trs, (m + 1) * 4, 0, 0);
      nxt[j] = has ? (t < 0 ? 0 : (t >= a.N ? (int)a.N - 1 : t)) : -1;
    }
    // (a wave wholly inside N, every one but the last column's, skips the per-block tests)
    const bool full = nw + 128 <= a.N;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      float v[8][4];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) v[i][e] = val(i, j, e);
      float mx = -INFINITY;
      if (full) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) mx = fmaxf(mx, v[i][e]);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (nw + i * 16 < a.N) mx = fmaxf(mx, v[i][e]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const bool mv = j * 16 + lr < rows;
      const int row = half * (int)a.T + (int)mw + j * 16 + lr;
      // the row's next-token logit, while the block's values are still the logits
      const int d = nxt[j] - (int)nw;   // the next token's offset in this wave's block
      const bool own = mv && d >= 0 && d < 128 && ((d >> 2) & 3) == lk;
      float tvv = 0.f;
      if (own) {   // rare (a 128-column block holds a row's next token about once in V / 128)
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (d == i * 16 + lk * 4 + e) tvv = v[i][e];
      }
      // exp(logit - max) in place, then four partial sums (element e of every block) added
      // in a fixed order: the 32 exponentials are independent of each other
      if (full) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) v[i][e] = __expf(v[i][e] - mx);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) v[i][e] = nw + i * 16 < a.N ? __expf(v[i][e] - mx) : 0.f;
      }
      float sp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) sp[e] += v[i][e];
      float se = (sp[0] + sp[1]) + (sp[2] + sp[3]);
      se += __shfl_xor(se, 16, 64);
      se += __shfl_xor(se, 32, 64);
      // (a wave wholly past N has no block of its own: index xnblk would be the next row's)
      const int vxp = (mv && lk == 0 && nw < a.N) ? (row * a.xnblk + (int)(nw >> 7)) * 8 : OFF_NONE;
      __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{__float_as_uint(mx), __float_as_uint(se)}, xps, vxp, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(tvv), xts, own ? row * 4 : OFF_NONE, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else if constexpr (PERM) {
    constexpr int ESZ = OUT_F32 ? 4 : 2;
    const bool res = a.resid != nullptr;
    const __amdgpu_buffer_rsrc_t ys = rows_rsrc(a.y, ((int64_t)half * a.T + mw) * a.N + nw, a.N, rows, ESZ);
    const int vy = (int)((lr * a.N + lk * 8) * ESZ);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      block_vals(j);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // (a pair past N is computed too; its store goes through an offset past the range)
        float o[8];
        pair_of(q, j, o);
        if (res) {
          const uint32_t t[4] = {tr[j][q].x, tr[j][q].y, tr[j][q].z, tr[j][q].w};
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            o[2 * w] += bf_lo(t[w]);
            o[2 * w + 1] += bf_hi(t[w]);
          }
        }
        if (EPI == ZOACT_EPI_RELU) {
#pragma unroll
          for (int f = 0; f < 8; ++f) o[f] = fmaxf(o[f], 0.0f);
        }
        // 8 consecutive features: one 16-byte store (two in fp32); none past N
        const int vo = pair_off(a, nw, q, lk, vy);
        const int so = (int)((j * 16 * a.N + q * 32) * ESZ);
        if (OUT_F32) {
          __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{__float_as_uint(o[0]), __float_as_uint(o[1]),
                                                         __float_as_uint(o[2]), __float_as_uint(o[3])},
                                                 ys, vo, so, 0);
          __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{__float_as_uint(o[4]), __float_as_uint(o[5]),
                                                         __float_as_uint(o[6]), __float_as_uint(o[7])},
                                                 ys, vo, so + 16, 0);
        } else {
          __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3]),
                                                         pack_bf16x2(o[4], o[5]), pack_bf16x2(o[6], o[7])},
                                                 ys, vo, so, 0);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    constexpr bool SW = EPI == ZOACT_EPI_SWIGLU;
    constexpr int ESZ = OUT_F32 ? 4 : 2;
    const bool res = a.resid != nullptr;
    const int64_t nout = SW ? a.N / 2 : a.N;
    const int64_t first = ((int64_t)half * a.T + mw) * nout + (SW ? nw / 2 : nw);
    const __amdgpu_buffer_rsrc_t ys = rows_rsrc(a.y, first, nout, rows, ESZ);
    const int vy = (int)((lr * nout + lk * 4) * ESZ);
    // output block b of token block j: the residual added, one store per lane (none for a
    // block past N)
    auto emit = [&](int j, int b, float (&o)[4], int voff) {
      if (res) {
        o[0] += bf_lo(tv[j][b].x);
        o[1] += bf_hi(tv[j][b].x);
        o[2] += bf_lo(tv[j][b].y);
        o[3] += bf_hi(tv[j][b].y);
      }
      if (EPI == ZOACT_EPI_RELU) {
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = fmaxf(o[e], 0.0f);
      }
      const int so = (int)((j * 16 * nout + b * 16) * ESZ);
      if (OUT_F32)
        __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{__float_as_uint(o[0]), __float_as_uint(o[1]),
                                                       __float_as_uint(o[2]), __float_as_uint(o[3])},
                                               ys, voff, so, 0);
      else
        __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])}, ys, voff,
                                              so, 0);
    };
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if constexpr (SW) {
        // blocks 2q (gate) and 2q + 1 (up) of the 16-interleaved fused projection give
        // output block q.  The token block's 32 values are read first, so the 16 outputs'
        // exp / reciprocal chains are independent work the scheduler can interleave (one at
        // a time, each waits out the latency of its transcendental steps).
        float gv[4][4], uv[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            gv[q][e] = val(2 * q, j, e);
            uv[q][e] = val(2 * q + 1, j, e);
          }
        float ov[4][4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) ov[q][e] = silu(gv[q][e]) * uv[q][e];
        // an output block past N: its store goes through an offset past the range (in the
        // wave's last row the block's own offset would still lie inside it)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float o[4] = {ov[q][0], ov[q][1], ov[q][2], ov[q][3]};
          emit(j, q, o, nw + q * 32 < a.N ? vy : OFF_NONE);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (nw + i * 16 >= a.N) continue;   // uniform
          float o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = val(i, j, e);
          emit(j, i, o, vy);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

template <int EPI, bool OUT_F32, bool CORR = false>
__device__ __forceinline__ void epilogue_regs(const GemmArgs& a, floatx4 (&acc)[8][8], uint4 (&tq)[8][4], int wave,
                                              int lane, int64_t m0, int64_t n0, int half, int tm, int tn) {
  if (a.bias) epilogue_regs_impl<EPI, OUT_F32, true, CORR>(a, acc, tq, wave, lane, m0, n0, half, tm, tn);
  else epilogue_regs_impl<EPI, OUT_F32, false, CORR>(a, acc, tq, wave, lane, m0, n0, half, tm, tn);
}

}  // namespace gemm
}  // namespace zoact

// Fused +/- adapted GEMM, four-wave schedule with 64-deep stages (gfx950, bf16 weights,
// precomputed C_h or r = 0).
//
// Same contraction and tiles as the 32-deep four-wave schedule: y[h] = x[h] W^T + b +
// p[h] C_h^T (Section 3, factored perturbed forward) over a 256-feature x 256-token
// workgroup tile, one wave per SIMD owning 128 x 128 outputs in 256 accumulator
// registers, 64 v_mfma_f32_16x16x32_bf16 per 32-deep sub-step with the next sub-step's
// fragments read from LDS meanwhile.  What changes is the global -> LDS path:
//
//  * A stage is 64 deep, so a row of an operand tile is one whole 128-byte line.  Each
//    direct-to-LDS load moves 8 rows x 128 bytes (every line it touches fully used),
//    where 32-deep stages move 16 rows x 64 bytes (half lines, the other half fetched
//    again a step later).  Rows are XOR-swizzled in LDS (chunk c of row r at chunk
//    c ^ (r & 7)), applied on the global side, so fragment reads are conflict-free.
//  * LDS holds five 32 KB operand slots used as a ring: stage S keeps W in slot 2S mod 5
//    and x in slot 2S+1 mod 5.  While stage S is computed (sub-steps 2S, 2S+1) the W of
//    stage S+2 goes into the slot stage S-1's x has left (during 2S) and its x into the
//    slot stage S's W leaves after 2S (during 2S+1); both are waited for at the end of
//    2S+2, one and a half to two and a half sub-steps later.  Eight loads per wave per
//    sub-step, as in the 32-deep schedule, and one workgroup barrier per stage.
//  * The fifth slot is the 32 KB the 32-deep schedule spends on C_h, so this schedule
//    reads C_h precomputed (zoact_perturb_coeffs) for the ceil(r/32) correction steps.
#include "gemm_4w_epi.hpp"

namespace zoact {

namespace {

using namespace gemm;

constexpr int NT = 256;
constexpr int SLOT_ELEMS = 256 * 64;                 // one operand tile, 64 deep (bf16 elements, 32 KB)
constexpr int NSLOT = 5;
constexpr int LDS_BYTES = NSLOT * SLOT_ELEMS * 2;    // 160 KB

// Byte offset of (row, 16-byte chunk c) in a 64-deep operand tile (rows of 128 bytes).
__device__ __forceinline__ int swz64(int row, int c) { return (row << 7) + ((c ^ (row & 7)) << 4); }

// One 1 KB load: rows row0 .. row0+7 (row0 % 8 == 0), depth k0 .. k0+63 -> LDS at dst.
// Lane l lands at dst + 16 l, i.e. row l >> 3, LDS chunk l & 7, which holds global
// chunk (l & 7) ^ (l >> 3).  The per-lane part of the address (`lane_off`, the same for
// every load of a wave) goes in the vector offset, the uniform part in the scalar one.
__device__ __forceinline__ int dma8_lane_off(int64_t ld) {
  const int lane = threadIdx.x & 63;
  return (int)((lane >> 3) * ld * 2 + (((lane & 7) ^ (lane >> 3)) << 4));
}
__device__ __forceinline__ void dma8(__amdgpu_buffer_rsrc_t src, int lane_off, int64_t ld, int64_t row0, int64_t k0,
                                     char* dst) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void_t*)dst, 16, lane_off, (int)((row0 * ld + k0) * 2), 0, 0);
}

__device__ __forceinline__ int mod5(int v) { return v >= 5 ? v - 5 : v; }

template <int EPI, bool OUT_F32>
__global__ void __launch_bounds__(NT, 1) gemm_4w64_kernel(GemmArgs a) {
  extern __shared__ __align__(16) uint16_t lds[];
  char* const lb = reinterpret_cast<char*>(lds);

  // ---- tile assignment (XCD-contiguous runs, grouped token-major order)
  const int ntiles = gridDim.x;
  int lin = blockIdx.x;
  if ((ntiles & 7) == 0) lin = (blockIdx.x & 7) * (ntiles >> 3) + (blockIdx.x >> 3);
  const int tiles_m = 2 * a.tiles_m_half;
  const int per_group = 4 * a.tiles_n;
  const int grp_t = lin / per_group;
  const int first_m = grp_t * 4;
  const int gsz = min(4, tiles_m - first_m);
  const int tm = first_m + (lin % per_group) % gsz;
  const int tn = (lin % per_group) / gsz;
  const int half = tm / a.tiles_m_half;
  const int64_t m0 = (int64_t)(tm % a.tiles_m_half) * 256;
  const int64_t n0 = (int64_t)tn * 256;
  const uint16_t* xh = a.x + (int64_t)half * a.T * a.K;
  const uint16_t* w = reinterpret_cast<const uint16_t*>(a.w);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: kept in SGPRs
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128;   // features of this wave
  const int wm0 = (wave >> 1) * 128;  // tokens of this wave
  const int NS = (int)(a.K >> 6);     // 64-deep stages

  const __amdgpu_buffer_rsrc_t wrs = buffer_rsrc(w, (uint32_t)(a.N * a.K * 2));
  const __amdgpu_buffer_rsrc_t xrs = buffer_rsrc(xh, (uint32_t)(a.T * a.K * 2));
  // this wave's 64 rows of one operand of stage st into slot `slot` (8 loads); `i` picks one
  const int loff = dma8_lane_off(a.K);
  auto dma_w = [&](int st, int slot, int i) {
    dma8(wrs, loff, a.K, n0 + wave * 64 + i * 8, (int64_t)st * 64,
         lb + slot * (SLOT_ELEMS * 2) + (wave * 64 + i * 8) * 128);
  };
  auto dma_x = [&](int st, int slot, int i) {
    dma8(xrs, loff, a.K, m0 + wave * 64 + i * 8, (int64_t)st * 64,
         lb + slot * (SLOT_ELEMS * 2) + (wave * 64 + i * 8) * 128);
  };

  floatx4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  bf16x8 fa0[8], fb0[8], fa1[8], fb1[8];

  // fragment offsets inside a slot: row (base + i * 16 + lr), chunk 4 h + lk; the swizzle
  // term depends on lr only, so k-half h has one per-lane offset
  const int fo0 = swz64(lr, lk), fo1 = swz64(lr, 4 + lk);
  auto frag = [&](int slot, int row0, int fo) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(lb + slot * (SLOT_ELEMS * 2) + row0 * 128 + fo);
  };

  // One 32-deep sub-step: 64 MFMAs on (fa, fb); the next sub-step's 16 fragments (slots
  // nws / nxs, k-half offset nfo) are read in the first four rows; one load of operand
  // `dma_x_side ? x : W` of stage dst_st into slot dslot after each row of MFMAs.
  auto sub_step = [&](bf16x8 (&fa)[8], bf16x8 (&fb)[8], bf16x8 (&na)[8], bf16x8 (&nb)[8], int nws, int nxs, int nfo,
                      bool dma_x_side, int dst_st, int dslot) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      if (dma_x_side) dma_x(dst_st, dslot, i);
      else dma_w(dst_st, dslot, i);
      if (i < 4) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int ii = 2 * i + h2;
          na[ii] = frag(nws, wn0 + ii * 16, nfo);
          nb[ii] = frag(nxs, wm0 + ii * 16, nfo);
        }
      }
      // issue order inside the row: each memory instruction right after an MFMA, so its
      // issue cycles fall in the shadow of that MFMA instead of between two rows
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // MFMA
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);    // the direct-to-LDS load
      if (i < 4) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one fragment read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x008, 7, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- prologue: stages 0 and 1 in flight (slots 0..3), stage 0 landed, fragments of
  // sub-step 0, then a barrier so that no slot is refilled before every wave has read it
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_w(0, 0, i);
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_x(0, 1, i);
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_w(1, 2, i);
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_x(1, 3, i);
  __builtin_amdgcn_s_waitcnt(WAIT_VM16);
  barrier();
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    fa0[i] = frag(0, wn0 + i * 16, fo0);
    fb0[i] = frag(1, wm0 + i * 16, fo0);
  }
  __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
  barrier();

  // ---- main loop: one stage (two sub-steps) per iteration.  s5 = 2S mod 5: stage S has
  // W in slot s5 and x in s5 + 1, stage S + 1 in s5 + 2 / s5 + 3, and stage S + 2 goes to
  // s5 + 4 (W, during sub-step 2S) and s5 (x, during 2S + 1).  Loads past the last stage
  // read the next rows or zeros into slots nobody reads again; the epilogue waits for them.
  // (The second sub-step sits under a test that always holds: written this way the
  // register allocator keeps every accumulator in place across the loop.)
  int s5 = 0;
  const int nsub = 2 * NS;
  for (int j = 0; j < nsub; j += 2) {
    const int st = j >> 1;
    const int sw1 = mod5(s5 + 2), sx1 = mod5(s5 + 3), sw2 = mod5(s5 + 4);
    // sub-step 2S: k-half 0 of stage S; reads k-half 1 of stage S; loads W of stage S + 2
    sub_step(fa0, fb0, fa1, fb1, s5, mod5(s5 + 1), fo1, false, st + 2, sw2);
    // stage S + 1 (issued during sub-steps 2S - 2 and 2S - 1) must have landed: the
    // eight loads of this sub-step may stay in flight
    __builtin_amdgcn_s_waitcnt(WAIT_VM8);
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    barrier();
    if (j + 1 < nsub) {
      // sub-step 2S + 1: k-half 1 of stage S; reads k-half 0 of stage S + 1; loads x of S + 2.
      // No barrier after it: sub-step 2S + 2 reads stage S + 1 (complete since the barrier
      // above) and loads into stage S's x slot (last read during 2S), so nothing it touches
      // can still be in use by a slower wave.
      sub_step(fa1, fb1, fa0, fb0, sw1, sx1, fo0, true, st + 2, s5);
      __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
      __builtin_amdgcn_sched_barrier(0);
    }
    s5 = sw1;
  }

  // ---- rank-r correction: [p[h] | C_h] as ceil(r/32) extra 32-deep steps, operands from
  // global memory (C_h precomputed); ranks not a multiple of 8 are gathered element-wise
  if (a.r > 0) {
    const int kts = (a.r + 31) >> 5;
    const uint16_t* ph = a.p + (int64_t)half * a.T * a.r;
    const uint16_t* chh = a.ch + (int64_t)half * a.ch_stride;
    const bool vec = (a.r & 7) == 0;
    const bf16x8 zero8 = {};
    auto row8 = [&](const uint16_t* rowp, int col) -> bf16x8 {
      if (vec) return col < a.r ? *reinterpret_cast<const bf16x8*>(rowp + col) : zero8;
      uint16_t e[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) e[q] = col + q < a.r ? rowp[col + q] : (uint16_t)0;
      const uint4 u = make_uint4(pack2(e[0], e[1]), pack2(e[2], e[3]), pack2(e[4], e[5]), pack2(e[6], e[7]));
      return __builtin_bit_cast(bf16x8, u);
    };
    for (int t = 0; t < kts; ++t) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int64_t m = m0 + wm0 + j * 16 + lr;
        m = m > a.T - 1 ? a.T - 1 : m;
        int64_t n = n0 + wn0 + j * 16 + lr;
        n = n > a.N - 1 ? a.N - 1 : n;
        const int col = t * 32 + lk * 8;
        fb0[j] = row8(ph + m * a.r, col);
        fa0[j] = row8(chh + n * a.r, col);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa0[i], fb0[j], acc[i][j], 0, 0, 0);
    }
  }

  epilogue_4w<EPI, OUT_F32>(a, acc, lds, wave, lane, m0, n0, half, tm, tn);
}

template <int EPI, bool OUT_F32>
hipError_t launch_4w64(const GemmArgs& a, hipStream_t s) {
  static bool attr_set = false;  // benign race: every thread sets the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_4w64_kernel<EPI, OUT_F32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const dim3 grid((unsigned)(2 * a.tiles_m_half * a.tiles_n));
  gemm_4w64_kernel<EPI, OUT_F32><<<grid, dim3(NT), LDS_BYTES, s>>>(a);
  return hipGetLastError();
}

}  // namespace

// Returns hipErrorNotSupported outside this schedule's coverage: bf16 weights; C_h
// precomputed (or r = 0), r <= 256; depth a multiple of 64; a half of x or the weights
// below 2 GiB.
hipError_t launch_linear_pm_4w64(const GemmArgs& a, int w_dtype, int epi, bool out_f32, hipStream_t s) {
  if (w_dtype != ZOACT_BF16) return hipErrorNotSupported;
  if (a.r > 0 && a.ch == nullptr) return hipErrorNotSupported;
  if (a.r > 256 || (a.K % 64) != 0) return hipErrorNotSupported;
  if (a.T * a.K * 2 >= (int64_t(1) << 31) || a.N * a.K * 2 >= (int64_t(1) << 31)) return hipErrorNotSupported;
#define ZO_4W64(EP, OF) \
  if (epi == EP && out_f32 == OF) return launch_4w64<EP, OF>(a, s);
  ZO_4W64(0, false)
  ZO_4W64(0, true)
  ZO_4W64(ZOACT_EPI_SWIGLU, false)
  ZO_4W64(ZOACT_EPI_RELU, false)
  ZO_4W64(EPI_MSE, false)
  ZO_4W64(EPI_XENT, false)
#undef ZO_4W64
  return hipErrorNotSupported;
}

}  // namespace zoact

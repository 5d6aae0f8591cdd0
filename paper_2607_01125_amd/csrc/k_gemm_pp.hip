// Fused +/- adapted GEMM, ping-pong schedule for gfx950 (bf16 weights, 0 <= r <= 64, r % 8 == 0).
//
// Same contraction as the generic kernel: y[h] = x[h] W^T + b + p[h] (C + s_h eps Z)^T
// (Section 3, factored perturbed forward), over a 256-feature x 256-token tile.
//
// Schedule (one workgroup of 8 wave64s per CU, 2 waves per SIMD):
//  * The waves form two groups of four (waves 0-3 and 4-7); each SIMD holds one wave
//    of each group.  The groups alternate between a compute phase (32 MFMAs on
//    fragments already in registers) and a memory phase (LDS -> register fragment
//    reads for their next compute phase, DMA issue, C +/- eps Z generation), switching
//    at workgroup barriers, so that every SIMD always has one wave feeding its matrix
//    core.  Group 1 starts one phase late.
//  * Global -> LDS uses the direct path (buffer_load_dwordx4 ... lds): each instruction
//    moves 64 x 16 bytes into a contiguous 1 KB run of LDS, 8 rows of a 64-deep stage.
//    The XOR swizzle of the LDS layout (16-byte chunk c of row r stored at chunk
//    c ^ (r & 7)) is applied on the global side.  Two stages of 64 KB (W + x): group 0
//    streams the W tile and group 1 the x tile of depth tile kt + 2 (8 runs per wave) in
//    the memory phase right after tile kt is released.  Buffer descriptors bound both
//    matrices: rows past the end read as 0.
//  * The perturbed coefficients C_h = bf16(C + s_h eps Z) of the tile's 256 features
//    are generated during the first memory phases into a dedicated 32 KB LDS region
//    (Z from its counter, nothing stored in HBM); the rank-r correction then runs as
//    one or two extra 32-deep steps against p[h] fragments read from global memory.
//  * The epilogue stages each wave's tile as fp32 through LDS and stores 16 bytes per
//    lane along the feature axis, with bias, residual and activation applied on rows.
//
// This schedule measured fastest of the variants tried on gfx950 (a four-wave 128 x 128
// schedule is limited by blocking vector-memory issue; a 32-deep four-stage ping-pong by
// the extra phase count).
//  * Barriers are raw s_barrier with explicit s_waitcnt (a full __syncthreads would wait
//    for the in-flight DMA at every phase switch).
#include "gemm_common.hpp"

namespace zoact {

namespace {

using namespace gemm;

constexpr int NT = 512;
constexpr int TILE_ELEMS = 256 * 64;            // one operand tile (bf16 elements, 32 KB)
constexpr int STAGE_ELEMS = 2 * TILE_ELEMS;     // W tile + x tile
constexpr int CH_ELEMS = 256 * 64;              // C_h region, 64 coefficient columns per feature
constexpr int LDS_BYTES = (2 * STAGE_ELEMS + CH_ELEMS) * 2;  // 160 KB

typedef __attribute__((address_space(3))) void lds_void_t;

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0,15:14], expcnt[6:4], lgkmcnt[11:8])
constexpr int WAIT_VM0 = 0x0F70;
constexpr int WAIT_LGKM0 = 0xC07F;
constexpr int WAIT_ALL0 = 0x0070;

__device__ __forceinline__ void barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
}

// Raw buffer resource over [base, base + bytes): loads at offsets past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// One 1 KB DMA run: rows row0 .. row0+7 of a [rows][ld] bf16 matrix, depth k0 .. k0+63,
// into LDS at `dst`; lane l fills row l >> 3, chunk l & 7, i.e. logical chunk (l&7)^(l>>3).
__device__ __forceinline__ void dma_run(__amdgpu_buffer_rsrc_t src, int64_t ld, int64_t row0, int64_t k0,
                                        uint16_t* dst) {
  const int lane = threadIdx.x & 63;
  const int64_t row = row0 + (lane >> 3);
  const int kc = (lane & 7) ^ (lane >> 3);
  const int off = (int)((row * ld + k0 + kc * 8) * 2);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void_t*)dst, 16, off, 0, 0, 0);
}

template <int EPI, bool OUT_F32, bool HAS_R>
__global__ void __launch_bounds__(NT, 1) gemm_pp_kernel(GemmArgs a) {
  extern __shared__ __align__(16) uint16_t lds[];

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
  const int sgn = a.sign_h[half];          // perturbation sign of this half
  const uint32_t qry = a.query_h[half];   // and its query index
  const uint16_t* xh = a.x + (int64_t)half * a.T * a.K;
  const uint16_t* w = reinterpret_cast<const uint16_t*>(a.w);

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int grp = wave >> 2;          // ping-pong group
  const int wq = wave & 3;            // index inside the group
  const int wn0 = (wave & 1) * 128;   // features of this wave
  const int wm0 = (wave >> 1) * 64;   // tokens of this wave
  const int nk = (int)(a.K >> 6);
  const int S = 2 * nk;               // 32-deep steps

  floatx4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  bf16x8 af[8], bfr[4];

  // DMA of depth tile kt into stage buf: group 0 moves W rows, group 1 x rows (8 runs per wave).
  const __amdgpu_buffer_rsrc_t drs = grp == 0 ? buffer_rsrc(w, (uint32_t)(a.N * a.K * 2))
                                              : buffer_rsrc(xh, (uint32_t)(a.T * a.K * 2));
  const int64_t drow0 = (grp == 0 ? n0 : m0) + wq * 64;
  const int doff = grp == 0 ? 0 : TILE_ELEMS;
  auto dma_tile = [&](int kt, int buf) {
    uint16_t* st = lds + buf * STAGE_ELEMS + doff + wq * 8 * 512;
    const int64_t k0 = (int64_t)kt * 64;
#pragma unroll
    for (int j = 0; j < 8; ++j) dma_run(drs, a.K, drow0 + j * 8, k0, st + j * 512);
  };
  auto load_frags = [&](int s) {
    const uint16_t* st = lds + ((s >> 1) & 1) * STAGE_ELEMS;
    const int kc = (s & 1) * 4 + lk;
#pragma unroll
    for (int i = 0; i < 8; ++i) af[i] = *reinterpret_cast<const bf16x8*>(st + swz(wn0 + i * 16 + lr, kc));
#pragma unroll
    for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(st + TILE_ELEMS + swz(wm0 + j * 16 + lr, kc));
  };
  auto compute = [&]() {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
  };
  // C_h chunk q of this thread: 4 coefficients (feature f, columns 4g .. 4g+3) -> LDS region.
  uint16_t* chreg = lds + 2 * STAGE_ELEMS;
  auto gen_chunk = [&](int q) {
    const int c = q * NT + threadIdx.x;
    const int f = c >> 4, g = c & 15;
    const int64_t n = n0 + f;
    uint2 packed = make_uint2(0u, 0u);
    if (4 * g < a.r && n < a.N) {
      const uint64_t e = (uint64_t)(a.coef_offset + n * a.r + 4 * g);
      const float4 z = gauss4(a.seed, a.step, qry, e);
      float cv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        cv[j] = a.c_bf16 ? bf2f(reinterpret_cast<const uint16_t*>(a.c)[e + j]) : reinterpret_cast<const float*>(a.c)[e + j];
      packed.x = pack2(perturbed_bf16(cv[0], z.x, a.eps, sgn), perturbed_bf16(cv[1], z.y, a.eps, sgn));
      packed.y = pack2(perturbed_bf16(cv[2], z.z, a.eps, sgn), perturbed_bf16(cv[3], z.w, a.eps, sgn));
    }
    *reinterpret_cast<uint2*>(chreg + swz(f, g >> 1) + (g & 1) * 4) = packed;
  };
  constexpr int QN = HAS_R ? (256 * 16) / NT : 0;  // 8 chunks per thread
  int q = 0;

  // ---- prologue: depth tiles 0 and 1 in flight, first fragments, group 1 one phase late
  dma_tile(0, 0);
  if (nk > 1) dma_tile(1, 1);
  __builtin_amdgcn_s_waitcnt(WAIT_VM0);
  barrier();
  load_frags(0);
  __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
  if (grp == 1) barrier();

  // one depth tile (two 32-deep steps) per iteration
  for (int kt = 0; kt < nk; ++kt) {
    const int s0 = 2 * kt;
    compute();
    barrier();
    {
      // memory phase for step s0 + 1; depth tile kt + 1 (DMA issued one phase pair ago)
      // must have landed before the next phase reads it.  C_h generation goes first: its
      // coefficient loads share the in-order vmcnt counter.
      if (HAS_R && q < QN) gen_chunk(q++);
      load_frags(s0 + 1);
      __builtin_amdgcn_s_waitcnt(WAIT_VM0);
      __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    }
    barrier();
    compute();
    barrier();
    if (s0 + 2 < S) {
      // memory phase for step s0 + 2 (depth tile kt + 1); stream tile kt + 2 into the
      // stage that tile kt has just released
      if (HAS_R && q < QN) gen_chunk(q++);
      load_frags(s0 + 2);
      if (kt + 2 < nk) dma_tile(kt + 2, kt & 1);
      __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    }
    barrier();
  }
  if (grp == 0) barrier();

  // ---- rank-r correction: [p[h] | C_h] as ceil(r/32) extra 32-deep steps
  if (HAS_R) {
    const int kts = (a.r + 31) >> 5;
    const uint16_t* ph = a.p + (int64_t)half * a.T * a.r;
    bf16x8 pf[2][4];
    const bf16x8 zero8 = {};
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int64_t m = m0 + wm0 + j * 16 + lr;
        m = m > a.T - 1 ? a.T - 1 : m;
        const int col = t * 32 + lk * 8;
        pf[t][j] = (t < kts && col < a.r) ? *reinterpret_cast<const bf16x8*>(ph + m * a.r + col) : zero8;
      }
    while (q < QN) gen_chunk(q++);
    __builtin_amdgcn_s_waitcnt(WAIT_ALL0);
    barrier();
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (t < kts) {
#pragma unroll
        for (int i = 0; i < 8; ++i) af[i] = *reinterpret_cast<const bf16x8*>(chreg + swz(wn0 + i * 16 + lr, t * 4 + lk));
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], pf[t][j], acc[i][j], 0, 0, 0);
      }
    }
  }

  // ---- epilogue through LDS: each wave stages its 128-feature x 64-token tile as fp32 in
  // its own 16 KB slice of the stage area, 32 tokens at a time, then applies bias, residual
  // and activation on rows and stores 16 bytes per lane along the feature axis.
  __builtin_amdgcn_s_waitcnt(WAIT_ALL0);
  barrier();
  constexpr int LDR = 132;  // padded fp32 row
  float* ep = reinterpret_cast<float*>(lds) + wave * (32 * LDR);
  const int64_t nout = (EPI == ZOACT_EPI_SWIGLU) ? a.N / 2 : a.N;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int j = pass * 2 + jj;
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<floatx4*>(ep + (jj * 16 + lr) * LDR + i * 16 + lk * 4) = acc[i][j];
    }
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    const int64_t tbase = m0 + wm0 + pass * 32;
    if (EPI == ZOACT_EPI_SWIGLU) {
      // 64 output features per wave: lane -> chunk c = lane & 7 (8 outputs), rows lane >> 3 + 8 it
      const int c = lane & 7;
      const int g0 = (c >> 1) * 32 + (c & 1) * 8;  // fused gate index inside the wave
      const int64_t ng = n0 + wn0 + g0;
      const int64_t fo = (n0 + wn0) / 2 + c * 8;  // output feature
      float bg[8], bu[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        bg[e] = (a.bias && ng < a.N) ? bf2f(a.bias[ng + e]) : 0.f;
        bu[e] = (a.bias && ng < a.N) ? bf2f(a.bias[ng + 16 + e]) : 0.f;
      }
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int tl = (lane >> 3) + 8 * it;
        const int64_t m = tbase + tl;
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
      for (int it = 0; it < 8; ++it) {
        const int tl = (lane >> 4) + 4 * it;
        const int64_t m = tbase + tl;
        if (m >= a.T || n >= a.N) continue;
        const int64_t row = (int64_t)half * a.T + m;
        const floatx4 v_lo = *reinterpret_cast<const floatx4*>(ep + tl * LDR + c * 8);
        const floatx4 v_hi = *reinterpret_cast<const floatx4*>(ep + tl * LDR + c * 8 + 4);
        float o[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = v_lo[e] + bb[e];
          o[e + 4] = v_hi[e] + bb[e + 4];
        }
        if (a.resid) {
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
}

template <int EPI, bool OUT_F32, bool HAS_R>
hipError_t launch_pp(const GemmArgs& a, hipStream_t s) {
  static bool attr_set = false;  // benign race: every thread sets the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_pp_kernel<EPI, OUT_F32, HAS_R>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const dim3 grid((unsigned)(2 * a.tiles_m_half * a.tiles_n));
  gemm_pp_kernel<EPI, OUT_F32, HAS_R><<<grid, dim3(NT), LDS_BYTES, s>>>(a);
  return hipGetLastError();
}

}  // namespace

// Returns hipErrorNotSupported when the layer is outside this kernel's coverage
// (INT4 weights, r > 64 or r % 8 != 0); the caller then uses the generic kernel.
hipError_t launch_linear_pm_pp(const GemmArgs& a, int w_dtype, int epi, bool out_f32, hipStream_t s) {
  if (w_dtype != ZOACT_BF16 || a.r > 64 || (a.r % 8) != 0 || (a.K % 64) != 0) return hipErrorNotSupported;
  // buffer offsets are 32-bit: each half of x and all of W must stay below 2 GiB
  if (a.T * a.K * 2 >= (int64_t(1) << 31) || a.N * a.K * 2 >= (int64_t(1) << 31)) return hipErrorNotSupported;
  const bool hr = a.r > 0;
#define ZO_PP(EP, OF, HR) \
  if (epi == EP && out_f32 == OF && hr == HR) return launch_pp<EP, OF, HR>(a, s);
  ZO_PP(0, false, true)
  ZO_PP(0, false, false)
  ZO_PP(0, true, false)
  ZO_PP(0, true, true)
  ZO_PP(ZOACT_EPI_SWIGLU, false, true)
  ZO_PP(ZOACT_EPI_SWIGLU, false, false)
  ZO_PP(ZOACT_EPI_RELU, false, true)
  ZO_PP(ZOACT_EPI_RELU, false, false)
#undef ZO_PP
  return hipErrorNotSupported;
}

}  // namespace zoact

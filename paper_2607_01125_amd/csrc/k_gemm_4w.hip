// Fused +/- adapted GEMM, four-wave software-pipelined schedule for gfx950
// (bf16 or group-128 INT4 weights; 0 <= r <= 256 with precomputed C_h, else r <= 64,
// r % 8 == 0).
//
// Same contraction as the other kernels: y[h] = x[h] W^T + b + p[h] (C + s_h eps Z)^T
// (Section 3, factored perturbed forward), over a 256-feature x 256-token tile.
//
//  * One wave per SIMD, each owning a 128 x 128 sub-tile: 64 fp32 accumulator blocks of
//    v_mfma_f32_16x16x32_bf16 (256 accumulator registers).  A wave reads 16 fragments per
//    32-deep step for 64 MFMAs, a quarter of a fragment per MFMA, which keeps the CU's LDS
//    traffic (about 128 bytes per clock) well below what the matrix cores consume.
//  * The fragments of step s + 1 are read from LDS while the 64 MFMAs of step s issue
//    (double-buffered fragment registers), so the matrix core never waits on LDS latency.
//  * Global -> LDS by the direct path (buffer_load_dwordx4 ... lds, 1 KB per instruction),
//    four 32 KB stages (W + x, 32-deep) in flight; stage s + 4 is issued at the start of
//    step s into the stage step s has just vacated, so each load has about three steps to
//    land.  The XOR swizzle (16-byte chunk c of row r at chunk c ^ ((r >> 1) & 3)) is
//    applied on the global side.  Buffer descriptors bound both matrices: rows past the
//    end read as 0.  One workgroup barrier per step.
//  * C_h = bf16(C + s_h eps Z) for the tile's 256 features is either read from the
//    precomputed array (zoact_perturb_coeffs) or generated in the prologue, while the first
//    stages are in flight, into a dedicated 32 KB LDS region; the rank-r correction runs
//    as ceil(r / 32) extra 32-deep steps against p[h] read from global memory.
//  * INT4 weights: the packed row and group scale of each lane's feature arrive by the
//    direct path six stages ahead; during step s every lane turns its row of stage s + 2
//    into bf16(q * s) in eight slices, one after each row of MFMAs, and writes it into the
//    W tile of that stage.  Only x travels through the bf16 stages.  The main loop's LDS
//    accesses to the packed ring and the W tile are inline assembly, so the compiler does
//    not drain the direct-to-LDS loads in flight before each of them.
#include "gemm_4w_epi.hpp"

namespace zoact {

namespace {

using namespace gemm;

constexpr int NT = 256;
constexpr int OP_ELEMS = 256 * 32;               // one operand tile (bf16 elements, 16 KB)
constexpr int STAGE_ELEMS = 2 * OP_ELEMS;        // W + x
constexpr int NSTAGE = 4;
constexpr int CH_ELEMS = 256 * 64;               // C_h region, 64 coefficient columns per feature
constexpr int LDS_BYTES = (NSTAGE * STAGE_ELEMS + CH_ELEMS) * 2;  // 160 KB
// INT4 weights: packed tiles (256 rows x 16 bytes) and their group scales arrive six stages
// ahead in their own ring; the C_h region is not used (C_h is read from the precomputed
// array).  A 2-byte direct-to-LDS load fills one 4-byte slot per lane, so a stage's 256
// scales take 1 KB.
constexpr int PK_STAGES = 6;
constexpr int PK_BYTES = 256 * 16;
constexpr int SC_BYTES = 256 * 4;
constexpr int LDS_BYTES_I4 = NSTAGE * STAGE_ELEMS * 2 + PK_STAGES * (PK_BYTES + SC_BYTES);  // 158 KB

// Element offset of (row, 16-byte chunk c) in a 32-deep operand tile (rows of 64 bytes).
__device__ __forceinline__ int swz32(int row, int c) { return (row << 5) + ((c ^ ((row >> 1) & 3)) << 3); }

// One 1 KB DMA run: rows row0 .. row0+15, depth k0 .. k0+31 -> LDS at dst.
__device__ __forceinline__ void dma_run(__amdgpu_buffer_rsrc_t src, int64_t ld, int64_t row0, int64_t k0,
                                        uint16_t* dst) {
  const int lane = threadIdx.x & 63;
  const int64_t row = row0 + (lane >> 2);
  const int c = (lane & 3) ^ ((lane >> 3) & 3);
  const int off = (int)((row * ld + k0 + c * 8) * 2);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void_t*)dst, 16, off, 0, 0, 0);
}

template <int EPI, bool OUT_F32, bool HAS_R, bool I4>
__global__ void __launch_bounds__(NT, 1) gemm_4w_kernel(GemmArgs a) {
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

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: kept in SGPRs
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128;   // features of this wave
  const int wm0 = (wave >> 1) * 128;  // tokens of this wave
  const int S = (int)(a.K >> 5);      // 32-deep steps

  // ---- C_h chunks (4 coefficients each), coefficient bits loaded before any DMA
  const int gmax = a.r <= 32 ? 8 : 16;
  const int qn = HAS_R ? (256 * gmax) / NT : 0;  // 8 or 16 chunks per thread
  uint32_t cbits[16][4];
  {
    const int esize = a.c_bf16 ? 2 : 4;
    const __amdgpu_buffer_rsrc_t crs =
        buffer_rsrc(static_cast<const char*>(a.c) + a.coef_offset * esize, (uint32_t)(a.N * a.r * esize));
    int base[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int c = q * NT + threadIdx.x;
      const int f = c / gmax, g = c % gmax;
      const int64_t n = n0 + f;
      const bool valid = HAS_R && q < qn && 4 * g < a.r && n < a.N;
      base[q] = valid ? (int)((n * a.r + 4 * g) * esize) : 0x7FFFFF00;
    }
    if (HAS_R && !I4 && a.ch == nullptr) {
      if (a.c_bf16) {
#pragma unroll
        for (int q = 0; q < 16; ++q)
#pragma unroll
          for (int j = 0; j < 4; ++j) cbits[q][j] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(crs, base[q] + 2 * j, 0, 0);
      } else {
#pragma unroll
        for (int q = 0; q < 16; ++q)
#pragma unroll
          for (int j = 0; j < 4; ++j) cbits[q][j] = __builtin_amdgcn_raw_buffer_load_b32(crs, base[q] + 4 * j, 0, 0);
      }
    }
  }
  uint16_t* chreg = lds + NSTAGE * STAGE_ELEMS;
  auto gen_chunk = [&](int q) {
    const int c = q * NT + threadIdx.x;
    const int f = c / gmax, g = c % gmax;
    const int64_t n = n0 + f;
    uint2 packed = make_uint2(0u, 0u);
    if (4 * g < a.r && n < a.N) {
      const uint64_t e = (uint64_t)(a.coef_offset + n * a.r + 4 * g);
      const float4 z = gauss4(a.seed, a.step, qry, e);
      float cv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) cv[j] = a.c_bf16 ? bf2f((uint16_t)cbits[q][j]) : __uint_as_float(cbits[q][j]);
      packed.x = pack2(perturbed_bf16(cv[0], z.x, a.eps, sgn), perturbed_bf16(cv[1], z.y, a.eps, sgn));
      packed.y = pack2(perturbed_bf16(cv[2], z.z, a.eps, sgn), perturbed_bf16(cv[3], z.w, a.eps, sgn));
    }
    *reinterpret_cast<uint2*>(chreg + swz(f, g >> 1) + (g & 1) * 4) = packed;
  };

  // ---- stage DMA: each wave moves 4 W runs and 4 x runs (16 rows each) per step
  const __amdgpu_buffer_rsrc_t wrs = buffer_rsrc(w, (uint32_t)(I4 ? a.N * a.K / 2 : a.N * a.K * 2));
  const __amdgpu_buffer_rsrc_t xrs = buffer_rsrc(xh, (uint32_t)(a.T * a.K * 2));
  const __amdgpu_buffer_rsrc_t srs = buffer_rsrc(a.wsc, (uint32_t)(I4 ? a.N * (a.K / 128) * 2 : 0));
  auto dma_x = [&](int st) {
    uint16_t* dst = lds + (st & (NSTAGE - 1)) * STAGE_ELEMS + wave * 4 * 512;
    const int64_t k0 = (int64_t)st * 32;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma_run(xrs, a.K, m0 + wave * 64 + j * 16, k0, dst + OP_ELEMS + j * 512);
  };
  auto dma_step = [&](int st) {
    uint16_t* dst = lds + (st & (NSTAGE - 1)) * STAGE_ELEMS + wave * 4 * 512;
    const int64_t k0 = (int64_t)st * 32;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma_run(wrs, a.K, n0 + wave * 64 + j * 16, k0, dst + j * 512);
    dma_x(st);
  };
  // INT4: row n0 + wave * 64 + lane of stage st: 16 packed bytes (32 depth values) into the
  // packed ring, and the row's group-128 scale into the scale ring
  char* const pk_base = reinterpret_cast<char*>(lds) + NSTAGE * STAGE_ELEMS * 2;
  char* const sc_base = pk_base + PK_STAGES * PK_BYTES;
  const int64_t my_row = n0 + wave * 64 + lane;
  auto dma_packed = [&](int st) {
    const int slot = st % PK_STAGES;
    const uint32_t poff = (uint32_t)(my_row * (a.K / 2) + (int64_t)st * 16);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void_t*)(pk_base + slot * PK_BYTES + wave * 1024), 16, poff, 0,
                                             0, 0);
    const uint32_t soff = (uint32_t)((my_row * (a.K / 128) + st / 4) * 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void_t*)(sc_base + slot * SC_BYTES + wave * 256), 2, soff, 0,
                                             0, 0);
  };
  // INT4: dequantise this lane's row of stage st (bf16(q * s), 32 values) into the W tile
  uint4 pk_q = make_uint4(0u, 0u, 0u, 0u);
  float pk_s = 0.f;
  auto pk_read = [&](int st) {
    const int slot = st % PK_STAGES;
    pk_q = *reinterpret_cast<const uint4*>(pk_base + slot * PK_BYTES + wave * 1024 + lane * 16);
    pk_s = bf2f((uint16_t)*reinterpret_cast<const uint32_t*>(sc_base + slot * SC_BYTES + wave * 256 + lane * 4));
  };
  // the same inside the main loop, as inline assembly: a plain LDS read here would make the
  // compiler wait for every direct-to-LDS load in flight.  The caller's end-of-step
  // lgkmcnt(0) lands the values before the next step uses them; the slot read was filled
  // three steps earlier and has been waited for.
  auto lds_addr = [](const void* p) {
    return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p);
  };
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  uint32_t pk_sbits = 0;
  u32x4 pk_qv = {0u, 0u, 0u, 0u};
  auto pk_read_async = [&](int st) {
    const int slot = st % PK_STAGES;
    asm volatile("ds_read_b128 %0, %1" : "=v"(pk_qv) : "v"(lds_addr(pk_base + slot * PK_BYTES + wave * 1024 + lane * 16)) : "memory");
    asm volatile("ds_read_b32 %0, %1" : "=v"(pk_sbits) : "v"(lds_addr(sc_base + slot * SC_BYTES + wave * 256 + lane * 4)) : "memory");
  };
  auto pk_take = [&]() {
    pk_q = make_uint4(pk_qv.x, pk_qv.y, pk_qv.z, pk_qv.w);
    pk_s = bf2f((uint16_t)pk_sbits);
  };
  auto pk_write = [&](int st, int c) {
    const uint32_t qw = c == 0 ? pk_q.x : (c == 1 ? pk_q.y : (c == 2 ? pk_q.z : pk_q.w));
    *reinterpret_cast<uint4*>(lds + (st & (NSTAGE - 1)) * STAGE_ELEMS + swz32(wave * 64 + lane, c)) =
        dequant8(qw, pk_s);
  };
  // the same in eight slices (half a 16-byte chunk each), one per row of MFMAs.  The store
  // is issued as inline assembly: the compiler would otherwise make it wait for every
  // direct-to-LDS load in flight (it cannot tell they target other LDS ranges), which would
  // drain the prefetch pipeline every step.  The W tile it writes has no load in flight, and
  // the end-of-step lgkmcnt(0) covers the store.
  auto lds_store16 = [&](const uint16_t* dst, uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3) {
    const u32x4 v = {a0, a1, a2, a3};
    asm volatile("ds_write_b128 %0, %1" ::"v"(lds_addr(dst)), "v"(v) : "memory");
  };
  uint32_t pk_half[2];
  auto pk_slice = [&](int st, int i) {
    const int c = i >> 1, hh = i & 1;
    const uint32_t qw = c == 0 ? pk_q.x : (c == 1 ? pk_q.y : (c == 2 ? pk_q.z : pk_q.w));
    const uint32_t q = qw >> (16 * hh);
    uint16_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = f2bf((float)(((int)(q << (28 - 4 * j))) >> 28) * pk_s);
    const uint32_t lo = pack2(o[0], o[1]), hi = pack2(o[2], o[3]);
    if (hh == 0) {
      pk_half[0] = lo;
      pk_half[1] = hi;
    } else {
      lds_store16(lds + (st & (NSTAGE - 1)) * STAGE_ELEMS + swz32(wave * 64 + lane, c), pk_half[0], pk_half[1], lo, hi);
    }
  };

  floatx4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
  bf16x8 fa0[8], fb0[8], fa1[8], fb1[8];

  auto read_frags = [&](int st, bf16x8 (&fa)[8], bf16x8 (&fb)[8]) {
    const uint16_t* sp = lds + (st & (NSTAGE - 1)) * STAGE_ELEMS;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      fa[i] = *reinterpret_cast<const bf16x8*>(sp + swz32(wn0 + i * 16 + lr, lk));
      fb[i] = *reinterpret_cast<const bf16x8*>(sp + OP_ELEMS + swz32(wm0 + i * 16 + lr, lk));
    }
  };
  // 64 MFMAs on (fa, fb) while the fragments of the next step are read into (na, nb) and
  // the 8 DMA runs of step dma_st are issued, one after each row of 8 MFMAs, so that the
  // CU's vector-memory path never holds the matrix core up.
  auto step_body = [&](bf16x8 (&fa)[8], bf16x8 (&fb)[8], bf16x8 (&na)[8], bf16x8 (&nb)[8], int next_st,
                       bool has_next, int dma_st, bool dma) {
    const uint16_t* sp = lds + (next_st & (NSTAGE - 1)) * STAGE_ELEMS;
    uint16_t* dst = lds + (dma_st & (NSTAGE - 1)) * STAGE_ELEMS + wave * 4 * 512;
    const int64_t k0 = (int64_t)dma_st * 32;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      if (dma) {
        if constexpr (I4) {
          // x runs in rows 0..3, the packed W and scales of stage dma_st + 2 in row 4, and one
          // slice of the dequantisation of stage next_st + 1 per row (its packed row was read
          // at the end of the previous step); the packed row of the next step's stage is read
          // after the last slice
          if (i < 4) dma_run(xrs, a.K, m0 + wave * 64 + i * 16, k0, dst + OP_ELEMS + i * 512);
          if (i == 4) dma_packed(dma_st + 2);
          pk_slice(next_st + 1, i);
          if (i == 7) pk_read_async(next_st + 2);
        } else {
          if (i < 4) dma_run(wrs, a.K, n0 + wave * 64 + i * 16, k0, dst + i * 512);
          else dma_run(xrs, a.K, m0 + wave * 64 + (i - 4) * 16, k0, dst + OP_ELEMS + (i - 4) * 512);
        }
      }
      // the next step's 16 fragment reads go out in the first half of the step, so they have
      // landed by the time the step ends
      if (has_next && i < 4) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int ii = 2 * i + h2;
          na[ii] = *reinterpret_cast<const bf16x8*>(sp + swz32(wn0 + ii * 16 + lr, lk));
          nb[ii] = *reinterpret_cast<const bf16x8*>(sp + OP_ELEMS + swz32(wm0 + ii * 16 + lr, lk));
        }
      }
      if constexpr (I4) {
        // rows that dequantise: interleave the conversion's VALU work between the MFMAs, so
        // the matrix core keeps busy while the wave converts (one wave per SIMD issues both)
        if (dma) {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);   // two VALU
          }
        }
      }
      // keep each row's MFMAs, DMA and fragment reads together (the loads stay spread over
      // the step instead of bunching at its ends)
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- prologue: coefficients, stages 0..3 in flight, C_h while they land, stages 0 and
  // 1 landed, fragments of step 0, then a barrier so that stage 0 may be refilled
  if constexpr (I4) {
    // x of stages 0..3, packed W of stages 0..5; all landed, then stages 0 and 1 dequantised
    // and the packed row of stage 2 (dequantised during step 0) read
    for (int st = 0; st < NSTAGE; ++st) dma_x(st);
    for (int st = 0; st < PK_STAGES; ++st) dma_packed(st);
    __builtin_amdgcn_s_waitcnt(WAIT_VM0);
    barrier();
    for (int st = 0; st < 2; ++st) {
      pk_read(st);
#pragma unroll
      for (int c = 0; c < 4; ++c) pk_write(st, c);
    }
    pk_read(2);
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    barrier();
  } else {
    const int npro = S < NSTAGE ? S : NSTAGE;
    for (int st = 0; st < npro; ++st) dma_step(st);
    if (HAS_R && a.ch == nullptr) {
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (q < qn) gen_chunk(q);
    }
    if (npro >= 4) __builtin_amdgcn_s_waitcnt(WAIT_VM16);
    else if (npro == 3) __builtin_amdgcn_s_waitcnt(WAIT_VM8);
    else __builtin_amdgcn_s_waitcnt(WAIT_VM0);
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    barrier();
  }
  read_frags(0, fa0, fb0);
  __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
  barrier();

  // ---- main loop, two steps per iteration (static fragment buffers).  At the end of step
  // s every wave has waited for the stage of step s + 2 (its own DMA two steps old), so
  // the barrier makes stage s + 2 visible before step s + 1 reads it.
  // Every step issues its DMA and its next-fragment reads, the last four included: their
  // stages are never read again (a DMA past the end of a row reads the next row, and past
  // the end of the matrix reads zeros), and the epilogue waits for all of them.  Constant
  // predicates leave the step free of branches.
  auto one_step = [&](int s, bf16x8 (&fa)[8], bf16x8 (&fb)[8], bf16x8 (&na)[8], bf16x8 (&nb)[8]) {
    step_body(fa, fb, na, nb, s + 1, true, s + 4, true);
    // the loads of steps s - 1 and s may stay in flight (8 runs per step; 6 with INT4 weights)
    __builtin_amdgcn_s_waitcnt(I4 ? WAIT_VM12 : WAIT_VM16);
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    barrier();
    if constexpr (I4) pk_take();
  };
  for (int s = 0; s < S; s += 2) {
    one_step(s, fa0, fb0, fa1, fb1);
    if (s + 1 < S) one_step(s + 1, fa1, fb1, fa0, fb0);
  }

  // ---- rank-r correction: [p[h] | C_h] as ceil(r/32) extra 32-deep steps.  Operands come
  // straight from global memory (p[h] rows, and C_h rows when precomputed; otherwise the
  // C_h region in LDS, r <= 64); a rank that is not a multiple of 8 is gathered element
  // by element, zero past r.
  if (HAS_R) {
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
        const int col = t * 32 + lk * 8;
        fb0[j] = row8(ph + m * a.r, col);
        if (I4 || a.ch != nullptr) {
          int64_t n = n0 + wn0 + j * 16 + lr;
          n = n > a.N - 1 ? a.N - 1 : n;
          fa0[j] = row8(chh + n * a.r, col);
        } else {
          fa0[j] = *reinterpret_cast<const bf16x8*>(chreg + swz(wn0 + j * 16 + lr, t * 4 + lk));
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa0[i], fb0[j], acc[i][j], 0, 0, 0);
    }
  }

  epilogue_4w<EPI, OUT_F32>(a, acc, lds, wave, lane, m0, n0, half, tm, tn);
}

template <int EPI, bool OUT_F32, bool HAS_R, bool I4>
hipError_t launch_4w(const GemmArgs& a, hipStream_t s) {
  constexpr int bytes = I4 ? LDS_BYTES_I4 : LDS_BYTES;
  static bool attr_set = false;  // benign race: every thread sets the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_4w_kernel<EPI, OUT_F32, HAS_R, I4>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const dim3 grid((unsigned)(2 * a.tiles_m_half * a.tiles_n));
  gemm_4w_kernel<EPI, OUT_F32, HAS_R, I4><<<grid, dim3(NT), bytes, s>>>(a);
  return hipGetLastError();
}

}  // namespace

// Returns hipErrorNotSupported outside this kernel's coverage: bf16 weights, or INT4 weights
// with the precomputed C_h (depth a multiple of 128); r <= 256 with the precomputed C_h,
// else r <= 64 and r % 8 == 0; depth a multiple of 32; a half of x or the weights below 2 GiB.
hipError_t launch_linear_pm_4w(const GemmArgs& a, int w_dtype, int epi, bool out_f32, hipStream_t s) {
  const bool i4 = w_dtype == ZOACT_INT4_G128;
  if (!(w_dtype == ZOACT_BF16 || (i4 && a.ch != nullptr && a.r > 0 && a.K % 128 == 0))) return hipErrorNotSupported;
  // ranks up to 256 and of any size read C_h precomputed; the in-kernel C_h covers r <= 64, r % 8 == 0
  if (a.ch == nullptr && (a.r > 64 || (a.r % 8) != 0)) return hipErrorNotSupported;
  if (a.r > 256 || (a.K % 32) != 0) return hipErrorNotSupported;
  if (a.T * a.K * 2 >= (int64_t(1) << 31) || a.N * a.K * 2 >= (int64_t(1) << 31)) return hipErrorNotSupported;
  // The correction-enabled instantiation also serves r = 0 (no chunks, no correction
  // steps): it is the one whose register assignment keeps the accumulators in AGPRs.
#define ZO_4W(EP, OF)                                               \
  if (epi == EP && out_f32 == OF)                                    \
    return i4 ? launch_4w<EP, OF, true, true>(a, s) : launch_4w<EP, OF, true, false>(a, s);
  ZO_4W(0, false)
  ZO_4W(0, true)
  ZO_4W(ZOACT_EPI_SWIGLU, false)
  ZO_4W(ZOACT_EPI_RELU, false)
  ZO_4W(EPI_MSE, false)
#undef ZO_4W
  return hipErrorNotSupported;
}

}  // namespace zoact

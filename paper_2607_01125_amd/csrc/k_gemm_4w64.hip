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
//  * Persistent workgroups (one per CU) walk their tiles back to back with the ring running
//    on: a tile's last two stages load the next tile's first two, so the next tile needs
//    no prologue, and the epilogue works from the accumulators without LDS while those
//    loads land.
#include <type_traits>

#include "gemm_4w_epi.hpp"

namespace zoact {

namespace {

using namespace gemm;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;
constexpr int SLOT_ELEMS = 256 * 64;                 // one operand tile, 64 deep (bf16 elements, 32 KB)
constexpr int NSLOT = 5;
constexpr int LDS_BYTES = NSLOT * SLOT_ELEMS * 2;    // 160 KB

// Byte offset of (row, 16-byte chunk c) in a 64-deep operand tile (rows of 128 bytes).
__device__ __forceinline__ int swz64(int row, int c) { return (row << 7) + ((c ^ (row & 7)) << 4); }

// One 1 KB load moves rows row0 .. row0+7 (row0 % 8 == 0), depth k0 .. k0+63 to LDS at
// dst: lane l lands at dst + 16 l, i.e. row l >> 3, LDS chunk l & 7, which holds global
// chunk (l & 7) ^ (l >> 3).  The per-lane part of the address (this offset, the same for
// every load of a wave) goes in the vector offset, the uniform part in the scalar one.
__device__ __forceinline__ int dma8_lane_off(int64_t ld) {
  const int lane = threadIdx.x & 63;
  return (int)((lane >> 3) * ld * 2 + (((lane & 7) ^ (lane >> 3)) << 4));
}

__device__ __forceinline__ int mod5(int v) { return v >= 5 ? v - 5 : v; }

// Split tail: with R = ntiles mod grid tiles left for a last, partly idle round (R at most
// half the grid), those R tiles are each computed as two halves of the depth by two
// workgroups (virtual tiles tail_first .. tail_first + 2R - 1, tail_first = ntiles - R), so
// the last round takes half the time.  The R tiles are the last tail_cols feature tiles
// with every token tile of both halves (R must be a multiple of the token tiles), so a
// tile and its twin in the other half are computed the same way: the two halves of the
// ± pair keep identical arithmetic.  A half tile stores its fp32 accumulators (in the
// accumulator layout, lane-major: coalesced) to tail_ws; a second kernel adds the two
// halves in the order first + second and runs the same epilogue.
struct VTile {
  int tile, k0, nst, kh;   // tile index, first 64-deep stage, stages, depth half (-1: whole)
};
__device__ __forceinline__ VTile vtile(const GemmArgs& a, int v, int NS) {
  if (v < a.tail_first) return VTile{v, 0, NS, -1};
  const int u = v - a.tail_first, h0 = (NS + 1) >> 1;
  return (u & 1) ? VTile{a.tail_first + (u >> 1), h0, NS - h0, 1} : VTile{a.tail_first + (u >> 1), 0, h0, 0};
}
// fp32 accumulators of half tile u (virtual index - tail_first): [u][wave][i * 8 + j][lane] x float4
__device__ __forceinline__ floatx4* tail_slot(const GemmArgs& a, int u, int wave) {
  return reinterpret_cast<floatx4*>(a.tail_ws) + ((int64_t)u * 4 + wave) * 64 * 64;
}

// Token tile, feature tile and half of virtual tile v of ntiles (XCD-contiguous runs,
// grouped token-major order: a workgroup's tiles v, v + grid, ... stay on its XCD when the
// grid is a multiple of 8).
struct TileGeom {
  int tm, tn, half;
  int64_t m0, n0;
};
__device__ __forceinline__ TileGeom tile_geom(const GemmArgs& a, int ntiles, int v, bool shared) {
  const int tiles_m = shared ? a.tiles_m_half : 2 * a.tiles_m_half;   // (shared input: one half's tokens)
  if (v >= a.tail_first) {   // split tail: feature tile columns past tiles_n - tail_cols
    const int t = v - a.tail_first;
    TileGeom g;
    g.tm = t % tiles_m;
    g.tn = a.tiles_n - a.tail_cols + t / tiles_m;
    g.half = shared ? 0 : g.tm / a.tiles_m_half;
    g.m0 = (int64_t)(g.tm % a.tiles_m_half) * 256;
    g.n0 = (int64_t)g.tn * 256;
    return g;
  }
  ntiles = a.tail_first;     // the tiles before the tail: tiles_n - tail_cols feature columns
  int lin = v;
  if ((ntiles & 7) == 0) lin = (v & 7) * (ntiles >> 3) + (v >> 3);
  const int per_group = 4 * (a.tiles_n - a.tail_cols);
  const int first_m = (lin / per_group) * 4;
  const int gsz = min(4, tiles_m - first_m);
  TileGeom g;
  g.tm = first_m + (lin % per_group) % gsz;
  g.tn = (lin % per_group) / gsz;
  g.half = shared ? 0 : g.tm / a.tiles_m_half;
  g.m0 = (int64_t)(g.tm % a.tiles_m_half) * 256;
  g.n0 = (int64_t)g.tn * 256;
  return g;
}

// Rank-r correction of one tile: [p[h] | C_h] as ceil(r/32) extra 32-deep steps added to
// the accumulators, operands from global memory (C_h precomputed) through buffer loads: rows
// past T or N read zeros (their outputs are not stored), columns past r are zeroed,
// element-wise when r is not a multiple of 8.  Past the plain feature range, C_h rows are
// shifted back by the range's width.  fa / fb are scratch fragment registers; with `pre`
// the first step's fragments come from pa / pb (rank_correction_pre).
template <bool PERM>
__device__ __forceinline__ void rank_correction(const GemmArgs& a, floatx4 (&acc)[8][8], bf16x8 (&fa)[8],
                                                bf16x8 (&fb)[8], const TileGeom& g, int p_half, int c_half,
                                                int wave, int lane, bool pre = false, const bf16x8* pa = nullptr,
                                                const bf16x8* pb = nullptr) {
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128, wm0 = (wave >> 1) * 128;
  const int prow = (lr >> 2) * 8 + (lr & 3);
  const int64_t plen = a.plain_end - a.plain_begin;
  const int kts = (a.r + 31) >> 5;
  const int64_t cn0 = g.n0 >= a.plain_end ? g.n0 - plen : g.n0;
  const __amdgpu_buffer_rsrc_t prs = buffer_rsrc(a.p + (int64_t)p_half * a.T * a.r, (uint32_t)(a.T * a.r * 2));
  const __amdgpu_buffer_rsrc_t crs =
      buffer_rsrc(a.ch + (int64_t)c_half * a.ch_stride, (uint32_t)((a.N - plen) * a.r * 2));
  const bool vec = (a.r & 7) == 0;
  const int pvo = ((wm0 + lr) * a.r + lk * 8) * 2, cvo = ((wn0 + (PERM ? prow : lr)) * a.r + lk * 8) * 2;
  // C_h rows of W block i (the permuted order with PERM): first row's byte offset
  auto crow = [&](int i) -> int {
    return (int)((cn0 + (PERM ? (i >> 1) * 32 + (i & 1) * 4 : i * 16)) * a.r * 2);
  };
  for (int t = 0; t < kts; ++t) {
    const int col = t * 32 + lk * 8;
    // every load issued before any result is used (one wait), then columns past r zeroed
    if (pre && t == 0) {
      const bool z = col >= a.r;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        fa[j] = z ? bf16x8{} : pa[j];
        fb[j] = z ? bf16x8{} : pb[j];
      }
    } else if (vec) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        fb[j] = __builtin_bit_cast(
            bf16x8, __builtin_amdgcn_raw_buffer_load_b128(prs, pvo, (int)((g.m0 + j * 16) * a.r * 2) + t * 64, 0));
        fa[j] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(crs, cvo, crow(j) + t * 64, 0));
      }
      if (col >= a.r) {
#pragma unroll
        for (int j = 0; j < 8; ++j) fb[j] = fa[j] = bf16x8{};
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint16_t ep[8], ec[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          ep[q] = __builtin_amdgcn_raw_buffer_load_b16(prs, pvo, (int)((g.m0 + j * 16) * a.r * 2) + t * 64 + 2 * q, 0);
          ec[q] = __builtin_amdgcn_raw_buffer_load_b16(crs, cvo, crow(j) + t * 64 + 2 * q, 0);
        }
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (col + q >= a.r) ep[q] = ec[q] = 0;
        fb[j] = __builtin_bit_cast(bf16x8, make_uint4(pack2(ep[0], ep[1]), pack2(ep[2], ep[3]), pack2(ep[4], ep[5]),
                                                       pack2(ep[6], ep[7])));
        fa[j] = __builtin_bit_cast(bf16x8, make_uint4(pack2(ec[0], ec[1]), pack2(ec[2], ec[3]), pack2(ec[4], ec[5]),
                                                       pack2(ec[6], ec[7])));
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  }
}

// The first 32-deep correction step's fragments (r a multiple of 8), loaded at the start of
// a tile so that their latency passes under its main loop (columns past r are zeroed where
// rank_correction takes them).  Only the SwiGLU kernel holds the 64 extra registers
// without spilling; there the loads cost the first stage's wait little and the correction
// ran 0.9% faster per gate|up launch.
template <bool PERM>
__device__ __forceinline__ void rank_correction_pre(const GemmArgs& a, const TileGeom& g, int p_half, int c_half,
                                                    int wave, int lane, bf16x8 (&pa)[8], bf16x8 (&pb)[8]) {
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128, wm0 = (wave >> 1) * 128;
  const int prow = (lr >> 2) * 8 + (lr & 3);
  const int64_t plen = a.plain_end - a.plain_begin;
  const int64_t cn0 = g.n0 >= a.plain_end ? g.n0 - plen : g.n0;
  const __amdgpu_buffer_rsrc_t prs = buffer_rsrc(a.p + (int64_t)p_half * a.T * a.r, (uint32_t)(a.T * a.r * 2));
  const __amdgpu_buffer_rsrc_t crs =
      buffer_rsrc(a.ch + (int64_t)c_half * a.ch_stride, (uint32_t)((a.N - plen) * a.r * 2));
  const int pvo = ((wm0 + lr) * a.r + lk * 8) * 2, cvo = ((wn0 + (PERM ? prow : lr)) * a.r + lk * 8) * 2;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    pb[j] = __builtin_bit_cast(bf16x8,
                               __builtin_amdgcn_raw_buffer_load_b128(prs, pvo, (int)((g.m0 + j * 16) * a.r * 2), 0));
    pa[j] = __builtin_bit_cast(
        bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                    crs, cvo, (int)((cn0 + (PERM ? (j >> 1) * 32 + (j & 1) * 4 : j * 16)) * a.r * 2), 0));
  }
}

// Persistent: the grid holds one workgroup per CU and each walks tiles v = blockIdx.x,
// + gridDim.x, ...  The stage ring runs on across tiles: the last two stages of a tile
// load the next tile's stages 0 and 1, and its last sub-step reads the next tile's first
// fragments, so the next tile starts without a prologue while this one finishes (rank
// correction, epilogue straight from the accumulators, no LDS).
template <int EPI, bool OUT_F32, bool SHARED>
__global__ void __launch_bounds__(NT, 1) gemm_4w64_kernel(GemmArgs a, int ntiles, int nvirt) {
  constexpr bool PERM = epi_perm(EPI);
  extern __shared__ __align__(16) uint16_t lds[];
  char* const lb = reinterpret_cast<char*>(lds);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // uniform: kept in SGPRs
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128;   // features of this wave
  const int wm0 = (wave >> 1) * 128;  // tokens of this wave
  const int NS = (int)(a.K >> 6);     // 64-deep stages (at least 2)
  const uint32_t xbytes = (uint32_t)(a.T * a.K * 2);

  const __amdgpu_buffer_rsrc_t wrs = buffer_rsrc(a.w, (uint32_t)(a.N * a.K * 2));
  const int loff = dma8_lane_off(a.K);
  // Load i (rows 8i .. 8i+7) of this wave's 64 rows of one operand into slot `slot`; `base`
  // is the byte offset of the wave's first row at the stage's depth (see src_base).
  const int row8_bytes = (int)(a.K * 16);   // 8 rows
  auto dma = [&](__amdgpu_buffer_rsrc_t rs, int base, int slot, int i) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(lb + slot * (SLOT_ELEMS * 2) + (wave * 64 + i * 8) * 128),
                                             16, loff, base + i * row8_bytes, 0, 0);
  };
  auto src_base = [&](int64_t rows, int64_t k0) -> int { return (int)(((rows + wave * 64) * a.K + k0) * 2); };

  floatx4 acc[8][8];
  bf16x8 fa0[8], fb0[8], fa1[8], fb1[8];

  // fragment offsets inside a slot.  x block j: row (wm0 + j * 16 + lr), chunk 4 kh + lk; the
  // swizzle term depends on lr only, so k-half kh has one per-lane offset.  W block i: the
  // same, or with PERM the rows of block pair q = i / 2 interleaved so that the outputs of
  // lane (lr, lk) in blocks 2q and 2q + 1 are 8 consecutive features: A-row r of block 2q + h
  // is feature q * 32 + (r / 4) * 8 + h * 4 + r % 4 (row r % 4 + 4 h modulo 8 for the swizzle).
  const int fo0 = swz64(lr, lk), fo1 = swz64(lr, 4 + lk);
  const int prow = (lr >> 2) * 8 + (lr & 3);
  const int fw[2][2] = {{PERM ? swz64(prow, lk) : fo0, PERM ? swz64(prow, 4 + lk) : fo1},
                        {PERM ? swz64(prow + 4, lk) : fo0, PERM ? swz64(prow + 4, 4 + lk) : fo1}};
  auto frag = [&](int slot, int row0, int fo) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(lb + slot * (SLOT_ELEMS * 2) + row0 * 128 + fo);
  };
  // W fragment of block i, k-half kh
  auto wfrag = [&](int slot, int i, int kh) -> bf16x8 {
    return frag(slot, PERM ? wn0 + (i >> 1) * 32 : wn0 + i * 16, fw[i & 1][kh]);
  };

  // One 32-deep sub-step: 64 MFMAs on (fa, fb); the next sub-step's 16 fragments (slots
  // nws / nxs, k-half nkh) are read in the first four rows; one load of operand
  // `rs` from byte offset `base` into slot dslot after each row of MFMAs.
  auto sub_step = [&](bf16x8 (&fa)[8], bf16x8 (&fb)[8], bf16x8 (&na)[8], bf16x8 (&nb)[8], int nws, int nxs, int nkh,
                      __amdgpu_buffer_rsrc_t rs, int base, int dslot) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      dma(rs, base, dslot, i);
      if (i < 4) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int ii = 2 * i + h2;
          na[ii] = wfrag(nws, ii, nkh);
          nb[ii] = frag(nxs, wm0 + ii * 16, nkh ? fo1 : fo0);
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

  int v = blockIdx.x;
  VTile vt = vtile(a, v, NS);
  TileGeom g = tile_geom(a, ntiles, vt.tile, SHARED);
  __amdgpu_buffer_rsrc_t xrs = buffer_rsrc(a.x + (int64_t)g.half * a.T * a.K, xbytes);

  // ---- prologue of the first tile: stages 0 and 1 in flight (slots 0..3), stage 0
  // landed in every wave's rows (the barrier)
  {
    const int64_t kb = (int64_t)vt.k0 * 64;
#pragma unroll
    for (int i = 0; i < 8; ++i) dma(wrs, src_base(g.n0, kb), 0, i);
#pragma unroll
    for (int i = 0; i < 8; ++i) dma(xrs, src_base(g.m0, kb), 1, i);
#pragma unroll
    for (int i = 0; i < 8; ++i) dma(wrs, src_base(g.n0, kb + 64), 2, i);
#pragma unroll
    for (int i = 0; i < 8; ++i) dma(xrs, src_base(g.m0, kb + 64), 3, i);
  }
  __builtin_amdgcn_s_waitcnt(WAIT_VM16);
  barrier();

  // s5 = 2S mod 5 over the whole sequence of stages (tiles back to back): stage S has W in
  // slot s5 and x in s5 + 1, stage S + 1 in s5 + 2 / s5 + 3, and stage S + 2 goes to
  // s5 + 4 (W, during sub-step 2S) and s5 (x, during 2S + 1).
  int s5 = 0;
  for (;;) {
    // fragments of the tile's first sub-step: stage 0 has landed (the prologue's barrier,
    // or the previous tile's barrier after its second-last sub-step) and its slots are
    // not refilled before sub-step 1.  (The previous tile's last sub-step read them too;
    // reading them again here keeps those registers free through its epilogue.)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      fa0[i] = wfrag(s5, i, 0);
      fb0[i] = frag(mod5(s5 + 1), wm0 + i * 16, fo0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int p_half = SHARED ? 0 : g.half, c_half = SHARED ? 1 : g.half;
    const bool corr = a.r > 0 && vt.kh <= 0 && !(g.n0 >= a.plain_begin && g.n0 < a.plain_end);
    // (the first correction step's operands requested now, see rank_correction_pre)
    const bool pre = EPI == ZOACT_EPI_SWIGLU && corr && (a.r & 7) == 0;
    bf16x8 cpa[8], cpb[8];
    if (pre) rank_correction_pre<PERM>(a, g, p_half, c_half, wave, lane, cpa, cpb);
    // nothing from LDS in flight when the main loop starts (as at the end of each of its
    // iterations), so the compiler places no LDS waits inside it
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    const int vn = v + (int)gridDim.x;
    const bool has_next = vn < nvirt;
    const VTile vtn = vtile(a, has_next ? vn : v, NS);
    const TileGeom gn = tile_geom(a, ntiles, vtn.tile, SHARED);
    const __amdgpu_buffer_rsrc_t xrs_n = buffer_rsrc(a.x + (int64_t)gn.half * a.T * a.K, xbytes);

    // ---- main loop: one stage (two sub-steps) per iteration.  Stages S + 2 past this
    // tile's end are the next tile's stages 0 and 1; after the last tile they re-read the
    // rows past the end (or zeros) into slots nobody reads again.
    // (The second sub-step sits under a test that always holds: written this way the
    // register allocator keeps every accumulator in place across the loop.)
    const int nst = vt.nst;
    const int nsub = 2 * nst;
    for (int j = 0; j < nsub; j += 2) {
      const int st = j >> 1;
      const bool nx = has_next && st + 2 >= nst;
      const int64_t kd = (int64_t)(nx ? vtn.k0 + st + 2 - nst : vt.k0 + st + 2) * 64;
      const int wb = src_base(nx ? gn.n0 : g.n0, kd), xb = src_base(nx ? gn.m0 : g.m0, kd);
      const __amdgpu_buffer_rsrc_t xr = nx ? xrs_n : xrs;
      const int sw1 = mod5(s5 + 2), sx1 = mod5(s5 + 3), sw2 = mod5(s5 + 4);
      // sub-step 2S: k-half 0 of stage S; reads k-half 1 of stage S; loads W of stage S + 2
      sub_step(fa0, fb0, fa1, fb1, s5, mod5(s5 + 1), 1, wrs, wb, sw2);
      // stage S + 1 (issued during sub-steps 2S - 2 and 2S - 1) must have landed: the
      // eight loads of this sub-step may stay in flight
      __builtin_amdgcn_s_waitcnt(WAIT_VM8);
      __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
      barrier();
      if (j + 1 < nsub) {
        // sub-step 2S + 1: k-half 1 of stage S; reads k-half 0 of stage S + 1 (the next
        // tile's stage 0 after the last stage); loads x of S + 2.  No barrier after it:
        // sub-step 2S + 2 reads stage S + 1 (complete since the barrier above) and loads
        // into stage S's x slot (last read during 2S), so nothing it touches can still be
        // in use by a slower wave.
        sub_step(fa1, fb1, fa0, fb0, sw1, sx1, 0, xr, xb, s5);
        __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
        __builtin_amdgcn_sched_barrier(0);
      }
      s5 = sw1;
    }

    // EPI_MSE: the target rows, requested now so that their latency overlaps what follows
    uint4 tq[8][4];
    epi_rows_early<EPI>(a, tq, wave, lane, g.m0, g.n0);
    if constexpr (SHARED) {
      // shared input: half 0 first, from the base with its correction applied in VGPR-form
      // MFMAs so that the base stays in the accumulators; half 1 then as in the stacked form
      epilogue_regs<EPI, OUT_F32, true>(a, acc, tq, wave, lane, g.m0, g.n0, 0, g.tm, g.tn);
      // (EPI_MSE: half 1 compares against the same target rows, still in tq)
    }

    // ---- rank-r correction (with the shared input: the shared p and C_1, for half 1); a
    // tile inside the plain feature range has none
    if (corr) rank_correction<PERM>(a, acc, fa1, fb1, g, p_half, c_half, wave, lane, pre, cpa, cpb);

    if (vt.kh >= 0) {
      // half a tile: its accumulators to the split tail's slot, the epilogue runs later
      floatx4* slot = tail_slot(a, v - a.tail_first, wave);
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          floatx4 t;
#pragma unroll
          for (int e = 0; e < 4; ++e) t[e] = acc_read(acc[i][j][e]);
          slot[(i * 8 + j) * 64 + lane] = t;
        }
    } else {
      epilogue_regs<EPI, OUT_F32>(a, acc, tq, wave, lane, g.m0, g.n0, SHARED ? 1 : g.half, g.tm, g.tn);
    }
    if (!has_next) break;
    v = vn;
    vt = vtn;
    g = gn;
    xrs = xrs_n;
  }
  // the loads past the last stage must land before the workgroup ends
  __builtin_amdgcn_s_waitcnt(WAIT_VM0);
}

// The split tail's R tiles: workgroup t adds the two halves of tile tail_first + t (first +
// second, the same order for every run) and runs the tile's epilogue on the sum.
template <int EPI, bool OUT_F32>
__global__ void __launch_bounds__(NT, 1) tail_combine_kernel(GemmArgs a, int ntiles) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x;
  const TileGeom g = tile_geom(a, ntiles, a.tail_first + t, false);
  const floatx4* h0 = tail_slot(a, 2 * t, wave);
  const floatx4* h1 = tail_slot(a, 2 * t + 1, wave);
  floatx4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = h0[(i * 8 + j) * 64 + lane] + h1[(i * 8 + j) * 64 + lane];
  uint4 tq[8][4];
  epilogue_regs<EPI, OUT_F32>(a, acc, tq, wave, lane, g.m0, g.n0, g.half, g.tm, g.tn);
}

// ---------------------------------------------------------------------------------------
// INT4 weights (group-128 scales) on the 64-deep persistent schedule.
//
// Only the packed weights and their scales travel global -> LDS: a stage's W is 256 rows x
// 32 bytes (8 KB, a quarter of the bf16 tile) plus one scale per row.  Each lane owns one
// row of the tile (wave * 64 + lane): it reads its packed half rows and writes bf16(q * s)
// into a bf16 W tile, the values zoact_dequant_int4 forms, so the fragments, MFMAs, rank
// correction and epilogue are those of the bf16 schedule with the dequantised weight (its
// results are the same bits).  A wave converts the rows it loaded itself, so the packed
// ring needs no barrier; the conversion of a stage is spread, four values (half a 16-byte
// chunk) per row of MFMAs, over the two sub-steps before the barrier that publishes it.
//
// LDS: four 32 KB bf16 slots (stage S: W in slot 2 (S & 1), x in 2 (S & 1) + 1) and a
// three-stage ring of packed W (8 KB) and scales (1 KB; a 2-byte direct-to-LDS load fills
// a 4-byte slot per lane).  Per stage S:
//  * sub-step 2S: MFMAs on k-half 0 of S while k-half 1 of S is read; packed W and scales
//    of stage S + 3 loaded into S's packed slot (converted by now); k-half 1 of W(S + 1)
//    converted.
//  * wait + barrier: x of S + 1 and packed W of S + 2 have landed (only S + 3's loads
//    may stay in flight); W(S + 1) is complete in LDS.
//  * sub-step 2S + 1: MFMAs on k-half 1 of S while k-half 0 of S + 1 is read; x of S + 2
//    loaded into x(S)'s slot and k-half 0 of W(S + 2) converted into W(S)'s slot (both
//    left at the barrier).
// x has one to two sub-steps to land, as in the bf16 ring; packed W three stages.
constexpr int I4_BF16_BYTES = 4 * SLOT_ELEMS * 2;                                 // 128 KB
constexpr int I4_PK_BYTES = 256 * 32;
constexpr int I4_SC_BYTES = 256 * 4;
constexpr int I4_LDS_BYTES = I4_BF16_BYTES + 3 * (I4_PK_BYTES + I4_SC_BYTES);    // 155 KB
constexpr int WAIT_VM3 = 0x0F73;

// Values 0..3 of dequant8: the four nibbles in the low 16 bits of q, scale s.
__device__ __forceinline__ uint2 dequant4(uint32_t q, float s) {
  uint16_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = ((int)(q << (28 - 4 * j))) >> 28;  // sign-extend nibble j
    o[j] = f2bf((float)v * s);
  }
  return make_uint2(pack2(o[0], o[1]), pack2(o[2], o[3]));
}

template <int EPI, bool OUT_F32>
__global__ void __launch_bounds__(NT, 1) gemm_i4w64_kernel(GemmArgs a, int ntiles) {
  constexpr bool PERM = epi_perm(EPI);
  extern __shared__ __align__(16) uint16_t lds[];
  char* const lb = reinterpret_cast<char*>(lds);
  char* const pkb = lb + I4_BF16_BYTES;
  char* const scb = pkb + 3 * I4_PK_BYTES;

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lk = lane >> 4;
  const int wn0 = (wave & 1) * 128;
  const int wm0 = (wave >> 1) * 128;
  const int NS = (int)(a.K >> 6);     // 64-deep stages (at least 4)
  const uint32_t xbytes = (uint32_t)(a.T * a.K * 2);
  const int64_t kp = a.K >> 1, kg = a.K >> 7;   // packed bytes and scale groups per row

  const __amdgpu_buffer_rsrc_t wrs = buffer_rsrc(a.w, (uint32_t)(a.N * kp));
  const __amdgpu_buffer_rsrc_t srs = buffer_rsrc(a.wsc, (uint32_t)(a.N * kg * 2));
  const int loff = dma8_lane_off(a.K);
  const int row8_bytes = (int)(a.K * 16);
  // x load i (rows 8i .. 8i+7 of this wave's 64) into bf16 slot `slot`
  auto dma_x = [&](__amdgpu_buffer_rsrc_t rs, int base, int slot, int i) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(lb + slot * (SLOT_ELEMS * 2) + (wave * 64 + i * 8) * 128),
                                             16, loff, base + i * row8_bytes, 0, 0);
  };
  auto x_base = [&](int64_t m0, int64_t k0) -> int { return (int)(((m0 + wave * 64) * a.K + k0) * 2); };
  // packed W of the stage at depth k0 for this wave's 64 rows into packed slot ps: load i
  // moves rows 32 i + l / 2, bytes 16 (l & 1) .. +15 (row-major 32-byte rows in LDS), then
  // one scale per row
  const int pk_loff = (int)((lane >> 1) * kp + (lane & 1) * 16);
  const int sc_loff = (int)(lane * kg * 2);
  auto dma_pk = [&](int64_t n0, int64_t k0, int ps, int i) {
    if (i < 2)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void_t*)(pkb + ps * I4_PK_BYTES + wave * 2048 + i * 1024), 16,
                                               pk_loff, (int)((n0 + wave * 64 + i * 32) * kp + (k0 >> 1)), 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void_t*)(scb + ps * I4_SC_BYTES + wave * 256), 2, sc_loff,
                                               (int)(((n0 + wave * 64) * kg + (k0 >> 7)) * 2), 0, 0);
  };
  // conversion of this lane's row: packed half row h of packed slot ps (16 bytes, 32
  // values) and its scale are read ahead (cv_read, then cv_wait); piece i
  // (0..7) turns values 4i .. 4i+3 into bf16, and every second piece stores a 16-byte chunk
  // of the bf16 row.  The packed reads and the chunk stores are inline assembly: as plain
  // LDS accesses the compiler would wait for every direct-to-LDS load in flight before
  // each of them (it cannot tell they touch other LDS ranges).  The packed rows read were
  // loaded by this wave and waited for; no load is in flight into the bf16 W slots.
  const int my_row = wave * 64 + lane;
  auto lds_addr = [](const void* p) {
    return (uint32_t)reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p);
  };
  u32x4 cq = {0u, 0u, 0u, 0u};
  uint32_t csb = 0;
  uint2 cpart = make_uint2(0u, 0u);
  auto cv_read = [&](int ps, int h) {
    asm volatile("ds_read_b128 %0, %1" : "=v"(cq) : "v"(lds_addr(pkb + ps * I4_PK_BYTES + my_row * 32 + h * 16)) : "memory");
    asm volatile("ds_read_b32 %0, %1" : "=v"(csb) : "v"(lds_addr(scb + ps * I4_SC_BYTES + wave * 256 + lane * 4)) : "memory");
  };
  // the wait for cv_read's values (and every other LDS access in flight): the compiler's
  // wait, then an empty inline assembly statement that takes and returns the values, so
  // that no use of them can be placed before the wait (the compiler does not know the
  // reads are in flight)
  auto cv_wait = [&]() {
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    asm volatile("" : "+v"(cq), "+v"(csb)::"memory");
  };
  auto cv_piece = [&](int wslot, int h, int i) {
    const uint2 d = dequant4(cq[i >> 1] >> ((i & 1) * 16), bf2f((uint16_t)csb));
    if ((i & 1) == 0) {
      cpart = d;
    } else {
      const u32x4 vv = {cpart.x, cpart.y, d.x, d.y};
      asm volatile("ds_write_b128 %0, %1" ::"v"(lds_addr(lb + wslot * (SLOT_ELEMS * 2) + swz64(my_row, 4 * h + (i >> 1)))),
                   "v"(vv) : "memory");
    }
  };

  floatx4 acc[8][8];
  bf16x8 fa0[8], fb0[8], fa1[8], fb1[8];
  const int fo0 = swz64(lr, lk), fo1 = swz64(lr, 4 + lk);
  const int prow = (lr >> 2) * 8 + (lr & 3);
  const int fw[2][2] = {{PERM ? swz64(prow, lk) : fo0, PERM ? swz64(prow, 4 + lk) : fo1},
                        {PERM ? swz64(prow + 4, lk) : fo0, PERM ? swz64(prow + 4, 4 + lk) : fo1}};
  auto frag = [&](int slot, int row0, int fo) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(lb + slot * (SLOT_ELEMS * 2) + row0 * 128 + fo);
  };
  auto wfrag = [&](int slot, int i, int kh) -> bf16x8 {
    return frag(slot, PERM ? wn0 + (i >> 1) * 32 : wn0 + i * 16, fw[i & 1][kh]);
  };

  // One 32-deep sub-step: 64 MFMAs on (fa, fb); the next sub-step's fragments (slots nws /
  // nxs, k-half nkh) read in the first four rows; one piece of the conversion of the half
  // row in cq (k-half ch) into bf16 slot cws per row.  SUB_B: an x load per row (rs, base -> slot dslot);
  // else the packed loads of stage (pn0, pk0) into packed slot ps in rows 0..2.
  auto sub_step = [&](auto sub_b, bf16x8 (&fa)[8], bf16x8 (&fb)[8], bf16x8 (&na)[8], bf16x8 (&nb)[8], int nws,
                      int nxs, int nkh, __amdgpu_buffer_rsrc_t rs, int base, int dslot, int64_t pn0, int64_t pk0,
                      int ps, int cws, int ch) {
    constexpr bool SUB_B = decltype(sub_b)::value;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      if constexpr (SUB_B) {
        dma_x(rs, base, dslot, i);
      } else {
        if (i < 3) dma_pk(pn0, pk0, ps, i);
      }
      if (i < 4) {
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
          const int ii = 2 * i + h2;
          na[ii] = wfrag(nws, ii, nkh);
          nb[ii] = frag(nxs, wm0 + ii * 16, nkh ? fo1 : fo0);
        }
      }
      cv_piece(cws, ch, i);
      const bool vm = SUB_B || i < 3;
      if (vm) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);    // the direct-to-LDS load
      }
      // the conversion arithmetic spread evenly over the row's MFMAs (measured 1-2% faster
      // than grouping it after fewer of them)
      if (i < 4) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one fragment read
          __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);  // conversion arithmetic
        }
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 7; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
        }
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);      // the rest of the row
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  using SubA = std::integral_constant<bool, false>;
  using SubB = std::integral_constant<bool, true>;

  int v = blockIdx.x;
  TileGeom g = tile_geom(a, ntiles, v, false);
  __amdgpu_buffer_rsrc_t xrs = buffer_rsrc(a.x + (int64_t)g.half * a.T * a.K, xbytes);

  // ---- prologue of the first tile: packed stages 0..2, x of stages 0 and 1; W of stage 0
  // and k-half 0 of W(1) converted (k-half 1 of W(1) is the first sub-step's), published by
  // the barrier
#pragma unroll
  for (int i = 0; i < 3; ++i) dma_pk(g.n0, 0, 0, i);
#pragma unroll
  for (int i = 0; i < 3; ++i) dma_pk(g.n0, 64, 1, i);
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_x(xrs, x_base(g.m0, 0), 1, i);
#pragma unroll
  for (int i = 0; i < 8; ++i) dma_x(xrs, x_base(g.m0, 64), 3, i);
#pragma unroll
  for (int i = 0; i < 3; ++i) dma_pk(g.n0, 128, 2, i);
  __builtin_amdgcn_s_waitcnt(WAIT_VM3);
  const int pslot[3][2] = {{0, 0}, {0, 1}, {1, 0}};   // (packed slot, half) -> bf16 slot 0, 0, 2
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    cv_read(pslot[c][0], pslot[c][1]);
    cv_wait();
#pragma unroll
    for (int i = 0; i < 8; ++i) cv_piece(c == 2 ? 2 : 0, pslot[c][1], i);
  }
  cv_read(1, 1);   // k-half 1 of W(1), converted by the first sub-step
  cv_wait();
  barrier();

  // global stage sequence (tiles back to back): stage gs in bf16 slots 2 par / 2 par + 1,
  // packed slot p3 = gs mod 3
  int par = 0, p3 = 0;
  for (;;) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      fa0[i] = wfrag(2 * par, i, 0);
      fb0[i] = frag(2 * par + 1, wm0 + i * 16, fo0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    __builtin_amdgcn_s_waitcnt(WAIT_LGKM0);
    const int vn = v + (int)gridDim.x;
    const bool has_next = vn < ntiles;
    const TileGeom gn = tile_geom(a, ntiles, has_next ? vn : v, false);
    const __amdgpu_buffer_rsrc_t xrs_n = buffer_rsrc(a.x + (int64_t)gn.half * a.T * a.K, xbytes);

    // ---- main loop: one stage per iteration.  Stages past this tile's end are the next
    // tile's (after the last tile: rows past the end or zeros, into slots nobody reads).
    // (cq holds k-half 1 of W(S + 1) when an iteration starts.  The second sub-step sits
    // under a test that always holds: written this way the register allocator keeps every
    // accumulator in place across the loop.)
    const int nsub = 2 * NS;
    for (int j = 0; j < nsub; j += 2) {
      const int st = j >> 1;
      const int par1 = par ^ 1;
      const int p31 = p3 == 2 ? 0 : p3 + 1, p32 = p31 == 2 ? 0 : p31 + 1;
      const bool nx3 = has_next && st + 3 >= NS;
      const int64_t k3 = (int64_t)(nx3 ? st + 3 - NS : st + 3) * 64;
      const bool nx2 = has_next && st + 2 >= NS;
      const int64_t k2 = (int64_t)(nx2 ? st + 2 - NS : st + 2) * 64;
      const int xb = x_base(nx2 ? gn.m0 : g.m0, k2);
      const __amdgpu_buffer_rsrc_t xr = nx2 ? xrs_n : xrs;
      // sub-step 2S: k-half 0 of S; reads k-half 1 of S; packed loads of S + 3; converts
      // k-half 1 of W(S + 1)
      sub_step(SubA{}, fa0, fb0, fa1, fb1, 2 * par, 2 * par + 1, 1, xr, xb, 0, nx3 ? gn.n0 : g.n0, k3, p3, 2 * par1, 1);
      // x of S + 1 and packed W of S + 2 have landed (S + 3's may stay in flight)
      __builtin_amdgcn_s_waitcnt(WAIT_VM3);
      cv_read(p32, 0);
      cv_wait();
      barrier();
      if (j + 1 < nsub) {
        // sub-step 2S + 1: k-half 1 of S; reads k-half 0 of S + 1; loads x of S + 2 into
        // x(S)'s slot; converts k-half 0 of W(S + 2) into W(S)'s slot
        sub_step(SubB{}, fa1, fb1, fa0, fb0, 2 * par1, 2 * par1 + 1, 0, xr, xb, 2 * par + 1, 0, 0, 0, 2 * par, 0);
        cv_read(p32, 1);
        cv_wait();
        __builtin_amdgcn_sched_barrier(0);
      }
      par = par1;
      p3 = p31;
    }

    uint4 tq[8][4];
    epi_rows_early<EPI>(a, tq, wave, lane, g.m0, g.n0);
    if (a.r > 0 && !(g.n0 >= a.plain_begin && g.n0 < a.plain_end))
      rank_correction<PERM>(a, acc, fa1, fb1, g, g.half, g.half, wave, lane);
    epilogue_regs<EPI, OUT_F32>(a, acc, tq, wave, lane, g.m0, g.n0, g.half, g.tm, g.tn);
    if (!has_next) break;
    v = vn;
    g = gn;
    xrs = xrs_n;
  }
  __builtin_amdgcn_s_waitcnt(WAIT_VM0);
}

template <int EPI, bool OUT_F32>
hipError_t launch_i4w64(const GemmArgs& a_in, hipStream_t s) {
  GemmArgs a = a_in;
  static bool attr_set = false;  // benign race: every thread sets the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_i4w64_kernel<EPI, OUT_F32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, I4_LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int ntiles = 2 * a.tiles_m_half * a.tiles_n;
  const int ncu = cu_count();
  if (ncu <= 0) return hipErrorInvalidDevice;
  const unsigned grid = (unsigned)(ntiles < ncu ? ntiles : ncu);
  a.tail_first = ntiles;
  a.tail_cols = 0;
  gemm_i4w64_kernel<EPI, OUT_F32><<<dim3(grid), dim3(NT), I4_LDS_BYTES, s>>>(a, ntiles);
  return hipGetLastError();
}

template <int EPI, bool OUT_F32, bool SHARED>
hipError_t launch_4w64(const GemmArgs& a_in, hipStream_t s) {
  GemmArgs a = a_in;
  static bool attr_set = false;  // benign race: every thread sets the same value
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_4w64_kernel<EPI, OUT_F32, SHARED>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, LDS_BYTES);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int ntiles = (SHARED ? 1 : 2) * a.tiles_m_half * a.tiles_n;
  const int ncu = cu_count();
  if (ncu <= 0) return hipErrorInvalidDevice;
  const unsigned grid = (unsigned)(ntiles < ncu ? ntiles : ncu);
  // the split tail where it applies: plain or ReLU outputs, a last round at most half
  // full after at least one full one and made of whole feature-tile columns, at least 4
  // stages (2 per half), a workspace
  const int rest = ntiles % (int)grid, tiles_m = 2 * a.tiles_m_half;
  const bool split = (EPI == 0 || EPI == ZOACT_EPI_RELU) && !SHARED && ntiles > (int)grid && rest > 0 &&
                     2 * rest <= (int)grid && rest % tiles_m == 0 && (a.K >> 6) >= 4 && a.tail_ws != nullptr &&
                     a.tail_ws_bytes >= (int64_t)rest * 2 * 4 * 64 * 64 * 16;
  a.tail_first = split ? ntiles - rest : ntiles;
  a.tail_cols = split ? rest / tiles_m : 0;
  const int nvirt = split ? ntiles + rest : ntiles;
  gemm_4w64_kernel<EPI, OUT_F32, SHARED><<<dim3(grid), dim3(NT), LDS_BYTES, s>>>(a, ntiles, nvirt);
  if constexpr ((EPI == 0 || EPI == ZOACT_EPI_RELU) && !SHARED) {
    if (split) tail_combine_kernel<EPI, OUT_F32><<<dim3((unsigned)rest), dim3(NT), 0, s>>>(a, ntiles);
  }
  return hipGetLastError();
}

}  // namespace

// Compute units of the current device (cached per device; every caller stores the same
// value, so concurrent first calls are harmless).  -1 on error.
int cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return -1;
  static int cache[64] = {};
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return -1;
    cache[dev] = n;
  }
  return cache[dev];
}


// Returns hipErrorNotSupported outside this schedule's coverage: bf16 weights; C_h
// precomputed (or r = 0), r <= 256; depth a multiple of 64, at least 128; a half of x,
// of p or of C_h, the weights, and the cross entropy's block partials, below 2 GiB.
// `shared`: x and p hold one half's rows, read by both (plain, ReLU or regression-loss
// epilogues; 8 <= r <= 32, a multiple of 8).
hipError_t launch_linear_pm_4w64(const GemmArgs& a, int w_dtype, int epi, bool out_f32, bool shared, hipStream_t s) {
  if (w_dtype != ZOACT_BF16 && w_dtype != ZOACT_INT4_G128) return hipErrorNotSupported;
  if (a.r > 0 && a.ch == nullptr) return hipErrorNotSupported;
  if (a.r > 256 || (a.K % 64) != 0 || a.K < 128) return hipErrorNotSupported;
  if (a.T * a.K * 2 >= (int64_t(1) << 31) || a.N * a.K * 2 >= (int64_t(1) << 31)) return hipErrorNotSupported;
  if (a.T * a.r * 2 >= (int64_t(1) << 31) || a.N * a.r * 2 >= (int64_t(1) << 31)) return hipErrorNotSupported;
  if (epi == EPI_XENT && 2 * a.T * (int64_t)a.xnblk * 8 >= (int64_t(1) << 31)) return hipErrorNotSupported;
  if (shared && (a.r < 8 || a.r > 32 || (a.r & 7) != 0)) return hipErrorNotSupported;
  if (a.plain_end > a.plain_begin && (shared || (a.plain_begin & 255) != 0 || (a.plain_end & 255) != 0))
    return hipErrorNotSupported;
  if (w_dtype == ZOACT_INT4_G128) {
    // packed weights: whole scale groups, at least four stages, plain / ReLU / SwiGLU outputs
    if (shared || a.wsc == nullptr || (a.K % 128) != 0 || a.K < 256) return hipErrorNotSupported;
    if (epi == 0 && !out_f32) return launch_i4w64<0, false>(a, s);
    if (epi == 0 && out_f32) return launch_i4w64<0, true>(a, s);
    if (epi == ZOACT_EPI_SWIGLU && !out_f32) return launch_i4w64<ZOACT_EPI_SWIGLU, false>(a, s);
    if (epi == ZOACT_EPI_RELU && !out_f32) return launch_i4w64<ZOACT_EPI_RELU, false>(a, s);
    return hipErrorNotSupported;
  }
#define ZO_4W64(EP, OF, SH) \
  if (epi == EP && out_f32 == OF && shared == SH) return launch_4w64<EP, OF, SH>(a, s);
  ZO_4W64(0, false, false)
  ZO_4W64(0, true, false)
  ZO_4W64(ZOACT_EPI_SWIGLU, false, false)
  ZO_4W64(ZOACT_EPI_RELU, false, false)
  ZO_4W64(EPI_MSE, false, false)
  ZO_4W64(EPI_XENT, false, false)
  ZO_4W64(0, false, true)
  ZO_4W64(0, true, true)
  ZO_4W64(ZOACT_EPI_RELU, false, true)
  ZO_4W64(EPI_MSE, false, true)
#undef ZO_4W64
  return hipErrorNotSupported;
}

}  // namespace zoact

// Z materialisation (test hook) and the ZO-Adam / ZO-SGD update over the arena.
//
// Algorithm 2: after the perturbed losses, the estimate g_B = a Z (a from the loss
// difference) drives an optimiser step on every coefficient matrix B_l; Section 5
// and Appendix B use Adam (weight decay 0) or SGD.  The two-sided form here uses
// a = (L+ - L-) / (2 eps) and regenerates the same Z the forward used.
//
// The update is HBM-bound: per coefficient it reads c, m, v and writes them back
// (24 bytes with fp32 C, 20 with bf16 C).  One thread owns one Philox counter
// block (4 consecutive arena indices, one Philox call) and moves them with
// 16-byte (8-byte for bf16 C) vector accesses; the arithmetic is fp32, one
// rounding per operation, in a fixed order.
#include "common.hpp"
#include "rng.hpp"

namespace zoact {

namespace {

__global__ void gen_z_kernel(uint64_t seed, uint32_t step, uint32_t query, int64_t e0, int64_t n, float* out) {
  const int64_t b0 = e0 >> 2;
  const int64_t b1 = (e0 + n - 1) >> 2;
  for (int64_t b = b0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b <= b1;
       b += (int64_t)gridDim.x * blockDim.x) {
    const float4 z = rng::gauss_block(seed, step, query, (uint64_t)b);
#pragma unroll
    for (int l = 0; l < 4; ++l) {
      const int64_t e = 4 * b + l;
      if (e >= e0 && e < e0 + n) out[e - e0] = rng::lane_of(z, l);
    }
  }
}

__device__ __forceinline__ float projected_grad(const float* loss_pm, float eps) {
#pragma clang fp contract(off)
  const float lp = loss_pm[0], lm = loss_pm[1];
  return (lp - lm) / (eps + eps);
}

struct AdamConst {
  float b1, b2, eps, wd, step_size, isb2, omb1, omb2;
};

__device__ __forceinline__ float adam_one(float c, float& m, float& v, float gh, const AdamConst& h) {
#pragma clang fp contract(off)
  if (h.wd != 0.0f) gh = gh + h.wd * c;
  m = h.b1 * m + h.omb1 * gh;
  v = h.b2 * v + h.omb2 * (gh * gh);
  const float d = __builtin_sqrtf(v) * h.isb2 + h.eps;
  return c - h.step_size * (m / d);
}

typedef float vf4 __attribute__((ext_vector_type(4)));
typedef uint32_t vu2 __attribute__((ext_vector_type(2)));

// Streaming (nontemporal) 16- and 8-byte accesses: every arena byte is touched once per
// step, so keeping it out of the caches leaves them to the data that is reused.
__device__ __forceinline__ vf4 ld_nt(const float* p) { return __builtin_nontemporal_load(reinterpret_cast<const vf4*>(p)); }
__device__ __forceinline__ void st_nt(float* p, vf4 v) { __builtin_nontemporal_store(v, reinterpret_cast<vf4*>(p)); }

// Four bf16 values (fp32 rounded to nearest even) in one 8-byte streaming store; p 8-byte aligned.
__device__ __forceinline__ void st4_bf16_nt(uint16_t* p, float a, float b, float c, float d) {
  const vu2 v = {(uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16), (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16)};
  __builtin_nontemporal_store(v, reinterpret_cast<vu2*>(p));
}

// C + s eps Z of one value for s in {-1, 0, +1} (fp32, no contraction).
__device__ __forceinline__ float pert_one(float c, float ez, int32_t s) {
#pragma clang fp contract(off)
  return s > 0 ? c + ez : (s < 0 ? c - ez : c);
}

// With NEXT, the same pass also writes the next step's perturbed coefficients from the C it
// leaves behind, exactly as perturb_kernel would over the whole arena (out bf16 [2][k]):
// out[h][e] = bf16(C'[e] + s_h (eps' Z(e; q'_h))), C' the stored value (bf16 C: the rounded
// one); with a non-finite g C is left unchanged and the perturbation is still written.
template <bool BF16C, bool NEXT>
__global__ void __launch_bounds__(256) adam_kernel(void* __restrict__ cptr, float* __restrict__ mptr,
                                                   float* __restrict__ vptr, int64_t k, const float* loss_pm,
                                                   uint64_t seed, uint32_t step, uint32_t query, float eps,
                                                   AdamConst h, uint32_t* status, zoact_pert_pair nx,
                                                   uint16_t* __restrict__ out) {
#pragma clang fp contract(off)
  const float g = projected_grad(loss_pm, eps);
  const bool upd = __builtin_isfinite(g);
  if (!upd) {
    if (status != nullptr && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, 1u);
    if (!NEXT) return;
  }
  // next perturbation of arena indices 4b .. 4b + nl - 1 from their stored values cs: a whole
  // block in two 8-byte stores when both halves' rows stay 8-byte aligned (k % 4 == 0)
  const bool vec_out = (k & 3) == 0;
  auto next_pert = [&](int64_t b, const float* cs, int nl) {
    const float4 za = rng::gauss_block(nx.seed, nx.step, nx.query[0], (uint64_t)b);
    const float4 zb = nx.query[0] == nx.query[1] ? za : rng::gauss_block(nx.seed, nx.step, nx.query[1], (uint64_t)b);
    if (nl == 4 && vec_out) {
      const int64_t e = 4 * b;
      st4_bf16_nt(out + e, pert_one(cs[0], nx.eps * za.x, nx.sign[0]), pert_one(cs[1], nx.eps * za.y, nx.sign[0]),
                  pert_one(cs[2], nx.eps * za.z, nx.sign[0]), pert_one(cs[3], nx.eps * za.w, nx.sign[0]));
      st4_bf16_nt(out + k + e, pert_one(cs[0], nx.eps * zb.x, nx.sign[1]), pert_one(cs[1], nx.eps * zb.y, nx.sign[1]),
                  pert_one(cs[2], nx.eps * zb.z, nx.sign[1]), pert_one(cs[3], nx.eps * zb.w, nx.sign[1]));
      return;
    }
    for (int l = 0; l < nl; ++l) {
      const int64_t e = 4 * b + l;
      const float c = cs[l];
      const float ea = nx.eps * rng::lane_of(za, l), eb = nx.eps * rng::lane_of(zb, l);
      out[e] = f2bf(nx.sign[0] > 0 ? c + ea : (nx.sign[0] < 0 ? c - ea : c));
      out[k + e] = f2bf(nx.sign[1] > 0 ? c + eb : (nx.sign[1] < 0 ? c - eb : c));
    }
  };
  const int64_t nb = (k + 3) >> 2;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nb; b += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e = 4 * b;
    if (e + 4 <= k) {
      float c0, c1, c2, c3;
      if (BF16C) {
        const vu2 cb = __builtin_nontemporal_load(reinterpret_cast<const vu2*>(reinterpret_cast<const uint16_t*>(cptr) + e));
        c0 = bf2f((uint16_t)(cb.x & 0xFFFFu)); c1 = bf2f((uint16_t)(cb.x >> 16));
        c2 = bf2f((uint16_t)(cb.y & 0xFFFFu)); c3 = bf2f((uint16_t)(cb.y >> 16));
      } else {
        const vf4 cf = ld_nt(reinterpret_cast<const float*>(cptr) + e);
        c0 = cf.x; c1 = cf.y; c2 = cf.z; c3 = cf.w;
      }
      if (upd) {
        vf4 m4 = ld_nt(mptr + e);
        vf4 v4 = ld_nt(vptr + e);
        const float4 z = rng::gauss_block(seed, step, query, (uint64_t)b);
        float mx = m4.x, my = m4.y, mz = m4.z, mw = m4.w, vx = v4.x, vy = v4.y, vz = v4.z, vw = v4.w;
        c0 = adam_one(c0, mx, vx, g * z.x, h);
        c1 = adam_one(c1, my, vy, g * z.y, h);
        c2 = adam_one(c2, mz, vz, g * z.z, h);
        c3 = adam_one(c3, mw, vw, g * z.w, h);
        st_nt(mptr + e, vf4{mx, my, mz, mw});
        st_nt(vptr + e, vf4{vx, vy, vz, vw});
        if (BF16C) {
          const vu2 cb = {(uint32_t)f2bf(c0) | ((uint32_t)f2bf(c1) << 16), (uint32_t)f2bf(c2) | ((uint32_t)f2bf(c3) << 16)};
          __builtin_nontemporal_store(cb, reinterpret_cast<vu2*>(reinterpret_cast<uint16_t*>(cptr) + e));
        } else {
          st_nt(reinterpret_cast<float*>(cptr) + e, vf4{c0, c1, c2, c3});
        }
      }
      if constexpr (NEXT) {
        const float cs[4] = {BF16C ? bf2f(f2bf(c0)) : c0, BF16C ? bf2f(f2bf(c1)) : c1, BF16C ? bf2f(f2bf(c2)) : c2,
                             BF16C ? bf2f(f2bf(c3)) : c3};
        next_pert(b, cs, 4);
      }
    } else {
      const float4 z = rng::gauss_block(seed, step, query, (uint64_t)b);
      float cs[4] = {0.f, 0.f, 0.f, 0.f};
      for (int l = 0; l < 4 && e + l < k; ++l) {
        float c = BF16C ? bf2f(reinterpret_cast<const uint16_t*>(cptr)[e + l])
                        : reinterpret_cast<const float*>(cptr)[e + l];
        if (upd) {
          float m = mptr[e + l], v = vptr[e + l];
          c = adam_one(c, m, v, g * rng::lane_of(z, l), h);
          mptr[e + l] = m;
          vptr[e + l] = v;
          if (BF16C) reinterpret_cast<uint16_t*>(cptr)[e + l] = f2bf(c);
          else reinterpret_cast<float*>(cptr)[e + l] = c;
        }
        cs[l] = BF16C ? bf2f(f2bf(c)) : c;
      }
      if constexpr (NEXT) next_pert(b, cs, (int)(k - e));
    }
  }
}

// adam_kernel<BF16C, true> for its common case: the next perturbation is the +/- pair of
// one query (signs +1, -1) and the arena holds whole Philox blocks (k % 4 == 0).  Per block
// the loads of C, m, v are issued first and both Gaussians (this step's, for the update, and
// the next step's) are formed while they are in flight; then the update, its stores, and
// the two 8-byte stores of the next step's C +/- eps Z.  Bit for bit adam_kernel<BF16C, true>.
template <bool BF16C>
__global__ void __launch_bounds__(256) adam_next_pm_kernel(void* __restrict__ cptr, float* __restrict__ mptr,
                                                           float* __restrict__ vptr, int64_t k, const float* loss_pm,
                                                           uint64_t seed, uint32_t step, uint32_t query, float eps,
                                                           AdamConst h, uint32_t* status, uint64_t nseed,
                                                           uint32_t nstep, uint32_t nquery, float neps,
                                                           uint16_t* __restrict__ out) {
#pragma clang fp contract(off)
  const float g = projected_grad(loss_pm, eps);
  const bool upd = __builtin_isfinite(g);
  if (!upd && status != nullptr && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, 1u);
  const int64_t nb = k >> 2;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nb; b += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e = 4 * b;
    float c[4];
    if (BF16C) {
      const vu2 cb = __builtin_nontemporal_load(reinterpret_cast<const vu2*>(reinterpret_cast<const uint16_t*>(cptr) + e));
      c[0] = bf2f((uint16_t)(cb.x & 0xFFFFu)); c[1] = bf2f((uint16_t)(cb.x >> 16));
      c[2] = bf2f((uint16_t)(cb.y & 0xFFFFu)); c[3] = bf2f((uint16_t)(cb.y >> 16));
    } else {
      const vf4 cf = ld_nt(reinterpret_cast<const float*>(cptr) + e);
      c[0] = cf.x; c[1] = cf.y; c[2] = cf.z; c[3] = cf.w;
    }
    vf4 m4 = {}, v4 = {};
    if (upd) {
      m4 = ld_nt(mptr + e);
      v4 = ld_nt(vptr + e);
    }
    const float4 zn = rng::gauss_block(nseed, nstep, nquery, (uint64_t)b);
    if (upd) {
      const float4 z = rng::gauss_block(seed, step, query, (uint64_t)b);
      float m[4] = {m4.x, m4.y, m4.z, m4.w}, v[4] = {v4.x, v4.y, v4.z, v4.w};
      const float zz[4] = {z.x, z.y, z.z, z.w};
#pragma unroll
      for (int l = 0; l < 4; ++l) c[l] = adam_one(c[l], m[l], v[l], g * zz[l], h);
      st_nt(mptr + e, vf4{m[0], m[1], m[2], m[3]});
      st_nt(vptr + e, vf4{v[0], v[1], v[2], v[3]});
      if (BF16C) {
#pragma unroll
        for (int l = 0; l < 4; ++l) c[l] = bf2f(f2bf(c[l]));   // the stored value
        const vu2 cb = {(uint32_t)f2bf(c[0]) | ((uint32_t)f2bf(c[1]) << 16),
                        (uint32_t)f2bf(c[2]) | ((uint32_t)f2bf(c[3]) << 16)};
        __builtin_nontemporal_store(cb, reinterpret_cast<vu2*>(reinterpret_cast<uint16_t*>(cptr) + e));
      } else {
        st_nt(reinterpret_cast<float*>(cptr) + e, vf4{c[0], c[1], c[2], c[3]});
      }
    }
    const float ez[4] = {neps * zn.x, neps * zn.y, neps * zn.z, neps * zn.w};
    st4_bf16_nt(out + e, c[0] + ez[0], c[1] + ez[1], c[2] + ez[2], c[3] + ez[3]);
    st4_bf16_nt(out + k + e, c[0] - ez[0], c[1] - ez[1], c[2] - ez[2], c[3] - ez[3]);
  }
}

template <bool BF16C>
__global__ void __launch_bounds__(256) sgd_kernel(void* __restrict__ cptr, int64_t k, const float* loss_pm,
                                                  uint64_t seed, uint32_t step, uint32_t query, float eps, float lr,
                                                  uint32_t* status) {
#pragma clang fp contract(off)
  const float g = projected_grad(loss_pm, eps);
  if (!__builtin_isfinite(g)) {
    if (status != nullptr && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, 1u);
    return;
  }
  const int64_t nb = (k + 3) >> 2;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nb; b += (int64_t)gridDim.x * blockDim.x) {
    const float4 z = rng::gauss_block(seed, step, query, (uint64_t)b);
    for (int l = 0; l < 4 && 4 * b + l < k; ++l) {
      const int64_t e = 4 * b + l;
      const float gh = g * rng::lane_of(z, l);
      if (BF16C) {
        uint16_t* c = reinterpret_cast<uint16_t*>(cptr);
        c[e] = f2bf(bf2f(c[e]) - lr * gh);
      } else {
        float* c = reinterpret_cast<float*>(cptr);
        c[e] = c[e] - lr * gh;
      }
    }
  }
}

// out[h][e - e0] = bf16(C[e] + s_h eps Z(e; q_h)) (s_h = 0: bf16(C[e])) for a range of whole
// Philox blocks (e0 % 4 == 0, n % 4 == 0): per block one 16-byte (8-byte with bf16 C)
// streaming load of C and one 8-byte streaming store per half.  HBM-bound: 8 (6) bytes per
// coefficient.
template <bool BF16C>
__global__ void __launch_bounds__(256) perturb_vec_kernel(const void* __restrict__ cptr, int64_t e0, int64_t n,
                                                          uint64_t seed, uint32_t step, uint32_t q0, uint32_t q1,
                                                          int32_t s0, int32_t s1, float eps,
                                                          uint16_t* __restrict__ out) {
#pragma clang fp contract(off)
  const int64_t nb = n >> 2, b0 = e0 >> 2;
  const bool same = q0 == q1;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nb; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = b0 + i;
    float c0, c1, c2, c3;
    if (BF16C) {
      const vu2 cb = __builtin_nontemporal_load(reinterpret_cast<const vu2*>(reinterpret_cast<const uint16_t*>(cptr) + 4 * b));
      c0 = bf2f((uint16_t)(cb.x & 0xFFFFu)); c1 = bf2f((uint16_t)(cb.x >> 16));
      c2 = bf2f((uint16_t)(cb.y & 0xFFFFu)); c3 = bf2f((uint16_t)(cb.y >> 16));
    } else {
      const vf4 cf = ld_nt(reinterpret_cast<const float*>(cptr) + 4 * b);
      c0 = cf.x; c1 = cf.y; c2 = cf.z; c3 = cf.w;
    }
    const float4 za = rng::gauss_block(seed, step, q0, (uint64_t)b);
    const float4 zb = same ? za : rng::gauss_block(seed, step, q1, (uint64_t)b);
    st4_bf16_nt(out + 4 * i, pert_one(c0, eps * za.x, s0), pert_one(c1, eps * za.y, s0), pert_one(c2, eps * za.z, s0),
                pert_one(c3, eps * za.w, s0));
    st4_bf16_nt(out + n + 4 * i, pert_one(c0, eps * zb.x, s1), pert_one(c1, eps * zb.y, s1),
                pert_one(c2, eps * zb.z, s1), pert_one(c3, eps * zb.w, s1));
  }
}

// The same for any range: one Philox block (4 arena indices) per thread and half, element
// by element.
template <bool BF16C>
__global__ void __launch_bounds__(256) perturb_kernel(const void* __restrict__ cptr, int64_t e0, int64_t n,
                                                      uint64_t seed, uint32_t step, uint32_t q0, uint32_t q1,
                                                      int32_t s0, int32_t s1, float eps, uint16_t* __restrict__ out) {
#pragma clang fp contract(off)
  const int64_t b0 = e0 >> 2, b1 = (e0 + n - 1) >> 2;
  const bool same = q0 == q1;
  for (int64_t b = b0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b <= b1; b += (int64_t)gridDim.x * blockDim.x) {
    const float4 za = rng::gauss_block(seed, step, q0, (uint64_t)b);
    const float4 zb = same ? za : rng::gauss_block(seed, step, q1, (uint64_t)b);
#pragma unroll
    for (int l = 0; l < 4; ++l) {
      const int64_t e = 4 * b + l;
      if (e < e0 || e >= e0 + n) continue;
      const float c = BF16C ? bf2f(reinterpret_cast<const uint16_t*>(cptr)[e]) : reinterpret_cast<const float*>(cptr)[e];
      const float ea = eps * rng::lane_of(za, l), eb = eps * rng::lane_of(zb, l);
      out[e - e0] = f2bf(s0 > 0 ? c + ea : (s0 < 0 ? c - ea : c));
      out[n + e - e0] = f2bf(s1 > 0 ? c + eb : (s1 < 0 ? c - eb : c));
    }
  }
}

// One-sided multi-query estimate of Algorithm 2: gh = (sum_j a_j Z^(j)) / q with
// a_j = (L_j - L_0) / eps, accumulated in fp32 with j ascending; then Adam (ADAM) or
// SGD on gh.  Returns false (no update anywhere) when some a_j is not finite.
__device__ __forceinline__ bool query_coeffs_finite(const float* losses, int q, float eps) {
#pragma clang fp contract(off)
  const float l0 = losses[0];
  for (int j = 1; j <= q; ++j)
    if (!__builtin_isfinite((losses[j] - l0) / eps)) return false;
  return true;
}

template <bool BF16C, bool ADAM>
__global__ void __launch_bounds__(256) step_q_kernel(void* __restrict__ cptr, float* __restrict__ mptr,
                                                     float* __restrict__ vptr, int64_t k, const float* losses, int q,
                                                     uint64_t seed, uint32_t step, float eps, AdamConst h, float lr,
                                                     uint32_t* status) {
#pragma clang fp contract(off)
  if (!query_coeffs_finite(losses, q, eps)) {
    if (status != nullptr && blockIdx.x == 0 && threadIdx.x == 0) atomicOr(status, 1u);
    return;
  }
  const float l0 = losses[0];
  const float qf = (float)q;
  const int64_t nb = (k + 3) >> 2;
  for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nb; b += (int64_t)gridDim.x * blockDim.x) {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int j = 1; j <= q; ++j) {
      const float aj = (losses[j] - l0) / eps;
      const float4 z = rng::gauss_block(seed, step, (uint32_t)j, (uint64_t)b);
      acc[0] = acc[0] + aj * z.x;
      acc[1] = acc[1] + aj * z.y;
      acc[2] = acc[2] + aj * z.z;
      acc[3] = acc[3] + aj * z.w;
    }
    const int64_t e = 4 * b;
    if (e + 4 <= k) {
      float cv[4], mv[4] = {0.f, 0.f, 0.f, 0.f}, vv[4] = {0.f, 0.f, 0.f, 0.f};
      if (BF16C) {
        const vu2 cb = __builtin_nontemporal_load(reinterpret_cast<const vu2*>(reinterpret_cast<const uint16_t*>(cptr) + e));
        cv[0] = bf2f((uint16_t)(cb.x & 0xFFFFu)); cv[1] = bf2f((uint16_t)(cb.x >> 16));
        cv[2] = bf2f((uint16_t)(cb.y & 0xFFFFu)); cv[3] = bf2f((uint16_t)(cb.y >> 16));
      } else {
        const vf4 cf = ld_nt(reinterpret_cast<const float*>(cptr) + e);
        cv[0] = cf.x; cv[1] = cf.y; cv[2] = cf.z; cv[3] = cf.w;
      }
      if (ADAM) {
        const vf4 m4 = ld_nt(mptr + e), v4 = ld_nt(vptr + e);
        mv[0] = m4.x; mv[1] = m4.y; mv[2] = m4.z; mv[3] = m4.w;
        vv[0] = v4.x; vv[1] = v4.y; vv[2] = v4.z; vv[3] = v4.w;
      }
#pragma unroll
      for (int l = 0; l < 4; ++l) {
        const float gh = acc[l] / qf;
        cv[l] = ADAM ? adam_one(cv[l], mv[l], vv[l], gh, h) : cv[l] - lr * gh;
      }
      if (ADAM) {
        st_nt(mptr + e, vf4{mv[0], mv[1], mv[2], mv[3]});
        st_nt(vptr + e, vf4{vv[0], vv[1], vv[2], vv[3]});
      }
      if (BF16C) {
        const vu2 cb = {(uint32_t)f2bf(cv[0]) | ((uint32_t)f2bf(cv[1]) << 16),
                        (uint32_t)f2bf(cv[2]) | ((uint32_t)f2bf(cv[3]) << 16)};
        __builtin_nontemporal_store(cb, reinterpret_cast<vu2*>(reinterpret_cast<uint16_t*>(cptr) + e));
      } else {
        st_nt(reinterpret_cast<float*>(cptr) + e, vf4{cv[0], cv[1], cv[2], cv[3]});
      }
    } else {
      for (int l = 0; l < 4 && e + l < k; ++l) {
        const float gh = acc[l] / qf;
        float c = BF16C ? bf2f(reinterpret_cast<const uint16_t*>(cptr)[e + l]) : reinterpret_cast<const float*>(cptr)[e + l];
        if (ADAM) {
          float m = mptr[e + l], v = vptr[e + l];
          c = adam_one(c, m, v, gh, h);
          mptr[e + l] = m;
          vptr[e + l] = v;
        } else {
          c = c - lr * gh;
        }
        if (BF16C) reinterpret_cast<uint16_t*>(cptr)[e + l] = f2bf(c);
        else reinterpret_cast<float*>(cptr)[e + l] = c;
      }
    }
  }
}

int64_t grid_for(int64_t blocks_of_four) {
  int64_t g = (blocks_of_four + 255) / 256;
  return g < 1 ? 1 : (g > (1 << 20) ? (1 << 20) : g);
}

}  // namespace

hipError_t launch_gen_z(uint64_t seed, uint32_t step, uint32_t query, int64_t e0, int64_t n, float* out,
                        hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nb = ((e0 + n - 1) >> 2) - (e0 >> 2) + 1;
  gen_z_kernel<<<dim3((unsigned)grid_for(nb)), dim3(256), 0, s>>>(seed, step, query, e0, n, out);
  return hipGetLastError();
}

hipError_t launch_perturb(const zoact_arena& A, int64_t e0, int64_t n, const zoact_pert_pair& p, uint16_t* out,
                          hipStream_t s) {
  const int64_t nb = ((e0 + n - 1) >> 2) - (e0 >> 2) + 1;
  const dim3 grid((unsigned)grid_for(nb));
  if ((e0 & 3) == 0 && (n & 3) == 0 && (reinterpret_cast<uintptr_t>(A.c) & 15u) == 0) {
    if (A.c_dtype == ZOACT_BF16)
      perturb_vec_kernel<true><<<grid, dim3(256), 0, s>>>(A.c, e0, n, p.seed, p.step, p.query[0], p.query[1],
                                                          p.sign[0], p.sign[1], p.eps, out);
    else
      perturb_vec_kernel<false><<<grid, dim3(256), 0, s>>>(A.c, e0, n, p.seed, p.step, p.query[0], p.query[1],
                                                           p.sign[0], p.sign[1], p.eps, out);
    return hipGetLastError();
  }
  if (A.c_dtype == ZOACT_BF16)
    perturb_kernel<true><<<grid, dim3(256), 0, s>>>(A.c, e0, n, p.seed, p.step, p.query[0], p.query[1], p.sign[0],
                                                    p.sign[1], p.eps, out);
  else
    perturb_kernel<false><<<grid, dim3(256), 0, s>>>(A.c, e0, n, p.seed, p.step, p.query[0], p.query[1], p.sign[0],
                                                     p.sign[1], p.eps, out);
  return hipGetLastError();
}

hipError_t launch_step_q(const zoact_arena& A, const float* losses, int32_t q, uint64_t seed, uint32_t step, float eps,
                         const zoact_adam* h, float lr, uint32_t* status, hipStream_t s) {
  if (A.k == 0) return hipSuccess;
  AdamConst c{};
  if (h) c = AdamConst{h->beta1, h->beta2, h->eps, h->weight_decay, h->step_size, h->inv_sqrt_bc2, h->one_minus_beta1,
                       h->one_minus_beta2};
  const dim3 grid((unsigned)grid_for((A.k + 3) >> 2));
  const bool bf = A.c_dtype == ZOACT_BF16;
#define ZO_Q(BF, AD) step_q_kernel<BF, AD><<<grid, dim3(256), 0, s>>>(A.c, A.m, A.v, A.k, losses, q, seed, step, eps, c, lr, status)
  if (h) {
    if (bf) ZO_Q(true, true); else ZO_Q(false, true);
  } else {
    if (bf) ZO_Q(true, false); else ZO_Q(false, false);
  }
#undef ZO_Q
  return hipGetLastError();
}

hipError_t launch_adam(const zoact_arena& A, const float* loss_pm, const zoact_pert& p, const zoact_adam& h,
                       uint32_t* status, const zoact_pert_pair* next, uint16_t* out, hipStream_t s) {
  if (A.k == 0) return hipSuccess;
  const AdamConst c{h.beta1, h.beta2, h.eps, h.weight_decay, h.step_size, h.inv_sqrt_bc2, h.one_minus_beta1,
                    h.one_minus_beta2};
  const dim3 grid((unsigned)grid_for((A.k + 3) >> 2));
  const zoact_pert_pair nx = next ? *next : zoact_pert_pair{};
#define ZO_ADAM(BF, NX)                                                                                             \
  adam_kernel<BF, NX><<<grid, dim3(256), 0, s>>>(A.c, A.m, A.v, A.k, loss_pm, p.seed, p.step, p.query, p.eps, c, \
                                                 status, nx, out)
  const bool bf = A.c_dtype == ZOACT_BF16;
  if (next && (A.k & 3) == 0 && next->query[0] == next->query[1] && next->sign[0] == 1 && next->sign[1] == -1) {
    if (bf)
      adam_next_pm_kernel<true><<<grid, dim3(256), 0, s>>>(A.c, A.m, A.v, A.k, loss_pm, p.seed, p.step, p.query, p.eps,
                                                            c, status, next->seed, next->step, next->query[0],
                                                            next->eps, out);
    else
      adam_next_pm_kernel<false><<<grid, dim3(256), 0, s>>>(A.c, A.m, A.v, A.k, loss_pm, p.seed, p.step, p.query,
                                                             p.eps, c, status, next->seed, next->step, next->query[0],
                                                             next->eps, out);
    return hipGetLastError();
  }
  if (next) {
    if (bf) ZO_ADAM(true, true); else ZO_ADAM(false, true);
  } else {
    if (bf) ZO_ADAM(true, false); else ZO_ADAM(false, false);
  }
#undef ZO_ADAM
  return hipGetLastError();
}

hipError_t launch_sgd(const zoact_arena& A, const float* loss_pm, const zoact_pert& p, float lr, uint32_t* status,
                      hipStream_t s) {
  if (A.k == 0) return hipSuccess;
  const dim3 grid((unsigned)grid_for((A.k + 3) >> 2));
  if (A.c_dtype == ZOACT_BF16)
    sgd_kernel<true><<<grid, dim3(256), 0, s>>>(A.c, A.k, loss_pm, p.seed, p.step, p.query, p.eps, lr, status);
  else
    sgd_kernel<false><<<grid, dim3(256), 0, s>>>(A.c, A.k, loss_pm, p.seed, p.step, p.query, p.eps, lr, status);
  return hipGetLastError();
}

}  // namespace zoact

// Shared device/host helpers of the ZO-Act HIP library (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "zoact.h"

namespace zoact {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// bf16 <-> fp32.  The conversion to bf16 is the hardware round-to-nearest-even.
__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

// Internal launchers return hipError_t from hipGetLastError() after the launch.
// Compute units of the current device (cached per device); -1 on error.
int cu_count();

hipError_t launch_perturb(const zoact_arena& A, int64_t e0, int64_t n, const zoact_pert_pair& p, uint16_t* out,
                          hipStream_t s);
hipError_t launch_gen_z(uint64_t seed, uint32_t step, uint32_t query, int64_t e0, int64_t n, float* out,
                        hipStream_t s);
hipError_t launch_adam(const zoact_arena& A, const float* loss_pm, const zoact_pert& p, const zoact_adam& h,
                       uint32_t* status, const zoact_pert_pair* next, uint16_t* out, hipStream_t s);
hipError_t launch_sgd(const zoact_arena& A, const float* loss_pm, const zoact_pert& p, float lr,
                      uint32_t* status, hipStream_t s);
// one-sided multi-query update: Adam when h != nullptr, else SGD with rate lr
hipError_t launch_step_q(const zoact_arena& A, const float* losses, int32_t q, uint64_t seed, uint32_t step, float eps,
                         const zoact_adam* h, float lr, uint32_t* status, hipStream_t s);
hipError_t launch_dequant_int4(const void* w, const void* scales, int64_t d_out, int64_t d_in, void* out,
                               hipStream_t s);
size_t project_ws_bytes(int64_t n_tok, int64_t d_in, int32_t r);
hipError_t launch_project_split(const void* x, int64_t n_tok, int64_t d_in, const void* ut, int32_t r, void* p,
                                void* ws, hipStream_t s);
hipError_t launch_project(const void* x, int32_t dtype, int64_t n_tok, int64_t d_in, const void* ut, int32_t r,
                          void* p, hipStream_t s);
// Norm (RMSNorm, or LayerNorm with bias b) of n_tok rows and the projection of its output,
// P = y U (bf16); hipErrorNotSupported outside the fused kernel's shapes.
hipError_t launch_norm_project(bool layernorm, const void* x, const void* w, const void* b, int64_t n_tok, int64_t d,
                               float eps, const void* ut, int r, void* y, void* p, hipStream_t s);
hipError_t launch_linear_pm(const zoact_linear& L, const zoact_arena* A, const void* x, int32_t x_dtype, int64_t T,
                            const void* p, const void* residual, uint32_t flags, const zoact_pert_pair& pert,
                            void* y, int32_t y_dtype, hipStream_t s);
// Adapted linear of both halves with the regression loss fused into the epilogue (y not
// stored): per-tile sums into part [2][tiles], then loss_pm[h] = sum / (T * d_out).
// y [2 T][N] fp32 = x [2 T][K] w^T, bf16 operands with dense rows (plain GEMM, no correction).
hipError_t launch_gemm_nt_f32(const uint16_t* x, int64_t T, const uint16_t* w, int64_t N, int64_t K, float* y,
                              hipStream_t s);
hipError_t launch_linear_mse(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T, uint32_t flags, const void* p,
                             const zoact_pert_pair& pert, const void* target, double* part, float* loss_pm,
                             hipStream_t s);
// The same with the partial sums in the library's static device scratch (no workspace).
hipError_t launch_linear_mse_noalloc(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T,
                                     uint32_t flags, const void* p, const zoact_pert_pair& pert, const void* target,
                                     float* loss_pm, hipStream_t s);
hipError_t launch_sum_mean(const double* part, int64_t n, double count, float* loss_pm, hipStream_t s);
// LM head of both halves with the next-token cross entropy fused into its epilogue (logits
// not stored); ws holds the per-row block partials, target logits and loss partials.
hipError_t launch_linear_xent(const zoact_linear& L, const zoact_arena* A, const void* x, int64_t T, const void* p,
                              const zoact_pert_pair& pert, const int32_t* tokens, int64_t S, float* loss_pm, void* ws,
                              hipStream_t s);
size_t linear_xent_ws_bytes(int64_t T, int64_t d_out);
hipError_t launch_xent_combine(const float2* xpart, const float* xtgt, int64_t T, int64_t S, int nblk, int64_t B,
                               double* part, float* loss_pm, hipStream_t s);
hipError_t launch_mse_pm(const void* y, int32_t dtype, const void* target, int64_t T, int64_t N, float* loss_pm,
                         void* ws, hipStream_t s);
hipError_t launch_xent_pm(const float* logits, const int32_t* tokens, int64_t B, int64_t S, int64_t V,
                          float* loss_pm, void* ws, hipStream_t s);
hipError_t launch_gram(const void* x, int32_t dtype, int64_t n_tok, int64_t d, int64_t ld, float* g, int accumulate,
                       hipStream_t s);
// `o` with every default resolved; `met` = false when tol > 0 and the final residual is above it.
hipError_t launch_basis_from_gram(const float* g, int64_t d, int32_t r, int32_t p, const zoact_eig_opts& o, void* ut,
                                  int32_t ut_dtype, float* ut_master, float* eigvals, zoact_eig_report* report, void* ws,
                                  hipStream_t s, bool& met);
size_t basis_ws_bytes(int64_t d, int32_t r, int32_t p);
// Algorithm 1 from the token-side Gram X X^T of bf16 X [n][ld] (D values per row,
// D % 64 == 0, r + p <= n): same outputs as the Gram form; ws of basis_rows_ws_bytes.
size_t basis_rows_ws_bytes(int64_t n, int64_t D, int32_t r, int32_t p);
hipError_t launch_basis_init_rows(const uint16_t* x, int64_t n, int64_t D, int64_t ld, int32_t r, int32_t p,
                                  const zoact_eig_opts& o, void* ut, int32_t ut_dtype, float* ut_master, float* eigvals,
                                  zoact_eig_report* report, void* ws, hipStream_t s, bool& met);

// Record the detail text of a failed call for zoact_last_error() and return `st`.
zoact_status set_error(zoact_status st, const char* msg);

// Deterministic two-stage reductions: partial sums per block, then one block sums them in order.
constexpr int kLossBlocks = 1024;

}  // namespace zoact

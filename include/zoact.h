/*
 * zoact.h -- C ABI of the ZO-Act forward-only step on MI355X (gfx950).
 *
 * ZO-Act (arXiv 2607.01125) fine-tunes a frozen model by adapting each linear
 * layer as W_eff = W + V_r B (Section 3): W and the activation basis V_r are
 * frozen, only the small coefficient matrix B is trained, and B is updated from
 * forward-only loss evaluations under Gaussian perturbations Z of B
 * (Algorithm 2), with an optimiser such as Adam.  V_r is computed once from a
 * calibration batch (Algorithm 1).
 *
 * Library orientation (PyTorch style): x [T][d_in] row-major, W [d_out][d_in],
 * the basis is stored transposed as U^T [r][d_in] (U = V_r), the coefficients
 * as C = B^T [d_out][r], so an adapted layer computes
 *     y = x W^T + b + (x U) C^T.
 * The step evaluates it twice on stacked halves of the batch, with C + eps Z
 * (half 0, "+") and C - eps Z (half 1, "-"), and then applies ZO-Adam with
 * g = (L+ - L-) / (2 eps).
 *
 * Conventions shared by every call:
 *  - Pointers are DEVICE pointers unless a comment says "host".  The caller owns
 *    every buffer; the library allocates and frees no memory on these paths and
 *    keeps no pointer after the call returns.  Buffers must stay valid until the
 *    stream reaches the enqueued work.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Every call only
 *    enqueues work on it and returns; none synchronises unless stated.
 *  - All shape, dtype and alignment checks run on the host before anything is
 *    enqueued; a failed check returns ZOACT_E_INVALID (or ZOACT_E_UNSUPPORTED)
 *    with no side effects.  A HIP launch error returns ZOACT_E_HIP.  The detail
 *    text of the last error on the calling thread is in zoact_last_error().
 *  - Device pointers must be 16-byte aligned; row lengths (d_in, d_out, r of
 *    bf16 tensors) must keep rows 16-byte aligned where stated.
 *  - bf16 values are stored as 16-bit patterns (uint16_t); conversions to bf16
 *    round to nearest, ties to even.
 *  - The arena: all coefficient matrices of a model live in one flat array of
 *    k = sum_l r * n_l entries (the paper's beta in R^k, Section 4).  A layer
 *    whose C starts at arena index `coef_offset` keeps C[n][i] at index
 *    coef_offset + n * r + i.  Z at arena index e for (seed, step, query) is a
 *    pure function of those four values and is never stored.
 *  - No C++ exception crosses this boundary.  The library is thread-safe; its
 *    only global state is the per-thread error text, and per GPU the static scratch
 *    array of zoact_linear_mse_pair_noalloc (and its cached device address).
 */
#ifndef ZOACT_H
#define ZOACT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t zoact_status;
enum {
  ZOACT_OK = 0,
  ZOACT_E_INVALID = 1,     /* bad argument, shape, dtype or alignment          */
  ZOACT_E_UNSUPPORTED = 2, /* valid request this build does not implement      */
  ZOACT_E_HIP = 3,         /* HIP runtime / launch failure                     */
  ZOACT_E_NOCONVERGE = 4,  /* eigensolver tolerance not met (result written)   */
  ZOACT_E_WORKSPACE = 5    /* workspace missing or too small                   */
};

/* Element types. */
enum { ZOACT_F32 = 0, ZOACT_BF16 = 1, ZOACT_INT4_G128 = 2 };

/* Flags of zoact_linear_fwd_pm. */
enum {
  ZOACT_EPI_NONE = 0,
  ZOACT_EPI_SWIGLU = 1u << 0, /* rows of W interleave gate/up in blocks of 16:
                                 fused rows 32j..32j+15 are gate features
                                 16j..16j+15 and rows 32j+16..32j+31 the matching
                                 up features; output y[t][f] = silu(gate)*up,
                                 width d_out/2                                    */
  ZOACT_EPI_RELU = 1u << 1,   /* y = max(0, .) before the store                   */
  ZOACT_SHARED_X = 1u << 2    /* both halves read the same input: x [T][d_in] and
                                 p [T][r] hold one copy; the base x W^T is formed
                                 once and each half adds its own rank-r correction
                                 to it (the same operations in the same order as
                                 with the input given twice, so the outputs are
                                 the same bits).  BF16 weights with L->ch (or
                                 r == 0), d_in % 64 == 0 and >= 128; not with
                                 ZOACT_EPI_SWIGLU.  Else ZOACT_E_UNSUPPORTED.      */
};

typedef void* zoact_stream; /* hipStream_t */

/* Perturbation of one evaluation: Z = Z(seed, step, query, arena index). */
typedef struct {
  uint64_t seed;
  uint32_t step;  /* optimiser step t (Algorithm 2's outer loop)          */
  uint32_t query; /* query index j (0 for the two-sided +/- pair)         */
  float eps;      /* perturbation scale (the paper's mu)                  */
} zoact_pert;

/* Perturbations of the two stacked halves of one evaluation, in general form: half h
 * evaluates C + sign[h] * eps * Z(seed, step, query[h]) with sign[h] in {-1, 0, +1}.
 * The two-sided pair is {query, query} with signs {+1, -1}; the one-sided multi-query
 * form of Algorithm 2 (Section 3's q-query average) evaluates the unperturbed model
 * (sign 0) and C + eps Z^(j) for queries j = 1..q, two per evaluation. */
typedef struct {
  uint64_t seed;
  uint32_t step;
  uint32_t query[2];
  int32_t sign[2];
  float eps;
} zoact_pert_pair;

/* One adapted (or plain, r = 0) linear layer. */
typedef struct {
  int32_t w_dtype;      /* ZOACT_F32, ZOACT_BF16 or ZOACT_INT4_G128               */
  const void* w;        /* F32/BF16: [d_out][d_in]; INT4: uint8 [d_out][d_in/2],
                           even column in the low nibble, two's complement,
                           values in [-7, 7]                                       */
  const void* w_scales; /* INT4: bf16 [d_out][d_in/128] (w = bf16(q * s)); else NULL */
  const void* bias;     /* [d_out] in the activation type, or NULL                 */
  const void* ut;       /* U^T [r][d_in] in the activation type; NULL iff r == 0   */
  int64_t d_in, d_out;
  int32_t r;            /* 0 <= r <= 256                                          */
  int64_t coef_offset;  /* arena index of C[0][0]                                 */
  const void* ch;       /* optional (BF16 activations): the perturbed coefficients
                           bf16(C +/- eps Z) of this layer from zoact_perturb_coeffs,
                           half 0 [d_out][r] at ch, half 1 at ch + ch_half_stride
                           elements; NULL = formed inside the kernel (same values).
                           r % 8 == 0: 16-byte aligned, stride a multiple of 8;
                           otherwise 2-byte alignment suffices                     */
  int64_t ch_half_stride;
  int64_t plain_begin;  /* output features [plain_begin, plain_end) are not adapted (a
                           projection fused with adapted ones, e.g. k inside q|k|v):
                           they get no correction and have no coefficient rows, so
                           feature n >= plain_end uses coefficient row
                           n - (plain_end - plain_begin).  Empty (equal) by default;
                           ignored when r == 0.  Non-empty needs BF16 activations,
                           BF16 weights (or INT4 with d_in % 128 == 0, d_in >= 256),
                           ch given, both bounds multiples of 256 and no
                           ZOACT_SHARED_X (else ZOACT_E_UNSUPPORTED or INVALID)       */
  int64_t plain_end;
  void* ws;             /* optional workspace (16-byte aligned) of ws_bytes >=
                           zoact_linear_workspace_bytes(): where the tiles leave a last
                           round of the persistent grid at most half full (for example
                           640 tiles on 256 compute units), BF16 plain or ReLU outputs
                           without ZOACT_SHARED_X, the depth of that round's tiles is
                           split over two workgroups and their halves summed (first +
                           second) before the epilogue: other summation order, same
                           bits in both halves of the pair.  NULL: not used.  Calls
                           that overlap on one workspace race.                        */
  size_t ws_bytes;
} zoact_linear;

/* The coefficient arena and its Adam moments (updated in place by zoact_step). */
typedef struct {
  int32_t c_dtype; /* ZOACT_F32 or ZOACT_BF16 */
  void* c;         /* [k] coefficients          */
  float* m;        /* [k] first moment, fp32    */
  float* v;        /* [k] second moment, fp32   */
  int64_t k;
} zoact_arena;

/* Host-computed Adam scalars for step t (float64 then one rounding to fp32):
   step_size = lr_t / (1 - beta1^t), inv_sqrt_bc2 = 1 / sqrt(1 - beta2^t),
   one_minus_beta1 = 1 - beta1, one_minus_beta2 = 1 - beta2. */
typedef struct {
  float beta1, beta2, eps, weight_decay;
  float step_size, inv_sqrt_bc2, one_minus_beta1, one_minus_beta2;
} zoact_adam;

/* Options of the eigensolver behind zoact_basis_from_gram (NULL = defaults; a field
   at 0 takes its default).  Fixed mode (adaptive == 0) runs max_iter subspace
   iterations and synchronises nothing unless tol > 0, in which case the call waits for
   the stream, reads the final residual and returns ZOACT_E_NOCONVERGE when it is above
   tol (the outputs are written all the same).  Adaptive mode (adaptive != 0, needs
   tol > 0) estimates the residual from the iteration's own products (one readback per
   check) after check_every and 2 check_every iterations, then at the iteration where the
   estimates' geometric rate predicts tol (at least check_every later; no further checks
   once that lies past max_iter or the estimate stops falling); it stops as soon as an
   estimate is at or below tol, then checks the exact residual and goes on iterating
   while that is above tol and iterations remain. */
typedef struct {
  int32_t oversample;  /* extra block columns p (default r)                     */
  int32_t max_iter;    /* subspace iterations, the most in adaptive mode (64)   */
  uint64_t seed;       /* seed of the random start block                        */
  float tol;           /* residual bound (0: none)                              */
  int32_t adaptive;    /* stop early once the residual is below tol             */
  int32_t check_every; /* iterations between adaptive checks (default 8)        */
} zoact_eig_opts;

/* Convergence report of one basis solve, written to device memory at the end of the
   call (in stream order).  resid = max_i ||G u_i - theta_i u_i|| / theta_1 of the
   returned basis (fp64 products); gap = theta_r / theta_{r+1}, the last kept over
   the first discarded Ritz value (1 means no gap: the top-r subspace is then not
   determined by G); iters = subspace iterations run; converged = resid <= tol, or 1
   when tol == 0. */
typedef struct {
  float resid;
  float gap;
  int32_t iters;
  int32_t converged;
} zoact_eig_report;

/* ------------------------------------------------------------------ info */
const char* zoact_version(void);
const char* zoact_status_str(zoact_status s);
/* Detail text of the last failed call on this thread ("" if none). */
const char* zoact_last_error(void);

/* ------------------------------------------------------ perturbation Z
 * Section 3: Z ~ N(0, I) in each layer's r x n coefficient space; Algorithm 2
 * draws a fresh Z per step and query.  Writes Z at arena indices e0 .. e0+n-1
 * to out[0 .. n-1] (fp32).  Generator: Philox4x32-10 with key = seed and counter
 * (lo32(e>>2), hi32(e>>2), step, query), lane e & 3, followed by Box-Muller in
 * quarter turns with series logarithm and sine/cosine (all fp32, no fused
 * multiply-add, correctly rounded division and square root).  The hot kernels
 * regenerate the same values internally; this entry point exists for testing.
 * Errors: n < 0, e0 < 0, out == NULL with n > 0 -> ZOACT_E_INVALID. */
zoact_status zoact_gen_z(uint64_t seed, uint32_t step, uint32_t query, int64_t e0, int64_t n,
                         float* out, zoact_stream stream);

/* ------------------------------------------------------ projection X U
 * The X V_r factor of the perturbed forward (Section 3, Y+ = XW + (X V_r)(B + mu Z)).
 * x [n_tok][d_in] and U^T [r][d_in] in dtype (F32 or BF16); p [n_tok][r] same
 * dtype, fp32 accumulation, one rounding on store.  1 <= r <= 256; d_in % 32 == 0
 * for BF16, x and ut 16-byte aligned.
 * ws (nullable, device): with BF16 and r <= 64, a workspace of at least
 * zoact_project_workspace_bytes(n_tok, d_in, r) bytes lets the depth be split over
 * workgroups as well (fewer U^T bytes per byte of x; fp32 partials, summed in a fixed
 * order by a second pass, so the same values on every run); calls that overlap on one
 * workspace race.  The split form is taken where it is the faster one (d_in > 4096 or
 * n_tok <= 4096); otherwise, with ws NULL or too small, the single-pass kernel (values
 * may differ from the split form in the last bit). */
size_t zoact_project_workspace_bytes(int64_t n_tok, int64_t d_in, int32_t r);
zoact_status zoact_project(const void* x, int32_t dtype, int64_t n_tok, int64_t d_in, const void* ut,
                           int32_t r, void* p, void* ws, size_t ws_bytes, zoact_stream stream);

/* The projection of a site whose input is a norm's output (the attention and MLP inputs
 * of a decoder layer), fused with that norm: y = RMSNorm(x) * w, or LayerNorm(x) * w + b,
 * over rows of d features (fp32 statistics, one rounding of y to bf16; eps as in the
 * norm), and p = y U (the X V_r factor of Section 3's perturbed forward) from the rounded
 * y, fp32 accumulation, one rounding.  x, y [rows][d], w, b [d], U^T [r][d], p [rows][r],
 * all bf16; the rows are read once.  The same values as the norm followed by zoact_project
 * up to the order of the fp32 sums.  Requirements: 16-byte aligned x, w, b, U^T, y;
 * d = 128, or d % 256 == 0 with d / 256 in {1, 2, 4, 8, 16, 20} (up to 5120); 1 <= r <= 128;
 * other shapes -> ZOACT_E_UNSUPPORTED (run the norm and zoact_project instead). */
zoact_status zoact_rmsnorm_project(const void* x, const void* w, int64_t rows, int64_t d, float eps, const void* ut,
                                   int32_t r, void* y, void* p, zoact_stream stream);
zoact_status zoact_layernorm_project(const void* x, const void* w, const void* b, int64_t rows, int64_t d, float eps,
                                     const void* ut, int32_t r, void* y, void* p, zoact_stream stream);

/* ------------------------------------------------------ fused +/- adapted linear
 * Section 3's perturbed forward evaluated for both signs in one pass over W:
 *   y[h] = epilogue(residual[h] + x[h] W^T + b + p[h] (C + s_h eps Z)^T),  s = (+1, -1)
 * x [2][T][d_in] and p [2][T][r] (from zoact_project on x; one copy of each,
 * [T][d_in] and [T][r], with ZOACT_SHARED_X) in the activation
 * dtype x_dtype (BF16 with BF16 or INT4 weights; F32 with F32 weights);
 * residual NULL or [2][T][d_out] in y's layout; y [2][T][d_out'] in y_dtype
 * (x_dtype, or F32 for logits), d_out' = d_out/2 with ZOACT_EPI_SWIGLU.
 * C is read from the arena at L->coef_offset (rows d_out, r per row) and
 * C +/- eps Z is formed in fp32 inside the kernel (rounded to bf16 for the
 * bf16 path); pert->eps == 0 gives two unperturbed halves.  With r == 0 the call
 * is a plain GEMM (arena and p may be NULL).  One rounding per output element.
 * Requirements: T >= 1; d_in % 64 == 0 (BF16/INT4) or % 4 (F32); INT4 needs
 * d_in % 128 == 0; d_out % 32 == 0 with SWIGLU (% 16 otherwise, BF16).
 * Errors: ZOACT_E_INVALID on shape/dtype mismatch, ZOACT_E_UNSUPPORTED for a
 * dtype combination not listed here. */
zoact_status zoact_linear_fwd_pm(const zoact_linear* L, const zoact_arena* A, const void* x,
                                 int32_t x_dtype, int64_t T, const void* p, const void* residual,
                                 uint32_t flags, const zoact_pert* pert, void* y, int32_t y_dtype,
                                 zoact_stream stream);
/* The same contraction with the general pair: half h uses C + pp->sign[h] eps
 * Z(pp->seed, pp->step, pp->query[h]).  zoact_linear_fwd_pm(pert) is this call with
 * {pert->query, pert->query} and signs {+1, -1}.  A precomputed L->ch must hold the
 * same pair (zoact_perturb_coeffs_pair with *pp). */
zoact_status zoact_linear_fwd_pair(const zoact_linear* L, const zoact_arena* A, const void* x,
                                   int32_t x_dtype, int64_t T, const void* p, const void* residual,
                                   uint32_t flags, const zoact_pert_pair* pp, void* y, int32_t y_dtype,
                                   zoact_stream stream);

/* Bytes of the optional zoact_linear workspace on the current device (one 256 KB tile
 * slot per compute unit). */
size_t zoact_linear_workspace_bytes(void);

/* INT4 weights to bf16: out[n][k] = bf16(q[n][k] * s[n][k / 128]), the dequantised weight
 * the INT4 GEMM forms in registers (same packing as zoact_linear.w).  At large token counts
 * a caller dequantises each INT4 layer once per forward into a bf16 buffer of its own and
 * runs the bf16 schedule on it: the in-register path converts every weight once per
 * 256-token tile.  w and out 16-byte aligned, out bf16 [d_out][d_in]; d_in % 128 == 0. */
zoact_status zoact_dequant_int4(const void* w, const void* w_scales, int64_t d_out, int64_t d_in, void* out,
                                zoact_stream stream);

/* ------------------------------------------------------ perturbed coefficients
 * out[h][e - e0] = bf16(fp32(C[e]) + s_h fp32(eps Z(e))), s = (+1, -1), for arena
 * indices e0 <= e < e0 + n: the C +/- eps Z of Section 3's perturbed forward, exactly
 * as the fused GEMM forms it.  Computing it once per step for a whole model (one
 * streaming pass over the arena) lets every GEMM workgroup read it instead of
 * regenerating Z; pass a layer's slice as zoact_linear.ch with ch_half_stride = n.
 * out bf16 [2][n], 16-byte aligned.  Errors: range outside the arena, n < 1. */
zoact_status zoact_perturb_coeffs(const zoact_arena* A, int64_t e0, int64_t n, const zoact_pert* pert, void* out,
                                  zoact_stream stream);
/* The general pair: out[h][e - e0] = bf16(fp32(C[e]) + sign[h] fp32(eps Z(e; query[h])))
 * (sign 0: bf16(C[e])). */
zoact_status zoact_perturb_coeffs_pair(const zoact_arena* A, int64_t e0, int64_t n, const zoact_pert_pair* pp,
                                       void* out, zoact_stream stream);

/* ------------------------------------------------------ losses of both halves
 * Algorithm 2 needs the loss under each perturbation; the two-sided step needs
 * L+ and L- (loss_pm[0], loss_pm[1], fp32, device).  Reductions are
 * deterministic (fixed order, no atomics) and use `ws` (>= zoact_loss_workspace_bytes()).
 * zoact_mse_pm: mean over T*N of (y[h] - target)^2; y [2][T][N], target [T][N], same dtype.
 * zoact_xent_pm: next-token cross entropy, mean over B*(S-1) positions of
 *   -log softmax(logits[h][b][s])[tokens[b][s+1]]; logits fp32 [2][B][S][V],
 *   tokens int32 [B][S] (host-validated range is the caller's duty; ids outside
 *   [0, V) are clamped). */
size_t zoact_loss_workspace_bytes(void);
/* Fused form of the single-layer regression loss: the adapted linear of both halves
 * (as zoact_linear_fwd_pair computes it, bias included, no residual or activation)
 * followed by loss_pm[h] = mean over T x d_out of (bf16(y[h]) - target)^2, without
 * storing y.  The sum of squares runs in the GEMM's epilogue (fp32 per lane, fp64
 * per wave: four partial sums per 256 x 256 tile) and a fixed-order fp64 sum over them;
 * it differs from zoact_linear_fwd_pair + zoact_mse_pm by summation order only.  BF16
 * activations, bf16 target [T][d_out] (16-byte aligned); BF16 or INT4 weights (INT4
 * with L->ch).  flags: 0, or ZOACT_SHARED_X when both halves' inputs are the same (x and p
 * then hold one copy, as in zoact_linear_fwd_pair).
 * ws: at least zoact_linear_mse_workspace_bytes(T, d_out) bytes (16-byte aligned).
 * Errors: shapes the fused kernel does not cover -> ZOACT_E_UNSUPPORTED. */
/* Fused LM head and next-token cross entropy: the linear of both halves (as
 * zoact_linear_fwd_pair computes it, logits in fp32, no residual or activation) followed by
 * zoact_xent_pm's loss, without storing the logits: the GEMM's epilogue keeps, per row and
 * 128-column block, the maximum and the sum of exp(logit - maximum) and the next token's
 * logit; a second pass merges the blocks per row (the online log-sum-exp rule) and sums
 * the rows in a fixed order.  x [2][B*S][d_in] bf16, tokens int32 [B][S] shared by both
 * halves (ids clamped to [0, d_out)), S >= 2.  BF16 activations and weights.
 * ws: zoact_linear_xent_workspace_bytes(B*S, d_out) bytes, 16-byte aligned.
 * Errors: shapes the fused kernel does not cover -> ZOACT_E_UNSUPPORTED. */
size_t zoact_linear_xent_workspace_bytes(int64_t T, int64_t d_out);
zoact_status zoact_linear_xent_pair(const zoact_linear* L, const zoact_arena* A, const void* x, int64_t B, int64_t S,
                                    const void* p, const zoact_pert_pair* pp, const int32_t* tokens, float* loss_pm,
                                    void* ws, size_t ws_bytes, zoact_stream stream);
size_t zoact_linear_mse_workspace_bytes(int64_t T, int64_t d_out);
zoact_status zoact_linear_mse_pair(const zoact_linear* L, const zoact_arena* A, const void* x, int64_t T,
                                   uint32_t flags, const void* p, const zoact_pert_pair* pp, const void* target,
                                   float* loss_pm, void* ws, size_t ws_bytes, zoact_stream stream);
/* zoact_linear_mse_pair without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  The per-tile partial sums go to a static device array of the library,
 * ZOACT_MSE_SCRATCH_BYTES per GPU, held by each GPU the library runs on until the process
 * ends; the call itself allocates and frees nothing.  Same arguments, kernels and results
 * (bit for bit) as zoact_linear_mse_pair.  Every call on one GPU shares that GPU's array:
 * calls whose work overlaps on one GPU (different streams, or other threads) race on it
 * and must be ordered by the caller.  Errors: a shape needing more than the scratch,
 * zoact_linear_mse_workspace_bytes(T, d_out) > ZOACT_MSE_SCRATCH_BYTES (T = 8192 tokens
 * per half allow d_out up to 1,048,576) -> ZOACT_E_INVALID; the others as
 * zoact_linear_mse_pair. */
#define ZOACT_MSE_SCRATCH_BYTES (1u << 20)
zoact_status zoact_linear_mse_pair_noalloc(const zoact_linear* L, const zoact_arena* A, const void* x, int64_t T,
                                           uint32_t flags, const void* p, const zoact_pert_pair* pp,
                                           const void* target, float* loss_pm, zoact_stream stream);
zoact_status zoact_mse_pm(const void* y, int32_t dtype, const void* target, int64_t T, int64_t N,
                          float* loss_pm, void* ws, size_t ws_bytes, zoact_stream stream);
zoact_status zoact_xent_pm(const float* logits, const int32_t* tokens, int64_t B, int64_t S, int64_t V,
                           float* loss_pm, void* ws, size_t ws_bytes, zoact_stream stream);

/* ------------------------------------------------------ ZO-Adam step
 * Algorithm 2's update in two-sided form: g = (L+ - L-) / (2 eps) from
 * loss_pm (device, fp32 [2]); for every arena index e: gh = g * Z(e) (+ wd*c),
 * then Adam on (c, m, v) in place in fp32 in the order
 *   m = b1 m + (1-b1) gh; v = b2 v + (1-b2) gh^2; d = sqrt(v) inv_sqrt_bc2 + eps_A;
 *   c = c - step_size (m / d)
 * (C rounded to bf16 on store when A->c_dtype == BF16).  A non-finite g leaves
 * the arena unchanged and ORs bit 0 into *dev_status (device, nullable).
 * zoact_step_sgd: c = c - lr * (g * Z(e)) (the paper's SGD variant). */
zoact_status zoact_step(const zoact_arena* A, const float* loss_pm, const zoact_pert* pert,
                        const zoact_adam* h, uint32_t* dev_status, zoact_stream stream);
zoact_status zoact_step_sgd(const zoact_arena* A, const float* loss_pm, const zoact_pert* pert, float lr,
                            uint32_t* dev_status, zoact_stream stream);
/* zoact_step, then zoact_perturb_coeffs(A, 0, A->k, next, ch_next) for the next step, in
 * one pass over the arena: both results bit for bit as the two calls give them (the
 * perturbation is formed from C as stored, after the update; with a non-finite g C is
 * unchanged and the perturbation is still written).  Saves one launch and one read of C
 * per step when a layer's coefficients are the whole arena.  ch_next bf16 [2][A->k],
 * 16-byte aligned; A->k >= 1. */
zoact_status zoact_step_perturb(const zoact_arena* A, const float* loss_pm, const zoact_pert* pert,
                                const zoact_adam* h, uint32_t* dev_status, const zoact_pert* next, void* ch_next,
                                zoact_stream stream);

/* ------------------------------------------------------ one-sided multi-query step
 * Algorithm 2 with q queries (Section 3's averaged forward-difference estimate):
 * losses (device, fp32 [q + 1]) holds the unperturbed loss L at losses[0] and the
 * loss under C + eps Z^(j) at losses[j], Z^(j) = Z(seed, step, query j), j = 1..q.
 * Per query a_j = (L_j - L) / eps in fp32; per arena index e, in fp32 with one
 * rounding per operation and j ascending,
 *   acc = 0; acc = acc + a_j * Z^(j)(e) for j = 1..q;  gh = acc / q,
 * then the Adam update of zoact_step on gh (zoact_step_q) or c = c - lr * gh
 * (zoact_step_q_sgd).  1 <= q <= 256.  A non-finite a_j leaves the arena unchanged
 * and ORs bit 0 into *dev_status (device, nullable). */
zoact_status zoact_step_q(const zoact_arena* A, const float* losses, int32_t q, uint64_t seed, uint32_t step,
                          float eps, const zoact_adam* h, uint32_t* dev_status, zoact_stream stream);
zoact_status zoact_step_q_sgd(const zoact_arena* A, const float* losses, int32_t q, uint64_t seed, uint32_t step,
                              float eps, float lr, uint32_t* dev_status, zoact_stream stream);

/* ------------------------------------------------------ one-shot basis (Algorithm 1)
 * Top-r right singular vectors of the calibration activations X_l, i.e. the top-r
 * eigenvectors of the uncentred Gram X^T X, largest first, each column signed so
 * that its largest-magnitude entry is positive.
 * zoact_gram: g [d][d] fp32 (+)= X^T X for x [n_tok] rows of d values (F32 or BF16)
 *   with row stride ld_x >= d elements; `accumulate` != 0 adds to g (chunked
 *   calibration batches).  BF16 needs d % 64 == 0, ld_x % 8 == 0 and x 16-byte aligned.
 * zoact_basis_from_gram: top-r eigenpairs of g by randomised block subspace
 *   iteration (block r + oversample), Rayleigh-Ritz and a Jacobi eigensolver of
 *   the projected block; writes ut [r][d] in ut_dtype (F32/BF16), optional
 *   ut_master fp32 [r][d], eigvals fp32 [r] (descending) and the convergence report
 *   (device, nullable; see zoact_eig_report).  Iteration control and synchronisation:
 *   see zoact_eig_opts.  Workspace: ws of at least zoact_basis_workspace_bytes(d, r,
 *   opts) bytes.
 * zoact_basis_init: zoact_gram followed by zoact_basis_from_gram, with g at the
 *   start of ws; ws needs zoact_basis_init_workspace_bytes(d, r, opts) bytes (the
 *   Gram d*d fp32, padded to 256 bytes, then the solver's workspace).  With fewer
 *   rows than features (BF16 x, n_tok < d, r + p <= n_tok, d % 64 == 0, ld_x % 8 ==
 *   0, x 16-byte aligned) and ws also large enough for it, the same singular vectors
 *   come from the thin SVD's other side (Section 3): the solver runs on the
 *   n_tok x n_tok token Gram X X^T, whose eigenvectors are X's left singular vectors
 *   V', and the basis is X^T V' with unit columns (signed as above); the eigenvalues
 *   are the same, and the report's residual is still that of the returned basis
 *   against X^T X (formed as X^T (X X^T) V' over the column norms).  A column whose
 *   singular value is exactly 0 (X of rank below r) is returned as zeros in this form.
 * Errors: r < 1, r > 256, r + p > d, n_tok < r, ld_x < d, negative tol or
 * check_every, adaptive with tol == 0 -> ZOACT_E_INVALID; a workspace that is NULL or
 * too small -> ZOACT_E_WORKSPACE; residual above tol -> ZOACT_E_NOCONVERGE (outputs
 * written, report->converged = 0). */
size_t zoact_basis_workspace_bytes(int64_t d, int32_t r, const zoact_eig_opts* opts);
size_t zoact_basis_init_workspace_bytes(int64_t d, int32_t r, const zoact_eig_opts* opts);
zoact_status zoact_gram(const void* x, int32_t x_dtype, int64_t n_tok, int64_t d, int64_t ld_x, float* g,
                        int32_t accumulate, zoact_stream stream);
zoact_status zoact_basis_from_gram(const float* g, int64_t d, int32_t r, const zoact_eig_opts* opts,
                                   void* ut, int32_t ut_dtype, float* ut_master, float* eigvals,
                                   zoact_eig_report* report, void* ws, size_t ws_bytes, zoact_stream stream);
zoact_status zoact_basis_init(const void* x, int32_t x_dtype, int64_t n_tok, int64_t d, int64_t ld_x, int32_t r,
                              const zoact_eig_opts* opts, void* ut, int32_t ut_dtype, float* ut_master,
                              float* eigvals, zoact_eig_report* report, void* ws, size_t ws_bytes,
                              zoact_stream stream);

#ifdef __cplusplus
}
#endif
#endif /* ZOACT_H */

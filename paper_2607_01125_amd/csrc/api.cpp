// extern "C" boundary of the ZO-Act HIP library: host-side validation, then a
// launch on the caller's stream.  Every check runs before anything is enqueued.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>

#include "common.hpp"

namespace {

thread_local std::string g_last_error;

zoact_status fail(zoact_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

zoact_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ZOACT_OK;
  if (e == hipErrorNotSupported) return fail(ZOACT_E_UNSUPPORTED, "%s: unsupported configuration", what);
  return fail(ZOACT_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

hipStream_t st(zoact_stream s) { return reinterpret_cast<hipStream_t>(s); }

bool float_type(int32_t t) { return t == ZOACT_F32 || t == ZOACT_BF16; }

#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) return fail(ZOACT_E_INVALID, __VA_ARGS__); \
  } while (0)

}  // namespace

namespace zoact {
zoact_status set_error(zoact_status st, const char* msg) {
  g_last_error = msg;
  return st;
}
}  // namespace zoact

extern "C" {

const char* zoact_version(void) { return "zoact-gfx950 0.1.0"; }

const char* zoact_status_str(zoact_status s) {
  switch (s) {
    case ZOACT_OK: return "ok";
    case ZOACT_E_INVALID: return "invalid argument";
    case ZOACT_E_UNSUPPORTED: return "unsupported";
    case ZOACT_E_HIP: return "HIP error";
    case ZOACT_E_NOCONVERGE: return "eigensolver did not converge";
    case ZOACT_E_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

const char* zoact_last_error(void) { return g_last_error.c_str(); }

zoact_status zoact_gen_z(uint64_t seed, uint32_t step, uint32_t query, int64_t e0, int64_t n, float* out,
                         zoact_stream stream) {
  CHECK(n >= 0 && e0 >= 0, "gen_z: negative range (e0=%lld, n=%lld)", (long long)e0, (long long)n);
  CHECK(n == 0 || out != nullptr, "gen_z: out is NULL");
  CHECK(e0 <= INT64_MAX - n, "gen_z: range overflows");
  return hip_status(zoact::launch_gen_z(seed, step, query, e0, n, out, st(stream)), "gen_z");
}

size_t zoact_project_workspace_bytes(int64_t n_tok, int64_t d_in, int32_t r) {
  if (n_tok < 1 || d_in < 1 || r < 1) return 0;
  return zoact::project_ws_bytes(n_tok, d_in, r);
}

zoact_status zoact_project(const void* x, int32_t dtype, int64_t n_tok, int64_t d_in, const void* ut, int32_t r, void* p,
                           void* ws, size_t ws_bytes, zoact_stream stream) {
  CHECK(float_type(dtype), "project: dtype must be F32 or BF16");
  CHECK(n_tok >= 1 && d_in >= 1, "project: empty shape (n_tok=%lld, d_in=%lld)", (long long)n_tok, (long long)d_in);
  CHECK(r >= 1 && r <= 256, "project: r=%d outside [1, 256]", r);
  CHECK(x && ut && p, "project: NULL pointer");
  if (dtype == ZOACT_BF16) {
    CHECK(d_in % 32 == 0, "project: bf16 needs d_in %% 32 == 0 (d_in=%lld)", (long long)d_in);
    CHECK(aligned16(x) && aligned16(ut), "project: x and ut must be 16-byte aligned");
    // the depth-split form where it measured faster: deep inputs, or few tokens (at
    // 8192 x 4096 the single pass is level with it)
    if (ws && r <= 64 && ws_bytes >= zoact::project_ws_bytes(n_tok, d_in, r) && (d_in > 4096 || n_tok <= 4096)) {
      CHECK(aligned16(ws), "project: ws must be 16-byte aligned");
      return hip_status(zoact::launch_project_split(x, n_tok, d_in, ut, r, p, ws, st(stream)), "project");
    }
  }
  return hip_status(zoact::launch_project(x, dtype, n_tok, d_in, ut, r, p, st(stream)), "project");
}

size_t zoact_linear_workspace_bytes(void) {
  const int n = zoact::cu_count();
  return n > 0 ? (size_t)n * 256 * 1024 : 0;
}

zoact_status zoact_dequant_int4(const void* w, const void* w_scales, int64_t d_out, int64_t d_in, void* out,
                                zoact_stream stream) {
  CHECK(w && w_scales && out, "dequant_int4: NULL pointer");
  CHECK(d_out >= 1 && d_in >= 128 && d_in % 128 == 0, "dequant_int4: need d_out >= 1 and d_in %% 128 == 0");
  CHECK(aligned16(w) && aligned16(out), "dequant_int4: w and out must be 16-byte aligned");
  return hip_status(zoact::launch_dequant_int4(w, w_scales, d_out, d_in, out, st(stream)), "dequant_int4");
}

static zoact_status validate_linear(const zoact_linear* L, const zoact_arena* A, const void* x, int32_t x_dtype,
                                    int64_t T, const void* p, const void* residual, uint32_t flags,
                                    const zoact_pert_pair* pert, const void* y, int32_t y_dtype) {
  CHECK(L != nullptr && pert != nullptr, "linear_fwd_pm: NULL layer or perturbation");
  for (int h = 0; h < 2; ++h)
    CHECK(pert->sign[h] >= -1 && pert->sign[h] <= 1, "linear_fwd_pm: sign[%d]=%d outside {-1, 0, 1}", h, pert->sign[h]);
  CHECK(x && y && L->w, "linear_fwd_pm: NULL x, y or w");
  CHECK(T >= 1, "linear_fwd_pm: T=%lld < 1", (long long)T);
  CHECK(L->d_in >= 1 && L->d_out >= 1, "linear_fwd_pm: empty layer");
  CHECK(L->r >= 0 && L->r <= 256, "linear_fwd_pm: r=%d outside [0, 256]", L->r);
  CHECK((flags & ~(uint32_t)(ZOACT_EPI_SWIGLU | ZOACT_EPI_RELU | ZOACT_SHARED_X)) == 0,
        "linear_fwd_pm: unknown flags 0x%x", flags);
  CHECK(!(flags & ZOACT_SHARED_X) || x_dtype == ZOACT_BF16, "linear_fwd_pm: SHARED_X needs BF16 activations");
  CHECK(!((flags & ZOACT_EPI_SWIGLU) && (flags & ZOACT_EPI_RELU)), "linear_fwd_pm: SWIGLU and RELU are exclusive");
  CHECK(float_type(x_dtype) && float_type(y_dtype), "linear_fwd_pm: activation types must be F32 or BF16");
  int64_t rows = L->d_out;   // coefficient rows of the layer
  if (L->r > 0) {
    CHECK(A != nullptr && A->c != nullptr, "linear_fwd_pm: r > 0 needs an arena");
    CHECK(L->ut != nullptr && p != nullptr, "linear_fwd_pm: r > 0 needs ut and p");
    CHECK(L->plain_begin >= 0 && L->plain_begin <= L->plain_end && L->plain_end <= L->d_out,
          "linear_fwd_pm: plain range [%lld, %lld) outside [0, d_out]", (long long)L->plain_begin,
          (long long)L->plain_end);
    if (L->plain_end > L->plain_begin) {
      CHECK(L->plain_begin % 256 == 0 && L->plain_end % 256 == 0,
            "linear_fwd_pm: plain range bounds must be multiples of 256");
      CHECK(L->ch != nullptr && x_dtype == ZOACT_BF16 && (L->w_dtype == ZOACT_BF16 || L->w_dtype == ZOACT_INT4_G128) &&
                !(flags & ZOACT_SHARED_X),
            "linear_fwd_pm: a plain range needs BF16 activations, BF16 or INT4 weights, ch, and no SHARED_X");
      rows -= L->plain_end - L->plain_begin;
    }
    CHECK(L->coef_offset >= 0 && L->coef_offset + rows * (int64_t)L->r <= A->k,
          "linear_fwd_pm: coefficient block [%lld, %lld) outside the arena (k=%lld)", (long long)L->coef_offset,
          (long long)(L->coef_offset + rows * (int64_t)L->r), (long long)A->k);
    CHECK(float_type(A->c_dtype), "linear_fwd_pm: arena dtype must be F32 or BF16");
  }
  if (flags & ZOACT_EPI_SWIGLU) CHECK(L->d_out % 32 == 0, "linear_fwd_pm: SWIGLU needs d_out %% 32 == 0");
  CHECK(L->ws == nullptr || aligned16(L->ws), "linear_fwd_pm: ws must be 16-byte aligned");
  if (L->ch != nullptr) {
    CHECK(x_dtype == ZOACT_BF16 && L->r > 0, "linear_fwd_pm: precomputed coefficients need BF16 activations and r > 0");
    CHECK(L->ch_half_stride >= rows * (int64_t)L->r && (reinterpret_cast<uintptr_t>(L->ch) & 1) == 0,
          "linear_fwd_pm: ch must be 2-byte aligned with a half stride >= (coefficient rows) * r");
    if (L->r % 8 == 0)
      CHECK(aligned16(L->ch) && L->ch_half_stride % 8 == 0,
            "linear_fwd_pm: with r %% 8 == 0, ch must be 16-byte aligned with a half stride that is a multiple of 8");
  }
  if (x_dtype == ZOACT_F32) {
    CHECK(L->w_dtype == ZOACT_F32 && y_dtype == ZOACT_F32, "linear_fwd_pm: F32 activations need F32 weights and output");
    CHECK(L->r == 0 || A->c_dtype == ZOACT_F32, "linear_fwd_pm: F32 path needs an F32 arena");
  } else {
    CHECK(L->w_dtype == ZOACT_BF16 || L->w_dtype == ZOACT_INT4_G128,
          "linear_fwd_pm: BF16 activations need BF16 or INT4 weights");
    CHECK(L->d_in % 64 == 0, "linear_fwd_pm: d_in=%lld must be a multiple of 64", (long long)L->d_in);
    CHECK(L->d_out % 16 == 0, "linear_fwd_pm: d_out=%lld must be a multiple of 16", (long long)L->d_out);
    CHECK(aligned16(x) && aligned16(L->w) && aligned16(y), "linear_fwd_pm: x, w, y must be 16-byte aligned");
    CHECK(residual == nullptr || aligned16(residual), "linear_fwd_pm: residual must be 16-byte aligned");
    if (L->w_dtype == ZOACT_INT4_G128) {
      CHECK(L->d_in % 128 == 0, "linear_fwd_pm: INT4 needs d_in %% 128 == 0 (d_in=%lld)", (long long)L->d_in);
      CHECK(L->w_scales != nullptr, "linear_fwd_pm: INT4 needs w_scales");
    }
  }
  return ZOACT_OK;
}

static zoact_status norm_project(bool layernorm, const void* x, const void* w, const void* b, int64_t rows, int64_t d,
                                 float eps, const void* ut, int32_t r, void* y, void* p, zoact_stream stream) {
  const char* who = layernorm ? "layernorm_project" : "rmsnorm_project";
  CHECK(x && w && ut && y && p && (!layernorm || b), "%s: NULL pointer", who);
  CHECK(rows >= 1 && d >= 1 && rows <= 0x7FFFFFFF, "%s: bad shape (rows=%lld, d=%lld)", who, (long long)rows,
        (long long)d);
  CHECK(r >= 1 && r <= 256, "%s: r=%d outside [1, 256]", who, r);
  CHECK(aligned16(x) && aligned16(w) && aligned16(ut) && aligned16(y) && (!layernorm || aligned16(b)),
        "%s: x, w, b, ut and y must be 16-byte aligned", who);
  return hip_status(zoact::launch_norm_project(layernorm, x, w, b, rows, d, eps, ut, r, y, p, st(stream)), who);
}

zoact_status zoact_rmsnorm_project(const void* x, const void* w, int64_t rows, int64_t d, float eps, const void* ut,
                                   int32_t r, void* y, void* p, zoact_stream stream) {
  return norm_project(false, x, w, nullptr, rows, d, eps, ut, r, y, p, stream);
}

zoact_status zoact_layernorm_project(const void* x, const void* w, const void* b, int64_t rows, int64_t d, float eps,
                                     const void* ut, int32_t r, void* y, void* p, zoact_stream stream) {
  return norm_project(true, x, w, b, rows, d, eps, ut, r, y, p, stream);
}

zoact_status zoact_linear_fwd_pair(const zoact_linear* L, const zoact_arena* A, const void* x, int32_t x_dtype,
                                   int64_t T, const void* p, const void* residual, uint32_t flags,
                                   const zoact_pert_pair* pert, void* y, int32_t y_dtype, zoact_stream stream) {
  const zoact_status v = validate_linear(L, A, x, x_dtype, T, p, residual, flags, pert, y, y_dtype);
  if (v != ZOACT_OK) return v;
  return hip_status(zoact::launch_linear_pm(*L, A, x, x_dtype, T, p, residual, flags, *pert, y, y_dtype, st(stream)),
                    "linear_fwd_pm");
}

static zoact_pert_pair pm_pair(const zoact_pert& p) {
  zoact_pert_pair pp{};
  pp.seed = p.seed;
  pp.step = p.step;
  pp.query[0] = pp.query[1] = p.query;
  pp.sign[0] = 1;
  pp.sign[1] = -1;
  pp.eps = p.eps;
  return pp;
}

zoact_status zoact_linear_fwd_pm(const zoact_linear* L, const zoact_arena* A, const void* x, int32_t x_dtype, int64_t T,
                                 const void* p, const void* residual, uint32_t flags, const zoact_pert* pert, void* y,
                                 int32_t y_dtype, zoact_stream stream) {
  CHECK(pert != nullptr, "linear_fwd_pm: NULL perturbation");
  const zoact_pert_pair pp = pm_pair(*pert);
  return zoact_linear_fwd_pair(L, A, x, x_dtype, T, p, residual, flags, &pp, y, y_dtype, stream);
}

zoact_status zoact_perturb_coeffs_pair(const zoact_arena* A, int64_t e0, int64_t n, const zoact_pert_pair* pp,
                                       void* out, zoact_stream stream) {
  CHECK(A != nullptr && pp != nullptr && out != nullptr && A->c != nullptr, "perturb_coeffs: NULL argument");
  CHECK(float_type(A->c_dtype), "perturb_coeffs: arena dtype must be F32 or BF16");
  CHECK(n >= 1 && e0 >= 0 && e0 + n <= A->k, "perturb_coeffs: range [%lld, %lld) outside the arena (k=%lld)",
        (long long)e0, (long long)(e0 + n), (long long)A->k);
  CHECK(aligned16(out), "perturb_coeffs: out must be 16-byte aligned");
  for (int h = 0; h < 2; ++h)
    CHECK(pp->sign[h] >= -1 && pp->sign[h] <= 1, "perturb_coeffs: sign[%d]=%d outside {-1, 0, 1}", h, pp->sign[h]);
  return hip_status(zoact::launch_perturb(*A, e0, n, *pp, static_cast<uint16_t*>(out), st(stream)), "perturb_coeffs");
}

zoact_status zoact_perturb_coeffs(const zoact_arena* A, int64_t e0, int64_t n, const zoact_pert* pert, void* out,
                                  zoact_stream stream) {
  CHECK(pert != nullptr, "perturb_coeffs: NULL argument");
  const zoact_pert_pair pp = pm_pair(*pert);
  return zoact_perturb_coeffs_pair(A, e0, n, &pp, out, stream);
}

size_t zoact_loss_workspace_bytes(void) { return (size_t)2 * zoact::kLossBlocks * sizeof(double); }

zoact_status zoact_mse_pm(const void* y, int32_t dtype, const void* target, int64_t T, int64_t N, float* loss_pm,
                          void* ws, size_t ws_bytes, zoact_stream stream) {
  CHECK(float_type(dtype), "mse_pm: dtype must be F32 or BF16");
  CHECK(y && target && loss_pm, "mse_pm: NULL pointer");
  CHECK(T >= 1 && N >= 1, "mse_pm: empty shape");
  CHECK(aligned16(y) && aligned16(target), "mse_pm: y and target must be 16-byte aligned");
  if (ws == nullptr || ws_bytes < zoact_loss_workspace_bytes())
    return fail(ZOACT_E_WORKSPACE, "mse_pm: workspace needs %zu bytes", zoact_loss_workspace_bytes());
  return hip_status(zoact::launch_mse_pm(y, dtype, target, T, N, loss_pm, ws, st(stream)), "mse_pm");
}

size_t zoact_linear_xent_workspace_bytes(int64_t T, int64_t d_out) {
  if (T < 1 || d_out < 1) return 0;
  return zoact::linear_xent_ws_bytes(T, d_out);
}

zoact_status zoact_linear_xent_pair(const zoact_linear* L, const zoact_arena* A, const void* x, int64_t B, int64_t S,
                                    const void* p, const zoact_pert_pair* pp, const int32_t* tokens, float* loss_pm,
                                    void* ws, size_t ws_bytes, zoact_stream stream) {
  CHECK(tokens != nullptr && loss_pm != nullptr, "linear_xent: NULL tokens or loss");
  CHECK(B >= 1 && S >= 2, "linear_xent: need B >= 1 and S >= 2");
  CHECK(L != nullptr && L->w_dtype == ZOACT_BF16, "linear_xent: needs a BF16 layer");
  // the shared validation of the layer, with x standing in for the unused output
  const zoact_status v = validate_linear(L, A, x, ZOACT_BF16, B * S, p, nullptr, 0, pp, x, ZOACT_F32);
  if (v != ZOACT_OK) return v;
  const size_t need = zoact_linear_xent_workspace_bytes(B * S, L->d_out);
  if (ws == nullptr || ws_bytes < need || !aligned16(ws))
    return fail(ZOACT_E_WORKSPACE, "linear_xent: workspace needs %zu bytes, 16-byte aligned", need);
  return hip_status(zoact::launch_linear_xent(*L, A, x, B * S, p, *pp, tokens, S, loss_pm, ws, st(stream)),
                    "linear_xent");
}

size_t zoact_linear_mse_workspace_bytes(int64_t T, int64_t d_out) {
  if (T < 1 || d_out < 1) return 0;
  // one fp64 partial sum per 256 x 256 tile and wave (four per tile)
  return (size_t)2 * (size_t)((T + 255) / 256) * (size_t)((d_out + 255) / 256) * 4 * sizeof(double);
}

zoact_status zoact_linear_mse_pair(const zoact_linear* L, const zoact_arena* A, const void* x, int64_t T,
                                   uint32_t flags, const void* p, const zoact_pert_pair* pp, const void* target,
                                   float* loss_pm, void* ws, size_t ws_bytes, zoact_stream stream) {
  CHECK(target != nullptr && loss_pm != nullptr, "linear_mse: NULL target or loss");
  CHECK(L != nullptr && aligned16(target), "linear_mse: NULL layer or misaligned target");
  CHECK((flags & ~(uint32_t)ZOACT_SHARED_X) == 0, "linear_mse: flags 0x%x (only ZOACT_SHARED_X applies)", flags);
  // the shared validation of the layer, with y standing in for the unused output
  const zoact_status v = validate_linear(L, A, x, ZOACT_BF16, T, p, nullptr, flags, pp, target, ZOACT_BF16);
  if (v != ZOACT_OK) return v;
  const size_t need = zoact_linear_mse_workspace_bytes(T, L->d_out);
  if (ws == nullptr || ws_bytes < need || !aligned16(ws))
    return fail(ZOACT_E_WORKSPACE, "linear_mse: workspace needs %zu bytes, 16-byte aligned", need);
  return hip_status(zoact::launch_linear_mse(*L, A, x, T, flags, p, *pp, target, static_cast<double*>(ws), loss_pm,
                                             st(stream)),
                    "linear_mse");
}

zoact_status zoact_linear_mse_pair_noalloc(const zoact_linear* L, const zoact_arena* A, const void* x, int64_t T,
                                           uint32_t flags, const void* p, const zoact_pert_pair* pp,
                                           const void* target, float* loss_pm, zoact_stream stream) {
  CHECK(target != nullptr && loss_pm != nullptr, "linear_mse_noalloc: NULL target or loss");
  CHECK(L != nullptr && aligned16(target), "linear_mse_noalloc: NULL layer or misaligned target");
  CHECK((flags & ~(uint32_t)ZOACT_SHARED_X) == 0, "linear_mse_noalloc: flags 0x%x (only ZOACT_SHARED_X applies)",
        flags);
  const zoact_status v = validate_linear(L, A, x, ZOACT_BF16, T, p, nullptr, flags, pp, target, ZOACT_BF16);
  if (v != ZOACT_OK) return v;
  const size_t need = zoact_linear_mse_workspace_bytes(T, L->d_out);
  CHECK(need <= (size_t)ZOACT_MSE_SCRATCH_BYTES,
        "linear_mse_noalloc: T=%lld, d_out=%lld need %zu bytes of partial sums, more than the static scratch "
        "of %zu bytes (use zoact_linear_mse_pair with a workspace)",
        (long long)T, (long long)L->d_out, need, (size_t)ZOACT_MSE_SCRATCH_BYTES);
  return hip_status(zoact::launch_linear_mse_noalloc(*L, A, x, T, flags, p, *pp, target, loss_pm, st(stream)),
                    "linear_mse_noalloc");
}

zoact_status zoact_xent_pm(const float* logits, const int32_t* tokens, int64_t B, int64_t S, int64_t V, float* loss_pm,
                           void* ws, size_t ws_bytes, zoact_stream stream) {
  CHECK(logits && tokens && loss_pm, "xent_pm: NULL pointer");
  CHECK(B >= 1 && S >= 2 && V >= 1, "xent_pm: need B >= 1, S >= 2, V >= 1");
  if (ws == nullptr || ws_bytes < zoact_loss_workspace_bytes())
    return fail(ZOACT_E_WORKSPACE, "xent_pm: workspace needs %zu bytes", zoact_loss_workspace_bytes());
  return hip_status(zoact::launch_xent_pm(logits, tokens, B, S, V, loss_pm, ws, st(stream)), "xent_pm");
}

static zoact_status check_arena(const zoact_arena* A, const float* loss_pm, const zoact_pert* p, const char* who) {
  CHECK(A != nullptr && p != nullptr && loss_pm != nullptr, "%s: NULL arena, loss or perturbation", who);
  CHECK(A->k >= 0, "%s: negative arena size", who);
  CHECK(float_type(A->c_dtype), "%s: arena dtype must be F32 or BF16", who);
  CHECK(A->k == 0 || A->c != nullptr, "%s: NULL coefficients", who);
  CHECK(aligned16(A->c) && aligned16(A->m) && aligned16(A->v), "%s: arena buffers must be 16-byte aligned", who);
  return ZOACT_OK;
}

zoact_status zoact_step(const zoact_arena* A, const float* loss_pm, const zoact_pert* p, const zoact_adam* h,
                        uint32_t* dev_status, zoact_stream stream) {
  zoact_status s = check_arena(A, loss_pm, p, "step");
  if (s != ZOACT_OK) return s;
  CHECK(h != nullptr, "step: NULL Adam scalars");
  CHECK(A->k == 0 || (A->m != nullptr && A->v != nullptr), "step: NULL moments");
  return hip_status(zoact::launch_adam(*A, loss_pm, *p, *h, dev_status, nullptr, nullptr, st(stream)), "step");
}

zoact_status zoact_step_perturb(const zoact_arena* A, const float* loss_pm, const zoact_pert* p, const zoact_adam* h,
                                uint32_t* dev_status, const zoact_pert* next, void* ch_next, zoact_stream stream) {
  zoact_status s = check_arena(A, loss_pm, p, "step_perturb");
  if (s != ZOACT_OK) return s;
  CHECK(h != nullptr && next != nullptr && ch_next != nullptr, "step_perturb: NULL Adam scalars, next or ch_next");
  CHECK(A->k >= 1, "step_perturb: empty arena");
  CHECK(A->m != nullptr && A->v != nullptr, "step_perturb: NULL moments");
  CHECK(aligned16(ch_next), "step_perturb: ch_next must be 16-byte aligned");
  const zoact_pert_pair pp = pm_pair(*next);
  return hip_status(zoact::launch_adam(*A, loss_pm, *p, *h, dev_status, &pp, static_cast<uint16_t*>(ch_next),
                                       st(stream)),
                    "step_perturb");
}

zoact_status zoact_step_sgd(const zoact_arena* A, const float* loss_pm, const zoact_pert* p, float lr,
                            uint32_t* dev_status, zoact_stream stream) {
  CHECK(A != nullptr && p != nullptr && loss_pm != nullptr, "step_sgd: NULL arena, loss or perturbation");
  CHECK(A->k >= 0 && float_type(A->c_dtype), "step_sgd: bad arena");
  CHECK(A->k == 0 || A->c != nullptr, "step_sgd: NULL coefficients");
  return hip_status(zoact::launch_sgd(*A, loss_pm, *p, lr, dev_status, st(stream)), "step_sgd");
}

static zoact_status check_step_q(const zoact_arena* A, const float* losses, int32_t q, const char* who) {
  CHECK(A != nullptr && losses != nullptr, "%s: NULL arena or losses", who);
  CHECK(q >= 1 && q <= 256, "%s: q=%d outside [1, 256]", who, q);
  CHECK(A->k >= 0 && float_type(A->c_dtype), "%s: bad arena", who);
  CHECK(A->k == 0 || A->c != nullptr, "%s: NULL coefficients", who);
  CHECK(aligned16(A->c) && aligned16(A->m) && aligned16(A->v), "%s: arena buffers must be 16-byte aligned", who);
  return ZOACT_OK;
}

zoact_status zoact_step_q(const zoact_arena* A, const float* losses, int32_t q, uint64_t seed, uint32_t step,
                          float eps, const zoact_adam* h, uint32_t* dev_status, zoact_stream stream) {
  zoact_status s = check_step_q(A, losses, q, "step_q");
  if (s != ZOACT_OK) return s;
  CHECK(h != nullptr, "step_q: NULL Adam scalars");
  CHECK(A->k == 0 || (A->m != nullptr && A->v != nullptr), "step_q: NULL moments");
  return hip_status(zoact::launch_step_q(*A, losses, q, seed, step, eps, h, 0.f, dev_status, st(stream)), "step_q");
}

zoact_status zoact_step_q_sgd(const zoact_arena* A, const float* losses, int32_t q, uint64_t seed, uint32_t step,
                              float eps, float lr, uint32_t* dev_status, zoact_stream stream) {
  zoact_status s = check_step_q(A, losses, q, "step_q_sgd");
  if (s != ZOACT_OK) return s;
  return hip_status(zoact::launch_step_q(*A, losses, q, seed, step, eps, nullptr, lr, dev_status, st(stream)),
                    "step_q_sgd");
}

// Options with every default resolved (r is the basis rank).
static zoact_eig_opts eig_resolve(int32_t r, const zoact_eig_opts* o) {
  zoact_eig_opts e{};
  e.oversample = (o && o->oversample > 0) ? o->oversample : r;
  e.max_iter = (o && o->max_iter > 0) ? o->max_iter : 64;
  e.seed = o ? o->seed : 0x5eedULL;
  e.tol = o ? o->tol : 0.f;
  e.adaptive = o ? o->adaptive : 0;
  e.check_every = (o && o->check_every > 0) ? o->check_every : 8;
  return e;
}

size_t zoact_basis_workspace_bytes(int64_t d, int32_t r, const zoact_eig_opts* opts) {
  if (d < 1 || r < 1) return 0;
  return zoact::basis_ws_bytes(d, r, eig_resolve(r, opts).oversample);
}

// Gram block at the start of the workspace, padded to 256 bytes so the solver's
// fp64 blocks after it stay aligned.
static size_t gram_ws_bytes(int64_t d) { return ((size_t)d * (size_t)d * sizeof(float) + 255) & ~(size_t)255; }

size_t zoact_basis_init_workspace_bytes(int64_t d, int32_t r, const zoact_eig_opts* opts) {
  const size_t solver = zoact_basis_workspace_bytes(d, r, opts);
  return solver ? gram_ws_bytes(d) + solver : 0;
}

zoact_status zoact_gram(const void* x, int32_t x_dtype, int64_t n_tok, int64_t d, int64_t ld_x, float* g,
                        int32_t accumulate, zoact_stream stream) {
  CHECK(x && g, "gram: NULL pointer");
  CHECK(float_type(x_dtype), "gram: dtype must be F32 or BF16");
  CHECK(n_tok >= 1 && d >= 1, "gram: empty shape");
  CHECK(ld_x >= d, "gram: row stride %lld < d = %lld", (long long)ld_x, (long long)d);
  if (x_dtype == ZOACT_BF16) {
    CHECK(d % 64 == 0, "gram: bf16 needs d %% 64 == 0");
    CHECK(ld_x % 8 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0,
          "gram: bf16 needs a row stride that is a multiple of 8 and x 16-byte aligned");
  }
  return hip_status(zoact::launch_gram(x, x_dtype, n_tok, d, ld_x, g, accumulate, st(stream)), "gram");
}

// The solver's argument checks, shared by the Gram and the token-side forms (n: rows of
// the Gram the iteration runs on).
static zoact_status eig_args(const char* fn, const void* ut, int32_t ut_dtype, int64_t n, int32_t r,
                             const zoact_eig_opts& o, const zoact_eig_opts* opts) {
  const int32_t p = o.oversample;
  CHECK(ut, "%s: NULL ut", fn);
  CHECK(float_type(ut_dtype), "%s: ut dtype must be F32 or BF16", fn);
  CHECK(r >= 1 && r <= 256, "%s: r=%d outside [1, 256]", fn, r);
  CHECK(n >= 2 && r + p <= n, "%s: r + oversample = %d exceeds d = %lld", fn, r + p, (long long)n);
  CHECK(r + p <= 512, "%s: block r + oversample = %d exceeds 512", fn, r + p);
  CHECK(o.tol >= 0.f, "%s: negative tol", fn);
  CHECK(!o.adaptive || o.tol > 0.f, "%s: adaptive mode needs tol > 0", fn);
  CHECK(!opts || (opts->max_iter >= 0 && opts->check_every >= 0 && opts->oversample >= 0), "%s: negative option", fn);
  return ZOACT_OK;
}

zoact_status zoact_basis_from_gram(const float* g, int64_t d, int32_t r, const zoact_eig_opts* opts, void* ut,
                                   int32_t ut_dtype, float* ut_master, float* eigvals, zoact_eig_report* report,
                                   void* ws, size_t ws_bytes, zoact_stream stream) {
  const zoact_eig_opts o = eig_resolve(r, opts);
  const int32_t p = o.oversample;
  CHECK(g, "basis_from_gram: NULL g");
  zoact_status s = eig_args("basis_from_gram", ut, ut_dtype, d, r, o, opts);
  if (s != ZOACT_OK) return s;
  const size_t need = zoact::basis_ws_bytes(d, r, p);
  if (ws == nullptr || ws_bytes < need) return fail(ZOACT_E_WORKSPACE, "basis_from_gram: workspace needs %zu bytes", need);
  bool met = true;
  s = hip_status(zoact::launch_basis_from_gram(g, d, r, p, o, ut, ut_dtype, ut_master, eigvals, report, ws, st(stream),
                                               met),
                 "basis_from_gram");
  if (s != ZOACT_OK) return s;
  if (!met) return fail(ZOACT_E_NOCONVERGE, "basis_from_gram: residual above tol %g after %d iterations", o.tol,
                        o.max_iter);
  return ZOACT_OK;
}

zoact_status zoact_basis_init(const void* x, int32_t x_dtype, int64_t n_tok, int64_t d, int64_t ld_x, int32_t r,
                              const zoact_eig_opts* opts, void* ut, int32_t ut_dtype, float* ut_master, float* eigvals,
                              zoact_eig_report* report, void* ws, size_t ws_bytes, zoact_stream stream) {
  CHECK(n_tok >= r, "basis_init: n_tok=%lld < r=%d", (long long)n_tok, r);
  const zoact_eig_opts o = eig_resolve(r, opts);
  const int32_t p = o.oversample;
  CHECK(r >= 1 && r <= 256 && d >= 2 && r + p <= d, "basis_init: bad r=%d for d=%lld", r, (long long)d);
  const size_t gbytes = gram_ws_bytes(d);
  const size_t need = gbytes + zoact::basis_ws_bytes(d, r, p);
  if (ws == nullptr || ws_bytes < need) return fail(ZOACT_E_WORKSPACE, "basis_init: workspace needs %zu bytes", need);
  // Fewer calibration rows than features: the same singular vectors from the n_tok x n_tok
  // token-side Gram (smaller to form and to iterate on), when its workspace fits in ws.
  const bool rows = x && x_dtype == ZOACT_BF16 && n_tok < d && r + p <= n_tok && d % 64 == 0 && ld_x >= d &&
                    ld_x % 8 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0 &&
                    zoact::basis_rows_ws_bytes(n_tok, d, r, p) <= ws_bytes;
  if (rows) {
    zoact_status s = eig_args("basis_init", ut, ut_dtype, n_tok, r, o, opts);
    if (s != ZOACT_OK) return s;
    bool met = true;
    s = hip_status(zoact::launch_basis_init_rows(static_cast<const uint16_t*>(x), n_tok, d, ld_x, r, p, o, ut,
                                                 ut_dtype, ut_master, eigvals, report, ws, st(stream), met),
                   "basis_init");
    if (s != ZOACT_OK) return s;
    if (!met) return fail(ZOACT_E_NOCONVERGE, "basis_init: residual above tol %g after %d iterations", o.tol,
                          o.max_iter);
    return ZOACT_OK;
  }
  float* g = static_cast<float*>(ws);
  zoact_status s = zoact_gram(x, x_dtype, n_tok, d, ld_x, g, 0, stream);
  if (s != ZOACT_OK) return s;
  return zoact_basis_from_gram(g, d, r, opts, ut, ut_dtype, ut_master, eigvals, report,
                               static_cast<char*>(ws) + gbytes, ws_bytes - gbytes, stream);
}

}  // extern "C"

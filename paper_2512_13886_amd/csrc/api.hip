// extern "C" entry points of liboptima.so: argument validation, then the
// launch sequences in hessian.hip, spectral.hip and solver.hip.
#include "common.h"

namespace optima {
size_t hessian_workspace_bytes(int64_t n_tok, int64_t d, int dtype);
optima_status hessian_accumulate(const void* X, int dtype, int64_t n_tok, int64_t d, float* H,
                                 int accumulate, void* ws, hipStream_t s);
optima_status hessian_damp(float* H, int64_t d, float rel, float* lambda_out, hipStream_t s);
optima_status hessian_jacobi(float* H, int64_t d, float* D, hipStream_t s);
size_t spectral_norm_workspace_bytes(int64_t d, int block);
optima_status spectral_norm(const float* H, int64_t d, const float* V0, int block, int max_iters,
                            float tol, void* ws, float* lambda_max, int32_t* iters,
                            hipStream_t s);
optima_status spectral_norm_noalloc(const float* H, int64_t d, const float* V0, int block,
                                    int max_iters, float tol, float* lambda_max, int32_t* iters,
                                    hipStream_t s);
size_t spectral_lanczos_workspace_bytes(int64_t d, int max_steps);
optima_status spectral_lanczos(const float* H, int64_t d, const float* v0, int max_steps,
                               float tol, void* ws, float* lambda_max, int32_t* steps,
                               hipStream_t s);
optima_status wanda_mask(const float* W0, int64_t n_cols, int64_t d, const void* col_sq,
                         int col_dtype, int64_t col_stride, int pattern, double sparsity,
                         uint8_t* mask, hipStream_t s);
size_t qp_workspace_bytes(int64_t d, int64_t n_cols);
size_t linear_forward_workspace_bytes(int64_t n_tok, int64_t d_in, int64_t d_out);
optima_status linear_forward(const void* X, int64_t n_tok, int64_t d_in, const float* W,
                             int64_t d_out, int act, void* Y, int y_dtype, const float* Y_ref,
                             double* err_out, void* ws, hipStream_t s);
optima_status qp_solve(const float* H, int64_t d, const float* lambda_max, const float* W0,
                       const uint8_t* mask, int64_t n_cols, const optima_solver_opts& o, void* ws,
                       float* W_out, const optima_solve_stats& stats, optima_solve_info* info,
                       hipStream_t s);
}  // namespace optima

namespace {
// Sizes are kept within 32-bit tile and row indices.
constexpr int64_t kMaxDim = int64_t(1) << 20;
constexpr int64_t kMaxCols = int64_t(1) << 24;

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}
}  // namespace

extern "C" {

const char* optima_status_string(optima_status status) {
  switch (status) {
    case OPTIMA_OK: return "OPTIMA_OK";
    case OPTIMA_E_INVAL: return "OPTIMA_E_INVAL: invalid argument";
    case OPTIMA_E_HIP: return "OPTIMA_E_HIP: HIP runtime error";
    case OPTIMA_E_NONFINITE: return "OPTIMA_E_NONFINITE: NaN or Inf in the input";
    case OPTIMA_E_WORKSPACE: return "OPTIMA_E_WORKSPACE: workspace missing or too small";
    case OPTIMA_E_UNSUPPORTED: return "OPTIMA_E_UNSUPPORTED: unsupported dtype or device";
    default: return "OPTIMA: unknown status";
  }
}

int optima_abi_version(void) { return 11; }

size_t optima_hessian_workspace_bytes(int64_t n_tok, int64_t d, int dtype) {
  if (n_tok < 0 || d < 1 || d > kMaxDim) return 0;
  if (dtype != OPTIMA_DTYPE_F32 && dtype != OPTIMA_DTYPE_BF16) return 0;
  return optima::hessian_workspace_bytes(n_tok, d, dtype);
}

optima_status optima_hessian_accumulate(const void* X, int dtype, int64_t n_tok, int64_t d,
                                        float* H, int accumulate, void* ws, size_t ws_bytes,
                                        hipStream_t stream) {
  if (dtype != OPTIMA_DTYPE_F32 && dtype != OPTIMA_DTYPE_BF16) return OPTIMA_E_UNSUPPORTED;
  if (!H || n_tok < 0 || d < 1 || d > kMaxDim) return OPTIMA_E_INVAL;
  if (n_tok > 0 && !X) return OPTIMA_E_INVAL;
  const size_t esz = dtype == OPTIMA_DTYPE_BF16 ? 2 : 4;
  if (n_tok > 0 && !optima::aligned16(X)) return OPTIMA_E_INVAL;
  if (X && overlaps(X, size_t(n_tok) * size_t(d) * esz, H, size_t(d) * size_t(d) * 4))
    return OPTIMA_E_INVAL;
  if (n_tok > 0) {
    const size_t need = optima::hessian_workspace_bytes(n_tok, d, dtype);
    if (!ws || ws_bytes < need) return OPTIMA_E_WORKSPACE;
  }
  return optima::hessian_accumulate(X, dtype, n_tok, d, H, accumulate ? 1 : 0, ws, stream);
}

optima_status optima_hessian_damp(float* H, int64_t d, float rel_damp, float* lambda_out,
                                  hipStream_t stream) {
  if (!H || !lambda_out || d < 1 || d > kMaxDim) return OPTIMA_E_INVAL;
  if (!(rel_damp >= 0.f)) return OPTIMA_E_INVAL;
  return optima::hessian_damp(H, d, rel_damp, lambda_out, stream);
}

optima_status optima_hessian_jacobi(float* H, int64_t d, float* scale_out, hipStream_t stream) {
  if (!H || !scale_out || d < 1 || d > kMaxDim) return OPTIMA_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(H) & 3) || (reinterpret_cast<uintptr_t>(scale_out) & 3))
    return OPTIMA_E_INVAL;
  if (overlaps(H, size_t(d) * size_t(d) * 4, scale_out, size_t(d) * 4)) return OPTIMA_E_INVAL;
  return optima::hessian_jacobi(H, d, scale_out, stream);
}

size_t optima_spectral_norm_workspace_bytes(int64_t d, int block) {
  if (d < 1 || d > kMaxDim || block < 1 || block > OPTIMA_SPECTRAL_MAX_BLOCK) return 0;
  return optima::spectral_norm_workspace_bytes(d, block);
}

optima_status optima_spectral_norm(const float* H, int64_t d, const float* V0, int block,
                                   int max_iters, float tol, void* ws, size_t ws_bytes,
                                   float* lambda_max, int32_t* iters, hipStream_t stream) {
  if (!H || !V0 || !lambda_max || d < 1 || d > kMaxDim || max_iters < 1 || !(tol >= 0.f))
    return OPTIMA_E_INVAL;
  if (block < 1 || block > OPTIMA_SPECTRAL_MAX_BLOCK) return OPTIMA_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(V0) & 3) || (reinterpret_cast<uintptr_t>(H) & 3))
    return OPTIMA_E_INVAL;
  if (!ws || ws_bytes < optima::spectral_norm_workspace_bytes(d, block))
    return OPTIMA_E_WORKSPACE;
  return optima::spectral_norm(H, d, V0, block, max_iters, tol, ws, lambda_max, iters, stream);
}

optima_status optima_spectral_norm_noalloc(const float* H, int64_t d, const float* V0, int block,
                                           int max_iters, float tol, float* lambda_max,
                                           int32_t* iters, hipStream_t stream) {
  if (!H || !V0 || !lambda_max || d < 1 || d > kMaxDim || max_iters < 1 || !(tol >= 0.f))
    return OPTIMA_E_INVAL;
  if (block < 1 || block > OPTIMA_SPECTRAL_MAX_BLOCK) return OPTIMA_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(V0) & 3) || (reinterpret_cast<uintptr_t>(H) & 3))
    return OPTIMA_E_INVAL;
  if (d > OPTIMA_SPECTRAL_NOALLOC_MAX_DIM) return OPTIMA_E_WORKSPACE;
  return optima::spectral_norm_noalloc(H, d, V0, block, max_iters, tol, lambda_max, iters,
                                       stream);
}

size_t optima_spectral_lanczos_workspace_bytes(int64_t d, int max_steps) {
  if (d < 1 || d > kMaxDim || max_steps < 1 || max_steps > OPTIMA_LANCZOS_MAX_STEPS) return 0;
  return optima::spectral_lanczos_workspace_bytes(d, max_steps);
}

optima_status optima_spectral_lanczos(const float* H, int64_t d, const float* v0, int max_steps,
                                      float tol, void* ws, size_t ws_bytes, float* lambda_max,
                                      int32_t* steps, hipStream_t stream) {
  if (!H || !v0 || !lambda_max || d < 1 || d > kMaxDim || !(tol >= 0.f)) return OPTIMA_E_INVAL;
  if (max_steps < 1 || max_steps > OPTIMA_LANCZOS_MAX_STEPS) return OPTIMA_E_INVAL;
  if ((reinterpret_cast<uintptr_t>(v0) & 3) || (reinterpret_cast<uintptr_t>(H) & 3))
    return OPTIMA_E_INVAL;
  if (!ws || ws_bytes < optima::spectral_lanczos_workspace_bytes(d, max_steps))
    return OPTIMA_E_WORKSPACE;
  return optima::spectral_lanczos(H, d, v0, max_steps, tol, ws, lambda_max, steps, stream);
}

optima_status optima_wanda_mask(const float* W0, int64_t n_cols, int64_t d, const void* col_sq,
                                int col_sq_dtype, int64_t col_sq_stride, int pattern,
                                double sparsity, uint8_t* mask, hipStream_t stream) {
  if (d < 1 || d > kMaxDim || n_cols < 0 || n_cols > kMaxCols) return OPTIMA_E_INVAL;
  if (n_cols == 0) return OPTIMA_OK;
  if (!W0 || !col_sq || !mask || col_sq_stride < 1) return OPTIMA_E_INVAL;
  if (col_sq_dtype != OPTIMA_DTYPE_F32 && col_sq_dtype != OPTIMA_DTYPE_F64)
    return OPTIMA_E_UNSUPPORTED;
  const size_t csz = col_sq_dtype == OPTIMA_DTYPE_F64 ? 8 : 4;
  if ((reinterpret_cast<uintptr_t>(W0) & 3) || (reinterpret_cast<uintptr_t>(mask) & 3) ||
      (reinterpret_cast<uintptr_t>(col_sq) % csz))
    return OPTIMA_E_INVAL;
  if (pattern == OPTIMA_MASK_2TO4) {
    if (d % 4) return OPTIMA_E_INVAL;
  } else if (pattern == OPTIMA_MASK_UNSTRUCTURED) {
    if (!(sparsity >= 0.0 && sparsity <= 1.0)) return OPTIMA_E_INVAL;
  } else {
    return OPTIMA_E_INVAL;
  }
  const size_t mbytes = size_t(n_cols) * size_t(d);
  if (overlaps(mask, mbytes, W0, mbytes * 4) ||
      overlaps(mask, mbytes, col_sq, (size_t(d - 1) * size_t(col_sq_stride) + 1) * csz))
    return OPTIMA_E_INVAL;
  return optima::wanda_mask(W0, n_cols, d, col_sq, col_sq_dtype, col_sq_stride, pattern,
                            sparsity, mask, stream);
}

size_t optima_linear_forward_workspace_bytes(int64_t n_tok, int64_t d_in, int64_t d_out) {
  if (n_tok < 0 || d_in < 64 || d_in > kMaxDim || d_in % 64 || d_out < 4 || d_out > kMaxDim ||
      d_out % 4)
    return 0;
  // one workgroup per 128 x 128 output tile; the grid stays below 2^31
  if ((n_tok + 127) / 128 * ((d_out + 127) / 128) >= (int64_t(1) << 31)) return 0;
  return optima::linear_forward_workspace_bytes(n_tok, d_in, d_out);
}

optima_status optima_linear_forward(const void* X, int64_t n_tok, int64_t d_in, const float* W,
                                    int64_t d_out, int act, void* Y, int y_dtype,
                                    const float* Y_ref, double* err_out, void* ws,
                                    size_t ws_bytes, hipStream_t stream) {
  const size_t need = optima_linear_forward_workspace_bytes(n_tok, d_in, d_out);
  if (!need) return OPTIMA_E_INVAL;
  // Nothing to do without Y or err_out; an error needs its reference (no
  // pointer is read when n_tok == 0).
  if (!W || (n_tok > 0 && !X) || (!Y && !err_out)) return OPTIMA_E_INVAL;
  if ((Y_ref && !err_out) || (err_out && n_tok > 0 && !Y_ref)) return OPTIMA_E_INVAL;
  if (act != OPTIMA_ACT_NONE && act != OPTIMA_ACT_SILU) return OPTIMA_E_INVAL;
  if (Y && y_dtype != OPTIMA_DTYPE_BF16 && y_dtype != OPTIMA_DTYPE_F32) return OPTIMA_E_INVAL;
  if ((X && !optima::aligned16(X)) || (reinterpret_cast<uintptr_t>(W) & 3)) return OPTIMA_E_INVAL;
  if (Y && (reinterpret_cast<uintptr_t>(Y) & (y_dtype == OPTIMA_DTYPE_F32 ? 15 : 7)))
    return OPTIMA_E_INVAL;
  if (Y_ref && !optima::aligned16(Y_ref)) return OPTIMA_E_INVAL;
  if (err_out && (reinterpret_cast<uintptr_t>(err_out) & 7)) return OPTIMA_E_INVAL;
  const size_t ybytes = size_t(n_tok) * size_t(d_out) * (Y && y_dtype == OPTIMA_DTYPE_BF16 ? 2 : 4);
  if (Y && (overlaps(Y, ybytes, X, size_t(n_tok) * size_t(d_in) * 2) ||
            overlaps(Y, ybytes, W, size_t(d_out) * size_t(d_in) * 4) ||
            (Y_ref && overlaps(Y, ybytes, Y_ref, size_t(n_tok) * size_t(d_out) * 4))))
    return OPTIMA_E_INVAL;
  if (!ws || ws_bytes < need) return OPTIMA_E_WORKSPACE;
  return optima::linear_forward(X, n_tok, d_in, W, d_out, act, Y, y_dtype, Y_ref, err_out, ws,
                                stream);
}

void optima_solver_opts_default(optima_solver_opts* o) {
  if (!o) return;
  o->max_iters = 100000;
  o->check_every = 64;
  o->fixed_iters = 0;
  o->eps_rel = 0.01f;
  o->eps_abs = 0.01f;
  o->beta_sufficient = 0.2f;
  o->beta_necessary = 0.8f;
  o->beta_artificial = 0.36f;
  o->step_safety = 1e-3f;
  o->restarts = 1;
  o->precision = OPTIMA_PREC_BF16X3;
  o->method = OPTIMA_METHOD_RAPDHG;
  o->col_scale = nullptr;
  o->sparse = 1;
  o->cooperative = 1;
}

size_t optima_qp_workspace_bytes(int64_t d, int64_t n_cols) {
  if (d < 1 || d > kMaxDim || n_cols < 0 || n_cols > kMaxCols) return 0;
  return optima::qp_workspace_bytes(d, n_cols);
}

optima_status optima_qp_solve_batched(const float* H, int64_t d, const float* lambda_max,
                                      const float* W0, const uint8_t* mask, int64_t n_cols,
                                      const optima_solver_opts* opts, void* ws, size_t ws_bytes,
                                      float* W_out, const optima_solve_stats* stats,
                                      optima_solve_info* info, hipStream_t stream) {
  if (!opts || d < 1 || d > kMaxDim || n_cols < 0 || n_cols > kMaxCols) return OPTIMA_E_INVAL;
  if (info) *info = optima_solve_info{};
  if (n_cols == 0) return OPTIMA_OK;
  if (opts->method != OPTIMA_METHOD_RAPDHG && opts->method != OPTIMA_METHOD_CG)
    return OPTIMA_E_INVAL;
  if (!H || !W0 || !mask || !W_out) return OPTIMA_E_INVAL;
  if (!lambda_max && opts->method == OPTIMA_METHOD_RAPDHG) return OPTIMA_E_INVAL;
  if (!optima::aligned16(H) || (reinterpret_cast<uintptr_t>(W0) & 3) ||
      (reinterpret_cast<uintptr_t>(W_out) & 3) ||
      (reinterpret_cast<uintptr_t>(opts->col_scale) & 3))
    return OPTIMA_E_INVAL;
  const size_t wbytes = size_t(n_cols) * size_t(d) * sizeof(float);
  if (overlaps(W0, wbytes, W_out, wbytes) || overlaps(H, size_t(d) * d * 4, W_out, wbytes) ||
      overlaps(mask, size_t(n_cols) * d, W_out, wbytes))
    return OPTIMA_E_INVAL;
  const optima_solver_opts& o = *opts;
  if (o.max_iters < 0 || o.check_every < 1) return OPTIMA_E_INVAL;
  if (o.sparse != 0 && o.sparse != 1) return OPTIMA_E_INVAL;
  if (o.cooperative != 0 && o.cooperative != 1) return OPTIMA_E_INVAL;
  if (o.precision != OPTIMA_PREC_FP32 && o.precision != OPTIMA_PREC_BF16X3)
    return OPTIMA_E_UNSUPPORTED;
  if (!(o.eps_rel >= 0.f) || !(o.eps_abs >= 0.f) || !(o.step_safety >= 0.f) ||
      !(o.beta_sufficient >= 0.f) || !(o.beta_necessary >= 0.f) || !(o.beta_artificial >= 0.f))
    return OPTIMA_E_INVAL;
  if (!ws || ws_bytes < optima::qp_workspace_bytes(d, n_cols)) return OPTIMA_E_WORKSPACE;
  optima_solve_stats st{};
  if (stats) st = *stats;
  return optima::qp_solve(H, d, lambda_max, W0, mask, n_cols, o, ws, W_out, st, info, stream);
}

}  // extern "C"

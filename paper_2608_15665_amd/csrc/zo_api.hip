// C ABI of libzo: argument validation on the host, then the launchers.
// Nothing here allocates device memory or synchronises the stream.
#include "zo_internal.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

namespace {
thread_local char g_detail[512] = "";

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

#define ZO_CHECK(cond, ...)           \
  do {                                \
    if (!(cond)) {                    \
      zo_set_error(__VA_ARGS__);      \
      return ZO_ERR_INVALID_ARG;      \
    }                                 \
  } while (0)

}  // namespace

void zo_set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_detail, sizeof(g_detail), fmt, ap);
  va_end(ap);
}

int zo_hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ZO_OK;
  zo_set_error("%s: %s", what, hipGetErrorString(e));
  return ZO_ERR_HIP;
}

extern "C" {

int zo_abi_version(void) { return ZO_ABI_VERSION; }

const char* zo_status_str(int s) {
  switch (s) {
    case ZO_OK: return "ok";
    case ZO_ERR_INVALID_ARG: return "invalid argument";
    case ZO_ERR_UNSUPPORTED: return "unsupported";
    case ZO_ERR_RANK_DEFICIENT: return "rank deficient";
    case ZO_ERR_NONFINITE: return "non-finite value";
    case ZO_ERR_HIP: return "HIP runtime error";
    case ZO_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

const char* zo_last_error_detail(void) { return g_detail; }

// ------------------------------------------------------------------ refresh
static int check_refresh(int count, const zo_panel* panels, int r) {
  ZO_CHECK(count >= 0, "refresh: count = %d < 0", count);
  ZO_CHECK(count == 0 || panels, "refresh: panels is NULL");
  ZO_CHECK(r >= 1 && r <= ZO_MAX_QR_RANK, "refresh: r = %d outside [1, %d]", r, ZO_MAX_QR_RANK);
  for (int p = 0; p < count; ++p) {
    const zo_panel& pn = panels[p];
    ZO_CHECK(pn.rows >= r, "refresh: panel %d has rows = %d < r = %d", p, pn.rows, r);
    ZO_CHECK(pn.rows <= (1 << 26), "refresh: panel %d rows = %d too large", p, pn.rows);
    ZO_CHECK(pn.omega && pn.q, "refresh: panel %d has a NULL omega or q", p);
    ZO_CHECK(aligned(pn.omega, 4) && aligned(pn.q, 4) && aligned(pn.r_diag, 4),
             "refresh: panel %d pointer not 4-byte aligned", p);
  }
  return ZO_OK;
}

size_t zo_subspace_refresh_workspace(int count, const zo_panel* panels, int r) {
  if (check_refresh(count, panels, r) != ZO_OK) return 0;
  size_t need = 0;
  zo_refresh_launch(count, panels, r, nullptr, nullptr, 0, nullptr, &need);
  return need;
}

int zo_subspace_refresh(int count, const zo_panel* panels, int r, int* info, void* workspace,
                        size_t ws_bytes, void* stream) {
  int st = check_refresh(count, panels, r);
  if (st != ZO_OK) return st;
  if (count == 0) return ZO_OK;
  size_t need = 0;
  zo_refresh_launch(count, panels, r, nullptr, nullptr, 0, nullptr, &need);
  if (ws_bytes < need || (need && !workspace)) {
    zo_set_error("refresh: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "refresh: workspace not 256-byte aligned");
  return zo_refresh_launch(count, panels, r, info, workspace, ws_bytes, (hipStream_t)stream,
                           nullptr);
}

int zo_subspace_refresh_noalloc(int count, const zo_panel* panels, int r, int* info, void* stream) {
  int st = check_refresh(count, panels, r);
  if (st != ZO_OK) return st;
  if (count == 0) return ZO_OK;
  size_t need = 0;
  zo_refresh_launch(count, panels, r, nullptr, nullptr, 0, nullptr, &need);
  if (need > (size_t)ZO_NOALLOC_SCRATCH_BYTES) {
    zo_set_error("refresh_noalloc: these %d panels need %zu bytes of scratch, more than the %zu-byte "
                 "static scratch; refresh them over several calls", count, need,
                 (size_t)ZO_NOALLOC_SCRATCH_BYTES);
    return ZO_ERR_WORKSPACE;
  }
  void* scratch = nullptr;
  if ((st = zo_refresh_scratch(&scratch)) != ZO_OK) return st;
  return zo_refresh_launch(count, panels, r, info, scratch, (size_t)ZO_NOALLOC_SCRATCH_BYTES,
                           (hipStream_t)stream, nullptr);
}

// --------------------------------------------------------- perturbed linear
static int check_plinear(int T, int m, int n, int r, int q, int nblk, long long xs, int in_dtype) {
  ZO_CHECK(T >= 1 && m >= 1 && n >= 1, "perturbed_linear: T, m, n must be >= 1 (got %d, %d, %d)",
           T, m, n);
  ZO_CHECK(r >= 1 && r <= ZO_MAX_RANK, "perturbed_linear: r = %d outside [1, %d]", r, ZO_MAX_RANK);
  ZO_CHECK(q >= 1 && q <= ZO_MAX_QUERIES, "perturbed_linear: q = %d outside [1, %d]", q,
           ZO_MAX_QUERIES);
  ZO_CHECK(nblk >= 1 && nblk <= ZO_MAX_BLOCKS, "perturbed_linear: nblk = %d outside [1, %d]", nblk,
           ZO_MAX_BLOCKS);
  ZO_CHECK(in_dtype == ZO_F32 || in_dtype == ZO_BF16 || in_dtype == ZO_F16,
           "perturbed_linear: bad in_dtype %d", in_dtype);
  ZO_CHECK(xs == 0 || xs >= (long long)T * n,
           "perturbed_linear: x_block_stride = %lld must be 0 or >= T*n", xs);
  ZO_CHECK((long long)T * nblk < (1LL << 31), "perturbed_linear: T * nblk too large");
  if (in_dtype != ZO_F32) {
    ZO_CHECK(m % 8 == 0 && n % 8 == 0, "perturbed_linear: 16-bit inputs need m %% 8 == 0 and "
             "n %% 8 == 0 (got m = %d, n = %d)", m, n);
    ZO_CHECK(xs % 8 == 0, "perturbed_linear: 16-bit x_block_stride must be a multiple of 8");
  }
  return ZO_OK;
}

size_t zo_perturbed_linear_workspace(int T, int m, int n, int r, int q, int nblk,
                                     long long x_block_stride, int in_dtype) {
  if (check_plinear(T, m, n, r, q, nblk, x_block_stride, in_dtype) != ZO_OK) return 0;
  PlinearPlan p;
  zo_plinear_plan(&p, T, m, n, r, q, nblk, x_block_stride, in_dtype, in_dtype);
  return p.ws_total;
}

static int check_plinear_call(int T, int m, int n, int r, int q, int nblk, long long xs,
                              int in_dtype, int out_dtype, const void* X, const void* W,
                              const void* Y, void* workspace, size_t ws_bytes, PlinearPlan* p) {
  int st = check_plinear(T, m, n, r, q, nblk, xs, in_dtype);
  if (st != ZO_OK) return st;
  ZO_CHECK(out_dtype == ZO_F32 || out_dtype == ZO_BF16 || out_dtype == ZO_F16,
           "perturbed_linear: bad out_dtype %d", out_dtype);
  if (out_dtype != ZO_F32 && out_dtype != in_dtype) {
    zo_set_error("perturbed_linear: out_dtype %d must be in_dtype (%d) or fp32", out_dtype, in_dtype);
    return ZO_ERR_UNSUPPORTED;
  }
  ZO_CHECK(X, "perturbed_linear: NULL tensor argument (X)");
  const size_t al = in_dtype != ZO_F32 ? 16 : 4;
  ZO_CHECK(aligned(X, al) && aligned(W, al) && aligned(Y, al),
           "perturbed_linear: X, W and Y must be %zu-byte aligned", al);
  zo_plinear_plan(p, T, m, n, r, q, nblk, xs, in_dtype, out_dtype);
  if (ws_bytes < p->ws_total || !workspace) {
    zo_set_error("perturbed_linear: workspace %zu bytes < required %zu", ws_bytes, p->ws_total);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "perturbed_linear: workspace not 256-byte aligned");
  return ZO_OK;
}

static int check_blocks(int q, int nblk, const int* blk_query, const int8_t* blk_sign, float eps,
                        const float* U, const float* V, const float* Z) {
  ZO_CHECK(blk_query && blk_sign, "perturbed_linear: blk_query / blk_sign is NULL");
  for (int b = 0; b < nblk; ++b) {
    ZO_CHECK(blk_query[b] >= 0 && blk_query[b] < q, "perturbed_linear: blk_query[%d] = %d outside "
             "[0, %d)", b, blk_query[b], q);
    ZO_CHECK(blk_sign[b] >= -1 && blk_sign[b] <= 1, "perturbed_linear: blk_sign[%d] = %d not in "
             "{-1, 0, 1}", b, (int)blk_sign[b]);
  }
  ZO_CHECK(isfinite(eps), "perturbed_linear: eps is not finite");
  ZO_CHECK(U && V && Z, "perturbed_linear: NULL tensor argument (U, V or Z)");
  ZO_CHECK(aligned(U, 4) && aligned(V, 4) && aligned(Z, 4), "perturbed_linear: U, V, Z alignment");
  return ZO_OK;
}

int zo_perturbed_linear(int T, int m, int n, int r, int q, int nblk, const int* blk_query,
                        const int8_t* blk_sign, float eps, int in_dtype, const void* X,
                        long long x_block_stride, const void* W, const float* U, const float* V,
                        const float* Z, int out_dtype, void* Y, void* workspace, size_t ws_bytes,
                        void* stream) {
  PlinearPlan p;
  int st = check_plinear(T, m, n, r, q, nblk, x_block_stride, in_dtype);
  if (st != ZO_OK) return st;
  if ((st = check_blocks(q, nblk, blk_query, blk_sign, eps, U, V, Z)) != ZO_OK) return st;
  ZO_CHECK(W && Y, "perturbed_linear: NULL tensor argument (W or Y)");
  st = check_plinear_call(T, m, n, r, q, nblk, x_block_stride, in_dtype, out_dtype, X, W, Y,
                          workspace, ws_bytes, &p);
  if (st != ZO_OK) return st;
  st = zo_plinear_prepare(p, blk_query, blk_sign, eps, X, U, V, Z, workspace, (hipStream_t)stream);
  if (st != ZO_OK) return st;
  return zo_plinear_apply(p, X, W, Y, workspace, (hipStream_t)stream);
}

int zo_perturbed_linear_prepare(int T, int m, int n, int r, int q, int nblk,
                                const int* blk_query, const int8_t* blk_sign, float eps,
                                int in_dtype, const void* X, long long x_block_stride,
                                const float* U, const float* V, const float* Z, void* workspace,
                                size_t ws_bytes, void* stream) {
  PlinearPlan p;
  int st = check_plinear(T, m, n, r, q, nblk, x_block_stride, in_dtype);
  if (st != ZO_OK) return st;
  if ((st = check_blocks(q, nblk, blk_query, blk_sign, eps, U, V, Z)) != ZO_OK) return st;
  // The output dtype does not enter the prepared operands.
  st = check_plinear_call(T, m, n, r, q, nblk, x_block_stride, in_dtype, in_dtype, X, nullptr,
                          nullptr, workspace, ws_bytes, &p);
  if (st != ZO_OK) return st;
  return zo_plinear_prepare(p, blk_query, blk_sign, eps, X, U, V, Z, workspace, (hipStream_t)stream);
}

size_t zo_perturbed_linear_group_workspace(int count, int T, int n, int r, int q, int nblk,
                                           long long x_block_stride, int in_dtype) {
  if (count < 1 || count > ZO_MAX_GROUP) return 0;
  if (check_plinear(T, 8, n, r, q, nblk, x_block_stride, in_dtype) != ZO_OK) return 0;
  PlinearPlan p;
  zo_plinear_plan(&p, T, 8, n, r, q, nblk, x_block_stride, in_dtype, in_dtype);
  return zo_plinear_group_ws(p, count);
}

int zo_perturbed_linear_prepare_group(int count, const int* m, int T, int n, int r, int q, int nblk,
                                      const int* blk_query, const int8_t* blk_sign, float eps, int in_dtype,
                                      const void* X, long long x_block_stride, const float* const* U,
                                      const float* const* V, const float* const* Z, void* const* workspace,
                                      const size_t* ws_bytes, void* group_ws, size_t group_ws_bytes,
                                      void* stream) {
  ZO_CHECK(count >= 1 && count <= ZO_MAX_GROUP, "prepare_group: count = %d outside [1, %d]", count,
           ZO_MAX_GROUP);
  ZO_CHECK(m && U && V && Z && workspace && ws_bytes, "prepare_group: NULL descriptor array");
  PlinearPlan plans[ZO_MAX_GROUP];
  int st;
  for (int i = 0; i < count; ++i) {
    if ((st = check_plinear(T, m[i], n, r, q, nblk, x_block_stride, in_dtype)) != ZO_OK) return st;
    if ((st = check_blocks(q, nblk, blk_query, blk_sign, eps, U[i], V[i], Z[i])) != ZO_OK) return st;
    if ((st = check_plinear_call(T, m[i], n, r, q, nblk, x_block_stride, in_dtype, in_dtype, X, nullptr, nullptr,
                                 workspace[i], ws_bytes[i], &plans[i])) != ZO_OK)
      return st;
  }
  const size_t need = zo_plinear_group_ws(plans[0], count);
  if (need > 0) {
    if (!group_ws || group_ws_bytes < need) {
      zo_set_error("prepare_group: group workspace %zu bytes < required %zu", group_ws_bytes, need);
      return ZO_ERR_WORKSPACE;
    }
    ZO_CHECK(aligned(group_ws, 256), "prepare_group: group workspace not 256-byte aligned");
  }
  // Each matrix keeps its prepared operands in its own workspace until its apply, and the group
  // scratch is read after every matrix's part has been written: no two of the regions the call
  // writes may overlap (a shared buffer would hand every apply the last matrix's operands).
  auto overlap = [](const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return na > 0 && nb > 0 && x < y + nb && y < x + na;
  };
  for (int i = 0; i < count; ++i) {
    for (int j = i + 1; j < count; ++j)
      ZO_CHECK(!overlap(workspace[i], plans[i].ws_total, workspace[j], plans[j].ws_total),
               "prepare_group: workspaces of matrices %d and %d overlap; each matrix needs its own", i, j);
    ZO_CHECK(!overlap(workspace[i], plans[i].ws_total, group_ws, need),
             "prepare_group: the group workspace overlaps matrix %d's workspace", i);
  }
  return zo_plinear_prepare_group(plans, count, blk_query, blk_sign, eps, X, U, V, Z, workspace, group_ws,
                                  (hipStream_t)stream);
}

int zo_perturbed_linear_apply_ex(int T, int m, int n, int r, int q, int nblk, int in_dtype,
                                 const void* X, long long x_block_stride, const void* W,
                                 int out_dtype, void* Y, int epilogue, const void* R,
                                 long long r_block_stride, void* workspace, size_t ws_bytes,
                                 void* stream) {
  PlinearPlan p;
  ZO_CHECK(W && Y, "perturbed_linear: NULL tensor argument (W or Y)");
  ZO_CHECK(epilogue == ZO_EPI_NONE || epilogue == ZO_EPI_RELU || epilogue == ZO_EPI_RESIDUAL ||
               epilogue == ZO_EPI_SILU_MUL,
           "perturbed_linear: bad epilogue %d", epilogue);
  const bool uses_r = epilogue == ZO_EPI_RESIDUAL || epilogue == ZO_EPI_SILU_MUL;
  if (uses_r) {
    ZO_CHECK(R, "perturbed_linear: epilogue %d with a NULL R", epilogue);
    ZO_CHECK(r_block_stride == 0 || r_block_stride >= (long long)T * m,
             "perturbed_linear: r_block_stride = %lld must be 0 or >= T*m", r_block_stride);
    ZO_CHECK(out_dtype == ZO_F32 || r_block_stride % 8 == 0,
             "perturbed_linear: 16-bit r_block_stride must be a multiple of 8");
    ZO_CHECK(aligned(R, out_dtype == ZO_F32 ? 4 : 16), "perturbed_linear: R alignment");
  }
  int st = check_plinear_call(T, m, n, r, q, nblk, x_block_stride, in_dtype, out_dtype, X, W, Y,
                              workspace, ws_bytes, &p);
  if (st != ZO_OK) return st;
  return zo_plinear_apply(p, X, W, Y, workspace, (hipStream_t)stream, epilogue, uses_r ? R : nullptr,
                          r_block_stride);
}

int zo_perturbed_linear_apply(int T, int m, int n, int r, int q, int nblk, int in_dtype,
                              const void* X, long long x_block_stride, const void* W,
                              int out_dtype, void* Y, void* workspace, size_t ws_bytes,
                              void* stream) {
  return zo_perturbed_linear_apply_ex(T, m, n, r, q, nblk, in_dtype, X, x_block_stride, W,
                                      out_dtype, Y, ZO_EPI_NONE, nullptr, 0, workspace, ws_bytes,
                                      stream);
}

// ------------------------------------------------------------- LoRA scheme
static int check_lora(int T, int m, int n, int rl, int r, int q, int nblk, long long xs,
                      int in_dtype) {
  ZO_CHECK(rl >= 1 && r >= 1 && rl + r <= ZO_MAX_RANK,
           "lora_perturbed_linear: r_L = %d, r = %d (need both >= 1, r_L + r <= %d)", rl, r,
           ZO_MAX_RANK);
  return check_plinear(T, m, n, rl + r, q, nblk, xs, in_dtype);
}

static int check_lora_factors(int q, int nblk, const int* blk_query, const int8_t* blk_sign,
                              float eps, float scale, const float* A, const float* UA,
                              const float* VA, const float* ZA, const float* B, const float* UB,
                              const float* VB, const float* ZB) {
  int st = check_blocks(q, nblk, blk_query, blk_sign, eps, UA, VA, ZA);
  if (st != ZO_OK) return st;
  ZO_CHECK(isfinite(scale), "lora_perturbed_linear: scale is not finite");
  ZO_CHECK(A && B && UB && VB && ZB, "lora_perturbed_linear: NULL tensor argument (A, B, U_B, V_B "
           "or Z_B)");
  ZO_CHECK(aligned(A, 4) && aligned(B, 4) && aligned(UB, 4) && aligned(VB, 4) && aligned(ZB, 4),
           "lora_perturbed_linear: adapter tensors must be 4-byte aligned");
  return ZO_OK;
}

size_t zo_lora_perturbed_linear_workspace(int T, int m, int n, int rl, int r, int q, int nblk,
                                          long long x_block_stride, int in_dtype) {
  if (check_lora(T, m, n, rl, r, q, nblk, x_block_stride, in_dtype) != ZO_OK) return 0;
  PlinearPlan p;
  zo_plinear_plan(&p, T, m, n, rl + r, q, nblk, x_block_stride, in_dtype, in_dtype);
  return p.ws_total;
}

int zo_lora_perturbed_linear_prepare(int T, int m, int n, int rl, int r, int q, int nblk,
                                     const int* blk_query, const int8_t* blk_sign, float eps,
                                     float scale, int in_dtype, const void* X,
                                     long long x_block_stride, const float* A, const float* UA,
                                     const float* VA, const float* ZA, const float* B,
                                     const float* UB, const float* VB, const float* ZB,
                                     void* workspace, size_t ws_bytes, void* stream) {
  PlinearPlan p;
  int st = check_lora(T, m, n, rl, r, q, nblk, x_block_stride, in_dtype);
  if (st != ZO_OK) return st;
  st = check_lora_factors(q, nblk, blk_query, blk_sign, eps, scale, A, UA, VA, ZA, B, UB, VB, ZB);
  if (st != ZO_OK) return st;
  st = check_plinear_call(T, m, n, rl + r, q, nblk, x_block_stride, in_dtype, in_dtype, X, nullptr,
                          nullptr, workspace, ws_bytes, &p);
  if (st != ZO_OK) return st;
  return zo_lora_prepare(p, rl, r, blk_query, blk_sign, eps, scale, X, A, UA, VA, ZA, B, UB, VB,
                         ZB, workspace, (hipStream_t)stream);
}

int zo_lora_perturbed_linear(int T, int m, int n, int rl, int r, int q, int nblk,
                             const int* blk_query, const int8_t* blk_sign, float eps, float scale,
                             int in_dtype, const void* X, long long x_block_stride, const void* W,
                             const float* A, const float* UA, const float* VA, const float* ZA,
                             const float* B, const float* UB, const float* VB, const float* ZB,
                             int out_dtype, void* Y, void* workspace, size_t ws_bytes,
                             void* stream) {
  PlinearPlan p;
  int st = check_lora(T, m, n, rl, r, q, nblk, x_block_stride, in_dtype);
  if (st != ZO_OK) return st;
  st = check_lora_factors(q, nblk, blk_query, blk_sign, eps, scale, A, UA, VA, ZA, B, UB, VB, ZB);
  if (st != ZO_OK) return st;
  ZO_CHECK(W && Y, "lora_perturbed_linear: NULL tensor argument (W or Y)");
  st = check_plinear_call(T, m, n, rl + r, q, nblk, x_block_stride, in_dtype, out_dtype, X, W, Y,
                          workspace, ws_bytes, &p);
  if (st != ZO_OK) return st;
  st = zo_lora_prepare(p, rl, r, blk_query, blk_sign, eps, scale, X, A, UA, VA, ZA, B, UB, VB, ZB,
                       workspace, (hipStream_t)stream);
  if (st != ZO_OK) return st;
  return zo_plinear_apply(p, X, W, Y, workspace, (hipStream_t)stream);
}

// ------------------------------------------------------- decoder layer
int zo_layernorm(long long rows, int d, int dtype, const void* X, const float* gamma,
                 const float* beta, float eps_ln, void* Y, void* stream) {
  ZO_CHECK(rows >= 0 && d >= 8 && d % 8 == 0, "layernorm: rows = %lld, d = %d (need d %% 8 == 0)",
           rows, d);
  ZO_CHECK(dtype == ZO_F32 || dtype == ZO_BF16 || dtype == ZO_F16, "layernorm: bad dtype %d", dtype);
  ZO_CHECK(isfinite(eps_ln) && eps_ln >= 0.f, "layernorm: eps_ln must be finite and >= 0");
  if (rows == 0) return ZO_OK;
  ZO_CHECK(X && Y && gamma && beta, "layernorm: NULL tensor argument");
  ZO_CHECK(aligned(X, 16) && aligned(Y, 16) && aligned(gamma, 16) && aligned(beta, 16),
           "layernorm: X, Y, gamma, beta must be 16-byte aligned");
  return zo_layernorm_launch(rows, d, dtype, X, gamma, beta, eps_ln, Y, (hipStream_t)stream);
}

int zo_rmsnorm(long long rows, int d, int dtype, const void* X, const float* gamma, float eps,
               void* Y, void* stream) {
  ZO_CHECK(rows >= 0 && d >= 8 && d % 8 == 0, "rmsnorm: rows = %lld, d = %d (need d %% 8 == 0)", rows, d);
  ZO_CHECK(dtype == ZO_F32 || dtype == ZO_BF16 || dtype == ZO_F16, "rmsnorm: bad dtype %d", dtype);
  ZO_CHECK(isfinite(eps) && eps >= 0.f, "rmsnorm: eps must be finite and >= 0");
  if (rows == 0) return ZO_OK;
  ZO_CHECK(X && Y && gamma, "rmsnorm: NULL tensor argument");
  ZO_CHECK(aligned(X, 16) && aligned(Y, 16) && aligned(gamma, 16),
           "rmsnorm: X, Y, gamma must be 16-byte aligned");
  return zo_layernorm_launch(rows, d, dtype, X, gamma, nullptr, eps, Y, (hipStream_t)stream, true);
}

static int check_rope(long long rows, int seq_len, int d, int heads, int dtype, float base) {
  ZO_CHECK(rows >= 0 && seq_len >= 1 && rows % seq_len == 0,
           "rope: rows = %lld, seq_len = %d (need rows %% seq_len == 0)", rows, seq_len);
  ZO_CHECK(heads >= 1 && d >= 16 && d % heads == 0 && (d / heads) % 16 == 0,
           "rope: d = %d, heads = %d (need a head dim that is a multiple of 16)", d, heads);
  ZO_CHECK(isfinite(base) && base > 1.f, "rope: base must be finite and > 1");
  if (dtype != ZO_BF16 && dtype != ZO_F16) {
    zo_set_error("rope: dtype %d unsupported (bf16 or fp16)", dtype);
    return ZO_ERR_UNSUPPORTED;
  }
  return ZO_OK;
}

int zo_rope(long long rows, int seq_len, int d, int heads, int dtype, void* X, float base,
            void* stream) {
  int st = check_rope(rows, seq_len, d, heads, dtype, base);
  if (st != ZO_OK) return st;
  if (rows == 0) return ZO_OK;
  ZO_CHECK(X && aligned(X, 16), "rope: X is NULL or not 16-byte aligned");
  return zo_rope_launch(rows, seq_len, d, heads, dtype, X, base, (hipStream_t)stream);
}

// kv_heads < 0: as many key/value heads as query heads (plain multi-head attention).
static int check_attention(int nblk, int T, int seq_len, int d, int heads, int dtype, int kv_heads = -1) {
  ZO_CHECK(nblk >= 1 && T >= 1 && seq_len >= 1 && T % seq_len == 0,
           "attention: nblk = %d, T = %d, seq_len = %d (need T %% seq_len == 0)", nblk, T, seq_len);
  ZO_CHECK(heads >= 1 && d % heads == 0, "attention: d = %d not a multiple of heads = %d", d, heads);
  if (kv_heads < 0) kv_heads = heads;
  ZO_CHECK(kv_heads >= 1 && heads % kv_heads == 0, "attention: heads = %d not a multiple of kv_heads = %d",
           heads, kv_heads);
  if (dtype != ZO_BF16 && dtype != ZO_F16) {
    zo_set_error("attention: dtype %d unsupported (bf16 or fp16)", dtype);
    return ZO_ERR_UNSUPPORTED;
  }
  const int dh = d / heads;
  if (dh != 64 && dh != 128) {
    zo_set_error("attention: head dim %d unsupported (64 or 128)", dh);
    return ZO_ERR_UNSUPPORTED;
  }
  ZO_CHECK((long long)nblk * T * d < (1LL << 40), "attention: tensors too large");
  return ZO_OK;
}

int zo_causal_attention(int nblk, int T, int seq_len, int d, int heads, int dtype, const void* Q,
                        const void* K, const void* V, void* O, void* stream) {
  int st = check_attention(nblk, T, seq_len, d, heads, dtype);
  if (st != ZO_OK) return st;
  ZO_CHECK(Q && K && V && O, "attention: NULL tensor argument");
  ZO_CHECK(aligned(Q, 16) && aligned(K, 16) && aligned(V, 16) && aligned(O, 16),
           "attention: Q, K, V, O must be 16-byte aligned");
  return zo_attention_launch(nblk, T, seq_len, d, heads, heads, dtype, Q, K, V, O, (hipStream_t)stream);
}

int zo_causal_attention_gqa(int nblk, int T, int seq_len, int d, int heads, int kv_heads, int dtype,
                            const void* Q, const void* K, const void* V, void* O, void* stream) {
  ZO_CHECK(kv_heads >= 1, "attention: kv_heads = %d must be >= 1", kv_heads);
  int st = check_attention(nblk, T, seq_len, d, heads, dtype, kv_heads);
  if (st != ZO_OK) return st;
  ZO_CHECK(Q && K && V && O, "attention: NULL tensor argument");
  ZO_CHECK(aligned(Q, 16) && aligned(K, 16) && aligned(V, 16) && aligned(O, 16),
           "attention: Q, K, V, O must be 16-byte aligned");
  return zo_attention_launch(nblk, T, seq_len, d, heads, kv_heads, dtype, Q, K, V, O, (hipStream_t)stream);
}

namespace {
struct DecoderWs {
  char *A, *Qb, *Kb, *Vb, *C, *H2, *F, *lin[3], *grp;
  size_t total;
};
// The largest perturbed-linear workspace of the layer's six matrices (the first layer's q, k, v
// read one shared input: their plans hold the fp32 base of the shared-X path).
static size_t decoder_lin_ws(int T, int d, int ffn, int r, int q, int nblk, int dtype) {
  const int shapes[3][2] = {{d, d}, {ffn, d}, {d, ffn}};
  size_t need = 0;
  for (const auto& sh : shapes) {
    for (const long long xs : {(long long)T * sh[1], 0LL}) {
      PlinearPlan p;
      zo_plinear_plan(&p, T, sh[0], sh[1], r, q, nblk, xs, dtype, dtype);
      need = p.ws_total > need ? p.ws_total : need;
    }
  }
  return need;
}
// The stacked projection of q, k, v (three matrices reading A, n = d).
static size_t decoder_grp_ws(int T, int d, int r, int q, int nblk, int dtype) {
  PlinearPlan p;
  zo_plinear_plan(&p, T, d, d, r, q, nblk, (long long)T * d, dtype, dtype);
  return zo_plinear_group_ws(p, 3);
}
static DecoderWs decoder_ws(int T, int d, int ffn, int r, int q, int nblk, int dtype, void* base) {
  const size_t es = dtype == ZO_F32 ? 4 : 2;
  const size_t act = zo_align256((size_t)nblk * T * d * es);
  WsCarver wc(base);
  DecoderWs w;
  w.A = (char*)wc.take(act);
  w.Qb = (char*)wc.take(act);
  w.Kb = (char*)wc.take(act);
  w.Vb = (char*)wc.take(act);
  w.C = (char*)wc.take(act);
  w.H2 = (char*)wc.take(act);
  w.F = (char*)wc.take((size_t)nblk * T * ffn * es);
  const size_t lin = decoder_lin_ws(T, d, ffn, r, q, nblk, dtype);
  for (auto& l : w.lin) l = (char*)wc.take(lin);
  w.grp = (char*)wc.take(decoder_grp_ws(T, d, r, q, nblk, dtype));
  w.total = wc.off;
  return w;
}
static int check_decoder(int T, int seq_len, int d, int heads, int ffn, int r, int q, int nblk, int dtype) {
  int st = check_attention(nblk, T, seq_len, d, heads, dtype);
  if (st != ZO_OK) return st;
  ZO_CHECK(ffn >= 8 && ffn % 8 == 0, "decoder: ffn = %d must be a positive multiple of 8", ffn);
  if ((st = check_plinear(T, d, d, r, q, nblk, (long long)T * d, dtype)) != ZO_OK) return st;
  if ((st = check_plinear(T, ffn, d, r, q, nblk, (long long)T * d, dtype)) != ZO_OK) return st;
  return check_plinear(T, d, ffn, r, q, nblk, (long long)T * ffn, dtype);
}
// Perturbed linears of one shape that read the same X: one stacked projection of X against
// all their V factors, then each one's fused GEMM in order (epilogue epi[i] with R[i], rs[i];
// a later one may read an earlier one's output as its R).
static int lin_group(int T, int m, int n, int r, int q, int nblk, long long xs, int dtype,
                     const int* blk_query, const int8_t* blk_sign, float eps, const void* X, int count,
                     const zo_matrix* const* mats, void* const* Y, const int* epi, const void* const* R,
                     const long long* rs, char* const* lin, void* grp, hipStream_t s) {
  PlinearPlan p[3];
  const float *U[3], *V[3], *Z[3];
  void* ws[3];
  for (int i = 0; i < count; ++i) {
    zo_plinear_plan(&p[i], T, m, n, r, q, nblk, xs, dtype, dtype);
    U[i] = mats[i]->U;
    V[i] = mats[i]->V;
    Z[i] = mats[i]->Z;
    ws[i] = lin[i];
  }
  int st = zo_plinear_prepare_group(p, count, blk_query, blk_sign, eps, X, U, V, Z, ws, grp, s);
  for (int i = 0; i < count && st == ZO_OK; ++i)
    st = zo_plinear_apply(p[i], X, mats[i]->W, Y[i], ws[i], s, epi[i], R[i], rs[i]);
  return st;
}
}  // namespace

size_t zo_decoder_layer_workspace(int T, int seq_len, int d, int heads, int ffn, int r, int q,
                                  int nblk, int dtype) {
  if (check_decoder(T, seq_len, d, heads, ffn, r, q, nblk, dtype) != ZO_OK) return 0;
  return decoder_ws(T, d, ffn, r, q, nblk, dtype, nullptr).total;
}

int zo_decoder_layer_forward(int T, int seq_len, int d, int heads, int ffn, int r, int q, int nblk,
                             const int* blk_query, const int8_t* blk_sign, float eps, float eps_ln,
                             int dtype, const void* H, long long h_block_stride,
                             const zo_decoder_layer* layer, void* H_out, void* workspace,
                             size_t ws_bytes, void* stream) {
  int st = check_decoder(T, seq_len, d, heads, ffn, r, q, nblk, dtype);
  if (st != ZO_OK) return st;
  ZO_CHECK(layer && H && H_out, "decoder: NULL argument (layer, H or H_out)");
  ZO_CHECK(h_block_stride == 0 || h_block_stride == (long long)T * d,
           "decoder: h_block_stride = %lld must be 0 (one H for every block) or T*d", h_block_stride);
  ZO_CHECK(isfinite(eps_ln) && eps_ln >= 0.f, "decoder: eps_ln must be finite and >= 0");
  const zo_matrix* mats[6] = {&layer->q, &layer->k, &layer->v, &layer->o, &layer->fc1, &layer->fc2};
  const char* names[6] = {"q", "k", "v", "o", "fc1", "fc2"};
  for (int i = 0; i < 6; ++i) {
    if ((st = check_blocks(q, nblk, blk_query, blk_sign, eps, mats[i]->U, mats[i]->V, mats[i]->Z)) != ZO_OK)
      return st;
    ZO_CHECK(mats[i]->W && aligned(mats[i]->W, 16), "decoder: %s W is NULL or not 16-byte aligned", names[i]);
  }
  ZO_CHECK(layer->ln1_gamma && layer->ln1_beta && layer->ln2_gamma && layer->ln2_beta,
           "decoder: NULL layer-norm parameter");
  ZO_CHECK(aligned(layer->ln1_gamma, 16) && aligned(layer->ln1_beta, 16) &&
               aligned(layer->ln2_gamma, 16) && aligned(layer->ln2_beta, 16),
           "decoder: layer-norm parameters must be 16-byte aligned");
  ZO_CHECK(aligned(H, 16) && aligned(H_out, 16), "decoder: H and H_out must be 16-byte aligned");
  const DecoderWs need = decoder_ws(T, d, ffn, r, q, nblk, dtype, nullptr);
  if (!workspace || ws_bytes < need.total) {
    zo_set_error("decoder: workspace %zu bytes < required %zu", ws_bytes, need.total);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "decoder: workspace not 256-byte aligned");
  const DecoderWs w = decoder_ws(T, d, ffn, r, q, nblk, dtype, workspace);
  hipStream_t s = (hipStream_t)stream;
  const long long Td = (long long)T * d, Tf = (long long)T * ffn;
  const bool shared = h_block_stride == 0;
  // One perturbed linear: prepare (X V, s eps U Z_j) then the fused GEMM.
  auto lin = [&](const zo_matrix* mt, int m, int n, const void* X, long long xs, void* Y, int epi,
                 const void* R, long long rs) -> int {
    PlinearPlan p;
    zo_plinear_plan(&p, T, m, n, r, q, nblk, xs, dtype, dtype);
    int e = zo_plinear_prepare(p, blk_query, blk_sign, eps, X, mt->U, mt->V, mt->Z, w.lin[0], s);
    if (e != ZO_OK) return e;
    return zo_plinear_apply(p, X, mt->W, Y, w.lin[0], s, epi, R, rs);
  };
  // A = LN1(H): once when every block shares H.
  if ((st = zo_layernorm_launch(shared ? T : (long long)nblk * T, d, dtype, H, layer->ln1_gamma,
                                layer->ln1_beta, eps_ln, w.A, s)) != ZO_OK)
    return st;
  const long long as = shared ? 0 : Td;
  // q, k, v read the same A: one stacked projection, then the three fused GEMMs.
  {
    const zo_matrix* const qkv[3] = {&layer->q, &layer->k, &layer->v};
    void* const out[3] = {w.Qb, w.Kb, w.Vb};
    const int epi[3] = {ZO_EPI_NONE, ZO_EPI_NONE, ZO_EPI_NONE};
    const void* const R[3] = {nullptr, nullptr, nullptr};
    const long long rs[3] = {0, 0, 0};
    if ((st = lin_group(T, d, d, r, q, nblk, as, dtype, blk_query, blk_sign, eps, w.A, 3, qkv, out, epi, R, rs,
                        w.lin, w.grp, s)) != ZO_OK)
      return st;
  }
  if ((st = zo_attention_launch(nblk, T, seq_len, d, heads, heads, dtype, w.Qb, w.Kb, w.Vb, w.C, s)) != ZO_OK)
    return st;
  // H2 = H + C Wo'^T;  A = LN2(H2);  F = relu(A W1'^T);  H_out = H2 + F W2'^T.
  if ((st = lin(&layer->o, d, d, w.C, Td, w.H2, ZO_EPI_RESIDUAL, H, h_block_stride)) != ZO_OK) return st;
  if ((st = zo_layernorm_launch((long long)nblk * T, d, dtype, w.H2, layer->ln2_gamma, layer->ln2_beta,
                                eps_ln, w.A, s)) != ZO_OK)
    return st;
  if ((st = lin(&layer->fc1, ffn, d, w.A, Td, w.F, ZO_EPI_RELU, nullptr, 0)) != ZO_OK) return st;
  return lin(&layer->fc2, d, ffn, w.F, Tf, H_out, ZO_EPI_RESIDUAL, w.H2, Td);
}

namespace {
struct LlamaWs {
  char *A, *Qb, *Kb, *Vb, *C, *H2, *G, *F, *lin[3], *grp;
  size_t total;
};
// The largest perturbed-linear workspace of the layer's seven matrices (d x d, ffn x d, d x ffn).
static LlamaWs llama_ws(int T, int d, int ffn, int r, int q, int nblk, int dtype, void* base) {
  const size_t es = dtype == ZO_F32 ? 4 : 2;
  const size_t act = zo_align256((size_t)nblk * T * d * es);
  const size_t wide = zo_align256((size_t)nblk * T * ffn * es);
  WsCarver wc(base);
  LlamaWs w;
  w.A = (char*)wc.take(act);
  w.Qb = (char*)wc.take(act);
  w.Kb = (char*)wc.take(act);
  w.Vb = (char*)wc.take(act);
  w.C = (char*)wc.take(act);
  w.H2 = (char*)wc.take(act);
  w.G = (char*)wc.take(wide);
  w.F = (char*)wc.take(wide);
  const size_t lin = decoder_lin_ws(T, d, ffn, r, q, nblk, dtype);
  for (auto& l : w.lin) l = (char*)wc.take(lin);
  w.grp = (char*)wc.take(decoder_grp_ws(T, d, r, q, nblk, dtype));  // q, k, v (gate, up need less)
  w.total = wc.off;
  return w;
}
}  // namespace

size_t zo_llama_layer_workspace(int T, int seq_len, int d, int heads, int ffn, int r, int q, int nblk,
                                int dtype) {
  if (check_decoder(T, seq_len, d, heads, ffn, r, q, nblk, dtype) != ZO_OK) return 0;
  if (check_rope((long long)nblk * T, seq_len, d, heads, dtype, 10000.f) != ZO_OK) return 0;
  return llama_ws(T, d, ffn, r, q, nblk, dtype, nullptr).total;
}

int zo_llama_layer_forward(int T, int seq_len, int d, int heads, int ffn, int r, int q, int nblk,
                           const int* blk_query, const int8_t* blk_sign, float eps, float eps_rms,
                           float rope_base, int dtype, const void* H, long long h_block_stride,
                           const zo_llama_layer* layer, void* H_out, void* workspace, size_t ws_bytes,
                           void* stream) {
  int st = check_decoder(T, seq_len, d, heads, ffn, r, q, nblk, dtype);
  if (st != ZO_OK) return st;
  if ((st = check_rope((long long)nblk * T, seq_len, d, heads, dtype, rope_base)) != ZO_OK) return st;
  ZO_CHECK(layer && H && H_out, "llama: NULL argument (layer, H or H_out)");
  ZO_CHECK(h_block_stride == 0 || h_block_stride == (long long)T * d,
           "llama: h_block_stride = %lld must be 0 (one H for every block) or T*d", h_block_stride);
  ZO_CHECK(isfinite(eps_rms) && eps_rms >= 0.f, "llama: eps_rms must be finite and >= 0");
  const zo_matrix* mats[7] = {&layer->q, &layer->k, &layer->v, &layer->o, &layer->gate, &layer->up, &layer->down};
  const char* names[7] = {"q", "k", "v", "o", "gate", "up", "down"};
  for (int i = 0; i < 7; ++i) {
    if ((st = check_blocks(q, nblk, blk_query, blk_sign, eps, mats[i]->U, mats[i]->V, mats[i]->Z)) != ZO_OK)
      return st;
    ZO_CHECK(mats[i]->W && aligned(mats[i]->W, 16), "llama: %s W is NULL or not 16-byte aligned", names[i]);
  }
  ZO_CHECK(layer->rms1_gamma && layer->rms2_gamma, "llama: NULL RMS-norm parameter");
  ZO_CHECK(aligned(layer->rms1_gamma, 16) && aligned(layer->rms2_gamma, 16),
           "llama: RMS-norm parameters must be 16-byte aligned");
  ZO_CHECK(aligned(H, 16) && aligned(H_out, 16), "llama: H and H_out must be 16-byte aligned");
  const LlamaWs need = llama_ws(T, d, ffn, r, q, nblk, dtype, nullptr);
  if (!workspace || ws_bytes < need.total) {
    zo_set_error("llama: workspace %zu bytes < required %zu", ws_bytes, need.total);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "llama: workspace not 256-byte aligned");
  const LlamaWs w = llama_ws(T, d, ffn, r, q, nblk, dtype, workspace);
  hipStream_t s = (hipStream_t)stream;
  const long long Td = (long long)T * d, Tf = (long long)T * ffn;
  const long long rows = (long long)nblk * T;
  const bool shared = h_block_stride == 0;
  auto lin = [&](const zo_matrix* mt, int m, int n, const void* X, long long xs, void* Y, int epi,
                 const void* R, long long rs) -> int {
    PlinearPlan p;
    zo_plinear_plan(&p, T, m, n, r, q, nblk, xs, dtype, dtype);
    int e = zo_plinear_prepare(p, blk_query, blk_sign, eps, X, mt->U, mt->V, mt->Z, w.lin[0], s);
    if (e != ZO_OK) return e;
    return zo_plinear_apply(p, X, mt->W, Y, w.lin[0], s, epi, R, rs);
  };
  // A = RMS1(H): once when every block shares H.
  if ((st = zo_layernorm_launch(shared ? T : rows, d, dtype, H, layer->rms1_gamma, nullptr, eps_rms, w.A, s,
                                true)) != ZO_OK)
    return st;
  const long long as = shared ? 0 : Td;
  // q, k, v read the same A: one stacked projection, then the three fused GEMMs.
  {
    const zo_matrix* const qkv[3] = {&layer->q, &layer->k, &layer->v};
    void* const out[3] = {w.Qb, w.Kb, w.Vb};
    const int epi[3] = {ZO_EPI_NONE, ZO_EPI_NONE, ZO_EPI_NONE};
    const void* const R[3] = {nullptr, nullptr, nullptr};
    const long long rs[3] = {0, 0, 0};
    if ((st = lin_group(T, d, d, r, q, nblk, as, dtype, blk_query, blk_sign, eps, w.A, 3, qkv, out, epi, R, rs,
                        w.lin, w.grp, s)) != ZO_OK)
      return st;
  }
  if ((st = zo_rope_launch(rows, seq_len, d, heads, dtype, w.Qb, rope_base, s)) != ZO_OK) return st;
  if ((st = zo_rope_launch(rows, seq_len, d, heads, dtype, w.Kb, rope_base, s)) != ZO_OK) return st;
  if ((st = zo_attention_launch(nblk, T, seq_len, d, heads, heads, dtype, w.Qb, w.Kb, w.Vb, w.C, s)) != ZO_OK)
    return st;
  // H2 = H + C Wo'^T;  A = RMS2(H2);  G = A Wg'^T;  F = silu(G) * (A Wu'^T);  H_out = H2 + F Wd'^T.
  if ((st = lin(&layer->o, d, d, w.C, Td, w.H2, ZO_EPI_RESIDUAL, H, h_block_stride)) != ZO_OK) return st;
  if ((st = zo_layernorm_launch(rows, d, dtype, w.H2, layer->rms2_gamma, nullptr, eps_rms, w.A, s, true)) != ZO_OK)
    return st;
  {  // gate and up read the same A: one stacked projection; F = silu(G) * (A Wu'^T)
    const zo_matrix* const gu[2] = {&layer->gate, &layer->up};
    void* const out[2] = {w.G, w.F};
    const int epi[2] = {ZO_EPI_NONE, ZO_EPI_SILU_MUL};
    const void* const R[2] = {nullptr, w.G};
    const long long rs[2] = {0, Tf};
    if ((st = lin_group(T, ffn, d, r, q, nblk, Td, dtype, blk_query, blk_sign, eps, w.A, 2, gu, out, epi, R, rs,
                        w.lin, w.grp, s)) != ZO_OK)
      return st;
  }
  return lin(&layer->down, d, ffn, w.F, Tf, H_out, ZO_EPI_RESIDUAL, w.H2, Td);
}

// ------------------------------------------------------- LoRA-scheme LLaMA-family layer
namespace {
struct LoraLayerWs {
  char *A, *Qb, *Kb, *Vb, *C, *H2, *G, *F, *lin;
  size_t total;
};
static LoraLayerWs lora_layer_ws(int T, int d, int dkv, int ffn, int rl, int r, int q, int nblk, int dtype,
                                 void* base) {
  const size_t es = 2;
  const size_t act = zo_align256((size_t)nblk * T * d * es), kv = zo_align256((size_t)nblk * T * dkv * es);
  const size_t wide = zo_align256((size_t)nblk * T * ffn * es);
  size_t lin = 0;
  for (int m : {d, dkv}) {
    for (const long long xs : {(long long)T * d, 0LL}) {  // per-block or shared input
      PlinearPlan p;
      zo_plinear_plan(&p, T, m, d, rl + r, q, nblk, xs, dtype, dtype);
      lin = p.ws_total > lin ? p.ws_total : lin;
    }
  }
  WsCarver wc(base);
  LoraLayerWs w;
  w.A = (char*)wc.take(act);
  w.Qb = (char*)wc.take(act);
  w.Kb = (char*)wc.take(kv);
  w.Vb = (char*)wc.take(kv);
  w.C = (char*)wc.take(act);
  w.H2 = (char*)wc.take(act);
  w.G = (char*)wc.take(wide);
  w.F = (char*)wc.take(wide);
  w.lin = (char*)wc.take(lin);
  w.total = wc.off;
  return w;
}
static int check_lora_layer(int T, int seq_len, int d, int heads, int kv_heads, int ffn, int rl, int r, int q,
                            int nblk, int dtype) {
  ZO_CHECK(kv_heads >= 1, "lora layer: kv_heads = %d must be >= 1", kv_heads);
  int st = check_attention(nblk, T, seq_len, d, heads, dtype, kv_heads);
  if (st != ZO_OK) return st;
  const int dkv = d / heads * kv_heads;
  ZO_CHECK(ffn >= 8 && ffn % 8 == 0, "lora layer: ffn = %d must be a positive multiple of 8", ffn);
  if ((st = check_lora(T, d, d, rl, r, q, nblk, (long long)T * d, dtype)) != ZO_OK) return st;
  if ((st = check_lora(T, dkv, d, rl, r, q, nblk, (long long)T * d, dtype)) != ZO_OK) return st;
  if ((st = check_plinear(T, ffn, d, 1, q, nblk, (long long)T * d, dtype)) != ZO_OK) return st;
  return check_plinear(T, d, ffn, 1, q, nblk, (long long)T * ffn, dtype);
}
}  // namespace

size_t zo_llama_lora_layer_workspace(int T, int seq_len, int d, int heads, int kv_heads, int ffn, int rl,
                                     int r, int q, int nblk, int dtype) {
  if (check_lora_layer(T, seq_len, d, heads, kv_heads, ffn, rl, r, q, nblk, dtype) != ZO_OK) return 0;
  if (check_rope((long long)nblk * T, seq_len, d, heads, dtype, 1e6f) != ZO_OK) return 0;
  return lora_layer_ws(T, d, d / heads * kv_heads, ffn, rl, r, q, nblk, dtype, nullptr).total;
}

int zo_llama_lora_layer_forward(int T, int seq_len, int d, int heads, int kv_heads, int ffn, int rl, int r,
                                int q, int nblk, const int* blk_query, const int8_t* blk_sign, float eps,
                                float scale, float eps_rms, float rope_base, int dtype, const void* H,
                                long long h_block_stride, const zo_llama_lora_layer* layer, void* H_out,
                                void* workspace, size_t ws_bytes, void* stream) {
  int st = check_lora_layer(T, seq_len, d, heads, kv_heads, ffn, rl, r, q, nblk, dtype);
  if (st != ZO_OK) return st;
  const int dkv = d / heads * kv_heads;
  if ((st = check_rope((long long)nblk * T, seq_len, d, heads, dtype, rope_base)) != ZO_OK) return st;
  ZO_CHECK(layer && H && H_out, "lora layer: NULL argument (layer, H or H_out)");
  ZO_CHECK(h_block_stride == 0 || h_block_stride == (long long)T * d,
           "lora layer: h_block_stride = %lld must be 0 (one H for every block) or T*d", h_block_stride);
  ZO_CHECK(isfinite(eps_rms) && eps_rms >= 0.f, "lora layer: eps_rms must be finite and >= 0");
  const zo_lora_matrix* ad[2] = {&layer->q, &layer->v};
  for (int i = 0; i < 2; ++i) {
    if ((st = check_lora_factors(q, nblk, blk_query, blk_sign, eps, scale, ad[i]->A, ad[i]->U_A, ad[i]->V_A,
                                 ad[i]->Z_A, ad[i]->B, ad[i]->U_B, ad[i]->V_B, ad[i]->Z_B)) != ZO_OK)
      return st;
    ZO_CHECK(ad[i]->W && aligned(ad[i]->W, 16), "lora layer: %s W is NULL or not 16-byte aligned",
             i ? "v" : "q");
  }
  const void* frozen[5] = {layer->k, layer->o, layer->gate, layer->up, layer->down};
  for (int i = 0; i < 5; ++i)
    ZO_CHECK(frozen[i] && aligned(frozen[i], 16), "lora layer: a frozen weight is NULL or not 16-byte aligned");
  ZO_CHECK(layer->rms1_gamma && layer->rms2_gamma && aligned(layer->rms1_gamma, 16) &&
               aligned(layer->rms2_gamma, 16),
           "lora layer: RMS-norm parameters NULL or not 16-byte aligned");
  ZO_CHECK(aligned(H, 16) && aligned(H_out, 16), "lora layer: H and H_out must be 16-byte aligned");
  const LoraLayerWs need = lora_layer_ws(T, d, dkv, ffn, rl, r, q, nblk, dtype, nullptr);
  if (!workspace || ws_bytes < need.total) {
    zo_set_error("lora layer: workspace %zu bytes < required %zu", ws_bytes, need.total);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "lora layer: workspace not 256-byte aligned");
  const LoraLayerWs w = lora_layer_ws(T, d, dkv, ffn, rl, r, q, nblk, dtype, workspace);
  hipStream_t s = (hipStream_t)stream;
  const long long Td = (long long)T * d, Tf = (long long)T * ffn;
  const long long rows = (long long)nblk * T;
  const bool shared = h_block_stride == 0;
  const long long as = shared ? 0 : Td;
  // An adapted matrix: both factors perturbed (X_b [A^T | V_A] times scale [B' | s eps B' U_A Z_A]).
  auto lora = [&](const zo_lora_matrix* mt, int m, void* Y) -> int {
    PlinearPlan p;
    zo_plinear_plan(&p, T, m, d, rl + r, q, nblk, as, dtype, dtype);
    int e = zo_lora_prepare(p, rl, r, blk_query, blk_sign, eps, scale, w.A, mt->A, mt->U_A, mt->V_A, mt->Z_A,
                            mt->B, mt->U_B, mt->V_B, mt->Z_B, w.lin, s);
    if (e != ZO_OK) return e;
    return zo_plinear_apply(p, w.A, mt->W, Y, w.lin, s);
  };
  // A = RMS1(H): once when every block shares H.
  if ((st = zo_layernorm_launch(shared ? T : rows, d, dtype, H, layer->rms1_gamma, nullptr, eps_rms, w.A, s,
                                true)) != ZO_OK)
    return st;
  if ((st = lora(&layer->q, d, w.Qb)) != ZO_OK) return st;
  if ((st = zo_gemm_plain(T, dkv, d, nblk, dtype, w.A, as, layer->k, w.Kb, ZO_EPI_NONE, nullptr, 0, s)) != ZO_OK)
    return st;
  if ((st = lora(&layer->v, dkv, w.Vb)) != ZO_OK) return st;
  if ((st = zo_rope_launch(rows, seq_len, d, heads, dtype, w.Qb, rope_base, s)) != ZO_OK) return st;
  if ((st = zo_rope_launch(rows, seq_len, dkv, kv_heads, dtype, w.Kb, rope_base, s)) != ZO_OK) return st;
  if ((st = zo_attention_launch(nblk, T, seq_len, d, heads, kv_heads, dtype, w.Qb, w.Kb, w.Vb, w.C, s)) != ZO_OK)
    return st;
  // H2 = H + C Wo^T;  A = RMS2(H2);  G = A Wg^T;  F = silu(G) * (A Wu^T);  H_out = H2 + F Wd^T.
  if ((st = zo_gemm_plain(T, d, d, nblk, dtype, w.C, Td, layer->o, w.H2, ZO_EPI_RESIDUAL, H, h_block_stride, s)) !=
      ZO_OK)
    return st;
  if ((st = zo_layernorm_launch(rows, d, dtype, w.H2, layer->rms2_gamma, nullptr, eps_rms, w.A, s, true)) != ZO_OK)
    return st;
  if ((st = zo_gemm_plain(T, ffn, d, nblk, dtype, w.A, Td, layer->gate, w.G, ZO_EPI_NONE, nullptr, 0, s)) != ZO_OK)
    return st;
  if ((st = zo_gemm_plain(T, ffn, d, nblk, dtype, w.A, Td, layer->up, w.F, ZO_EPI_SILU_MUL, w.G, Tf, s)) != ZO_OK)
    return st;
  return zo_gemm_plain(T, d, ffn, nblk, dtype, w.F, Tf, layer->down, H_out, ZO_EPI_RESIDUAL, w.H2, Td, s);
}

// ------------------------------------------------------------------ update
static int check_update(int count, const zo_update_item* items, int r, int q, int w_dtype,
                        bool moments = true) {
  ZO_CHECK(count >= 0, "update: count = %d < 0", count);
  ZO_CHECK(count == 0 || items, "update: items is NULL");
  ZO_CHECK(r >= 1 && r <= ZO_MAX_RANK, "update: r = %d outside [1, %d]", r, ZO_MAX_RANK);
  ZO_CHECK(q >= 1 && q <= ZO_MAX_QUERIES, "update: q = %d outside [1, %d]", q, ZO_MAX_QUERIES);
  ZO_CHECK(w_dtype == ZO_F32 || w_dtype == ZO_BF16 || w_dtype == ZO_F16, "update: bad w_dtype %d",
           w_dtype);
  for (int i = 0; i < count; ++i) {
    const zo_update_item& it = items[i];
    ZO_CHECK(it.m >= 1 && it.n >= 1, "update: item %d has m = %d, n = %d", i, it.m, it.n);
    ZO_CHECK((long long)it.m * it.n < (1LL << 40), "update: item %d too large", i);
    ZO_CHECK(it.W && it.U && it.V && it.Z, "update: item %d has a NULL tensor", i);
    ZO_CHECK(!moments || (it.M1 && it.M2), "update: item %d has a NULL moment", i);
    if (w_dtype != ZO_F32) {
      ZO_CHECK(it.n % 8 == 0, "update: 16-bit W needs n %% 8 == 0 (item %d, n = %d)", i, it.n);
      ZO_CHECK(it.n <= (1 << 20), "update: 16-bit W needs n <= %d (item %d, n = %d)", 1 << 20, i,
               it.n);
      ZO_CHECK(aligned(it.W, 16) && aligned(it.w_f32_out, 16),
               "update: item %d W / w_f32_out not 16-byte aligned", i);
      ZO_CHECK((long long)((it.m + 127) / 128) * ((it.n + 255) / 256) < (1LL << 30),
               "update: item %d too large", i);
    } else {
      ZO_CHECK(aligned(it.W, 4) && aligned(it.w_f32_out, 4), "update: item %d alignment", i);
      ZO_CHECK((long long)it.m * it.n < (1LL << 38), "update: item %d too large", i);
    }
  }
  return ZO_OK;
}

size_t zo_subspace_adam_update_workspace(int count, const zo_update_item* items, int r, int q,
                                         int w_dtype) {
  if (check_update(count, items, r, q, w_dtype) != ZO_OK) return 0;
  size_t need = 0;
  zo_update_launch(count, items, w_dtype, r, q, nullptr, 1, 0.f, 0.f, 0.f, 0.f, 0, nullptr,
                   nullptr, 0, nullptr, &need);
  return need;
}

int zo_subspace_adam_update(int count, const zo_update_item* items, int w_dtype, int r, int q,
                            const float* g, int t, float lr, float beta1, float beta2,
                            float eps_adam, int* nonfinite_flag, void* workspace, size_t ws_bytes,
                            void* stream) {
  int st = check_update(count, items, r, q, w_dtype);
  if (st != ZO_OK) return st;
  ZO_CHECK(g, "update: g is NULL");
  ZO_CHECK(t >= 1, "update: Adam step t = %d must be >= 1", t);
  ZO_CHECK(isfinite(lr), "update: lr is not finite");
  ZO_CHECK(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f,
           "update: betas must lie in [0, 1)");
  ZO_CHECK(eps_adam >= 0.f && isfinite(eps_adam), "update: eps_adam must be finite and >= 0");
  if (count == 0) return ZO_OK;
  size_t need = 0;
  zo_update_launch(count, items, w_dtype, r, q, nullptr, 1, 0.f, 0.f, 0.f, 0.f, 0, nullptr,
                   nullptr, 0, nullptr, &need);
  if (ws_bytes < need || !workspace) {
    zo_set_error("update: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "update: workspace not 256-byte aligned");
  return zo_update_launch(count, items, w_dtype, r, q, g, t, lr, beta1, beta2, eps_adam, 0,
                          nonfinite_flag, workspace, ws_bytes, (hipStream_t)stream, nullptr);
}

size_t zo_subspace_sgd_update_workspace(int count, const zo_update_item* items, int r, int q,
                                        int w_dtype) {
  if (check_update(count, items, r, q, w_dtype, false) != ZO_OK) return 0;
  size_t need = 0;
  zo_update_launch(count, items, w_dtype, r, q, nullptr, 1, 0.f, 0.f, 0.f, 0.f, 1, nullptr,
                   nullptr, 0, nullptr, &need);
  return need;
}

int zo_subspace_sgd_update(int count, const zo_update_item* items, int w_dtype, int r, int q,
                           const float* g, float lr, int* nonfinite_flag, void* workspace,
                           size_t ws_bytes, void* stream) {
  int st = check_update(count, items, r, q, w_dtype, false);
  if (st != ZO_OK) return st;
  ZO_CHECK(g, "update: g is NULL");
  ZO_CHECK(isfinite(lr), "update: lr is not finite");
  if (count == 0) return ZO_OK;
  size_t need = 0;
  zo_update_launch(count, items, w_dtype, r, q, nullptr, 1, 0.f, 0.f, 0.f, 0.f, 1, nullptr,
                   nullptr, 0, nullptr, &need);
  if (ws_bytes < need || !workspace) {
    zo_set_error("update: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  ZO_CHECK(aligned(workspace, 256), "update: workspace not 256-byte aligned");
  return zo_update_launch(count, items, w_dtype, r, q, g, 1, lr, 0.f, 0.f, 0.f, 1,
                          nonfinite_flag, workspace, ws_bytes, (hipStream_t)stream, nullptr);
}

// ------------------------------------------------------------------- losses
size_t zo_sq_loss_workspace(int nblk, int T, int m) {
  if (nblk < 1 || T < 1 || m < 1) return 0;
  size_t need = 0;
  zo_sq_loss_launch(nblk, T, m, ZO_F32, nullptr, nullptr, nullptr, nullptr, 0, nullptr, &need);
  return need;
}

int zo_sq_loss(int nblk, int T, int m, int dtype, const void* Y, const void* Ystar, double* out,
               void* workspace, size_t ws_bytes, void* stream) {
  ZO_CHECK(nblk >= 1 && T >= 1 && m >= 1, "sq_loss: nblk, T, m must be >= 1");
  ZO_CHECK(nblk <= 65535, "sq_loss: nblk = %d too large", nblk);
  ZO_CHECK(dtype == ZO_F32 || dtype == ZO_BF16 || dtype == ZO_F16, "sq_loss: bad dtype %d", dtype);
  ZO_CHECK(Y && Ystar && out, "sq_loss: NULL tensor argument");
  size_t need = 0;
  zo_sq_loss_launch(nblk, T, m, dtype, nullptr, nullptr, nullptr, nullptr, 0, nullptr, &need);
  if (ws_bytes < need || !workspace) {
    zo_set_error("sq_loss: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  return zo_sq_loss_launch(nblk, T, m, dtype, Y, Ystar, out, workspace, ws_bytes,
                           (hipStream_t)stream, nullptr);
}

int zo_combine_central(int q, const double* L, float eps, float* g, void* stream) {
  ZO_CHECK(q >= 1, "combine_central: q = %d < 1", q);
  ZO_CHECK(L && g, "combine_central: NULL tensor argument");
  ZO_CHECK(isfinite(eps) && eps != 0.f, "combine_central: eps must be finite and non-zero");
  return zo_combine_central_launch(q, L, eps, g, (hipStream_t)stream);
}

int zo_combine_forward(int q, const double* L, float eps, float* g, void* stream) {
  ZO_CHECK(q >= 1, "combine_forward: q = %d < 1", q);
  ZO_CHECK(L && g, "combine_forward: NULL tensor argument");
  ZO_CHECK(isfinite(eps) && eps != 0.f, "combine_forward: eps must be finite and non-zero");
  return zo_combine_forward_launch(q, L, eps, g, (hipStream_t)stream);
}

}  // extern "C"

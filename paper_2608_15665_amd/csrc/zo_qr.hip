// Subspace refresh of SubZero+: Haar-distributed factor of a Gaussian panel
// (Eq. 11, Alg. 1) -- thin QR with each column of Q multiplied by the sign of
// the matching diagonal entry of R, so the corrected R has diag(R) > 0.
//
// That corrected factor is the unique Q with Q^T Q = I and Omega = Q R,
// diag(R) > 0.  It is computed here by CholeskyQR2 in float64 (Fukaya,
// Nakatsukasa, Yanagisawa, Yamamoto, 2014): R1 = chol(Omega^T Omega),
// Q1 = Omega R1^-1, R2 = chol(Q1^T Q1), Q = Q1 R2^-1, R = R2 R1.  A Cholesky
// factor has a positive diagonal, so the sign correction is built in.  The
// second pass restores orthogonality to working precision.  What limits the
// method is a pivot of the first factorisation sinking into the rounding noise
// of the Gram matrix, which takes a column within ~1e-8 of the span of the
// earlier ones (column scaling alone does not: the relative pivots are scale
// free).  Gaussian panels, whose condition number is about
// (sqrt(rows) + sqrt(r)) / (sqrt(rows) - sqrt(r)), essentially never get there.
//
// Five launches per call, each over every panel of the call (the panel
// descriptors sit in a table in the workspace, written by k_cqr_fill; a row
// launch's workgroup finds its panel by binary search over the table), all
// float64 with fixed-order sums (the result is bitwise reproducible):
//   k_cqr_rows<0>  per chunk of CHUNK rows: partial Omega^T Omega
//   k_cqr_chol     per panel: sum of the partials, Cholesky -> R1, and
//                  X1 = R1^-1 (rows of the identity through forward substitution)
//   k_cqr_rows<1>  per chunk: Q1 = Omega X1, partial Q1^T Q1
//   k_cqr_chol     per panel: R2, X2 = R2^-1, M = X1 X2; diag(R) = diag(R2) diag(R1); info
//   k_cqr_rows<2>  per chunk: Q = Omega M, written as fp32
// The row passes (r <= 64) run on v_mfma_f64_16x16x4_f64, each wave on its own
// quarter of the chunk: the Gram matrix as sums of 4-row outer products over
// its upper 16 x 16 tiles, the products 16 rows at a time.  The product's
// output registers are, lane for lane, the operands of the Gram MFMAs of its
// rows (output lane l, register v holds row 4 v + l / 16, column l % 16, the
// layout an operand's k = l / 16, i = l % 16 asks for), so Q1 never leaves the
// registers.  The four waves' partial Gram matrices are added in wave order.
// A pivot that is not positive marks the panel rank deficient at that column
// (an exactly zero column gives a zero pivot): R's row there is zero, the Q
// column is zero, and the other columns are formed as if it were absent.
#include "zo_internal.h"

#include <algorithm>
#include <mutex>
#include <vector>

namespace {

constexpr int CHUNK = 2048;       // rows per workgroup of the r <= 64 path (CHUNK / 4 per wave)
constexpr int WROWS = CHUNK / 4;
constexpr int BIG_CHUNK = 1024;   // rows per workgroup of the r > 64 path
constexpr int FILL_PANELS = 48;   // descriptors per k_cqr_fill launch (kernel arguments)

typedef double f64x4 __attribute__((ext_vector_type(4)));

struct CqrPanel {
  const float* omega;
  float* q;
  float* r_diag;
  int* info;
  double* part;  // partial Gram matrices, one RP x RP per chunk
  double* R1;    // RP x RP: R1 (its diagonal is needed at the end)
  double* X1;    // RP x RP: R1^-1
  double* M;     // RP x RP: R1^-1 R2^-1
  int rows, chunk_begin;
};
struct CqrArgs {
  const CqrPanel* p;  // the call's descriptor table (workspace)
  int count, r;
};
struct CqrFill {
  CqrPanel p[FILL_PANELS];
  CqrPanel* dst;
  int n;
};

// Copies n host descriptors (kernel arguments) into the table, one 32-bit word per thread.
__global__ __launch_bounds__(256) void k_cqr_fill(CqrFill f) {
  constexpr int W = (int)(sizeof(CqrPanel) / 4);
  static_assert(sizeof(CqrPanel) % 4 == 0, "descriptor of whole words");
  const int x = blockIdx.x * 256 + threadIdx.x;
  if (x < f.n * W) ((uint32_t*)f.dst)[x] = ((const uint32_t*)f.p)[x];
}

// The panel that row workgroup wg belongs to: the last k with chunk_begin <= wg
// (chunk_begin is non-decreasing from 0; a panel without rows has no chunks).
__device__ __forceinline__ int find_panel(const CqrArgs& a, int wg) {
  int lo = 0, hi = a.count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.p[mid].chunk_begin <= wg) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ f64x4 mfma64(double a, double b, f64x4 c) {
  return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// PASS 0: partial Omega^T Omega of this chunk.  PASS 1: partial Q1^T Q1 with
// Q1 = Omega X1.  PASS 2: Q = Omega M written as fp32.  Entries outside the
// panel's rows x r read as zero.  A Gram tile (ta <= tb) accumulates, per
// 4-row step, the MFMA of the rows' columns 16 ta + i (A) and 16 tb + j (B):
// lane l brings row base + l / 16, column 16 t + l % 16 as the operand of
// tile t.  A product 16 rows x RP takes the row's columns in K steps of 4:
// step kk, lane l multiplies column c = (l / 16) KS + kk of row base + l % 16
// with Mx row c (any one-to-one map of (step, lane group) to columns sums the
// same terms).
template <int RK, int PASS>
__global__ __launch_bounds__(256) void k_cqr_rows(CqrArgs a) {
  constexpr int RP = 16 * RK, KS = RP / 4, NPAIR = RK * (RK + 1) / 2;
  __shared__ double Mx[PASS == 0 ? 1 : RP * RP];
  __shared__ double red[PASS == 2 ? 1 : NPAIR * 256];
  const CqrPanel P = a.p[find_panel(a, blockIdx.x)];
  const int chunk = blockIdx.x - P.chunk_begin;
  const int r = a.r, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  if (PASS >= 1) {
    const double* src = PASS == 1 ? P.X1 : P.M;
    for (int x = tid; x < RP * RP; x += 256) Mx[x] = src[x];
    __syncthreads();
  }
  const int row0 = chunk * CHUNK + wave * WROWS;
  const int nrow = min(WROWS, P.rows - row0);  // this wave's rows (none past the end)
  // Omega entries as loaded (fp32, zero outside the panel); widened to float64 at use (exact).
  auto om = [&](int row, int col) -> float {
    return (row < P.rows && col < r) ? P.omega[(size_t)row * r + col] : 0.f;
  };
  f64x4 acc[NPAIR];
#pragma unroll
  for (int p = 0; p < NPAIR; ++p) acc[p] = (f64x4){0.0, 0.0, 0.0, 0.0};
  // The Gram tiles over 4 rows whose tile-t operands are v[t].
  auto gram = [&](const double* v) {
    int p = 0;
#pragma unroll
    for (int ta = 0; ta < RK; ++ta)
#pragma unroll
      for (int tb = ta; tb < RK; ++tb, ++p) acc[p] = mfma64(v[ta], v[tb], acc[p]);
  };
  if (PASS == 0) {
    // 32 rows per step (eight 4-row Gram steps), the next step's loads issued before the MFMAs.
    float nx[8][RK];
    auto load = [&](int s) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int t = 0; t < RK; ++t) nx[u][t] = om(row0 + s + 4 * u + g, 16 * t + l16);
    };
    if (nrow > 0) load(0);
    for (int s = 0; s < nrow; s += 32) {
      float cur[8][RK];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int t = 0; t < RK; ++t) cur[u][t] = nx[u][t];
      if (s + 32 < nrow) load(s + 32);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        double v[RK];
#pragma unroll
        for (int t = 0; t < RK; ++t) v[t] = (double)cur[u][t];
        gram(v);
      }
    }
  } else {
    float nx[KS];
    auto load = [&](int s) {
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) nx[kk] = om(row0 + s + l16, g * KS + kk);
    };
    if (nrow > 0) load(0);
    for (int s = 0; s < nrow; s += 16) {
      float av[KS];
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) av[kk] = nx[kk];
      if (s + 16 < nrow) load(s + 16);
      // The RK product chains interleaved (each still sums its K steps in order).
      f64x4 q[RK];
#pragma unroll
      for (int t = 0; t < RK; ++t) q[t] = (f64x4){0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const double x = (double)av[kk];
#pragma unroll
        for (int t = 0; t < RK; ++t) q[t] = mfma64(x, Mx[(g * KS + kk) * RP + 16 * t + l16], q[t]);
      }
      // q[t][v]: row row0 + s + 4 v + g, column 16 t + l16.
      if (PASS == 1) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          double w[RK];
#pragma unroll
          for (int t = 0; t < RK; ++t) w[t] = q[t][v];
          gram(w);
        }
      } else {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = row0 + s + 4 * v + g;
          if (row >= P.rows) continue;
#pragma unroll
          for (int t = 0; t < RK; ++t)
            if (16 * t + l16 < r) P.q[(size_t)row * r + 16 * t + l16] = (float)q[t][v];
        }
      }
    }
  }
  if (PASS == 2) return;
  // The waves' partials added in wave order, then written as the chunk's upper tiles.
  for (int w = 0; w < 4; ++w) {
    if (wave == w) {
#pragma unroll
      for (int p = 0; p < NPAIR; ++p)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          double& d = red[p * 256 + v * 64 + lane];
          d = w == 0 ? acc[p][v] : d + acc[p][v];
        }
    }
    __syncthreads();
  }
  double* out = P.part + (size_t)chunk * RP * RP;
  for (int x = tid; x < NPAIR * 256; x += 256) {
    int p = x >> 8, ta = 0;
    while (p >= RK - ta) { p -= RK - ta; ++ta; }
    const int tb = ta + p, v = (x >> 6) & 3, l = x & 63;
    out[(size_t)(16 * ta + 4 * v + (l >> 4)) * RP + 16 * tb + (l & 15)] = red[x];
  }
}

// Sum of the chunk partials (upper triangle, chunk order) and the Cholesky
// factor G = R^T R, row by row: R_kk = sqrt(G_kk - sum_{i<k} R_ik^2),
// R_kj = (G_kj - sum_{i<k} R_ik R_ij) / R_kk (a pivot that is not positive
// gives a zero row).  Then X = R^-1 row by row: row i of X is e_i pushed
// through the forward substitution x_j = (x_j - sum_{l<j} x_l R_lj) / R_jj
// (zero where R_jj = 0), so Omega X is exactly that substitution applied to
// Omega's rows.  FINAL: this is R2; M = X1 X2, diag(R) = diag(R2) diag(R1), info.
template <int RK, bool FINAL>
__global__ __launch_bounds__(256) void k_cqr_chol(CqrArgs a) {
  constexpr int RP = 16 * RK;
  __shared__ double G[RP * RP];
  __shared__ double X[RP * RP];
  __shared__ double X1s[FINAL ? RP * RP : 1];
  __shared__ double inv[RP];
  const CqrPanel& P = a.p[blockIdx.x];
  const int r = a.r, tid = threadIdx.x;
  const int nchunk = (P.rows + CHUNK - 1) / CHUNK;
  // Entry x = tid + 256 e of G: the chunks' partials added in chunk order, the loads of one
  // chunk for all of a thread's entries in flight together.
  constexpr int EPT = RP * RP / 256;
  double gs[EPT];
#pragma unroll
  for (int e = 0; e < EPT; ++e) gs[e] = 0.0;
  for (int c = 0; c < nchunk; ++c) {
    const double* pc = P.part + (size_t)c * RP * RP;
    double v[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int x = tid + 256 * e, i = x / RP, j = x % RP;
      v[e] = (i <= j && j < r) ? pc[x] : 0.0;
    }
#pragma unroll
    for (int e = 0; e < EPT; ++e) gs[e] += v[e];
  }
#pragma unroll
  for (int e = 0; e < EPT; ++e) G[tid + 256 * e] = gs[e];
  __syncthreads();
  for (int k = 0; k < r; ++k) {
    if (tid == 0) {
      double d = G[k * RP + k];
      for (int i = 0; i < k; ++i) d = fma(-G[i * RP + k], G[i * RP + k], d);
      G[k * RP + k] = d > 0.0 ? sqrt(d) : 0.0;
    }
    __syncthreads();
    const double rkk = G[k * RP + k];
    for (int j = k + 1 + tid; j < r; j += 256) {
      double s = G[k * RP + j];
      for (int i = 0; i < k; ++i) s = fma(-G[i * RP + k], G[i * RP + j], s);
      G[k * RP + j] = rkk > 0.0 ? s / rkk : 0.0;
    }
    __syncthreads();
  }
  for (int j = tid; j < RP; j += 256) {
    const double d = j < r ? G[j * RP + j] : 0.0;
    inv[j] = d > 0.0 ? 1.0 / d : 0.0;
  }
  __syncthreads();
  if (tid < RP) {
    double x[RP];
#pragma unroll
    for (int j = 0; j < RP; ++j) {
      double s = j == tid ? 1.0 : 0.0;
#pragma unroll
      for (int l = 0; l < j; ++l) s = fma(-x[l], G[l * RP + j], s);
      x[j] = s * inv[j];
    }
#pragma unroll
    for (int j = 0; j < RP; ++j) X[tid * RP + j] = x[j];
  }
  __syncthreads();
  if (!FINAL) {
    for (int x = tid; x < RP * RP; x += 256) {
      const int i = x / RP, j = x % RP;
      P.R1[x] = i <= j ? G[x] : 0.0;
      P.X1[x] = X[x];
    }
    return;
  }
  // M = X1 X2, X1 staged in LDS.
  for (int x = tid; x < RP * RP; x += 256) X1s[x] = P.X1[x];
  __syncthreads();
  for (int x = tid; x < RP * RP; x += 256) {
    const int i = x / RP, j = x % RP;
    double s = 0.0;
    for (int k = 0; k < RP; ++k) s = fma(X1s[i * RP + k], X[k * RP + j], s);
    P.M[x] = s;
  }
  if (tid == 0) {
    int bad = 0;
    for (int k = 0; k < r; ++k) {
      const double d = G[k * RP + k] * P.R1[k * RP + k];
      if (P.r_diag) P.r_diag[k] = (float)d;
      if (d == 0.0 && bad == 0) bad = k + 1;
    }
    if (P.info) *P.info = bad;
  }
}

size_t panel_ws(int rows, int RP) {
  const size_t nchunk = (size_t)(rows + CHUNK - 1) / CHUNK;
  return zo_align256(nchunk * RP * RP * 8) + 3 * zo_align256((size_t)RP * RP * 8);
}

template <int RK>
int run_batch(const CqrArgs& ca, int wg, hipStream_t stream) {
  int st;
  if (wg > 0) hipLaunchKernelGGL((k_cqr_rows<RK, 0>), dim3(wg), dim3(256), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_rows")) != ZO_OK) return st;
  hipLaunchKernelGGL((k_cqr_chol<RK, false>), dim3(ca.count), dim3(256), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_chol")) != ZO_OK) return st;
  if (wg > 0) hipLaunchKernelGGL((k_cqr_rows<RK, 1>), dim3(wg), dim3(256), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_rows")) != ZO_OK) return st;
  hipLaunchKernelGGL((k_cqr_chol<RK, true>), dim3(ca.count), dim3(256), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_chol")) != ZO_OK) return st;
  if (wg > 0) hipLaunchKernelGGL((k_cqr_rows<RK, 2>), dim3(wg), dim3(256), 0, stream, ca);
  return zo_hip_status(hipGetLastError(), "k_cqr_rows");
}

// ---------------------------------------------------------------- 64 < r <= 128
// Wide panels are padded to RP = 128.  Neither an RP x RP operand next to a
// 128-row block nor a thread-private row of R^-1 fits at that width, so the
// same five launches are arranged differently:
//   rows: 256 threads, 64 rows in LDS at a time; the product Omega Mx streams
//         Mx through LDS 32 rows of K at a time (4 x 4 register tiles, two per
//         thread); the chunk's partial Gram is stored as its 528 upper 4 x 4
//         blocks.
//   chol: one RP x (RP + 1) LDS array holds R in its upper part (R_ij at
//         [i][j + 1]) and R^-1 transposed in its lower part (X_ij at [j][i]).
//         Cholesky and the inverse are right-looking: after column k is final,
//         every later entry takes its fused update from it.  Each entry sees
//         the same updates in the same order (k = 0, 1, ...) as the left-looking
//         sums of the narrow kernel, with the same zero-pivot rule.
constexpr int BIG_RP = 128;
constexpr int BIG_NT = 256;
constexpr int BIG_RW = 64;                      // rows per pass
constexpr int BIG_KC = 32;                      // K rows of Mx staged at a time
constexpr int BIG_NB = BIG_RP / 4;              // 4 x 4 blocks per side
constexpr int BIG_NBLK = BIG_NB * (BIG_NB + 1) / 2;

// Index of upper block (bi <= bj) in row-major order over the upper triangle.
__device__ __forceinline__ int big_blk(int bi, int bj) {
  return bi * BIG_NB - bi * (bi - 1) / 2 + (bj - bi);
}

template <int PASS>
__global__ __launch_bounds__(BIG_NT) void k_cqr_rows_big(CqrArgs a) {
  constexpr int RP = BIG_RP, NB = BIG_NB, NBLK = BIG_NBLK;
  constexpr int BPT = (NBLK + BIG_NT - 1) / BIG_NT;
  __shared__ __attribute__((aligned(16))) double rowbuf[BIG_RW][RP + 1];
  __shared__ __attribute__((aligned(16))) double Mk[PASS == 0 ? 2 : BIG_KC * RP];
  const CqrPanel& P = a.p[find_panel(a, blockIdx.x)];
  const int chunk = blockIdx.x - P.chunk_begin;
  const int r = a.r, tid = threadIdx.x;
  for (int x = tid; x < BIG_RW * (RP - r); x += BIG_NT)
    rowbuf[x / (RP - r)][r + x % (RP - r)] = 0.0;
  int bi[BPT], bj[BPT];
  double g[BPT][4][4];
#pragma unroll
  for (int t = 0; t < BPT; ++t) {
    int b = tid + t * BIG_NT, ii = 0;
    if (b >= NBLK) b = -1;
    if (b >= 0) {
      int rem = b;
      while (rem >= NB - ii) { rem -= NB - ii; ++ii; }
      bi[t] = ii;
      bj[t] = ii + rem;
    } else {
      bi[t] = bj[t] = -1;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) g[t][u][v] = 0.0;
  }
  // Product tiles: column group cg, row groups rg0 and rg0 + 8.
  const int cg = tid & 31, rg0 = tid >> 5;
  const int nkc = (r + BIG_KC - 1) / BIG_KC;
  const double* Msrc = PASS == 1 ? P.X1 : P.M;
  const int row_end = min((chunk + 1) * BIG_CHUNK, P.rows);
  for (int base = chunk * BIG_CHUNK; base < row_end; base += BIG_RW) {
    const int nrow = min(BIG_RW, row_end - base);
    __syncthreads();  // the previous block's rows have been consumed
    {
      const float* src = P.omega + (size_t)base * r;
      for (int x = tid; x < nrow * r; x += BIG_NT) rowbuf[x / r][x % r] = (double)src[x];
      for (int x = tid; x < (BIG_RW - nrow) * r; x += BIG_NT) rowbuf[nrow + x / r][x % r] = 0.0;
    }
    if (PASS >= 1) {
      double acc[2][4][4];
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[t][u][v] = 0.0;
      for (int kc = 0; kc < nkc; ++kc) {
        __syncthreads();  // rows stored / previous Mk slice consumed
        for (int x = tid; x < BIG_KC * RP; x += BIG_NT) Mk[x] = Msrc[(size_t)kc * BIG_KC * RP + x];
        __syncthreads();
#pragma unroll 4
        for (int kk = 0; kk < BIG_KC; ++kk) {
          const int k = kc * BIG_KC + kk;
          const double2 m01 = *(const double2*)&Mk[kk * RP + 4 * cg];
          const double2 m23 = *(const double2*)&Mk[kk * RP + 4 * cg + 2];
          const double m[4] = {m01.x, m01.y, m23.x, m23.y};
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int rg = rg0 + 8 * t;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const double av = rowbuf[4 * rg + u][k];
#pragma unroll
              for (int v = 0; v < 4; ++v) acc[t][u][v] = fma(av, m[v], acc[t][u][v]);
            }
          }
        }
      }
      __syncthreads();  // every thread has read its rows of Omega
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int rg = rg0 + 8 * t;
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) rowbuf[4 * rg + u][4 * cg + v] = acc[t][u][v];
      }
    }
    __syncthreads();
    if (PASS == 2) {
      float* dst = P.q + (size_t)base * r;
      for (int x = tid; x < nrow * r; x += BIG_NT) dst[x] = (float)rowbuf[x / r][x % r];
      continue;
    }
    for (int rr = 0; rr < nrow; ++rr) {
      const double* row = rowbuf[rr];
#pragma unroll
      for (int t = 0; t < BPT; ++t) {
        if (bi[t] < 0) continue;
        double u[4], v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          u[e] = row[4 * bi[t] + e];
          v[e] = row[4 * bj[t] + e];
        }
#pragma unroll
        for (int p = 0; p < 4; ++p)
#pragma unroll
          for (int q = 0; q < 4; ++q) g[t][p][q] = fma(u[p], v[q], g[t][p][q]);
      }
    }
  }
  if (PASS == 2) return;
  double* out = P.part + (size_t)chunk * NBLK * 16;
#pragma unroll
  for (int t = 0; t < BPT; ++t) {
    if (bi[t] < 0) continue;
    double* o = out + (size_t)big_blk(bi[t], bj[t]) * 16;
#pragma unroll
    for (int p = 0; p < 4; ++p)
#pragma unroll
      for (int q = 0; q < 4; ++q) o[p * 4 + q] = g[t][p][q];
  }
}

template <bool FINAL>
__global__ __launch_bounds__(BIG_NT) void k_cqr_chol_big(CqrArgs a) {
  constexpr int RP = BIG_RP, NBLK = BIG_NBLK;
  __shared__ double A[RP][RP + 1];  // R_ij at [i][j + 1], X_ij at [j][i]  (i <= j)
  __shared__ double inv[RP];
  __shared__ double dg[RP];
  const CqrPanel& P = a.p[blockIdx.x];
  const int r = a.r, tid = threadIdx.x;
  const int nchunk = (P.rows + BIG_CHUNK - 1) / BIG_CHUNK;
  for (int x = tid; x < RP * RP; x += BIG_NT) {
    const int i = x / RP, j = x % RP;
    if (i > j) continue;
    double s = 0.0;
    if (j < r) {
      const size_t e = (size_t)big_blk(i >> 2, j >> 2) * 16 + (i & 3) * 4 + (j & 3);
      for (int c = 0; c < nchunk; ++c) s += P.part[(size_t)c * NBLK * 16 + e];
    }
    A[i][j + 1] = s;
    A[j][i] = (i == j && i < r) ? 1.0 : 0.0;
  }
  __syncthreads();
  // Cholesky: G = R^T R, right-looking.
  for (int k = 0; k < r; ++k) {
    if (tid == 0) {
      const double d = A[k][k + 1];
      A[k][k + 1] = d > 0.0 ? sqrt(d) : 0.0;
    }
    __syncthreads();
    const double rkk = A[k][k + 1];
    for (int j = k + 1 + tid; j < r; j += BIG_NT) A[k][j + 1] = rkk > 0.0 ? A[k][j + 1] / rkk : 0.0;
    __syncthreads();
    for (int i = k + 1 + (tid >> 5); i < r; i += BIG_NT / 32) {
      const double rki = A[k][i + 1];
      for (int j = i + (tid & 31); j < r; j += 32) A[i][j + 1] = fma(-rki, A[k][j + 1], A[i][j + 1]);
    }
    __syncthreads();
  }
  for (int j = tid; j < RP; j += BIG_NT) {
    const double d = j < r ? A[j][j + 1] : 0.0;
    inv[j] = d > 0.0 ? 1.0 / d : 0.0;
  }
  __syncthreads();
  // X = R^-1: rows of the identity through the forward substitution, column by
  // column; X_ij = 0 for i > j, and column j is final once scaled by 1 / R_jj.
  for (int j = 0; j < r; ++j) {
    for (int i = tid; i <= j; i += BIG_NT) A[j][i] *= inv[j];
    __syncthreads();
    for (int jj = j + 1 + (tid >> 5); jj < r; jj += BIG_NT / 32) {
      const double rjj = A[j][jj + 1];
      for (int i = tid & 31; i <= j; i += 32) A[jj][i] = fma(-A[j][i], rjj, A[jj][i]);
    }
    __syncthreads();
  }
  if (!FINAL) {
    for (int x = tid; x < RP * RP; x += BIG_NT) {
      const int i = x / RP, j = x % RP;
      P.R1[x] = i <= j ? A[i][j + 1] : 0.0;
      P.X1[x] = i <= j ? A[j][i] : 0.0;
    }
    return;
  }
  for (int k = tid; k < RP; k += BIG_NT) dg[k] = A[k][k + 1];
  __syncthreads();
  // R2 is no longer needed: X1 takes its place, then M = X1 X2.
  for (int x = tid; x < RP * RP; x += BIG_NT) {
    const int i = x / RP, j = x % RP;
    if (i <= j) A[i][j + 1] = P.X1[x];
  }
  __syncthreads();
  for (int x = tid; x < RP * RP; x += BIG_NT) {
    const int i = x / RP, j = x % RP;
    double s = 0.0;
    for (int k = i; k <= j; ++k) s = fma(A[i][k + 1], A[j][k], s);
    P.M[x] = s;
  }
  if (tid == 0) {
    int bad = 0;
    for (int k = 0; k < r; ++k) {
      const double d = dg[k] * P.R1[k * RP + k];
      if (P.r_diag) P.r_diag[k] = (float)d;
      if (d == 0.0 && bad == 0) bad = k + 1;
    }
    if (P.info) *P.info = bad;
  }
}

size_t panel_ws_big(int rows) {
  const size_t nchunk = (size_t)(rows + BIG_CHUNK - 1) / BIG_CHUNK;
  return zo_align256(nchunk * BIG_NBLK * 16 * 8) + 3 * zo_align256((size_t)BIG_RP * BIG_RP * 8);
}

int run_batch_big(const CqrArgs& ca, int wg, hipStream_t stream) {
  int st;
  if (wg > 0) hipLaunchKernelGGL(k_cqr_rows_big<0>, dim3(wg), dim3(BIG_NT), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_rows_big")) != ZO_OK) return st;
  hipLaunchKernelGGL(k_cqr_chol_big<false>, dim3(ca.count), dim3(BIG_NT), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_chol_big")) != ZO_OK) return st;
  if (wg > 0) hipLaunchKernelGGL(k_cqr_rows_big<1>, dim3(wg), dim3(BIG_NT), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_rows_big")) != ZO_OK) return st;
  hipLaunchKernelGGL(k_cqr_chol_big<true>, dim3(ca.count), dim3(BIG_NT), 0, stream, ca);
  if ((st = zo_hip_status(hipGetLastError(), "k_cqr_chol_big")) != ZO_OK) return st;
  if (wg > 0) hipLaunchKernelGGL(k_cqr_rows_big<2>, dim3(wg), dim3(BIG_NT), 0, stream, ca);
  return zo_hip_status(hipGetLastError(), "k_cqr_rows_big");
}

}  // namespace

int zo_refresh_launch(int count, const zo_panel* panels, int r, int* info, void* ws,
                      size_t ws_bytes, hipStream_t stream, size_t* ws_needed) {
  const bool big = r > 64;
  const int RK = big ? BIG_RP / 16 : (r + 15) / 16;
  const int RP = 16 * RK;
  const int chunk_rows = big ? BIG_CHUNK : CHUNK;
  size_t need = zo_align256((size_t)count * sizeof(CqrPanel));
  for (int p = 0; p < count; ++p) need += big ? panel_ws_big(panels[p].rows) : panel_ws(panels[p].rows, RP);
  if (ws_needed) *ws_needed = need;
  if (!ws || count == 0) return ZO_OK;
  if (ws_bytes < need) {
    zo_set_error("refresh: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  WsCarver wc(ws);
  CqrPanel* tab = (CqrPanel*)wc.take((size_t)count * sizeof(CqrPanel));
  std::vector<CqrPanel> host((size_t)count);
  long long wg = 0;
  for (int p = 0; p < count; ++p) {
    CqrPanel& e = host[p];
    const int nchunk = (panels[p].rows + chunk_rows - 1) / chunk_rows;
    e.omega = panels[p].omega;
    e.q = panels[p].q;
    e.r_diag = panels[p].r_diag;
    e.info = info ? info + p : nullptr;
    e.part = (double*)wc.take((size_t)nchunk * (big ? BIG_NBLK * 16 : RP * RP) * 8);
    e.R1 = (double*)wc.take((size_t)RP * RP * 8);
    e.X1 = (double*)wc.take((size_t)RP * RP * 8);
    e.M = (double*)wc.take((size_t)RP * RP * 8);
    e.rows = panels[p].rows;
    e.chunk_begin = (int)wg;
    wg += nchunk;
  }
  if (wg > 0x7fffffffLL) {
    zo_set_error("refresh: too many row chunks (%lld)", wg);
    return ZO_ERR_UNSUPPORTED;
  }
  int st;
  for (int c0 = 0; c0 < count; c0 += FILL_PANELS) {
    CqrFill f{};
    f.n = std::min(FILL_PANELS, count - c0);
    for (int i = 0; i < f.n; ++i) f.p[i] = host[c0 + i];
    f.dst = tab + c0;
    const int words = f.n * (int)(sizeof(CqrPanel) / 4);
    hipLaunchKernelGGL(k_cqr_fill, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, stream, f);
    if ((st = zo_hip_status(hipGetLastError(), "k_cqr_fill")) != ZO_OK) return st;
  }
  CqrArgs ca{};
  ca.p = tab;
  ca.count = count;
  ca.r = r;
  switch (big ? 0 : RK) {
    case 0: return run_batch_big(ca, (int)wg, stream);
    case 1: return run_batch<1>(ca, (int)wg, stream);
    case 2: return run_batch<2>(ca, (int)wg, stream);
    case 3: return run_batch<3>(ca, (int)wg, stream);
    default: return run_batch<4>(ca, (int)wg, stream);
  }
}

// ---------------------------------------------------------------- no-allocation variant
// The scratch of zo_subspace_refresh_noalloc: a static device array, one copy per GPU the
// library runs on, held until the process ends.  The row passes write every partial Gram
// entry the Cholesky launch reads, and the Cholesky launch writes all of R1, X1 and M, so
// nothing in it has to start at zero and what an earlier call left there is never read.
// In host code the array's name is a stand-in, not a device address: the device address is
// looked up once per device (hipGetSymbolAddress, with that device current) and only that
// pointer is handed to kernels.
static __device__ __align__(256) char scratch[ZO_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES];
}  // namespace

int zo_refresh_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return zo_hip_status(e, "refresh_noalloc: hipGetDevice");
  if (dev < 0 || dev >= MAX_DEVICES) {
    zo_set_error("refresh_noalloc: device %d outside [0, %d)", dev, MAX_DEVICES);
    return ZO_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return zo_hip_status(e, "refresh_noalloc: hipGetSymbolAddress");
    if (!p || (uintptr_t)p % 256 != 0) {
      zo_set_error("refresh_noalloc: scratch address %p unusable", p);
      return ZO_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return ZO_OK;
}

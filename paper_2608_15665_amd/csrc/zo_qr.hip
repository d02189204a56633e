// Subspace refresh of SubZero+: Haar-distributed factor of a Gaussian panel
// (Eq. 11, Alg. 1) -- thin QR with each column of Q multiplied by the sign of
// the matching diagonal entry of R, so the corrected R has diag(R) > 0.
//
// Tall-skinny QR as a reduction tree (TSQR) of Householder factorisations,
// float64 throughout:
//   up pass    level 0: each leaf is a block of at most BMAX rows of the
//              panel; level l >= 1: each node stacks the R factors (r x r) of
//              up to G children.  A node loads its block into LDS
//              (column-major float64), runs r Householder steps (one wave
//              per trailing column: dot product by wave reduction, then the
//              rank-1 update), writes its R, then forms its explicit Q in
//              place by backward accumulation and writes it.
//   down pass  from the root: the root's Q is multiplied by diag(s),
//              s_k = sgn(R_kk) with sgn(0) = +1; every child's Q is
//              multiplied by its r x r slice of the parent's final Q.  The
//              leaves write the float32 panel output.
// The final Q equals the panel's unique thin-QR factor with positive
// diag(R), whatever sign convention the reflectors use.
#include "zo_internal.h"

#include <vector>

namespace {

constexpr int NT = 256;
constexpr int LDS_DOUBLES = 16384;  // 128 KB node block (plus padding of the leading dimension)
constexpr int MAX_LEAF_ROWS = 1024;
constexpr int MAX_FANIN = 16;
constexpr int PANELS_PER_LAUNCH = 16;  // keeps the kernel-argument struct under 2 KB

struct QrEntry {
  const float* omega;
  float* q;
  float* r_diag;
  int* info;
  double* Qn;         // Q of this level's nodes
  double* Rn;         // R of this level's nodes (r x r each)
  const double* Rc;   // children's R (up pass, level >= 1)
  const double* Mp;   // parent's final Q (down pass, below the top)
  double* Qf;         // this level's final Q (down pass, level >= 1)
  int rows, nodes, child_nodes, G, leaf_base, leaf_extra, is_top, wg_begin;
};
struct QrArgs {
  QrEntry e[PANELS_PER_LAUNCH];
  int count, r, level;
};

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ int find_entry(const QrArgs& a) {
  int k = 0;
  while (k + 1 < a.count && (int)blockIdx.x >= a.e[k + 1].wg_begin) ++k;
  return k;
}

__device__ __forceinline__ void leaf_rows(const QrEntry& e, int node, int* rs, int* nr) {
  *rs = node * e.leaf_base + min(node, e.leaf_extra);
  *nr = e.leaf_base + (node < e.leaf_extra ? 1 : 0);
}

// Householder QR of the nr x r block in LDS (column-major, leading dim ld).
// On return the upper triangle holds R, the reflector vectors (v_0 = 1
// implied) sit below the diagonal and tau[] holds their scalars.
__device__ void householder_lds(double* A, int ld, int nr, int r, double* tau, double* red) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int k = 0; k < r; ++k) {
    double* ck = A + (size_t)k * ld;
    double s = 0.0;
    for (int i = k + 1 + tid; i < nr; i += NT) s += ck[i] * ck[i];
    s = wave_sum(s);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (tid == 0) {
      const double xn2 = (red[0] + red[1]) + (red[2] + red[3]);
      const double alpha = ck[k];
      double t = 0.0, scale = 0.0, beta = alpha;
      if (xn2 > 0.0) {
        beta = -copysign(sqrt(alpha * alpha + xn2), alpha);
        t = (beta - alpha) / beta;
        scale = 1.0 / (alpha - beta);
      }
      tau[k] = t;
      red[4] = scale;
      ck[k] = beta;
    }
    __syncthreads();
    const double scale = red[4];
    const double tk = tau[k];
    if (tk != 0.0)
      for (int i = k + 1 + tid; i < nr; i += NT) ck[i] *= scale;
    __syncthreads();
    if (tk != 0.0) {
      for (int j = k + 1 + wave; j < r; j += NT / 64) {
        double* cj = A + (size_t)j * ld;
        double w = 0.0;
        for (int i = k + 1 + lane; i < nr; i += 64) w += ck[i] * cj[i];
        w = wave_sum(w) + cj[k];
        const double tw = tk * w;
        for (int i = k + 1 + lane; i < nr; i += 64) cj[i] -= tw * ck[i];
        if (lane == 0) cj[k] -= tw;
      }
    }
    __syncthreads();
  }
}

// Explicit thin Q (nr x r) from the reflectors, in place (backward accumulation).
__device__ void form_q_lds(double* A, int ld, int nr, int r, const double* tau) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int k = r - 1; k >= 0; --k) {
    double* ck = A + (size_t)k * ld;
    const double tk = tau[k];
    if (tk != 0.0) {
      for (int j = k + 1 + wave; j < r; j += NT / 64) {
        double* cj = A + (size_t)j * ld;
        double w = 0.0;
        for (int i = k + 1 + lane; i < nr; i += 64) w += ck[i] * cj[i];
        w = wave_sum(w) + cj[k];
        const double tw = tk * w;
        for (int i = k + 1 + lane; i < nr; i += 64) cj[i] -= tw * ck[i];
        if (lane == 0) cj[k] -= tw;
      }
    }
    __syncthreads();
    for (int i = tid; i < nr; i += NT) {
      double v;
      if (i < k) v = 0.0;
      else if (i == k) v = 1.0 - tk;
      else v = -tk * ck[i];
      ck[i] = v;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(NT) void k_qr_up(QrArgs a) {
  __shared__ double A[LDS_DOUBLES + ZO_MAX_QR_RANK];
  __shared__ double tau[ZO_MAX_QR_RANK];
  __shared__ double red[8];
  const QrEntry& e = a.e[find_entry(a)];
  const int node = blockIdx.x - e.wg_begin;
  const int r = a.r, tid = threadIdx.x;
  int nr, ld;
  double* qout;
  if (a.level == 0) {
    int rs;
    leaf_rows(e, node, &rs, &nr);
    ld = nr | 1;  // odd leading dimension: column-strided LDS access spreads over banks
    for (int x = tid; x < nr * r; x += NT) {
      const int i = x / r, c = x % r;
      A[(size_t)c * ld + i] = (double)e.omega[(size_t)(rs + i) * r + c];
    }
    qout = e.Qn + (size_t)rs * r;
  } else {
    const int c0 = node * e.G;
    const int c1 = min(c0 + e.G, e.child_nodes);
    nr = (c1 - c0) * r;
    ld = nr | 1;
    const double* src = e.Rc + (size_t)c0 * r * r;  // stacked r x r row-major blocks
    for (int x = tid; x < nr * r; x += NT) {
      const int i = x / r, c = x % r;
      A[(size_t)c * ld + i] = src[x];
    }
    qout = e.Qn + (size_t)node * e.G * r * r;
  }
  __syncthreads();
  householder_lds(A, ld, nr, r, tau, red);
  double* Rout = e.Rn + (size_t)node * r * r;
  for (int x = tid; x < r * r; x += NT) {
    const int i = x / r, c = x % r;
    Rout[x] = i <= c ? A[(size_t)c * ld + i] : 0.0;
  }
  if (e.is_top && tid == 0) {
    int bad = 0;
    for (int k = 0; k < r; ++k) {
      const double d = A[(size_t)k * ld + k];
      if (e.r_diag) e.r_diag[k] = (float)fabs(d);
      if (d == 0.0 && bad == 0) bad = k + 1;
    }
    if (e.info) *e.info = bad;
  }
  __syncthreads();
  form_q_lds(A, ld, nr, r, tau);
  for (int x = tid; x < nr * r; x += NT) {
    const int i = x / r, c = x % r;
    qout[x] = A[(size_t)c * ld + i];
  }
}

__global__ __launch_bounds__(NT) void k_qr_down(QrArgs a) {
  __shared__ double M[ZO_MAX_QR_RANK * ZO_MAX_QR_RANK];
  const QrEntry& e = a.e[find_entry(a)];
  const int node = blockIdx.x - e.wg_begin;
  const int r = a.r, tid = threadIdx.x;
  if (e.is_top) {
    const double* R = e.Rn;  // the root's R
    for (int x = tid; x < r * r; x += NT) {
      const int i = x / r, c = x % r;
      M[x] = i == c ? (R[(size_t)i * r + i] < 0.0 ? -1.0 : 1.0) : 0.0;
    }
  } else {
    const int p = node / e.G, cl = node % e.G;
    const double* src = e.Mp + ((size_t)p * e.G + cl) * r * r;
    for (int x = tid; x < r * r; x += NT) M[x] = src[x];
  }
  __syncthreads();
  int nr;
  const double* Qsrc;
  if (a.level == 0) {
    int rs;
    leaf_rows(e, node, &rs, &nr);
    Qsrc = e.Qn + (size_t)rs * r;
    float* out = e.q + (size_t)rs * r;
    for (int x = tid; x < nr * r; x += NT) {
      const int i = x / r, c = x % r;
      const double* qi = Qsrc + (size_t)i * r;
      double s = 0.0;
      for (int k = 0; k < r; ++k) s += qi[k] * M[k * r + c];
      out[x] = (float)s;
    }
  } else {
    const int c0 = node * e.G;
    const int c1 = min(c0 + e.G, e.child_nodes);
    nr = (c1 - c0) * r;
    Qsrc = e.Qn + (size_t)node * e.G * r * r;
    double* out = e.Qf + (size_t)node * e.G * r * r;
    for (int x = tid; x < nr * r; x += NT) {
      const int i = x / r, c = x % r;
      const double* qi = Qsrc + (size_t)i * r;
      double s = 0.0;
      for (int k = 0; k < r; ++k) s += qi[k] * M[k * r + c];
      out[x] = s;
    }
  }
}

struct PanelPlan {
  int rows, nleaf, G, top, leaf_base, leaf_extra;
  std::vector<int> nodes;           // per level
  std::vector<size_t> q_off, r_off, qf_off;  // doubles, per level
  size_t q_total, r_total, qf_total;
};

PanelPlan plan_panel(int rows, int r) {
  PanelPlan p;
  p.rows = rows;
  int bmax = LDS_DOUBLES / r;
  if (bmax > MAX_LEAF_ROWS) bmax = MAX_LEAF_ROWS;
  p.G = bmax / r;
  if (p.G > MAX_FANIN) p.G = MAX_FANIN;
  p.nleaf = (rows + bmax - 1) / bmax;
  p.leaf_base = rows / p.nleaf;
  p.leaf_extra = rows % p.nleaf;
  p.nodes.push_back(p.nleaf);
  while (p.nodes.back() > 1) p.nodes.push_back((p.nodes.back() + p.G - 1) / p.G);
  p.top = (int)p.nodes.size() - 1;
  size_t q = 0, rr = 0, qf = 0;
  for (int l = 0; l <= p.top; ++l) {
    p.q_off.push_back(q);
    p.r_off.push_back(rr);
    p.qf_off.push_back(qf);
    if (l == 0) {
      q += (size_t)rows * r;
    } else {
      q += (size_t)p.nodes[l] * p.G * r * r;
      qf += (size_t)p.nodes[l] * p.G * r * r;
    }
    rr += (size_t)p.nodes[l] * r * r;
  }
  p.q_total = q;
  p.r_total = rr;
  p.qf_total = qf;
  return p;
}

}  // namespace

int zo_refresh_launch(int count, const zo_panel* panels, int r, int* info, void* ws,
                      size_t ws_bytes, hipStream_t stream, size_t* ws_needed) {
  std::vector<PanelPlan> plans;
  plans.reserve(count);
  size_t need = 0;
  int max_top = 0;
  for (int p = 0; p < count; ++p) {
    plans.push_back(plan_panel(panels[p].rows, r));
    const PanelPlan& pl = plans.back();
    need += zo_align256(pl.q_total * 8) + zo_align256(pl.r_total * 8) + zo_align256(pl.qf_total * 8);
    if (pl.top > max_top) max_top = pl.top;
  }
  if (ws_needed) *ws_needed = need;
  if (!ws) return ZO_OK;
  if (ws_bytes < need) {
    zo_set_error("refresh: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  std::vector<double*> qb(count), rb(count), qfb(count);
  WsCarver wc(ws);
  for (int p = 0; p < count; ++p) {
    qb[p] = (double*)wc.take(plans[p].q_total * 8);
    rb[p] = (double*)wc.take(plans[p].r_total * 8);
    qfb[p] = (double*)wc.take(plans[p].qf_total * 8);
  }
  int st;
  // Up pass, level by level; down pass from the highest root to the leaves.
  for (int pass = 0; pass < 2; ++pass) {
    for (int step = 0; step <= max_top; ++step) {
      const int level = pass == 0 ? step : max_top - step;
      for (int c0 = 0; c0 < count; c0 += PANELS_PER_LAUNCH) {
        QrArgs qa{};
        qa.r = r;
        qa.level = level;
        int n = 0, wg = 0;
        for (int p = c0; p < count && p < c0 + PANELS_PER_LAUNCH; ++p) {
          const PanelPlan& pl = plans[p];
          if (level > pl.top) continue;
          QrEntry e{};
          e.omega = panels[p].omega;
          e.q = panels[p].q;
          e.r_diag = panels[p].r_diag;
          e.info = info ? info + p : nullptr;
          e.Qn = qb[p] + pl.q_off[level];
          e.Rn = rb[p] + pl.r_off[level];
          e.Rc = level > 0 ? rb[p] + pl.r_off[level - 1] : nullptr;
          e.Mp = level < pl.top ? qfb[p] + pl.qf_off[level + 1] : nullptr;
          e.Qf = level > 0 ? qfb[p] + pl.qf_off[level] : nullptr;
          e.rows = pl.rows;
          e.nodes = pl.nodes[level];
          e.child_nodes = level > 0 ? pl.nodes[level - 1] : 0;
          e.G = pl.G;
          e.leaf_base = pl.leaf_base;
          e.leaf_extra = pl.leaf_extra;
          e.is_top = level == pl.top;
          e.wg_begin = wg;
          wg += e.nodes;
          qa.e[n++] = e;
        }
        if (n == 0) continue;
        qa.count = n;
        if (pass == 0)
          hipLaunchKernelGGL(k_qr_up, dim3(wg), dim3(NT), 0, stream, qa);
        else
          hipLaunchKernelGGL(k_qr_down, dim3(wg), dim3(NT), 0, stream, qa);
        if ((st = zo_hip_status(hipGetLastError(), pass == 0 ? "k_qr_up" : "k_qr_down")) != ZO_OK)
          return st;
      }
    }
  }
  return ZO_OK;
}

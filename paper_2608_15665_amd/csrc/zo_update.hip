// Subspace Adam update of SubZero+ (Eqs. 6-10, tail of Alg. 3).
//
// Three launches per chunk of up to ITEMS_PER_LAUNCH matrices:
//   k_adam_rr   one workgroup per matrix: Zbar = (1/q) sum_j g_j Z_j, the two
//               r x r moments (Eqs. 7-8), the bias-corrected direction S
//               (Eq. 9, Adam form), all in float64; writes M1, M2 (fp32) and
//               S (float64, workspace) -- or, if any entry is non-finite,
//               leaves the state alone, raises the flag and marks the item
//               skipped.
//   k_us        L = lr U S (m x rp) and V (n x rp), zero padded to rp columns.
//               bf16 W: each as a hi + lo pair of bf16 (x = hi + lo to about
//               16 significant bits); fp32 W: L in fp32.
//   k_update_*  W <- W - L V^T in place.
//
// bf16 W (k_update_bf16): memory bound -- 4 bytes of HBM traffic per weight
// against 2 r MACs.  At r = 64 that is 32 FLOP/B, above the fp32 VALU ridge
// of the chip, so the rank-r product runs on v_mfma_f32_16x16x32_bf16 as
// hi*hi + hi*lo + lo*hi (3 MFMAs per 32-deep K step).  Each wave owns a strip
// of 64 columns whose V fragments stay in registers, and walks down rows 16
// at a time.  The A operand rows are the strip's columns in a permuted order
// so that the 16 accumulator values a lane ends with are 16 ADJACENT columns
// of one row: the lane reads and writes its W values as two 16-byte vectors.
#include "zo_internal.h"

namespace {

constexpr int ITEMS_PER_LAUNCH = 16;
constexpr int UPD_ROWS = 128;  // rows per workgroup (8 steps of 16 per wave)
constexpr int UPD_COLS = 256;  // columns per workgroup (4 waves x 64)

struct ItemRR {
  const float* Z;
  float* M1;
  float* M2;
  float* zbar_out;
  double* S;  // workspace, r x r
  int* skip;  // workspace
};
struct RRArgs {
  ItemRR it[ITEMS_PER_LAUNCH];
  const float* g;
  int* nonfinite_flag;
  int r, q;
  double beta1, beta2, eps_adam, bc1, bc2;
};

__global__ __launch_bounds__(256) void k_adam_rr(RRArgs a) {
  const ItemRR& it = a.it[blockIdx.x];
  const int rr = a.r * a.r;
  int bad = 0;
  for (int e = threadIdx.x; e < rr; e += 256) {
    double zb = 0.0;
    for (int j = 0; j < a.q; ++j) zb += (double)a.g[j] * (double)it.Z[(size_t)j * rr + e];
    zb /= (double)a.q;
    const double m1 = a.beta1 * (double)it.M1[e] + (1.0 - a.beta1) * zb;
    const double m2 = a.beta2 * (double)it.M2[e] + (1.0 - a.beta2) * zb * zb;
    const double s = (m1 / a.bc1) / (sqrt(m2 / a.bc2) + a.eps_adam);
    if (!isfinite(zb) || !isfinite(s)) bad = 1;
    if (it.zbar_out) it.zbar_out[e] = (float)zb;
  }
  bad = __syncthreads_or(bad);
  if (bad) {
    if (threadIdx.x == 0) {
      *it.skip = 1;
      if (a.nonfinite_flag) *a.nonfinite_flag = 1;
    }
    return;
  }
  // Second pass writes the state, recomputed identically.  Element e is read
  // and written by the same thread only, so no barrier is needed.
  for (int e = threadIdx.x; e < rr; e += 256) {
    double zb = 0.0;
    for (int j = 0; j < a.q; ++j) zb += (double)a.g[j] * (double)it.Z[(size_t)j * rr + e];
    zb /= (double)a.q;
    const double m1 = a.beta1 * (double)it.M1[e] + (1.0 - a.beta1) * zb;
    const double m2 = a.beta2 * (double)it.M2[e] + (1.0 - a.beta2) * zb * zb;
    it.S[e] = (m1 / a.bc1) / (sqrt(m2 / a.bc2) + a.eps_adam);
    it.M1[e] = (float)m1;
    it.M2[e] = (float)m2;
  }
  if (threadIdx.x == 0) *it.skip = 0;
}

struct ItemUS {
  const float* U;
  const float* V;
  const double* S;
  const int* skip;
  void* L;   // bf16: hi then lo (2 x m x rp); fp32: m x rp
  void* Vs;  // bf16: hi then lo (2 x n x rp); unused for fp32
  int m, n;
  long long begin;  // first flat index of this item in the launch
};
struct USArgs {
  ItemUS it[ITEMS_PER_LAUNCH];
  int count, r, rp, bf16;
  float lr;
  long long total;
};

__global__ __launch_bounds__(256) void k_us(USArgs a) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= a.total) return;
  int k = 0;
  while (k + 1 < a.count && idx >= a.it[k + 1].begin) ++k;
  const ItemUS& it = a.it[k];
  if (*it.skip) return;
  const long long e = idx - it.begin;
  const long long nl = (long long)it.m * a.rp;
  if (e < nl) {
    const int i = (int)(e / a.rp), c = (int)(e % a.rp);
    float v = 0.f;
    if (c < a.r) {
      double acc = 0.0;
      for (int t = 0; t < a.r; ++t) acc += (double)it.U[(size_t)i * a.r + t] * it.S[t * a.r + c];
      v = (float)((double)a.lr * acc);
    }
    if (a.bf16) {
      const bf16_t hi = f32_to_bf16(v);
      const bf16_t lo = f32_to_bf16(v - bf16_to_f32(hi));
      ((bf16_t*)it.L)[e] = hi;
      ((bf16_t*)it.L)[nl + e] = lo;
    } else {
      ((float*)it.L)[e] = v;
    }
  } else {
    const long long f = e - nl;  // only launched for bf16
    const int i = (int)(f / a.rp), c = (int)(f % a.rp);
    const float v = c < a.r ? it.V[(size_t)i * a.r + c] : 0.f;
    const bf16_t hi = f32_to_bf16(v);
    const bf16_t lo = f32_to_bf16(v - bf16_to_f32(hi));
    const long long nv = (long long)it.n * a.rp;
    ((bf16_t*)it.Vs)[f] = hi;
    ((bf16_t*)it.Vs)[nv + f] = lo;
  }
}

struct ItemUpd {
  void* W;
  float* wout;
  const void* L;
  const void* Vs;  // bf16 path: split V; fp32 path: V itself (n x r)
  const int* skip;
  int m, n;
  int strips, wg_begin;
};
struct UpdArgs {
  ItemUpd it[ITEMS_PER_LAUNCH];
  int count, r, rp;
};

__device__ __forceinline__ bf16x8 ld_frag(const bf16_t* p, bool ok) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if (ok) v = *(const u32x4*)p;
  return __builtin_bit_cast(bf16x8, v);
}

template <int RPK>  // rp = 32 * RPK
__global__ __launch_bounds__(256) void k_update_bf16(UpdArgs a) {
  constexpr int RP = 32 * RPK;
  int k = 0;
  while (k + 1 < a.count && (int)blockIdx.x >= a.it[k + 1].wg_begin) ++k;
  const ItemUpd& it = a.it[k];
  if (*it.skip) return;
  const int local = blockIdx.x - it.wg_begin;
  const int strip = local % it.strips;
  const int rchunk = local / it.strips;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col0 = strip * UPD_COLS + wave * 64;
  const int row0 = rchunk * UPD_ROWS;
  const int m = it.m, n = it.n;
  if (col0 >= n) return;

  const bf16_t* __restrict__ Lh = (const bf16_t*)it.L;
  const bf16_t* __restrict__ Ll = Lh + (size_t)m * RP;
  const bf16_t* __restrict__ Vh = (const bf16_t*)it.Vs;
  const bf16_t* __restrict__ Vl = Vh + (size_t)n * RP;
  const int l16 = lane & 15, g = lane >> 4;

  // V fragments of the strip (A operand): row rho = l16 of tile t is column
  // col0 + 16 (rho / 4) + 4 t + rho % 4.
  bf16x8 vh[RPK][4], vl[RPK][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int col = col0 + 16 * (l16 >> 2) + 4 * t + (l16 & 3);
    const bool ok = col < n;
#pragma unroll
    for (int kk = 0; kk < RPK; ++kk) {
      const size_t off = (size_t)col * RP + kk * 32 + g * 8;
      vh[kk][t] = ld_frag(Vh + off, ok);
      vl[kk][t] = ld_frag(Vl + off, ok);
    }
  }

  bf16_t* __restrict__ W = (bf16_t*)it.W;
  const int cbase = col0 + 16 * g;  // this lane's 16 adjacent columns
  const bool c0ok = cbase < n, c1ok = cbase + 8 < n;
  const int rend = min(row0 + UPD_ROWS, m);
  for (int rs = row0; rs < rend; rs += 16) {
    const int row = rs + l16;
    const bool rok = row < m;
    bf16x8 uh[RPK], ul[RPK];
#pragma unroll
    for (int kk = 0; kk < RPK; ++kk) {
      const size_t off = (size_t)row * RP + kk * 32 + g * 8;
      uh[kk] = ld_frag(Lh + off, rok);
      ul[kk] = ld_frag(Ll + off, rok);
    }
    u32x4 w0 = {0u, 0u, 0u, 0u}, w1 = {0u, 0u, 0u, 0u};
    bf16_t* wp = W + (size_t)row * n + cbase;
    if (rok && c0ok) w0 = *(const u32x4*)wp;
    if (rok && c1ok) w1 = *(const u32x4*)(wp + 8);
    f32x4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      acc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < RPK; ++kk) {
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vh[kk][t], uh[kk], acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vh[kk][t], ul[kk], acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vl[kk][t], uh[kk], acc[t], 0, 0, 0);
      }
    }
    // acc[t][c] is column cbase + 4 t + c.
    uint32_t wv[8] = {w0[0], w0[1], w0[2], w0[3], w1[0], w1[1], w1[2], w1[3]};
    float nv[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint32_t word = wv[e >> 1];
      const float old = __uint_as_float((e & 1) ? (word & 0xffff0000u) : (word << 16));
      nv[e] = old - acc[e >> 2][e & 3];
    }
    if (rok) {
      if (c0ok) {
        u32x4 o = {pack_bf16x2(nv[0], nv[1]), pack_bf16x2(nv[2], nv[3]), pack_bf16x2(nv[4], nv[5]),
                   pack_bf16x2(nv[6], nv[7])};
        *(u32x4*)wp = o;
      }
      if (c1ok) {
        u32x4 o = {pack_bf16x2(nv[8], nv[9]), pack_bf16x2(nv[10], nv[11]),
                   pack_bf16x2(nv[12], nv[13]), pack_bf16x2(nv[14], nv[15])};
        *(u32x4*)(wp + 8) = o;
      }
      if (it.wout) {
        float* fo = it.wout + (size_t)row * n + cbase;
        if (c0ok) {
          *(f32x4*)fo = (f32x4){nv[0], nv[1], nv[2], nv[3]};
          *(f32x4*)(fo + 4) = (f32x4){nv[4], nv[5], nv[6], nv[7]};
        }
        if (c1ok) {
          *(f32x4*)(fo + 8) = (f32x4){nv[8], nv[9], nv[10], nv[11]};
          *(f32x4*)(fo + 12) = (f32x4){nv[12], nv[13], nv[14], nv[15]};
        }
      }
    }
  }
}

// fp32 W: one thread per weight, fp32 FMA over the r columns.
__global__ __launch_bounds__(256) void k_update_f32(UpdArgs a) {
  int k = 0;
  while (k + 1 < a.count && (int)blockIdx.x >= a.it[k + 1].wg_begin) ++k;
  const ItemUpd& it = a.it[k];
  if (*it.skip) return;
  const long long e = (long long)(blockIdx.x - it.wg_begin) * 256 + threadIdx.x;
  if (e >= (long long)it.m * it.n) return;
  const int i = (int)(e / it.n), c = (int)(e % it.n);
  const float* L = (const float*)it.L;  // m x rp (rp = r)
  const float* V = (const float*)it.Vs; // n x r
  float d = 0.f;
  for (int t = 0; t < a.r; ++t) d = fmaf(L[(size_t)i * a.rp + t], V[(size_t)c * a.r + t], d);
  float* W = (float*)it.W;
  const float nv = W[e] - d;
  W[e] = nv;
  if (it.wout) it.wout[e] = nv;
}

struct Layout {
  size_t s, skip, L, Vs, total;
};
Layout item_layout(int m, int n, int r, int rp, int bf16) {
  Layout l;
  l.s = zo_align256((size_t)r * r * 8);
  l.skip = 256;
  l.L = zo_align256((size_t)m * rp * (bf16 ? 4 : 4));  // bf16: hi+lo; fp32: one
  l.Vs = bf16 ? zo_align256((size_t)n * rp * 4) : 0;
  l.total = l.s + l.skip + l.L + l.Vs;
  return l;
}

}  // namespace

int zo_update_launch(int count, const zo_update_item* items, int w_dtype, int r, int q,
                     const float* g, int t, float lr, float beta1, float beta2, float eps_adam,
                     int* nonfinite_flag, void* ws, size_t ws_bytes, hipStream_t stream,
                     size_t* ws_needed) {
  const int bf16 = w_dtype == ZO_BF16;
  const int rp = bf16 ? (r + 31) / 32 * 32 : r;
  size_t need = 0;
  for (int i = 0; i < count; ++i) need += item_layout(items[i].m, items[i].n, r, rp, bf16).total;
  if (ws_needed) *ws_needed = need;
  if (!ws) return ZO_OK;
  if (ws_bytes < need) {
    zo_set_error("update: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  if (bf16 && rp / 32 > 4) {
    zo_set_error("update: r = %d above %d", r, ZO_MAX_RANK);
    return ZO_ERR_UNSUPPORTED;
  }
  WsCarver wc(ws);
  int st;
  for (int c0 = 0; c0 < count; c0 += ITEMS_PER_LAUNCH) {
    const int cn = count - c0 < ITEMS_PER_LAUNCH ? count - c0 : ITEMS_PER_LAUNCH;
    RRArgs ra{};
    USArgs ua{};
    UpdArgs pa{};
    ra.g = g;
    ra.nonfinite_flag = nonfinite_flag;
    ra.r = r;
    ra.q = q;
    ra.beta1 = beta1;
    ra.beta2 = beta2;
    ra.eps_adam = eps_adam;
    ra.bc1 = 1.0 - pow((double)beta1, (double)t);
    ra.bc2 = 1.0 - pow((double)beta2, (double)t);
    ua.count = pa.count = cn;
    ua.r = pa.r = r;
    ua.rp = pa.rp = rp;
    ua.bf16 = bf16;
    ua.lr = lr;
    long long us_total = 0;
    int wg_total = 0;
    for (int k = 0; k < cn; ++k) {
      const zo_update_item& src = items[c0 + k];
      const Layout lay = item_layout(src.m, src.n, r, rp, bf16);
      double* S = (double*)wc.take(lay.s);
      int* skip = (int*)wc.take(lay.skip);
      void* L = wc.take(lay.L);
      void* Vs = lay.Vs ? wc.take(lay.Vs) : nullptr;
      ra.it[k] = ItemRR{src.Z, src.M1, src.M2, src.zbar_out, S, skip};
      ua.it[k] = ItemUS{src.U, src.V, S, skip, L, Vs, src.m, src.n, us_total};
      us_total += (long long)src.m * rp + (bf16 ? (long long)src.n * rp : 0);
      ItemUpd u{};
      u.W = src.W;
      u.wout = src.w_f32_out;
      u.L = L;
      u.Vs = bf16 ? Vs : (const void*)src.V;
      u.skip = skip;
      u.m = src.m;
      u.n = src.n;
      u.wg_begin = wg_total;
      if (bf16) {
        u.strips = (src.n + UPD_COLS - 1) / UPD_COLS;
        wg_total += u.strips * ((src.m + UPD_ROWS - 1) / UPD_ROWS);
      } else {
        u.strips = 1;
        wg_total += (int)(((long long)src.m * src.n + 255) / 256);
      }
      pa.it[k] = u;
    }
    ua.total = us_total;
    hipLaunchKernelGGL(k_adam_rr, dim3(cn), dim3(256), 0, stream, ra);
    if ((st = zo_hip_status(hipGetLastError(), "k_adam_rr")) != ZO_OK) return st;
    hipLaunchKernelGGL(k_us, dim3((unsigned)((us_total + 255) / 256)), dim3(256), 0, stream, ua);
    if ((st = zo_hip_status(hipGetLastError(), "k_us")) != ZO_OK) return st;
    if (wg_total > 0) {
      if (!bf16) {
        hipLaunchKernelGGL(k_update_f32, dim3(wg_total), dim3(256), 0, stream, pa);
      } else {
        switch (rp / 32) {
          case 1: hipLaunchKernelGGL(k_update_bf16<1>, dim3(wg_total), dim3(256), 0, stream, pa); break;
          case 2: hipLaunchKernelGGL(k_update_bf16<2>, dim3(wg_total), dim3(256), 0, stream, pa); break;
          case 3: hipLaunchKernelGGL(k_update_bf16<3>, dim3(wg_total), dim3(256), 0, stream, pa); break;
          default: hipLaunchKernelGGL(k_update_bf16<4>, dim3(wg_total), dim3(256), 0, stream, pa); break;
        }
      }
      if ((st = zo_hip_status(hipGetLastError(), "k_update")) != ZO_OK) return st;
    }
  }
  return ZO_OK;
}

// The network a SubZero+ query evaluates (the forward inside Eq. 5 / the query
// loop of Alg. 3), as a pre-LN decoder layer of the OPT family whose six weight
// matrices are all perturbed in their own subspaces (Eq. 4):
//   A = LN1(H);  Q, K, V = A Wq'^T, A Wk'^T, A Wv'^T;  C = causal attention;
//   H2 = H + C Wo'^T;  F = relu(LN2(H2) W1'^T);  H3 = H2 + F W2'^T.
// The six products are the perturbed linears of zo_gemm.hip (the ReLU and the
// residual additions fused into their epilogues); this file adds the row
// normalisation, the attention, and the host sequence of one layer.
//
// k_layernorm: one wave per row, three passes over the row (sum, squared
// deviations, output; RMS normalisation skips the first), statistics in fp32
// with fixed-order wave sums.  Rows of
// up to 8192 elements are read once into registers (k_layernorm_reg, NC
// 512-element chunks, every load in flight at once); longer rows are re-read
// by each pass from L1/L2 (k_layernorm).  Both do the same operations in the
// same order, so their results are identical.
//
// k_attention<F16, DH, W>: one workgroup (W = 4 or 8 waves) per (block, sequence,
// head, tile of 32 W queries); keys in tiles of 64 through LDS (loaded into
// registers a tile ahead, both K and V stored row-major), online softmax in
// fp32.  Each wave owns AT_NG = 2 groups of 16 queries that share every K and
// V fragment it reads from LDS (two groups measured 9-18 % faster than one once
// the accumulators sit in VGPRs: 240 registers, two waves per SIMD), skips the
// tiles whose keys all follow its queries, and computes the transposed
// products, which keeps every step in registers:
//   S^T = K Q^T  (v_mfma_f32_16x16x32: A = K rows from LDS, B = the wave's Q
//                 rows held in registers); lane (l16, g) of a 16 x 16 result
//                 holds query l16 and keys 4g .. 4g+3, so a query's softmax
//                 statistics are a sum over its lane and the 4 lanes l16 + 16g;
//   O^T += V^T P^T, 32 keys per MFMA.  The MFMA's k slots of lane group g are
//                 given the keys that lane already holds for P (4g .. 4g+3 of
//                 each of two 16-key tiles); V^T's fragment takes the same keys
//                 from two transposed reads (ds_read_b64_tr_b16) of the
//                 row-major V tile.  A sum over k does not depend on how the k
//                 slots are assigned to keys, as long as both operands use the
//                 same assignment.
// P enters as a hi + lo pair of 16-bit values (two MFMAs), so the product is
// ~2^-16 accurate before the output's rounding; P is computed as
// 2^((s - m) scale + 12) on the raw logits s (the common factor cancels in the
// normalisation and keeps fp16 low parts out of the subnormal range), with the
// running maximum m moved only when a logit exceeds it by more than 2^3.
#include "zo_internal.h"

#include <type_traits>

namespace {

// ---------------------------------------------------------------- layer norm
template <int DT>
__device__ __forceinline__ void load8(const void* X, size_t idx, float* v) {
  if constexpr (DT == ZO_F32) {
    const f32x4 a = *(const f32x4*)((const float*)X + idx);
    const f32x4 b = *(const f32x4*)((const float*)X + idx + 4);
    v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
    v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
  } else {
    const u32x4 u = *(const u32x4*)((const uint16_t*)X + idx);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (DT == ZO_BF16) {
        v[2 * e] = bf16_to_f32((bf16_t)u[e]);
        v[2 * e + 1] = bf16_to_f32((bf16_t)(u[e] >> 16));
      } else {
        v[2 * e] = f16_to_f32((uint16_t)u[e]);
        v[2 * e + 1] = f16_to_f32((uint16_t)(u[e] >> 16));
      }
    }
  }
}

template <int DT>
__device__ __forceinline__ void store8(void* Y, size_t idx, const float* v) {
  if constexpr (DT == ZO_F32) {
    *(f32x4*)((float*)Y + idx) = (f32x4){v[0], v[1], v[2], v[3]};
    *(f32x4*)((float*)Y + idx + 4) = (f32x4){v[4], v[5], v[6], v[7]};
  } else if constexpr (DT == ZO_BF16) {
    *(u32x4*)((uint16_t*)Y + idx) = (u32x4){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                            pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
  } else {
    *(u32x4*)((uint16_t*)Y + idx) = (u32x4){pack_f16x2(v[0], v[1]), pack_f16x2(v[2], v[3]),
                                            pack_f16x2(v[4], v[5]), pack_f16x2(v[6], v[7])};
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Rows of d elements (d % 8 == 0), 4 rows per workgroup, one per wave.  RMS: no centring
// (the mean is taken as 0 and the sum pass skipped) and no beta (fmaf with 0 is the rounded
// product), i.e. x / sqrt(mean(x^2) + eps) * gamma.
template <int DT, bool RMS>
__global__ __launch_bounds__(256) void k_layernorm(const void* __restrict__ X,
                                                   const float* __restrict__ gamma,
                                                   const float* __restrict__ beta, void* Y,
                                                   long long rows, int d, float eps_ln) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const size_t base = (size_t)row * d;
  float v[8];
  float mean = 0.f;
  if constexpr (!RMS) {
    float s = 0.f;
    for (int c = lane * 8; c < d; c += 512) {
      load8<DT>(X, base + c, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[e];
    }
    mean = wave_sum(s) / (float)d;
  }
  float q = 0.f;
  for (int c = lane * 8; c < d; c += 512) {
    load8<DT>(X, base + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) q = fmaf(v[e] - mean, v[e] - mean, q);
  }
  const float rstd = 1.f / sqrtf(wave_sum(q) / (float)d + eps_ln);
  for (int c = lane * 8; c < d; c += 512) {
    load8<DT>(X, base + c, v);
    const f32x4 g0 = *(const f32x4*)(gamma + c), g1 = *(const f32x4*)(gamma + c + 4);
    f32x4 b0 = {0.f, 0.f, 0.f, 0.f}, b1 = {0.f, 0.f, 0.f, 0.f};
    if constexpr (!RMS) {
      b0 = *(const f32x4*)(beta + c);
      b1 = *(const f32x4*)(beta + c + 4);
    }
    const float g[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
    const float b[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = fmaf((v[e] - mean) * rstd, g[e], b[e]);
    store8<DT>(Y, base + c, v);
  }
}

// Rows of d <= 512 NC elements held in registers as loaded (8 elements per lane and chunk:
// one 16-byte word for 16-bit types, two for fp32), widened to fp32 at each use (exact).
template <int DT>
struct Raw8 {
  static constexpr int W = DT == ZO_F32 ? 2 : 1;
  u32x4 w[W];
  __device__ __forceinline__ void load(const void* X, size_t idx) {
    const u32x4* p = DT == ZO_F32 ? (const u32x4*)((const float*)X + idx) : (const u32x4*)((const uint16_t*)X + idx);
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = p[i];
  }
  __device__ __forceinline__ float at(int e) const {
    if constexpr (DT == ZO_F32) return __uint_as_float(w[e >> 2][e & 3]);
    const uint32_t u = w[0][e >> 1];
    const uint16_t h = (uint16_t)((e & 1) ? (u >> 16) : u);
    if constexpr (DT == ZO_BF16) return bf16_to_f32((bf16_t)h);
    return f16_to_f32(h);
  }
};

template <int DT, int NC, bool RMS>
__global__ __launch_bounds__(256) void k_layernorm_reg(const void* __restrict__ X,
                                                       const float* __restrict__ gamma,
                                                       const float* __restrict__ beta, void* Y,
                                                       long long rows, int d, float eps_ln) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int lane = threadIdx.x & 63;
  const size_t base = (size_t)row * d;
  Raw8<DT> v[NC];
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int c = lane * 8 + 512 * k;
    if (c < d) v[k].load(X, base + c);
  }
  float mean = 0.f;
  if constexpr (!RMS) {
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      if (lane * 8 + 512 * k < d) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s += v[k].at(e);
      }
    }
    mean = wave_sum(s) / (float)d;
  }
  float q = 0.f;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    if (lane * 8 + 512 * k < d) {
#pragma unroll
      for (int e = 0; e < 8; ++e) q = fmaf(v[k].at(e) - mean, v[k].at(e) - mean, q);
    }
  }
  const float rstd = 1.f / sqrtf(wave_sum(q) / (float)d + eps_ln);
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int c = lane * 8 + 512 * k;
    if (c < d) {
      const f32x4 g0 = *(const f32x4*)(gamma + c), g1 = *(const f32x4*)(gamma + c + 4);
      f32x4 b0 = {0.f, 0.f, 0.f, 0.f}, b1 = {0.f, 0.f, 0.f, 0.f};
      if constexpr (!RMS) {
        b0 = *(const f32x4*)(beta + c);
        b1 = *(const f32x4*)(beta + c + 4);
      }
      const float g[8] = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
      const float b[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = fmaf((v[k].at(e) - mean) * rstd, g[e], b[e]);
      store8<DT>(Y, base + c, o);
    }
  }
}

// Rotary positions, in place.  A thread owns 8 dimensions i of the first half of one head
// (and their partners dh/2 further on) in ROPE_RB consecutive rows.  The frequency
// 2^(i k), k = -2 log2(base) / dh, is formed once per thread in fp64; each angle p 2^(i k)
// is formed and reduced to [-pi, pi] in fp64, so that sincosf sees an argument that is
// exact to fp32 rounding at any position (a direct fp32 product p * theta would carry an
// absolute error of about p * 2^-24 radians: 2.4e-4 at p = 4095, a quarter of a bf16 ulp).
constexpr int ROPE_RB = 8;

template <int DT>
__global__ __launch_bounds__(256) void k_rope(void* X, long long rows, int seq_len, int d, int dh, double k) {
  const int cpr = d / 16;   // (head, 8-dimension chunk) pairs per row
  const int cph = dh / 16;  // chunks per half head
  const long long t = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long groups = (rows + ROPE_RB - 1) / ROPE_RB;
  if (t >= groups * cpr) return;
  const int cc = (int)(t % cpr);
  const int h = cc / cph, c = cc % cph;
  const long long r0 = (t / cpr) * ROPE_RB;
  const long long r1 = r0 + ROPE_RB < rows ? r0 + ROPE_RB : rows;
  double theta[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) theta[e] = exp2((double)(8 * c + e) * k);
  constexpr double kTwoPi = 6.283185307179586, kInvTwoPi = 0.15915494309189535;
  for (long long row = r0; row < r1; ++row) {
    const double pos = (double)(row % seq_len);
    const size_t ia = (size_t)row * d + (size_t)h * dh + 8 * c, ib = ia + dh / 2;
    float a[8], b[8], na[8], nb[8];
    load8<DT>(X, ia, a);
    load8<DT>(X, ib, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const double ang = pos * theta[e];
      const float red = (float)fma(-rint(ang * kInvTwoPi), kTwoPi, ang);
      float sn, cs;
      sincosf(red, &sn, &cs);
      na[e] = a[e] * cs - b[e] * sn;
      nb[e] = b[e] * cs + a[e] * sn;
    }
    store8<DT>(X, ia, na);
    store8<DT>(X, ib, nb);
  }
}

// ---------------------------------------------------------------- attention
constexpr int AT_NG = 2;               // 16-query groups per wave
// Waves per workgroup: 4, or 8 for sequences of 512 or more (the K/V tile a workgroup loads
// then serves 256 queries; at 256 keys per sequence the causal tiles 8 waves would walk in
// step cost more than that saves).
constexpr int AT_K = 64;               // keys per tile

struct AttnArgs {
  const void* Q;
  const void* K;
  const void* V;
  void* O;
  int T, seq_len, d, heads, qtiles;  // qtiles = ceil(seq_len / queries per workgroup)
  int dkv, group;                    // K/V row length (kv_heads dh); query heads per K/V head
  float scale_log2;                  // log2(e) / sqrt(dh)
};

template <bool F16>
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                   __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Two fp32 values rounded to nearest even into a packed pair of 16-bit values (one
// v_cvt_pk_bf16_f32 / v_cvt_pk_f16_f32), and back.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
template <bool F16>
__device__ __forceinline__ uint32_t cvt_pk(float x, float y) {
  if constexpr (F16)
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){x, y}, f16x2_t));
  else
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){x, y}, bf16x2_t));
}
template <bool F16>
__device__ __forceinline__ float unpk(uint32_t pk, int half) {
  const uint16_t h = (uint16_t)(half ? pk >> 16 : pk);
  if constexpr (F16)
    return f16_to_f32(h);
  else
    return bf16_to_f32(h);
}

typedef short i16x4_t __attribute__((ext_vector_type(4)));
// ds_read_b64_tr_b16: within each 16-lane group, lane i reads 4 consecutive 16-bit values
// D[i][0..3] at its own address, and lane j receives D[j/4 + 4e][j%4] for e = 0..3.  With
// lane i addressing row (r0 + i/4), columns c0 + 4 (i%4) of a row-major tile, lane j thus
// receives column c0 + j of rows r0 .. r0+3: a transposed fragment.
__device__ __forceinline__ u32x2 ds_read_tr(const uint16_t* p) {
  const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4_t*)(p));
  return __builtin_bit_cast(u32x2, v);
}

template <bool F16, int DH, int W>
__global__ __launch_bounds__(64 * W) void k_attention(AttnArgs a) {
  constexpr int NT = 64 * W;              // threads
  constexpr int AT_Q = 16 * AT_NG * W;    // queries per workgroup
  constexpr int KS = DH / 32;         // 32-deep k steps of Q K^T
  constexpr int DT = DH / 16;         // 16-dim tiles of the output
  constexpr int KROW = DH + 8;        // LDS row of the K tile (elements), padded
  constexpr int VROW = DH + 16;       // LDS row of the V tile (elements): 16 rows of a
                                      // transposed read fall on distinct banks
  constexpr int C8 = DH / 8;          // 16-byte chunks per head row
  constexpr int KCH = AT_K * C8 / NT;    // K (and V) chunks per thread per tile
  static_assert(KCH * NT == AT_K * C8, "tile / thread mismatch");
  __shared__ __attribute__((aligned(16))) uint16_t Ks[AT_K * KROW];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[AT_K * VROW];

  // Workgroup -> (block, sequence, head, query tile).
  int w = blockIdx.x;
  const int qt = w % a.qtiles;
  w /= a.qtiles;
  const int head = w % a.heads;
  w /= a.heads;
  const int nseq = a.T / a.seq_len;
  const int seq = w % nseq;
  const int blk = w / nseq;
  const long long row0 = (long long)blk * a.T + (long long)seq * a.seq_len;  // first row of the sequence
  const int col0 = head * DH;
  const int col0kv = (head / a.group) * DH;  // the key/value head of this query head
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, g = lane >> 4;
  const int q0 = qt * AT_Q;  // first query of the tile (within the sequence)
  const uint16_t* __restrict__ Kg = (const uint16_t*)a.K;
  const uint16_t* __restrict__ Vg = (const uint16_t*)a.V;

  // This lane's queries (one per group) and their rows as B operands of S^T = K Q^T.
  int myq[AT_NG];
  bf16x8 qf[AT_NG][KS];
#pragma unroll
  for (int gq = 0; gq < AT_NG; ++gq) {
    myq[gq] = q0 + wave * 16 * AT_NG + 16 * gq + l16;
    const int qc = min(myq[gq], a.seq_len - 1);
    const uint16_t* qp = (const uint16_t*)a.Q + (size_t)(row0 + qc) * a.d + col0 + 8 * g;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      qf[gq][kk] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + 32 * kk));
  }
  const int wq0 = q0 + wave * 16 * AT_NG;  // the wave's first query

  f32x4 o[AT_NG][DT];
  float mrow[AT_NG], lsum[AT_NG];
#pragma unroll
  for (int gq = 0; gq < AT_NG; ++gq) {
#pragma unroll
    for (int t = 0; t < DT; ++t) o[gq][t] = (f32x4){0.f, 0.f, 0.f, 0.f};
    mrow[gq] = -1e30f;  // running max of the raw logits
    lsum[gq] = 0.f;     // this lane's part of the running sum
  }

  // K and V tiles are loaded into registers a tile ahead: chunk x = tid + NT c is key x / C8,
  // dims 8 (x % C8); both are stored row-major (V is read transposed by ds_read_tr).  Rows
  // past the sequence are clamped to its last row (their keys are masked).
  u32x4 kreg[KCH], vreg[KCH];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      const int x = tid + NT * c;
      const size_t off = (size_t)(row0 + min(k0 + x / C8, a.seq_len - 1)) * a.dkv + col0kv + 8 * (x % C8);
      kreg[c] = *(const u32x4*)(Kg + off);
      vreg[c] = *(const u32x4*)(Vg + off);
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int c = 0; c < KCH; ++c) {
      const int x = tid + NT * c;
      *(u32x4*)&Ks[(x / C8) * KROW + 8 * (x % C8)] = kreg[c];
      *(u32x4*)&Vs[(x / C8) * VROW + 8 * (x % C8)] = vreg[c];
    }
  };

  const int kend = min(a.seq_len, q0 + AT_Q);  // keys beyond the tile's last query are never seen
  load_tile(0);
  for (int k0 = 0; k0 < kend; k0 += AT_K) {
    __syncthreads();  // the previous tile has been consumed
    store_tile();
    __syncthreads();
    if (k0 + AT_K < kend) load_tile(k0 + AT_K);
    if (k0 > wq0 + 16 * AT_NG - 1) continue;  // every key of the tile is after the wave's queries

    // S^T for 4 key subtiles of 16: st[gq][t][i] = key k0 + 16 t + 4 g + i, query myq[gq].
    f32x4 st[AT_NG][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int gq = 0; gq < AT_NG; ++gq) st[gq][t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8 kf = *(const bf16x8*)&Ks[(16 * t + l16) * KROW + 32 * kk + 8 * g];
#pragma unroll
        for (int gq = 0; gq < AT_NG; ++gq) st[gq][t] = mfma16<F16>(kf, qf[gq][kk], st[gq][t]);
      }
    }
    // Mask keys after the query (only a tile that reaches past the wave's first query has
    // any), online softmax on the raw logits, P = 2^((s - m) scale + 12) as hi + lo 16-bit
    // pairs in the B-operand order of the P V MFMA.  The running maximum m moves only when
    // some query of the wave has a logit more than 3 (log2 units) above it, so most tiles
    // skip the rescale of O; P then stays below 2^15 (within fp16's range), and the first
    // tile sets m to its row maximum, whose P is exactly 2^12.
    const bool diag = k0 + AT_K - 1 > wq0;
    uint32_t ph[AT_NG][4][2], pl[AT_NG][4][2];
#pragma unroll
    for (int gq = 0; gq < AT_NG; ++gq) {
      float tmax = -1e30f;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if (diag && k0 + 16 * t + 4 * g + i > myq[gq]) st[gq][t][i] = -INFINITY;
          tmax = fmaxf(tmax, st[gq][t][i]);
        }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
      if (__ballot((tmax - mrow[gq]) * a.scale_log2 > 3.f)) {
        const float mnew = fmaxf(mrow[gq], tmax);
        const float alpha = __builtin_amdgcn_exp2f((mrow[gq] - mnew) * a.scale_log2);
        mrow[gq] = mnew;
        lsum[gq] *= alpha;
#pragma unroll
        for (int t = 0; t < DT; ++t) o[gq][t] *= alpha;
      }
      const float m = mrow[gq];
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; i += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(st[gq][t][i] - m, a.scale_log2, 12.f));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(st[gq][t][i + 1] - m, a.scale_log2, 12.f));
          lsum[gq] += p0 + p1;
          const uint32_t h = cvt_pk<F16>(p0, p1);
          ph[gq][t][i / 2] = h;
          pl[gq][t][i / 2] = cvt_pk<F16>(p0 - unpk<F16>(h, 0), p1 - unpk<F16>(h, 1));
        }
    }
    // O^T += V^T P^T over two 32-key chunks c (subtiles 2c and 2c+1): lane group g's k slots
    // are keys 32c + 4g + (0..3) and 32c + 16 + 4g + (0..3); V^T's fragment (dim 16t + l16 of
    // those keys) comes from two transposed reads of the row-major V tile.
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      bf16x8 bh[AT_NG], bl[AT_NG];
#pragma unroll
      for (int gq = 0; gq < AT_NG; ++gq) {
        bh[gq] = __builtin_bit_cast(bf16x8, (u32x4){ph[gq][2 * c][0], ph[gq][2 * c][1], ph[gq][2 * c + 1][0],
                                                    ph[gq][2 * c + 1][1]});
        bl[gq] = __builtin_bit_cast(bf16x8, (u32x4){pl[gq][2 * c][0], pl[gq][2 * c][1], pl[gq][2 * c + 1][0],
                                                    pl[gq][2 * c + 1][1]});
      }
      const uint16_t* vb = &Vs[(32 * c + 4 * g + (l16 >> 2)) * VROW + 4 * (l16 & 3)];
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const u32x2 v0 = ds_read_tr(vb + 16 * t), v1 = ds_read_tr(vb + 16 * VROW + 16 * t);
        const bf16x8 af = __builtin_bit_cast(bf16x8, (u32x4){v0[0], v0[1], v1[0], v1[1]});
#pragma unroll
        for (int gq = 0; gq < AT_NG; ++gq) {
          o[gq][t] = mfma16<F16>(af, bh[gq], o[gq][t]);
          o[gq][t] = mfma16<F16>(af, bl[gq], o[gq][t]);
        }
      }
    }
  }
  // Normalise by the row sums (over the 4 lane groups) and store dims 16 t + 4 g .. +3.
#pragma unroll
  for (int gq = 0; gq < AT_NG; ++gq) {
    float l = lsum[gq] + __shfl_xor(lsum[gq], 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (myq[gq] >= a.seq_len) continue;
    const float inv = 1.f / l;
    uint16_t* op = (uint16_t*)a.O + (size_t)(row0 + myq[gq]) * a.d + col0 + 4 * g;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const float y0 = o[gq][t][0] * inv, y1 = o[gq][t][1] * inv;
      const float y2 = o[gq][t][2] * inv, y3 = o[gq][t][3] * inv;
      const u32x2 pk = F16 ? (u32x2){pack_f16x2(y0, y1), pack_f16x2(y2, y3)}
                           : (u32x2){pack_bf16x2(y0, y1), pack_bf16x2(y2, y3)};
      *(u32x2*)(op + 16 * t) = pk;
    }
  }
}

// Register-resident rows in buckets of 2, 4, 8, 10 or 16 chunks of 512; longer rows re-read.
template <int DT, bool RMS>
void layernorm_dispatch(dim3 grid, dim3 block, hipStream_t stream, const void* X, const float* gamma,
                        const float* beta, void* Y, long long rows, int d, float eps_ln) {
  if (d <= 1024)
    hipLaunchKernelGGL((k_layernorm_reg<DT, 2, RMS>), grid, block, 0, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else if (d <= 2048)
    hipLaunchKernelGGL((k_layernorm_reg<DT, 4, RMS>), grid, block, 0, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else if (d <= 4096)
    hipLaunchKernelGGL((k_layernorm_reg<DT, 8, RMS>), grid, block, 0, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else if (d <= 5120)
    hipLaunchKernelGGL((k_layernorm_reg<DT, 10, RMS>), grid, block, 0, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else if (d <= 8192)
    hipLaunchKernelGGL((k_layernorm_reg<DT, 16, RMS>), grid, block, 0, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else
    hipLaunchKernelGGL((k_layernorm<DT, RMS>), grid, block, 0, stream, X, gamma, beta, Y, rows, d, eps_ln);
}

template <int DT>
void layernorm_dispatch_rms(bool rms, dim3 grid, dim3 block, hipStream_t stream, const void* X,
                            const float* gamma, const float* beta, void* Y, long long rows, int d,
                            float eps_ln) {
  if (rms)
    layernorm_dispatch<DT, true>(grid, block, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else
    layernorm_dispatch<DT, false>(grid, block, stream, X, gamma, beta, Y, rows, d, eps_ln);
}

}  // namespace

int zo_layernorm_launch(long long rows, int d, int dtype, const void* X, const float* gamma,
                        const float* beta, float eps_ln, void* Y, hipStream_t stream, bool rms) {
  if (rows <= 0) return ZO_OK;
  const dim3 grid((unsigned)((rows + 3) / 4)), block(256);
  if (dtype == ZO_BF16)
    layernorm_dispatch_rms<ZO_BF16>(rms, grid, block, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else if (dtype == ZO_F16)
    layernorm_dispatch_rms<ZO_F16>(rms, grid, block, stream, X, gamma, beta, Y, rows, d, eps_ln);
  else
    layernorm_dispatch_rms<ZO_F32>(rms, grid, block, stream, X, gamma, beta, Y, rows, d, eps_ln);
  return zo_hip_status(hipGetLastError(), "k_layernorm");
}

int zo_rope_launch(long long rows, int seq_len, int d, int heads, int dtype, void* X, float base,
                   hipStream_t stream) {
  const int dh = d / heads;
  const long long threads = (rows + ROPE_RB - 1) / ROPE_RB * (d / 16);
  if (threads <= 0) return ZO_OK;
  const long long wg = (threads + 255) / 256;
  if (wg > 0x7fffffffLL) {
    zo_set_error("rope: too many rows (%lld)", rows);
    return ZO_ERR_UNSUPPORTED;
  }
  const double k = -2.0 * log2((double)base) / (double)dh;
  if (dtype == ZO_BF16)
    hipLaunchKernelGGL(k_rope<ZO_BF16>, dim3((unsigned)wg), dim3(256), 0, stream, X, rows, seq_len, d, dh, k);
  else
    hipLaunchKernelGGL(k_rope<ZO_F16>, dim3((unsigned)wg), dim3(256), 0, stream, X, rows, seq_len, d, dh, k);
  return zo_hip_status(hipGetLastError(), "k_rope");
}

int zo_attention_launch(int nblk, int T, int seq_len, int d, int heads, int kv_heads, int dtype,
                        const void* Q, const void* K, const void* V, void* O, hipStream_t stream) {
  AttnArgs a;
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.O = O;
  a.T = T;
  a.seq_len = seq_len;
  a.d = d;
  a.heads = heads;
  a.dkv = d / heads * kv_heads;
  a.group = heads / kv_heads;
  const int W = seq_len >= 512 ? 8 : 4;
  const int qpw = 16 * AT_NG * W;
  a.qtiles = (seq_len + qpw - 1) / qpw;
  const int dh = d / heads;
  a.scale_log2 = 1.4426950408889634f / sqrtf((float)dh);
  const long long wg = (long long)nblk * (T / seq_len) * heads * a.qtiles;
  if (wg <= 0) return ZO_OK;
  if (wg > 0x7fffffffLL) {
    zo_set_error("attention: too many workgroups (%lld)", wg);
    return ZO_ERR_UNSUPPORTED;
  }
  const dim3 grid((unsigned)wg), block(64 * W);
  const bool f16 = dtype == ZO_F16;
#define ZO_ATTN(F, D, WW) hipLaunchKernelGGL((k_attention<F, D, WW>), grid, block, 0, stream, a)
  if (W == 8) {
    if (dh == 64) {
      if (f16) ZO_ATTN(true, 64, 8); else ZO_ATTN(false, 64, 8);
    } else {
      if (f16) ZO_ATTN(true, 128, 8); else ZO_ATTN(false, 128, 8);
    }
  } else {
    if (dh == 64) {
      if (f16) ZO_ATTN(true, 64, 4); else ZO_ATTN(false, 64, 4);
    } else {
      if (f16) ZO_ATTN(true, 128, 4); else ZO_ATTN(false, 128, 4);
    }
  }
#undef ZO_ATTN
  return zo_hip_status(hipGetLastError(), "k_attention");
}

// Perturbed linear layer of SubZero+ (Eq. 4 inside the forward of Eq. 5).
//
//   Y_b = X_b W^T + (X_b V) (s_b eps U Z_{j(b)})^T
//
// Launches per call (bf16 inputs):
//   1. k_transpose_v : V (n x r fp32) -> Vt2 (2 rp x n bf16): rows [0, rp) the
//                      high bf16 part of V^T, rows [rp, 2 rp) the low part
//                      (V = hi + lo to ~16 bits); rp = r rounded up to 32
//                      (16 for fp32 inputs).
//   2. k_bprime      : B_b = s_b eps U Z_{j(b)} (fp32) written as the K segment
//                      [B_hi | B_lo | B_hi] (bf16, 3 rp wide), every block.
//   3. projection    : P = X_x Vt2_hi^T + X_x Vt2_lo^T of every distinct X block,
//                      written as the K segment [P_hi | P_hi | P_lo] (bf16,
//                      3 rp wide).  k_proj for one factor of 64 or 128 rows
//                      (or a pair of 64), the main GEMM with the EPI_PROJ
//                      epilogues for a stack of factors that read the same X;
//                      otherwise an fp32 projection followed by k_pcombine.
//   4. main GEMM     : Y_b = X_b W^T + P_{x(b)} B_b^T, the rank-r term added as
//                      one more 3 rp-deep K segment into the same fp32
//                      accumulators: hi*hi + hi*lo + lo*hi, so the correction
//                      carries ~2^-16 relative error instead of the 2^-8 of
//                      plain bf16 operands.
// fp16 inputs: the same launches.  X W^T runs on the fp16 MFMA; the rank-r
// segment keeps its bf16 hi/lo operands (eps U Z_j entries are near fp16's
// smallest normal, and bf16 has fp32's range) on the bf16 MFMA, as more
// k-tiles of the same pipeline.  The projection X_x Vt2^T runs on the fp16
// MFMA with Vt2 the fp16 hi/lo split of 256 V (the low parts of entries near
// 1/sqrt(n) then stay normal); the combine multiplies by 1/256 (exact).
// fp32 inputs: Vt (rp x n), P = X Vt^T and B_b in fp32, fp32 FMA throughout.
//
// The main GEMM (k_gemm_main) is described where it is defined.  The
// register-staged GEMM (k_gemm_bf16: the projection of wide factors and the
// fallback when K is not a multiple of 32) computes a BM x BN tile of Y_b^T
// with v_mfma_f32_32x32x16_bf16: the A operand is the W tile (rows = output
// columns), the B operand the X tile (rows = tokens), both K-contiguous and
// staged through LDS in 128-byte rows with an XOR swizzle of the 16-byte
// chunks, double buffered.  Workgroup ids are remapped so that the tiles one
// XCD runs concurrently are contiguous, then grouped 8 token tiles deep so the
// tiles in flight on an XCD share their W and X panels in that XCD's L2.
#include "zo_internal.h"

#include <type_traits>

namespace {

constexpr int BK = 64;  // bf16 elements per K tile = 128 bytes per LDS row

// Internal epilogues of the shared-X fan-out (beyond zo_epilogue's values): R is an fp32 T x m
// base X W^T shared by every block, added to the block's rank-r term before the rounding.
constexpr int EPI_BASE = 16;       // Y_b = base + result
constexpr int EPI_BASE_RELU = 17;  // Y_b = max(base + result, 0)
// The prepare's projection of a stack of 16-bit factors (A = the stacked [V_hi; V_lo] rows, 2 rp
// per factor, rp = 32 or 64): P = (hi part + lo part) * unscale of every factor, written to the
// factor's own buffer as [P_hi | P_hi | P_lo] (bf16, 3 rp per token); Y is not used.
constexpr int EPI_PROJ32 = 18;
constexpr int EPI_PROJ64 = 19;

// Swizzle of the 16-byte chunk index within a 128-byte LDS row; conflict free
// for ds_read_b128 of 8 or 16 consecutive rows at one logical chunk.
__device__ __forceinline__ int swz(int row) { return ((row >> 1) ^ ((row & 1) << 2)) & 7; }

struct GemmArgs {
  const bf16_t* A;            // rows_a x K (shared by all blocks)
  const bf16_t* B;            // per block rows_b x K
  long long b_block_stride;   // elements; 0 = shared
  int rows_a, rows_b, K, nblk;
  const bf16_t* ca;           // correction A operand: per block rows_a x rc
  long long ca_block_stride;
  const bf16_t* cb;           // correction B operand: per block rows_b x rc
  long long cb_block_stride;
  int rc;                     // multiple of 16; 0 = no correction
  void* Y;                    // per block rows_b x ldy
  long long y_block_stride;
  int ldy, out_dtype;          // zo_dtype of Y
  int epi;                     // zo_epilogue
  const void* R;               // ZO_EPI_RESIDUAL / SILU_MUL: same type and layout as Y (ldy)
  long long r_block_stride;    // elements; 0 = one R shared by all blocks
  int tiles_a, tiles_b, total_tiles;
  int blk_inner;               // k_gemm_main: 1 = the blocks of one output tile run consecutively
  // EPI_PROJ32 / EPI_PROJ64: factor f's output (nblk x rows_b tokens x 3 rp), the number of
  // factors, and the scale of the combined projection (1, or 1/256 for fp16 inputs).
  bf16_t* pc[ZO_MAX_GROUP];
  int pcount;
  float unscale;
};

// Four fp32 accumulator values as element idx.. of an OUT-typed (zo_dtype) array.
template <int OUT>
__device__ __forceinline__ void store4(char* base, size_t idx, float v0, float v1, float v2,
                                       float v3) {
  if constexpr (OUT == ZO_BF16)
    *(u32x2*)(base + idx * 2) = (u32x2){pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
  else if constexpr (OUT == ZO_F16)
    *(u32x2*)(base + idx * 2) = (u32x2){pack_f16x2(v0, v1), pack_f16x2(v2, v3)};
  else
    *(f32x4*)(base + idx * 4) = (f32x4){v0, v1, v2, v3};
}

// Four OUT-typed values at element idx.. as fp32.
template <int OUT>
__device__ __forceinline__ f32x4 load4(const char* base, size_t idx) {
  if constexpr (OUT == ZO_F32) {
    return *(const f32x4*)(base + idx * 4);
  } else {
    const u32x2 r = *(const u32x2*)(base + idx * 2);
    if constexpr (OUT == ZO_BF16)
      return (f32x4){bf16_to_f32((bf16_t)r[0]), bf16_to_f32((bf16_t)(r[0] >> 16)),
                     bf16_to_f32((bf16_t)r[1]), bf16_to_f32((bf16_t)(r[1] >> 16))};
    else
      return (f32x4){f16_to_f32((uint16_t)r[0]), f16_to_f32((uint16_t)(r[0] >> 16)),
                     f16_to_f32((uint16_t)r[1]), f16_to_f32((uint16_t)(r[1] >> 16))};
  }
}

// Four OUT-typed values at element idx.. as fp32, added to v0..v3.
template <int OUT>
__device__ __forceinline__ void add4(const char* base, size_t idx, float& v0, float& v1, float& v2,
                                     float& v3) {
  const f32x4 r = load4<OUT>(base, idx);
  v0 += r[0]; v1 += r[1]; v2 += r[2]; v3 += r[3];
}

// silu(x) = x / (1 + e^-x) from the hardware exponential and reciprocal (about 1 ulp each,
// so a few fp32 ulps in all, far below the output's 16-bit rounding): the IEEE expf and
// division cost ~28 VALU instructions per element, and the epilogue of a 256 x 256 tile
// applies it to 256 values per lane while the matrix cores idle.  e^-x overflows to +inf
// for x < -88, and the reciprocal then gives 0: silu(x) -> -0, its limit.
__device__ __forceinline__ float silu(float x) {
  return x * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(x * -1.4426950408889634f));
}

// v0..v3 multiplied by silu of the four OUT-typed values at element idx.. (fp32).
template <int OUT>
__device__ __forceinline__ void mul4_silu(const char* base, size_t idx, float& v0, float& v1, float& v2,
                                          float& v3) {
  const f32x4 r = load4<OUT>(base, idx);
  v0 *= silu(r[0]); v1 *= silu(r[1]); v2 *= silu(r[2]); v3 *= silu(r[3]);
}

// The fused epilogue on four fp32 accumulator values, then the store: ReLU, the residual R
// (same layout as Y) added, or the product with silu(R), before the single rounding to OUT.
// Eight OUT-typed values at element idx.. as fp32 (16-bit: one 16-byte load; fp32: element
// loads, since an fp32 R need only be 4-byte aligned).
template <int OUT>
__device__ __forceinline__ void load8(const char* base, size_t idx, float* v) {
  if constexpr (OUT == ZO_F32) {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = ((const float*)base)[idx + e];
  } else {
    const u32x4 r = *(const u32x4*)(base + idx * 2);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if constexpr (OUT == ZO_BF16) {
        v[2 * e] = bf16_to_f32((bf16_t)r[e]);
        v[2 * e + 1] = bf16_to_f32((bf16_t)(r[e] >> 16));
      } else {
        v[2 * e] = f16_to_f32((uint16_t)r[e]);
        v[2 * e + 1] = f16_to_f32((uint16_t)(r[e] >> 16));
      }
    }
  }
}

// Eight fp32 values stored as OUT at element idx.. (idx a multiple of 8, 16-byte aligned rows).
template <int OUT>
__device__ __forceinline__ void store8(char* base, size_t idx, const float* v) {
  if constexpr (OUT == ZO_F32) {
    *(f32x4*)(base + idx * 4) = (f32x4){v[0], v[1], v[2], v[3]};
    *(f32x4*)(base + idx * 4 + 16) = (f32x4){v[4], v[5], v[6], v[7]};
  } else if constexpr (OUT == ZO_BF16) {
    *(u32x4*)(base + idx * 2) = (u32x4){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                        pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
  } else {
    *(u32x4*)(base + idx * 2) = (u32x4){pack_f16x2(v[0], v[1]), pack_f16x2(v[2], v[3]),
                                        pack_f16x2(v[4], v[5]), pack_f16x2(v[6], v[7])};
  }
}

template <int OUT, int EPI>
__device__ __forceinline__ void finish4(char* Yb, const char* Rb, size_t idx, float v0, float v1,
                                        float v2, float v3) {
  if constexpr (EPI == ZO_EPI_RELU) {
    v0 = fmaxf(v0, 0.f); v1 = fmaxf(v1, 0.f); v2 = fmaxf(v2, 0.f); v3 = fmaxf(v3, 0.f);
  } else if constexpr (EPI == ZO_EPI_RESIDUAL) {
    add4<OUT>(Rb, idx, v0, v1, v2, v3);
  } else if constexpr (EPI == ZO_EPI_SILU_MUL) {
    mul4_silu<OUT>(Rb, idx, v0, v1, v2, v3);
  }
  store4<OUT>(Yb, idx, v0, v1, v2, v3);
}

// The same with the output type and epilogue chosen at run time (kernels with few
// accumulators live).
template <int OUT>
__device__ __forceinline__ void finish4_epi(char* Yb, const char* Rb, size_t idx, int epi, float v0,
                                            float v1, float v2, float v3) {
  if (epi == ZO_EPI_RELU)
    finish4<OUT, ZO_EPI_RELU>(Yb, Rb, idx, v0, v1, v2, v3);
  else if (epi == ZO_EPI_RESIDUAL)
    finish4<OUT, ZO_EPI_RESIDUAL>(Yb, Rb, idx, v0, v1, v2, v3);
  else if (epi == ZO_EPI_SILU_MUL)
    finish4<OUT, ZO_EPI_SILU_MUL>(Yb, Rb, idx, v0, v1, v2, v3);
  else
    finish4<OUT, ZO_EPI_NONE>(Yb, Rb, idx, v0, v1, v2, v3);
}
__device__ __forceinline__ void finish4_rt(char* Yb, const char* Rb, size_t idx, int out_dtype,
                                           int epi, float v0, float v1, float v2, float v3) {
  if (out_dtype == ZO_BF16)
    finish4_epi<ZO_BF16>(Yb, Rb, idx, epi, v0, v1, v2, v3);
  else if (out_dtype == ZO_F16)
    finish4_epi<ZO_F16>(Yb, Rb, idx, epi, v0, v1, v2, v3);
  else
    finish4_epi<ZO_F32>(Yb, Rb, idx, epi, v0, v1, v2, v3);
}

// 32x32x16 MFMA on 16-byte fragments of eight 16-bit values: fp16 or bf16.
template <bool F16>
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                   __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 16x16x32 MFMA on 16-byte fragments of eight 16-bit values, fp16 or bf16, accumulating in place
// into c.  Lane l holds row l % 16 of A (and of B's transpose) at k (l / 16) 8 .. + 7; the
// result's lane l holds rows 4 (l / 16) .. + 3 of column l % 16.
//
// Written as inline assembly with c tied to the destination in AGPRs.  With the builtin, a
// kernel holding 64 such accumulators next to 128 fragment registers (every VGPR and AGPR in
// use) gets the untied form for part of its MFMAs: those write a fresh AGPR quad, and each
// trip round the loop then starts with ~300 AGPR/VGPR copies that put the accumulators back.
// The hazard recognizer does not look inside inline assembly, so the caller provides what it
// would: 2 wait states between a VALU write of c and the first MFMA reading it, and 12 (8
// passes + 4) between the last MFMA and any other instruction reading or writing c.  Fragment
// registers are only ever sources A and B, which need no wait before being overwritten.
template <bool F16>
__device__ __forceinline__ void mfma16(f32x4& c, bf16x8 a, bf16x8 b) {
  if constexpr (F16)
    asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
  else
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

template <int WM, int WN, int TM, int TN, bool F16>
__global__ __launch_bounds__(WM* WN * 64) void k_gemm_bf16(GemmArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int BM = WM * TM * 32;
  constexpr int BN = WN * TN * 32;
  constexpr int CA = BM * 8 / NT;
  constexpr int CB = BN * 8 / NT;
  constexpr int RSTEP = NT / 8;
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0, "tile/thread mismatch");
  static_assert(RSTEP % 16 == 0, "swizzle must be invariant over the row step");
  __shared__ __attribute__((aligned(16))) char lds[2 * (BM + BN) * 128];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WM;
  const int wn = wave / WM;

  // XCD-aware remap: hardware deals workgroup w to XCD w % 8; give each XCD a
  // contiguous range of logical tiles.
  const int w = blockIdx.x;
  const int nt = a.total_tiles;
  const int xcd = w & 7, widx = w >> 3;
  const int lt = xcd * (nt >> 3) + min(xcd, nt & 7) + widx;
  // Grouped raster: 8 token tiles (across blocks) per column sweep.
  constexpr int GROUP = 8;
  const int total_bt = a.nblk * a.tiles_b;
  const int per_group = GROUP * a.tiles_a;
  const int grp = lt / per_group;
  const int first = grp * GROUP;
  const int gsize = min(GROUP, total_bt - first);
  const int rem = lt - grp * per_group;
  const int bt = first + rem % gsize;
  const int at = rem / gsize;
  const int blk = bt / a.tiles_b;
  const int t0 = (bt % a.tiles_b) * BN;
  const int m0 = at * BM;

  const bf16_t* __restrict__ Ag = a.A;
  const bf16_t* __restrict__ Bg = a.B + (long long)blk * a.b_block_stride;

  const int lrow = tid >> 3;
  const int kc = tid & 7;
  const int pc = kc ^ swz(lrow);

  u32x4 ra[CA], rb[CB];
  auto load_tiles = [&](int k0) {
    const int kk = k0 + kc * 8;
    const bool kin = kk < a.K;
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int row = m0 + lrow + RSTEP * i;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (kin && row < a.rows_a) v = *(const u32x4*)(Ag + (size_t)row * a.K + kk);
      ra[i] = v;
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int row = t0 + lrow + RSTEP * i;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (kin && row < a.rows_b) v = *(const u32x4*)(Bg + (size_t)row * a.K + kk);
      rb[i] = v;
    }
  };
  auto store_tiles = [&](int buf) {
    char* la = lds + buf * (BM + BN) * 128;
    char* lb = la + BM * 128;
#pragma unroll
    for (int i = 0; i < CA; ++i) *(u32x4*)(la + (lrow + RSTEP * i) * 128 + pc * 16) = ra[i];
#pragma unroll
    for (int i = 0; i < CB; ++i) *(u32x4*)(lb + (lrow + RSTEP * i) * 128 + pc * 16) = rb[i];
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int fr = lane & 31;
  const int fh = lane >> 5;
  const int fsw = swz(fr);
  auto compute = [&](int buf) {
    const char* la = lds + buf * (BM + BN) * 128;
    const char* lb = la + BM * 128;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int ch = ((ks * 2 + fh) ^ fsw) * 16;
      bf16x8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *(const bf16x8*)(la + (wm * TM * 32 + i * 32 + fr) * 128 + ch);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *(const bf16x8*)(lb + (wn * TN * 32 + j * 32 + fr) * 128 + ch);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<F16>(fa[i], fb[j], acc[i][j]);
    }
  };

  const int nk = (a.K + BK - 1) / BK;
  load_tiles(0);
  store_tiles(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tiles((kt + 1) * BK);
    compute(cur);
    if (kt + 1 < nk) store_tiles(cur ^ 1);
    __syncthreads();
  }

  // Rank-rc correction: one more K segment with operands read straight from
  // global memory (16 bytes per lane per fragment); bf16 for every input type.
  if (a.rc > 0) {
    const bf16_t* __restrict__ Cg = a.ca + (long long)blk * a.ca_block_stride;
    const bf16_t* __restrict__ Dg = a.cb + (long long)blk * a.cb_block_stride;
    for (int k0 = 0; k0 < a.rc; k0 += 16) {
      bf16x8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int row = m0 + wm * TM * 32 + i * 32 + fr;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (row < a.rows_a) v = *(const u32x4*)(Cg + (size_t)row * a.rc + k0 + fh * 8);
        fa[i] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int row = t0 + wn * TN * 32 + j * 32 + fr;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (row < a.rows_b) v = *(const u32x4*)(Dg + (size_t)row * a.rc + k0 + fh * 8);
        fb[j] = __builtin_bit_cast(bf16x8, v);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
  }

  // Store: lane holds token fr (+32j) and 4 adjacent output columns per a.
  const int osz = a.out_dtype == ZO_F32 ? 4 : 2;
  char* Yb = (char*)a.Y + (long long)blk * a.y_block_stride * osz;
  const char* Rb = (const char*)a.R + (long long)blk * a.r_block_stride * osz;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int tok = t0 + wn * TN * 32 + j * 32 + fr;
    if (tok >= a.rows_b) continue;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int col = m0 + wm * TM * 32 + i * 32 + q4 * 8 + fh * 4;
        if (col >= a.rows_a) continue;
        finish4_rt(Yb, Rb, (size_t)tok * a.ldy + col, a.out_dtype, a.epi, acc[i][j][q4 * 4 + 0],
                   acc[i][j][q4 * 4 + 1], acc[i][j][q4 * 4 + 2], acc[i][j][q4 * 4 + 3]);
      }
    }
  }
}

// fp32 path: plain 64x64 tile GEMM, fp32 FMA, with the same correction term.
struct F32Args {
  const float* A;  // rows_a x K
  const float* B;  // per block rows_b x K
  long long b_block_stride;
  int rows_a, rows_b, K;
  const float* ca;  // per block rows_a x rc
  long long ca_block_stride;
  const float* cb;  // per block rows_b x rc
  long long cb_block_stride;
  int rc;
  float* Y;
  long long y_block_stride;
  int ldy;
  int epi;                    // zo_epilogue
  const float* R;             // ZO_EPI_RESIDUAL: added to Y (same layout)
  long long r_block_stride;
  const float* base;          // nullptr, or a rows_b x ldy matrix added before the epilogue
};

__global__ __launch_bounds__(256) void k_gemm_f32(F32Args a) {
  __shared__ float sb[16][68];
  __shared__ float sa[16][68];
  const int blk = blockIdx.z;
  const int t0 = blockIdx.y * 64;
  const int c0 = blockIdx.x * 64;
  const float* __restrict__ B = a.B + (long long)blk * a.b_block_stride;
  const float* __restrict__ A = a.A;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < a.K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = threadIdx.x + 256 * i;
      const int row = e >> 4, kk = e & 15;
      const int k = k0 + kk;
      sb[kk][row] = (t0 + row < a.rows_b && k < a.K) ? B[(size_t)(t0 + row) * a.K + k] : 0.f;
      sa[kk][row] = (c0 + row < a.rows_a && k < a.K) ? A[(size_t)(c0 + row) * a.K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(sb[kk][ty * 4 + i], sa[kk][tx * 4 + j], acc[i][j]);
    __syncthreads();
  }
  if (a.rc > 0) {
    const float* __restrict__ C = a.ca + (long long)blk * a.ca_block_stride;
    const float* __restrict__ D = a.cb + (long long)blk * a.cb_block_stride;
    for (int c = 0; c < a.rc; ++c) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tok = t0 + ty * 4 + i;
        const float p = tok < a.rows_b ? D[(size_t)tok * a.rc + c] : 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = c0 + tx * 4 + j;
          const float q = col < a.rows_a ? C[(size_t)col * a.rc + c] : 0.f;
          acc[i][j] = fmaf(p, q, acc[i][j]);
        }
      }
    }
  }
  float* Y = a.Y + (long long)blk * a.y_block_stride;
  const float* R = a.R + (long long)blk * a.r_block_stride;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = t0 + ty * 4 + i;
    if (tok >= a.rows_b) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = c0 + tx * 4 + j;
      if (col >= a.rows_a) continue;
      float v = acc[i][j];
      if (a.base) v += a.base[(size_t)tok * a.ldy + col];
      if (a.epi == ZO_EPI_RELU) v = fmaxf(v, 0.f);
      if (a.epi == ZO_EPI_RESIDUAL) v += R[(size_t)tok * a.ldy + col];
      if (a.epi == ZO_EPI_SILU_MUL) v *= silu(R[(size_t)tok * a.ldy + col]);
      Y[(size_t)tok * a.ldy + col] = v;
    }
  }
}

// Vt[a][k] = V[k][a] for a < r, 0 for r <= a < rp.  16-bit: hi part in rows
// [0, rp), low part (V - hi, rounded) in rows [rp, 2 rp); fp16 splits 256 V.
// Factor blockIdx.y of a group that shares n, r and rp.
struct TvArgs {
  const float* V[ZO_MAX_GROUP];
  void* Vt[ZO_MAX_GROUP];
  int n, r, rp, dtype;
};
__global__ __launch_bounds__(256) void k_transpose_v(TvArgs t) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const int n = t.n, r = t.r, rp = t.rp;
  if (idx >= (long long)rp * n) return;
  const float* __restrict__ V = t.V[blockIdx.y];
  const int a = (int)(idx / n), k = (int)(idx % n);
  const float v = a < r ? V[(size_t)k * r + a] : 0.f;
  put_split(t.Vt[blockIdx.y], idx, (long long)rp * n, v, t.dtype);
}

// P = (P2[:, :rp] + P2[:, rp:]) * unscale (fp32; unscale a power of two; P2 rows ld2 apart),
// written as [P_hi | P_hi | P_lo] (bf16, 3 rp wide).
__global__ __launch_bounds__(256) void k_pcombine(const float* __restrict__ P2, long long rows,
                                                   int rp, int ld2, float unscale,
                                                   bf16_t* __restrict__ Pc) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= rows * rp) return;
  const long long t = idx / rp;
  const int a = (int)(idx % rp);
  const float p = (P2[t * ld2 + a] + P2[t * ld2 + rp + a]) * unscale;
  const bf16_t hi = f32_to_bf16(p);
  const bf16_t lo = f32_to_bf16(p - bf16_to_f32(hi));
  bf16_t* o = Pc + t * 3 * rp;
  o[a] = hi;
  o[rp + a] = hi;
  o[2 * rp + a] = lo;
}

// B_b[i][a] = s_b eps sum_c U[i][c] Z_{j(b)}[c][a] (a < r; 0 for r <= a < rp).
// fp32 output: m x rp per block.  bf16 output: m x 3 rp per block as
// [B_hi | B_lo | B_hi].
// One workgroup forms C = eps U Z_j for R rows and one query j: Z_j and the
// workgroup's U rows are staged in LDS, and each thread owns RR rows (R / RR
// apart) and 8 adjacent columns (K ascending, one fused multiply-add per term,
// as a plain dot product).
// It then writes s_b C for every block b of query j, 16 bytes per store, so a
// wave's three stores of a block cover 8 whole rows of [B_hi | B_lo | B_hi]
// (3 KB contiguous at rp = 64).  The bf16 split is odd in its argument (round
// to nearest even is symmetric), so the blocks of one query share one product.
template <int RPK>
struct BpShape {
  static constexpr int RP = 32 * RPK;
  static constexpr int G = RP / 8;    // column groups of a row
  // Rows per thread: wider factors take more, so the staged Z_j rows serve more outputs.
  static constexpr int RR = RPK <= 2 ? 1 : (RPK == 3 ? 2 : 4);
  static constexpr int RT = 256 / G;  // rows per pass of the 256 threads (RP = 96: 21, 4 idle)
  static constexpr int R = RR * RT;   // rows per workgroup
};

// Factor blockIdx.z of a group that shares r, rp, the blocks and eps (one factor: a group of 1);
// the grid covers the tallest factor.
struct BpArgs {
  const float* U[ZO_MAX_GROUP];
  const float* Z[ZO_MAX_GROUP];
  void* Bp[ZO_MAX_GROUP];
  int m[ZO_MAX_GROUP];
  int r, rp, nblk, out_bf16;
  float eps;
  BlkTable tab;
};

template <int RPK>
__global__ __launch_bounds__(256) void k_bprime(BpArgs a) {
  constexpr int RP = BpShape<RPK>::RP, G = BpShape<RPK>::G, RR = BpShape<RPK>::RR;
  constexpr int RT = BpShape<RPK>::RT, R = BpShape<RPK>::R;
  constexpr int UL = RP + 4;  // floats per staged U row (rows 4 banks apart)
  __shared__ __attribute__((aligned(16))) float Zl[32 * RP];  // 32 rows of Z_j at a time
  __shared__ __attribute__((aligned(16))) float Ul[R * UL];
  const int f = blockIdx.z;
  const int m = a.m[f], r = a.r, rp = a.rp, nblk = a.nblk, out_bf16 = a.out_bf16;
  const float eps = a.eps;
  const float* __restrict__ U = a.U[f];
  const float* __restrict__ Z = a.Z[f];
  void* const Bp = a.Bp[f];
  const int j = blockIdx.y;
  const int i0 = blockIdx.x * R;
  if (i0 >= m) return;  // past a shorter factor: the whole workgroup, before any barrier
  const int tid = threadIdx.x;
  const float* __restrict__ Zj = Z + (size_t)j * r * r;
  for (int x = tid; x < R * RP; x += 256) {
    const int i = x / RP, k = x % RP;
    Ul[i * UL + k] = (i0 + i < m && k < r) ? U[(size_t)(i0 + i) * r + k] : 0.f;
  }
  const int row = tid / G, cg = tid % G;
  // Threads past the last row still take part in the staging and its barriers.
  const bool live = row < RT && i0 + row < m;
  float acc[RR][8];
#pragma unroll
  for (int q = 0; q < RR; ++q)
#pragma unroll
    for (int y = 0; y < 8; ++y) acc[q][y] = 0.f;
  const float* __restrict__ zc = Zl + cg * 8;
  for (int k0 = 0; k0 < r; k0 += 32) {
    const int kn = min(32, r - k0);
    if (k0) __syncthreads();  // every thread is done with the previous rows of Z_j
    for (int x = tid; x < kn * RP; x += 256) {
      const int k = x / RP, c = x % RP;
      Zl[x] = c < r ? Zj[(k0 + k) * r + c] : 0.f;
    }
    __syncthreads();
    if (live) {
      const int kn4 = kn & ~3;
      int k = 0;
      for (; k < kn4; k += 4) {
        f32x4 u[RR];
#pragma unroll
        for (int q = 0; q < RR; ++q) u[q] = *(const f32x4*)(Ul + (row + q * RT) * UL + k0 + k);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const f32x4 z0 = *(const f32x4*)(zc + (k + e) * RP);
          const f32x4 z1 = *(const f32x4*)(zc + (k + e) * RP + 4);
#pragma unroll
          for (int q = 0; q < RR; ++q) {
            acc[q][0] = fmaf(u[q][e], z0[0], acc[q][0]);
            acc[q][1] = fmaf(u[q][e], z0[1], acc[q][1]);
            acc[q][2] = fmaf(u[q][e], z0[2], acc[q][2]);
            acc[q][3] = fmaf(u[q][e], z0[3], acc[q][3]);
            acc[q][4] = fmaf(u[q][e], z1[0], acc[q][4]);
            acc[q][5] = fmaf(u[q][e], z1[1], acc[q][5]);
            acc[q][6] = fmaf(u[q][e], z1[2], acc[q][6]);
            acc[q][7] = fmaf(u[q][e], z1[3], acc[q][7]);
          }
        }
      }
      for (; k < kn; ++k) {
#pragma unroll
        for (int q = 0; q < RR; ++q) {
          const float u = Ul[(row + q * RT) * UL + k0 + k];
#pragma unroll
          for (int y = 0; y < 8; ++y) acc[q][y] = fmaf(u, zc[k * RP + y], acc[q][y]);
        }
      }
    }
  }
  if (!live) return;
#pragma unroll
  for (int q = 0; q < RR; ++q) {
    const int i = i0 + row + q * RT;
    if (i >= m) break;
    float v[8];
#pragma unroll
    for (int y = 0; y < 8; ++y) v[y] = eps * acc[q][y];
    if (out_bf16) {
      // hi / lo of eps C (the sign is applied per block below).
      u32x4 hp, lp;
#pragma unroll
      for (int y = 0; y < 4; ++y) {
        const float a0 = v[2 * y], a1 = v[2 * y + 1];
        hp[y] = pack_bf16x2(a0, a1);
        lp[y] = pack_bf16x2(a0 - bf16_to_f32(f32_to_bf16(a0)), a1 - bf16_to_f32(f32_to_bf16(a1)));
      }
      for (int b = 0; b < nblk; ++b) {
        const int code = a.tab.code[b];
        if ((code & 0xffff) != j) continue;
        const int s = (code >> 16) - 1;
        // Negation flips the sign bits; zero times the sign is +0.
        const uint32_t flip = s < 0 ? 0x80008000u : 0u;
        const u32x4 h = s == 0 ? (u32x4){0u, 0u, 0u, 0u} : (hp ^ flip);
        const u32x4 l = s == 0 ? (u32x4){0u, 0u, 0u, 0u} : (lp ^ flip);
        bf16_t* o = (bf16_t*)Bp + ((long long)b * m + i) * 3 * rp + cg * 8;
        *(u32x4*)o = h;
        *(u32x4*)(o + rp) = l;
        *(u32x4*)(o + 2 * rp) = h;
      }
    } else {
      // fp32 keeps rp == round16(r) wide rows; RP may exceed rp (whole groups of 8).
      if (cg * 8 >= rp) break;
      for (int b = 0; b < nblk; ++b) {
        const int code = a.tab.code[b];
        if ((code & 0xffff) != j) continue;
        const float s = (float)((code >> 16) - 1);
        float* o = (float*)Bp + ((long long)b * m + i) * rp + cg * 8;
        *(f32x4*)o = (f32x4){s * v[0], s * v[1], s * v[2], s * v[3]};
        *(f32x4*)(o + 4) = (f32x4){s * v[4], s * v[5], s * v[6], s * v[7]};
      }
    }
  }
}

template <int WM, int WN, int TM, int TN, bool F16>
int launch_gemm_bf16(GemmArgs a, hipStream_t stream) {
  constexpr int BM = WM * TM * 32, BN = WN * TN * 32;
  a.tiles_a = (a.rows_a + BM - 1) / BM;
  a.tiles_b = (a.rows_b + BN - 1) / BN;
  const long long total = (long long)a.tiles_a * a.tiles_b * a.nblk;
  if (total <= 0) return ZO_OK;
  if (total > 0x7fffffffLL) {
    zo_set_error("perturbed linear: too many tiles (%lld)", total);
    return ZO_ERR_UNSUPPORTED;
  }
  a.total_tiles = (int)total;
  hipLaunchKernelGGL((k_gemm_bf16<WM, WN, TM, TN, F16>), dim3(a.total_tiles), dim3(WM * WN * 64), 0,
                     stream, a);
  return zo_hip_status(hipGetLastError(), "k_gemm_bf16");
}


// ---------------------------------------------------------------------------
// Main GEMM for K % 32 == 0: the kernel every model-shaped call takes.
//
// 256 x 256 output tile per workgroup of 4 waves (one per SIMD), each wave a 128 x 128
// sub-tile held in 64 accumulators of the 16x16x32 MFMA (256 AGPRs, updated in place).
//
// K is walked in tiles of 64, so every LDS row holds 128 bytes: one whole cache line per row,
// which the load path moves ~1.6x faster than 64-byte half lines (measured with load-only
// kernels of the same traffic).  Tiles are brought in by direct global->LDS buffer loads
// (buffer_load_dwordx4 ... lds: 8 rows x 128 B per instruction, a per-lane row offset fixed for
// the whole loop and the k offset in a scalar register, so the loop has no address arithmetic).
// Row r keeps its 16-byte chunk c at position c ^ f(r), f(r) = (r >> 1) & 7: the fragment reads
// (16 consecutive rows at one chunk per 16-lane group) are conflict free.
//
// LDS ring: the 160 KB as 5 slots of 32 KB, one per part of a tile (part A = the 256 W rows,
// part B = the 256 X rows): A(t) in slot 2t % 5, B(t) in slot (2t+1) % 5.  A tile is two
// 32-deep substeps of 64 MFMAs each, with one barrier between them.  Substep 0 runs the MFMAs of
// the tile's first half, reads the fragments of its second half and issues A(k+2) (into the
// slot B(k-1) vacated); then the wave waits for everything but A(k+2) and meets the others at
// the barrier: every wave is done reading tile k and tile k+1 has landed.  Substep 1 runs the
// second half, reads tile k+1's first half and issues B(k+2) into tile k's A slot.  So every
// part has a whole tile or more to land.  The loads are spread one per eight MFMAs and the
// fragment reads one per four, in the order the next substep first uses them; scheduling
// fences after every MFMA keep that interleave (left to itself the compiler bunches the reads
// and loads, and the wave's MFMA issue stalls behind them).
//
// The rank-rc correction is rc/64 more k-tiles through the same pipeline, with the A operand
// taken from ca (per block, rows_a x rc) and the B operand from cb (per block, rows_b x rc).
// The last tile of a segment whose length is an odd multiple of 32 holds 32 valid columns: only
// its first substep is computed (the other half of its rows is loaded but never read).  So
// every accumulator sees its k terms in ascending order, 32 at a time, whatever the tiling.
// Rows past rows_a / rows_b are loaded from the last valid row (never stored).  F16: the main
// tiles run the fp16 MFMA and the correction tiles (bf16 hi/lo operands) the bf16 MFMA.  OUT
// (zo_dtype of Y) and EPI (zo_epilogue) are template parameters: with all 256 accumulators
// live, one store path per instantiation keeps the epilogue free of per-store branches (a
// run-time choice there made the compiler keep spilled VGPR copies of the accumulators, one of
// which it stored wrongly).
//
// Each operand's buffer descriptor spans its rows x K (or rc) elements, so the host takes this
// kernel only when every such span is below 2^32 bytes.
constexpr int MAIN_RB = 128;               // bytes per LDS row (64 bf16)
constexpr int MAIN_PART = 256 * MAIN_RB;   // one part of a tile: 32 KB
constexpr int MAIN_SLOTS = 5;

__device__ __forceinline__ int f8(int r) { return (r >> 1) & 7; }

// Byte offset of a lane's DMA row (clamped to the operand's last row) at k = 0 in an operand of
// the given width (elements per row), its 16-byte chunk lch.
__device__ __forceinline__ unsigned dma_off(int row, int rows, int width, int lch) {
  return (unsigned)min(row, rows - 1) * (unsigned)width * 2u + (unsigned)lch * 16u;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, (int)bytes, 0x00020000);
}

template <bool F16, int OUT, int EPI>
__global__ __launch_bounds__(256, 1) void k_gemm_main(GemmArgs a) {
  constexpr int RB = MAIN_RB, PART = MAIN_PART;
  __shared__ __attribute__((aligned(1024))) char lds[MAIN_SLOTS * PART];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;

  // XCD-aware tile order (each XCD a contiguous range), grouped 8 token tiles deep.  With
  // blk_inner the block index runs fastest (the shared-X fan-out: the blocks of one tile read
  // the same base tile, which then comes from the XCD's L2).
  const int w = blockIdx.x;
  const int nt = a.total_tiles;
  const int xcd = w & 7, widx = w >> 3;
  const int lt0 = xcd * (nt >> 3) + min(xcd, nt & 7) + widx;
  const int lt = a.blk_inner ? lt0 / a.nblk : lt0;
  const int nbt = a.blk_inner ? a.tiles_b : a.nblk * a.tiles_b;  // (block, token tile) pairs in the raster
  constexpr int GROUP = 8;
  const int per_group = GROUP * a.tiles_a, grp = lt / per_group, first = grp * GROUP;
  const int gsize = min(GROUP, nbt - first), rem = lt - grp * per_group;
  const int bt = first + rem % gsize, at = rem / gsize;
  // The decode is uniform but its divisions run on the VALU: pin the results to scalar
  // registers, so the buffer descriptors built from them are scalar too.
  const int blk = __builtin_amdgcn_readfirstlane(a.blk_inner ? lt0 % a.nblk : bt / a.tiles_b);
  const int t0 = __builtin_amdgcn_readfirstlane((bt % a.tiles_b) * 256);
  const int m0 = __builtin_amdgcn_readfirstlane(at * 256);

  // Tiles: main segment [0, NTM) over K, rank-rc segment [NTM, NT) over rc.
  const int NTM = (a.K + 63) / 64, NT = NTM + (a.rc + 63) / 64;
  const bool halfM = (a.K & 63) != 0, halfR = (a.rc & 63) != 0;
  const bf16_t* const Bblk = a.B + (long long)blk * a.b_block_stride;
  const bf16_t* const Cblk = a.ca + (long long)blk * a.ca_block_stride;
  const bf16_t* const Dblk = a.cb + (long long)blk * a.cb_block_stride;
  const __amdgpu_buffer_rsrc_t rsA = make_rsrc(a.A, (unsigned)a.rows_a * a.K * 2);
  const __amdgpu_buffer_rsrc_t rsB = make_rsrc(Bblk, (unsigned)a.rows_b * a.K * 2);
  // DMA: load i (0..7) of a wave writes rows 8 (wave + 4 i) .. + 7 of a part; lane l writes row
  // l / 8 at physical chunk l % 8, which holds logical chunk (l % 8) ^ f(row) (f(row) does not
  // depend on i).  Per-lane byte offsets of the four operands at k = 0.
  const int drow = lane >> 3;
  const int lch = (lane & 7) ^ f8(8 * wave + drow);
  unsigned voA[8], voB[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = 8 * (wave + 4 * i) + drow;
    const unsigned ra = (unsigned)min(m0 + row, a.rows_a - 1), rb = (unsigned)min(t0 + row, a.rows_b - 1);
    voA[i] = ra * (unsigned)a.K * 2u + lch * 16u;
    voB[i] = rb * (unsigned)a.K * 2u + lch * 16u;
  }
  // The rank segment's row offsets are formed where its few tiles load (a couple of VALU
  // instructions each) rather than kept through the main loop.
#define voC(i) dma_off(m0 + 8 * (wave + 4 * (i)) + drow, a.rows_a, a.rc, lch)
#define voD(i) dma_off(t0 + 8 * (wave + 4 * (i)) + drow, a.rows_b, a.rc, lch)
  char* const ldsw = lds + 8 * wave * RB;
  // Loads i in [I0, I1) of part A (W rows) or B (X rows) of tile t into slot sl; tiles past the
  // end are not loaded.  MAIN: t is known to be a main-segment tile.  The rank segment's
  // descriptor is built after its base is chosen (a scalar select), so it stays in scalar
  // registers.
  auto load_A = [&](int sl, int t, auto MAIN, auto I0, auto I1) {
    const bool m = decltype(MAIN)::value || t < NTM;
    if (!m && t >= NT) return;
    char* d = ldsw + sl * PART;
    const __amdgpu_buffer_rsrc_t r = m ? rsA : make_rsrc(Cblk, (unsigned)a.rows_a * a.rc * 2);
    const unsigned so = (unsigned)(m ? t : t - NTM) * 128u;
#pragma unroll
    for (int i = decltype(I0)::value; i < decltype(I1)::value; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(d + 32 * RB * i), 16, m ? voA[i] : voC(i), so, 0, 0);
  };
  auto load_B = [&](int sl, int t, auto MAIN, auto I0, auto I1) {
    const bool m = decltype(MAIN)::value || t < NTM;
    if (!m && t >= NT) return;
    char* d = ldsw + sl * PART;
    const __amdgpu_buffer_rsrc_t r = m ? rsB : make_rsrc(Dblk, (unsigned)a.rows_b * a.rc * 2);
    const unsigned so = (unsigned)(m ? t : t - NTM) * 128u;
#pragma unroll
    for (int i = decltype(I0)::value; i < decltype(I1)::value; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(d + 32 * RB * i), 16, m ? voB[i] : voD(i), so, 0, 0);
  };
  using Main = std::true_type;
  using Any = std::false_type;
  using I0 = std::integral_constant<int, 0>;
  using I4 = std::integral_constant<int, 4>;
  using I8 = std::integral_constant<int, 8>;

  // Fragments (16x16x32): lane l reads row (16 i + l % 16) of its wave's 128 rows of a part at
  // k-quarter l / 16 of a 32-deep substep, i.e. logical chunk 4 s + l / 16 of the row.  The
  // rows of one fragment start at a multiple of 16, so f of a fragment row is f(l % 16).
  const int fr = lane & 15, fq = lane >> 4;
  const int ff = f8(fr);
  const int offA = (wm * 128 + fr) * RB, offB = (wn * 128 + fr) * RB;
  bf16x8 F0a[8], F0b[8], F1a[8], F1b[8];
  // Fragments of substep s (k 32 s .. 32 s + 31 of the tile) from the slots sa (A) and sb (B).
  auto frags = [&](int sa, int sb, int s, bf16x8* fa, bf16x8* fb) {
    const int ch = ((4 * s + fq) ^ ff) * 16;
    const char* pa = lds + sa * PART + offA + ch;
    const char* pb = lds + sb * PART + offB + ch;
#pragma unroll
    for (int i = 0; i < 8; ++i) fa[i] = *(const bf16x8*)(pa + i * 16 * RB);
#pragma unroll
    for (int j = 0; j < 8; ++j) fb[j] = *(const bf16x8*)(pb + j * 16 * RB);
  };
  // acc[i][j]: output columns (A rows) 16 i + 4 (l / 16) .. + 3, token (B row) 16 j + l % 16 of
  // the wave's 128 x 128.
  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.f;
  // The zeros are in place (in AGPRs) at least 2 wait states before any MFMA reads them.
#pragma unroll
  for (int i = 0; i < 8; ++i)
    asm volatile("s_nop 1" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]),
                 "+a"(acc[i][4]), "+a"(acc[i][5]), "+a"(acc[i][6]), "+a"(acc[i][7]));
  auto mma = [&](const bf16x8* fa, const bf16x8* fb, auto f16) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) mfma16<decltype(f16)::value>(acc[i][j], fa[i], fb[j]);
  };
  // The n-th fragment read of substep s from slots sa / sb, in the order the next substep first
  // uses them: A0 (MFMA 0), B0..B7 (MFMAs 0..7), then A1..A7 (MFMAs 8, 16, ..., 56).
  auto frag1 = [&](int sa, int sb, int s, int n, bf16x8* fa, bf16x8* fb) {
    const int ch = ((4 * s + fq) ^ ff) * 16;
    if (n >= 1 && n <= 8)
      fb[n - 1] = *(const bf16x8*)(lds + sb * PART + offB + ch + (n - 1) * 16 * RB);
    else {
      const int x = n == 0 ? 0 : n - 8;
      fa[x] = *(const bf16x8*)(lds + sa * PART + offA + ch + x * 16 * RB);
    }
  };
  // One load (i of 8) of part A / B of main-segment tile t into slot sl.
  auto load1_A = [&](int sl, int t, int i) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, (lds_ptr_t)(ldsw + sl * PART + 32 * RB * i), 16, voA[i],
                                             (unsigned)t * 128u, 0, 0);
  };
  auto load1_B = [&](int sl, int t, int i) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsB, (lds_ptr_t)(ldsw + sl * PART + 32 * RB * i), 16, voB[i],
                                             (unsigned)t * 128u, 0, 0);
  };
  // One steady-state substep, written out in issue order: MFMA x (x = 0..63, accumulator
  // x / 8, x % 8), the next substep's fragment read x / 4 after every fourth MFMA (fragments
  // (ra, rb, rs) into na / nb, in frag1's order: the B fragments, which the next substep's first
  // eight MFMAs all use, are read early), and load ld(x / 8) after every eighth, each group fenced so the
  // compiler keeps the interleave (left to itself it bunches the reads and loads, and the wave's
  // MFMA issue stalls behind them).
  auto substep = [&](const bf16x8* fa, const bf16x8* fb, int ra, int rb, int rs, bf16x8* na, bf16x8* nb,
                     auto ld, auto f16) {
#pragma unroll
    for (int x = 0; x < 64; ++x) {
      mfma16<decltype(f16)::value>(acc[x >> 3][x & 7], fa[x >> 3], fb[x & 7]);
      if (x % 4 == 0) frag1(ra, rb, rs, x / 4, na, nb);
      if (x % 8 == 3) ld(x / 8);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Prologue: A0, B0, A1 and B1.  Tile k then issues A(k+2) before its barrier (into the slot
  // tile k-1's B part vacated) and B(k+2) after it (into tile k's A slot), so every part has a
  // whole tile or more to land.
  load_A(0, 0, Any{}, I0{}, I8{});
  load_B(1, 0, Any{}, I0{}, I8{});
  load_A(2, 1, Any{}, I0{}, I8{});
  load_B(3, 1, Any{}, I0{}, I8{});
  if (NT > 1)
    asm volatile("s_waitcnt vmcnt(16)" ::: "memory");  // this wave's loads of tile 0 landed
  else
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  frags(0, 1, 0, F0a, F0b);

  // Tile k, a full main tile with main tiles k+1 and k+2 after it; K5 = k % 5 makes every slot a
  // compile-time constant.  Substep 0 (MFMAs of k-half 0, reads of half 1) issues A(k+2); the
  // barrier follows the last reads of tile k; substep 1 (MFMAs of half 1, reads of tile k+1's
  // half 0) issues B(k+2) into tile k's A slot.
  auto body_main = [&](int k, auto K5, auto f16) {
    constexpr int k5 = decltype(K5)::value;
    constexpr int sa = (2 * k5) % 5, sb = (2 * k5 + 1) % 5;                       // tile k
    constexpr int na = (2 * k5 + 2) % 5, nb = (2 * k5 + 3) % 5, a2 = (2 * k5 + 4) % 5;  // k+1, A(k+2)
    substep(F0a, F0b, sa, sb, 1, F1a, F1b, [&](int i) { load1_A(a2, k + 2, i); }, f16);
    asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)" ::: "memory");  // all but A(k+2)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    substep(F1a, F1b, na, nb, 0, F0a, F0b, [&](int i) { load1_B(sa, k + 2, i); }, f16);
  };
  // One load (i of 8) of part A / B of tile t (either segment; t < NT) into slot sl.  The
  // segment is a uniform choice: scalar selects of the descriptor and k offset, one VALU select
  // of the row offset.
  const __amdgpu_buffer_rsrc_t rsC = make_rsrc(Cblk, (unsigned)a.rows_a * a.rc * 2);
  const __amdgpu_buffer_rsrc_t rsD = make_rsrc(Dblk, (unsigned)a.rows_b * a.rc * 2);
  auto load1g_A = [&](int sl, int t, int i) {
    const bool m = t < NTM;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(m ? rsA : rsC, (lds_ptr_t)(ldsw + sl * PART + 32 * RB * i), 16,
                                             m ? voA[i] : voC(i), (unsigned)(m ? t : t - NTM) * 128u, 0, 0);
  };
  auto load1g_B = [&](int sl, int t, int i) {
    const bool m = t < NTM;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(m ? rsB : rsD, (lds_ptr_t)(ldsw + sl * PART + 32 * RB * i), 16,
                                             m ? voB[i] : voD(i), (unsigned)(m ? t : t - NTM) * 128u, 0, 0);
  };
  // Tile k as body_main, with run-time slots and loads from either segment: the tiles that
  // follow the unrolled main loop (the last main tiles and the rank segment), up to NT - 3.
  // Needs tile k full and tiles k + 1, k + 2 to exist.
  auto body_rt = [&](int k, auto f16) {
    const int sa = (2 * k) % 5, sb = (2 * k + 1) % 5;
    const int na = (2 * k + 2) % 5, nb = (2 * k + 3) % 5, a2 = (2 * k + 4) % 5;
    substep(F0a, F0b, sa, sb, 1, F1a, F1b, [&](int i) { load1g_A(a2, k + 2, i); }, f16);
    asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)" ::: "memory");  // all but A(k+2)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    substep(F1a, F1b, na, nb, 0, F0a, F0b, [&](int i) { load1g_B(sa, k + 2, i); }, f16);
  };
  // Any tile (run-time slots, loads of either segment or none, half tiles: their second
  // 32-deep half is loaded but never read).  The loads go out together here: only the last two
  // tiles and half tiles take this path.
  auto body_any = [&](int k, auto f16) {
    const int sa = (2 * k) % 5, sb = (2 * k + 1) % 5, na = (2 * k + 2) % 5, nb = (2 * k + 3) % 5;
    const int a2 = (2 * k + 4) % 5;
    const bool half = k == NTM - 1 ? halfM : (k == NT - 1 ? halfR : false);
    load_A(a2, k + 2, Any{}, I0{}, I8{});
    if (!half) frags(sa, sb, 1, F1a, F1b);
    mma(F0a, F0b, f16);
    // The last loads issued are A(k+2)'s when it exists; otherwise none may stay outstanding.
    if (k + 2 < NT)
      asm volatile("s_waitcnt vmcnt(8) lgkmcnt(0)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (k + 1 < NT) frags(na, nb, 0, F0a, F0b);
    load_B(sa, k + 2, Any{}, I0{}, I8{});
    if (!half) mma(F1a, F1b, f16);
  };
  using MT = std::integral_constant<bool, F16>;
  // body_main needs k + 2 <= NTM - 1 (main-segment loads) and tile k full: k <= NTM - 3.
  const int P = NTM >= 3 ? (NTM - 2) / 5 * 5 : 0;
  int k = 0;
  for (; k < P; k += 5) {
    body_main(k, std::integral_constant<int, 0>{}, MT{});
    body_main(k + 1, std::integral_constant<int, 1>{}, MT{});
    body_main(k + 2, std::integral_constant<int, 2>{}, MT{});
    body_main(k + 3, std::integral_constant<int, 3>{}, MT{});
    body_main(k + 4, std::integral_constant<int, 4>{}, MT{});
  }
  // The rest: body_rt while the tile is full and two more follow, else body_any (only a
  // segment's last tile can be a half tile).
  const int e1 = min(halfM ? NTM - 1 : NTM, NT - 2);
  for (; k < e1; ++k) body_rt(k, MT{});
  for (; k < NTM; ++k) body_any(k, MT{});
  for (; k < NT - 2; ++k) body_rt(k, std::false_type{});
  for (; k < NT; ++k) body_any(k, std::false_type{});
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // drain before the stores and exit
  // 24 wait states after the last MFMA before the accumulators are read.  They then pass
  // through empty statements ordered after the wait, so no read or copy of them can be placed
  // ahead of it.
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int i = 0; i < 8; ++i)
    asm volatile("" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]), "+a"(acc[i][4]),
                 "+a"(acc[i][5]), "+a"(acc[i][6]), "+a"(acc[i][7]));
#undef voC
#undef voD

  // Epilogue through LDS.  The accumulator layout gives each lane 4 adjacent outputs of one
  // token, so stores straight from the registers would touch 32 token rows per instruction
  // with 16 bytes each; staged through the (now free) ring, every lane writes 16 contiguous
  // bytes and a wave's store covers whole rows.  16-bit outputs without R are rounded
  // once and staged as stored (256 token rows of 512 bytes); otherwise the fp32 values are
  // staged in two halves of 128 token rows of 1 KB, and R is applied to them before the single
  // rounding.  Rows are padded by 16 bytes (pitch 528 / 1040), so that the writes (8 consecutive
  // rows at one chunk per 8 lanes) spread over the banks and every lane's staging addresses are
  // one base register plus immediates.
  char* Yb = (char*)a.Y + (long long)blk * a.y_block_stride * (OUT == ZO_F32 ? 4 : 2);
  const char* Rb = (const char*)a.R + (long long)blk * a.r_block_stride * (OUT == ZO_F32 ? 4 : 2);
  __syncthreads();  // every wave is past its last fragment reads: the ring is free
  __builtin_amdgcn_sched_barrier(0);  // nothing of the epilogue moves above the barrier
  // The lane index again, from the lane masks rather than the work-item id: the compiler then
  // recomputes these few values here instead of keeping (and spilling) the loop's copies.
  const int el = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int efr = el & 31, efh = el >> 5;
  const int e16 = el & 15, eq = el >> 4;  // the accumulator layout's token row and column quarter
  if constexpr (EPI == EPI_PROJ32 || EPI == EPI_PROJ64) {
    // A wave's 128 A rows hold whole factors (2 rp rows each: the hi rows, then the lo rows), so
    // a factor column's hi and lo sums are accumulators i and i + rp / 16 of one lane.  Combined,
    // split and rounded here, they go straight to the factor's buffer (a lane writes 4 adjacent
    // columns of one token; the output is 3 rp / (2 K) of the bytes read, so no staging).
    constexpr int RP = EPI == EPI_PROJ32 ? 32 : 64, R16 = RP / 16, NFW = 128 / (2 * RP);
#pragma unroll
    for (int f = 0; f < NFW; ++f) {
      const int gf = (m0 + wm * 128) / (2 * RP) + f;
      if (gf >= a.pcount) break;
      bf16_t* const pc = a.pc[gf];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int tok = t0 + wn * 128 + 16 * j + e16;
        if (tok >= a.rows_b) continue;
        bf16_t* const o = pc + ((long long)blk * a.rows_b + tok) * (3 * RP) + 4 * eq;
#pragma unroll
        for (int ii = 0; ii < R16; ++ii) {
          const int ih = f * 2 * R16 + ii, il = ih + R16;
          float hv[4], lv[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float pv = (acc[ih][j][e] + acc[il][j][e]) * a.unscale;
            hv[e] = bf16_to_f32(f32_to_bf16(pv));
            lv[e] = pv - hv[e];
          }
          const u32x2 hi = (u32x2){pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3])};
          const u32x2 lo = (u32x2){pack_bf16x2(lv[0], lv[1]), pack_bf16x2(lv[2], lv[3])};
          *(u32x2*)(o + 16 * ii) = hi;
          *(u32x2*)(o + RP + 16 * ii) = hi;
          *(u32x2*)(o + 2 * RP + 16 * ii) = lo;
        }
      }
    }
  } else if constexpr (OUT != ZO_F32 && (EPI == ZO_EPI_NONE || EPI == ZO_EPI_RELU)) {
    constexpr int PITCH = 528;
    // acc[i][j]: token row wn 128 + 16 j + l % 16, columns wm 128 + 16 i + 4 (l / 16) .. + 3.
    char* const wb = lds + (wn * 128 + e16) * PITCH + wm * 256 + eq * 8;
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = acc[i][j][e];
          if constexpr (EPI == ZO_EPI_RELU) v[e] = fmaxf(v[e], 0.f);
        }
        *(u32x2*)(wb + j * 16 * PITCH + i * 32) =
            OUT == ZO_BF16 ? (u32x2){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])}
                           : (u32x2){pack_f16x2(v[0], v[1]), pack_f16x2(v[2], v[3])};
      }
    __syncthreads();
    // Pass it of wave w: rows 8 it + 2 w + lane / 32, whole (512 bytes each), 16-byte chunk
    // lane % 32 (columns 8 (lane % 32) ..).
    const char* const rb = lds + (2 * wave + efh) * PITCH + efr * 16;
    const int col = m0 + efr * 8;
#pragma unroll 8
    for (int it = 0; it < 32; ++it) {
      const u32x4 v = *(const u32x4*)(rb + it * 8 * PITCH);
      const int tok = t0 + it * 8 + 2 * wave + efh;
      // Non-temporal: the output streams past the caches (1-2% faster at K = 5120 in A/B).
      if (tok < a.rows_b && col < a.rows_a) __builtin_nontemporal_store(v, (u32x4*)(Yb + ((size_t)tok * a.ldy + col) * 2));
    }
  } else {
    constexpr int PITCH = 1040;
    // Half h holds j = 4 h .. 4 h + 3: staging row wn 64 + 16 (j % 4) + l % 16 is tile token
    // wn 128 + 16 j + l % 16; 16-byte chunk wm 32 + 4 i + l / 16 holds its columns 4 chunk .. + 3.
    char* const wb = lds + (wn * 64 + e16) * PITCH + wm * 512 + eq * 16;
    // Read-back pass it of wave w: staging rows 8 it + lr8, columns 64 w + 8 lc8 .. + 7.
    const int lr8 = el & 7, lc8 = el >> 3;
    const char* const rb = lds + lr8 * PITCH + (wave * 8 + lc8) * 32;
    const int col = m0 + (wave * 8 + lc8) * 8;
    // R of the half's read-back passes is requested before its staging writes, so that its
    // latency overlaps them (one load chain per half instead of one per few passes).
    constexpr bool HAS_R = EPI == ZO_EPI_RESIDUAL || EPI == ZO_EPI_SILU_MUL || EPI == EPI_BASE ||
                           EPI == EPI_BASE_RELU;
    constexpr bool R32 = EPI == EPI_BASE || EPI == EPI_BASE_RELU;  // the fp32 base
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if (h) __syncthreads();  // the first half's read-back is done
      u32x4 rpre[HAS_R ? 16 : 1][R32 || OUT == ZO_F32 ? 2 : 1];
      if constexpr (HAS_R) {
#pragma unroll
        for (int it = 0; it < 16; ++it) {
          const int sr = it * 8 + lr8;
          const int tok = t0 + (sr >> 6) * 128 + h * 64 + (sr & 63);
          const size_t idx = (size_t)min(tok, a.rows_b - 1) * a.ldy + min(col, a.rows_a - 8);
          if constexpr (R32) {  // 32-byte aligned rows
            rpre[it][0] = *(const u32x4*)(Rb + idx * 4);
            rpre[it][1] = *(const u32x4*)(Rb + idx * 4 + 16);
          } else if constexpr (OUT == ZO_F32) {  // an fp32 R need only be 4-byte aligned
            float r8[8];
            load8<ZO_F32>(Rb, idx, r8);
            rpre[it][0] = __builtin_bit_cast(u32x4, (f32x4){r8[0], r8[1], r8[2], r8[3]});
            rpre[it][1] = __builtin_bit_cast(u32x4, (f32x4){r8[4], r8[5], r8[6], r8[7]});
          } else {
            rpre[it][0] = *(const u32x4*)(Rb + idx * 2);
          }
        }
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int i = 0; i < 8; ++i) *(f32x4*)(wb + jj * 16 * PITCH + i * 64) = acc[i][4 * h + jj];
      __syncthreads();
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int sr = it * 8 + lr8;
        const f32x4 lo = *(const f32x4*)(rb + it * 8 * PITCH);
        const f32x4 hi = *(const f32x4*)(rb + it * 8 * PITCH + 16);
        const int tok = t0 + (sr >> 6) * 128 + h * 64 + (sr & 63);
        if (tok >= a.rows_b || col >= a.rows_a) continue;
        const size_t idx = (size_t)tok * a.ldy + col;
        float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        if constexpr (EPI != ZO_EPI_NONE) {
          float rv[8];
          if constexpr (HAS_R) {
            if constexpr (R32 || OUT == ZO_F32) {
              const f32x4 r0 = __builtin_bit_cast(f32x4, rpre[it][0]), r1 = __builtin_bit_cast(f32x4, rpre[it][1]);
              rv[0] = r0[0]; rv[1] = r0[1]; rv[2] = r0[2]; rv[3] = r0[3];
              rv[4] = r1[0]; rv[5] = r1[1]; rv[6] = r1[2]; rv[7] = r1[3];
            } else {
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t u = rpre[it][0][e];
                if constexpr (OUT == ZO_BF16) {
                  rv[2 * e] = bf16_to_f32((bf16_t)u);
                  rv[2 * e + 1] = bf16_to_f32((bf16_t)(u >> 16));
                } else {
                  rv[2 * e] = f16_to_f32((uint16_t)u);
                  rv[2 * e + 1] = f16_to_f32((uint16_t)(u >> 16));
                }
              }
            }
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if constexpr (EPI == ZO_EPI_RELU) v[e] = fmaxf(v[e], 0.f);
            else if constexpr (EPI == ZO_EPI_RESIDUAL || EPI == EPI_BASE) v[e] += rv[e];
            else if constexpr (EPI == EPI_BASE_RELU) v[e] = fmaxf(v[e] + rv[e], 0.f);
            else v[e] *= silu(rv[e]);
          }
        }
        store8<OUT>(Yb, idx, v);
      }
    }
  }
}

// Projection of the prepare pass with the combine fused: for every X block and every factor f
// of a stack of `count` (each 2 RP rows of Vt2: the hi rows, then the lo rows),
//   P = (X_b Vt2_hi^T + X_b Vt2_lo^T) * unscale,  written as [P_hi | P_hi | P_lo] (bf16, 3 RP),
// which is the left operand of the fused GEMM's rank-r segment.  The projection reads every X
// block once and is bound by that stream, so the tile is narrow: 256 tokens x 128 factor rows
// per workgroup, the 4 waves side by side along the tokens (64 tokens x 128 rows each, 8 x 4
// accumulators of the 16x16x32 MFMA), so a k-tile's MFMAs (1024 cycles per wave) take less time
// than its 32 KB of X takes to arrive.  A factor's hi and lo rows lie in the same tile and the
// same lane (accumulators i and i + RP / 16), so the combine, the hi/lo split and the rounding
// happen in registers and the fp32 projection never goes to memory.  Every accumulator sums
// its k terms in ascending order, 32 at a time, as in the main GEMM: the values are those of
// the unfused projection followed by the separate combine.
//
// K is walked in tiles of 64 through a 3-stage LDS ring (X part 32 KB, factor part 16 KB per
// stage; rows swizzled as in the main GEMM), filled by direct global->LDS loads two tiles ahead,
// with one barrier per tile.  Rows past T or past the stack are loaded from the last valid row
// and not stored.
constexpr int PJ_XPART = 256 * 128;
constexpr int PJ_STAGE = PJ_XPART + 128 * 128;

struct ProjArgs {
  const bf16_t* V;           // rows_v x K: the stacked Vt2 of `count` factors
  const bf16_t* X;           // per block T x K
  long long x_block_stride;  // elements
  int rows_v, T, K, count;
  int tiles_t, tiles_c, total_tiles;
  float unscale;             // 1, or 1/256 for fp16 (whose Vt2 holds 256 V)
  bf16_t* pc[ZO_MAX_GROUP];  // factor f's output: (nx T) x 3 RP
};

template <bool F16, int RP>
__global__ __launch_bounds__(256, 1) void k_proj(ProjArgs a) {
  static_assert(RP == 32 || RP == 64, "factors of 64 or 128 rows");
  constexpr int NF = 128 / (2 * RP);  // factors per tile
  constexpr int R16 = RP / 16;
  __shared__ __attribute__((aligned(1024))) char lds[3 * PJ_STAGE];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // XCD-aware order; the factor tiles of one token tile are adjacent, so its X tile comes
  // from the XCD's L2 after the first of them.
  const int w = blockIdx.x, nt = a.total_tiles;
  const int xcd = w & 7, widx = w >> 3;
  const int lt = xcd * (nt >> 3) + min(xcd, nt & 7) + widx;
  const int ct = __builtin_amdgcn_readfirstlane(lt % a.tiles_c);
  const int bt = lt / a.tiles_c;
  const int blk = __builtin_amdgcn_readfirstlane(bt / a.tiles_t);
  const int t0 = __builtin_amdgcn_readfirstlane((bt % a.tiles_t) * 256);
  const int c0 = ct * 128;
  const __amdgpu_buffer_rsrc_t rsX =
      make_rsrc(a.X + (long long)blk * a.x_block_stride, (unsigned)a.T * a.K * 2);
  const __amdgpu_buffer_rsrc_t rsV = make_rsrc(a.V, (unsigned)a.rows_v * a.K * 2);
  // DMA: load i of a wave writes rows 8 (wave + 4 i) .. + 7 of a part (8 loads for the 256 X
  // rows, 4 for the 128 factor rows); lane l writes row l / 8 at physical chunk l % 8.
  const int drow = lane >> 3;
  const int lch = (lane & 7) ^ f8(8 * wave + drow);
  unsigned voX[8], voV[4];
#pragma unroll
  for (int i = 0; i < 8; ++i) voX[i] = dma_off(t0 + 8 * (wave + 4 * i) + drow, a.T, a.K, lch);
#pragma unroll
  for (int i = 0; i < 4; ++i) voV[i] = dma_off(c0 + 8 * (wave + 4 * i) + drow, a.rows_v, a.K, lch);
  char* const ldsw = lds + 8 * wave * 128;
  auto load = [&](int st, int t) {
    char* d = ldsw + st * PJ_STAGE;
    const unsigned so = (unsigned)t * 128u;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsX, (lds_ptr_t)(d + 32 * 128 * i), 16, voX[i], so, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsV, (lds_ptr_t)(d + PJ_XPART + 32 * 128 * i), 16, voV[i], so,
                                               0, 0);
  };
  // Fragments of substep s: factor rows 16 i + l % 16 (A operand, i < 8) and the wave's tokens
  // 64 wave + 16 j + l % 16 (B operand, j < 4), chunk 4 s + l / 16.
  const int fr = lane & 15, fq = lane >> 4;
  const int ff = f8(fr);
  auto frags = [&](int st, int s, bf16x8* fa, bf16x8* fb) {
    const int ch = ((4 * s + fq) ^ ff) * 16;
    const char* pv = lds + st * PJ_STAGE + PJ_XPART + fr * 128 + ch;
    const char* px = lds + st * PJ_STAGE + (wave * 64 + fr) * 128 + ch;
#pragma unroll
    for (int i = 0; i < 8; ++i) fa[i] = *(const bf16x8*)(pv + i * 16 * 128);
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[j] = *(const bf16x8*)(px + j * 16 * 128);
  };
  // acc[i][j]: factor rows 16 i + 4 (l / 16) .. + 3 of the tile, token 64 wave + 16 j + l % 16.
  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[i][j][e] = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)  // the zeros in place 2 wait states before the first MFMA
    asm volatile("s_nop 1" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]));
  auto mma = [&](const bf16x8* fa, const bf16x8* fb) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) mfma16<F16>(acc[i][j], fa[i], fb[j]);
  };

  const int NT = (a.K + 63) / 64;
  const bool half = (a.K & 63) != 0;  // the last tile holds 32 valid columns
  load(0, 0);
  if (NT > 1) {
    load(1, 1);
    asm volatile("s_waitcnt vmcnt(12)" ::: "memory");  // this wave's loads of tile 0 landed
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
  // Tile t (both 32-deep substeps, or only the first for the last tile of an odd K / 32).
  auto tile = [&](int t, bool two) {
    const int st = t % 3;
    if (t + 2 < NT) load((t + 2) % 3, t + 2);  // into the stage tile t - 1 vacated
    bf16x8 fa[8], fb[4], ga[8], gb[4];
    frags(st, 0, fa, fb);
    if (two) frags(st, 1, ga, gb);
    mma(fa, fb);
    if (two) mma(ga, gb);
    // Tile t + 1 landed (only tile t + 2's loads may be in flight) and this wave's reads of
    // stage st are done; after the barrier every wave may overwrite it.
    if (t + 2 < NT)
      asm volatile("s_waitcnt vmcnt(12) lgkmcnt(0)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  const int NTF = half ? NT - 1 : NT;
  for (int t = 0; t < NTF; ++t) tile(t, true);
  if (half) tile(NT - 1, false);
  // 24 wait states after the last MFMA, then the accumulators pass through tied empty
  // statements so that no read of them is placed ahead of the wait.
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int i = 0; i < 8; ++i)
    asm volatile("" : "+a"(acc[i][0]), "+a"(acc[i][1]), "+a"(acc[i][2]), "+a"(acc[i][3]));

#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int gf = ct * NF + f;
    if (gf >= a.count) break;
    bf16_t* const pc = a.pc[gf];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tok = t0 + wave * 64 + 16 * j + fr;
      if (tok >= a.T) continue;
      bf16_t* const o = pc + ((long long)blk * a.T + tok) * (3 * RP) + 4 * fq;
#pragma unroll
      for (int ii = 0; ii < R16; ++ii) {
        const int ih = f * 2 * R16 + ii, il = ih + R16;
        float hv[4], lv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pv = (acc[ih][j][e] + acc[il][j][e]) * a.unscale;
          const bf16_t h = f32_to_bf16(pv);
          hv[e] = bf16_to_f32(h);
          lv[e] = pv - hv[e];
        }
        const u32x2 hi = (u32x2){pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3])};
        const u32x2 lo = (u32x2){pack_bf16x2(lv[0], lv[1]), pack_bf16x2(lv[2], lv[3])};
        *(u32x2*)(o + 16 * ii) = hi;
        *(u32x2*)(o + RP + 16 * ii) = hi;
        *(u32x2*)(o + 2 * RP + 16 * ii) = lo;
      }
    }
  }
}

template <bool F16, int OUT>
void launch_main_epi(const GemmArgs& a, dim3 grid, hipStream_t stream) {
  if constexpr (OUT != ZO_F32) {  // the projection epilogues write bf16 whatever OUT is
    if (a.epi == EPI_PROJ32) {
      hipLaunchKernelGGL((k_gemm_main<F16, OUT, EPI_PROJ32>), grid, dim3(256), 0, stream, a);
      return;
    }
    if (a.epi == EPI_PROJ64) {
      hipLaunchKernelGGL((k_gemm_main<F16, OUT, EPI_PROJ64>), grid, dim3(256), 0, stream, a);
      return;
    }
  }
  if (a.epi == EPI_BASE)
    hipLaunchKernelGGL((k_gemm_main<F16, OUT, EPI_BASE>), grid, dim3(256), 0, stream, a);
  else if (a.epi == EPI_BASE_RELU)
    hipLaunchKernelGGL((k_gemm_main<F16, OUT, EPI_BASE_RELU>), grid, dim3(256), 0, stream, a);
  else if (a.epi == ZO_EPI_RELU)
    hipLaunchKernelGGL((k_gemm_main<F16, OUT, ZO_EPI_RELU>), grid, dim3(256), 0, stream, a);
  else if (a.epi == ZO_EPI_RESIDUAL)
    hipLaunchKernelGGL((k_gemm_main<F16, OUT, ZO_EPI_RESIDUAL>), grid, dim3(256), 0, stream, a);
  else if (a.epi == ZO_EPI_SILU_MUL)
    hipLaunchKernelGGL((k_gemm_main<F16, OUT, ZO_EPI_SILU_MUL>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((k_gemm_main<F16, OUT, ZO_EPI_NONE>), grid, dim3(256), 0, stream, a);
}

// Whether k_gemm_main can take a call: K a multiple of 32 and every operand's buffer descriptor
// span (rows x K, rows x rc elements of 2 bytes) below 2^32 bytes.
bool main_gemm_fits(const GemmArgs& a) {
  const unsigned long long lim = (1ull << 32) - 256;
  return a.K % 32 == 0 && (unsigned long long)a.rows_a * a.K * 2 <= lim &&
         (unsigned long long)a.rows_b * a.K * 2 <= lim && (unsigned long long)a.rows_a * a.rc * 2 <= lim &&
         (unsigned long long)a.rows_b * a.rc * 2 <= lim;
}

int launch_gemm_main(GemmArgs a, bool f16, hipStream_t stream) {
  a.tiles_a = (a.rows_a + 255) / 256;
  a.tiles_b = (a.rows_b + 255) / 256;
  const long long total = (long long)a.tiles_a * a.tiles_b * a.nblk;
  if (total <= 0) return ZO_OK;
  if (total > 0x7fffffffLL) {
    zo_set_error("perturbed linear: too many tiles (%lld)", total);
    return ZO_ERR_UNSUPPORTED;
  }
  a.total_tiles = (int)total;
  const dim3 grid(a.total_tiles);
  if (a.out_dtype == ZO_F32) {
    if (f16)
      launch_main_epi<true, ZO_F32>(a, grid, stream);
    else
      launch_main_epi<false, ZO_F32>(a, grid, stream);
  } else if (f16) {
    launch_main_epi<true, ZO_F16>(a, grid, stream);
  } else {
    launch_main_epi<false, ZO_BF16>(a, grid, stream);
  }
  return zo_hip_status(hipGetLastError(), "k_gemm_main");
}

}  // namespace

int zo_plinear_plan(PlinearPlan* p, int T, int m, int n, int r, int q, int nblk,
                    long long x_block_stride, int in_dtype, int out_dtype) {
  p->T = T;
  p->m = m;
  p->n = n;
  p->r = r;
  p->in16 = in_dtype != ZO_F32;
  p->in_dtype = in_dtype;
  p->out_dtype = out_dtype;
  // 16-bit: a multiple of 32 so the 3 rp-deep rank-r segment is whole 32-wide k-tiles.
  p->rp = p->in16 ? (r + 31) / 32 * 32 : (r + 15) / 16 * 16;
  p->q = q;
  p->nblk = nblk;
  p->x_block_stride = x_block_stride;
  p->nx = x_block_stride == 0 ? 1 : nblk;
  const size_t rows = (size_t)p->nx * T;
  if (p->in16) {
    p->ws_vt = zo_align256((size_t)2 * p->rp * n * 2);       // Vt hi and lo, bf16
    p->ws_p2 = zo_align256(rows * 2 * p->rp * 4);            // X Vt2^T, fp32
    p->ws_p = zo_align256(rows * 3 * p->rp * 2);             // [P_hi | P_hi | P_lo]
    p->ws_bp = zo_align256((size_t)nblk * m * 3 * p->rp * 2);  // [B_hi | B_lo | B_hi]
  } else {
    p->ws_vt = zo_align256((size_t)p->rp * n * 4);
    p->ws_p2 = 0;
    p->ws_p = zo_align256(rows * p->rp * 4);
    p->ws_bp = zo_align256((size_t)nblk * m * p->rp * 4);
  }
  p->fan = p->nx == 1 && nblk > 1;
  p->ws_base = p->fan ? zo_align256((size_t)T * m * 4) : 0;
  p->ws_total = p->ws_vt + p->ws_p2 + p->ws_p + p->ws_bp + p->ws_base;
  return ZO_OK;
}

BlkTable zo_blk_table(int nblk, const int* blk_query, const int8_t* blk_sign) {
  BlkTable tab;
  for (int b = 0; b < nblk; ++b) tab.code[b] = blk_query[b] | ((int)(blk_sign[b] + 1) << 16);
  return tab;
}

PlinearWs zo_plinear_ws(const PlinearPlan& p, void* ws) {
  WsCarver wc(ws);
  PlinearWs w;
  w.vt = wc.take(p.ws_vt);
  w.p2 = p.ws_p2 ? wc.take(p.ws_p2) : nullptr;
  w.pp = wc.take(p.ws_p);
  w.bp = wc.take(p.ws_bp);
  w.base = p.ws_base ? wc.take(p.ws_base) : nullptr;
  return w;
}

// Vt2 of `count` factors that share n, r and rp (plans[i] gives factor i's; V[i] -> vt[i]).
static int launch_transpose_v(const PlinearPlan* plans, int count, const float* const* V, void* const* vt,
                              hipStream_t stream) {
  const PlinearPlan& p = plans[0];
  TvArgs t{};
  for (int i = 0; i < count; ++i) {
    t.V[i] = V[i];
    t.Vt[i] = vt[i];
  }
  t.n = p.n;
  t.r = p.r;
  t.rp = p.rp;
  t.dtype = p.in_dtype;
  const long long total = (long long)p.rp * p.n;
  hipLaunchKernelGGL(k_transpose_v, dim3((unsigned)((total + 255) / 256), (unsigned)count), dim3(256), 0, stream,
                     t);
  return zo_hip_status(hipGetLastError(), "k_transpose_v");
}

// B' of `count` factors that share r, rp, the blocks and eps (heights may differ): one launch.
static int launch_bprime(const PlinearPlan* plans, int count, const BlkTable& tab, float eps,
                         const float* const* U, const float* const* Z, void* const* bp, hipStream_t stream) {
  const PlinearPlan& p = plans[0];
  BpArgs a{};
  int mmax = 0;
  for (int i = 0; i < count; ++i) {
    a.U[i] = U[i];
    a.Z[i] = Z[i];
    a.Bp[i] = bp[i];
    a.m[i] = plans[i].m;
    mmax = std::max(mmax, plans[i].m);
  }
  a.r = p.r;
  a.rp = p.rp;
  a.nblk = p.nblk;
  a.out_bf16 = p.in16;
  a.eps = eps;
  a.tab = tab;
  auto grid = [&](int rows) { return dim3((unsigned)((mmax + rows - 1) / rows), (unsigned)p.q, (unsigned)count); };
  switch ((p.r + 31) / 32) {
    case 1: hipLaunchKernelGGL(k_bprime<1>, grid(BpShape<1>::R), dim3(256), 0, stream, a); break;
    case 2: hipLaunchKernelGGL(k_bprime<2>, grid(BpShape<2>::R), dim3(256), 0, stream, a); break;
    case 3: hipLaunchKernelGGL(k_bprime<3>, grid(BpShape<3>::R), dim3(256), 0, stream, a); break;
    default: hipLaunchKernelGGL(k_bprime<4>, grid(BpShape<4>::R), dim3(256), 0, stream, a); break;
  }
  return zo_hip_status(hipGetLastError(), "k_bprime");
}

int zo_plinear_prepare(const PlinearPlan& p, const int* blk_query, const int8_t* blk_sign,
                       float eps, const void* X, const float* U, const float* V, const float* Z,
                       void* ws, hipStream_t stream) {
  const PlinearWs w = zo_plinear_ws(p, ws);
  int st;
  void* vt = w.vt;
  void* bp = w.bp;
  if ((st = launch_transpose_v(&p, 1, &V, &vt, stream)) != ZO_OK) return st;
  if ((st = launch_bprime(&p, 1, zo_blk_table(p.nblk, blk_query, blk_sign), eps, &U, &Z, &bp, stream)) != ZO_OK)
    return st;
  return zo_plinear_project(p, X, ws, stream);
}

// The 16-bit projection GEMM P2 = X_x Vt2^T of every distinct X block: A = vt (rows_a rows,
// n deep), output fp32 rows_a wide.
static int launch_projection(const PlinearPlan& p, const void* X, const void* vt, int rows_a, void* p2,
                             hipStream_t stream) {
  GemmArgs g{};
  g.A = (const bf16_t*)vt;
  g.B = (const bf16_t*)X;
  g.b_block_stride = p.x_block_stride;
  g.rows_a = rows_a;
  g.rows_b = p.T;
  g.K = p.n;
  g.nblk = p.nx;
  g.rc = 0;
  g.Y = p2;
  g.y_block_stride = (long long)p.T * rows_a;
  g.ldy = rows_a;
  g.out_dtype = ZO_F32;
  // From 128 rows on, the main GEMM's pipeline (256 x 256 tiles: the 2 rp = 128 rows of one
  // r = 64 factor fill half a tile, a stacked q, k, v projection 384 of 512 rows): it keeps the X
  // stream and the MFMAs overlapped better than the register-staged kernel even with the idle
  // rows (OPT-13B-shaped stack: prepare 130 -> 103 ms per step).  Otherwise 64 x 256 tiles;
  // 64 x 128 when that leaves fewer than two workgroups per CU.  Tile shapes change no
  // element's arithmetic.
  const bool f16 = p.in_dtype == ZO_F16;
  if (rows_a >= 128 && main_gemm_fits(g)) return launch_gemm_main(g, f16, stream);
  const long long tiles = (long long)p.nx * ((p.T + 255) / 256) * ((rows_a + 63) / 64);
  if (tiles < 512)
    return f16 ? launch_gemm_bf16<1, 4, 2, 1, true>(g, stream) : launch_gemm_bf16<1, 4, 2, 1, false>(g, stream);
  return f16 ? launch_gemm_bf16<1, 4, 2, 2, true>(g, stream) : launch_gemm_bf16<1, 4, 2, 2, false>(g, stream);
}

static int launch_pcombine(const PlinearPlan& p, const float* p2, int ld2, void* pp, hipStream_t stream) {
  const long long prow = (long long)p.nx * p.T;
  hipLaunchKernelGGL(k_pcombine, dim3((unsigned)((prow * p.rp + 255) / 256)), dim3(256), 0, stream, p2,
                     prow, p.rp, ld2, p.in_dtype == ZO_F16 ? 1.f / ZO_F16_RSCALE : 1.f, (bf16_t*)pp);
  return zo_hip_status(hipGetLastError(), "k_pcombine");
}

// A stack of `count` 16-bit factors (rp = 32 or 64; vt: count x 2 rp rows) projected on the main
// GEMM with the combine in its epilogue, factor i's [P_hi | P_hi | P_lo] into pc[i].  False when
// the stack does not fit that kernel (the caller then projects to fp32 and combines apart).
static bool proj_main_fits(const PlinearPlan& p, int count) {
  GemmArgs g{};
  g.rows_a = count * 2 * p.rp;
  g.rows_b = p.T;
  g.K = p.n;
  return p.in16 && (p.rp == 32 || p.rp == 64) && count >= 1 && count <= ZO_MAX_GROUP && g.rows_a >= 128 &&
         main_gemm_fits(g);
}

static int launch_proj_main(const PlinearPlan& p, const void* X, const void* vt, int count, bf16_t* const* pc,
                            hipStream_t stream) {
  GemmArgs g{};
  g.A = (const bf16_t*)vt;
  g.B = (const bf16_t*)X;
  g.b_block_stride = p.x_block_stride;
  g.rows_a = count * 2 * p.rp;
  g.rows_b = p.T;
  g.K = p.n;
  g.nblk = p.nx;
  g.rc = 0;
  g.out_dtype = p.in_dtype;  // selects the F16 / BF16 instantiation; nothing is written to Y
  g.epi = p.rp == 32 ? EPI_PROJ32 : EPI_PROJ64;
  for (int i = 0; i < count; ++i) g.pc[i] = pc[i];
  g.pcount = count;
  g.unscale = p.in_dtype == ZO_F16 ? 1.f / ZO_F16_RSCALE : 1.f;
  return launch_gemm_main(g, p.in_dtype == ZO_F16, stream);
}

// The fused projection (k_proj): 16-bit factors of 64 or 128 rows (rp = 32 or 64), each
// operand's buffer descriptor below 2^32 bytes.
static bool proj_fused_fits(const PlinearPlan& p, int count) {
  const unsigned long long lim = (1ull << 32) - 256;
  return p.in16 && (p.rp == 32 || p.rp == 64) && p.n % 32 == 0 && count >= 1 && count <= ZO_MAX_GROUP &&
         (unsigned long long)p.T * p.n * 2 <= lim && (unsigned long long)count * 2 * p.rp * p.n * 2 <= lim;
}

// [P_hi | P_hi | P_lo] of `count` stacked factors (vt: count x 2 rp rows) for every distinct X
// block, into pc[i] for factor i.
static int launch_proj_fused(const PlinearPlan& p, const void* X, const void* vt, int count,
                             bf16_t* const* pc, hipStream_t stream) {
  ProjArgs a{};
  a.V = (const bf16_t*)vt;
  a.X = (const bf16_t*)X;
  a.x_block_stride = p.x_block_stride;
  a.rows_v = count * 2 * p.rp;
  a.T = p.T;
  a.K = p.n;
  a.count = count;
  a.tiles_t = (p.T + 255) / 256;
  a.tiles_c = (a.rows_v + 127) / 128;
  const long long total = (long long)p.nx * a.tiles_t * a.tiles_c;
  if (total <= 0) return ZO_OK;
  if (total > 0x7fffffffLL) {
    zo_set_error("perturbed linear: too many projection tiles (%lld)", total);
    return ZO_ERR_UNSUPPORTED;
  }
  a.total_tiles = (int)total;
  a.unscale = p.in_dtype == ZO_F16 ? 1.f / ZO_F16_RSCALE : 1.f;
  for (int i = 0; i < count; ++i) a.pc[i] = pc[i];
  const dim3 grid((unsigned)total);
  const bool f16 = p.in_dtype == ZO_F16;
  if (p.rp == 32) {
    if (f16) hipLaunchKernelGGL((k_proj<true, 32>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((k_proj<false, 32>), grid, dim3(256), 0, stream, a);
  } else {
    if (f16) hipLaunchKernelGGL((k_proj<true, 64>), grid, dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((k_proj<false, 64>), grid, dim3(256), 0, stream, a);
  }
  return zo_hip_status(hipGetLastError(), "k_proj");
}

size_t zo_plinear_group_ws(const PlinearPlan& p, int count) {
  if (!p.in16 || count < 2) return 0;
  return zo_align256((size_t)count * 2 * p.rp * p.n * 2) +
         zo_align256((size_t)p.nx * p.T * count * 2 * p.rp * 4);
}

int zo_plinear_prepare_group(const PlinearPlan* plans, int count, const int* blk_query,
                             const int8_t* blk_sign, float eps, const void* X, const float* const* U,
                             const float* const* V, const float* const* Z, void* const* ws, void* gws,
                             hipStream_t stream) {
  int st;
  if (count < 2 || !plans[0].in16) {
    for (int i = 0; i < count; ++i)
      if ((st = zo_plinear_prepare(plans[i], blk_query, blk_sign, eps, X, U[i], V[i], Z[i], ws[i], stream)) !=
          ZO_OK)
        return st;
    return ZO_OK;
  }
  const PlinearPlan& p0 = plans[0];
  const int w2 = 2 * p0.rp;  // rows of one matrix's Vt2 (a multiple of 64: whole projection tiles)
  char* gvt = (char*)gws;
  float* gp2 = (float*)(gvt + zo_align256((size_t)count * w2 * p0.n * 2));
  const BlkTable tab = zo_blk_table(p0.nblk, blk_query, blk_sign);
  // Vt2 and B' of every factor of the group: one launch each.
  void* vts[ZO_MAX_GROUP];
  void* bps[ZO_MAX_GROUP];
  for (int i = 0; i < count; ++i) {
    vts[i] = gvt + (size_t)i * w2 * p0.n * 2;
    bps[i] = zo_plinear_ws(plans[i], ws[i]).bp;
  }
  if ((st = launch_transpose_v(plans, count, V, vts, stream)) != ZO_OK) return st;
  if ((st = launch_bprime(plans, count, tab, eps, U, Z, bps, stream)) != ZO_OK) return st;
  // A stack of several factors stays on the main GEMM's 256-row tiles (two factors of 128 rows
  // per X tile: the stacked q, k, v run 0.50 ms there against 0.72 ms in three 128-row tiles of
  // k_proj), with the combine in its epilogue; only a 64-row pair shares one 128-row tile.
  bf16_t* pc[ZO_MAX_GROUP];
  for (int i = 0; i < count; ++i) pc[i] = (bf16_t*)zo_plinear_ws(plans[i], ws[i]).pp;
  if (2 * p0.rp * count <= 128 && proj_fused_fits(p0, count)) return launch_proj_fused(p0, X, gvt, count, pc, stream);
  if (proj_main_fits(p0, count)) return launch_proj_main(p0, X, gvt, count, pc, stream);
  if ((st = launch_projection(p0, X, gvt, count * w2, gp2, stream)) != ZO_OK) return st;
  for (int i = 0; i < count; ++i)
    if ((st = launch_pcombine(plans[i], gp2 + (size_t)i * w2, count * w2, zo_plinear_ws(plans[i], ws[i]).pp,
                              stream)) != ZO_OK)
      return st;
  return ZO_OK;
}

int zo_plinear_project(const PlinearPlan& p, const void* X, void* ws, hipStream_t stream) {
  const PlinearWs w = zo_plinear_ws(p, ws);
  void* vt = w.vt;
  void* p2 = w.p2;
  void* pp = w.pp;
  int st;
  const long long xs = p.x_block_stride;
  if (p.in16) {
    if (proj_fused_fits(p, 1)) {
      bf16_t* pc = (bf16_t*)pp;
      return launch_proj_fused(p, X, vt, 1, &pc, stream);
    }
    if ((st = launch_projection(p, X, vt, 2 * p.rp, p2, stream)) != ZO_OK) return st;
    return launch_pcombine(p, (const float*)p2, 2 * p.rp, pp, stream);
  }
  F32Args g{};
  g.A = (const float*)vt;
  g.B = (const float*)X;
  g.b_block_stride = xs;
  g.rows_a = p.rp;
  g.rows_b = p.T;
  g.K = p.n;
  g.rc = 0;
  g.Y = (float*)pp;
  g.y_block_stride = (long long)p.T * p.rp;
  g.ldy = p.rp;
  dim3 grid((p.rp + 63) / 64, (p.T + 63) / 64, p.nx);
  hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, stream, g);
  return zo_hip_status(hipGetLastError(), "k_gemm_f32 (projection)");
}

int zo_gemm_plain(int T, int m, int n, int nblk, int dtype, const void* X, long long x_block_stride,
                  const void* W, void* Y, int epi, const void* R, long long r_block_stride,
                  hipStream_t stream) {
  GemmArgs h{};
  h.A = (const bf16_t*)W;
  h.B = (const bf16_t*)X;
  h.b_block_stride = x_block_stride;
  h.rows_a = m;
  h.rows_b = T;
  h.K = n;
  h.nblk = nblk;
  h.rc = 0;
  h.Y = Y;
  h.y_block_stride = (long long)T * m;
  h.ldy = m;
  h.out_dtype = dtype;
  h.epi = epi;
  h.R = R;
  h.r_block_stride = r_block_stride;
  const bool f16 = dtype == ZO_F16;
  if (main_gemm_fits(h)) return launch_gemm_main(h, f16, stream);
  return f16 ? launch_gemm_bf16<2, 4, 4, 2, true>(h, stream) : launch_gemm_bf16<2, 4, 4, 2, false>(h, stream);
}

// Shared X (one X for every block): X W^T once into the fp32 base, then per block only the
// rank-r term, added to the base before the epilogue (plain or ReLU; the others take the
// per-block path).  The MFMA work drops from nblk products to one.
static int apply_fan(const PlinearPlan& p, const PlinearWs& w, const void* X, const void* W, void* Y,
                     hipStream_t stream, int epi) {
  const bool f16 = p.in_dtype == ZO_F16;
  GemmArgs b{};
  b.A = (const bf16_t*)W;
  b.B = (const bf16_t*)X;
  b.rows_a = p.m;
  b.rows_b = p.T;
  b.K = p.n;
  b.nblk = 1;
  b.Y = w.base;
  b.ldy = p.m;
  b.out_dtype = ZO_F32;
  b.epi = ZO_EPI_NONE;
  GemmArgs h{};
  h.A = (const bf16_t*)W;
  h.B = (const bf16_t*)X;
  h.rows_a = p.m;
  h.rows_b = p.T;
  h.K = 0;
  h.nblk = p.nblk;
  h.ca = (const bf16_t*)w.bp;
  h.ca_block_stride = (long long)p.m * 3 * p.rp;
  h.cb = (const bf16_t*)w.pp;
  h.cb_block_stride = 0;
  h.rc = 3 * p.rp;
  h.Y = Y;
  h.y_block_stride = (long long)p.T * p.m;
  h.ldy = p.m;
  h.out_dtype = p.out_dtype;
  h.epi = epi == ZO_EPI_RELU ? EPI_BASE_RELU : EPI_BASE;
  h.R = w.base;
  h.r_block_stride = 0;
  h.blk_inner = 1;
  int st = launch_gemm_main(b, f16, stream);
  if (st != ZO_OK) return st;
  // No main-segment tiles here (K = 0): f16 only selects the fp16 output type.
  return launch_gemm_main(h, f16, stream);
}

static bool fan_fits(const PlinearPlan& p, int epi) {
  if (!p.fan || !p.in16 || (epi != ZO_EPI_NONE && epi != ZO_EPI_RELU)) return false;
  GemmArgs b{};
  b.rows_a = p.m;
  b.rows_b = p.T;
  b.K = p.n;
  GemmArgs h{};
  h.rows_a = p.m;
  h.rows_b = p.T;
  h.rc = 3 * p.rp;
  return main_gemm_fits(b) && main_gemm_fits(h);
}

int zo_plinear_apply(const PlinearPlan& p, const void* X, const void* W, void* Y, void* ws,
                     hipStream_t stream, int epi, const void* R, long long r_block_stride) {
  const PlinearWs w = zo_plinear_ws(p, ws);
  void* pp = w.pp;
  void* bp = w.bp;
  const long long xs = p.x_block_stride;
  if (fan_fits(p, epi)) return apply_fan(p, w, X, W, Y, stream, epi);
  if (p.in16) {
    GemmArgs h{};
    h.A = (const bf16_t*)W;
    h.B = (const bf16_t*)X;
    h.b_block_stride = xs;
    h.rows_a = p.m;
    h.rows_b = p.T;
    h.K = p.n;
    h.nblk = p.nblk;
    h.ca = (const bf16_t*)bp;
    h.ca_block_stride = (long long)p.m * 3 * p.rp;
    h.cb = (const bf16_t*)pp;
    h.cb_block_stride = p.nx == 1 ? 0 : (long long)p.T * 3 * p.rp;
    h.rc = 3 * p.rp;
    h.Y = Y;
    h.y_block_stride = (long long)p.T * p.m;
    h.ldy = p.m;
    h.out_dtype = p.out_dtype;
    h.epi = epi;
    h.R = R;
    h.r_block_stride = r_block_stride;
    const bool f16 = p.in_dtype == ZO_F16;
    if (main_gemm_fits(h)) return launch_gemm_main(h, f16, stream);
    return f16 ? launch_gemm_bf16<2, 4, 4, 2, true>(h, stream) : launch_gemm_bf16<2, 4, 4, 2, false>(h, stream);
  }
  F32Args h{};
  h.A = (const float*)W;
  h.B = (const float*)X;
  h.b_block_stride = xs;
  h.rows_a = p.m;
  h.rows_b = p.T;
  h.K = p.n;
  h.ca = (const float*)bp;
  h.ca_block_stride = (long long)p.m * p.rp;
  h.cb = (const float*)pp;
  h.cb_block_stride = p.nx == 1 ? 0 : (long long)p.T * p.rp;
  h.rc = p.rp;
  h.Y = (float*)Y;
  h.y_block_stride = (long long)p.T * p.m;
  h.ldy = p.m;
  h.epi = epi;
  h.R = (const float*)R;
  h.r_block_stride = r_block_stride;
  if (p.fan) {
    // Shared X: X W^T once into the base, then each block's rank-r term added to it.
    F32Args b = h;
    b.rc = 0;
    b.Y = (float*)w.base;
    b.y_block_stride = 0;
    b.epi = ZO_EPI_NONE;
    b.R = nullptr;
    b.r_block_stride = 0;
    hipLaunchKernelGGL(k_gemm_f32, dim3((p.m + 63) / 64, (p.T + 63) / 64, 1), dim3(256), 0, stream, b);
    int st = zo_hip_status(hipGetLastError(), "k_gemm_f32 (shared X)");
    if (st != ZO_OK) return st;
    h.K = 0;
    h.base = (const float*)w.base;
  }
  dim3 grid((p.m + 63) / 64, (p.T + 63) / 64, p.nblk);
  hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, stream, h);
  return zo_hip_status(hipGetLastError(), "k_gemm_f32");
}

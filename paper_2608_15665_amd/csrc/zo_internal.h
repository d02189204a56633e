// Internal declarations shared by the HIP sources of libzo (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "zo.h"

typedef uint16_t bf16_t;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// ---------------------------------------------------------------- host side
void zo_set_error(const char* fmt, ...);
int zo_hip_status(hipError_t e, const char* what);

static inline size_t zo_align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Carves consecutive 256-byte aligned regions out of a workspace.
struct WsCarver {
  char* base;
  size_t off;
  explicit WsCarver(void* p) : base((char*)p), off(0) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += zo_align256(bytes);
    return p;
  }
};

// ---------------------------------------------------------------- device side
__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Round to nearest even with gfx950's conversion instruction (v_cvt_pk_bf16_f32);
// NaN stays NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}

// Two values in one instruction: lo in bits 0..15, hi in bits 16..31.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// IEEE binary16: conversion from fp32 rounds to nearest even (v_cvt_f16_f32
// under the default mode), overflowing to infinity.
__device__ __forceinline__ float f16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}
__device__ __forceinline__ uint16_t f32_to_f16(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  return (uint32_t)f32_to_f16(lo) | ((uint32_t)f32_to_f16(hi) << 16);
}

// fp16 inputs: the projection's right factor (V, or LoRA's [A ; V_A^T]) is
// split into fp16 hi + lo after scaling by this power of two, so that the low
// parts of entries near 1/sqrt(n) stay normal numbers; the projection undoes
// it exactly.  Entries must stay below 65504 / 256 in magnitude.
constexpr float ZO_F16_RSCALE = 256.f;

// Element idx of the projection's right factor: fp32 as is; 16-bit as a hi
// part at idx and the rounded remainder at lo_off + idx (fp16: of 256 v).
__device__ __forceinline__ void put_split(void* Vt, long long idx, long long lo_off, float v,
                                          int dtype) {
  if (dtype == ZO_BF16) {
    const bf16_t hi = f32_to_bf16(v);
    ((bf16_t*)Vt)[idx] = hi;
    ((bf16_t*)Vt)[lo_off + idx] = f32_to_bf16(v - bf16_to_f32(hi));
  } else if (dtype == ZO_F16) {
    const float x = v * ZO_F16_RSCALE;
    const uint16_t hi = f32_to_f16(x);
    ((uint16_t*)Vt)[idx] = hi;
    ((uint16_t*)Vt)[lo_off + idx] = f32_to_f16(x - f16_to_f32(hi));
  } else {
    ((float*)Vt)[idx] = v;
  }
}

// ---------------------------------------------------------------- launchers
// Perturbed linear (zo_gemm.hip).
struct PlinearPlan {
  int T, m, n, r, rp, q, nblk, nx;  // nx: number of distinct X blocks (1 or nblk)
  long long x_block_stride;
  int in16;                 // 16-bit inputs (bf16 or fp16): MFMA path
  int in_dtype, out_dtype;  // zo_dtype values
  int fan;                  // one X shared by nblk > 1 blocks: X W^T once, then the blocks' terms
  size_t ws_vt, ws_p2, ws_p, ws_bp, ws_base;  // bytes of each workspace region
  size_t ws_total;
};
int zo_plinear_plan(PlinearPlan* p, int T, int m, int n, int r, int q, int nblk,
                    long long x_block_stride, int in_dtype, int out_dtype);
// Workspace regions of a plan, in carving order.
struct PlinearWs {
  void* vt;  // right factor, transposed: bf16 2 rp x n (hi rows, then lo rows); fp32 rp x n
  void* p2;  // bf16 inputs: X_b Vt^T in fp32, 2 rp wide (nullptr for fp32)
  void* pp;  // left correction operand per X block: bf16 [P_hi | P_hi | P_lo]; fp32 rp wide
  void* bp;  // right correction operand per block: bf16 [B_hi | B_lo | B_hi]; fp32 rp wide
  void* base;  // shared X only: X W^T in fp32, T x m (nullptr otherwise)
};
PlinearWs zo_plinear_ws(const PlinearPlan& p, void* ws);
// Query table of a call: j(b) and s(b) packed as j | (s + 1) << 16.
struct BlkTable {
  int code[ZO_MAX_BLOCKS];
};
BlkTable zo_blk_table(int nblk, const int* blk_query, const int8_t* blk_sign);
// P = X_b Vt^T for every distinct X block, from the vt region already filled.
int zo_plinear_project(const PlinearPlan& p, const void* X, void* ws, hipStream_t stream);
// LoRA scheme: fills vt with [A ; V_A^T] and bp with the per-block right factor
// (plan rank r = rl + rs), then projects.
int zo_lora_prepare(const PlinearPlan& p, int rl, int rs, const int* blk_query,
                    const int8_t* blk_sign, float eps, float scale, const void* X, const float* A,
                    const float* UA, const float* VA, const float* ZA, const float* B,
                    const float* UB, const float* VB, const float* ZB, void* ws,
                    hipStream_t stream);
int zo_plinear_prepare(const PlinearPlan& p, const int* blk_query, const int8_t* blk_sign,
                       float eps, const void* X, const float* U, const float* V,
                       const float* Z, void* ws, hipStream_t stream);
// Prepare of `count` perturbed linears that read the same X (plans equal but for m; 16-bit):
// their Vt2 factors stacked into one projection GEMM, so X is read once for all of them.
// ws[i] is matrix i's own workspace (apply reads it afterwards); gws holds the stacked
// factors and projections, zo_plinear_group_ws bytes.  Results are bitwise those of
// separate prepares (every projection tile covers one matrix's rows).  fp32 plans, or
// count < 2, take the separate prepares.
size_t zo_plinear_group_ws(const PlinearPlan& p, int count);
// X_b W^T for every block with no perturbation (a frozen matrix): the fused GEMM without its
// rank-r segment, with the same epilogues.  16-bit inputs and outputs of one type.
int zo_gemm_plain(int T, int m, int n, int nblk, int dtype, const void* X, long long x_block_stride,
                  const void* W, void* Y, int epi, const void* R, long long r_block_stride,
                  hipStream_t stream);
int zo_plinear_prepare_group(const PlinearPlan* plans, int count, const int* blk_query,
                             const int8_t* blk_sign, float eps, const void* X, const float* const* U,
                             const float* const* V, const float* const* Z, void* const* ws, void* gws,
                             hipStream_t stream);
// Decoder-layer pieces (zo_decoder.hip).
int zo_layernorm_launch(long long rows, int d, int dtype, const void* X, const float* gamma,
                        const float* beta, float eps_ln, void* Y, hipStream_t stream, bool rms = false);
int zo_rope_launch(long long rows, int seq_len, int d, int heads, int dtype, void* X, float base,
                   hipStream_t stream);
int zo_attention_launch(int nblk, int T, int seq_len, int d, int heads, int kv_heads, int dtype,
                        const void* Q, const void* K, const void* V, void* O, hipStream_t stream);
int zo_plinear_apply(const PlinearPlan& p, const void* X, const void* W, void* Y, void* ws,
                     hipStream_t stream, int epi = ZO_EPI_NONE, const void* R = nullptr,
                     long long r_block_stride = 0);

// Subspace update (zo_update.hip): Adam (sgd = 0) or plain SGD in the subspace (sgd = 1,
// S = Zbar; the moments are neither read nor written).
int zo_update_launch(int count, const zo_update_item* items, int w_dtype, int r, int q,
                     const float* g, int t, float lr, float beta1, float beta2,
                     float eps_adam, int sgd, int* nonfinite_flag, void* ws, size_t ws_bytes,
                     hipStream_t stream, size_t* ws_needed);

// Subspace refresh, CholeskyQR2 (zo_qr.hip).
int zo_refresh_launch(int count, const zo_panel* panels, int r, int* info, void* ws,
                      size_t ws_bytes, hipStream_t stream, size_t* ws_needed);
// Device address of the current device's static refresh scratch (ZO_NOALLOC_SCRATCH_BYTES),
// looked up on the first call per device and cached.
int zo_refresh_scratch(void** ptr);

// Loss helpers (zo_loss.hip).
int zo_sq_loss_launch(int nblk, int T, int m, int dtype, const void* Y, const void* Ystar,
                      double* out, void* ws, size_t ws_bytes, hipStream_t stream,
                      size_t* ws_needed);
int zo_combine_central_launch(int q, const double* L, float eps, float* g,
                              hipStream_t stream);
int zo_combine_forward_launch(int q, const double* L, float eps, float* g, hipStream_t stream);

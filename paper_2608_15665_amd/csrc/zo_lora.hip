// LoRA scheme of SubZero+: the trainable parameters of an adapted layer are the
// two adapter factors A (r_L x n) and B (m x r_L), each perturbed in its own
// rank-r subspace (Eq. 4 and Alg. 2 applied to every trainable matrix; the
// paper's LoRA runs use r_L = 8, alpha = 16).  Query j with sign s gives
//   A' = A + s eps U_A Z_A,j V_A^T,   B' = B + s eps U_B Z_B,j V_B^T,
//   Y_b = X_b W^T + scale (X_b A'^T) B'^T          (scale = alpha / r_L).
// The adapter branch is a rank-(r_L + r) correction of the frozen-base GEMM:
//   X_b A'^T = X_b A^T + s eps (X_b V_A) (U_A Z_A,j)^T, so
//   Y_b = X_b W^T + P_b Bt_b^T  with  P_b = X_b [A^T | V_A]        (T x (r_L + r)),
//                                     Bt_b = scale [B' | s eps B' U_A Z_A,j]  (m x (r_L + r)).
// P_b depends on the activations only, so it is formed once per distinct X
// block by the same projection pass as the full-tuning path; Bt_b is tiny.  The
// fused GEMM of the full-tuning path then runs unchanged with rank r_L + r.
#include "zo_internal.h"

namespace {

// Vt rows a < rl: A[a][:]; rows rl <= a < rl + rs: V_A[:][a - rl]; zero up to rp.
// 16-bit: hi part in rows [0, rp), low part (x - hi, rounded) in rows [rp, 2 rp);
// fp16 splits 256 x (the projection scales back exactly).
__global__ __launch_bounds__(256) void k_lora_vt(const float* __restrict__ A,
                                                 const float* __restrict__ VA, int n, int rl,
                                                 int rs, int rp, void* Vt, int dtype) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (long long)rp * n) return;
  const int a = (int)(idx / n), k = (int)(idx % n);
  float v = 0.f;
  if (a < rl)
    v = A[(size_t)a * n + k];
  else if (a < rl + rs)
    v = VA[(size_t)k * rs + (a - rl)];
  put_split(Vt, idx, (long long)rp * n, v, dtype);
}

// B'[i][c] = B[i][c] + s eps sum_e U_B[i][e] sum_f Z_B[e][f] V_B[c][f].
__device__ __forceinline__ float lora_bp(const float* __restrict__ B, const float* __restrict__ UB,
                                         const float* __restrict__ VB, const float* __restrict__ ZBj,
                                         int i, int c, int rl, int rs, float se) {
  float acc = 0.f;
  for (int e = 0; e < rs; ++e) {
    float zv = 0.f;
    for (int f = 0; f < rs; ++f) zv = fmaf(ZBj[e * rs + f], VB[(size_t)c * rs + f], zv);
    acc = fmaf(UB[(size_t)i * rs + e], zv, acc);
  }
  return fmaf(se, acc, B[(size_t)i * rl + c]);
}

// Bt_b[i][a]: scale B'[i][a] for a < rl; scale s eps sum_c B'[i][c] (U_A Z_A,j)[c][a - rl]
// for rl <= a < rl + rs; zero up to rp.  Layouts as the full-tuning right factor:
// fp32 m x rp per block, bf16 m x 3 rp per block as [hi | lo | hi].
__global__ __launch_bounds__(256) void k_lora_bprime(
    const float* __restrict__ B, const float* __restrict__ UB, const float* __restrict__ VB,
    const float* __restrict__ ZB, const float* __restrict__ UA, const float* __restrict__ ZA, int m,
    int rl, int rs, int rp, int nblk, float eps, float scale, BlkTable tab, void* Bp,
    int out_bf16) {
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long per = (long long)m * rp;
  if (idx >= per * nblk) return;
  const int b = (int)(idx / per);
  const long long rem = idx - (long long)b * per;
  const int i = (int)(rem / rp), a = (int)(rem % rp);
  const int code = tab.code[b];
  const int j = code & 0xffff;
  const float se = (float)((code >> 16) - 1) * eps;
  const float* __restrict__ ZBj = ZB + (size_t)j * rs * rs;
  float v = 0.f;
  if (a < rl) {
    v = scale * lora_bp(B, UB, VB, ZBj, i, a, rl, rs, se);
  } else if (a < rl + rs) {
    const int f = a - rl;
    const float* __restrict__ ZAj = ZA + (size_t)j * rs * rs;
    float acc = 0.f;
    for (int c = 0; c < rl; ++c) {
      float uz = 0.f;
      for (int e = 0; e < rs; ++e) uz = fmaf(UA[(size_t)c * rs + e], ZAj[e * rs + f], uz);
      acc = fmaf(lora_bp(B, UB, VB, ZBj, i, c, rl, rs, se), uz, acc);
    }
    v = scale * se * acc;
  }
  if (out_bf16) {
    const bf16_t hi = f32_to_bf16(v);
    const bf16_t lo = f32_to_bf16(v - bf16_to_f32(hi));
    bf16_t* o = (bf16_t*)Bp + ((long long)b * m + i) * 3 * rp;
    o[a] = hi;
    o[rp + a] = lo;
    o[2 * rp + a] = hi;
  } else {
    ((float*)Bp)[idx] = v;
  }
}

}  // namespace

int zo_lora_prepare(const PlinearPlan& p, int rl, int rs, const int* blk_query,
                    const int8_t* blk_sign, float eps, float scale, const void* X, const float* A,
                    const float* UA, const float* VA, const float* ZA, const float* B,
                    const float* UB, const float* VB, const float* ZB, void* ws,
                    hipStream_t stream) {
  const PlinearWs w = zo_plinear_ws(p, ws);
  int st;
  {
    const long long total = (long long)p.rp * p.n;
    hipLaunchKernelGGL(k_lora_vt, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream, A,
                       VA, p.n, rl, rs, p.rp, w.vt, p.in_dtype);
    if ((st = zo_hip_status(hipGetLastError(), "k_lora_vt")) != ZO_OK) return st;
  }
  {
    const BlkTable tab = zo_blk_table(p.nblk, blk_query, blk_sign);
    const long long total = (long long)p.nblk * p.m * p.rp;
    hipLaunchKernelGGL(k_lora_bprime, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, stream,
                       B, UB, VB, ZB, UA, ZA, p.m, rl, rs, p.rp, p.nblk, eps, scale, tab, w.bp,
                       p.in16);
    if ((st = zo_hip_status(hipGetLastError(), "k_lora_bprime")) != ZO_OK) return st;
  }
  return zo_plinear_project(p, X, ws, stream);
}

// Loss helpers for driving the hot path on a one-layer regression problem:
// per-block squared error and the central difference of Eq. 3 per query.
// Both reduce in float64 in a fixed order (deterministic, no atomics).
#include "zo_internal.h"

namespace {

constexpr int LOSS_CHUNK = 65536;  // elements per workgroup

__global__ __launch_bounds__(256) void k_sq_partial(const void* Y, const void* Ystar, int dtype,
                                                    long long per_block, int nchunk,
                                                    double* partial) {
  __shared__ double red[4];
  const int c = blockIdx.x, b = blockIdx.y;
  const long long lo = (long long)c * LOSS_CHUNK;
  const long long hi = min(lo + (long long)LOSS_CHUNK, per_block);
  double s = 0.0;
  if (dtype == ZO_BF16) {
    const bf16_t* y = (const bf16_t*)Y + (long long)b * per_block;
    const bf16_t* ys = (const bf16_t*)Ystar;
    for (long long e = lo + threadIdx.x; e < hi; e += 256) {
      const double d = (double)bf16_to_f32(y[e]) - (double)bf16_to_f32(ys[e]);
      s += d * d;
    }
  } else if (dtype == ZO_F16) {
    const uint16_t* y = (const uint16_t*)Y + (long long)b * per_block;
    const uint16_t* ys = (const uint16_t*)Ystar;
    for (long long e = lo + threadIdx.x; e < hi; e += 256) {
      const double d = (double)f16_to_f32(y[e]) - (double)f16_to_f32(ys[e]);
      s += d * d;
    }
  } else {
    const float* y = (const float*)Y + (long long)b * per_block;
    const float* ys = (const float*)Ystar;
    for (long long e = lo + threadIdx.x; e < hi; e += 256) {
      const double d = (double)y[e] - (double)ys[e];
      s += d * d;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) partial[(long long)b * nchunk + c] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ void k_sq_final(const double* partial, int nchunk, int nblk, int T, double* out) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nblk) return;
  double s = 0.0;
  for (int c = 0; c < nchunk; ++c) s += partial[(long long)b * nchunk + c];
  out[b] = 0.5 * s / (double)T;
}

__global__ void k_central(int q, const double* L, float eps, float* g) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < q) g[j] = (float)((L[2 * j] - L[2 * j + 1]) / (2.0 * (double)eps));
}

__global__ void k_forward(int q, const double* L, float eps, float* g) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < q) g[j] = (float)((L[1 + j] - L[0]) / (double)eps);
}

}  // namespace

int zo_sq_loss_launch(int nblk, int T, int m, int dtype, const void* Y, const void* Ystar,
                      double* out, void* ws, size_t ws_bytes, hipStream_t stream,
                      size_t* ws_needed) {
  const long long per = (long long)T * m;
  const int nchunk = (int)((per + LOSS_CHUNK - 1) / LOSS_CHUNK);
  const size_t need = zo_align256((size_t)nblk * nchunk * sizeof(double));
  if (ws_needed) *ws_needed = need;
  if (!ws) return ZO_OK;
  if (ws_bytes < need) {
    zo_set_error("sq_loss: workspace %zu bytes < required %zu", ws_bytes, need);
    return ZO_ERR_WORKSPACE;
  }
  double* partial = (double*)ws;
  hipLaunchKernelGGL(k_sq_partial, dim3(nchunk, nblk), dim3(256), 0, stream, Y, Ystar,
                     dtype, per, nchunk, partial);
  int st = zo_hip_status(hipGetLastError(), "k_sq_partial");
  if (st != ZO_OK) return st;
  hipLaunchKernelGGL(k_sq_final, dim3((nblk + 63) / 64), dim3(64), 0, stream, partial, nchunk,
                     nblk, T, out);
  return zo_hip_status(hipGetLastError(), "k_sq_final");
}

int zo_combine_central_launch(int q, const double* L, float eps, float* g, hipStream_t stream) {
  hipLaunchKernelGGL(k_central, dim3((q + 63) / 64), dim3(64), 0, stream, q, L, eps, g);
  return zo_hip_status(hipGetLastError(), "k_central");
}

int zo_combine_forward_launch(int q, const double* L, float eps, float* g, hipStream_t stream) {
  hipLaunchKernelGGL(k_forward, dim3((q + 63) / 64), dim3(64), 0, stream, q, L, eps, g);
  return zo_hip_status(hipGetLastError(), "k_forward");
}

// Loss helpers for driving the hot path on a one-layer regression problem:
// per-block squared error and the central difference of Eq. 3 per query.
// Both reduce in float64 in a fixed order (deterministic, no atomics).
#include "zo_internal.h"

namespace {

constexpr int LOSS_CHUNK = 65536;  // elements per workgroup

// Squared differences of the block's chunk, summed in float64 per thread, then over the
// workgroup in a fixed order.  With 16-byte alignment (VEC: the block's rows start on 16-byte
// boundaries) each thread reads 16 bytes of Y and of Y* per step; otherwise one element.
template <int DT, bool VEC>
__device__ __forceinline__ double sq_chunk(const void* Y, const void* Ystar, long long per_block, int b,
                                           long long lo, long long hi) {
  constexpr int E = DT == ZO_F32 ? 4 : 8;  // elements per 16 bytes
  auto val = [](const void* p, long long e) -> double {
    if constexpr (DT == ZO_BF16) return (double)bf16_to_f32(((const bf16_t*)p)[e]);
    else if constexpr (DT == ZO_F16) return (double)f16_to_f32(((const uint16_t*)p)[e]);
    else return (double)((const float*)p)[e];
  };
  const char* y = (const char*)Y + (long long)b * per_block * (DT == ZO_F32 ? 4 : 2);
  double s = 0.0;
  if constexpr (VEC) {
    for (long long e = lo + (long long)threadIdx.x * E; e < hi; e += 256LL * E) {
      const u32x4 a = *(const u32x4*)(y + e * (16 / E));
      const u32x4 c = *(const u32x4*)((const char*)Ystar + e * (16 / E));
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (DT == ZO_F32) {
          const double d = (double)__uint_as_float(a[k]) - (double)__uint_as_float(c[k]);
          s += d * d;
        } else {
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint16_t ya = (uint16_t)(a[k] >> (16 * h)), yc = (uint16_t)(c[k] >> (16 * h));
            const double d = DT == ZO_BF16 ? (double)bf16_to_f32(ya) - (double)bf16_to_f32(yc)
                                           : (double)f16_to_f32(ya) - (double)f16_to_f32(yc);
            s += d * d;
          }
        }
      }
    }
  } else {
    for (long long e = lo + threadIdx.x; e < hi; e += 256) {
      const double d = val(y, e) - val(Ystar, e);
      s += d * d;
    }
  }
  return s;
}

__global__ __launch_bounds__(256) void k_sq_partial(const void* Y, const void* Ystar, int dtype,
                                                    long long per_block, int nchunk, int vec,
                                                    double* partial) {
  __shared__ double red[4];
  const int c = blockIdx.x, b = blockIdx.y;
  const long long lo = (long long)c * LOSS_CHUNK;
  const long long hi = min(lo + (long long)LOSS_CHUNK, per_block);
  double s;
  if (dtype == ZO_BF16)
    s = vec ? sq_chunk<ZO_BF16, true>(Y, Ystar, per_block, b, lo, hi) : sq_chunk<ZO_BF16, false>(Y, Ystar, per_block, b, lo, hi);
  else if (dtype == ZO_F16)
    s = vec ? sq_chunk<ZO_F16, true>(Y, Ystar, per_block, b, lo, hi) : sq_chunk<ZO_F16, false>(Y, Ystar, per_block, b, lo, hi);
  else
    s = vec ? sq_chunk<ZO_F32, true>(Y, Ystar, per_block, b, lo, hi) : sq_chunk<ZO_F32, false>(Y, Ystar, per_block, b, lo, hi);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) partial[(long long)b * nchunk + c] = (red[0] + red[1]) + (red[2] + red[3]);
}

// One wave per block: lane l sums the chunk partials l, l + 64, ... in order, then the lanes
// are added in a fixed butterfly.
__global__ __launch_bounds__(64) void k_sq_final(const double* partial, int nchunk, int nblk, int T,
                                                 double* out) {
  const int b = blockIdx.x, l = threadIdx.x;
  double s = 0.0;
  for (int c = l; c < nchunk; c += 64) s += partial[(long long)b * nchunk + c];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (l == 0) out[b] = 0.5 * s / (double)T;
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
  // 16-byte loads when every block and both bases start on 16-byte boundaries (the chunks are
  // whole multiples of 16 bytes).
  const int esz = dtype == ZO_F32 ? 4 : 2;
  const int vec = (per * esz) % 16 == 0 && (uintptr_t)Y % 16 == 0 && (uintptr_t)Ystar % 16 == 0;
  hipLaunchKernelGGL(k_sq_partial, dim3(nchunk, nblk), dim3(256), 0, stream, Y, Ystar,
                     dtype, per, nchunk, vec, partial);
  int st = zo_hip_status(hipGetLastError(), "k_sq_partial");
  if (st != ZO_OK) return st;
  hipLaunchKernelGGL(k_sq_final, dim3(nblk), dim3(64), 0, stream, partial, nchunk, nblk, T, out);
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

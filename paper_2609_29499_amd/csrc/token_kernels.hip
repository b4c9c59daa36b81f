// Token-level kernels of the request loop: INT8 embedding lookup and greedy argmax, both reading
// their token ids from device memory so that a whole request (prefill + decode steps) is enqueued
// without a host round trip per token.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

// x[t][k] = scale[id] * table[id][k] for id = ids[t]; an id outside the vocabulary gives NaN rows
__global__ __launch_bounds__(kBlock) void embed_kernel(const int8_t* __restrict__ table,
                                                       const float* __restrict__ scale, int V, int d,
                                                       const int* __restrict__ ids, float* x) {
  const int t = blockIdx.x;
  const int id = ids[t];
  const bool ok = id >= 0 && id < V;
  const float s = ok ? scale[id] : __builtin_nanf("");
  const int8_t* row = table + size_t(ok ? id : 0) * d;
  float* out = x + size_t(t) * d;
  for (int k4 = threadIdx.x; k4 < d / 4; k4 += kBlock) {
    const char4 w = reinterpret_cast<const char4*>(row)[k4];
    reinterpret_cast<float4*>(out)[k4] = make_float4(s * float(w.x), s * float(w.y), s * float(w.z), s * float(w.w));
  }
}

// best of (v, i) and (w, j): the larger value, the lower index among equal ones
__device__ __forceinline__ void take_better(float& v, int& i, float w, int j) {
  if (w > v || (w == v && j < i)) {
    v = w;
    i = j;
  }
}

// ids_out[r] = argmax of logits row r (finite logits; the lowest id among equal maxima)
__global__ __launch_bounds__(kBlock) void argmax_kernel(const float* __restrict__ logits, int V,
                                                        int* ids_out) {
  __shared__ float sv[kBlock / kWave];
  __shared__ int si[kBlock / kWave];
  const float* row = logits + size_t(blockIdx.x) * V;
  float best = -INFINITY;
  int bi = 0;
  for (int i = threadIdx.x; i < V; i += kBlock) take_better(best, bi, row[i], i);
#pragma unroll
  for (int m = 1; m < kWave; m <<= 1) {
    const float w = __shfl_xor(best, m, kWave);
    const int j = __shfl_xor(bi, m, kWave);
    take_better(best, bi, w, j);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) {
    sv[wave] = best;
    si[wave] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kBlock / kWave; ++w) take_better(best, bi, sv[w], si[w]);
    ids_out[blockIdx.x] = bi;
  }
}

}  // namespace

hipError_t launch_embed(const int8_t* table, const float* scale, int V, int d, const int* ids,
                        int n, float* x, hipStream_t s) {
  if (n < 1) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_kernel, dim3(n), dim3(kBlock), 0, s, table, scale, V, d, ids, x);
  return hipGetLastError();
}

hipError_t launch_argmax(const float* logits, int n, int V, int* ids_out, hipStream_t s) {
  if (n < 1) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(n), dim3(kBlock), 0, s, logits, V, ids_out);
  return hipGetLastError();
}

}  // namespace tasp

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

// the workgroup's best (value, index) into thread 0 (take_better is associative and commutative,
// so the order of the reduction does not change the result)
__device__ __forceinline__ void block_best(float& best, int& bi, float* sv, int* si) {
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
  if (threadIdx.x == 0)
    for (int w = 1; w < kBlock / kWave; ++w) take_better(best, bi, sv[w], si[w]);
}

// ids_out[r] = argmax of logits row r (finite logits; the lowest id among equal maxima).
// Grid (chunks, rows): workgroup c takes logits [c K, (c + 1) K) of its row, K = kArgmaxChunk
// (all of them for a grid of one chunk), 16 independent loads per thread and pass. With several
// chunks, each workgroup stores its best (value, index) device-coherent and counts itself done;
// the last of the row reduces the partials and resets the counter.
__global__ __launch_bounds__(kBlock) void argmax_kernel(const float* __restrict__ logits, int V,
                                                        int* ids_out, float* part, int* cnt) {
  __shared__ float sv[kBlock / kWave];
  __shared__ int si[kBlock / kWave];
  __shared__ int last;
  constexpr int U = kArgmaxChunk / kBlock;
  const int n_ch = gridDim.x, c = blockIdx.x, r = blockIdx.y;
  const float* row = logits + size_t(r) * V;
  const int k0 = n_ch == 1 ? 0 : c * kArgmaxChunk;
  const int k1 = n_ch == 1 ? V : min(V, k0 + kArgmaxChunk);
  float best = -INFINITY;
  int bi = k0;
  for (int base = k0; base < k1; base += kArgmaxChunk) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = base + u * kBlock + int(threadIdx.x);
      v[u] = i < k1 ? row[i] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) take_better(best, bi, v[u], min(base + u * kBlock + int(threadIdx.x), k1 - 1));
  }
  block_best(best, bi, sv, si);
  if (n_ch == 1) {
    if (threadIdx.x == 0) ids_out[r] = bi;
    return;
  }
  const __amdgpu_buffer_rsrc_t rp = make_rsrc(part + size_t(r) * n_ch * 2, uint32_t(n_ch) * 8u);
  if (threadIdx.x == 0) {
    buf_store8_device(make_int2(__float_as_int(best), bi), rp, uint32_t(c) * 8u);
    __builtin_amdgcn_s_waitcnt(0);                      // the partial is at the coherence point
    last = __hip_atomic_fetch_add(cnt + r, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == n_ch - 1;
    if (last) __hip_atomic_store(cnt + r, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!last) return;
  best = -INFINITY;
  bi = 0;
  if (int(threadIdx.x) < n_ch) {
    const int2 pv = buf_load8_device(rp, uint32_t(threadIdx.x) * 8u);
    best = __int_as_float(pv.x);
    bi = pv.y;
  }
  block_best(best, bi, sv, si);
  if (threadIdx.x == 0) ids_out[r] = bi;
}

}  // namespace

hipError_t launch_embed(const int8_t* table, const float* scale, int V, int d, const int* ids,
                        int n, float* x, hipStream_t s) {
  if (n < 1) return hipSuccess;
  if (d % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_kernel, dim3(n), dim3(kBlock), 0, s, table, scale, V, d, ids, x);
  return hipGetLastError();
}

hipError_t launch_argmax(const float* logits, int n, int V, int* ids_out, float* part, int* cnt,
                         hipStream_t s) {
  if (n < 1) return hipSuccess;
  if (V < 1) return hipErrorInvalidValue;
  const int chunks = (V + kArgmaxChunk - 1) / kArgmaxChunk;
  const int n_ch = (part && cnt && n <= kArgmaxMaxRows && chunks <= kArgmaxMaxChunks) ? chunks : 1;
  hipLaunchKernelGGL(argmax_kernel, dim3(n_ch, n), dim3(kBlock), 0, s, logits, V, ids_out, part, cnt);
  return hipGetLastError();
}

}  // namespace tasp

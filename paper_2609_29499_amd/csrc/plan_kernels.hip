// Plan compilation kernels: dependency closure with ascending index lists, and the gathers that
// pack retained rows / columns of the INT8 store into contiguous panels.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

// Writes the ascending positions i < n with flag(i) != 0 to out[0..count) and returns count.
// Integer-only: a wave ballot gives each lane its rank inside 64 flags; four wave totals give the
// workgroup offset; a running base carries across 256-wide tiles. All threads get the count.
template <class Flag>
__device__ int block_compact(int n, Flag flag, int* out, int* wave_cnt) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int base = 0;
  for (int t0 = 0; t0 < n; t0 += kBlock) {
    const int i = t0 + tid;
    const bool f = (i < n) && flag(i);
    const unsigned long long bal = __ballot(f);
    const int rank = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wave_cnt[w] = __popcll(bal);
    __syncthreads();
    int off = base;
    for (int k = 0; k < w; ++k) off += wave_cnt[k];
    if (f) out[off + rank] = i;
    const int total = wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3];
    __syncthreads();
    base += total;
  }
  return base;
}

__global__ __launch_bounds__(kBlock) void closure_kernel(
    const uint8_t* __restrict__ q_keep, const uint8_t* __restrict__ kv_keep,
    const uint8_t* __restrict__ ffn_keep, int Hq, int Hkv, int F, int* q_idx, int* kv_idx,
    int* q_kvslot, int* slot_start, int* ffn_idx, int* counts) {
  __shared__ uint8_t qc[256];
  __shared__ uint8_t kvc[64];
  __shared__ int lq[256];
  __shared__ int lkv[64];
  __shared__ int wave_cnt[4];
  const int l = blockIdx.x, tid = threadIdx.x;
  const int r = Hq / Hkv;
  const uint8_t* q = q_keep + size_t(l) * Hq;
  const uint8_t* kv = kv_keep ? kv_keep + size_t(l) * Hkv : nullptr;
  // a query head survives only if its own group is kept; it is never moved to another group
  if (tid < Hq) qc[tid] = (q[tid] != 0) && (kv == nullptr || kv[tid / r] != 0);
  __syncthreads();
  // a KV group is active iff at least one of its query heads survived
  if (tid < Hkv) {
    uint8_t any = 0;
    for (int h = tid * r; h < (tid + 1) * r; ++h) any |= qc[h];
    kvc[tid] = any;
  }
  __syncthreads();
  const int m_q = block_compact(Hq, [&](int i) { return qc[i] != 0; }, lq, wave_cnt);
  const int m_kv = block_compact(Hkv, [&](int i) { return kvc[i] != 0; }, lkv, wave_cnt);
  const uint8_t* f = ffn_keep + size_t(l) * F;
  const int c = block_compact(F, [&](int i) { return f[i] != 0; }, ffn_idx + size_t(l) * F,
                              wave_cnt);
  // slots: the retained group of head q_idx[i] is lkv[q_kvslot[i]]; heads of one slot are a
  // contiguous run of the ascending head list because groups are contiguous head ranges
  if (tid < m_q) {
    const int g = lq[tid] / r;
    int slot = 0;
    for (int j = 0; j < m_kv; ++j) slot += (lkv[j] < g);
    q_idx[size_t(l) * Hq + tid] = lq[tid];
    q_kvslot[size_t(l) * Hq + tid] = slot;
  }
  if (tid <= m_kv) {
    int first = 0;
    if (tid < m_kv) {
      for (int i = 0; i < m_q; ++i) first += (lq[i] / r < lkv[tid]);
    } else {
      first = m_q;
    }
    slot_start[size_t(l) * (Hkv + 1) + tid] = first;
  }
  if (tid < m_kv) kv_idx[size_t(l) * Hkv + tid] = lkv[tid];
  if (tid == 0) {
    counts[l * 4 + 0] = m_q;
    counts[l * 4 + 1] = m_kv;
    counts[l * 4 + 2] = c;
    counts[l * 4 + 3] = 0;
  }
}

// One workgroup per destination row; 16-byte copies.
__global__ __launch_bounds__(kBlock) void gather_head_rows_kernel(
    int8_t* __restrict__ dst, const int8_t* __restrict__ src, const int* __restrict__ idx, int dh,
    int K, float* dst_scale, const float* __restrict__ src_scale) {
  const int row = blockIdx.x;
  const int i = row / dh, e = row % dh;
  const size_t srow = size_t(idx[i]) * dh + e;
  const int4* s = reinterpret_cast<const int4*>(src + srow * K);
  int4* d = reinterpret_cast<int4*>(dst + size_t(row) * K);
  for (int v = threadIdx.x; v < K / 16; v += kBlock) d[v] = s[v];
  if (threadIdx.x == 0) dst_scale[row] = src_scale[srow];
}

__global__ __launch_bounds__(kBlock) void gather_rows_kernel(
    int8_t* __restrict__ dst, const int8_t* __restrict__ src, const int* __restrict__ idx, int K,
    float* dst_scale, const float* __restrict__ src_scale) {
  const int row = blockIdx.x;
  const size_t srow = size_t(idx[row]);
  const int4* s = reinterpret_cast<const int4*>(src + srow * K);
  int4* d = reinterpret_cast<int4*>(dst + size_t(row) * K);
  for (int v = threadIdx.x; v < K / 16; v += kBlock) d[v] = s[v];
  if (threadIdx.x == 0) dst_scale[row] = src_scale[srow];
}

// One workgroup per row; each retained head contributes dh contiguous bytes (dh % 16 == 0).
__global__ __launch_bounds__(kBlock) void gather_head_cols_kernel(
    int8_t* __restrict__ dst, int dst_ld, const int8_t* __restrict__ src, int src_ld,
    const int* __restrict__ idx, int n, int dh) {
  const int row = blockIdx.x;
  const int per_head = dh / 16;
  const int8_t* s = src + size_t(row) * src_ld;
  int8_t* d = dst + size_t(row) * dst_ld;
  for (int u = threadIdx.x; u < n * per_head; u += kBlock) {
    const int i = u / per_head, v = u % per_head;
    *reinterpret_cast<int4*>(d + i * dh + v * 16) =
        *reinterpret_cast<const int4*>(s + size_t(idx[i]) * dh + v * 16);
  }
  for (int j = n * dh + threadIdx.x; j < dst_ld; j += kBlock) d[j] = 0;
}

__global__ __launch_bounds__(kBlock) void gather_cols_kernel(
    int8_t* __restrict__ dst, int dst_ld, const int8_t* __restrict__ src, int src_ld,
    const int* __restrict__ idx, int n) {
  const int row = blockIdx.x;
  const int8_t* s = src + size_t(row) * src_ld;
  int8_t* d = dst + size_t(row) * dst_ld;
  for (int j = threadIdx.x; j < dst_ld; j += kBlock) d[j] = (j < n) ? s[idx[j]] : int8_t(0);
}

// Streaming copy with 4 independent 16-byte loads in flight per thread.
__global__ __launch_bounds__(kBlock) void copy_kernel(int4* __restrict__ dst,
                                                      const int4* __restrict__ src, size_t n) {
  const size_t stride = size_t(gridDim.x) * kBlock;
  size_t i = size_t(blockIdx.x) * kBlock + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const int4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    dst[i] = a;
    dst[i + stride] = b;
    dst[i + 2 * stride] = c;
    dst[i + 3 * stride] = d;
  }
  for (; i < n; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(kBlock) void fill_zero_kernel(uint32_t* __restrict__ dst, size_t n) {
  const size_t stride = size_t(gridDim.x) * kBlock;
  for (size_t i = size_t(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride) dst[i] = 0u;
}

int grid_for(size_t n) {
  size_t g = (n + kBlock - 1) / kBlock;
  if (g > 2048) g = 2048;
  return g ? int(g) : 1;
}

}  // namespace

hipError_t launch_closure(const uint8_t* q_keep, const uint8_t* kv_keep, const uint8_t* ffn_keep,
                          int L, int Hq, int Hkv, int F, int* q_idx, int* kv_idx, int* q_kvslot,
                          int* slot_start, int* ffn_idx, int* counts, hipStream_t s) {
  hipLaunchKernelGGL(closure_kernel, dim3(L), dim3(kBlock), 0, s, q_keep, kv_keep, ffn_keep, Hq,
                     Hkv, F, q_idx, kv_idx, q_kvslot, slot_start, ffn_idx, counts);
  return hipGetLastError();
}

hipError_t launch_gather_head_rows(int8_t* dst, const int8_t* src, const int* idx, int n, int dh,
                                   int K, float* dst_scale, const float* src_scale, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_head_rows_kernel, dim3(n * dh), dim3(kBlock), 0, s, dst, src, idx, dh,
                     K, dst_scale, src_scale);
  return hipGetLastError();
}

hipError_t launch_gather_rows(int8_t* dst, const int8_t* src, const int* idx, int n, int K,
                              float* dst_scale, const float* src_scale, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_rows_kernel, dim3(n), dim3(kBlock), 0, s, dst, src, idx, K, dst_scale,
                     src_scale);
  return hipGetLastError();
}

hipError_t launch_gather_head_cols(int8_t* dst, int dst_ld, const int8_t* src, int src_ld,
                                   const int* idx, int n, int dh, int rows, hipStream_t s) {
  if (rows == 0 || dst_ld == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_head_cols_kernel, dim3(rows), dim3(kBlock), 0, s, dst, dst_ld, src,
                     src_ld, idx, n, dh);
  return hipGetLastError();
}

hipError_t launch_gather_cols(int8_t* dst, int dst_ld, const int8_t* src, int src_ld,
                              const int* idx, int n, int rows, hipStream_t s) {
  if (rows == 0 || dst_ld == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_cols_kernel, dim3(rows), dim3(kBlock), 0, s, dst, dst_ld, src, src_ld,
                     idx, n);
  return hipGetLastError();
}

hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(copy_kernel, dim3(grid_for(n)), dim3(kBlock), 0, s,
                     reinterpret_cast<int4*>(dst), reinterpret_cast<const int4*>(src), n);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(n)), dim3(kBlock), 0, s,
                     reinterpret_cast<uint32_t*>(dst), n);
  return hipGetLastError();
}

}  // namespace tasp

// Greedy dependency-closed mask construction on the GPU (paper, Sec. "Dependency-Closed Masks and
// Cache-Consistent Routing"; candidate costs from Eqs. flop-attn and flop-mlp).
//
// Candidates, in index order, are every layer's query heads followed by its SwiGLU channel groups.
//   1. keys: score / active FLOPs in float64 (a head carries its own cost plus 1/r of its KV
//      group's), negated so that an ascending sort gives descending keys; signed zeros are
//      folded to one zero, and a non-finite score raises the status word;
//   2. a stable device radix sort (rocPRIM) of (key, index): equal keys keep ascending index;
//   3. one workgroup scans the sorted order. The order is staged through LDS in chunks; one
//      thread walks it, accepting a candidate when its marginal cost (plus its KV group's, if
//      the group is not open yet) fits the remaining budget, and recording the acceptance in LDS
//      bytes; the workgroup then writes q_keep, kv_keep and the per-channel ffn_keep.
// The scan is sequential by nature (each decision depends on the budget left by all earlier
// ones); it touches a few bytes per candidate and runs once per mask.
#include <rocprim/device/device_radix_sort.hpp>

#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

constexpr int kScanChunk = 4096;       // sorted indices staged per round

__global__ __launch_bounds__(kBlock) void mask_keys_kernel(MaskArgs a, double* keys, int* idx) {
  const int i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= a.n_cand) return;
  const int per = a.Hq + a.nG;
  const int l = i / per, u = i % per;
  const bool head = u < a.Hq;
  const float s = head ? a.head_scores[size_t(l) * a.Hq + u] : a.chan_scores[size_t(l) * a.nG + (u - a.Hq)];
  if (!isfinite(s)) atomicOr(a.status, 1u);
  const double c = head ? a.head_rank_cost : double(a.chan_cost);
  double k = double(s) / c;
  if (k == 0.0) k = 0.0;
  keys[i] = -k;
  idx[i] = i;
}

__global__ __launch_bounds__(kBlock) void mask_scan_kernel(MaskArgs a, const int* order) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  int* chunk = reinterpret_cast<int*>(lds);                          // kScanChunk indices
  unsigned char* q_acc = lds + kScanChunk * sizeof(int);             // [L][Hq]
  unsigned char* kv_acc = q_acc + size_t(a.L) * a.Hq;                // [L][Hkv]
  unsigned char* g_acc = kv_acc + size_t(a.L) * a.Hkv;               // [L][nG]
  const int tid = threadIdx.x;
  const int nq = a.L * a.Hq, nkv = a.L * a.Hkv, ng = a.L * a.nG;
  for (int i = tid; i < nq + nkv + ng; i += kBlock) q_acc[i] = 0;
  __syncthreads();
  const int per = a.Hq + a.nG, r = a.Hq / a.Hkv;
  unsigned long long spent = 0;
  for (int c0 = 0; c0 < a.n_cand; c0 += kScanChunk) {
    const int n = min(kScanChunk, a.n_cand - c0);
    for (int i = tid; i < n; i += kBlock) chunk[i] = order[c0 + i];
    __syncthreads();
    if (tid == 0) {
      for (int k = 0; k < n; ++k) {
        const int i = chunk[k];
        const int l = i / per, u = i % per;
        if (u < a.Hq) {
          const int g = l * a.Hkv + u / r;
          const unsigned long long cost = a.head_cost + (kv_acc[g] ? 0ull : a.group_cost);
          if (spent + cost > a.budget) continue;
          spent += cost;
          q_acc[l * a.Hq + u] = 1;
          kv_acc[g] = 1;
        } else {
          if (spent + a.chan_cost > a.budget) continue;
          spent += a.chan_cost;
          g_acc[l * a.nG + (u - a.Hq)] = 1;
        }
      }
    }
    __syncthreads();
  }
  for (int i = tid; i < nq; i += kBlock) a.q_keep[i] = q_acc[i];
  for (int i = tid; i < nkv; i += kBlock) a.kv_keep[i] = kv_acc[i];
  const long nf = long(a.L) * a.nG * a.granule;
  for (long i = tid; i < nf; i += kBlock) {
    const long l = i / (long(a.nG) * a.granule), ch = i % (long(a.nG) * a.granule);
    a.ffn_keep[i] = g_acc[l * a.nG + ch / a.granule];
  }
  if (tid == 0) *a.spent = spent;
}

}  // namespace

size_t mask_scan_lds_bytes(int L, int Hq, int Hkv, int nG) {
  return kScanChunk * sizeof(int) + size_t(L) * (Hq + Hkv + nG);
}

hipError_t mask_sort_temp_bytes(int n, size_t* bytes) {
  return rocprim::radix_sort_pairs(nullptr, *bytes, static_cast<double*>(nullptr),
                                   static_cast<double*>(nullptr), static_cast<int*>(nullptr),
                                   static_cast<int*>(nullptr), size_t(n), 0, 64);
}

hipError_t launch_build_mask(const MaskArgs& a, void* temp, size_t temp_bytes, double* keys_in,
                             double* keys_out, int* idx_in, int* idx_out, hipStream_t s) {
  hipLaunchKernelGGL(mask_keys_kernel, dim3((a.n_cand + kBlock - 1) / kBlock), dim3(kBlock), 0, s,
                     a, keys_in, idx_in);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  size_t tb = temp_bytes;
  e = rocprim::radix_sort_pairs(temp, tb, keys_in, keys_out, idx_in, idx_out, size_t(a.n_cand), 0,
                                64, s);
  if (e != hipSuccess) return e;
  const size_t lds = mask_scan_lds_bytes(a.L, a.Hq, a.Hkv, a.nG);
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(&mask_scan_kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, int(lds));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mask_scan_kernel, dim3(1), dim3(kBlock), lds, s, a, idx_out);
  return hipGetLastError();
}

}  // namespace tasp

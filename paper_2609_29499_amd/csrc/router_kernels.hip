// Router inference (paper, Sec. "Dependency-Closed Masks and Cache-Consistent Routing"; appendix
// paragraph "Router feature specification"): per prompt, a feature vector of hashed character
// trigrams (projected by a frozen random map), length, proxy-LM log-probability, character-class
// counts and five task descriptors; a three-layer MLP over it; temperature-scaled softmax; the
// dense plan when the top probability is below tau.
//
//   1. router_features_kernel, one workgroup of 1024 threads per prompt. The prompt is staged
//      through LDS in chunks with a small halo on both sides (bytes outside the prompt read as
//      zero, which no pattern byte equals; all byte loads of a chunk are in flight together).
//      Every position is examined by one thread: its case-folded trigram's
//      32-bit FNV-1a hash goes into an LDS histogram by an LDS atomic increment (integer, so the
//      histogram does not depend on the order of the increments), its byte is classified, and
//      the descriptor patterns that can start there are matched. Counts and descriptor bits are
//      combined by LDS atomics; the workgroup writes the term frequencies [n_bins] and the 11
//      scalar features;
//   2. router_dense_kernel, launched three times (projection, hidden layer 1, hidden layer 2):
//      one wave per output row, lanes strided over the row, up to 8 prompts per workgroup
//      sharing each weight load; bias and ReLU in the epilogue;
//   3. router_head_kernel, one workgroup per prompt: the task logits, softmax of logits /
//      temperature (shifted by the maximum), the top probability (lowest task on ties) and the
//      decision.
// Everything is float32 except the text scan, which is integer and exact.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

constexpr int kFeatBlock = 1024;      // threads of the features kernel (one workgroup per prompt)
constexpr int kChunk = 8192;          // prompt bytes staged per round
constexpr int kHalo = 16;             // bytes kept on either side of a chunk (patterns need <= 9)
constexpr int kStaged = kChunk + 2 * kHalo;
constexpr int kStage = (kStaged + kFeatBlock - 1) / kFeatBlock;   // byte loads per thread
constexpr int kDenseRows = kBlock / kWave;   // output rows per workgroup
constexpr int kDensePrompts = 8;             // prompts per workgroup

enum : unsigned { kNumbered = 1u, kFence = 2u, kTranslate = 4u, kOptA = 8u, kOptB = 16u,
                  kRetrieval = 32u };

__device__ __forceinline__ unsigned fold(unsigned c) { return (c - 65u < 26u) ? c + 32u : c; }
__device__ __forceinline__ bool is_digit(unsigned c) { return c - 48u < 10u; }
__device__ __forceinline__ bool is_letter(unsigned c) { return (c | 32u) - 97u < 26u; }
__device__ __forceinline__ bool is_alnum(unsigned c) { return is_digit(c) || is_letter(c); }
__device__ __forceinline__ bool is_operator(unsigned c) {
  return c == '+' || c == '-' || c == '*' || c == '/' || c == '=' || c == '<' || c == '>' ||
         c == '%' || c == '^';
}
__device__ __forceinline__ bool is_code_punct(unsigned c) {
  return c == '{' || c == '}' || c == '[' || c == ']' || c == '(' || c == ')' || c == ';' ||
         c == '_' || c == '#' || c == '`' || c == '\\' || c == '|' || c == '&';
}

// FNV-1a (32-bit) of three bytes
__device__ __forceinline__ uint32_t fnv1a3(unsigned b0, unsigned b1, unsigned b2) {
  uint32_t h = 2166136261u;
  h = (h ^ b0) * 16777619u;
  h = (h ^ b1) * 16777619u;
  h = (h ^ b2) * 16777619u;
  return h;
}

// t points at the position's byte inside the staged chunk; t[-1] .. t[kHalo - 1] are readable
template <int N>
__device__ __forceinline__ bool folded_is(const uint8_t* t, const char (&w)[N]) {
#pragma unroll
  for (int i = 0; i < N - 1; ++i)
    if (fold(t[i]) != unsigned(w[i])) return false;
  return true;
}

__device__ __forceinline__ unsigned patterns_at(const uint8_t* t, bool line_start, bool word_start) {
  unsigned f = 0;
  if (line_start) {
    int k = 0;
    while (k < 3 && is_digit(t[k])) ++k;
    if (k > 0 && (t[k] == '.' || t[k] == ')') && t[k + 1] == ' ') f |= kNumbered;
    unsigned lab = 0xffu;
    if (t[0] == '(' && t[1] - 65u < 4u && t[2] == ')' && t[3] == ' ') lab = t[1] - 65u;
    else if (t[0] - 65u < 4u && (t[1] == '.' || t[1] == ')') && t[2] == ' ') lab = t[0] - 65u;
    if (lab == 0) f |= kOptA;
    if (lab == 1) f |= kOptB;
  }
  if (t[0] == '`' && t[1] == '`' && t[2] == '`') f |= kFence;
  if (folded_is(t, "translat")) f |= kTranslate;
  if (word_start) {
    if ((folded_is(t, "who") && !is_letter(t[3])) || (folded_is(t, "when") && !is_letter(t[4])) ||
        (folded_is(t, "where") && !is_letter(t[5])) || (folded_is(t, "which") && !is_letter(t[5])))
      f |= kRetrieval;
  }
  return f;
}

__global__ __launch_bounds__(kFeatBlock) void router_features_kernel(RouterFeatArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint32_t hist[];     // [n_bins]
  __shared__ uint8_t tb[kStaged];
  __shared__ int cnt[4];
  __shared__ unsigned flags;
  const int b = blockIdx.x, tid = threadIdx.x;
  long start = 0, end = a.n_text;
  if (a.offsets) {
    start = min(max(long(a.offsets[b]), 0L), long(a.n_text));
    end = min(max(long(a.offsets[b + 1]), start), long(a.n_text));
  }
  const int n = int(end - start);
  // this prompt's bytes; loads at an offset past them return zero without touching memory
  const __amdgpu_buffer_rsrc_t rt = make_rsrc(a.text + start, uint32_t(n));
  for (int i = tid; i < a.n_bins; i += kFeatBlock) hist[i] = 0u;
  if (tid < 4) cnt[tid] = 0;
  if (tid == 0) flags = 0u;
  __syncthreads();
  int cd = 0, co = 0, cc = 0, cq = 0;
  unsigned fl = 0;
  const uint32_t nb = uint32_t(a.n_bins);
  for (int c0 = 0; c0 < n; c0 += kChunk) {
    uint8_t v[kStage];
#pragma unroll
    for (int u = 0; u < kStage; ++u) {
      const int i = u * kFeatBlock + tid;
      const long q = long(c0) - kHalo + i;
      v[u] = __builtin_amdgcn_raw_buffer_load_b8(
          rt, (i < kStaged && q >= 0 && q < n) ? int(q) : int(kOOB), 0, 0);
    }
    __syncthreads();                                   // the previous chunk is consumed
#pragma unroll
    for (int u = 0; u < kStage; ++u) {
      const int i = u * kFeatBlock + tid;
      if (i < kStaged) tb[i] = v[u];
    }
    __syncthreads();
    const int lim = min(kChunk, n - c0);
    for (int i = tid; i < lim; i += kFeatBlock) {
      const int p = c0 + i;
      const uint8_t* t = tb + kHalo + i;
      const unsigned c = t[0];
      if (p + 3 <= n) atomicAdd(&hist[fnv1a3(fold(t[0]), fold(t[1]), fold(t[2])) % nb], 1u);
      cd += is_digit(c);
      co += is_operator(c);
      cc += is_code_punct(c);
      cq += (c == '?');
      const unsigned prev = t[-1];
      fl |= patterns_at(t, p == 0 || prev == '\n', p == 0 || !is_alnum(prev));
    }
  }
  atomicAdd(&cnt[0], cd);
  atomicAdd(&cnt[1], co);
  atomicAdd(&cnt[2], cc);
  atomicAdd(&cnt[3], cq);
  atomicOr(&flags, fl);
  __syncthreads();
  const float inv_n = float(max(1, n - 2));
  float* tf = a.tf + size_t(b) * a.n_bins;
  for (int i = tid; i < a.n_bins; i += kFeatBlock) tf[i] = float(hist[i]) / inv_n;
  if (tid == 0) {
    float* f = a.feats + size_t(b) * a.ld_feats + a.proj_dim;
    const unsigned g = flags;
    f[0] = log1pf(float(n));
    f[1] = a.logprob[b];
    f[2] = log1pf(float(cnt[0]));
    f[3] = log1pf(float(cnt[1]));
    f[4] = log1pf(float(cnt[2]));
    f[5] = log1pf(float(cnt[3]));
    f[6] = (g & kNumbered) ? 1.0f : 0.0f;
    f[7] = (g & kFence) ? 1.0f : 0.0f;
    f[8] = (g & kTranslate) ? 1.0f : 0.0f;
    f[9] = ((g & kOptA) && (g & kOptB)) ? 1.0f : 0.0f;
    f[10] = (g & kRetrieval) ? 1.0f : 0.0f;
  }
}

__global__ __launch_bounds__(kBlock) void router_dense_kernel(RouterDenseArgs a) {
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * kDenseRows + (threadIdx.x >> 6);
  const int b0 = blockIdx.y * kDensePrompts;
  if (j >= a.N) return;                               // whole waves leave together
  const int nb = min(kDensePrompts, a.B - b0);
  const float* w = a.w + size_t(j) * a.K;
  float acc[kDensePrompts];
#pragma unroll
  for (int u = 0; u < kDensePrompts; ++u) acc[u] = 0.0f;
  for (int k = lane; k < a.K; k += kWave) {
    const float wk = w[k];
#pragma unroll
    for (int u = 0; u < kDensePrompts; ++u)
      if (u < nb) acc[u] = fmaf(wk, a.x[size_t(b0 + u) * a.ldx + k], acc[u]);
  }
  const float bias = a.bias ? a.bias[j] : 0.0f;
#pragma unroll
  for (int u = 0; u < kDensePrompts; ++u) {
    const float v = wave_sum(acc[u]) + bias;
    if (lane == 0 && u < nb) a.y[size_t(b0 + u) * a.ldy + j] = a.relu ? fmaxf(v, 0.0f) : v;
  }
}

__global__ __launch_bounds__(kBlock) void router_head_kernel(RouterHeadArgs a) {
  __shared__ float z[kMaxRouterTasks];
  const int b = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* h = a.h + size_t(b) * a.K;
  for (int t = wave; t < a.n_tasks; t += kBlock / kWave) {
    const float* w = a.w + size_t(t) * a.K;
    float acc = 0.0f;
    for (int k = lane; k < a.K; k += kWave) acc = fmaf(w[k], h[k], acc);
    acc = wave_sum(acc);
    if (lane == 0) z[t] = acc + a.bias[t];
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  float u[kMaxRouterTasks];
  float m = -INFINITY;
  for (int t = 0; t < a.n_tasks; ++t) {
    u[t] = z[t] / a.temperature;
    m = fmaxf(m, u[t]);
  }
  float s = 0.0f;
  for (int t = 0; t < a.n_tasks; ++t) {
    u[t] = expf(u[t] - m);
    s += u[t];
  }
  float best = -1.0f;
  int task = 0;
  float* p = a.probs + size_t(b) * a.n_tasks;
  for (int t = 0; t < a.n_tasks; ++t) {
    const float v = u[t] / s;
    p[t] = v;
    if (v > best) {
      best = v;
      task = t;
    }
  }
  a.choice[b] = (best >= a.tau) ? task : -1;
}

}  // namespace

size_t router_features_lds_bytes(int n_bins) { return size_t(n_bins) * sizeof(uint32_t); }

hipError_t launch_router_features(const RouterFeatArgs& a, int n_prompts, hipStream_t s) {
  if (n_prompts < 1) return hipSuccess;
  const size_t lds = router_features_lds_bytes(a.n_bins);
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&router_features_kernel),
      hipFuncAttributeMaxDynamicSharedMemorySize, int(router_features_lds_bytes(kMaxRouterBins)));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(router_features_kernel, dim3(n_prompts), dim3(kFeatBlock), lds, s, a);
  return hipGetLastError();
}

hipError_t launch_router_dense(const RouterDenseArgs& a, hipStream_t s) {
  if (a.B < 1 || a.N < 1) return hipSuccess;
  const dim3 grid((a.N + kDenseRows - 1) / kDenseRows, (a.B + kDensePrompts - 1) / kDensePrompts);
  hipLaunchKernelGGL(router_dense_kernel, grid, dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_router_head(const RouterHeadArgs& a, int n_prompts, hipStream_t s) {
  if (n_prompts < 1) return hipSuccess;
  if (a.n_tasks < 1 || a.n_tasks > kMaxRouterTasks) return hipErrorInvalidValue;
  hipLaunchKernelGGL(router_head_kernel, dim3(n_prompts), dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

}  // namespace tasp

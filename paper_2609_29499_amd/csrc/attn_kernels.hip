// Decode attention over the retained KV groups only (grouped-query attention, one new token).
//
// Grid (n_split, m_kv, B): workgroup (s, j, b) serves retained group slot j of sequence b over
// cache rows [s*chunk, min((s+1)*chunk, pos+1)) for all of that group's retained query heads
// (1..8), so each K/V row is read from HBM once for every head that uses it. The workgroup
//   1. rotates its heads' raw q (RoPE at pos, table from the plan) into LDS, pre-scaled by
//      log2(e)/sqrt(d_h) so the softmax works in base 2;
//   2. if its range holds row pos: rotates the new k, rounds k and v to BF16, appends them to the
//      cache and keeps the rounded values in LDS (the same values later steps will read);
//   3. scores: d_h/8 lanes share one cache row (16-byte loads), dot products reduced with
//      shuffles inside the lane group, scores kept in LDS;
//   4. exact softmax of its range (max, exp2, sum), then P V with the same row mapping;
//   5. writes (max, sum, unnormalised output) per head; the last workgroup of the group (atomic
//      counter, reset by that workgroup) merges the ranges by log-sum-exp and writes o.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

constexpr int kMaxHeads = 8;
constexpr int kMaxChunk = 512;

template <int DH>
__global__ __launch_bounds__(kBlock) void attn_decode_kernel(AttnArgs a) {
  constexpr int LPR = DH / 8;          // lanes per cache row
  constexpr int RPW = kWave / LPR;     // rows per wave per step
  constexpr int RPB = RPW * 4;         // rows per workgroup per step
  constexpr int HALF = DH / 2;
  __shared__ float q_s[kMaxHeads][DH];
  __shared__ float sc[kMaxHeads][kMaxChunk];
  __shared__ float red[4][kMaxHeads][DH];
  __shared__ float knew[DH], vnew[DH];
  __shared__ float m_s[kMaxHeads], l_s[kMaxHeads];
  __shared__ int last_flag;

  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = a.kv_idx[j];
  const int h0 = a.slot_start[j];
  const int nh = a.slot_start[j + 1] - h0;
  const int t0 = s * a.chunk;
  const int t1 = min(t0 + a.chunk, a.pos + 1);
  const int n = t1 - t0;
  const float* qkv = a.qkv + size_t(b) * a.ld_qkv;
  const float* cs = a.rope_cos + size_t(a.pos) * HALF;
  const float* sn = a.rope_sin + size_t(a.pos) * HALF;
  const float qscale = kLog2e * rsqrtf(float(DH));
  const size_t row_base = (size_t(b) * a.Hkv + g) * a.S;
  uint16_t* kc = a.kc + row_base * DH;
  uint16_t* vc = a.vc + row_base * DH;
  const bool has_new = (t1 == a.pos + 1);

  // 1-2. rotary embedding of the heads' queries and, in the last range, the new key
  for (int i = tid; i < nh * DH; i += kBlock) {
    const int h = i / DH, e = i % DH;
    const float* qh = qkv + size_t(h0 + h) * DH;
    const int p = e % HALF;
    const float v = (e < HALF) ? qh[e] * cs[p] - qh[e + HALF] * sn[p]
                               : qh[e] * cs[p] + qh[e - HALF] * sn[p];
    q_s[h][e] = v * qscale;
  }
  if (has_new && tid < DH) {
    const float* kh = qkv + size_t(a.m_q + j) * DH;
    const float* vh = qkv + size_t(a.m_q + a.m_kv + j) * DH;
    const int e = tid, p = e % HALF;
    const float kr = (e < HALF) ? kh[e] * cs[p] - kh[e + HALF] * sn[p]
                                : kh[e] * cs[p] + kh[e - HALF] * sn[p];
    const uint16_t kb = f32_to_bf16(kr), vb = f32_to_bf16(vh[e]);
    kc[size_t(a.pos) * DH + e] = kb;
    vc[size_t(a.pos) * DH + e] = vb;
    knew[e] = bf16_to_f32(kb);
    vnew[e] = bf16_to_f32(vb);
  }
  __syncthreads();

  const int lr = lane % LPR;           // dims [8 lr, 8 lr + 8)
  const int rb = wave * RPW + lane / LPR;
  float qr[kMaxHeads][8];
#pragma unroll
  for (int h = 0; h < kMaxHeads; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) qr[h][i] = (h < nh) ? q_s[h][lr * 8 + i] : 0.0f;

  // 3. scores
  for (int t = t0 + rb; t - rb < t1; t += RPB) {
    float kf[8];
    const bool valid = t < t1;
    if (valid && t == a.pos) {
#pragma unroll
      for (int i = 0; i < 8; ++i) kf[i] = knew[lr * 8 + i];
    } else if (valid) {
      const uint4 w = *reinterpret_cast<const uint4*>(kc + size_t(t) * DH + lr * 8);
      kf[0] = bf16_lo(w.x); kf[1] = bf16_hi(w.x); kf[2] = bf16_lo(w.y); kf[3] = bf16_hi(w.y);
      kf[4] = bf16_lo(w.z); kf[5] = bf16_hi(w.z); kf[6] = bf16_lo(w.w); kf[7] = bf16_hi(w.w);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) kf[i] = 0.0f;
    }
#pragma unroll
    for (int h = 0; h < kMaxHeads; ++h) {
      if (h >= nh) break;
      float d = 0.0f;
#pragma unroll
      for (int i = 0; i < 8; ++i) d = fmaf(qr[h][i], kf[i], d);
#pragma unroll
      for (int m = LPR / 2; m >= 1; m >>= 1) d += __shfl_xor(d, m, kWave);
      if (valid && lr == 0) sc[h][t - t0] = d;
    }
  }
  __syncthreads();

  // 4. softmax of this range, one wave per head
  for (int h = wave; h < nh; h += 4) {
    float mx = -INFINITY;
    for (int t = lane; t < n; t += kWave) mx = fmaxf(mx, sc[h][t]);
    mx = wave_max(mx);
    float sum = 0.0f;
    for (int t = lane; t < n; t += kWave) {
      const float p = exp2f(sc[h][t] - mx);
      sc[h][t] = p;
      sum += p;
    }
    sum = wave_sum(sum);
    if (lane == 0) {
      m_s[h] = mx;
      l_s[h] = sum;
    }
  }
  __syncthreads();

  float acc[kMaxHeads][8];
#pragma unroll
  for (int h = 0; h < kMaxHeads; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;
  for (int t = t0 + rb; t < t1; t += RPB) {
    float vf[8];
    if (t == a.pos) {
#pragma unroll
      for (int i = 0; i < 8; ++i) vf[i] = vnew[lr * 8 + i];
    } else {
      const uint4 w = *reinterpret_cast<const uint4*>(vc + size_t(t) * DH + lr * 8);
      vf[0] = bf16_lo(w.x); vf[1] = bf16_hi(w.x); vf[2] = bf16_lo(w.y); vf[3] = bf16_hi(w.y);
      vf[4] = bf16_lo(w.z); vf[5] = bf16_hi(w.z); vf[6] = bf16_lo(w.w); vf[7] = bf16_hi(w.w);
    }
#pragma unroll
    for (int h = 0; h < kMaxHeads; ++h) {
      if (h >= nh) break;
      const float p = sc[h][t - t0];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[h][i] = fmaf(p, vf[i], acc[h][i]);
    }
  }
  // reduce over the rows of a wave (lanes that share lr), then over the 4 waves in LDS
#pragma unroll
  for (int h = 0; h < kMaxHeads; ++h) {
    if (h >= nh) break;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float v = acc[h][i];
#pragma unroll
      for (int m = LPR; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
      acc[h][i] = v;
    }
  }
  if (lane < LPR) {
#pragma unroll
    for (int h = 0; h < kMaxHeads; ++h) {
      if (h >= nh) break;
#pragma unroll
      for (int i = 0; i < 8; ++i) red[wave][h][lr * 8 + i] = acc[h][i];
    }
  }
  __syncthreads();

  float* ob = a.o + size_t(b) * a.ld_o;
  if (a.n_split == 1) {
    for (int i = tid; i < nh * DH; i += kBlock) {
      const int h = i / DH, e = i % DH;
      const float v = red[0][h][e] + red[1][h][e] + red[2][h][e] + red[3][h][e];
      ob[size_t(h0 + h) * DH + e] = v / l_s[h];
    }
    return;
  }

  // 5. partial results, then the last workgroup of this group merges them
  constexpr int PS = DH + 2;
  float* part = a.part + (size_t(b) * a.m_kv + j) * size_t(a.n_split) * kMaxHeads * PS;
  for (int i = tid; i < nh * DH; i += kBlock) {
    const int h = i / DH, e = i % DH;
    part[(size_t(s) * kMaxHeads + h) * PS + 2 + e] =
        red[0][h][e] + red[1][h][e] + red[2][h][e] + red[3][h][e];
  }
  if (tid < nh) {
    part[(size_t(s) * kMaxHeads + tid) * PS + 0] = m_s[tid];
    part[(size_t(s) * kMaxHeads + tid) * PS + 1] = l_s[tid];
  }
  __threadfence();
  __syncthreads();
  int* cnt = a.counters + size_t(b) * a.Hkv + j;
  if (tid == 0) last_flag = (atomicAdd(cnt, 1) == a.n_split - 1);
  __syncthreads();
  if (!last_flag) return;
  __threadfence();
  for (int i = tid; i < nh * DH; i += kBlock) {
    const int h = i / DH, e = i % DH;
    float M = -INFINITY;
    for (int k = 0; k < a.n_split; ++k) M = fmaxf(M, ld_coherent(&part[(size_t(k) * kMaxHeads + h) * PS]));
    float L = 0.0f, A = 0.0f;
    for (int k = 0; k < a.n_split; ++k) {
      const float* pk = &part[(size_t(k) * kMaxHeads + h) * PS];
      const float w = exp2f(ld_coherent(pk) - M);
      L = fmaf(ld_coherent(pk + 1), w, L);
      A = fmaf(ld_coherent(pk + 2 + e), w, A);
    }
    ob[size_t(h0 + h) * DH + e] = A / L;
  }
  if (tid == 0) *cnt = 0;
}

}  // namespace

hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t s) {
  if (a.m_kv == 0 || a.B == 0) return hipSuccess;
  const dim3 grid(a.n_split, a.m_kv, a.B);
  if (a.dh == 128)
    hipLaunchKernelGGL(attn_decode_kernel<128>, grid, dim3(kBlock), 0, s, a);
  else if (a.dh == 64)
    hipLaunchKernelGGL(attn_decode_kernel<64>, grid, dim3(kBlock), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

int attn_max_chunk() { return kMaxChunk; }

}  // namespace tasp

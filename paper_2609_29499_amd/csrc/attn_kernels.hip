// Decode attention over the retained KV groups only (grouped-query attention, one new token).
//
// Grid (n_split, m_kv, B): workgroup (s, j, b) serves retained group slot j of sequence b over
// cache rows [s*chunk, (s+1)*chunk), the last split over [s*chunk, pos+1) (it may be longer or
// shorter than chunk), for all of that group's retained query heads
// (1..8), so each K/V row is read from HBM once for every head that uses it. The slot -> group
// and slot -> head-range tables of the layer travel inside the kernel arguments, so the cache
// loads do not wait for an index load. The workgroup
//   1. issues the K and V loads of its first 64-row sub-block, then rotates its heads' raw q
//      (RoPE at pos, table from the plan) into LDS, pre-scaled by log2(e)/sqrt(d_h) so the
//      softmax works in base 2; if its range holds row pos it also rotates the new k, rounds k
//      and v to BF16, appends them to the cache and keeps the rounded values in LDS (the values
//      every later step reads);
//   2. per sub-block (the next one's loads already in flight): d_h/8 lanes share a cache row (16-byte loads; rows outside the range use an
//      out-of-range buffer offset, so no branch sits around a load); the per-row dot products are
//      reduced across the row's lanes with DPP, and an online softmax (running max and sum per
//      head, rescaled accumulators) folds the sub-block into P V. The head count is a template
//      parameter, so every per-head loop is unrolled and independent chains interleave;
//   3. when the range is split, writes (max, sum, unnormalised output) per head with
//      device-coherent stores, waits for them to complete and counts itself done on the
//      (group slot, sequence) counter; the workgroup that brings the count to n_split reads every
//      split's record back with device-coherent loads, merges them by log-sum-exp, writes o and
//      resets the counter for the next launch. Nothing waits on another workgroup, and no L2
//      write-back is needed (an earlier version fenced every workgroup, which serialised on the
//      write-backs; a second merge kernel cost a launch and a round trip through memory).
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

constexpr int kMaxHeads = 8;
constexpr int kSub = 64;               // rows per sub-block (two in flight per workgroup)
constexpr int kMinChunk = 2 * kSub;    // rows per split are a multiple of this
constexpr int kMaxSplit = 256;
constexpr int kMergeBatch = 16;        // split records in flight per thread while merging
constexpr int kNumCu = 256;

__device__ __forceinline__ void unpack_bf16x8(const int4& w, float (&f)[8]) {
  f[0] = bf16_lo(uint32_t(w.x)); f[1] = bf16_hi(uint32_t(w.x));
  f[2] = bf16_lo(uint32_t(w.y)); f[3] = bf16_hi(uint32_t(w.y));
  f[4] = bf16_lo(uint32_t(w.z)); f[5] = bf16_hi(uint32_t(w.z));
  f[6] = bf16_lo(uint32_t(w.w)); f[7] = bf16_hi(uint32_t(w.w));
}

__device__ __forceinline__ float4 rope4(const float4& a, const float4& b, const float4& c,
                                        const float4& s, bool first_half) {
  // first half: a cos - b sin (b = partner); second half: a cos + b sin
  const float sg = first_half ? -1.0f : 1.0f;
  return make_float4(fmaf(sg * b.x, s.x, a.x * c.x), fmaf(sg * b.y, s.y, a.y * c.y),
                     fmaf(sg * b.z, s.z, a.z * c.z), fmaf(sg * b.w, s.w, a.w * c.w));
}

template <int DH>
struct AttnSmem {
  float q_s[kMaxHeads][DH];
  float sc[kMaxHeads][kSub];
  float red[4][kMaxHeads][DH];
  float knew[DH];
  float vnew[DH];
  float m_s[kMaxHeads], l_s[kMaxHeads], al_s[kMaxHeads];
  int last;                            // this workgroup merges the splits
};

template <int LPR>
__device__ __forceinline__ float row_group_sum(float v) {
  return LPR == 16 ? row16_sum(v) : row8_sum(v);
}

// One attention output element: float32 row b of o, or the hi/lo BF16 operand of the batched
// projections (rows 2b and 2b + 1).
__device__ __forceinline__ void store_o(const AttnArgs& a, int b, int col, float v) {
  if (a.o_hl) {
    const uint16_t hi = f32_to_bf16(v);
    a.o_hl[size_t(2 * b) * a.ld_ohl + col] = hi;
    a.o_hl[size_t(2 * b + 1) * a.ld_ohl + col] = f32_to_bf16(v - bf16_to_f32(hi));
  } else {
    a.o[size_t(b) * a.ld_o + col] = v;
  }
}

template <int DH, int NH>
__device__ __forceinline__ void attn_body(const AttnArgs& a, AttnSmem<DH>& sm, int s, int j,
                                          int b) {
  constexpr int LPR = DH / 8;          // lanes per cache row
  constexpr int RPW = kWave / LPR;     // rows per wave per step
  constexpr int RPB = RPW * 4;         // rows per workgroup per step
  constexpr int U = kSub / RPB;        // steps per sub-block
  constexpr int HALF = DH / 2;
  constexpr int Q4 = DH / 4;           // float4 per head row
  constexpr int PS = DH + 4;           // partial record: max, sum, pad, DH accumulators
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = a.kv_idx[j];
  const int h0 = a.slot_start[j];
  const int t0 = s * a.chunk;
  const int t1 = (s == a.n_split - 1) ? a.pos + 1 : t0 + a.chunk;
  const float* qkv = a.qkv + size_t(b) * a.ld_qkv;
  const size_t row_base = (size_t(b) * a.Hkv + g) * a.S;
  uint16_t* kc = a.kc + row_base * DH;
  uint16_t* vc = a.vc + row_base * DH;
  const bool has_new = (t1 == a.pos + 1);
  // this group's cache rows 0..pos-1 (row pos is taken from LDS)
  const uint32_t group_bytes = uint32_t(a.pos) * DH * 2u;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kc, group_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vc, group_bytes);
  const int lr = lane % LPR;           // dims [8 lr, 8 lr + 8)
  const int rb = wave * RPW + lane / LPR;
  auto row_off = [&](int t) -> uint32_t {
    return (t < t1 && t < a.pos) ? uint32_t(t) * (DH * 2u) + uint32_t(lr) * 16u : kOOB;
  };

  // K and V of one sub-block: U rows per lane
  struct KV {
    int4 k[U], v[U];
  };
  auto issue = [&](int tb, KV& f) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      f.k[u] = buf_load16_stream(rk, row_off(tb + rb + u * RPB));
      f.v[u] = buf_load16_stream(rv, row_off(tb + rb + u * RPB));
    }
  };
  KV fa, fb;
  issue(t0, fa);

  // 1. RoPE of the queries (and of the new key): item (h, i4) rotates float4 i4 of the first half
  //    with its partner in the second half
  {
    const float4* cs4 = reinterpret_cast<const float4*>(a.rope_cos + size_t(a.pos) * HALF);
    const float4* sn4 = reinterpret_cast<const float4*>(a.rope_sin + size_t(a.pos) * HALF);
    const float qscale = kLog2e * rsqrtf(float(DH));
    constexpr int H4 = HALF / 4;
    const int nitems = (NH + (has_new ? 1 : 0)) * H4;
    if (tid < nitems) {
      const int h = tid / H4, i4 = tid % H4;
      const bool is_k = h == NH;
      const float* src = is_k ? qkv + size_t(a.m_q + j) * DH : qkv + size_t(h0 + h) * DH;
      const float4 x1 = reinterpret_cast<const float4*>(src)[i4];
      const float4 x2 = reinterpret_cast<const float4*>(src)[i4 + H4];
      const float4 c = cs4[i4], sn = sn4[i4];
      float4 y1 = rope4(x1, x2, c, sn, true), y2 = rope4(x2, x1, c, sn, false);
      if (!is_k) {
        y1.x *= qscale; y1.y *= qscale; y1.z *= qscale; y1.w *= qscale;
        y2.x *= qscale; y2.y *= qscale; y2.z *= qscale; y2.w *= qscale;
        reinterpret_cast<float4*>(sm.q_s[h])[i4] = y1;
        reinterpret_cast<float4*>(sm.q_s[h])[i4 + H4] = y2;
      } else {
        const float e1[4] = {y1.x, y1.y, y1.z, y1.w}, e2[4] = {y2.x, y2.y, y2.z, y2.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint16_t b1 = f32_to_bf16(e1[q]), b2 = f32_to_bf16(e2[q]);
          kc[size_t(a.pos) * DH + i4 * 4 + q] = b1;
          kc[size_t(a.pos) * DH + HALF + i4 * 4 + q] = b2;
          sm.knew[i4 * 4 + q] = bf16_to_f32(b1);
          sm.knew[HALF + i4 * 4 + q] = bf16_to_f32(b2);
        }
      }
    }
    if (has_new && tid >= 128 && tid < 128 + Q4) {
      const int i4 = tid - 128;
      const float4 v = reinterpret_cast<const float4*>(qkv + size_t(a.m_q + a.m_kv + j) * DH)[i4];
      const float e[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint16_t bv = f32_to_bf16(e[q]);
        vc[size_t(a.pos) * DH + i4 * 4 + q] = bv;
        sm.vnew[i4 * 4 + q] = bf16_to_f32(bv);
      }
    }
    if (tid < NH) {
      sm.m_s[tid] = -INFINITY;
      sm.l_s[tid] = 0.0f;
    }
  }
  __syncthreads();

  float qr[NH][8];
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) qr[h][i] = sm.q_s[h][lr * 8 + i];
  float acc[NH][8];
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[h][i] = 0.0f;

  // 2. sub-blocks with an online softmax; the next sub-block's K and V are in flight while the
  //    current one is scored and accumulated
  auto process = [&](const KV& f, int tb) {
    float d[U][NH];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = tb + rb + u * RPB;
      float kf[8];
      unpack_bf16x8(f.k[u], kf);
      if (has_new && t == a.pos) {
#pragma unroll
        for (int i = 0; i < 8; ++i) kf[i] = sm.knew[lr * 8 + i];
      }
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        float x = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) x = fmaf(qr[h][i], kf[i], x);
        d[u][h] = x;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int h = 0; h < NH; ++h) d[u][h] = row_group_sum<LPR>(d[u][h]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = tb + rb + u * RPB;
      if (lr == 0) {
#pragma unroll
        for (int h = 0; h < NH; ++h) sm.sc[h][t - tb] = (t < t1) ? d[u][h] : -INFINITY;
      }
    }
    __syncthreads();
    for (int h = wave; h < NH; h += 4) {
      const float v0 = sm.sc[h][lane];
      const float mo = sm.m_s[h];
      const float mn = fmaxf(mo, wave_max(v0));
      const float p0 = exp2f(v0 - mn);
      sm.sc[h][lane] = p0;
      const float sum = wave_sum(p0);
      if (lane == 0) {
        const float al = exp2f(mo - mn);
        sm.al_s[h] = al;
        sm.l_s[h] = sm.l_s[h] * al + sum;
        sm.m_s[h] = mn;
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < NH; ++h) {
      const float al = sm.al_s[h];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[h][i] *= al;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = tb + rb + u * RPB;
      float vf[8];
      unpack_bf16x8(f.v[u], vf);
      if (has_new && t == a.pos) {
#pragma unroll
        for (int i = 0; i < 8; ++i) vf[i] = sm.vnew[lr * 8 + i];
      }
#pragma unroll
      for (int h = 0; h < NH; ++h) {
        const float p = sm.sc[h][t - tb];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[h][i] = fmaf(p, vf[i], acc[h][i]);
      }
    }
    __syncthreads();
  };
  for (int tb = t0; tb < t1; tb += 2 * kSub) {
    issue(tb + kSub, fb);
    process(fa, tb);
    issue(tb + 2 * kSub, fa);
    if (tb + kSub < t1) process(fb, tb + kSub);
  }
  // reduce over the rows of a wave (lanes that share lr), then over the 4 waves in LDS
#pragma unroll
  for (int h = 0; h < NH; ++h)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      float v = acc[h][i];
#pragma unroll
      for (int m = LPR; m < kWave; m <<= 1) v += __shfl_xor(v, m, kWave);
      acc[h][i] = v;
    }
  if (lane < LPR) {
#pragma unroll
    for (int h = 0; h < NH; ++h)
#pragma unroll
      for (int i = 0; i < 8; ++i) sm.red[wave][h][lr * 8 + i] = acc[h][i];
  }
  __syncthreads();

  if (a.n_split == 1) {
    for (int i = tid; i < NH * DH; i += kBlock) {
      const int h = i / DH, e = i % DH;
      const float v = sm.red[0][h][e] + sm.red[1][h][e] + sm.red[2][h][e] + sm.red[3][h][e];
      store_o(a, b, (h0 + h) * DH + e, v / sm.l_s[h]);
    }
    return;
  }
  // 3. partial results: record per (split, head) = [max, sum, 0, 0, acc[DH]] (float4-aligned),
  //    written device-coherent; the last split of (j, b) to finish merges all of them
  const size_t rec0 = (size_t(b) * a.m_kv + j) * size_t(a.n_split) * kMaxHeads * PS;
  const __amdgpu_buffer_rsrc_t rp =
      make_rsrc(a.part + rec0, uint32_t(a.n_split) * kMaxHeads * PS * 4u);
  for (int i = tid; i < NH * Q4; i += kBlock) {
    const int h = i / Q4, e4 = i % Q4;
    float4 v;
    v.x = sm.red[0][h][4 * e4 + 0] + sm.red[1][h][4 * e4 + 0] + sm.red[2][h][4 * e4 + 0] + sm.red[3][h][4 * e4 + 0];
    v.y = sm.red[0][h][4 * e4 + 1] + sm.red[1][h][4 * e4 + 1] + sm.red[2][h][4 * e4 + 1] + sm.red[3][h][4 * e4 + 1];
    v.z = sm.red[0][h][4 * e4 + 2] + sm.red[1][h][4 * e4 + 2] + sm.red[2][h][4 * e4 + 2] + sm.red[3][h][4 * e4 + 2];
    v.w = sm.red[0][h][4 * e4 + 3] + sm.red[1][h][4 * e4 + 3] + sm.red[2][h][4 * e4 + 3] + sm.red[3][h][4 * e4 + 3];
    buf_store16_device(__builtin_bit_cast(int4, v), rp,
                       uint32_t(((s * kMaxHeads + h) * PS + 4) * 4 + e4 * 16));
  }
  if (tid < NH)
    buf_store8_device(__builtin_bit_cast(int2, make_float2(sm.m_s[tid], sm.l_s[tid])), rp,
                      uint32_t((s * kMaxHeads + tid) * PS * 4));
  __builtin_amdgcn_s_waitcnt(0);        // this thread's records have reached the coherence point
  __syncthreads();                      // ... and every thread's
  int* cnt = a.cnt + size_t(b) * a.m_kv + j;
  if (tid == 0) {
    const int done = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sm.last = (done == a.n_split - 1);
  }
  __syncthreads();
  if (!sm.last) return;
  if (tid == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // merge: thread (h, e4) combines 4 output dims of one head over all splits, kMergeBatch records
  // in flight at once, with a running log-sum-exp across batches
  if (tid >= NH * Q4) return;
  const int h = tid / Q4, e4 = tid % Q4;
  float M = -INFINITY, L = 0.0f;
  float4 A = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  for (int k0 = 0; k0 < a.n_split; k0 += kMergeBatch) {
    float2 ml[kMergeBatch];
    float4 av[kMergeBatch];
#pragma unroll
    for (int q = 0; q < kMergeBatch; ++q) {
      const uint32_t rec = uint32_t((min(k0 + q, a.n_split - 1) * kMaxHeads + h) * PS * 4);
      ml[q] = __builtin_bit_cast(float2, buf_load8_device(rp, rec));
      av[q] = __builtin_bit_cast(float4, buf_load16_device(rp, rec + 16u + uint32_t(e4) * 16u));
    }
    float bm = M;
#pragma unroll
    for (int q = 0; q < kMergeBatch; ++q) bm = fmaxf(bm, ml[q].x);
    const float rs = exp2f(M - bm);             // rescale what was merged so far
    L *= rs;
    A.x *= rs; A.y *= rs; A.z *= rs; A.w *= rs;
#pragma unroll
    for (int q = 0; q < kMergeBatch; ++q) {
      const float w = (k0 + q < a.n_split) ? exp2f(ml[q].x - bm) : 0.0f;
      L = fmaf(ml[q].y, w, L);
      A.x = fmaf(av[q].x, w, A.x); A.y = fmaf(av[q].y, w, A.y);
      A.z = fmaf(av[q].z, w, A.z); A.w = fmaf(av[q].w, w, A.w);
    }
    M = bm;
  }
  const float inv = 1.0f / L;
  const int col = (h0 + h) * DH + 4 * e4;
  if (a.o_hl) {
    store_o(a, b, col + 0, A.x * inv);
    store_o(a, b, col + 1, A.y * inv);
    store_o(a, b, col + 2, A.z * inv);
    store_o(a, b, col + 3, A.w * inv);
  } else {
    *reinterpret_cast<float4*>(a.o + size_t(b) * a.ld_o + col) =
        make_float4(A.x * inv, A.y * inv, A.z * inv, A.w * inv);
  }
}

// NHM bounds the retained heads of every group slot in the launch: the register budget is set by
// the largest head count compiled into the kernel, so layers whose groups keep few heads run with
// fewer registers and more resident workgroups.
template <int DH, int NHM>
__global__ __launch_bounds__(kBlock) void attn_decode_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) AttnSmem<DH> sm;
  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int nh = a.slot_start[j + 1] - a.slot_start[j];
  if (NHM == 1 || nh == 1) { attn_body<DH, 1>(a, sm, s, j, b); return; }
  if (NHM == 2 || nh == 2) { attn_body<DH, (NHM >= 2 ? 2 : 1)>(a, sm, s, j, b); return; }
  if (NHM == 4) {
    if (nh == 3) attn_body<DH, (NHM >= 3 ? 3 : 1)>(a, sm, s, j, b);
    else attn_body<DH, (NHM >= 4 ? 4 : 1)>(a, sm, s, j, b);
    return;
  }
  switch (nh) {
    case 3: attn_body<DH, 3>(a, sm, s, j, b); break;
    case 4: attn_body<DH, 4>(a, sm, s, j, b); break;
    case 5: attn_body<DH, 5>(a, sm, s, j, b); break;
    case 6: attn_body<DH, 6>(a, sm, s, j, b); break;
    case 7: attn_body<DH, 7>(a, sm, s, j, b); break;
    default: attn_body<DH, 8>(a, sm, s, j, b); break;
  }
}

}  // namespace

template <int DH>
hipError_t launch_partials(const AttnArgs& a, dim3 grid, int nhm, hipStream_t s) {
  if (nhm <= 1) hipLaunchKernelGGL((attn_decode_kernel<DH, 1>), grid, dim3(kBlock), 0, s, a);
  else if (nhm == 2) hipLaunchKernelGGL((attn_decode_kernel<DH, 2>), grid, dim3(kBlock), 0, s, a);
  else if (nhm <= 4) hipLaunchKernelGGL((attn_decode_kernel<DH, 4>), grid, dim3(kBlock), 0, s, a);
  else hipLaunchKernelGGL((attn_decode_kernel<DH, 8>), grid, dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

template <int DH, int NHM>
int resident_blocks() {
  static const int n = [] {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_decode_kernel<DH, NHM>, kBlock,
                                                     0) != hipSuccess || per_cu < 1)
      per_cu = 1;
    return per_cu * kNumCu;
  }();
  return n;
}

template <int DH>
int resident_for(int nhm) {
  if (nhm <= 1) return resident_blocks<DH, 1>();
  if (nhm == 2) return resident_blocks<DH, 2>();
  if (nhm <= 4) return resident_blocks<DH, 4>();
  return resident_blocks<DH, 8>();
}

hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t s) {
  if (a.m_kv == 0 || a.B == 0) return hipSuccess;
  if (a.chunk < kMinChunk || a.chunk % kMinChunk != 0 || (a.dh != 64 && a.dh != 128))
    return hipErrorInvalidValue;
  // every split holds at least one row, and the merge takes at most kMaxSplit records
  if (a.n_split < 1 || a.n_split > kMaxSplit || long(a.n_split - 1) * a.chunk > a.pos)
    return hipErrorInvalidValue;
  int nhm = 0;
  for (int j = 0; j < a.m_kv; ++j) nhm = std::max(nhm, a.slot_start[j + 1] - a.slot_start[j]);
  if (nhm < 1 || nhm > kMaxHeads) return hipErrorInvalidValue;
  if (a.n_split > 1 && (!a.part || !a.cnt)) return hipErrorInvalidValue;
  const dim3 grid(a.n_split, a.m_kv, a.B);
  return (a.dh == 128) ? launch_partials<128>(a, grid, nhm, s) : launch_partials<64>(a, grid, nhm, s);
}

int attn_min_chunk() { return kMinChunk; }
int attn_max_split() { return kMaxSplit; }
int attn_resident_blocks(int dh, int nhm) {
  return dh == 128 ? resident_for<128>(nhm) : resident_for<64>(nhm);
}

}  // namespace tasp

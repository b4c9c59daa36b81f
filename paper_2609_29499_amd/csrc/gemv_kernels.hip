// Decode-time GEMVs over compacted panels: y = s * (P x), float32 x and float32 accumulation,
// INT8 panels for the projections and the dense BF16 LM head, for one sequence. They stream the
// panel from HBM; at the 8B layer shape each launch is short enough that its fixed costs (launch,
// first-byte latency, the last wave's work) weigh as much as the stream.
//
// Work decomposition: rows are taken in groups (2 rows for QKV, O and down; 4 for the LM head;
// for gate/up one SwiGLU channel = its gate and up rows). A tile is one group x 1 KiB of each of
// its rows (the LM head: 2 KiB); a wave reads whole contiguous KiB, 16 bytes
// per lane. Several workgroups per CU and small tiles keep the slowest wave's share short. Each
// wave owns a contiguous range of whole groups and walks its tiles with two register buffers in
// ping-pong: the next tile's buffer loads are in flight while the current tile is dequantised and
// accumulated, so arithmetic overlaps the stream. Loads are branch-free: lanes past a row end and
// tiles past the wave's range use an out-of-range buffer offset, which returns zeros without
// memory traffic. The prologue stages the input vector in LDS (RMS-normalised when a gain is
// given, the inverse RMS being applied in the epilogue); the first tiles are issued around it (see
// the kernel), and the epilogue's per-row operands (scales, residual) are wave-uniform scalar
// loads, which do not queue behind the vector loads.
//
// INT8 dequantisation happens in registers: each byte b is XOR-ed with 0x80 so that
// v_cvt_f32_ubyte gives b + 128 exactly; the bias is removed once per row as 128 * sum(x); the
// per-row scale is applied after the wave reduction, fused with the epilogue (store, residual
// add or SwiGLU). BF16 weights are widened by a shift.
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

// Rows per group: 2 for the INT8 projections (gate/up: one channel = its gate and up rows), 4 for
// the BF16 LM head. At the 8B shapes 2-row groups measured 4-8 % faster per launch than 4-row
// groups (twice the waves, half the bytes in flight per wave).
constexpr int rows_per_group(int mode) { return mode == GEMV_LMHEAD ? 4 : 2; }
constexpr int kC = 2;             // 1 KiB chunks per tile of the LM head (INT8 projections: 1)
constexpr int kWgPerCu = 4;
constexpr int kNumCu = 256;
constexpr size_t kMaxGemvLds = 159 * 1024;     // gfx950: 160 KiB of LDS per workgroup, minus statics

__device__ __forceinline__ void fma_bytes(float& acc, uint32_t word, const float4& x) {
  const uint32_t u = word ^ 0x80808080u;
  acc = fmaf(float(u & 0xffu), x.x, acc);
  acc = fmaf(float((u >> 8) & 0xffu), x.y, acc);
  acc = fmaf(float((u >> 16) & 0xffu), x.z, acc);
  acc = fmaf(float(u >> 24), x.w, acc);
}

__device__ __forceinline__ void fma_bf16x4(float& acc, uint32_t w0, uint32_t w1, const float4& x) {
  acc = fmaf(bf16_lo(w0), x.x, acc);
  acc = fmaf(bf16_hi(w0), x.y, acc);
  acc = fmaf(bf16_lo(w1), x.z, acc);
  acc = fmaf(bf16_hi(w1), x.w, acc);
}

// Stage B input rows of K floats into LDS (swizzled, zero padded to KP).
// Thread t owns the float4 at columns 1024 i + 4 t (i < KP / 1024); loads are issued in
// batches of 8 (4 for BF16 rows) before any use. With a gain the LDS holds x * gamma and the
// row's inverse RMS is returned in xscale (applied after the dot product: W (c x) = c (W x));
// without, xscale = 1.
// For INT8 rows bias = 128 * sum of the staged values (removes the +128 of the byte conversion).
// `after_first` runs right after the first batch of input loads is issued: the caller may issue
// its first weight tile there. Vector loads retire in issue order, so waiting for the input
// batch then does not wait for the weights, and the weight stream starts before the input
// arrives.
template <int B, bool NORM, bool I8, int NW, class F>
__device__ __forceinline__ void stage_inputs(const float* __restrict__ x, int ldx, int K, int KP,
                                             const uint16_t* __restrict__ gamma, float eps,
                                             float* xs, float* red2, float* xscale, float* bias,
                                             F&& after_first) {
  constexpr int kBatch = I8 ? 8 : 4;                    // BF16 rows: fewer registers in flight
  const int tid = threadIdx.x;
  const int n4 = (K + 3) >> 2;                          // float4 slots holding valid columns
  constexpr int NT = NW * kWave;                        // threads of the workgroup
  const int npass = (KP + 4 * NT - 1) / (4 * NT);       // passes of one float4 per thread
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(gamma, uint32_t(NORM ? K : 0) * 2u);
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + size_t(b) * ldx, uint32_t(n4) * 16u);
    float ss = 0.0f, sx = 0.0f;
    int4 xv[kBatch];
    int2 gv[kBatch];
    auto load_batch = [&](int i0) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int c4 = (i0 + u) * NT + tid;             // float4 index
        xv[u] = buf_load16(rx, c4 < n4 ? uint32_t(c4) * 16u : kOOB);
        if (NORM)
          gv[u] = __builtin_bit_cast(int2, __builtin_amdgcn_raw_buffer_load_b64(
                                               rg, c4 < n4 ? int(uint32_t(c4) * 8u) : int(kOOB), 0, 0));
      }
    };
    auto store_batch = [&](int i0) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int i = i0 + u;
        if (i >= npass) break;
        const int k = (i * NT + tid) << 2;
        if (k >= KP) break;
        float4 v = __builtin_bit_cast(float4, xv[u]);
        // columns K.. of a partial float4 are zero
        if (k + 0 >= K) v.x = 0.0f;
        if (k + 1 >= K) v.y = 0.0f;
        if (k + 2 >= K) v.z = 0.0f;
        if (k + 3 >= K) v.w = 0.0f;
        if (NORM) {
          ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, ss))));
          v.x *= bf16_lo(uint32_t(gv[u].x));
          v.y *= bf16_hi(uint32_t(gv[u].x));
          v.z *= bf16_lo(uint32_t(gv[u].y));
          v.w *= bf16_hi(uint32_t(gv[u].y));
        }
        sx += (v.x + v.y) + (v.z + v.w);
        *reinterpret_cast<float4*>(xs + size_t(b) * KP + (I8 ? xs_slot_i8(k) : xs_slot_bf16(k))) = v;
      }
    };
    // the first batch is peeled so that the caller's loads sit between its issue and its use
    // without a branch around them
    load_batch(0);
    if (b == 0) after_first();
    store_batch(0);
    for (int i0 = kBatch; i0 < npass; i0 += kBatch) {
      load_batch(i0);
      store_batch(i0);
    }
    // one block reduction for both sums
    ss = wave_sum(ss);
    sx = wave_sum(sx);
    __syncthreads();
    if ((tid & 63) == 0) {
      red2[(tid >> 6) * 2] = ss;
      red2[(tid >> 6) * 2 + 1] = sx;
    }
    __syncthreads();
    float tss = 0.0f, tsx = 0.0f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      tss += red2[2 * w];
      tsx += red2[2 * w + 1];
    }
    xscale[b] = NORM ? rsqrtf(tss / float(K) + eps) : 1.0f;
    bias[b] = I8 ? 128.0f * tsx : 0.0f;
  }
  __syncthreads();
}

// At most 128 VGPRs, so that four waves share each SIMD (the grid is sized for that). NW waves
// per workgroup: 4, or 8 where the staged input leaves room for fewer than four workgroups per
// CU (the same waves per CU with half the staging).
template <int B, int MODE, int NW>
__global__ __launch_bounds__(NW * kWave) __attribute__((amdgpu_waves_per_eu(4))) void gemv_kernel(GemvArgs a) {
  constexpr int kR = rows_per_group(MODE);
  // 1 KiB chunks per tile: 1 for the INT8 projections (gate/up 1.5 % faster than 2 or 4 at the 8B
  // shape; QKV, O and down at the 70B shape 8.73 -> 8.65 ms per token, the 8B layer unchanged),
  // 2 for the LM head
  constexpr int kC = (MODE == GEMV_LMHEAD) ? ::tasp::kC : 1;
  constexpr bool BF = (MODE == GEMV_LMHEAD);
  constexpr bool NORM = (MODE != GEMV_RESID);
  constexpr int CPC = BF ? 512 : 1024;                 // columns per 1 KiB chunk
  constexpr int LCOL = BF ? 8 : 16;                    // columns per lane load
  extern __shared__ __attribute__((aligned(16))) float xs[];
  __shared__ float red2[2 * NW];
  const float* __restrict__ scale = a.scale;
  const float* __restrict__ scale2 = a.scale2;
  const float* __restrict__ resid = a.resid;
  const int K = a.K, N = a.N;
  const int KP = (K + 1023) & ~1023;
  const int nchunks = (K + CPC - 1) / CPC;
  // tiles per group; at least one, so that an empty input (no retained heads or channels) still
  // writes the epilogue (residual + 0)
  const int KB = max(1, (nchunks + kC - 1) / kC);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * NW + (threadIdx.x >> 6));
  const int nwaves = gridDim.x * NW;
  constexpr int CH = kR / 2;                           // gate/up: channels per group
  const int per_group = (MODE == GEMV_GATEUP) ? CH : kR;
  const int G = (N + per_group - 1) / per_group;
  const int g0 = int((long(wave) * G) / nwaves), g1 = int((long(wave + 1) * G) / nwaves);
  const int t_begin = g0 * KB, t_end = g1 * KB;
  const uint32_t row_bytes = BF ? uint32_t(K) * 2u : uint32_t(a.ld);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, uint32_t(N) * row_bytes);
  const __amdgpu_buffer_rsrc_t rw2 =
      make_rsrc(MODE == GEMV_GATEUP ? a.w2 : a.w, uint32_t(N) * row_bytes);

  auto row_of = [&](int gi, int r) {
    return (MODE == GEMV_GATEUP) ? gi * CH + (r % CH) : gi * kR + r;
  };
  // A wave issuing its next tile's loads runs at raised priority, so that the address stream is
  // not held behind other waves' dequantisation (measured 1 % on gate/up).
  auto issue = [&](int t, int4 (&w)[kC][kR]) {
    __builtin_amdgcn_s_setprio(2);
    const bool ok_t = t < t_end;
    const int gi = ok_t ? t / KB : 0;
    const int kb = t - gi * KB;
#pragma unroll
    for (int u = 0; u < kC; ++u) {
      const int k = (kb * kC + u) * CPC + lane * LCOL;
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const int row = row_of(gi, r);
        const bool ok = ok_t && (row < N) && (k < K);
        const uint32_t off = ok ? uint32_t(row) * row_bytes + uint32_t(k) * (BF ? 2u : 1u) : kOOB;
        w[u][r] = buf_load16_stream((MODE == GEMV_GATEUP && r >= CH) ? rw2 : rw, off);
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };

  // Epilogue operands (scales, residual) of the wave's first group: scalar loads issued ahead of
  // the staging and held (the empty asm below keeps them there), so their latency is hidden by it
  // instead of stalling the first group's epilogue (measured 0.2 us per 8B layer step).
  float s1p[kR], s2p[CH], resp[B][kR];
  {
    const int row0 = row_of(g0, 0);
#pragma unroll
    for (int r = 0; r < kR; ++r) {
      const int row = min(MODE == GEMV_GATEUP ? row0 + (r % CH) : row0 + r, N - 1);
      s1p[r] = BF ? 1.0f : scale[row];
      if (MODE == GEMV_GATEUP && r < CH) s2p[r] = scale2[row];
#pragma unroll
      for (int b = 0; b < B; ++b)
        resp[b][r] = (MODE == GEMV_RESID) ? resid[size_t(b) * a.ldy + row] : 0.0f;
    }
  }

  // The first weight tile is issued between the input loads and their use, so that the weight
  // stream starts one memory latency before the staged input is ready (for gate/up too: at the
  // 70B shape 8.86 -> 8.75 ms per token, neutral at the 8B layer).
  int4 wa[kC][kR], wb[kC][kR];
  float xscale[B], bias[B];
  stage_inputs<B, NORM, !BF, NW>(a.x, a.ldx, K, KP, a.gamma, a.eps, xs, red2, xscale, bias,
                                 [&] { issue(t_begin, wa); });
  issue(t_begin + 1, wb);
#pragma unroll
  for (int r = 0; r < kR; ++r) {
    asm volatile("" : "+s"(s1p[r]));
#pragma unroll
    for (int b = 0; b < B; ++b) asm volatile("" : "+s"(resp[b][r]));
  }
#pragma unroll
  for (int r = 0; r < CH; ++r) asm volatile("" : "+s"(s2p[r]));

  float acc[B][kR];
  float s1[kR], s2[CH], res[B][kR];
  auto process = [&](const int4 (&w)[kC][kR], int t) {
    const int gi = t / KB;
    const int kb = t - gi * KB;
    const int row0 = row_of(gi, 0);
    if (kb == 0) {
#pragma unroll
      for (int b = 0; b < B; ++b)
#pragma unroll
        for (int r = 0; r < kR; ++r) acc[b][r] = 0.0f;
      // epilogue operands: wave-uniform addresses -> scalar loads
      if (gi == g0) {
#pragma unroll
        for (int r = 0; r < kR; ++r) {
          s1[r] = s1p[r];
          if (MODE == GEMV_GATEUP && r < CH) s2[r] = s2p[r];
#pragma unroll
          for (int b = 0; b < B; ++b) res[b][r] = resp[b][r];
        }
      } else
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const int row = min(MODE == GEMV_GATEUP ? row0 + (r % CH) : row0 + r, N - 1);
        s1[r] = BF ? 1.0f : scale[row];
        if (MODE == GEMV_GATEUP && r < CH) s2[r] = scale2[row];
#pragma unroll
        for (int b = 0; b < B; ++b)
          res[b][r] = (MODE == GEMV_RESID) ? resid[size_t(b) * a.ldy + row] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < kC; ++u) {
      const int c = kb * kC + u;
      if (c >= nchunks) break;
#pragma unroll
      for (int b = 0; b < B; ++b) {
        if (BF) {
          const float4* xp = reinterpret_cast<const float4*>(xs + size_t(b) * KP) + ((c << 1) << 6) + lane;
          const float4 x0 = xp[0], x1 = xp[64];
#pragma unroll
          for (int r = 0; r < kR; ++r) {
            fma_bf16x4(acc[b][r], uint32_t(w[u][r].x), uint32_t(w[u][r].y), x0);
            fma_bf16x4(acc[b][r], uint32_t(w[u][r].z), uint32_t(w[u][r].w), x1);
          }
        } else {
          const float4* xp = reinterpret_cast<const float4*>(xs + size_t(b) * KP) + ((c << 2) << 6) + lane;
          const float4 x0 = xp[0], x1 = xp[64], x2 = xp[128], x3 = xp[192];
#pragma unroll
          for (int r = 0; r < kR; ++r) {
            fma_bytes(acc[b][r], uint32_t(w[u][r].x), x0);
            fma_bytes(acc[b][r], uint32_t(w[u][r].y), x1);
            fma_bytes(acc[b][r], uint32_t(w[u][r].z), x2);
            fma_bytes(acc[b][r], uint32_t(w[u][r].w), x3);
          }
        }
      }
    }
    if (kb != KB - 1) return;
    float tot[B][kR];
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int r = 0; r < kR; ++r) tot[b][r] = wave_sum(acc[b][r]);
    if (lane != 0) return;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float* yb = a.y + size_t(b) * a.ldy;
      if (MODE == GEMV_GATEUP) {
#pragma unroll
        for (int r = 0; r < CH; ++r) {
          const int ch = row0 + r;
          if (ch >= N) continue;
          const float g = s1[r] * xscale[b] * (tot[b][r] - bias[b]);
          const float u = s2[r] * xscale[b] * (tot[b][r + CH] - bias[b]);
          yb[ch] = g / (1.0f + exp2f(-g * kLog2e)) * u;
        }
      } else {
#pragma unroll
        for (int r = 0; r < kR; ++r) {
          const int row = row0 + r;
          if (row >= N) continue;
          yb[row] = res[b][r] + s1[r] * xscale[b] * (tot[b][r] - bias[b]);
        }
      }
    }
  };

  for (int t = t_begin; t < t_end; t += 2) {
    process(wa, t);
    issue(t + 2, wa);
    if (t + 1 < t_end) process(wb, t + 1);
    issue(t + 3, wb);
  }
}

// One wave per group up to the workgroups that fit on the chip at once: kWgPerCu per CU, fewer
// when the staged input limits them (160 KiB of LDS per CU). Past that, waves take several groups
// each, so that no workgroup waits for a second round and stages the input again.
int gemv_per_cu(size_t lds) {
  constexpr size_t kLdsPerCu = 160 * 1024;
  const int by_lds = int(kLdsPerCu / std::max<size_t>(lds + 64, 1));
  return std::max(1, std::min(kWgPerCu, by_lds));
}

int gemv_grid(int n_groups, int per_cu, int nw) {
  const int grid = std::min((n_groups + nw - 1) / nw, kNumCu * per_cu);
  return grid < 1 ? 1 : grid;
}

template <int B, int MODE, int NW>
hipError_t launch_mode(const GemvArgs& a, int grid, size_t lds, hipStream_t s) {
  // dynamic LDS above 64 KiB must be allowed per kernel; done once per instantiation
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&gemv_kernel<B, MODE, NW>),
      hipFuncAttributeMaxDynamicSharedMemorySize, int(kMaxGemvLds));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((gemv_kernel<B, MODE, NW>), dim3(grid), dim3(NW * kWave), lds, s, a);
  return hipGetLastError();
}

template <int B, int MODE>
hipError_t launch_mode_nw(const GemvArgs& a, int n_groups, size_t lds, hipStream_t s) {
  // a wide input (staging LDS for fewer than kWgPerCu workgroups per CU) gets 8-wave workgroups,
  // so that each CU still holds about 16 waves of loads in flight
  const int per_cu = gemv_per_cu(lds);
  if (per_cu < kWgPerCu) return launch_mode<B, MODE, 8>(a, gemv_grid(n_groups, per_cu, 8), lds, s);
  return launch_mode<B, MODE, 4>(a, gemv_grid(n_groups, per_cu, 4), lds, s);
}

template <int B>
hipError_t launch_gemv_b(GemvMode mode, const GemvArgs& a, hipStream_t s) {
  if (a.N < 1) return hipSuccess;                       // no output rows: nothing to launch
  const int per_group = (mode == GEMV_GATEUP) ? rows_per_group(mode) / 2 : rows_per_group(mode);
  const size_t lds = gemv_lds_bytes(B, a.K);
  const int n_groups = (a.N + per_group - 1) / per_group;
  if (lds > kMaxGemvLds) return hipErrorInvalidValue;
  switch (mode) {
    case GEMV_QKV: return launch_mode_nw<B, GEMV_QKV>(a, n_groups, lds, s);
    case GEMV_RESID: return launch_mode_nw<B, GEMV_RESID>(a, n_groups, lds, s);
    case GEMV_GATEUP: return launch_mode_nw<B, GEMV_GATEUP>(a, n_groups, lds, s);
    case GEMV_LMHEAD: return launch_mode_nw<B, GEMV_LMHEAD>(a, n_groups, lds, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

size_t gemv_lds_bytes(int B, int K) { return size_t(B) * ((K + 1023) & ~1023) * sizeof(float); }

hipError_t launch_gemv(GemvMode mode, const GemvArgs& a, hipStream_t s) {
  // one sequence; batches of 2..8 run on the matrix cores
  if (a.B != 1) return hipErrorInvalidValue;
  return launch_gemv_b<1>(mode, a, s);
}

}  // namespace tasp

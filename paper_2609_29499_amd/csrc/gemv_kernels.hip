// Decode-time GEMVs over compacted panels: y = s * (P x) with INT8 P, float32 x and float32
// accumulation, memory-bound on the panel stream.
//
// Layout of the work: a workgroup stages its input vector (RMS-normalised in the prologue when a
// gain is given) in LDS once, then each wave walks row groups (4 rows, or 2 SwiGLU channels =
// 2 gate + 2 up rows) in a grid-stride loop. For a row group a lane issues 16-byte loads at chunk
// offset 16*lane of every 1 KiB chunk of each row, so a wave reads whole contiguous KiB; 4 chunks
// x 4 rows are in flight per lane before any arithmetic. Dequantisation happens in registers:
// each int8 byte b is XOR-ed with 0x80 so that v_cvt_f32_ubyte gives b + 128 exactly, and the
// bias is removed once per row as 128 * sum(x). The per-row scale is applied after the wave
// reduction, together with the fused epilogue (plain store, residual add, or SwiGLU).
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

constexpr int kRowsPerGroup = 4;
constexpr int kChunksInFlight = 4;
constexpr int kWgPerCu = 2;
constexpr int kNumCu = 256;

__device__ __forceinline__ void fma_bytes(float& acc, uint32_t word, const float4& x) {
  const uint32_t u = word ^ 0x80808080u;
  acc = fmaf(float(u & 0xffu), x.x, acc);
  acc = fmaf(float((u >> 8) & 0xffu), x.y, acc);
  acc = fmaf(float((u >> 16) & 0xffu), x.z, acc);
  acc = fmaf(float(u >> 24), x.w, acc);
}

// Stage B input rows of K floats into LDS (swizzled, zero padded to KP) and return sum(x) per row.
template <int B, bool NORM, bool I8>
__device__ __forceinline__ void stage_inputs(const float* __restrict__ x, int ldx, int K, int KP,
                                             const uint16_t* __restrict__ gamma, float eps,
                                             float* xs, float* red, float* sumx) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int b = 0; b < B; ++b) {
    const float* xr = x + size_t(b) * ldx;
    float inv = 1.0f;
    if (NORM) {
      float ss = 0.0f;
      for (int k = tid; k < K; k += kBlock) {
        const float v = xr[k];
        ss = fmaf(v, v, ss);
      }
      ss = block_sum(ss, red);
      inv = rsqrtf(ss / float(K) + eps);
    }
    float sx = 0.0f;
    for (int k = tid; k < KP; k += kBlock) {
      float v = 0.0f;
      if (k < K) {
        v = xr[k];
        if (NORM) v = (v * inv) * bf16_to_f32(gamma[k]);
      }
      xs[size_t(b) * KP + (I8 ? xs_slot_i8(k) : xs_slot_bf16(k))] = v;
      sx += v;
    }
    sumx[b] = block_sum(sx, red);
  }
  __syncthreads();
}

template <int B, int MODE>
__global__ __launch_bounds__(kBlock) void gemv_i8_kernel(GemvArgs a) {
  extern __shared__ __attribute__((aligned(16))) float xs[];
  __shared__ float red[4];
  const int K = a.K;
  const int KP = (K + 1023) & ~1023;
  float sumx[B];
  stage_inputs<B, MODE != GEMV_RESID, true>(a.x, a.ldx, K, KP, a.gamma, a.eps, xs, red, sumx);

  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kBlock / kWave) + (threadIdx.x >> 6);
  const int nwaves = gridDim.x * (kBlock / kWave);
  const int per_group = (MODE == GEMV_GATEUP) ? 2 : kRowsPerGroup;
  const int n_groups = (a.N + per_group - 1) / per_group;
  const int nchunks = (K + 1023) >> 10;

  for (int gi = wave; gi < n_groups; gi += nwaves) {
    const int8_t* rp[kRowsPerGroup];
    bool rv[kRowsPerGroup];
    int row0;
    if (MODE == GEMV_GATEUP) {
      row0 = gi * 2;
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) {
        const int ch = row0 + (r & 1);
        rv[r] = ch < a.N;
        rp[r] = (r < 2 ? a.w : a.w2) + size_t(rv[r] ? ch : 0) * a.ld;
      }
    } else {
      row0 = gi * kRowsPerGroup;
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) {
        rv[r] = row0 + r < a.N;
        rp[r] = a.w + size_t(rv[r] ? row0 + r : 0) * a.ld;
      }
    }
    float acc[B][kRowsPerGroup];
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) acc[b][r] = 0.0f;

    for (int c0 = 0; c0 < nchunks; c0 += kChunksInFlight) {
      int4 wv[kChunksInFlight][kRowsPerGroup];
#pragma unroll
      for (int u = 0; u < kChunksInFlight; ++u) {
        const int k = ((c0 + u) << 10) + (lane << 4);
#pragma unroll
        for (int r = 0; r < kRowsPerGroup; ++r) {
          if (rv[r] && c0 + u < nchunks && k < K)
            wv[u][r] = *reinterpret_cast<const int4*>(rp[r] + k);
          else
            wv[u][r] = make_int4(int(0x80808080u), int(0x80808080u), int(0x80808080u),
                                 int(0x80808080u));
        }
      }
#pragma unroll
      for (int u = 0; u < kChunksInFlight; ++u) {
        const int c = c0 + u;
        if (c >= nchunks) break;
#pragma unroll
        for (int b = 0; b < B; ++b) {
          const float4* xp =
              reinterpret_cast<const float4*>(xs + size_t(b) * KP) + ((c << 2) << 6) + lane;
          const float4 x0 = xp[0], x1 = xp[64], x2 = xp[128], x3 = xp[192];
#pragma unroll
          for (int r = 0; r < kRowsPerGroup; ++r) {
            fma_bytes(acc[b][r], uint32_t(wv[u][r].x), x0);
            fma_bytes(acc[b][r], uint32_t(wv[u][r].y), x1);
            fma_bytes(acc[b][r], uint32_t(wv[u][r].z), x2);
            fma_bytes(acc[b][r], uint32_t(wv[u][r].w), x3);
          }
        }
      }
    }

#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) acc[b][r] = wave_sum(acc[b][r]);

    if (lane == 0) {
#pragma unroll
      for (int b = 0; b < B; ++b) {
        if (b >= a.B) break;
        const float bias = 128.0f * sumx[b];
        float* yb = a.y + size_t(b) * a.ldy;
        if (MODE == GEMV_GATEUP) {
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            if (!rv[r]) continue;
            const int ch = row0 + r;
            const float g = a.scale[ch] * (acc[b][r] - bias);
            const float u = a.scale2[ch] * (acc[b][r + 2] - bias);
            yb[ch] = g / (1.0f + exp2f(-g * kLog2e)) * u;
          }
        } else {
#pragma unroll
          for (int r = 0; r < kRowsPerGroup; ++r) {
            if (!rv[r]) continue;
            const int row = row0 + r;
            const float v = a.scale[row] * (acc[b][r] - bias);
            if (MODE == GEMV_RESID)
              yb[row] = a.resid[size_t(b) * a.ldy + row] + v;
            else
              yb[row] = v;
          }
        }
      }
    }
  }
}

// Dense BF16 LM head: logits = W_lm RMSNorm(r). A 16-byte lane load holds 8 BF16 weights.
template <int B>
__global__ __launch_bounds__(kBlock) void lmhead_kernel(LmHeadArgs a) {
  extern __shared__ __attribute__((aligned(16))) float xs[];
  __shared__ float red[4];
  const int K = a.K;
  const int KP = (K + 511) & ~511;
  float sumx[B];
  stage_inputs<B, true, false>(a.x, a.ldx, K, KP, a.gamma, a.eps, xs, red, sumx);
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kBlock / kWave) + (threadIdx.x >> 6);
  const int nwaves = gridDim.x * (kBlock / kWave);
  const int n_groups = (a.V + kRowsPerGroup - 1) / kRowsPerGroup;
  const int nchunks = (K + 511) >> 9;
  for (int gi = wave; gi < n_groups; gi += nwaves) {
    const int row0 = gi * kRowsPerGroup;
    const uint16_t* rp[kRowsPerGroup];
    bool rv[kRowsPerGroup];
#pragma unroll
    for (int r = 0; r < kRowsPerGroup; ++r) {
      rv[r] = row0 + r < a.V;
      rp[r] = a.w + size_t(rv[r] ? row0 + r : 0) * K;
    }
    float acc[B][kRowsPerGroup];
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) acc[b][r] = 0.0f;
    for (int c0 = 0; c0 < nchunks; c0 += kChunksInFlight) {
      int4 wv[kChunksInFlight][kRowsPerGroup];
#pragma unroll
      for (int u = 0; u < kChunksInFlight; ++u) {
        const int k = ((c0 + u) << 9) + (lane << 3);
#pragma unroll
        for (int r = 0; r < kRowsPerGroup; ++r) {
          if (rv[r] && c0 + u < nchunks && k < K)
            wv[u][r] = *reinterpret_cast<const int4*>(rp[r] + k);
          else
            wv[u][r] = make_int4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int u = 0; u < kChunksInFlight; ++u) {
        const int c = c0 + u;
        if (c >= nchunks) break;
#pragma unroll
        for (int b = 0; b < B; ++b) {
          const float4* xp =
              reinterpret_cast<const float4*>(xs + size_t(b) * KP) + ((c << 1) << 6) + lane;
          const float4 x0 = xp[0], x1 = xp[64];
#pragma unroll
          for (int r = 0; r < kRowsPerGroup; ++r) {
            const uint32_t w0 = wv[u][r].x, w1 = wv[u][r].y, w2 = wv[u][r].z, w3 = wv[u][r].w;
            float s = acc[b][r];
            s = fmaf(bf16_lo(w0), x0.x, s);
            s = fmaf(bf16_hi(w0), x0.y, s);
            s = fmaf(bf16_lo(w1), x0.z, s);
            s = fmaf(bf16_hi(w1), x0.w, s);
            s = fmaf(bf16_lo(w2), x1.x, s);
            s = fmaf(bf16_hi(w2), x1.y, s);
            s = fmaf(bf16_lo(w3), x1.z, s);
            s = fmaf(bf16_hi(w3), x1.w, s);
            acc[b][r] = s;
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int r = 0; r < kRowsPerGroup; ++r) acc[b][r] = wave_sum(acc[b][r]);
    if (lane == 0) {
#pragma unroll
      for (int b = 0; b < B; ++b) {
        if (b >= a.B) break;
#pragma unroll
        for (int r = 0; r < kRowsPerGroup; ++r)
          if (rv[r]) a.y[size_t(b) * a.ldy + row0 + r] = acc[b][r];
      }
    }
  }
}

template <int B>
hipError_t launch_gemv_b(GemvMode mode, const GemvArgs& a, hipStream_t s) {
  const int per_group = (mode == GEMV_GATEUP) ? 2 : kRowsPerGroup;
  const int n_groups = (a.N + per_group - 1) / per_group;
  int grid = (n_groups + 3) / 4;
  if (grid > kNumCu * kWgPerCu) grid = kNumCu * kWgPerCu;
  if (grid < 1) grid = 1;
  const size_t lds = gemv_lds_bytes(B, a.K);
  switch (mode) {
    case GEMV_QKV:
      hipLaunchKernelGGL((gemv_i8_kernel<B, GEMV_QKV>), dim3(grid), dim3(kBlock), lds, s, a);
      break;
    case GEMV_RESID:
      hipLaunchKernelGGL((gemv_i8_kernel<B, GEMV_RESID>), dim3(grid), dim3(kBlock), lds, s, a);
      break;
    case GEMV_GATEUP:
      hipLaunchKernelGGL((gemv_i8_kernel<B, GEMV_GATEUP>), dim3(grid), dim3(kBlock), lds, s, a);
      break;
  }
  return hipGetLastError();
}

template <int B>
hipError_t launch_lmhead_b(const LmHeadArgs& a, hipStream_t s) {
  const int n_groups = (a.V + kRowsPerGroup - 1) / kRowsPerGroup;
  int grid = (n_groups + 3) / 4;
  if (grid > kNumCu * kWgPerCu) grid = kNumCu * kWgPerCu;
  const size_t lds = size_t(B) * ((a.K + 511) & ~511) * sizeof(float);
  hipLaunchKernelGGL((lmhead_kernel<B>), dim3(grid), dim3(kBlock), lds, s, a);
  return hipGetLastError();
}

}  // namespace

size_t gemv_lds_bytes(int B, int K) { return size_t(B) * ((K + 1023) & ~1023) * sizeof(float); }

hipError_t launch_gemv(GemvMode mode, const GemvArgs& a, hipStream_t s) {
  switch (a.B) {
    case 1: return launch_gemv_b<1>(mode, a, s);
    case 2: return launch_gemv_b<2>(mode, a, s);
    case 3: return launch_gemv_b<3>(mode, a, s);
    case 4: return launch_gemv_b<4>(mode, a, s);
    case 5: return launch_gemv_b<5>(mode, a, s);
    case 6: return launch_gemv_b<6>(mode, a, s);
    case 7: return launch_gemv_b<7>(mode, a, s);
    case 8: return launch_gemv_b<8>(mode, a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_lmhead(const LmHeadArgs& a, hipStream_t s) {
  switch (a.B) {
    case 1: return launch_lmhead_b<1>(a, s);
    case 2: return launch_lmhead_b<2>(a, s);
    case 3: return launch_lmhead_b<3>(a, s);
    case 4: return launch_lmhead_b<4>(a, s);
    case 5: return launch_lmhead_b<5>(a, s);
    case 6: return launch_lmhead_b<6>(a, s);
    case 7: return launch_lmhead_b<7>(a, s);
    case 8: return launch_lmhead_b<8>(a, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace tasp

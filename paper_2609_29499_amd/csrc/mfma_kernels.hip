// Batched decode (2..8 sequences) on the matrix cores: y = s * (P u) for every compacted panel P,
// with v_mfma_f32_16x16x32_bf16 and float32 accumulation.
//
// Activation operand. The 16 columns of the MFMA tile carry 8 sequences twice: column 2b holds
// bf16(v) and column 2b+1 holds bf16(v - bf16(v)) for sequence b, so the pair keeps 16 significant
// bits of every activation and one MFMA pass evaluates both halves. The operand lives in HBM as a
// [16][ldx] BF16 matrix; rows >= 2B are never read (their lanes use an out-of-range offset) and
// columns >= K hold finite values that meet zero panel columns. It is written by the epilogue of
// whichever kernel produced the activation (RMSNorm gain applied, the inverse RMS deferred: the
// producer also writes per-16-row-tile sums of squares, which the consumer reduces).
//
// Weights. INT8 rows are widened in registers (sign-extend, convert, keep the upper 16 bits: exact,
// since |w| <= 127 needs 7 significant bits); the BF16 LM head is used as is. One workgroup owns
// one tile of 16 output rows (gate/up: 8 channels, rows 0-7 gate and 8-15 up, so SwiGLU is local)
// and its waves split the K range; every lane streams 16 contiguous bytes of its row per step with
// branch-free buffer loads, double-buffered so the next steps' loads are in flight during the
// current steps' MFMAs. The partial tiles of the waves are summed through LDS, then the epilogue
// applies scale, inverse RMS, residual / SwiGLU, and writes the next operand.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kPF = 4;                 // steps per load batch (two batches in flight)
constexpr int kMaxSsqPerLane = 16;     // sums-of-squares partials per lane: d_model <= 16384

// Two float32 holding values exact in BF16 -> packed BF16 pair (lo in the low half).
__device__ __forceinline__ uint32_t pack_exact(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// 8 signed INT8 weights (two words) -> 8 BF16 values.
__device__ __forceinline__ bf16x8 widen_i8(uint32_t w0, uint32_t w1) {
  int4 r;
  r.x = int(pack_exact(float(int8_t(w0 & 0xffu)), float(int8_t((w0 >> 8) & 0xffu))));
  r.y = int(pack_exact(float(int8_t((w0 >> 16) & 0xffu)), float(int8_t(w0 >> 24))));
  r.z = int(pack_exact(float(int8_t(w1 & 0xffu)), float(int8_t((w1 >> 8) & 0xffu))));
  r.w = int(pack_exact(float(int8_t((w1 >> 16) & 0xffu)), float(int8_t(w1 >> 24))));
  return __builtin_bit_cast(bf16x8, r);
}

__device__ __forceinline__ void store_hilo(uint16_t* xo, int ldxo, int b, int col, float v) {
  const uint16_t hi = f32_to_bf16(v);
  xo[size_t(2 * b) * ldxo + col] = hi;
  xo[size_t(2 * b + 1) * ldxo + col] = f32_to_bf16(v - bf16_to_f32(hi));
}

struct Frag {
  int4 a;        // 16 weight bytes (INT8) or 8 BF16 weights
  int4 x0, x1;   // activation fragments for the step's two MFMAs (x1 unused for BF16 weights)
};

template <int MODE, int WAVES>
__global__ __launch_bounds__(WAVES * kWave) void mfma_gemv_kernel(MfmaArgs a) {
  constexpr bool BF = (MODE == MM_LMHEAD);
  constexpr int KS = BF ? 32 : 64;                      // k per wave step
  __shared__ float red[WAVES][4][kWave];
  __shared__ float tile_s[16][17];
  __shared__ float rs[8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int tile = blockIdx.x;
  const int B = a.B, N = a.N, K = a.K;

  // ---- this lane's weight row and activation column
  int row;
  uint32_t row_base;
  const uint32_t row_bytes = uint32_t(a.ld) * (BF ? 2u : 1u);
  if (MODE == MM_GATEUP) {
    row = tile * 8 + (r & 7);
    row_base = (r < 8 ? 0u : a.w2_off) + uint32_t(row) * row_bytes;
  } else {
    row = tile * 16 + r;
    row_base = uint32_t(row) * row_bytes;
  }
  const bool row_ok = row < N;
  const uint32_t w_bytes = (MODE == MM_GATEUP) ? a.w2_off + uint32_t(N) * row_bytes
                                               : uint32_t(N) * row_bytes;
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, w_bytes);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, uint32_t(2 * B) * uint32_t(a.ldx) * 2u);
  const uint32_t x_base = uint32_t(r) * uint32_t(a.ldx) * 2u;   // >= the record count when r >= 2B

  // ---- this wave's steps
  const int n_steps = (K + KS - 1) / KS;
  const int s0 = (wave * n_steps) / WAVES, s1 = ((wave + 1) * n_steps) / WAVES;
  const int lane_k = q * (BF ? 8 : 16);                 // first k of the lane inside a step

  // RMS partials first (all loads issued before any use): they are L2 hits and retire ahead of
  // the weight stream. Wave w reduces sequences w and w + WAVES; n_ssq <= 16 * 64.
  float ssq_v[2][kMaxSsqPerLane];
  const bool rms = a.ssq != nullptr;
  if (rms) {
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(a.ssq, uint32_t(B) * uint32_t(a.n_ssq) * 4u);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int b = wave + u * WAVES;
#pragma unroll
      for (int i = 0; i < kMaxSsqPerLane; ++i) {
        const int j = i * kWave + lane;
        const uint32_t off = (b < B && j < a.n_ssq) ? (uint32_t(b) * uint32_t(a.n_ssq) + uint32_t(j)) * 4u : kOOB;
        ssq_v[u][i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rq, int(off), 0, 0));
      }
    }
  }
  // epilogue operands of the threads that write outputs
  float e_s1 = 1.0f, e_s2 = 1.0f, e_res = 0.0f, e_g = 0.0f;
  {
    if (MODE == MM_GATEUP) {
      const int ch = tile * 8 + (tid & 7), b = tid >> 3;
      if (b < B && ch < N) { e_s1 = a.scale[ch]; e_s2 = a.scale2[ch]; }
    } else if (MODE != MM_LMHEAD) {
      const int gr = tile * 16 + (tid & 15), b = tid >> 4;
      if (b < B && gr < N) {
        e_s1 = a.scale[gr];
        if (MODE == MM_RESID) {
          e_res = a.resid[size_t(b) * a.ldy + gr];
          if (a.gamma_next) e_g = bf16_to_f32(a.gamma_next[gr]);
        }
      }
    }
  }

  auto issue = [&](int t, Frag (&f)[kPF]) {
#pragma unroll
    for (int u = 0; u < kPF; ++u) {
      const int step = t + u;
      const int k = step * KS + lane_k;
      const bool ok = step < s1;
      const uint32_t wo = (ok && row_ok && k < a.ld) ? row_base + uint32_t(k) * (BF ? 2u : 1u) : kOOB;
      const uint32_t xo = ok ? x_base + uint32_t(k) * 2u : kOOB;
      f[u].a = buf_load16(rw, wo);
      f[u].x0 = buf_load16(rx, xo);
      if (!BF) f[u].x1 = buf_load16(rx, xo + 16u);
    }
  };

  f32x4 acc0 = {0.0f, 0.0f, 0.0f, 0.0f}, acc1 = {0.0f, 0.0f, 0.0f, 0.0f};
  auto process = [&](const Frag (&f)[kPF], int t) {
#pragma unroll
    for (int u = 0; u < kPF; ++u) {
      if (t + u >= s1) break;
      if (BF) {
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f[u].a),
                                                       __builtin_bit_cast(bf16x8, f[u].x0), acc0, 0, 0, 0);
      } else {
        const bf16x8 w_lo = widen_i8(uint32_t(f[u].a.x), uint32_t(f[u].a.y));
        const bf16x8 w_hi = widen_i8(uint32_t(f[u].a.z), uint32_t(f[u].a.w));
        acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w_lo, __builtin_bit_cast(bf16x8, f[u].x0), acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w_hi, __builtin_bit_cast(bf16x8, f[u].x1), acc1, 0, 0, 0);
      }
    }
  };

  Frag fa[kPF], fb[kPF];
  issue(s0, fa);
  if (rms) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int b = wave + u * WAVES;
      float t = 0.0f;
#pragma unroll
      for (int i = 0; i < kMaxSsqPerLane; ++i) t += ssq_v[u][i];
      t = wave_sum(t);
      if (b < B && lane == 0) rs[b] = rsqrtf(t * a.inv_d + a.eps);
    }
  }
  for (int t = s0; t < s1; t += 2 * kPF) {
    issue(t + kPF, fb);
    process(fa, t);
    issue(t + 2 * kPF, fa);
    process(fb, t + kPF);
  }

  // ---- sum the waves' partial tiles: lane holds D[4q + i][r]
#pragma unroll
  for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc0[i] + acc1[i];
  __syncthreads();
  if (tid < 256) {
    const int i = tid >> 6, l = tid & 63;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) v += red[w][i][l];
    tile_s[4 * (l >> 4) + i][l & 15] = v;
  }
  __syncthreads();

  // ---- epilogue
  if (MODE == MM_GATEUP) {
    const int chl = tid & 7, b = tid >> 3, ch = tile * 8 + chl;
    if (b >= B || ch >= N) return;
    const float rb = rms ? rs[b] : 1.0f;
    const float g = (tile_s[chl][2 * b] + tile_s[chl][2 * b + 1]) * e_s1 * rb;
    const float u = (tile_s[8 + chl][2 * b] + tile_s[8 + chl][2 * b + 1]) * e_s2 * rb;
    store_hilo(a.xo, a.ldxo, b, ch, g / (1.0f + exp2f(-g * kLog2e)) * u);
    return;
  }
  const int rl = tid & 15, b = tid >> 4, gr = tile * 16 + rl;
  if (b >= B) return;                                   // whole rows of 16 lanes stay together
  const float rb = rms ? rs[b] : 1.0f;
  const float dot = tile_s[rl][2 * b] + tile_s[rl][2 * b + 1];
  if (MODE == MM_RESID) {
    const float v = gr < N ? e_res + dot * e_s1 * rb : 0.0f;
    if (gr < N) a.y[size_t(b) * a.ldy + gr] = v;
    if (a.gamma_next) {
      if (gr < N) store_hilo(a.xo, a.ldxo, b, gr, v * e_g);
      const float ss = row16_sum(v * v);
      if (rl == 0) a.ssq_out[size_t(b) * a.n_tiles_out + tile] = ss;
    }
    return;
  }
  if (gr >= N) return;
  a.y[size_t(b) * a.ldy + gr] = (MODE == MM_LMHEAD) ? dot * rb : dot * e_s1 * rb;
}

// First operand of a step: u = x * gamma as hi/lo BF16 and per-16-element sums of squares of x.
__global__ __launch_bounds__(kBlock) void mfma_prep_kernel(const float* __restrict__ x, int ldx, int D,
                                                           const uint16_t* __restrict__ gamma,
                                                           uint16_t* xo, int ldxo, float* ssq,
                                                           int n_tiles) {
  const int b = blockIdx.y, i = blockIdx.x * kBlock + threadIdx.x;
  const float v = i < D ? x[size_t(b) * ldx + i] : 0.0f;
  if (i < D) store_hilo(xo, ldxo, b, i, v * bf16_to_f32(gamma[i]));
  const float ss = row16_sum(v * v);
  if ((threadIdx.x & 15) == 0 && i < D) ssq[size_t(b) * n_tiles + (i >> 4)] = ss;
}

template <int MODE, int WAVES>
hipError_t launch_mm(const MfmaArgs& a, int grid, hipStream_t s) {
  hipLaunchKernelGGL((mfma_gemv_kernel<MODE, WAVES>), dim3(grid), dim3(WAVES * kWave), 0, s, a);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_mm_mode(const MfmaArgs& a, hipStream_t s) {
  const int tiles = (MODE == MM_GATEUP) ? (a.N + 7) / 8 : (a.N + 15) / 16;
  if (tiles == 0) return hipSuccess;
  // small panels: more waves per tile so that enough loads are in flight
  return tiles >= 1024 ? launch_mm<MODE, 4>(a, tiles, s) : launch_mm<MODE, 8>(a, tiles, s);
}

}  // namespace

hipError_t launch_mfma_gemv(MfmaMode mode, const MfmaArgs& a, hipStream_t s) {
  if (a.B < 1 || a.B > 8 || a.K < 0 || a.K > a.ld || a.ld % 16 != 0 || a.ldx % 64 != 0 ||
      a.ldx < a.K || (a.ssq && a.n_ssq > kMaxSsqPerLane * kWave))
    return hipErrorInvalidValue;
  switch (mode) {
    case MM_QKV: return launch_mm_mode<MM_QKV>(a, s);
    case MM_RESID: return launch_mm_mode<MM_RESID>(a, s);
    case MM_GATEUP: return launch_mm_mode<MM_GATEUP>(a, s);
    case MM_LMHEAD: return launch_mm_mode<MM_LMHEAD>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_mfma_prep(const float* x, int ldx, int D, const uint16_t* gamma, uint16_t* xo,
                            int ldxo, float* ssq, int B, hipStream_t s) {
  if (D % 16 != 0 || B < 1 || B > 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_prep_kernel, dim3((D + kBlock - 1) / kBlock, B), dim3(kBlock), 0, s, x,
                     ldx, D, gamma, xo, ldxo, ssq, D / 16);
  return hipGetLastError();
}

}  // namespace tasp

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

constexpr int kStepsPerBatch = 4;      // 16-row weight loads per lane and load batch
constexpr int kNumCu = 256;
constexpr int kMmTwoTileRows = 8192;   // panels at least this tall use two row tiles per wave
constexpr int kSsqBatch = 8;           // sums-of-squares partials loaded per thread and round

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

template <int RT>
struct Frag {
  int4 a[RT];    // 16 weight bytes (INT8) or 8 BF16 weights of each row tile
  int4 x0, x1;   // activation fragments for the step's two k halves (x1 unused for BF16 weights)
};

// Per-thread epilogue operands of one tile (thread -> (row, sequence) of the output tile).
struct EpiOps {
  float s1, s2, res, g;
};

// Persistent: workgroup w serves tiles w, w + grid, ... A tile is RT row tiles of 16 rows (gate/up:
// 8 RT channels, gate rows then up rows); every wave computes all RT row tiles over its K run,
// so each activation fragment it loads feeds RT MFMAs. The waves split each tile's K range into
// equal runs of spw steps (a multiple of the batch; steps past K are skipped), so every wave reaches a
// tile boundary at the same flattened step and the cross-wave reduction lines up. The load
// stream runs across tile boundaries: the first steps of the next tile are in flight while the
// current tile is reduced and stored.
template <int MODE, int WAVES, int RT>
__global__ __launch_bounds__(WAVES * kWave) void mfma_gemv_kernel(MfmaArgs a) {
  constexpr int kPF = kStepsPerBatch / RT;             // steps per load batch (two batches in flight)
  constexpr bool BF = (MODE == MM_LMHEAD);
  constexpr bool GU = (MODE == MM_GATEUP);
  constexpr int KS = BF ? 32 : 64;                      // k per wave step
  constexpr int ROWS = 16 * RT;                         // tile rows
  constexpr int RPT = GU ? 8 * RT : ROWS;               // output rows (channels) per tile
  __shared__ float red[WAVES][4 * RT][kWave];
  __shared__ float tile_s[ROWS][17];
  __shared__ float rs[8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int B = a.B, N = a.N, K = a.K;
  const int n_tiles = (N + RPT - 1) / RPT;
  const int grid = gridDim.x, wg = blockIdx.x;
  const int my_tiles = wg < n_tiles ? (n_tiles - 1 - wg) / grid + 1 : 0;
  const int n_steps = (K + KS - 1) / KS;
  // at least one batch per tile, so that an empty input still writes its epilogue
  const int spw = max(kPF, ((n_steps + WAVES - 1) / WAVES + kPF - 1) / kPF * kPF);
  const int total = my_tiles * spw;

  const uint32_t esz = BF ? 2u : 1u;
  const uint32_t row_bytes = uint32_t(a.ld) * esz;
  const uint32_t w_bytes = GU ? a.w2_off + uint32_t(N) * row_bytes : uint32_t(N) * row_bytes;
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, w_bytes);
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, uint32_t(2 * B) * uint32_t(a.ldx) * 2u);
  const uint32_t x_base = uint32_t(r) * uint32_t(a.ldx) * 2u;   // >= the record count when r >= 2B
  const int lane_k = q * (BF ? 8 : 16);                 // first k of the lane inside a step

  // row of this lane in row tile rt of a tile, and the byte offset of its panel
  auto lane_row = [&](int tile, int rt) {
    if (GU) return tile * RPT + (RT == 1 ? (r & 7) : r);
    return tile * ROWS + 16 * rt + r;
  };
  auto lane_half = [&](int rt) -> uint32_t {
    if (!GU) return 0u;
    return (RT == 1 ? (r >= 8) : (rt == 1)) ? a.w2_off : 0u;
  };

  // epilogue thread roles and their operand resources (out-of-range offsets read zero)
  const int e_b = tid / RPT, e_r = tid % RPT;           // gate/up: channel e_r, else row e_r
  const __amdgpu_buffer_rsrc_t rs1 = make_rsrc(BF ? nullptr : a.scale, BF ? 0u : uint32_t(N) * 4u);
  const __amdgpu_buffer_rsrc_t rs2 = make_rsrc(GU ? a.scale2 : nullptr, GU ? uint32_t(N) * 4u : 0u);
  const bool resid_on = (MODE == MM_RESID);
  const __amdgpu_buffer_rsrc_t rres =
      make_rsrc(resid_on ? a.resid : nullptr, resid_on ? uint32_t(B) * uint32_t(a.ldy) * 4u : 0u);
  const bool gam_on = resid_on && a.gamma_next != nullptr;
  const __amdgpu_buffer_rsrc_t rgam = make_rsrc(gam_on ? a.gamma_next : nullptr, gam_on ? uint32_t(N) * 2u : 0u);

  auto load_ops = [&](int tile, EpiOps& e) {
    const int row = tile * RPT + e_r;
    const bool ok = e_b < B && row < N;
    const uint32_t o4 = ok ? uint32_t(row) * 4u : kOOB;
    e.s1 = BF ? 1.0f : __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs1, int(o4), 0, 0));
    e.s2 = GU ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs2, int(o4), 0, 0)) : 1.0f;
    e.res = resid_on ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                           rres, int(ok ? (uint32_t(e_b) * uint32_t(a.ldy) + uint32_t(row)) * 4u : kOOB), 0, 0))
                     : 0.0f;
    e.g = gam_on ? bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rgam, int(ok ? uint32_t(row) * 2u : kOOB), 0, 0))
                 : 0.0f;
  };

  EpiOps ops0{}, ops1{};
  auto issue = [&](int g, Frag<RT> (&f)[kPF]) {
    const int i = g / spw, jb = g - i * spw;
    const int tile = wg + i * grid;
    const bool ok_t = g < total;
    if (ok_t && jb == 0) {
      if (i & 1) load_ops(tile, ops1); else load_ops(tile, ops0);
    }
#pragma unroll
    for (int u = 0; u < kPF; ++u) {
      const int step = wave * spw + jb + u;
      const int k = step * KS + lane_k;
      const bool ok = ok_t && step < n_steps;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int row = lane_row(tile, rt);
        const uint32_t wo = (ok && row < N && k < a.ld)
                                ? lane_half(rt) + uint32_t(row) * row_bytes + uint32_t(k) * esz : kOOB;
        f[u].a[rt] = buf_load16_stream(rw, wo);
      }
      const uint32_t xo = ok ? x_base + uint32_t(k) * 2u : kOOB;
      f[u].x0 = buf_load16(rx, xo);
      if (!BF) f[u].x1 = buf_load16(rx, xo + 16u);
    }
  };

  f32x4 acc0[RT], acc1[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    acc0[rt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    acc1[rt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  auto epilogue = [&](int tile, const EpiOps& e) {
    // sum the waves' partial tiles: lane holds D[4q + i][r] of each row tile
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][4 * rt + i][lane] = acc0[rt][i] + acc1[rt][i];
      acc0[rt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      acc1[rt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    __syncthreads();
    for (int idx = tid; idx < 256 * RT; idx += WAVES * kWave) {
      const int ri = idx >> 6, l = idx & 63;            // ri = 4 rt + i
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) v += red[w][ri][l];
      tile_s[16 * (ri >> 2) + 4 * (l >> 4) + (ri & 3)][l & 15] = v;
    }
    __syncthreads();
    const int b = e_b;
    if (b >= B) return;
    const float rb = a.ssq ? rs[b] : 1.0f;
    if (GU) {
      const int ch = tile * RPT + e_r;
      if (ch >= N) return;
      const float gv = (tile_s[e_r][2 * b] + tile_s[e_r][2 * b + 1]) * e.s1 * rb;
      const float uv = (tile_s[RPT + e_r][2 * b] + tile_s[RPT + e_r][2 * b + 1]) * e.s2 * rb;
      store_hilo(a.xo, a.ldxo, b, ch, gv / (1.0f + exp2f(-gv * kLog2e)) * uv);
      return;
    }
    const int gr = tile * RPT + e_r;
    const float dot = tile_s[e_r][2 * b] + tile_s[e_r][2 * b + 1];
    if (MODE == MM_RESID) {
      const float v = gr < N ? e.res + dot * e.s1 * rb : 0.0f;
      if (gr < N) a.y[size_t(b) * a.ldy + gr] = v;
      if (gam_on) {                                     // each 16-lane row: one sequence, 16 rows
        if (gr < N) store_hilo(a.xo, a.ldxo, b, gr, v * e.g);
        const float ss = row16_sum(v * v);
        if ((e_r & 15) == 0 && gr < N) a.ssq_out[size_t(b) * a.n_tiles_out + (gr >> 4)] = ss;
      }
      return;
    }
    if (gr < N) a.y[size_t(b) * a.ldy + gr] = dot * e.s1 * rb;
  };

  auto process = [&](const Frag<RT> (&f)[kPF], int g) {
    if (g >= total) return;
    const int i = g / spw, jb = g - i * spw;
#pragma unroll
    for (int u = 0; u < kPF; ++u) {
      if (wave * spw + jb + u >= n_steps) break;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if (BF) {
          acc0[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f[u].a[rt]),
                                                             __builtin_bit_cast(bf16x8, f[u].x0), acc0[rt], 0, 0, 0);
        } else {
          const bf16x8 w_lo = widen_i8(uint32_t(f[u].a[rt].x), uint32_t(f[u].a[rt].y));
          const bf16x8 w_hi = widen_i8(uint32_t(f[u].a[rt].z), uint32_t(f[u].a[rt].w));
          acc0[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w_lo, __builtin_bit_cast(bf16x8, f[u].x0), acc0[rt], 0, 0, 0);
          acc1[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w_hi, __builtin_bit_cast(bf16x8, f[u].x1), acc1[rt], 0, 0, 0);
        }
      }
    }
    if (jb + kPF == spw) {
      if (i & 1) epilogue(wg + i * grid, ops1); else epilogue(wg + i * grid, ops0);
    }
  };

  Frag<RT> fa[kPF], fb[kPF];
  issue(0, fa);
  // inverse RMS of every sequence, once per workgroup: thread t sums the partials
  // ssq[t / 32][j], j = t % 32 (mod 32); visible after the first epilogue barrier
  if (a.ssq && tid < 256) {
    const int b = tid >> 5;
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(a.ssq, uint32_t(B) * uint32_t(a.n_ssq) * 4u);
    float v = 0.0f;
    for (int j0 = 0; j0 < a.n_ssq; j0 += 32 * kSsqBatch) {
      float t[kSsqBatch];
#pragma unroll
      for (int u = 0; u < kSsqBatch; ++u) {
        const int j = j0 + u * 32 + (tid & 31);
        const uint32_t off = (b < B && j < a.n_ssq) ? (uint32_t(b) * uint32_t(a.n_ssq) + uint32_t(j)) * 4u : kOOB;
        t[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rq, int(off), 0, 0));
      }
#pragma unroll
      for (int u = 0; u < kSsqBatch; ++u) v += t[u];
    }
    v = row16_sum(v);
    v += __shfl_xor(v, 16, kWave);
    if ((tid & 31) == 0 && b < B) rs[b] = rsqrtf(v * a.inv_d + a.eps);
  }
  for (int g = 0; g < total; g += 2 * kPF) {
    issue(g + kPF, fb);
    process(fa, g);
    issue(g + 2 * kPF, fa);
    process(fb, g + kPF);
  }
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

template <int MODE, int WAVES, int RT>
hipError_t launch_mm(const MfmaArgs& a, hipStream_t s) {
  const int rpt = (MODE == MM_GATEUP) ? 8 * RT : 16 * RT;
  const int tiles = (a.N + rpt - 1) / rpt;
  if (tiles == 0) return hipSuccess;
  // resident workgroups per CU at this kernel's register and LDS use, queried once
  static int per_cu = [] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, mfma_gemv_kernel<MODE, WAVES, RT>,
                                                     WAVES * kWave, 0) != hipSuccess || n < 1)
      n = 1;
    return n;
  }();
  const int grid = tiles < per_cu * kNumCu ? tiles : per_cu * kNumCu;
  hipLaunchKernelGGL((mfma_gemv_kernel<MODE, WAVES, RT>), dim3(grid), dim3(WAVES * kWave), 0, s, a);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_mm_mode(const MfmaArgs& a, hipStream_t s) {
  // two row tiles per wave halve the activation reads per weight byte; panels with few rows
  // keep one so that every CU gets a tile, with more waves per tile so that enough loads fly
  const int rows = (MODE == MM_GATEUP) ? 2 * a.N : a.N;
  if (rows >= kMmTwoTileRows) return launch_mm<MODE, 4, 2>(a, s);
  return launch_mm<MODE, 8, 1>(a, s);
}

}  // namespace

hipError_t launch_mfma_gemv(MfmaMode mode, const MfmaArgs& a, hipStream_t s) {
  if (a.B < 1 || a.B > 8 || a.K < 0 || a.K > a.ld || a.ld % 16 != 0 || a.ldx % 64 != 0 ||
      a.ldx < a.K)
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

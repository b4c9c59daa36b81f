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
//
// Groupwise store (shared-store plans). The weights come from the store through the plan's row
// map (QKV, gate/up) or 16-column piece map (O, down, staged in LDS), and a lane's 16 bytes lie in
// one piece, hence in one group of 128 columns: it loads the group's BF16 scale with them and
// forms w = q * s in float32, exact (7 + 8 significant bits), then splits it into BF16 hi and lo
// parts (exact as well: the lo part keeps at most 7 bits). Both parts meet the hi/lo activation
// columns, so one step costs four MFMAs instead of two and no per-row scale remains.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kStepsPerBatch = 4;      // 16-row weight loads per lane and load batch
constexpr int kNumCu = 256;
constexpr int kMmTwoTileRows = 8192;   // panels at least this tall use two row tiles per wave
constexpr int kMmFourTileRows = 15360; // and four from here (240 tiles of 64 rows: every CU but 16 busy)
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
  uint32_t gs[RT];   // groupwise store: the BF16 scale of the row tile's 16 bytes
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t cvt_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// 8 signed INT8 weights (two words) times a group scale -> the exact products as BF16 hi and lo
__device__ __forceinline__ void widen_scaled(uint32_t w0, uint32_t w1, float sc, bf16x8& hi, bf16x8& lo) {
  const uint32_t w[2] = {w0, w1};
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float f0 = float(int8_t(w[i] & 0xffu)) * sc, f1 = float(int8_t((w[i] >> 8) & 0xffu)) * sc;
    const float f2 = float(int8_t((w[i] >> 16) & 0xffu)) * sc, f3 = float(int8_t(w[i] >> 24)) * sc;
    h[2 * i] = cvt_bf16x2(f0, f1);
    h[2 * i + 1] = cvt_bf16x2(f2, f3);
    l[2 * i] = cvt_bf16x2(f0 - bf16_lo(h[2 * i]), f1 - bf16_hi(h[2 * i]));
    l[2 * i + 1] = cvt_bf16x2(f2 - bf16_lo(h[2 * i + 1]), f3 - bf16_hi(h[2 * i + 1]));
  }
  hi = __builtin_bit_cast(bf16x8, make_int4(int(h[0]), int(h[1]), int(h[2]), int(h[3])));
  lo = __builtin_bit_cast(bf16x8, make_int4(int(l[0]), int(l[1]), int(l[2]), int(l[3])));
}

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
template <int MODE, int WAVES, int RT, bool SH>
__global__ __launch_bounds__(WAVES * kWave) void mfma_gemv_kernel(MfmaArgs a) {
  constexpr int kPF = kStepsPerBatch / RT;             // steps per load batch (two batches in flight)
  constexpr bool BF = (MODE == MM_LMHEAD);
  static_assert(!(SH && BF), "the LM head is dense BF16 in every store");
  extern __shared__ int cmap_s[];                      // groupwise store with a column map
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
  const uint32_t row_bytes = SH ? uint32_t(a.sv.ld) : uint32_t(a.ld) * esz;
  const uint32_t w_bytes = SH ? uint32_t(a.sv.store_rows) * row_bytes
                              : (GU ? a.w2_off + uint32_t(N) * row_bytes : uint32_t(N) * row_bytes);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(SH ? static_cast<const void*>(a.sv.w) : a.w, w_bytes);
  const __amdgpu_buffer_rsrc_t rw2 = make_rsrc(SH && GU ? a.sv.w2 : nullptr, SH && GU ? w_bytes : 0u);
  const uint32_t sgroups = SH ? uint32_t(a.sv.ld / 128) : 0u;
  const __amdgpu_buffer_rsrc_t rg1 = make_rsrc(SH ? a.sv.gs : nullptr, SH ? uint32_t(a.sv.store_rows) * sgroups * 2u : 0u);
  const __amdgpu_buffer_rsrc_t rg2 = make_rsrc(SH && GU ? a.sv.gs2 : nullptr,
                                               SH && GU ? uint32_t(a.sv.store_rows) * sgroups * 2u : 0u);
  const bool has_cols = SH && a.sv.cols != nullptr;
  if (has_cols) {                                       // column map of the plan's K range
    for (int i = tid; i < (K + 15) / 16; i += WAVES * kWave) cmap_s[i] = a.sv.cols[i];
    __syncthreads();
  }
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, uint32_t(2 * B) * uint32_t(a.ldx) * 2u);
  const uint32_t x_base = uint32_t(r) * uint32_t(a.ldx) * 2u;   // >= the record count when r >= 2B
  const int lane_k = q * (BF ? 8 : 16);                 // first k of the lane inside a step

  // row of this lane in row tile rt of a tile, and the byte offset of its panel
  // (gate/up with RT >= 2: row tiles 0 .. RT/2 - 1 hold the gate rows of the tile's channels,
  // RT/2 .. RT - 1 their up rows)
  auto lane_row = [&](int tile, int rt) {
    if (GU) return tile * RPT + (RT == 1 ? (r & 7) : 16 * (rt % (RT > 1 ? RT / 2 : 1)) + r);
    return tile * ROWS + 16 * rt + r;
  };
  // gate/up: whether the lane's rows of row tile rt are up rows, and their byte offset
  auto lane_up = [&](int rt) -> bool { return GU && (RT == 1 ? (r >= 8) : (rt >= RT / 2)); };
  auto lane_half = [&](int rt) -> uint32_t { return lane_up(rt) ? a.w2_off : 0u; };

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
    e.s1 = (BF || SH) ? 1.0f : __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs1, int(o4), 0, 0));
    e.s2 = (GU && !SH) ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs2, int(o4), 0, 0)) : 1.0f;
    e.res = resid_on ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                           rres, int(ok ? (uint32_t(e_b) * uint32_t(a.ldy) + uint32_t(row)) * 4u : kOOB), 0, 0))
                     : 0.0f;
    e.g = gam_on ? bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rgam, int(ok ? uint32_t(row) * 2u : kOOB), 0, 0))
                 : 0.0f;
  };

  EpiOps ops0{}, ops1{};
  // groupwise store: store row of this lane in each row tile of the current tile (row map loads
  // once per tile)
  int srow_tile = -1;
  int srow[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) srow[rt] = -1;
  auto issue = [&](int g, Frag<RT> (&f)[kPF]) {
    const int i = g / spw, jb = g - i * spw;
    const int tile = wg + i * grid;
    const bool ok_t = g < total;
    if (ok_t && jb == 0) {
      // select values, not references (a select of addresses puts both structs in memory)
      EpiOps e;
      load_ops(tile, e);
      const bool odd = (i & 1) != 0;
      ops1.s1 = odd ? e.s1 : ops1.s1; ops1.s2 = odd ? e.s2 : ops1.s2;
      ops1.res = odd ? e.res : ops1.res; ops1.g = odd ? e.g : ops1.g;
      ops0.s1 = odd ? ops0.s1 : e.s1; ops0.s2 = odd ? ops0.s2 : e.s2;
      ops0.res = odd ? ops0.res : e.res; ops0.g = odd ? ops0.g : e.g;
    }
    if (SH && ok_t && tile != srow_tile) {
      srow_tile = tile;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int row = lane_row(tile, rt);
        srow[rt] = row < N ? (a.sv.rows ? a.sv.rows[row] : row) : -1;
      }
    }
#pragma unroll
    for (int u = 0; u < kPF; ++u) {
      const int step = wave * spw + jb + u;
      const int k = step * KS + lane_k;
      const bool ok = ok_t && step < n_steps;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        if constexpr (SH) {
          const bool okr = ok && srow[rt] >= 0 && k < K;
          const int scol = okr ? (has_cols ? cmap_s[k >> 4] : k) : 0;
          const uint32_t wo = okr ? uint32_t(srow[rt]) * row_bytes + uint32_t(scol) : kOOB;
          const uint32_t so = okr ? (uint32_t(srow[rt]) * sgroups + uint32_t(scol) / 128u) * 2u : kOOB;
          if constexpr (GU) {
            // gate and up rows of one wave come from two store matrices: a resource must be
            // wave-uniform, so each lane loads from both with the other offset out of range
            // (no traffic) and keeps the union
            const bool up = lane_up(rt);
            const int4 g4 = buf_load16_stream(rw, up ? kOOB : wo);
            const int4 u4 = buf_load16_stream(rw2, up ? wo : kOOB);
            f[u].a[rt] = make_int4(g4.x | u4.x, g4.y | u4.y, g4.z | u4.z, g4.w | u4.w);
            f[u].gs[rt] = __builtin_amdgcn_raw_buffer_load_b16(rg1, int(up ? kOOB : so), 0, 0) |
                          __builtin_amdgcn_raw_buffer_load_b16(rg2, int(up ? so : kOOB), 0, 0);
          } else {
            f[u].a[rt] = buf_load16_stream(rw, wo);
            f[u].gs[rt] = __builtin_amdgcn_raw_buffer_load_b16(rg1, int(so), 0, 0);
          }
        } else {
          const int row = lane_row(tile, rt);
          const uint32_t wo = (ok && row < N && k < a.ld)
                                  ? lane_half(rt) + uint32_t(row) * row_bytes + uint32_t(k) * esz : kOOB;
          f[u].a[rt] = buf_load16_stream(rw, wo);
        }
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
        } else if constexpr (SH) {
          const float sc = bf16_to_f32(uint16_t(f[u].gs[rt]));
          bf16x8 h0, l0, h1, l1;
          widen_scaled(uint32_t(f[u].a[rt].x), uint32_t(f[u].a[rt].y), sc, h0, l0);
          widen_scaled(uint32_t(f[u].a[rt].z), uint32_t(f[u].a[rt].w), sc, h1, l1);
          const bf16x8 x0 = __builtin_bit_cast(bf16x8, f[u].x0), x1 = __builtin_bit_cast(bf16x8, f[u].x1);
          acc0[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(h0, x0, acc0[rt], 0, 0, 0);
          acc1[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(h1, x1, acc1[rt], 0, 0, 0);
          acc0[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(l0, x0, acc0[rt], 0, 0, 0);
          acc1[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(l1, x1, acc1[rt], 0, 0, 0);
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

template <int MODE, int WAVES, int RT, bool SH>
hipError_t launch_mm(const MfmaArgs& a, hipStream_t s) {
  const int rpt = (MODE == MM_GATEUP) ? 8 * RT : 16 * RT;
  const int tiles = (a.N + rpt - 1) / rpt;
  if (tiles == 0) return hipSuccess;
  // dynamic LDS: the column map of a groupwise-store projection
  const size_t lds = (SH && a.sv.cols) ? size_t((a.K + 15) / 16) * 4 : 0;
  // resident workgroups per CU at this kernel's register and LDS use, queried once
  static int per_cu = [] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, mfma_gemv_kernel<MODE, WAVES, RT, SH>,
                                                     WAVES * kWave, SH ? 8192 : 0) != hipSuccess || n < 1)
      n = 1;
    return n;
  }();
  const int grid = tiles < per_cu * kNumCu ? tiles : per_cu * kNumCu;
  hipLaunchKernelGGL((mfma_gemv_kernel<MODE, WAVES, RT, SH>), dim3(grid), dim3(WAVES * kWave), lds, s, a);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_mm_mode(const MfmaArgs& a, hipStream_t s) {
  // two row tiles per wave halve the activation reads per weight byte; panels with few rows
  // keep one so that every CU gets a tile, with more waves per tile so that enough loads fly
  const int rows = (MODE == MM_GATEUP) ? 2 * a.N : a.N;
  if constexpr (MODE != MM_LMHEAD) {
    if (a.sv.gs) {
      if (rows >= kMmTwoTileRows) return launch_mm<MODE, 4, 2, true>(a, s);
      return launch_mm<MODE, 8, 1, true>(a, s);
    }
  }
  // four row tiles for the tallest panels (the 8B gate/up at batch 8: 23.1 -> 22.1 us)
  if (MODE == MM_GATEUP && rows >= kMmFourTileRows) return launch_mm<MODE, 4, 4, false>(a, s);
  if (rows >= kMmTwoTileRows) return launch_mm<MODE, 4, 2, false>(a, s);
  return launch_mm<MODE, 8, 1, false>(a, s);
}

}  // namespace

hipError_t launch_mfma_gemv(MfmaMode mode, const MfmaArgs& a, hipStream_t s) {
  if (a.sv.gs) {
    // groupwise store: plan columns within the operand, store rows of 16-byte multiples in 128
    // column groups, a column map only for piece-aligned K, no LM head
    if (mode == MM_LMHEAD || a.B < 1 || a.B > 8 || a.K < 0 || a.K % 16 != 0 || a.ldx % 64 != 0 ||
        a.ldx < a.K || a.sv.ld % 128 != 0 || a.sv.store_rows < 1 ||
        (mode == MM_GATEUP && (!a.sv.w2 || !a.sv.gs2)))
      return hipErrorInvalidValue;
    if (size_t((a.K + 15) / 16) * 4 > 64 * 1024) return hipErrorInvalidValue;
  } else if (a.B < 1 || a.B > 8 || a.K < 0 || a.K > a.ld || a.ld % 16 != 0 || a.ldx % 64 != 0 ||
             a.ldx < a.K) {
    return hipErrorInvalidValue;
  }
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

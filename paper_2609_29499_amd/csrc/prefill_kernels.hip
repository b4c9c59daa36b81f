// Prefill projections on the matrix cores: C[t][n] = sum_k A[t][k] P[n][k] for the T tokens of a
// prompt chunk, with v_mfma_f32_16x16x32_bf16 and float32 accumulation.
//
// Operands. The activation A is carried as two BF16 planes, hi = bf16(v) and lo = bf16(v - hi),
// and every tile is multiplied twice (hi, then lo, into the same accumulator), so activations keep
// 16 significant bits; INT8 panel rows are widened exactly to BF16 while they are staged in LDS
// (the dense BF16 LM head is staged as is). The inverse RMS of an RMSNorm input is applied per
// token in the epilogue (W (c x) = c (W x)); the producer of an operand writes x * gamma and
// per-64-row sums of squares of x, which the consumer reduces once per workgroup.
//
// Tiling. A workgroup computes 128 tokens x 128 panel rows (gate/up: 64 channels, each wave's
// 64 rows being 32 gate rows and the 32 up rows of the same channels, so SwiGLU stays in
// registers). Four waves in a 2 x 2 arrangement own 64 x 64 each as 4 x 4 MFMA tiles. K advances
// in chunks of 32: the global loads of the next three chunks are in flight (in registers) while
// the current chunk's MFMAs run from LDS (double-buffered, one barrier per chunk). LDS rows hold
// one chunk (32 BF16) with their 16-byte quarters XOR-swizzled by row (bank-conflict free).
//
// Split K. Panels of d_model rows (QKV, O, down) give few tiles at prompt lengths of a few
// hundred tokens (256 at 512 tokens: one workgroup per CU, latency-bound K loops). Their K range
// is then split over blockIdx.z so that the launch holds about as many workgroups as the chip
// keeps resident; each split writes its scaled partial tile to a float32 buffer and a second
// kernel sums the splits in a fixed order and applies the epilogue (residual, next operand, sums
// of squares).
//
// Groupwise store (shared-store plans). Panel rows come from the store through the plan's row map
// (QKV, gate/up) and plan columns through its 16-column piece map (O, down; staged in LDS); each
// thread's 16 staged bytes lie in one piece, hence in one group of 128 columns with one BF16
// scale. The staged weight is the exact product q * s (7 + 8 significant bits) split into BF16 hi
// and lo planes (both exact), and a tile pair costs three MFMAs (a_hi w_hi, a_lo w_hi, a_hi w_lo;
// a_lo w_lo is below 2^-16 of the product) with no per-row scale left for the epilogue.
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kTMax = 128;             // tokens per workgroup tile (largest)
constexpr int kTN = 128;               // panel rows per workgroup tile
constexpr int kKC = 32;                // k per chunk
constexpr int kLdsRow = 32;            // BF16 per LDS row (one chunk of k)
constexpr int kSsqBlk = 64;            // rows per sum-of-squares partial
constexpr long kPfMinTiles = 384;      // fewer 128-token tiles than this: use 64-token tiles
constexpr int kMaxKSplit = 4;          // K splits per tile at most
constexpr int kMinSplitChunks = 8;     // k chunks per split at least
constexpr long kSplitRowCap = 2048;    // (tokens x splits) the partial buffer is sized for
constexpr int kNumCu = 256;

template <int TM, bool SH>
struct PfSmem {
  uint16_t a[2][2][TM * kLdsRow];      // [buffer][hi/lo][swizzled token row]
  uint16_t b[2][SH ? 2 : 1][kTN * kLdsRow];   // [buffer][hi/lo (store weights)][swizzled panel row]
  float rs[TM];                        // inverse RMS of the tile's tokens
};

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t cvt_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// 16 signed INT8 weights times their group scale -> the exact products as BF16 hi and lo parts
// (each as two 16-byte halves)
__device__ __forceinline__ void widen16_scaled(const int4& w, float sc, int4& hlo, int4& hhi,
                                               int4& llo, int4& lhi) {
  const uint32_t v[4] = {uint32_t(w.x), uint32_t(w.y), uint32_t(w.z), uint32_t(w.w)};
  uint32_t h[8], l[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float f0 = float(int8_t(v[i] & 0xffu)) * sc, f1 = float(int8_t((v[i] >> 8) & 0xffu)) * sc;
    const float f2 = float(int8_t((v[i] >> 16) & 0xffu)) * sc, f3 = float(int8_t(v[i] >> 24)) * sc;
    h[2 * i] = cvt_bf16x2(f0, f1);
    h[2 * i + 1] = cvt_bf16x2(f2, f3);
    l[2 * i] = cvt_bf16x2(f0 - bf16_lo(h[2 * i]), f1 - bf16_hi(h[2 * i]));
    l[2 * i + 1] = cvt_bf16x2(f2 - bf16_lo(h[2 * i + 1]), f3 - bf16_hi(h[2 * i + 1]));
  }
  hlo = make_int4(int(h[0]), int(h[1]), int(h[2]), int(h[3]));
  hhi = make_int4(int(h[4]), int(h[5]), int(h[6]), int(h[7]));
  llo = make_int4(int(l[0]), int(l[1]), int(l[2]), int(l[3]));
  lhi = make_int4(int(l[4]), int(l[5]), int(l[6]), int(l[7]));
}

// LDS offset (BF16 elements) of 16-byte quarter qu of LDS row `row`. Quarters are XOR-swizzled
// with bits 1-4 of the row: the 8 or 16 lanes served together by a 16-byte read (one fragment
// column: 16 consecutive rows, one quarter) or write (4 consecutive rows, all quarters) then
// touch distinct banks.
__device__ __forceinline__ int lds_q(int row, int qu) {
  return row * kLdsRow + 8 * (qu ^ (((row >> 1) ^ (row >> 3)) & 3));
}

__device__ __forceinline__ uint32_t pack_exact(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}

// 16 signed INT8 -> 16 BF16 (exact), as two 16-byte halves
__device__ __forceinline__ void widen16(const int4& w, int4& lo, int4& hi) {
  const uint32_t v[4] = {uint32_t(w.x), uint32_t(w.y), uint32_t(w.z), uint32_t(w.w)};
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = pack_exact(float(int8_t(v[i] & 0xffu)), float(int8_t((v[i] >> 8) & 0xffu)));
    o[2 * i + 1] = pack_exact(float(int8_t((v[i] >> 16) & 0xffu)), float(int8_t(v[i] >> 24)));
  }
  lo = make_int4(int(o[0]), int(o[1]), int(o[2]), int(o[3]));
  hi = make_int4(int(o[4]), int(o[5]), int(o[6]), int(o[7]));
}

__device__ __forceinline__ void store_hilo_pf(uint16_t* xo, size_t plane, int ld, int t, int col, float v) {
  const uint16_t hi = f32_to_bf16(v);
  xo[size_t(t) * ld + col] = hi;
  xo[plane + size_t(t) * ld + col] = f32_to_bf16(v - bf16_to_f32(hi));
}

// Epilogue of a prefill projection tile: lane (r, q) of wave (wm, wn) holds tokens 4q + i of each
// of its token tiles for panel row r of each row tile; rs = inverse RMS of the tile's tokens.
template <int MODE, int TM, bool SH>
__device__ __forceinline__ void pf_epilogue(const PfArgs& a, const f32x4 (&acc)[TM / 32][4],
                                            const float* rs, int m0, int n0, int bz, int wm, int wn,
                                            int q, int r) {
  constexpr bool BF = (MODE == MM_LMHEAD);
  constexpr bool GU = (MODE == MM_GATEUP);
  constexpr int MT = TM / 32;
  const int T = a.T, N = a.N;
  if (!GU && !BF && a.part) {
    // split K: this split's scaled partial; the reduction adds the splits and the epilogue
    float* part = a.part + size_t(bz) * T * N;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int tl = wm * (TM / 2) + mt * 16 + 4 * q + i;
        const int t = m0 + tl;
        if (t >= T) continue;
        const float rb = a.ssq ? rs[tl] : 1.0f;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
          const int n = n0 + wn * 64 + nt * 16 + r;
          if (n < N) part[size_t(t) * N + n] = acc[mt][nt][i] * (SH ? 1.0f : a.scale[n]) * rb;
        }
      }
    return;
  }
  const bool resid_on = (MODE == MM_RESID);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tl = wm * (TM / 2) + mt * 16 + 4 * q + i;
      const int t = m0 + tl;
      const bool t_ok = t < T;
      const float rb = a.ssq ? rs[tl] : 1.0f;
      if (GU) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int ch = n0 + 32 * wn + 16 * nt + r;
          if (t_ok && ch < N) {
            const float gv = acc[mt][nt][i] * (SH ? 1.0f : a.scale[ch]) * rb;
            const float uv = acc[mt][nt + 2][i] * (SH ? 1.0f : a.scale2[ch]) * rb;
            store_hilo_pf(a.xo, a.plane_o, a.ldxo, t, ch, gv / (1.0f + exp2f(-gv * kLog2e)) * uv);
          }
        }
        continue;
      }
      float ss = 0.0f;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int n = n0 + wn * 64 + nt * 16 + r;
        const bool ok = t_ok && n < N;
        float v = 0.0f;
        if (MODE == MM_LMHEAD) {
          v = acc[mt][nt][i] * rb;
        } else if (resid_on) {
          v = ok ? a.resid[size_t(t) * a.ldy + n] + acc[mt][nt][i] * (SH ? 1.0f : a.scale[n]) : 0.0f;
          if (ok && a.gamma_next) store_hilo_pf(a.xo, a.plane_o, a.ldxo, t, n, v * bf16_to_f32(a.gamma_next[n]));
          ss = fmaf(v, v, ss);
        } else {
          v = ok ? acc[mt][nt][i] * (SH ? 1.0f : a.scale[n]) * rb : 0.0f;
        }
        if (ok) a.y[size_t(t) * a.ldy + n] = v;
      }
      if (resid_on && a.gamma_next) {
        ss = row16_sum(ss);                             // the 16 lanes of this token
        if (r == 0 && t_ok && n0 + wn * 64 < N) a.ssq_out[size_t(t) * a.n_ssq_out + (n0 + wn * 64) / kSsqBlk] = ss;
      }
    }
  }
}

template <int MODE, int TM, bool SH>
__global__ __launch_bounds__(kBlock) void pf_gemm_kernel(PfArgs a) {
  constexpr bool BF = (MODE == MM_LMHEAD);
  constexpr bool GU = (MODE == MM_GATEUP);
  static_assert(!(SH && BF), "the LM head is dense BF16 in every store");
  constexpr int MT = TM / 32;                           // token tiles of 16 per wave
  constexpr int APT = TM / 32;                          // A pieces per thread and chunk
  __shared__ __attribute__((aligned(16))) PfSmem<TM, SH> sm;
  extern __shared__ int cmap_s[];                       // groupwise store: column map of K

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int T = a.T, N = a.N, K = a.K;
  const int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  const int m0 = by * TM;
  const int n0 = bx * (GU ? kTN / 2 : kTN);           // first row (gate/up: first channel)
  // this workgroup's k chunks: split bz of gridDim.z
  const int nk_all = (K + kKC - 1) / kKC;
  const int kc0 = int((long(bz) * nk_all) / gridDim.z);
  const int nk = int((long(bz + 1) * nk_all) / gridDim.z) - kc0;

  // ---- global -> register staging of one chunk
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(a.x, uint32_t(2 * a.plane) * 2u);
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
  // groupwise store: store row of this thread's staged panel row (fixed for the workgroup)
  int srow = -1;
  bool srow_up = false;
  // A pieces: thread t loads pieces t + 256 i (i < APT): plane, token row, 16-byte quarter
  auto a_off = [&](int i, int k0) -> uint32_t {
    const int p = tid + kBlock * i;
    const int plane = p / (4 * TM), row = (p >> 2) & (TM - 1), qu = p & 3;
    const int t = m0 + row;
    const int k = k0 + 8 * qu;
    return (t < T && k < a.ldx) ? uint32_t(plane) * uint32_t(a.plane) * 2u + (uint32_t(t) * uint32_t(a.ldx) + uint32_t(k)) * 2u
                                : kOOB;
  };
  // B rows of this thread: INT8 row t / 2, half t % 2 (16 bytes); BF16 rows p / 4, quarter p % 4
  auto w_row = [&](int lr) -> int {                     // panel row of LDS row lr
    if (!GU) return n0 + lr;
    return n0 + 32 * (lr >> 6) + (lr & 31);             // channel
  };
  auto w_off = [&](int lr, int kbyte) -> uint32_t {
    const int row = w_row(lr);
    const bool up = GU && ((lr & 63) >= 32);
    const bool ok = (GU ? row < N : row < N) && kbyte < int(row_bytes);
    return ok ? (up ? a.w2_off : 0u) + uint32_t(row) * row_bytes + uint32_t(kbyte) : kOOB;
  };
  struct Stage {
    int4 av[APT];
    int4 bv[2];
    uint32_t gs;                                        // groupwise store: scale of bv[0]
  };
  auto load = [&](int kc, Stage& st) {
    const int k0 = (kc0 + kc) * kKC;
#pragma unroll
    for (int i = 0; i < APT; ++i) st.av[i] = buf_load16(ra, kc < nk ? a_off(i, k0) : kOOB);
    if (BF) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int p = tid + kBlock * i;
        st.bv[i] = buf_load16(rw, kc < nk ? w_off(p >> 2, (k0 + 8 * (p & 3)) * 2) : kOOB);
      }
    } else if constexpr (SH) {
      const int k = k0 + 16 * (tid & 1);
      const bool ok = kc < nk && srow >= 0 && k < K;
      const int scol = ok ? (has_cols ? cmap_s[k >> 4] : k) : 0;
      const uint32_t wo = ok ? uint32_t(srow) * row_bytes + uint32_t(scol) : kOOB;
      const uint32_t so = ok ? (uint32_t(srow) * sgroups + uint32_t(scol) / 128u) * 2u : kOOB;
      if constexpr (GU) {
        // gate and up rows come from two store matrices (resources must be wave-uniform): load
        // from both, the other offset out of range, and keep the union
        const int4 g4 = buf_load16(rw, srow_up ? kOOB : wo);
        const int4 u4 = buf_load16(rw2, srow_up ? wo : kOOB);
        st.bv[0] = make_int4(g4.x | u4.x, g4.y | u4.y, g4.z | u4.z, g4.w | u4.w);
        st.gs = __builtin_amdgcn_raw_buffer_load_b16(rg1, int(srow_up ? kOOB : so), 0, 0) |
                __builtin_amdgcn_raw_buffer_load_b16(rg2, int(srow_up ? so : kOOB), 0, 0);
      } else {
        st.bv[0] = buf_load16(rw, wo);
        st.gs = __builtin_amdgcn_raw_buffer_load_b16(rg1, int(so), 0, 0);
      }
    } else {
      st.bv[0] = buf_load16(rw, kc < nk ? w_off(tid >> 1, k0 + 16 * (tid & 1)) : kOOB);
    }
  };
  auto commit = [&](int buf, const Stage& st) {
#pragma unroll
    for (int i = 0; i < APT; ++i) {
      const int p = tid + kBlock * i;
      const int plane = p / (4 * TM), row = (p >> 2) & (TM - 1), qu = p & 3;
      *reinterpret_cast<int4*>(&sm.a[buf][plane][lds_q(row, qu)]) = st.av[i];
    }
    if (BF) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int p = tid + kBlock * i;
        *reinterpret_cast<int4*>(&sm.b[buf][0][lds_q(p >> 2, p & 3)]) = st.bv[i];
      }
    } else if constexpr (SH) {
      int4 hlo, hhi, llo, lhi;
      widen16_scaled(st.bv[0], bf16_to_f32(uint16_t(st.gs)), hlo, hhi, llo, lhi);
      const int row = tid >> 1, h = tid & 1;
      *reinterpret_cast<int4*>(&sm.b[buf][0][lds_q(row, 2 * h)]) = hlo;
      *reinterpret_cast<int4*>(&sm.b[buf][0][lds_q(row, 2 * h + 1)]) = hhi;
      *reinterpret_cast<int4*>(&sm.b[buf][1][lds_q(row, 2 * h)]) = llo;
      *reinterpret_cast<int4*>(&sm.b[buf][1][lds_q(row, 2 * h + 1)]) = lhi;
    } else {
      int4 lo, hi;
      widen16(st.bv[0], lo, hi);
      const int row = tid >> 1, h = tid & 1;
      *reinterpret_cast<int4*>(&sm.b[buf][0][lds_q(row, 2 * h)]) = lo;
      *reinterpret_cast<int4*>(&sm.b[buf][0][lds_q(row, 2 * h + 1)]) = hi;
    }
  };

  if constexpr (SH) {
    const int lr = tid >> 1, row = w_row(lr);
    srow_up = GU && ((lr & 63) >= 32);
    srow = row < N ? (a.sv.rows ? a.sv.rows[row] : row) : -1;
    if (has_cols) {                                     // column map of the plan's K range
      for (int i = tid; i < (K + 15) / 16; i += kBlock) cmap_s[i] = a.sv.cols[i];
      __syncthreads();
    }
  }

  // three chunks in flight in registers: chunk c is loaded while chunk c - 3 is computed and
  // committed to LDS after chunk c - 1 has been computed
  Stage s0, s1, s2;
  load(0, s0);
  load(1, s1);
  load(2, s2);

  // ---- inverse RMS of the tile's tokens (RMSNorm inputs): thread t sums half of token t / 2
  if (a.ssq) {
    const int row = tid >> 1, half = tid & 1, t = m0 + row;
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(a.ssq, uint32_t(T) * uint32_t(a.n_ssq) * 4u);
    float v = 0.0f;
    for (int j0 = 0; j0 < a.n_ssq; j0 += 16) {
      float tv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + 2 * u + half;
        tv[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                              rq, int((t < T && j < a.n_ssq) ? (uint32_t(t) * uint32_t(a.n_ssq) + uint32_t(j)) * 4u : kOOB), 0, 0));
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) v += tv[u];
    }
    v += __shfl_xor(v, 1, kWave);
    if (half == 0) sm.rs[row] = rsqrtf(v * a.inv_d + a.eps);
  }

  commit(0, s0);
  __syncthreads();

  f32x4 acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto step = [&](int kc, Stage& mine, const Stage& next) {
    const int buf = kc & 1;
    load(kc + 3, mine);                                 // chunk kc was committed already
    bf16x8 bw[4], bl[SH ? 4 : 1];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      bw[nt] = *reinterpret_cast<const bf16x8*>(&sm.b[buf][0][lds_q(wn * 64 + nt * 16 + r, q)]);
      if constexpr (SH) bl[nt] = *reinterpret_cast<const bf16x8*>(&sm.b[buf][1][lds_q(wn * 64 + nt * 16 + r, q)]);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int ar = lds_q(wm * (TM / 2) + mt * 16 + r, q);
      const bf16x8 ahi = *reinterpret_cast<const bf16x8*>(&sm.a[buf][0][ar]);
      const bf16x8 alo = *reinterpret_cast<const bf16x8*>(&sm.a[buf][1][ar]);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bw[nt], acc[mt][nt], 0, 0, 0);
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bw[nt], acc[mt][nt], 0, 0, 0);
        if constexpr (SH) acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bl[nt], acc[mt][nt], 0, 0, 0);
      }
    }
    if (kc + 1 < nk) commit(buf ^ 1, next);
    __syncthreads();
  };
  for (int kc = 0; kc < nk; kc += 3) {
    step(kc, s0, s1);
    if (kc + 1 < nk) step(kc + 1, s1, s2);
    if (kc + 2 < nk) step(kc + 2, s2, s0);
  }

  pf_epilogue<MODE, TM, SH>(a, acc, sm.rs, m0, n0, bz, wm, wn, q, r);
}

// ---- per-row INT8 panels: operands copied straight from memory into LDS
//
// The activation planes and the INT8 panel rows go from memory to LDS by buffer loads with an LDS
// destination (no register staging, no LDS store instructions), through four stages, so that
// the loads of the next three chunks are in flight while a chunk is multiplied; one barrier
// per chunk. INT8 panel bytes stay INT8 in LDS (half the LDS traffic of BF16) and each wave widens
// its 8-byte fragments exactly to BF16 before the MFMAs. An LDS-destination load writes lane l's
// 16 bytes at l * 16 from the wave's base, so the bank swizzle is applied on the memory side: the
// lane that fills LDS slot s of a row fetches the row's 16-byte piece s ^ swizzle(row). Used
// when K is a whole number of chunks, so that no load crosses the end of a panel row.

template <int TM>
struct PfDmaStage {
  uint16_t a[2][TM * kLdsRow];         // [hi/lo][token row x 32 BF16], quarters swizzled
  uint8_t b[kTN * kKC];                // [panel row x 32 INT8], 16-byte halves swizzled
};

// slot of quarter qu (16 bytes) of A row `row` (the 8 lanes served together by a 16-byte read,
// 8 consecutive rows of one quarter, hit distinct banks), and of half h of B row `row` (an
// 8-byte read of 16 consecutive rows meets each bank at most twice, the least for 8-byte reads
// of one word position)
__device__ __forceinline__ int dma_a_q(int row, int qu) { return qu ^ (((row >> 1) ^ (row >> 3)) & 3); }
__device__ __forceinline__ int dma_b_h(int row, int h) { return h ^ ((row >> 3) & 1); }

// s_waitcnt: vector memory count <= n, the other counters not waited on
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// 8 signed INT8 (two words) -> 8 BF16 (exact)
__device__ __forceinline__ bf16x8 widen8(uint32_t w0, uint32_t w1) {
  const uint32_t v[2] = {w0, w1};
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    o[2 * i] = pack_exact(float(int8_t(v[i] & 0xffu)), float(int8_t((v[i] >> 8) & 0xffu)));
    o[2 * i + 1] = pack_exact(float(int8_t((v[i] >> 16) & 0xffu)), float(int8_t(v[i] >> 24)));
  }
  return __builtin_bit_cast(bf16x8, make_int4(int(o[0]), int(o[1]), int(o[2]), int(o[3])));
}

template <int MODE, int TM>
__global__ __launch_bounds__(kBlock) void pf_dma_kernel(PfArgs a) {
  constexpr bool GU = (MODE == MM_GATEUP);
  constexpr int MT = TM / 32;                           // token tiles of 16 per wave
  constexpr int A_PER_WAVE = TM / 32;                   // A loads (16 rows x 64 B) per wave and chunk
  constexpr int PER_CHUNK = A_PER_WAVE + 1;             // + one B load (32 rows x 32 B)
  static_assert(MODE == MM_QKV || MODE == MM_RESID || MODE == MM_GATEUP, "INT8 projections");
  __shared__ __attribute__((aligned(16))) PfDmaStage<TM> st0;
  __shared__ __attribute__((aligned(16))) PfDmaStage<TM> st1;
  __shared__ __attribute__((aligned(16))) PfDmaStage<TM> st2;
  __shared__ __attribute__((aligned(16))) PfDmaStage<TM> st3;
  // the inverse RMS of the tile's tokens goes to LDS after the last chunk, over stage 0
  float* rs = reinterpret_cast<float*>(&st0);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int wm = wave >> 1, wn = wave & 1;
  const int T = a.T, N = a.N;
  const int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
  const int m0 = by * TM;
  const int n0 = bx * (GU ? kTN / 2 : kTN);
  const int nk_all = (a.K + kKC - 1) / kKC;
  const int kc0 = int((long(bz) * nk_all) / gridDim.z);
  const int nk = int((long(bz + 1) * nk_all) / gridDim.z) - kc0;

  const __amdgpu_buffer_rsrc_t ra = make_rsrc(a.x, uint32_t(2 * a.plane) * 2u);
  const uint32_t row_bytes = uint32_t(a.ld);
  const __amdgpu_buffer_rsrc_t rw =
      make_rsrc(a.w, GU ? a.w2_off + uint32_t(N) * row_bytes : uint32_t(N) * row_bytes);

  // this lane's share of a chunk's loads: A load j covers plane (i / (TM / 16)) rows
  // 16 (i % (TM / 16)) .. + 16 with i = wave + 4 j; the B load covers LDS rows 32 wave .. + 32
  uint32_t a_base[A_PER_WAVE];
  int a_lds[A_PER_WAVE];
#pragma unroll
  for (int j = 0; j < A_PER_WAVE; ++j) {
    const int i = wave + 4 * j;
    const int plane = i / (TM / 16), r0 = (i % (TM / 16)) * 16;
    const int row = r0 + (lane >> 2), t = m0 + row;
    const int k8 = 8 * dma_a_q(row, lane & 3);          // BF16 column of this lane's piece
    a_base[j] = t < T ? uint32_t(plane) * a.plane * 2u + (uint32_t(t) * uint32_t(a.ldx) + uint32_t(k8)) * 2u
                      : kOOB;
    a_lds[j] = plane * (TM * kLdsRow) + r0 * kLdsRow;   // wave-uniform (BF16 elements)
  }
  const int b_lr = 32 * wave + (lane >> 1);
  const int b_row = GU ? n0 + 32 * (b_lr >> 6) + (b_lr & 31) : n0 + b_lr;
  const bool b_up = GU && ((b_lr & 63) >= 32);
  const int b_k = 16 * dma_b_h(b_lr, lane & 1);
  const uint32_t b_base =
      b_row < N ? (b_up ? a.w2_off : 0u) + uint32_t(b_row) * row_bytes + uint32_t(b_k) : kOOB;

  auto issue = [&](int kc, PfDmaStage<TM>& S) {
    const int k0 = (kc0 + kc) * kKC;
#pragma unroll
    for (int j = 0; j < A_PER_WAVE; ++j) {
      // columns past ldx are beyond the plane row: never read (ldx is a multiple of 64)
      const uint32_t off = a_base[j] == kOOB ? kOOB : a_base[j] + uint32_t(k0) * 2u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, static_cast<void*>(&S.a[0][a_lds[j]]), 16, int(off), 0, 0, 0);
    }
    const uint32_t boff = (b_base == kOOB || k0 + b_k >= int(row_bytes)) ? kOOB : b_base + uint32_t(k0);
    // (the LDS operand is passed as void*: a typed pointer leaves the host stub of the kernel
    // unemitted)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, static_cast<void*>(&S.b[32 * wave * kKC]), 16, int(boff), 0, 0, 0);
  };

  // the inverse RMS loads go first, so that waiting for them does not wait for the chunks
  float rsv = 0.0f;
  {
    const int row = tid >> 1, half = tid & 1, t = m0 + row;
    if (a.ssq && row < TM) {
      const __amdgpu_buffer_rsrc_t rq = make_rsrc(a.ssq, uint32_t(T) * uint32_t(a.n_ssq) * 4u);
      for (int j0 = 0; j0 < a.n_ssq; j0 += 16) {
        float tv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + 2 * u + half;
          tv[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                rq, int((t < T && j < a.n_ssq) ? (uint32_t(t) * uint32_t(a.n_ssq) + uint32_t(j)) * 4u : kOOB), 0, 0));
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) rsv += tv[u];
      }
    }
  }
  if (nk > 0) issue(0, st0);
  if (nk > 1) issue(1, st1);
  if (nk > 2) issue(2, st2);
  if (a.ssq) {
    rsv += __shfl_xor(rsv, 1, kWave);
    rsv = rsqrtf(rsv * a.inv_d + a.eps);
  }

  f32x4 acc[MT][4];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  auto compute = [&](const PfDmaStage<TM>& S) {
    bf16x8 bw[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      const int lr = wn * 64 + nt * 16 + r;
      const uint2 w = *reinterpret_cast<const uint2*>(&S.b[lr * kKC + 16 * dma_b_h(lr, q >> 1) + 8 * (q & 1)]);
      bw[nt] = widen8(w.x, w.y);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int row = wm * (TM / 2) + mt * 16 + r;
      const int o = row * kLdsRow + 8 * dma_a_q(row, q);
      const bf16x8 ahi = *reinterpret_cast<const bf16x8*>(&S.a[0][o]);
      const bf16x8 alo = *reinterpret_cast<const bf16x8*>(&S.a[1][o]);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bw[nt], acc[mt][nt], 0, 0, 0);
        acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bw[nt], acc[mt][nt], 0, 0, 0);
      }
    }
  };
  // chunk kc sits in stage kc % 4: wait for this wave's loads of it (those of later chunks may
  // stay in flight), meet the other waves (their loads of it have landed, and all of them are
  // done with the stage loaded next), load chunk kc + 3 into the stage chunk kc - 1 used,
  // multiply chunk kc
  auto step = [&](int kc, const PfDmaStage<TM>& cur, PfDmaStage<TM>& nxt) {
    if (kc + 2 < nk) wait_vm<2 * PER_CHUNK>();
    else if (kc + 1 < nk) wait_vm<PER_CHUNK>();
    else wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    if (kc + 3 < nk) issue(kc + 3, nxt);
    compute(cur);
  };
  for (int kc = 0; kc < nk; kc += 4) {
    step(kc, st0, st3);
    if (kc + 1 < nk) step(kc + 1, st1, st0);
    if (kc + 2 < nk) step(kc + 2, st2, st1);
    if (kc + 3 < nk) step(kc + 3, st3, st2);
  }
  __syncthreads();                                      // every wave is done with the stages
  if (a.ssq && (tid & 1) == 0 && (tid >> 1) < TM) rs[tid >> 1] = rsv;
  __syncthreads();
  pf_epilogue<MODE, TM, false>(a, acc, rs, m0, n0, bz, wm, wn, q, r);
}

// First operand of a prefill: x * gamma as hi/lo planes and per-64-element sums of squares of x.
// Thread = four consecutive elements of token blockIdx.y; 16 lanes cover one 64-element block.
__global__ __launch_bounds__(kBlock) void pf_prep_kernel(const float* __restrict__ x, int D,
                                                         const uint16_t* __restrict__ gamma,
                                                         uint16_t* xo, size_t plane, int ldxo,
                                                         float* ssq, int n_ssq) {
  const int t = blockIdx.y, i0 = (blockIdx.x * kBlock + threadIdx.x) * 4;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + size_t(t) * D, uint32_t(D) * 4u);
  const float4 v = __builtin_bit_cast(float4, buf_load16(rx, i0 < D ? uint32_t(i0) * 4u : kOOB));
  float ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, v.w * v.w)));
  if (i0 < D) {
    const float e[4] = {v.x * bf16_to_f32(gamma[i0]), v.y * bf16_to_f32(gamma[i0 + 1]),
                        v.z * bf16_to_f32(gamma[i0 + 2]), v.w * bf16_to_f32(gamma[i0 + 3])};
    uint32_t hi[2], lo[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const uint16_t h0 = f32_to_bf16(e[2 * k]), h1 = f32_to_bf16(e[2 * k + 1]);
      hi[k] = uint32_t(h0) | (uint32_t(h1) << 16);
      lo[k] = uint32_t(f32_to_bf16(e[2 * k] - bf16_to_f32(h0))) |
              (uint32_t(f32_to_bf16(e[2 * k + 1] - bf16_to_f32(h1))) << 16);
    }
    uint16_t* row = xo + size_t(t) * ldxo + i0;          // 8-byte aligned: ldxo % 64 == 0
    *reinterpret_cast<uint2*>(row) = make_uint2(hi[0], hi[1]);
    *reinterpret_cast<uint2*>(row + plane) = make_uint2(lo[0], lo[1]);
  }
  ss = row16_sum(ss);
  if ((threadIdx.x & 15) == 0 && i0 < D) ssq[size_t(t) * n_ssq + i0 / kSsqBlk] = ss;
}

// Sum of the K splits of a prefill projection (in split order) and the projection's epilogue:
// MM_QKV stores the sum; MM_RESID adds the residual, stores the row and, with a next gain, writes
// the next operand's hi/lo planes and the per-64-row sums of squares. Thread = one (token, row);
// a wave covers 64 consecutive rows, i.e. one sum-of-squares block.
template <int MODE>
__global__ __launch_bounds__(kBlock) void pf_split_reduce_kernel(PfArgs a, int ks) {
  const int t = blockIdx.y, n = blockIdx.x * kBlock + threadIdx.x;
  const int T = a.T, N = a.N;
  const bool ok = n < N;
  float v = 0.0f;
  if (ok)
    for (int z = 0; z < ks; ++z) v += a.part[(size_t(z) * T + t) * N + n];
  if (MODE == MM_RESID) {
    if (ok) {
      v += a.resid[size_t(t) * a.ldy + n];
      a.y[size_t(t) * a.ldy + n] = v;
      if (a.gamma_next) store_hilo_pf(a.xo, a.plane_o, a.ldxo, t, n, v * bf16_to_f32(a.gamma_next[n]));
    }
    if (a.gamma_next) {
      const float ss = wave_sum(ok ? v * v : 0.0f);
      if ((threadIdx.x & 63) == 0 && ok) a.ssq_out[size_t(t) * a.n_ssq_out + n / kSsqBlk] = ss;
    }
  } else if (ok) {
    a.y[size_t(t) * a.ldy + n] = v;
  }
}

// RoPE of the T tokens' q and k at positions pos0 + t. q (scaled by log2(e) / sqrt(d_h)) goes to
// the attention operand as hi/lo planes [2][m_q][T][d_h]; k and v are rounded to BF16 and
// written to the cache rows pos0 + t of their retained groups. An item is four consecutive
// rotation pairs (q, k) or four consecutive v elements.
__device__ __forceinline__ void store_bf16x4(uint16_t* dst, const float (&v)[4]) {
  const uint32_t a = uint32_t(f32_to_bf16(v[0])) | (uint32_t(f32_to_bf16(v[1])) << 16);
  const uint32_t b = uint32_t(f32_to_bf16(v[2])) | (uint32_t(f32_to_bf16(v[3])) << 16);
  *reinterpret_cast<uint2*>(dst) = make_uint2(a, b);
}

__global__ __launch_bounds__(kBlock) void pf_rope_kernel(PfRopeArgs a) {
  const int t = blockIdx.x;
  const int dh = a.dh, half = dh / 2, h4 = half / 4;
  const float* row = a.qkv + size_t(t) * a.ld_qkv;
  const int pos = a.pos0 + t;
  const float* cs = a.rope_cos + size_t(pos) * half;
  const float* sn = a.rope_sin + size_t(pos) * half;
  const float qscale = kLog2e * rsqrtf(float(dh));
  const int nq = a.m_q * h4, nk = a.m_kv * h4, nv = a.m_kv * (dh / 4);
  for (int it = threadIdx.x; it < nq + nk + nv; it += kBlock) {
    if (it < nq + nk) {
      const bool is_q = it < nq;
      const int u = is_q ? it : it - nq;
      const int h = u / h4, i = 4 * (u % h4);
      const float* src = row + (is_q ? h * dh : (a.m_q + h) * dh);
      const float4 x1 = *reinterpret_cast<const float4*>(src + i);
      const float4 x2 = *reinterpret_cast<const float4*>(src + i + half);
      const float4 c = *reinterpret_cast<const float4*>(cs + i);
      const float4 sv = *reinterpret_cast<const float4*>(sn + i);
      const float sc = is_q ? qscale : 1.0f;
      const float y1[4] = {(x1.x * c.x - x2.x * sv.x) * sc, (x1.y * c.y - x2.y * sv.y) * sc,
                           (x1.z * c.z - x2.z * sv.z) * sc, (x1.w * c.w - x2.w * sv.w) * sc};
      const float y2[4] = {(x2.x * c.x + x1.x * sv.x) * sc, (x2.y * c.y + x1.y * sv.y) * sc,
                           (x2.z * c.z + x1.z * sv.z) * sc, (x2.w * c.w + x1.w * sv.w) * sc};
      if (is_q) {
        uint16_t* qo = a.q_out + (size_t(h) * a.T_ld + t) * dh;
        float l1[4], l2[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          l1[e] = y1[e] - bf16_to_f32(f32_to_bf16(y1[e]));
          l2[e] = y2[e] - bf16_to_f32(f32_to_bf16(y2[e]));
        }
        store_bf16x4(qo + i, y1);
        store_bf16x4(qo + i + half, y2);
        store_bf16x4(qo + a.q_plane + i, l1);
        store_bf16x4(qo + a.q_plane + i + half, l2);
      } else {
        uint16_t* kc = a.kc + (size_t(a.kv_idx[h]) * a.S + pos) * dh;
        store_bf16x4(kc + i, y1);
        store_bf16x4(kc + i + half, y2);
      }
    } else {
      const int u = it - nq - nk;
      const int j = u / (dh / 4), e = 4 * (u % (dh / 4));
      const float4 v = *reinterpret_cast<const float4*>(row + (a.m_q + a.m_kv + j) * dh + e);
      const float w[4] = {v.x, v.y, v.z, v.w};
      store_bf16x4(a.vc + (size_t(a.kv_idx[j]) * a.S + pos) * dh + e, w);
    }
  }
}

template <int MODE, int TM, bool SH>
int pf_resident() {
  static const int n = [] {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, pf_gemm_kernel<MODE, TM, SH>, kBlock,
                                                     SH ? 8192 : 0) != hipSuccess || per_cu < 1)
      per_cu = 1;
    return per_cu * kNumCu;
  }();
  return n;
}

template <int MODE, int TM>
int pf_dma_resident() {
  static const int n = [] {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, pf_dma_kernel<MODE, TM>, kBlock, 0) !=
            hipSuccess || per_cu < 1)
      per_cu = 1;
    return per_cu * kNumCu;
  }();
  return n;
}

template <int MODE, int TM, bool SH>
hipError_t launch_pf_tm(const PfArgs& a, hipStream_t s) {
  const int rows_per_tile = (MODE == MM_GATEUP) ? kTN / 2 : kTN;
  const int gx = (a.N + rows_per_tile - 1) / rows_per_tile, gy = (a.T + TM - 1) / TM;
  if (gx == 0 || gy == 0) return hipSuccess;
  // per-row INT8 panels with K in whole chunks take the LDS-destination kernel
  constexpr bool kDmaMode = !SH && (MODE == MM_QKV || MODE == MM_RESID || MODE == MM_GATEUP);
  const bool dma = kDmaMode && a.K % kKC == 0 && a.K > 0;
  // K splits: as many as keep every workgroup resident, at least kMinSplitChunks chunks each,
  // and no more than the partial buffer holds
  int ks = 1;
  if ((MODE == MM_QKV || MODE == MM_RESID) && a.part) {
    const long tiles = long(gx) * gy;
    const long per_split = long(a.T) * a.N;
    int resident = pf_resident<MODE, TM, SH>();
    if constexpr (kDmaMode) {
      if (dma) resident = pf_dma_resident<MODE, TM>();
    }
    ks = int(std::min<long>(kMaxKSplit, resident / tiles));
    ks = std::min(ks, ((a.K + kKC - 1) / kKC) / kMinSplitChunks);
    ks = int(std::min<long>(ks, per_split > 0 ? long(a.part_floats / size_t(per_split)) : 1));
    ks = std::max(ks, 1);
  }
  PfArgs b = a;
  if (ks == 1) b.part = nullptr;
  const size_t lds = (SH && a.sv.cols) ? size_t((a.K + 15) / 16) * 4 : 0;
  bool launched = false;
  if constexpr (kDmaMode) {
    if (dma) {
      hipLaunchKernelGGL((pf_dma_kernel<MODE, TM>), dim3(gx, gy, ks), dim3(kBlock), 0, s, b);
      launched = true;
    }
  }
  if (!launched)
    hipLaunchKernelGGL((pf_gemm_kernel<MODE, TM, SH>), dim3(gx, gy, ks), dim3(kBlock), lds, s, b);
  if (ks == 1) return hipGetLastError();
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((pf_split_reduce_kernel<MODE == MM_QKV ? MM_QKV : MM_RESID>),
                     dim3((a.N + kBlock - 1) / kBlock, a.T), dim3(kBlock), 0, s, b, ks);
  return hipGetLastError();
}

template <int MODE, bool SH>
hipError_t launch_pf_sh(const PfArgs& a, hipStream_t s) {
  // 128-token tiles halve the panel re-reads; smaller ones when that leaves CUs idle
  const int rows_per_tile = (MODE == MM_GATEUP) ? kTN / 2 : kTN;
  const long tiles = long((a.N + rows_per_tile - 1) / rows_per_tile) * ((a.T + kTMax - 1) / kTMax);
  if (tiles >= kPfMinTiles) return launch_pf_tm<MODE, kTMax, SH>(a, s);
  return launch_pf_tm<MODE, kTMax / 2, SH>(a, s);
}

template <int MODE>
hipError_t launch_pf(const PfArgs& a, hipStream_t s) {
  if constexpr (MODE != MM_LMHEAD) {
    if (a.sv.gs) return launch_pf_sh<MODE, true>(a, s);
  }
  return launch_pf_sh<MODE, false>(a, s);
}

}  // namespace

hipError_t launch_pf_gemm(MfmaMode mode, const PfArgs& a, hipStream_t s) {
  if (a.sv.gs) {
    // groupwise store: piece-aligned plan columns, 128-column scale groups, no LM head
    if (mode == MM_LMHEAD || a.T < 1 || a.K < 0 || a.K % 16 != 0 || a.ldx % 64 != 0 ||
        a.ldx < a.K || a.sv.ld % 128 != 0 || a.sv.store_rows < 1 ||
        (mode == MM_GATEUP && (!a.sv.w2 || !a.sv.gs2)) || size_t((a.K + 15) / 16) * 4 > 64 * 1024)
      return hipErrorInvalidValue;
  } else if (a.T < 1 || a.K < 0 || a.K > a.ld || a.ld % 16 != 0 || a.ldx % 64 != 0 || a.ldx < a.K) {
    return hipErrorInvalidValue;
  }
  switch (mode) {
    case MM_QKV: return launch_pf<MM_QKV>(a, s);
    case MM_RESID: return launch_pf<MM_RESID>(a, s);
    case MM_GATEUP: return launch_pf<MM_GATEUP>(a, s);
    case MM_LMHEAD: return launch_pf<MM_LMHEAD>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_pf_prep(const float* x, int D, int T, const uint16_t* gamma, uint16_t* xo,
                          size_t plane, int ldxo, float* ssq, hipStream_t s) {
  if (D % 16 != 0 || T < 1 || ldxo % 4 != 0 || plane % 4 != 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pf_prep_kernel, dim3((D + 4 * kBlock - 1) / (4 * kBlock), T), dim3(kBlock), 0, s, x, D,
                     gamma, xo, plane, ldxo, ssq, (D + kSsqBlk - 1) / kSsqBlk);
  return hipGetLastError();
}

hipError_t launch_pf_rope(const PfRopeArgs& a, hipStream_t s) {
  if (a.T < 1) return hipSuccess;
  hipLaunchKernelGGL(pf_rope_kernel, dim3(a.T), dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

int pf_ssq_block() { return kSsqBlk; }

size_t pf_split_buffer_floats(int max_prefill, int n_max) {
  // splits pay while the tiles leave CUs idle, i.e. up to a few hundred tokens; past the cap the
  // launch takes fewer splits
  const long rows = std::min<long>(long(kMaxKSplit) * std::max(max_prefill, 0), kSplitRowCap);
  return size_t(rows) * size_t(std::max(n_max, 0));
}

}  // namespace tasp

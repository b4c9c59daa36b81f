// Decode attention over the retained KV groups only (grouped-query attention, one new token per
// sequence), on the matrix cores.
//
// Grid (n_split, m_kv, B): workgroup (s, j, b) serves retained group slot j of sequence b over
// cache rows [s*chunk, (s+1)*chunk), the last split over [s*chunk, pos + 1), for all of that
// group's retained query heads (1..8), so each K/V row is read from HBM once for every head that
// uses it. The slot -> group and slot -> head-range tables of the layer travel inside the kernel
// arguments, so the cache loads do not wait for an index load. Splits hold a multiple of 64 rows
// (attn_mfma_split for one sequence, attn_mfma_split_batched for a batch), at most 32 of them.
//
// The workgroup rotates its heads' raw q (RoPE at pos, table from the plan) into LDS, pre-scaled
// by log2(e)/sqrt(d_h) so the softmax works in base 2; the last split also rotates the new k and
// rounds k and v to BF16 (the values every later step reads) and appends them to the cache after
// its tile loads. Nothing inside a split waits on the other waves: wave w owns the 16-row tiles
// w, w + 4, ... of the split and keeps the K and V loads of its next two tiles in flight
// (branch-free buffer loads; rows outside the range use an out-of-range offset). Per tile:
//   * S = K Q^T on v_mfma_f32_16x16x32_bf16: the tile's K rows are the A operand straight from the
//     cache (lane (r, q) loads row r, dims 32 kk + 8 q .. + 8), the retained heads' rotated q the
//     B operand as a hi/lo BF16 pair, so lane (r, q) receives the scores of tile rows 4 q .. 4 q + 3
//     for head r. BF16 K is exact; only q's 16-bit hi/lo split rounds.
//   * Online softmax per head over the wave's rows (the running max is exchanged between the four
//     lanes of a head).
//   * O += P V on v_mfma_f32_16x16x16_bf16: the probabilities are already in the A-operand layout
//     (head r, rows 4 q .. 4 q + 3), split into hi/lo BF16; V is the B operand, which needs 4 rows
//     of one dimension per lane, so the tile's V goes through a per-wave LDS buffer holding
//     8-byte units (dimension, group of 4 rows), XOR-swizzled so that both the writes (8 dims of 4
//     rows per lane) and the reads (one unit per lane) meet at most 2 lanes per bank.
// The new token's row is in no tile: the last split folds it into its result after its tiles (one
// online-softmax step per head). The waves meet once, in LDS. When the range is split, each
// workgroup writes (max, sum, unnormalised output) per head with device-coherent stores, waits for
// them to complete and counts itself done on the (group slot, sequence) counter; the workgroup
// that brings the count to n_split reads every split's record back with device-coherent loads,
// merges them by log-sum-exp, writes o and resets the counter for the next launch. Nothing waits
// on another workgroup, and no L2 write-back is needed (an earlier version fenced every
// workgroup, which serialised on the write-backs; a second merge kernel cost a launch and a round
// trip through memory).
#include <algorithm>
#include <type_traits>
#include <utility>

#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

constexpr int kMaxHeads = 8;
constexpr int kNumCu = 256;
constexpr int kMfmaChunk = 64;         // rows per split of the matrix-core kernel: a multiple of this
constexpr int kMfmaTargetSplits = 32;  // split count beyond which its splits grow
constexpr int kMfmaMaxSplit = 32;      // its merge handles up to this many splits

__device__ __forceinline__ float4 rope4(const float4& a, const float4& b, const float4& c,
                                        const float4& s, bool first_half) {
  // first half: a cos - b sin (b = partner); second half: a cos + b sin
  const float sg = first_half ? -1.0f : 1.0f;
  return make_float4(fmaf(sg * b.x, s.x, a.x * c.x), fmaf(sg * b.y, s.y, a.y * c.y),
                     fmaf(sg * b.z, s.z, a.z * c.z), fmaf(sg * b.w, s.w, a.w * c.w));
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

template <int DH, int NHM>
struct AttnMfmaSmem {
  float q_s[NHM][DH];
  uint16_t knew_b[DH];                 // the new key and value, BF16 bits
  uint16_t vnew_b[DH];
  uint2 vt[4][DH * 4];                 // per wave: units (dim, row group of 4) of the tile's V
  float wm[4][NHM], wl[4][NHM];
  float wacc[4][NHM][DH];              // per wave: unnormalised outputs
  float mw[kMfmaMaxSplit][NHM];        // merge: per (split, head) weight
  float mlsum[NHM];                    // merge: per head, the weighted sum of the splits' sums
  float4 mpart[kBlock];                // merge: per-thread partial outputs
  int last;
};

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef short __attribute__((ext_vector_type(4))) s16x4_t;

// LDS unit of V element rows [4 g, 4 g + 4) of dimension dim (index into AttnMfmaSmem::vt[w])
__device__ __forceinline__ int vt_unit(int dim, int g) {
  return (dim * 4 + g) ^ (((dim >> 3) & 7) << 2);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// two floats -> packed BF16 (hardware round to nearest even), and the packed value back as floats
__device__ __forceinline__ uint32_t cvt_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}
// maximum over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four lanes of one MFMA output column)
__device__ __forceinline__ float col_max4(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
__device__ __forceinline__ float col_sum4(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}

template <int DH, int NH, int NHM>
__device__ __forceinline__ void attn_mfma_body(const AttnArgs& a, AttnMfmaSmem<DH, NHM>& sm, int s,
                                               int j, int b) {
  constexpr int NKC = DH / 32;         // k chunks of the score MFMAs
  constexpr int NDT = DH / 16;         // output dimension tiles
  constexpr int LPR = DH / 8;          // lanes per V row (16-byte loads)
  constexpr int RG = kWave / LPR;      // V row groups per wave
  constexpr int RPG = 16 / RG;         // rows of a tile per row group (4 at d_h 128, 2 at 64)
  constexpr int HALF = DH / 2;
  constexpr int Q4 = DH / 4;
  constexpr int PS = DH + 4;           // partial record: max, sum, pad, DH accumulators
  static_assert(NH <= NHM, "head count above the shared-memory bound");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, qq = lane >> 4;         // MFMA fragment coordinates
  const int c = lane % LPR, rg = lane / LPR;       // V: dims [8 c, 8 c + 8) of row group rg
  const int g = a.kv_idx[j];
  const int h0 = a.slot_start[j];
  const int t0 = s * a.chunk;
  const int t1 = (s == a.n_split - 1) ? a.pos + 1 : t0 + a.chunk;
  const bool has_new = (t1 == a.pos + 1);
  // the tiles cover the split's cache rows [t0, tr); the new row (pos) of the last split is
  // folded into its record after them, so that split runs as many tiles as the others
  const int tr = has_new ? a.pos : t1;
  const int n_tiles = (tr - t0 + 15) / 16;
  const float* qkv = a.qkv + size_t(b) * a.ld_qkv;
  const size_t row_base = (size_t(b) * a.Hkv + g) * a.S;
  uint16_t* kc = a.kc + row_base * DH;
  uint16_t* vc = a.vc + row_base * DH;
  // this group's cache rows 0..pos-1 (row pos comes from LDS)
  const uint32_t group_bytes = uint32_t(a.pos) * DH * 2u;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kc, group_bytes);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vc, group_bytes);

  // RoPE inputs first (from L2: the QKV projection just wrote them), so that waiting for them does
  // not wait for the cache rows: item (h, i4) rotates float4 i4 of the first half of head h (h ==
  // NH: the new key) with its partner in the second half; threads 192 .. 192 + DH/4 take the new
  // value. Every address is valid (indices clamped), so the loads need no branch.
  constexpr int H4 = HALF / 4;
  const int nitems = (NH + (has_new ? 1 : 0)) * H4;
  const bool rope_item = tid < nitems;
  const int rh = rope_item ? tid / H4 : 0, ri4 = rope_item ? tid % H4 : 0;
  const bool is_k = rope_item && rh == NH;
  const float4* src4 = reinterpret_cast<const float4*>(
      is_k ? qkv + size_t(a.m_q + j) * DH : qkv + size_t(h0 + min(rh, NH - 1)) * DH);
  const float4 x1 = src4[ri4], x2 = src4[ri4 + H4];
  const float4 cc = reinterpret_cast<const float4*>(a.rope_cos + size_t(a.pos) * HALF)[ri4];
  const float4 sn = reinterpret_cast<const float4*>(a.rope_sin + size_t(a.pos) * HALF)[ri4];
  const bool v_item = has_new && tid >= 192 && tid < 192 + Q4;
  const int vi4 = v_item ? tid - 192 : 0;
  const float4 vx = reinterpret_cast<const float4*>(qkv + size_t(a.m_q + a.m_kv + j) * DH)[vi4];

  // K (A-fragment layout) and V (row-group layout) of one tile; rows outside [t0, t1) and row
  // pos read as zeros through out-of-range offsets
  struct Tile {
    int4 k[NKC], v[RPG];
  };
  auto issue = [&](int ti, Tile& f) {
    const int tb = t0 + 16 * ti;
    const int tk = tb + r;
#pragma unroll
    for (int kk = 0; kk < NKC; ++kk)
      f.k[kk] = buf_load16_stream(rk, (ti < n_tiles && tk < tr)
                                          ? uint32_t(tk) * (DH * 2u) + uint32_t(32 * kk + 8 * qq) * 2u
                                          : kOOB);
#pragma unroll
    for (int u = 0; u < RPG; ++u) {
      const int tv = tb + rg * RPG + u;
      f.v[u] = buf_load16_stream(rv, (ti < n_tiles && tv < tr)
                                         ? uint32_t(tv) * (DH * 2u) + uint32_t(c) * 16u : kOOB);
    }
  };
  Tile fa, fb;
  issue(wave, fa);
  issue(wave + 4, fb);

  // RoPE of the queries (pre-scaled by log2(e)/sqrt(d_h)) into LDS; the new key and value, rounded
  // to BF16, into LDS (they reach the cache at the end: a global store issued before the tile
  // loads are consumed would hold up the waits for them, one in-order counter covering both)
  if (rope_item) {
    const float qscale = kLog2e * rsqrtf(float(DH));
    float4 y1 = rope4(x1, x2, cc, sn, true), y2 = rope4(x2, x1, cc, sn, false);
    if (!is_k) {
      y1.x *= qscale; y1.y *= qscale; y1.z *= qscale; y1.w *= qscale;
      y2.x *= qscale; y2.y *= qscale; y2.z *= qscale; y2.w *= qscale;
      reinterpret_cast<float4*>(sm.q_s[rh])[ri4] = y1;
      reinterpret_cast<float4*>(sm.q_s[rh])[ri4 + H4] = y2;
    } else {
      const float e1[4] = {y1.x, y1.y, y1.z, y1.w}, e2[4] = {y2.x, y2.y, y2.z, y2.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sm.knew_b[ri4 * 4 + e] = f32_to_bf16(e1[e]);
        sm.knew_b[HALF + ri4 * 4 + e] = f32_to_bf16(e2[e]);
      }
    }
  }
  if (v_item) {
    const float e[4] = {vx.x, vx.y, vx.z, vx.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) sm.vnew_b[vi4 * 4 + k] = f32_to_bf16(e[k]);
  }
  __syncthreads();

  // q fragments (B operand of the scores): column r = head r (zero for r >= NH), hi and lo parts
  bf16x8_t qh[NKC], ql[NKC];
  {
    const int hr = r < NH ? r : 0;
#pragma unroll
    for (int kk = 0; kk < NKC; ++kk) {
      uint32_t hi[4], lo[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v0 = r < NH ? sm.q_s[hr][32 * kk + 8 * qq + 2 * e] : 0.0f;
        const float v1 = r < NH ? sm.q_s[hr][32 * kk + 8 * qq + 2 * e + 1] : 0.0f;
        hi[e] = cvt_bf16x2(v0, v1);
        lo[e] = cvt_bf16x2(v0 - bf16_lo(hi[e]), v1 - bf16_hi(hi[e]));
      }
      qh[kk] = __builtin_bit_cast(bf16x8_t, make_int4(int(hi[0]), int(hi[1]), int(hi[2]), int(hi[3])));
      ql[kk] = __builtin_bit_cast(bf16x8_t, make_int4(int(lo[0]), int(lo[1]), int(lo[2]), int(lo[3])));
    }
  }

  float m_run = -INFINITY, l_run = 0.0f;          // head r; l_run sums this lane's rows only
  f32x4_t o[NDT];                                  // lane (r, q): heads 4 q + i, dim 16 d + r
#pragma unroll
  for (int d = 0; d < NDT; ++d) o[d] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  uint2* vt = sm.vt[wave];

  auto process = [&](const Tile& f, int ti) {
    const int tb = t0 + 16 * ti;
    // scores
    f32x4_t sc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kk = 0; kk < NKC; ++kk) {
      const bf16x8_t af = __builtin_bit_cast(bf16x8_t, f.k[kk]);
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, qh[kk], sc, 0, 0, 0);
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, ql[kk], sc, 0, 0, 0);
    }
    // V of the tile into the wave's transposition buffer: this lane's rows rg RPG + u, 8 dims
    {
      int4 vw[RPG];
#pragma unroll
      for (int u = 0; u < RPG; ++u) vw[u] = f.v[u];
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        const int dim = 8 * c + dd;
        const int comp = dd >> 1;
        // v_perm_b32 selectors: low halves of (lo word, hi word), or their high halves
        const uint32_t sel = (dd & 1) ? 0x07060302u : 0x05040100u;
        uint32_t wv[RPG];
#pragma unroll
        for (int u = 0; u < RPG; ++u)
          wv[u] = uint32_t(comp == 0 ? vw[u].x : comp == 1 ? vw[u].y : comp == 2 ? vw[u].z : vw[u].w);
        if constexpr (RPG == 4) {
          vt[vt_unit(dim, rg)] = make_uint2(__builtin_amdgcn_perm(wv[1], wv[0], sel),
                                            __builtin_amdgcn_perm(wv[3], wv[2], sel));
        } else {
          // d_h 64: rows 2 rg, 2 rg + 1 are the low or high half of unit (dim, rg / 2)
          reinterpret_cast<uint32_t*>(&vt[vt_unit(dim, rg >> 1)])[rg & 1] =
              __builtin_amdgcn_perm(wv[1], wv[0], sel);
        }
      }
    }
    // online softmax per head (column r)
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (tb + 4 * qq + i >= tr) sc[i] = -INFINITY;
      mx = fmaxf(mx, sc[i]);
    }
    mx = col_max4(mx);
    const float mn = fmaxf(m_run, mx);           // finite: row tb < tr is in the tile
    const float al = __builtin_amdgcn_exp2f(m_run - mn);
    float pr[4], ps = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pr[i] = __builtin_amdgcn_exp2f(sc[i] - mn);
      ps += pr[i];
    }
    l_run = fmaf(l_run, al, ps);
    m_run = mn;
    // P as the A operand (head r, rows 4 q .. 4 q + 3), hi and lo parts
    const uint32_t ah0 = cvt_bf16x2(pr[0], pr[1]), ah1 = cvt_bf16x2(pr[2], pr[3]);
    const uint32_t al0 = cvt_bf16x2(pr[0] - bf16_lo(ah0), pr[1] - bf16_hi(ah0));
    const uint32_t al1 = cvt_bf16x2(pr[2] - bf16_lo(ah1), pr[3] - bf16_hi(ah1));
    const s16x4_t pah = __builtin_bit_cast(s16x4_t, make_uint2(ah0, ah1));
    const s16x4_t pal = __builtin_bit_cast(s16x4_t, make_uint2(al0, al1));
    // rescale output rows 4 q + i (head 4 q + i, whose factor lane 4 q + i holds); a wave's first
    // tile starts from zero outputs
    if (ti != wave) {
      float ar[4];
      const float a0 = lane_value(al, 0), a1 = lane_value(al, 1), a2 = lane_value(al, 2), a3 = lane_value(al, 3);
      if constexpr (NH > 4) {
        const float a4 = lane_value(al, 4), a5 = lane_value(al, 5), a6 = lane_value(al, 6), a7 = lane_value(al, 7);
        ar[0] = qq ? a4 : a0; ar[1] = qq ? a5 : a1; ar[2] = qq ? a6 : a2; ar[3] = qq ? a7 : a3;
      } else {
        ar[0] = a0; ar[1] = a1; ar[2] = a2; ar[3] = a3;       // rows of qq > 0 are unused heads
      }
#pragma unroll
      for (int d = 0; d < NDT; ++d)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[d][i] *= ar[i];
    }
#pragma unroll
    for (int d = 0; d < NDT; ++d) {
      const s16x4_t vb = __builtin_bit_cast(s16x4_t, vt[vt_unit(16 * d + r, qq)]);
      o[d] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pah, vb, o[d], 0, 0, 0);
      o[d] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pal, vb, o[d], 0, 0, 0);
    }
  };
  for (int ti = wave; ti < n_tiles; ti += 8) {
    process(fa, ti);
    issue(ti + 8, fa);
    if (ti + 4 < n_tiles) process(fb, ti + 4);
    issue(ti + 12, fb);
  }

  // the new row goes to the cache now
  if (has_new && tid < DH / 8) {
    *reinterpret_cast<int4*>(kc + size_t(a.pos) * DH + 8 * tid) =
        *reinterpret_cast<const int4*>(&sm.knew_b[8 * tid]);
    *reinterpret_cast<int4*>(vc + size_t(a.pos) * DH + 8 * tid) =
        *reinterpret_cast<const int4*>(&sm.vnew_b[8 * tid]);
  }
  // the wave's running max and sum per head, and its unnormalised outputs, to LDS
  l_run = col_sum4(l_run);
  if (qq == 0 && r < NH) {
    sm.wm[wave][r] = m_run;
    sm.wl[wave][r] = l_run;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * qq + i;
    if (h < NH) {
#pragma unroll
      for (int d = 0; d < NDT; ++d) sm.wacc[wave][h][16 * d + r] = o[d][i];
    }
  }
  __syncthreads();

  // the workgroup's record: thread (h, e4) combines 4 dims of head h over the waves
  const int h = tid / Q4, e4 = tid % Q4;
  const bool item = tid < NH * Q4;
  float M = -INFINITY, L = 0.0f;
  float4 A = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (item) {
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, sm.wm[w][h]);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      // 0 for a wave without rows (and for every wave when the split has no cache rows)
      const float sw = (M == -INFINITY) ? 0.0f : exp2f(sm.wm[w][h] - M);
      L = fmaf(sm.wl[w][h], sw, L);
      const float4 v = reinterpret_cast<const float4*>(&sm.wacc[w][h][0])[e4];
      A.x = fmaf(v.x, sw, A.x); A.y = fmaf(v.y, sw, A.y);
      A.z = fmaf(v.z, sw, A.z); A.w = fmaf(v.w, sw, A.w);
    }
  }
  if (has_new) {
    // the new row: its score against head h (the pre-scaled q times the BF16 key, this thread's
    // 4 dims summed over the head's Q4 consecutive threads), then one online-softmax step
    float p = 0.0f;
    if (item) {
      const float4 qv = reinterpret_cast<const float4*>(sm.q_s[h])[e4];
      const uint2 kb = *reinterpret_cast<const uint2*>(&sm.knew_b[4 * e4]);
      p = fmaf(qv.x, bf16_lo(kb.x), fmaf(qv.y, bf16_hi(kb.x), fmaf(qv.z, bf16_lo(kb.y), qv.w * bf16_hi(kb.y))));
    }
#pragma unroll
    for (int off = 1; off < Q4; off <<= 1) p += __shfl_xor(p, off, kWave);
    if (item) {
      const uint2 vb = *reinterpret_cast<const uint2*>(&sm.vnew_b[4 * e4]);
      const float Mn = fmaxf(M, p);
      const float co = exp2f(M - Mn), cn = exp2f(p - Mn);     // co = 0 when M = -inf
      L = fmaf(L, co, cn);
      A.x = fmaf(A.x, co, cn * bf16_lo(vb.x)); A.y = fmaf(A.y, co, cn * bf16_hi(vb.x));
      A.z = fmaf(A.z, co, cn * bf16_lo(vb.y)); A.w = fmaf(A.w, co, cn * bf16_hi(vb.y));
      M = Mn;
    }
  }
  auto store4 = [&](const float4& v) {
    const int col = (h0 + h) * DH + 4 * e4;
    if (a.o_hl) {
      store_o(a, b, col + 0, v.x);
      store_o(a, b, col + 1, v.y);
      store_o(a, b, col + 2, v.z);
      store_o(a, b, col + 3, v.w);
    } else {
      *reinterpret_cast<float4*>(a.o + size_t(b) * a.ld_o + col) = v;
    }
  };
  if (a.n_split == 1) {
    if (item) {
      const float inv = 1.0f / L;
      store4(make_float4(A.x * inv, A.y * inv, A.z * inv, A.w * inv));
    }
    return;
  }
  // record per (split, head) = [max, sum, 0, 0, acc[DH]], written device-coherent; the last
  // split of (j, b) to finish merges them all
  const size_t rec0 = (size_t(b) * a.m_kv + j) * size_t(a.n_split) * kMaxHeads * PS;
  const __amdgpu_buffer_rsrc_t rp =
      make_rsrc(a.part + rec0, uint32_t(a.n_split) * kMaxHeads * PS * 4u);
  if (item) {
    buf_store16_device(__builtin_bit_cast(int4, A), rp,
                       uint32_t(((s * kMaxHeads + h) * PS + 4) * 4 + e4 * 16));
    if (e4 == 0)
      buf_store8_device(__builtin_bit_cast(int2, make_float2(M, L)), rp,
                        uint32_t((s * kMaxHeads + h) * PS * 4));
  }
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
  // merge (n_split <= kMfmaMaxSplit): (1) thread (head, split) reads that record's (max, sum); the
  // head's maximum M and the total of the sums weighted by exp2(max - M) are lane reductions, and
  // every split's weight goes to LDS; (2) thread (part, head, 4 dims) sums weighted accumulators
  // over splits part, part + NPARTS, ... with all of its record loads in flight at once; (3) the
  // parts are added and divided by the head's total.
  constexpr int ITEMS = NH * Q4;
  constexpr int NPARTS = ITEMS * 4 <= kBlock ? 4 : (ITEMS * 2 <= kBlock ? 2 : 1);
  constexpr int PER_PART = kMfmaMaxSplit / NPARTS;
  static_assert(kMfmaMaxSplit * NHM <= kBlock && kMfmaMaxSplit <= kWave &&
                    (kMfmaMaxSplit & (kMfmaMaxSplit - 1)) == 0,
                "one (max, sum) per thread, a head's records in one wave");
  const int part = tid / ITEMS, it = tid % ITEMS, mh = it / Q4, me4 = it % Q4;
  float4 av[PER_PART];
  {
    // every record load of the merge is issued before the first use of any of them; thread
    // (head mhl, split ms) = (tid / 32, tid % 32) takes that record's (max, sum), so each head's
    // records sit in 32 consecutive lanes and their maximum and weighted sum are lane reductions
    const int ms = tid & (kMfmaMaxSplit - 1), mhl = tid / kMfmaMaxSplit;
    const bool mi = ms < a.n_split && mhl < NH;
    const float2 ml = __builtin_bit_cast(
        float2, buf_load8_device(rp, mi ? uint32_t((ms * kMaxHeads + mhl) * PS * 4) : kOOB));
#pragma unroll
    for (int q = 0; q < PER_PART; ++q) {
      const int mq = part + NPARTS * q;
      av[q] = __builtin_bit_cast(
          float4, buf_load16_device(rp, (part < NPARTS && mq < a.n_split)
                                            ? uint32_t((mq * kMaxHeads + mh) * PS * 4 + 16 + me4 * 16)
                                            : kOOB));
    }
    float mm = mi ? ml.x : -INFINITY;
#pragma unroll
    for (int off = 1; off < kMfmaMaxSplit; off <<= 1) mm = fmaxf(mm, __shfl_xor(mm, off, kWave));
    const float w = mi ? exp2f(ml.x - mm) : 0.0f;        // every split has rows: mm is finite
    float lw = ml.y * w;
#pragma unroll
    for (int off = 1; off < kMfmaMaxSplit; off <<= 1) lw += __shfl_xor(lw, off, kWave);
    if (mi) sm.mw[ms][mhl] = w;
    if (ms == 0 && mhl < NH) sm.mlsum[mhl] = lw;
    __syncthreads();
  }
  if (part < NPARTS) {
    float4 acc4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
    for (int q = 0; q < PER_PART; ++q) {
      const int ms = part + NPARTS * q;
      const float w = ms < a.n_split ? sm.mw[ms][mh] : 0.0f;
      acc4.x = fmaf(av[q].x, w, acc4.x); acc4.y = fmaf(av[q].y, w, acc4.y);
      acc4.z = fmaf(av[q].z, w, acc4.z); acc4.w = fmaf(av[q].w, w, acc4.w);
    }
    sm.mpart[tid] = acc4;
  }
  __syncthreads();
  if (tid < ITEMS) {
    float4 v = sm.mpart[tid];
#pragma unroll
    for (int pp = 1; pp < NPARTS; ++pp) {
      const float4 u = sm.mpart[pp * ITEMS + tid];
      v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
    }
    const float inv = 1.0f / sm.mlsum[mh];
    store4(make_float4(v.x * inv, v.y * inv, v.z * inv, v.w * inv));   // h == mh, e4 == me4 here
  }
}

template <int DH, int NHM>
__global__ __launch_bounds__(kBlock) void attn_mfma_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) AttnMfmaSmem<DH, NHM> sm;
  const int s = blockIdx.x, j = blockIdx.y, b = blockIdx.z;
  const int nh = a.slot_start[j + 1] - a.slot_start[j];
  if constexpr (NHM == 1) {
    attn_mfma_body<DH, 1, NHM>(a, sm, s, j, b);
  } else if constexpr (NHM == 2) {
    if (nh == 1) attn_mfma_body<DH, 1, NHM>(a, sm, s, j, b);
    else attn_mfma_body<DH, 2, NHM>(a, sm, s, j, b);
  } else if constexpr (NHM == 4) {
    switch (nh) {
      case 1: attn_mfma_body<DH, 1, NHM>(a, sm, s, j, b); break;
      case 2: attn_mfma_body<DH, 2, NHM>(a, sm, s, j, b); break;
      case 3: attn_mfma_body<DH, 3, NHM>(a, sm, s, j, b); break;
      default: attn_mfma_body<DH, 4, NHM>(a, sm, s, j, b); break;
    }
  } else {
    switch (nh) {
      case 1: attn_mfma_body<DH, 1, NHM>(a, sm, s, j, b); break;
      case 2: attn_mfma_body<DH, 2, NHM>(a, sm, s, j, b); break;
      case 3: attn_mfma_body<DH, 3, NHM>(a, sm, s, j, b); break;
      case 4: attn_mfma_body<DH, 4, NHM>(a, sm, s, j, b); break;
      case 5: attn_mfma_body<DH, 5, NHM>(a, sm, s, j, b); break;
      case 6: attn_mfma_body<DH, 6, NHM>(a, sm, s, j, b); break;
      case 7: attn_mfma_body<DH, 7, NHM>(a, sm, s, j, b); break;
      default: attn_mfma_body<DH, 8, NHM>(a, sm, s, j, b); break;
    }
  }
}

}  // namespace

template <int DH>
hipError_t launch_mfma_dh(const AttnArgs& a, dim3 grid, int nhm, hipStream_t s) {
  if (nhm <= 1) hipLaunchKernelGGL((attn_mfma_kernel<DH, 1>), grid, dim3(kBlock), 0, s, a);
  else if (nhm == 2) hipLaunchKernelGGL((attn_mfma_kernel<DH, 2>), grid, dim3(kBlock), 0, s, a);
  else if (nhm <= 4) hipLaunchKernelGGL((attn_mfma_kernel<DH, 4>), grid, dim3(kBlock), 0, s, a);
  else hipLaunchKernelGGL((attn_mfma_kernel<DH, 8>), grid, dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t s) {
  if (a.m_kv == 0 || a.B == 0) return hipSuccess;
  if (a.dh != 64 && a.dh != 128) return hipErrorInvalidValue;
  // splits of chunk rows (a multiple of the 64-row tile group), the last one holding the
  // remainder up to pos (at least the new row), at most kMfmaMaxSplit records for the merge
  if (a.chunk < kMfmaChunk || a.chunk % kMfmaChunk != 0 || a.n_split < 1 ||
      a.n_split > kMfmaMaxSplit || long(a.n_split - 1) * a.chunk > a.pos)
    return hipErrorInvalidValue;
  int nhm = 0;
  for (int j = 0; j < a.m_kv; ++j) nhm = std::max(nhm, a.slot_start[j + 1] - a.slot_start[j]);
  if (nhm < 1 || nhm > kMaxHeads) return hipErrorInvalidValue;
  if (a.n_split > 1 && (!a.part || !a.cnt)) return hipErrorInvalidValue;
  const dim3 grid(a.n_split, a.m_kv, a.B);
  return (a.dh == 128) ? launch_mfma_dh<128>(a, grid, nhm, s) : launch_mfma_dh<64>(a, grid, nhm, s);
}

void attn_mfma_split(int total, int* chunk, int* n_split) {
  // the smallest multiple of 64 rows that keeps the split count at 32 or fewer, and at least 128
  // rows (two tiles per wave, the second's loads in flight during the first) once the context
  // holds 256; the remainder joins the last split. At 2048 positions 16 splits of 128 rows
  // measured faster than 32 of 64 (fewer records to merge), at 4096 positions 32 of 128 faster
  // than 16 or 22 longer ones.
  const int n64 = total / kMfmaChunk;
  if (n64 <= 1) {
    *chunk = kMfmaChunk;
    *n_split = 1;
    return;
  }
  int k = (n64 + kMfmaTargetSplits - 1) / kMfmaTargetSplits;
  if (k < 2 && n64 >= 4) k = 2;
  *chunk = kMfmaChunk * k;
  *n_split = std::max(1, total / *chunk);
}
void attn_mfma_split_batched(int total, int units, int* chunk, int* n_split) {
  // a batch: about one workgroup per CU over all (sequence, group slot) units. The cache rows
  // (total - 1; the new one is folded into the last split) are cut into splits of a multiple of
  // 64 rows, at least 128 once the context holds 256, the last one shorter. At 8 sequences of
  // 8192 positions: 4 splits of 2048 rows.
  const int cached = total - 1;
  const int n64 = total / kMfmaChunk;
  if (n64 <= 1 || units >= kNumCu) {
    attn_mfma_split(total, chunk, n_split);
    return;
  }
  const int target = std::max(1, std::min(kNumCu / std::max(units, 1), kMfmaTargetSplits));
  int rows = (cached + target - 1) / target;
  rows = (rows + kMfmaChunk - 1) / kMfmaChunk * kMfmaChunk;
  if (rows < 2 * kMfmaChunk && n64 >= 4) rows = 2 * kMfmaChunk;
  *chunk = rows;
  *n_split = std::max(1, (cached + rows - 1) / rows);
}
int attn_mfma_max_split(int max_seq) {
  // both rules split total <= max_seq rows into at most ceil(total / 64) and at most 32 splits
  return std::max(1, std::min((max_seq + kMfmaChunk - 1) / kMfmaChunk, kMfmaTargetSplits));
}
}  // namespace tasp

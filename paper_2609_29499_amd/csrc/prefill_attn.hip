// Causal prefill attention on the matrix cores, over the retained heads only.
//
// Grid (retained heads, query blocks of 64): workgroup (h, qb) serves queries 64 qb .. 64 qb + 63
// of retained head h, wave w the 16 queries 64 qb + 16 w + i. Query blocks are dealt last first
// (blockIdx.y = 0 is the last block): the longest rows of the causal triangle start first and
// the short ones fill in behind them. Cache rows 0 .. pos0 + last query of
// the block are walked in sub-blocks of 64, staged in LDS once per workgroup (K row-major, V
// transposed into units of 4 rows x 1 dimension), the next sub-block's rows loaded into registers
// while the current one is computed; one barrier per sub-block. Per 16-row tile:
//   * S^T = K Q^T on v_mfma_f32_16x16x32_bf16: K rows are the A operand, q (hi/lo BF16 planes, in
//     base-2 units: q carries log2(e) / sqrt(d_h)) the B operand, so lane (r, c) receives the
//     scores of query r against rows 4 c .. 4 c + 3 of the tile, which is exactly the A-operand
//     layout of v_mfma_f32_16x16x16_bf16: P never leaves the registers;
//   * causal mask, online softmax per query (the query's four lanes exchange maxima and sums by
//     lane permutes);
//   * O += P V on v_mfma_f32_16x16x16_bf16 with P split into hi/lo BF16 and V units read from LDS;
//     the output holds query 4 c + i in lane (r, c), so the per-query rescale factors move there
//     by a lane permute.
// The output O / l is written as the hi/lo operand of the O projection.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef short __attribute__((ext_vector_type(4))) s16x4;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

constexpr int kQB = 64;                // queries per workgroup (16 per wave)
constexpr int kKB = 64;                // cache rows per sub-block
constexpr int kVtRow = kKB + 4;        // BF16 per transposed-V row (8-byte pad)

template <int DH>
struct PaSmem {
  uint16_t k[2][kKB * (DH + 8)];       // [buffer][row][dim]
  uint16_t vt[2][DH * kVtRow];         // [buffer][dim][row]
};

__device__ __forceinline__ uint32_t cvt_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// reductions over the four lanes r, r + 16, r + 32, r + 48 (one query's lanes)
__device__ __forceinline__ float quad_max(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(q[0]), __uint_as_float(q[1]));
}
__device__ __forceinline__ float quad_sum(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(q[0]) + __uint_as_float(q[1]);
}
// value of lane `src` (wave-wide read)
__device__ __forceinline__ float lane_read(float v, int src) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(v)));
}

template <int DH>
__global__ __launch_bounds__(kBlock) void pf_attn_kernel(PfAttnArgs a) {
  constexpr int NKC = DH / 32;         // k chunks of the score MFMAs
  constexpr int NDT = DH / 16;         // output dimension tiles
  constexpr int KROW = DH + 8;
  constexpr int PPK = DH / 8;          // 16-byte pieces per cache row
  constexpr int STAGERS = 16 * PPK;    // threads staging a sub-block: 16 row quads x PPK pieces
  static_assert(STAGERS <= kBlock, "sub-block staging");
  __shared__ __attribute__((aligned(16))) PaSmem<DH> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, c = lane >> 4;
  const int h = blockIdx.x, qb = gridDim.y - 1 - blockIdx.y;
  int j = 0;                                            // group slot of head h
  while (j + 1 < a.m_kv && a.slot_start[j + 1] <= h) ++j;
  const int g = a.kv_idx[j];
  const int t_block = qb * kQB, t_first = t_block + 16 * wave;
  const int kv_end = a.pos0 + min(t_block + kQB, a.T);  // rows 0 .. kv_end - 1 are attended
  const int n_sb = (kv_end + kKB - 1) / kKB;
  const int wave_last = a.pos0 + min(t_first + 15, a.T - 1);   // last row this wave attends
  const uint16_t* kc = a.kc + size_t(g) * a.S * DH;
  const uint16_t* vc = a.vc + size_t(g) * a.S * DH;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kc, uint32_t(kv_end) * DH * 2u);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vc, uint32_t(kv_end) * DH * 2u);

  // q fragments (B operand): lane (r, c) holds query t_first + r, dimensions 32 kk + 8 c .. + 8
  bf16x8 qf[2][NKC];
  {
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(a.q, uint32_t(2 * a.q_plane) * 2u);
    const int t = t_first + r;
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int kk = 0; kk < NKC; ++kk) {
        const uint32_t off = t < a.T ? (uint32_t(pl) * uint32_t(a.q_plane) +
                                        (uint32_t(h) * uint32_t(a.T_ld) + uint32_t(t)) * DH + 32u * kk + 8u * c) * 2u
                                     : kOOB;
        qf[pl][kk] = __builtin_bit_cast(bf16x8, buf_load16(rq, off));
      }
  }
  f32x4 o[NDT];
#pragma unroll
  for (int d = 0; d < NDT; ++d) o[d] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float m_run = -INFINITY, l_run = 0.0f;                // of query t_first + r (lanes r + 16 c)
  const int qpos = a.pos0 + t_first + r;

  // staging: thread s < STAGERS holds rows 4 (s / PPK) .. + 3, piece s % PPK of K and of V
  const bool stager = tid < STAGERS;
  const int s_row = 4 * (tid / PPK), s_pc = tid % PPK;
  int4 pk[4], pv[4];
  auto load_sb = [&](int sb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = sb * kKB + s_row + i;
      const uint32_t off = (stager && t < kv_end) ? (uint32_t(t) * DH + 8u * s_pc) * 2u : kOOB;
      pk[i] = buf_load16(rk, off);
      pv[i] = buf_load16(rv, off);
    }
  };
  auto stage_sb = [&](int buf) {
    if (!stager) return;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<int4*>(&sm.k[buf][(s_row + i) * KROW + 8 * s_pc]) = pk[i];
    // V: 4 rows x 8 dimensions -> 8 units of (1 dimension, 4 rows)
    const uint32_t w[4][4] = {{uint32_t(pv[0].x), uint32_t(pv[0].y), uint32_t(pv[0].z), uint32_t(pv[0].w)},
                              {uint32_t(pv[1].x), uint32_t(pv[1].y), uint32_t(pv[1].z), uint32_t(pv[1].w)},
                              {uint32_t(pv[2].x), uint32_t(pv[2].y), uint32_t(pv[2].z), uint32_t(pv[2].w)},
                              {uint32_t(pv[3].x), uint32_t(pv[3].y), uint32_t(pv[3].z), uint32_t(pv[3].w)}};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint2 lo = make_uint2(__builtin_amdgcn_perm(w[1][e], w[0][e], 0x05040100u),
                                  __builtin_amdgcn_perm(w[3][e], w[2][e], 0x05040100u));
      const uint2 hi = make_uint2(__builtin_amdgcn_perm(w[1][e], w[0][e], 0x07060302u),
                                  __builtin_amdgcn_perm(w[3][e], w[2][e], 0x07060302u));
      *reinterpret_cast<uint2*>(&sm.vt[buf][(8 * s_pc + 2 * e) * kVtRow + s_row]) = lo;
      *reinterpret_cast<uint2*>(&sm.vt[buf][(8 * s_pc + 2 * e + 1) * kVtRow + s_row]) = hi;
    }
  };

  load_sb(0);
  for (int sb = 0; sb < n_sb; ++sb) {
    const int buf = sb & 1, tb = sb * kKB;
    stage_sb(buf);                                      // this buffer's readers finished at sb - 2
    if (sb + 1 < n_sb) load_sb(sb + 1);
    __syncthreads();
    if (tb > wave_last) continue;                       // every row of the sub-block is after the wave's queries
    // scores: tile ct, lane (r, c): query t_first + r, rows tb + 16 ct + 4 c + i
    f32x4 sc[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      sc[ct] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kk = 0; kk < NKC; ++kk) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&sm.k[buf][(16 * ct + r) * KROW + 32 * kk + 8 * c]);
        sc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[0][kk], sc[ct], 0, 0, 0);
        sc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[1][kk], sc[ct], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = tb + 16 * ct + 4 * c + i;
        sc[ct][i] = row > qpos ? -INFINITY : sc[ct][i];
        mx = fmaxf(mx, sc[ct][i]);
      }
    mx = quad_max(mx);
    const float mn = fmaxf(m_run, mx);
    const float base = mn == -INFINITY ? 0.0f : mn;     // a query with no row yet stays empty
    float ps = 0.0f;
    s16x4 ph[4], pl[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      float pv4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pv4[i] = __builtin_amdgcn_exp2f(sc[ct][i] - base);
        ps += pv4[i];
      }
      const uint32_t h0 = cvt_bf16x2(pv4[0], pv4[1]), h1 = cvt_bf16x2(pv4[2], pv4[3]);
      const uint32_t l0 = cvt_bf16x2(pv4[0] - bf16_lo(h0), pv4[1] - bf16_hi(h0));
      const uint32_t l1 = cvt_bf16x2(pv4[2] - bf16_lo(h1), pv4[3] - bf16_hi(h1));
      ph[ct] = __builtin_bit_cast(s16x4, make_uint2(h0, h1));
      pl[ct] = __builtin_bit_cast(s16x4, make_uint2(l0, l1));
    }
    ps = quad_sum(ps);
    const float alpha = __builtin_amdgcn_exp2f(m_run - base);   // 0 while m_run is -inf
    l_run = l_run * alpha + ps;
    m_run = mn;
    // the output rows of lane (r, c) are queries 4 c + i: their factors sit in lanes 4 c + i
    float al[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) al[i] = lane_read(alpha, 4 * c + i);
#pragma unroll
    for (int d = 0; d < NDT; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) o[d][i] *= al[i];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int d = 0; d < NDT; ++d) {
        const s16x4 vb = __builtin_bit_cast(
            s16x4, *reinterpret_cast<const uint2*>(&sm.vt[buf][(16 * d + r) * kVtRow + 16 * ct + 4 * c]));
        o[d] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ph[ct], vb, o[d], 0, 0, 0);
        o[d] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pl[ct], vb, o[d], 0, 0, 0);
      }
  }

  // O / l as the hi/lo operand of the O projection: lane (r, c) holds queries t_first + 4 c + i,
  // dimensions 16 d + r
  float inv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) inv[i] = 1.0f / lane_read(l_run, 4 * c + i);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int t = t_first + 4 * c + i;
    if (t >= a.T) continue;
#pragma unroll
    for (int d = 0; d < NDT; ++d) {
      const float v = o[d][i] * inv[i];
      const uint16_t hi = f32_to_bf16(v);
      const size_t at = size_t(t) * a.ldo + size_t(h) * DH + 16 * d + r;
      a.o[at] = hi;
      a.o[a.o_plane + at] = f32_to_bf16(v - bf16_to_f32(hi));
    }
  }
}

}  // namespace

hipError_t launch_pf_attn(const PfAttnArgs& a, hipStream_t s) {
  if (a.m_kv == 0 || a.T < 1) return hipSuccess;
  const int m_q = a.slot_start[a.m_kv];
  if (m_q < 1 || a.m_kv > 64) return hipErrorInvalidValue;
  const dim3 grid(m_q, (a.T + kQB - 1) / kQB);
  if (a.dh == 128) hipLaunchKernelGGL((pf_attn_kernel<128>), grid, dim3(kBlock), 0, s, a);
  else if (a.dh == 64) hipLaunchKernelGGL((pf_attn_kernel<64>), grid, dim3(kBlock), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tasp

// Causal prefill attention on the matrix cores, over the retained heads only.
//
// Grid (retained heads, work units): a unit serves queries 64 qb .. 64 qb + 63 of retained head h
// (wave w the 16 queries 64 qb + 16 w + i) over cache rows 0 .. pos0 + last query of the block,
// walked in sub-blocks of 64. Query blocks are dealt last first (blockIdx.y = 0 is the last
// block): the longest rows of the causal triangle start first and the short ones fill in behind
// them. A block whose rows span more than split_sb sub-blocks is served by two units (chunk 0:
// sub-blocks 0 .. split_sb - 1, chunk 1: the rest), so that the last blocks do not leave the
// chip waiting on one long chain: each writes its running maxima, sums and unnormalised outputs
// to a record (device-coherent, in the lanes' own layout), counts itself done, and the second to
// finish combines the other's record with its own registers (the scheme of the decode
// attention's splits). Sub-blocks are staged in LDS once per workgroup (K row-major, V
// transposed into units of 4 rows x 1 dimension), the next sub-block's rows loaded into
// registers while the current one is computed; one barrier per sub-block. Per 16-row tile:
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
#include <algorithm>

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

// 4-byte device-coherent accesses (cache-policy bit sc1, as the 16-byte ones of the common
// header) for the split records
__device__ __forceinline__ float buf_load4f_device(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, kCpolDevice));
}
__device__ __forceinline__ void buf_store4f_device(float v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, (int)off, 0, kCpolDevice);
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

// sub-blocks of cache rows that query block qb attends
__host__ __device__ inline int sub_blocks(const PfAttnArgs& a, int qb) {
  const int kv_end = a.pos0 + (qb * kQB + kQB < a.T ? qb * kQB + kQB : a.T);
  return (kv_end + kKB - 1) / kKB;
}
// A CU retires sub-blocks at about the same rate with one workgroup or two (the loop is
// issue-bound), so the kernel takes about max(longest chain, all sub-blocks / CUs) sub-block
// times. Blocks are split (in halves of the longest block's chain) only where the longest chain
// dominates: at least kMinSplitChain sub-blocks and over 1.5 times the per-CU share. Measured on
// the 8B layer: 512 tokens 22.3 -> 17.5 us; at 2048 tokens, where the share (37) exceeds the
// chain (32), splitting made it slower (84 -> 86 us).
constexpr int kMinSplitChain = 4;
constexpr int kNumCuAttn = 256;
int choose_split_sb(const PfAttnArgs& a, int m_q) {
  const int nqb = (a.T + kQB - 1) / kQB;
  const int longest = sub_blocks(a, nqb - 1);
  long total = 0;
  for (int qb = 0; qb < nqb; ++qb) total += sub_blocks(a, qb);
  total *= m_q;
  if (longest < kMinSplitChain || 2L * longest * kNumCuAttn <= 3L * total) return 0;
  return (longest + 1) / 2;
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
  const int h = blockIdx.x;
  // unit -> (query block, chunk): blocks last first, each block's chunks in order
  const int nqb = (a.T + kQB - 1) / kQB;
  const int ssb = a.part ? a.split_sb : 0;
  int qb = nqb - 1, ch = 0;
  for (int u = blockIdx.y; qb >= 0; --qb) {
    const int n = (ssb > 0 && sub_blocks(a, qb) > ssb) ? 2 : 1;
    if (u < n) {
      ch = u;
      break;
    }
    u -= n;
  }
  if (qb < 0) return;                                   // past the units (not launched)
  int j = 0;                                            // group slot of head h
  while (j + 1 < a.m_kv && a.slot_start[j + 1] <= h) ++j;
  const int g = a.kv_idx[j];
  const int t_block = qb * kQB, t_first = t_block + 16 * wave;
  const int kv_end = a.pos0 + min(t_block + kQB, a.T);  // rows 0 .. kv_end - 1 are attended
  const int n_sb = (kv_end + kKB - 1) / kKB;
  const bool split = ssb > 0 && n_sb > ssb;
  const int sb_begin = (split && ch == 1) ? ssb : 0;
  const int sb_end = (split && ch == 0) ? ssb : n_sb;
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

  load_sb(sb_begin);
  for (int sb = sb_begin; sb < sb_end; ++sb) {
    const int buf = (sb - sb_begin) & 1, tb = sb * kKB;
    stage_sb(buf);                                      // this buffer's readers finished at sb - 2
    if (sb + 1 < sb_end) load_sb(sb + 1);
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

  float inv[4];
  if (split) {
    // record of (h, qb, ch): per wave, o[d][i] of every lane, then (max, sum) of every lane
    constexpr int WREC = NDT * 4 * kWave + 2 * kWave;
    const size_t rec_floats = size_t(4) * WREC;
    const size_t slot = (size_t(h) * nqb + qb) * 2;
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(a.part, uint32_t(a.part_floats * 4u));
    const uint32_t mine = uint32_t(((slot + ch) * rec_floats + size_t(wave) * WREC) * 4u);
    const uint32_t other = uint32_t(((slot + 1 - ch) * rec_floats + size_t(wave) * WREC) * 4u);
#pragma unroll
    for (int d = 0; d < NDT; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) buf_store4f_device(o[d][i], rp, mine + uint32_t(((d * 4 + i) * kWave + lane) * 4));
    buf_store4f_device(m_run, rp, mine + uint32_t((NDT * 4 * kWave + lane) * 4));
    buf_store4f_device(l_run, rp, mine + uint32_t((NDT * 4 * kWave + kWave + lane) * 4));
    __builtin_amdgcn_s_waitcnt(0);                      // this thread's record is at the coherence point
    __syncthreads();                                    // ... and every thread's
    __shared__ int last;
    int* cnt = a.cnt + size_t(h) * nqb + qb;
    if (tid == 0) {
      last = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 1;
      if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!last) return;
    // the other chunk's maximum and sum of query t_first + r, and the combined weights; chunk 0
    // holds row 0 for every query, so the combined maximum is finite
    const float m_o = buf_load4f_device(rp, other + uint32_t((NDT * 4 * kWave + lane) * 4));
    const float l_o = buf_load4f_device(rp, other + uint32_t((NDT * 4 * kWave + kWave + lane) * 4));
    float oo[NDT][4];
#pragma unroll
    for (int d = 0; d < NDT; ++d)
#pragma unroll
      for (int i = 0; i < 4; ++i) oo[d][i] = buf_load4f_device(rp, other + uint32_t(((d * 4 + i) * kWave + lane) * 4));
    const float mm = fmaxf(m_run, m_o);
    const float ws = __builtin_amdgcn_exp2f(m_run - mm), wo = __builtin_amdgcn_exp2f(m_o - mm);
    const float lsum = l_run * ws + l_o * wo;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float s_i = lane_read(ws, 4 * c + i), o_i = lane_read(wo, 4 * c + i);
      inv[i] = 1.0f / lane_read(lsum, 4 * c + i);
#pragma unroll
      for (int d = 0; d < NDT; ++d) o[d][i] = o[d][i] * s_i + oo[d][i] * o_i;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) inv[i] = 1.0f / lane_read(l_run, 4 * c + i);
  }
  // O / l as the hi/lo operand of the O projection: lane (r, c) holds queries t_first + 4 c + i,
  // dimensions 16 d + r
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

size_t pf_attn_record_floats(int max_prefill, int n_q_heads, int dh) {
  const size_t nqb = size_t(std::max(max_prefill, 0) + kQB - 1) / kQB;
  return nqb * size_t(std::max(n_q_heads, 0)) * 2 * 4 * (size_t(dh / 16) * 4 * kWave + 2 * kWave);
}

hipError_t launch_pf_attn(const PfAttnArgs& a0, hipStream_t s) {
  if (a0.m_kv == 0 || a0.T < 1) return hipSuccess;
  const int m_q = a0.slot_start[a0.m_kv];
  if (m_q < 1 || a0.m_kv > 64) return hipErrorInvalidValue;
  // blocks are split only when the records and counters of every (head, block) fit
  PfAttnArgs a = a0;
  const int nqb = (a.T + kQB - 1) / kQB;
  if (!a.part || !a.cnt || a.part_floats < pf_attn_record_floats(a.T, m_q, a.dh) ||
      a.part_floats * 4 >= size_t(kOOB) || long(a.cnt_len) < long(m_q) * nqb)
    a.part = nullptr;
  a.split_sb = a.part ? choose_split_sb(a, m_q) : 0;
  if (a.split_sb == 0) a.part = nullptr;
  int units = nqb;
  for (int qb = 0; qb < nqb && a.part; ++qb) units += sub_blocks(a, qb) > a.split_sb ? 1 : 0;
  const dim3 grid(m_q, units);
  if (a.dh == 128) hipLaunchKernelGGL((pf_attn_kernel<128>), grid, dim3(kBlock), 0, s, a);
  else if (a.dh == 64) hipLaunchKernelGGL((pf_attn_kernel<64>), grid, dim3(kBlock), 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace tasp

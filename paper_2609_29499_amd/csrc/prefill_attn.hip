// Causal prefill attention on the matrix cores, over the retained KV groups only.
//
// Grid (query blocks of 16, retained group slots): workgroup (qb, j) serves queries
// 16 qb .. 16 qb + 15 of every retained head of slot j, so each K/V row staged in LDS is shared by
// the group's heads. Cache rows 0 .. pos0 + last query are walked in sub-blocks of 64:
//   * K (row-major) and V (transposed, dimension-major) of the sub-block are staged in LDS, rows
//     past the causal end read as zeros; the next sub-block's rows are loaded into registers
//     while the current one is computed;
//   * per head, S = Q K^T with v_mfma_f32_16x16x32_bf16 (q as hi/lo BF16 planes, K exact BF16),
//     already in base-2 units (q carries log2(e) / sqrt(d_h)); rows after a query's position are
//     masked; an online softmax keeps each query row's running max and sum in the four rows a
//     lane holds of the MFMA output;
//   * P goes through LDS (the MFMA output layout is transposed with respect to its operand layout)
//     as hi/lo planes and O += P V accumulates in registers.
// The output O / l is written as the hi/lo operand of the O projection.
#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kQB = 16;                // queries per workgroup
constexpr int kKB = 64;                // cache rows per sub-block
constexpr int kVtRow = kKB + 8;        // BF16 per transposed-V row (padding)
constexpr int kPRow = kKB + 8;

template <int DH>
struct PaSmem {
  uint16_t k[kKB * (DH + 8)];          // [row][dim]
  uint16_t vt[DH * kVtRow];            // [dim][row]
  uint16_t p[4][2][kQB * kPRow];       // [wave][hi/lo][query][row]
};

__device__ __forceinline__ bf16x8 lds8(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

template <int DH, int UPW>
__global__ __launch_bounds__(kBlock) void pf_attn_kernel(PfAttnArgs a) {
  constexpr int NKC = DH / 32;         // k chunks of the score MFMAs
  constexpr int NDT = DH / 16;         // output dimension tiles
  constexpr int KROW = DH + 8;
  __shared__ __attribute__((aligned(16))) PaSmem<DH> sm;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, q = lane >> 4;
  const int qb = blockIdx.x, j = blockIdx.y;
  const int h0 = a.slot_start[j], nh = a.slot_start[j + 1] - h0;
  const int g = a.kv_idx[j];
  const int t_first = qb * kQB;
  const int kv_end = a.pos0 + min(t_first + kQB, a.T);  // rows 0 .. kv_end - 1 are attended
  const int n_sb = (kv_end + kKB - 1) / kKB;
  const uint16_t* kc = a.kc + size_t(g) * a.S * DH;
  const uint16_t* vc = a.vc + size_t(g) * a.S * DH;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kc, uint32_t(kv_end) * DH * 2u);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vc, uint32_t(kv_end) * DH * 2u);

  // ---- per unit (head): q fragments, output accumulators, running max / sum of 4 query rows
  bf16x8 qf[UPW][2][NKC];
  f32x4 o[UPW][NDT];
  float m_run[UPW][4], l_run[UPW][4];
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(a.q, uint32_t(2 * a.q_plane) * 2u);
#pragma unroll
  for (int u = 0; u < UPW; ++u) {
    const int h = wave + 4 * u;
    const int t = t_first + r;
    const bool ok = h < nh && t < a.T;
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int kk = 0; kk < NKC; ++kk) {
        const uint32_t off = ok ? (uint32_t(pl) * uint32_t(a.q_plane) +
                                   (uint32_t(h0 + h) * uint32_t(a.T_ld) + uint32_t(t)) * DH + 32u * kk + 8u * q) * 2u
                                : kOOB;
        qf[u][pl][kk] = __builtin_bit_cast(bf16x8, buf_load16(rq, off));
      }
#pragma unroll
    for (int d = 0; d < NDT; ++d) o[u][d] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m_run[u][i] = -INFINITY;
      l_run[u][i] = 0.0f;
    }
  }

  // K / V pieces of one sub-block per thread: piece tid + kBlock i is row p / PPR, 16-byte
  // column piece p % PPR. The next sub-block's pieces are loaded into registers while the current
  // one is computed from LDS.
  constexpr int PPR = DH / 8;                           // 16-byte pieces per row
  constexpr int KPT = kKB * PPR / kBlock;               // pieces per thread
  static_assert(kKB * PPR % kBlock == 0, "sub-block pieces must divide over the workgroup");
  int4 pk[KPT], pv[KPT];
  auto load_sb = [&](int sb) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int p = tid + kBlock * i;
      const int t = sb * kKB + p / PPR;
      const uint32_t off = t < kv_end ? (uint32_t(t) * DH + 8u * (p % PPR)) * 2u : kOOB;
      pk[i] = buf_load16(rk, off);
      pv[i] = buf_load16(rv, off);
    }
  };
  load_sb(0);

  for (int sb = 0; sb < n_sb; ++sb) {
    const int tb = sb * kKB;
    // ---- stage K and transposed V of rows tb .. tb + 63, then start loading the next rows
    __syncthreads();                                    // previous sub-block fully consumed
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const int p = tid + kBlock * i;
      const int row = p / PPR, c8 = p % PPR;
      *reinterpret_cast<int4*>(&sm.k[row * KROW + 8 * c8]) = pk[i];
      const uint32_t w[4] = {uint32_t(pv[i].x), uint32_t(pv[i].y), uint32_t(pv[i].z), uint32_t(pv[i].w)};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sm.vt[(8 * c8 + 2 * e) * kVtRow + row] = uint16_t(w[e] & 0xffffu);
        sm.vt[(8 * c8 + 2 * e + 1) * kVtRow + row] = uint16_t(w[e] >> 16);
      }
    }
    if (sb + 1 < n_sb) load_sb(sb + 1);
    __syncthreads();

#pragma unroll
    for (int u = 0; u < UPW; ++u) {
      const int h = wave + 4 * u;
      const bool active = h < nh;                      // wave-uniform
      if (active) {
        // scores of 16 queries x 64 rows: tile ct holds rows tb + 16 ct + r
        f32x4 s[4];
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
          s[ct] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int kk = 0; kk < NKC; ++kk) {
            const bf16x8 kf = lds8(&sm.k[(16 * ct + r) * KROW + 32 * kk + 8 * q]);
            s[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[u][0][kk], kf, s[ct], 0, 0, 0);
            s[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[u][1][kk], kf, s[ct], 0, 0, 0);
          }
        }
        // causal mask and online softmax; lane holds query rows 4q + i, cache row tb + 16 ct + r
        float alpha[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int qpos = a.pos0 + t_first + 4 * q + i;
          float mx = -INFINITY;
#pragma unroll
          for (int ct = 0; ct < 4; ++ct) {
            const int t = tb + 16 * ct + r;
            if (t > qpos) s[ct][i] = -INFINITY;
            mx = fmaxf(mx, s[ct][i]);
          }
          mx = row16_max(mx);
          const float mn = fmaxf(m_run[u][i], mx);
          float sum = 0.0f;
#pragma unroll
          for (int ct = 0; ct < 4; ++ct) {
            const float pv = exp2f(s[ct][i] - mn);
            s[ct][i] = pv;
            sum += pv;
          }
          sum = row16_sum(sum);
          alpha[i] = exp2f(m_run[u][i] - mn);
          l_run[u][i] = l_run[u][i] * alpha[i] + sum;
          m_run[u][i] = mn;
        }
#pragma unroll
        for (int d = 0; d < NDT; ++d)
#pragma unroll
          for (int i = 0; i < 4; ++i) o[u][d][i] *= alpha[i];
        // P (hi/lo) to LDS in operand layout [query][row]
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float pv = s[ct][i];
            const uint16_t hi = f32_to_bf16(pv);
            const int at = (4 * q + i) * kPRow + 16 * ct + r;
            sm.p[wave][0][at] = hi;
            sm.p[wave][1][at] = f32_to_bf16(pv - bf16_to_f32(hi));
          }
      }
      __syncthreads();                                  // P visible across the wave's lanes
      if (active) {
#pragma unroll
        for (int k2 = 0; k2 < kKB / 32; ++k2) {
          const bf16x8 phi = lds8(&sm.p[wave][0][r * kPRow + 32 * k2 + 8 * q]);
          const bf16x8 plo = lds8(&sm.p[wave][1][r * kPRow + 32 * k2 + 8 * q]);
#pragma unroll
          for (int d = 0; d < NDT; ++d) {
            const bf16x8 vf = lds8(&sm.vt[(16 * d + r) * kVtRow + 32 * k2 + 8 * q]);
            o[u][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(phi, vf, o[u][d], 0, 0, 0);
            o[u][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(plo, vf, o[u][d], 0, 0, 0);
          }
        }
      }
      __syncthreads();                                  // P buffer reused by the next unit
    }
  }

  // ---- O / l as the hi/lo operand of the O projection: lane holds query 4q + i, dim 16 d + r
#pragma unroll
  for (int u = 0; u < UPW; ++u) {
    const int h = wave + 4 * u;
    if (h >= nh) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = t_first + 4 * q + i;
      if (t >= a.T) continue;
      const float inv = 1.0f / l_run[u][i];
#pragma unroll
      for (int d = 0; d < NDT; ++d) {
        const float v = o[u][d][i] * inv;
        const uint16_t hi = f32_to_bf16(v);
        const size_t at = size_t(t) * a.ldo + size_t(h0 + h) * DH + 16 * d + r;
        a.o[at] = hi;
        a.o[a.o_plane + at] = f32_to_bf16(v - bf16_to_f32(hi));
      }
    }
  }
}

template <int DH>
hipError_t launch_dh(const PfAttnArgs& a, int nhm, hipStream_t s) {
  const dim3 grid((a.T + kQB - 1) / kQB, a.m_kv);
  if (nhm <= 4) hipLaunchKernelGGL((pf_attn_kernel<DH, 1>), grid, dim3(kBlock), 0, s, a);
  else hipLaunchKernelGGL((pf_attn_kernel<DH, 2>), grid, dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pf_attn(const PfAttnArgs& a, hipStream_t s) {
  if (a.m_kv == 0 || a.T < 1) return hipSuccess;
  int nhm = 0;
  for (int j = 0; j < a.m_kv; ++j) nhm = nhm > a.slot_start[j + 1] - a.slot_start[j] ? nhm : a.slot_start[j + 1] - a.slot_start[j];
  if (nhm < 1 || nhm > 8) return hipErrorInvalidValue;
  if (a.dh == 128) return launch_dh<128>(a, nhm, s);
  if (a.dh == 64) return launch_dh<64>(a, nhm, s);
  return hipErrorInvalidValue;
}

}  // namespace tasp

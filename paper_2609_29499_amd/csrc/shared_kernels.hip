// Decode GEMVs of a shared-store plan (paper, appendix "Backing-store semantics": every mask
// indexes one immutable packed store and owns no weight bytes; Table "configuration": symmetric
// groupwise INT8 with group size 128 and BF16 scales). One sequence, float32 activations.
//
// A plan's GEMV reads the store through two maps built at compile time:
//   rows: plan row -> store row (the retained query heads' rows, then K and V rows of the
//         retained groups for QKV; the retained channels for gate / up), null for all rows;
//   cols: plan piece of 16 columns -> store column of its first element (the retained heads'
//         columns of W_o, the retained channel blocks of W_down), null for all columns.
// Work decomposition follows the per-row kernel: groups of 2 rows (gate/up: one channel's gate
// and up row), tiles of 1 KiB per row in the plan's column space, each wave a contiguous
// range of groups with two register buffers in ping-pong. A lane's 16 bytes lie in one piece,
// hence in one scale group: it loads the group's BF16 scale with them, forms the 16-byte dot
// product in float32 (byte XOR 0x80 converted exactly to b + 128) and adds
// scale * (dot - 128 * sum of the piece's 16 inputs); the piece sums are staged in LDS with the
// input. The column map is staged in LDS for all tiles but each wave's first, whose map entries
// every lane loads itself.
#include <algorithm>

#include "device_common.hpp"
#include "kernels.hpp"

namespace tasp {
namespace {

// Rows per group: 2 (gate/up: one channel = its gate and up row), twice the waves of 4-row
// groups (measured 7 % faster per 8B layer step).
constexpr int kR = 2;
constexpr int kCH = kR / 2;
constexpr int kC = 1;                 // 1 KiB chunks per tile (2 measured 1 % slower at the 8B layer)
constexpr int kNumCu = 256;
constexpr int kWgPerCu = 4;
constexpr int kScaleGroup = 128;

__device__ __forceinline__ float dot_bytes(uint32_t word, const float4& x, float acc) {
  const uint32_t u = word ^ 0x80808080u;
  acc = fmaf(float(u & 0xffu), x.x, acc);
  acc = fmaf(float((u >> 8) & 0xffu), x.y, acc);
  acc = fmaf(float((u >> 16) & 0xffu), x.z, acc);
  acc = fmaf(float(u >> 24), x.w, acc);
  return acc;
}

// NW waves per workgroup: 4, or 8 where the staged input leaves room for fewer than four
// workgroups per CU (the same waves per CU with half the staging)
template <int MODE, int NW>
__global__ __launch_bounds__(NW * kWave) __attribute__((amdgpu_waves_per_eu(4))) void shared_gemv_kernel(
    SharedGemvArgs a) {
  constexpr bool NORM = (MODE != GEMV_RESID);
  extern __shared__ __attribute__((aligned(16))) float lds[];
  __shared__ float red[NW];
  constexpr int NT = NW * kWave;
  const int K = a.K, N = a.N;
  const int KP = (K + 1023) & ~1023;
  const int NP = KP >> 4;                                 // pieces staged
  float* xs = lds;                                        // [KP], lane-swizzled
  float* xsum = lds + KP;                                 // [NP] sums of the pieces' inputs
  int* cmap = reinterpret_cast<int*>(xsum + NP);          // [NP] store column of each piece
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * NW + (tid >> 6));
  const int nwaves = gridDim.x * NW;
  const int nchunks = (K + 1023) >> 10;
  const int KB = max(1, (nchunks + kC - 1) / kC);
  const int per_group = (MODE == GEMV_GATEUP) ? kCH : kR;
  const int G = (N + per_group - 1) / per_group;
  const int g0 = int((long(wave) * G) / nwaves), g1 = int((long(wave + 1) * G) / nwaves);
  const int t_begin = g0 * KB, t_end = g1 * KB;
  const uint32_t ld = uint32_t(a.ld), lds_groups = uint32_t(a.ld / kScaleGroup);
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.w, uint32_t(a.store_rows) * ld);
  const __amdgpu_buffer_rsrc_t rw2 = make_rsrc(MODE == GEMV_GATEUP ? a.w2 : a.w, uint32_t(a.store_rows) * ld);
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.s, uint32_t(a.store_rows) * lds_groups * 2u);
  const __amdgpu_buffer_rsrc_t rs2 =
      make_rsrc(MODE == GEMV_GATEUP ? a.s2 : a.s, uint32_t(a.store_rows) * lds_groups * 2u);
  const int* __restrict__ rows = a.rows;

  auto row_of = [&](int gi, int r) {
    return (MODE == GEMV_GATEUP) ? gi * kCH + (r % kCH) : gi * kR + r;
  };
  // first: the column-map entries come from c_first (the lane's own, loaded from memory) instead
  // of the staged map
  auto issue = [&](int t, int4 (&w)[kC][kR], uint32_t (&sv)[kC][kR], const int (&c_first)[kC],
                   bool first) {
    const bool ok_t = t < t_end;
    const int gi = ok_t ? t / KB : 0;
    const int kb = t - gi * KB;
    int srow[kR];
#pragma unroll
    for (int r = 0; r < kR; ++r) {
      const int row = row_of(gi, r);
      srow[r] = (ok_t && row < N) ? (rows ? rows[row] : row) : -1;
    }
#pragma unroll
    for (int u = 0; u < kC; ++u) {
      const int k = (kb * kC + u) * 1024 + lane * 16;
      const int scol = (a.cols && k < K) ? (first ? c_first[u] : cmap[k >> 4]) : k;
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const bool ok = srow[r] >= 0 && k < K;
        const uint32_t off = ok ? uint32_t(srow[r]) * ld + uint32_t(scol) : kOOB;
        const uint32_t soff =
            ok ? (uint32_t(srow[r]) * lds_groups + uint32_t(scol) / kScaleGroup) * 2u : kOOB;
        const bool second = (MODE == GEMV_GATEUP && r >= kCH);
        w[u][r] = buf_load16_stream(second ? rw2 : rw, off);
        sv[u][r] = __builtin_amdgcn_raw_buffer_load_b16(second ? rs2 : rs, int(soff), 0, 0);
      }
    }
  };

  int4 wa[kC][kR], wb[kC][kR];
  uint32_t sa[kC][kR], sb[kC][kR];

  // Staging. The wave's first tile is issued between the first batch of input loads and their
  // use: vector loads retire in issue order, so waiting for that batch then does not wait for
  // the weights, and the weight stream starts one memory latency before the input is ready. A
  // column-mapped kernel first loads each lane's map entries of that tile itself (ahead of the
  // inputs, so that waiting for them does not wait for the inputs either); the rest of the map
  // rides with the input batches. Every load of a batch is issued (out-of-range offsets return
  // zeros) and consumed, so that the wait counts are the same on every path.
  const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.cols, a.cols ? uint32_t(K >> 4) * 4u : 0u);
  int c_first[kC];
  {
    const int kb0 = t_begin - (t_begin / KB) * KB;
#pragma unroll
    for (int u = 0; u < kC; ++u) {
      const int q = (kb0 * kC + u) * 64 + lane;
      c_first[u] = __builtin_amdgcn_raw_buffer_load_b32(rc, t_begin < t_end ? q * 4 : int(kOOB), 0, 0);
    }
  }
  {
    // float4 loads per thread in flight: a second batch waits for the first tile as well (loads
    // retire in order), so the gain-free kernels, with registers to spare, take 12 (the 8B
    // down projection's retained channels in one batch)
    constexpr int kSB = NORM ? 8 : 12;
    const int n4 = K >> 2;
    const int n4p = KP >> 2;                             // float4 slots staged
    const int npass = (n4p + NT - 1) / NT;               // one float4 per thread per pass
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.x, uint32_t(n4) * 16u);
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.gamma, uint32_t(NORM ? K : 0) * 2u);
    float ss = 0.0f;
    int4 xv[kSB];
    int2 gv[NORM ? kSB : 1];
    int cm[kSB];
    auto load_batch = [&](int i0) {
#pragma unroll
      for (int u = 0; u < kSB; ++u) {
        const int c4 = (i0 + u) * NT + tid;            // float4 slot; piece c4 / 4
        const bool ok = i0 + u < npass && c4 < n4;
        xv[u] = buf_load16(rx, ok ? uint32_t(c4) * 16u : kOOB);
        if constexpr (NORM)
          gv[u] = __builtin_bit_cast(int2, __builtin_amdgcn_raw_buffer_load_b64(
                                               rg, ok ? int(uint32_t(c4) * 8u) : int(kOOB), 0, 0));
        cm[u] = __builtin_amdgcn_raw_buffer_load_b32(rc, ok ? (c4 >> 2) * 4 : int(kOOB), 0, 0);
      }
    };
    auto store_batch = [&](int i0) {
#pragma unroll
      for (int u = 0; u < kSB; ++u) {
        const int c4 = (i0 + u) * NT + tid;
        float4 v = __builtin_bit_cast(float4, xv[u]);
        if constexpr (NORM) {
          ss = fmaf(v.x, v.x, fmaf(v.y, v.y, fmaf(v.z, v.z, fmaf(v.w, v.w, ss))));
          v.x *= bf16_lo(uint32_t(gv[u].x));
          v.y *= bf16_hi(uint32_t(gv[u].x));
          v.z *= bf16_lo(uint32_t(gv[u].y));
          v.w *= bf16_hi(uint32_t(gv[u].y));
        }
        // a piece is four consecutive float4 slots, held by four consecutive lanes
        float p = (v.x + v.y) + (v.z + v.w);
        p += dpp<kQuadXor1>(p);
        p += dpp<kQuadXor2>(p);
        if (i0 + u < npass && (NT == 256 || c4 < n4p)) {   // 256 threads: passes end at KP
          *reinterpret_cast<float4*>(xs + xs_slot_i8(c4 << 2)) = v;
          if ((tid & 3) == 0) {
            xsum[c4 >> 2] = p;
            cmap[c4 >> 2] = cm[u];
          }
        }
      }
    };
    load_batch(0);
    issue(t_begin, wa, sa, c_first, true);
    store_batch(0);
    for (int i0 = kSB; i0 < npass; i0 += kSB) {
      load_batch(i0);
      store_batch(i0);
    }
    if (NORM) {
      ss = wave_sum(ss);
      if (lane == 0) red[tid >> 6] = ss;
    }
    __syncthreads();
  }
  float red_sum = 0.0f;
#pragma unroll
  for (int w = 0; w < NW; ++w) red_sum += red[w];
  const float xscale = NORM ? rsqrtf(red_sum / float(K) + a.eps) : 1.0f;

  float acc[kR], res[kR];
  auto process = [&](const int4 (&w)[kC][kR], const uint32_t (&sv)[kC][kR], int t) {
    const int gi = t / KB;
    const int kb = t - gi * KB;
    const int row0 = row_of(gi, 0);
    if (kb == 0) {
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        acc[r] = 0.0f;
        res[r] = (MODE == GEMV_RESID) ? a.resid[min(row0 + r, N - 1)] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < kC; ++u) {
      const int c = kb * kC + u;
      if (c >= nchunks) break;
      const float4* xp = reinterpret_cast<const float4*>(xs) + ((c << 2) << 6) + lane;
      const float4 x0 = xp[0], x1 = xp[64], x2 = xp[128], x3 = xp[192];
      const float bias = 128.0f * xsum[(c << 6) + lane];
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        float d = dot_bytes(uint32_t(w[u][r].x), x0, 0.0f);
        d = dot_bytes(uint32_t(w[u][r].y), x1, d);
        d = dot_bytes(uint32_t(w[u][r].z), x2, d);
        d = dot_bytes(uint32_t(w[u][r].w), x3, d);
        acc[r] = fmaf(bf16_to_f32(uint16_t(sv[u][r])), d - bias, acc[r]);
      }
    }
    if (kb != KB - 1) return;
    float tot[kR];
#pragma unroll
    for (int r = 0; r < kR; ++r) tot[r] = wave_sum(acc[r]);
    if (lane != 0) return;
    if (MODE == GEMV_GATEUP) {
#pragma unroll
      for (int r = 0; r < kCH; ++r) {
        const int ch = row0 + r;
        if (ch >= N) continue;
        const float g = xscale * tot[r];
        const float u = xscale * tot[r + kCH];
        a.y[ch] = g / (1.0f + exp2f(-g * kLog2e)) * u;
      }
    } else {
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const int row = row0 + r;
        if (row >= N) continue;
        a.y[row] = res[r] + xscale * tot[r];
      }
    }
  };

  for (int t = t_begin; t < t_end; t += 2) {
    issue(t + 1, wb, sb, c_first, false);
    process(wa, sa, t);
    issue(t + 2, wa, sa, c_first, false);
    if (t + 1 < t_end) process(wb, sb, t + 1);
  }
}

template <int MODE, int NW>
hipError_t launch_shared_nw(const SharedGemvArgs& a, int grid, size_t lds, hipStream_t s) {
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&shared_gemv_kernel<MODE, NW>),
      hipFuncAttributeMaxDynamicSharedMemorySize, int(kMaxSharedGemvLds));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((shared_gemv_kernel<MODE, NW>), dim3(grid), dim3(NW * kWave), lds, s, a);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_shared_mode(const SharedGemvArgs& a, int groups, int per_cu, size_t lds, hipStream_t s) {
  // one wave per group up to the workgroups resident at once; past that, waves take several
  // groups each
  const int nw = per_cu < kWgPerCu ? 8 : 4;
  const int grid = std::max(1, std::min((groups + nw - 1) / nw, kNumCu * per_cu));
  return nw == 8 ? launch_shared_nw<MODE, 8>(a, grid, lds, s) : launch_shared_nw<MODE, 4>(a, grid, lds, s);
}

// the retained rows and column pieces of every layer in store coordinates (one workgroup per
// layer; integer only)
__global__ __launch_bounds__(kBlock) void shared_maps_kernel(SharedMapsArgs a) {
  const int l = blockIdx.x, tid = threadIdx.x;
  const int mq = a.counts[l * 4], mkv = a.counts[l * 4 + 1], c = a.counts[l * 4 + 2];
  const int dh = a.dh;
  const int* qi = a.q_idx + size_t(l) * a.Hq;
  const int* kvi = a.kv_idx + size_t(l) * a.Hkv;
  const int* fi = a.ffn_idx + size_t(l) * a.F;
  int* qr = a.qkv_rows + size_t(l) * (a.Hq + 2 * a.Hkv) * dh;
  for (int r = tid; r < (mq + 2 * mkv) * dh; r += kBlock) {
    const int blk = r / dh, e = r - blk * dh;
    int srow;
    if (blk < mq) srow = qi[blk] * dh + e;                                    // query rows
    else if (blk < mq + mkv) srow = (a.Hq + kvi[blk - mq]) * dh + e;          // K rows
    else srow = (a.Hq + a.Hkv + kvi[blk - mq - mkv]) * dh + e;               // V rows
    qr[r] = srow;
  }
  int* oc = a.o_cols + size_t(l) * (a.Hq * dh / 16);
  for (int q = tid; q < mq * dh / 16; q += kBlock) {
    const int col = q * 16;
    oc[q] = qi[col / dh] * dh + col % dh;
  }
  int* dc = a.down_cols + size_t(l) * (a.F / 16);
  for (int q = tid; q < c / 16; q += kBlock) dc[q] = fi[q * 16];
}

}  // namespace

size_t shared_gemv_lds_bytes(int K) {
  const size_t KP = (size_t(K) + 1023) & ~size_t(1023);
  return KP * 4 + (KP / 16) * 8;
}

hipError_t launch_shared_gemv(GemvMode mode, const SharedGemvArgs& a, hipStream_t s) {
  if (a.K % 16 || a.ld % kScaleGroup || a.N < 0) return hipErrorInvalidValue;
  const size_t lds = shared_gemv_lds_bytes(a.K);
  if (lds > kMaxSharedGemvLds) return hipErrorInvalidValue;
  const int per_group = (mode == GEMV_GATEUP) ? kCH : kR;
  // workgroups resident per CU: kWgPerCu, fewer when the staged input limits them
  const int groups = (a.N + per_group - 1) / per_group;
  const int per_cu = std::max(1, std::min(kWgPerCu, int((160 * 1024) / (lds + 64))));
  switch (mode) {
    case GEMV_QKV: return launch_shared_mode<GEMV_QKV>(a, groups, per_cu, lds, s);
    case GEMV_RESID: return launch_shared_mode<GEMV_RESID>(a, groups, per_cu, lds, s);
    case GEMV_GATEUP: return launch_shared_mode<GEMV_GATEUP>(a, groups, per_cu, lds, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_shared_maps(const SharedMapsArgs& a, int n_layers, hipStream_t s) {
  if (n_layers < 1 || a.dh % 16 || a.F % 16) return hipErrorInvalidValue;
  hipLaunchKernelGGL(shared_maps_kernel, dim3(n_layers), dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

}  // namespace tasp

// Host runtime of libtasp: validation, mask closure for sizing and cross-checking, the workspace
// layout of a plan, plan compilation, and the launch sequences of decode.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "tasp.h"

struct tasp_plan_s;

namespace {

thread_local std::string g_err;

tasp_status fail(tasp_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(TASP_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kAlign = 256;
constexpr size_t kLdsLimit = 159 * 1024;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
int round_up16(int v) { return (v + 15) / 16 * 16; }
int round_up64(int v) { return (v + 63) / 64 * 64; }

// ----------------------------------------------------------------------- closure on the host

struct Closed {
  std::vector<uint8_t> q, kv, f;     // closed bits [L][Hq], [L][Hkv], [L][F]
  std::vector<int> m_q, m_kv, c;
};

tasp_status check_desc(const tasp_model_desc* d) {
  if (!d) return fail(TASP_ERR_INVALID_ARG, "desc is NULL");
  if (d->n_layers < 1 || d->d_model < 16 || d->n_q_heads < 1 || d->n_kv_heads < 1 ||
      d->d_ffn < 1 || d->vocab < 0 || d->max_batch < 1 || d->max_seq < 1 || d->max_prefill < 0)
    return fail(TASP_ERR_SHAPE, "non-positive dimension in model desc");
  if (d->d_model % 16) return fail(TASP_ERR_SHAPE, "d_model %% 16 != 0 (%d)", d->d_model);
  if (d->d_model > 16384) return fail(TASP_ERR_SHAPE, "d_model > 16384 (%d)", d->d_model);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(TASP_ERR_SHAPE, "head_dim must be 64 or 128 (%d)", d->head_dim);
  if (d->n_q_heads % d->n_kv_heads)
    return fail(TASP_ERR_SHAPE, "n_q_heads %% n_kv_heads != 0");
  if (d->n_q_heads / d->n_kv_heads > 8)
    return fail(TASP_ERR_SHAPE, "more than 8 query heads per KV group");
  if (d->n_q_heads > 256 || d->n_kv_heads > 64)
    return fail(TASP_ERR_SHAPE, "at most 256 query heads and 64 KV heads");
  if (d->d_ffn % 16) return fail(TASP_ERR_SHAPE, "d_ffn %% 16 != 0 (%d)", d->d_ffn);
  if (d->max_batch > 8) return fail(TASP_ERR_SHAPE, "max_batch > 8");
  if (d->max_prefill > 4096) return fail(TASP_ERR_SHAPE, "max_prefill > 4096");
  if (!(d->rms_eps > 0.0f) || !(d->rope_theta > 0.0))
    return fail(TASP_ERR_SHAPE, "rms_eps and rope_theta must be positive");
  // every panel (and the BF16 LM head) must be addressable by a 31-bit buffer offset
  const double big = double(1u << 31) - 1.0;
  const double D = d->d_model, qkv_rows = double(d->n_q_heads + 2 * d->n_kv_heads) * d->head_dim;
  if (qkv_rows * D > big || double(d->d_ffn) * D > big || D * d->n_q_heads * d->head_dim > big ||
      double(d->vocab) * D * 2.0 > big)
    return fail(TASP_ERR_SHAPE, "a weight panel exceeds 2^31 bytes");
  // the batched gate/up kernel addresses both panels from the gate panel with 32-bit offsets
  if (2.0 * double(d->d_ffn) * D + 2.0 * kAlign > 4294967295.0)
    return fail(TASP_ERR_SHAPE, "gate + up panels exceed 2^32 bytes");
  // batch 1 stages every GEMV input vector in LDS (batches 2..8 run on the matrix cores)
  const int widest = std::max({d->d_model, d->n_q_heads * d->head_dim, d->d_ffn});
  if (tasp::gemv_lds_bytes(1, widest) > kLdsLimit)
    return fail(TASP_ERR_UNSUPPORTED, "widest GEMV input exceeds LDS (%d)", widest);
  return TASP_OK;
}

tasp_status host_close(const tasp_model_desc* d, const tasp_mask* m, Closed* out) {
  const int L = d->n_layers, Hq = d->n_q_heads, Hkv = d->n_kv_heads, F = d->d_ffn;
  const int r = Hq / Hkv;
  out->q.assign(size_t(L) * Hq, 1);
  out->kv.assign(size_t(L) * Hkv, 1);
  out->f.assign(size_t(L) * F, 1);
  if (m) {
    if (!m->q_keep || !m->ffn_keep)
      return fail(TASP_ERR_INVALID_ARG, "mask q_keep / ffn_keep is NULL");
    auto check = [](const uint8_t* p, size_t n, const char* what) -> tasp_status {
      for (size_t i = 0; i < n; ++i)
        if (p[i] > 1) return fail(TASP_ERR_MASK, "%s[%zu] = %d is not 0 or 1", what, i, int(p[i]));
      return TASP_OK;
    };
    tasp_status s;
    if ((s = check(m->q_keep, out->q.size(), "q_keep")) != TASP_OK) return s;
    if (m->kv_keep && (s = check(m->kv_keep, out->kv.size(), "kv_keep")) != TASP_OK) return s;
    if ((s = check(m->ffn_keep, out->f.size(), "ffn_keep")) != TASP_OK) return s;
    for (int l = 0; l < L; ++l)
      for (int h = 0; h < Hq; ++h) {
        const bool g_in = m->kv_keep ? m->kv_keep[size_t(l) * Hkv + h / r] != 0 : true;
        out->q[size_t(l) * Hq + h] = (m->q_keep[size_t(l) * Hq + h] != 0) && g_in;
      }
    std::memcpy(out->f.data(), m->ffn_keep, out->f.size());
  }
  out->m_q.assign(L, 0);
  out->m_kv.assign(L, 0);
  out->c.assign(L, 0);
  for (int l = 0; l < L; ++l) {
    for (int g = 0; g < Hkv; ++g) {
      uint8_t any = 0;
      for (int h = g * r; h < (g + 1) * r; ++h) any |= out->q[size_t(l) * Hq + h];
      out->kv[size_t(l) * Hkv + g] = any;
      out->m_kv[l] += any;
    }
    for (int h = 0; h < Hq; ++h) out->m_q[l] += out->q[size_t(l) * Hq + h];
    for (int j = 0; j < F; ++j) out->c[l] += out->f[size_t(l) * F + j];
  }
  return TASP_OK;
}

// ----------------------------------------------------------------------- workspace layout

struct LayerLayout {
  size_t qkv, s_qkv, o, s_o, g, u, s_g, s_u, dn, s_d, an, fn;
  int n_qkv, ld_o, ld_d;
};

struct Layout {
  std::vector<LayerLayout> layers;
  size_t mask_q, mask_kv, mask_f;
  size_t idx_q, idx_kv, idx_slot, idx_slot_start, idx_ffn, counts;
  size_t final_norm, lm_head, rope_cos, rope_sin;
  size_t r_mid, r_io0, r_io1, qkv_buf, o_buf, h_buf, part, acnt;
  size_t xd, xo, xh, ssq;            // batched path: hi/lo operands and sums of squares
  size_t pxd, pxw, pq, pqkv, pr_mid, pr_io0, pr_io1, pssq;   // prefill scratch
  size_t ppart, ppart_floats;                                // prefill K-split partials and
                                                             // split attention records
  size_t pacnt;                      // prefill attention: counter per (head, query block)
  int pacnt_len = 0;
  size_t arg_part, arg_cnt;          // request loop: argmax partials and counters
  size_t qkv_rows, o_cols, down_cols;                        // shared-store plans: maps
  size_t zero_begin, zero_end;       // scratch cleared at compile
  size_t total;
  size_t scratch_total = 0;          // shared-store plans: bytes of the separate scratch arena
  int n_split_max, ld_qkv, ld_obuf, ld_h, ld_xd, ld_xo, ld_xh, ld_xw;
};

// Decode and prefill scratch of a plan (every format): residuals, q/k/v, attention partials and
// split counters, batched operands (max_batch > 1) and prefill operands (max_prefill > 0).
// zero_begin .. zero_end is cleared at compile; the prefill split partials after it are written
// in full before they are read.
template <class Take>
void scratch_layout(Layout& Y, const tasp_model_desc* d, Take&& take, size_t& off) {
  const int D = d->d_model, Hq = d->n_q_heads, Hkv = d->n_kv_heads;
  const int dh = d->head_dim, F = d->d_ffn, B = d->max_batch;
  Y.n_split_max = tasp::attn_mfma_max_split(d->max_seq);
  Y.ld_qkv = (Hq + 2 * Hkv) * dh;
  Y.ld_obuf = Hq * dh;
  Y.ld_h = round_up16(F);
  Y.zero_begin = off;
  Y.r_mid = take(size_t(B) * D * 4);
  Y.r_io0 = take(size_t(B) * D * 4);
  Y.r_io1 = take(size_t(B) * D * 4);
  Y.qkv_buf = take(size_t(B) * Y.ld_qkv * 4);
  Y.o_buf = take(size_t(B) * Y.ld_obuf * 4);
  Y.h_buf = take(size_t(B) * Y.ld_h * 4);
  Y.part = take(size_t(B) * Hkv * Y.n_split_max * 8 * (dh + 4) * 4);
  Y.acnt = take(size_t(B) * Hkv * 4);
  Y.ld_xd = round_up64(D);
  Y.ld_xo = round_up64(Hq * dh);
  Y.ld_xh = round_up64(F);
  const bool batched = B > 1;
  Y.xd = take(batched ? size_t(16) * Y.ld_xd * 2 : 0);
  Y.xo = take(batched ? size_t(16) * Y.ld_xo * 2 : 0);
  Y.xh = take(batched ? size_t(16) * Y.ld_xh * 2 : 0);
  Y.ssq = take(batched ? size_t(B) * (D / 16) * 4 : 0);
  // prefill of up to P tokens: hi/lo operand planes, q planes, q/k/v, residuals, RMS partials
  const size_t P = size_t(d->max_prefill);
  Y.ld_xw = round_up64(std::max(Hq * dh, F));
  Y.pxd = take(2 * P * Y.ld_xd * 2);
  Y.pxw = take(2 * P * Y.ld_xw * 2);
  Y.pq = take(2 * size_t(Hq) * P * dh * 2);
  Y.pqkv = take(P * Y.ld_qkv * 4);
  Y.pr_mid = take(P * D * 4);
  Y.pr_io0 = take(P * D * 4);
  Y.pr_io1 = take(P * D * 4);
  Y.pssq = take(P * ((D + 63) / 64) * 4);
  Y.pacnt_len = int(size_t(Hq) * ((P + 63) / 64));
  Y.pacnt = take(size_t(Y.pacnt_len) * 4);
  Y.arg_cnt = take(size_t(tasp::kArgmaxMaxRows) * 4);
  Y.zero_end = off;
  Y.arg_part = take(size_t(tasp::kArgmaxMaxRows) * tasp::kArgmaxMaxChunks * 2 * 4);
  Y.ppart_floats = P ? std::max(tasp::pf_split_buffer_floats(int(P), std::max(D, Y.ld_qkv)),
                                tasp::pf_attn_record_floats(int(P), Hq, dh))
                     : 0;
  Y.ppart = take(Y.ppart_floats * 4);
}

Layout make_layout(const tasp_model_desc* d, const Closed& c) {
  Layout Y;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, kAlign);
    return at;
  };
  const int L = d->n_layers, D = d->d_model, Hq = d->n_q_heads, Hkv = d->n_kv_heads;
  const int dh = d->head_dim, F = d->d_ffn;
  Y.layers.resize(L);
  for (int l = 0; l < L; ++l) {
    LayerLayout& P = Y.layers[l];
    P.n_qkv = (c.m_q[l] + 2 * c.m_kv[l]) * dh;
    P.ld_o = c.m_q[l] * dh;
    P.ld_d = round_up16(c.c[l]);
    P.qkv = take(size_t(P.n_qkv) * D);
    P.s_qkv = take(size_t(P.n_qkv) * 4);
    P.o = take(size_t(D) * P.ld_o);
    P.s_o = take(size_t(D) * 4);
    P.g = take(size_t(c.c[l]) * D);
    P.u = take(size_t(c.c[l]) * D);
    P.s_g = take(size_t(c.c[l]) * 4);
    P.s_u = take(size_t(c.c[l]) * 4);
    P.dn = take(size_t(D) * P.ld_d);
    P.s_d = take(size_t(D) * 4);
    P.an = take(size_t(D) * 2);
    P.fn = take(size_t(D) * 2);
  }
  Y.mask_q = take(size_t(L) * Hq);
  Y.mask_kv = take(size_t(L) * Hkv);
  Y.mask_f = take(size_t(L) * F);
  Y.idx_q = take(size_t(L) * Hq * 4);
  Y.idx_kv = take(size_t(L) * Hkv * 4);
  Y.idx_slot = take(size_t(L) * Hq * 4);
  Y.idx_slot_start = take(size_t(L) * (Hkv + 1) * 4);
  Y.idx_ffn = take(size_t(L) * F * 4);
  Y.counts = take(size_t(L) * 4 * 4);
  Y.final_norm = d->vocab ? take(size_t(D) * 2) : 0;
  Y.lm_head = d->vocab ? take(size_t(d->vocab) * D * 2) : 0;
  Y.rope_cos = take(size_t(d->max_seq) * (dh / 2) * 4);
  Y.rope_sin = take(size_t(d->max_seq) * (dh / 2) * 4);
  scratch_layout(Y, d, take, off);
  Y.total = off;
  return Y;
}

// A shared-store plan holds no weights: masks and index lists, the maps into the store and the
// RoPE table (Y.total bytes, the same for every mask). Its decode / prefill scratch is a separate
// arena of Y.scratch_total bytes (offsets relative to the arena) that plans may share.
Layout make_shared_layout(const tasp_model_desc* d) {
  Layout Y{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, kAlign);
    return at;
  };
  const int L = d->n_layers, Hq = d->n_q_heads, Hkv = d->n_kv_heads;
  const int dh = d->head_dim, F = d->d_ffn;
  Y.mask_q = take(size_t(L) * Hq);
  Y.mask_kv = take(size_t(L) * Hkv);
  Y.mask_f = take(size_t(L) * F);
  Y.idx_q = take(size_t(L) * Hq * 4);
  Y.idx_kv = take(size_t(L) * Hkv * 4);
  Y.idx_slot = take(size_t(L) * Hq * 4);
  Y.idx_slot_start = take(size_t(L) * (Hkv + 1) * 4);
  Y.idx_ffn = take(size_t(L) * F * 4);
  Y.counts = take(size_t(L) * 4 * 4);
  Y.qkv_rows = take(size_t(L) * (Hq + 2 * Hkv) * dh * 4);
  Y.o_cols = take(size_t(L) * (Hq * dh / 16) * 4);
  Y.down_cols = take(size_t(L) * (F / 16) * 4);
  Y.rope_cos = take(size_t(d->max_seq) * (dh / 2) * 4);
  Y.rope_sin = take(size_t(d->max_seq) * (dh / 2) * 4);
  Y.total = off;
  size_t soff = 0;
  auto stake = [&](size_t bytes) {
    const size_t at = soff;
    soff = align_up(soff + bytes, kAlign);
    return at;
  };
  scratch_layout(Y, d, stake, soff);
  Y.scratch_total = soff;
  return Y;
}

uint64_t fnv1a(uint64_t h, const void* p, size_t n) {
  const uint8_t* b = static_cast<const uint8_t*>(p);
  for (size_t i = 0; i < n; ++i) {
    h ^= b[i];
    h *= 1099511628211ull;
  }
  return h;
}

// Retained per-token FLOPs of one layer (paper, Eqs. flop-attn and flop-mlp).
double layer_flops(const tasp_model_desc* d, int m_q, int m_kv, int c) {
  const double D = d->d_model, dh = d->head_dim;
  return 2.0 * D * dh * (m_q + 2.0 * m_kv) + 2.0 * dh * m_q * D + 6.0 * D * c;
}

}  // namespace

// ------------------------------------------------------------------------------- the plan

struct LayerPlan {
  int m_q, m_kv, c, n_qkv, ld_o, ld_d;
  int8_t *qkv, *o, *g, *u, *dn;
  float *s_qkv, *s_o, *s_g, *s_u, *s_d;
  uint16_t *an, *fn;
  std::vector<int> q_idx, kv_idx, q_kvslot, ffn_idx, slot_start;
};

// a shared-store plan's view of one store layer and its maps (device pointers)
struct SharedLayer {
  const int8_t *qkv, *o, *g, *u, *d;
  const uint16_t *s_qkv, *s_o, *s_g, *s_u, *s_d;
  const int *qkv_rows, *o_cols, *ffn_rows, *down_cols;
};

struct tasp_plan_s {
  tasp_model_desc desc;
  bool shared = false;               // indexes a groupwise store instead of owning panels
  std::vector<SharedLayer> sl;
  uint64_t sig;
  double ratio;
  uint64_t weight_bytes, scale_bytes;
  std::vector<LayerPlan> layers;
  uint16_t *final_norm, *lm_head;
  float *rope_cos, *rope_sin;
  float *r_mid, *r_io[2], *qkv_buf, *o_buf, *h_buf, *part;
  int* acnt;                       // attention split counters [B][H_kv], zero between launches
  int n_split_max, ld_qkv, ld_obuf, ld_h;
  uint16_t *xd, *xo, *xh;            // batched path operands [16][ld_x*]
  float* ssq;                        // [max_batch][d_model / 16]
  int ld_xd, ld_xo, ld_xh;
  uint16_t *pxd, *pxw, *pq;          // prefill operands: [2][max_prefill][ld_xd | ld_xw], q planes
  float *pqkv, *pr_mid, *pr_io[2], *pssq;
  float* ppart;                      // prefill K-split partials, split attention records
  size_t ppart_floats;
  int* pacnt;                        // prefill attention counters, zero between launches
  int pacnt_len;
  float* arg_part;                   // argmax partials and counters (zero between launches)
  int* arg_cnt;
  int ld_xw;
};

namespace {

// Pointers of a plan into the decode / prefill scratch of its workspace (scratch_layout).
void set_scratch(tasp_plan_s* p, const Layout& Y, char* ws) {
  auto at = [&](size_t off) { return ws + off; };
  p->r_mid = reinterpret_cast<float*>(at(Y.r_mid));
  p->r_io[0] = reinterpret_cast<float*>(at(Y.r_io0));
  p->r_io[1] = reinterpret_cast<float*>(at(Y.r_io1));
  p->qkv_buf = reinterpret_cast<float*>(at(Y.qkv_buf));
  p->o_buf = reinterpret_cast<float*>(at(Y.o_buf));
  p->h_buf = reinterpret_cast<float*>(at(Y.h_buf));
  p->part = reinterpret_cast<float*>(at(Y.part));
  p->acnt = reinterpret_cast<int*>(at(Y.acnt));
  p->n_split_max = Y.n_split_max; p->ld_qkv = Y.ld_qkv; p->ld_obuf = Y.ld_obuf; p->ld_h = Y.ld_h;
  p->xd = reinterpret_cast<uint16_t*>(at(Y.xd));
  p->xo = reinterpret_cast<uint16_t*>(at(Y.xo));
  p->xh = reinterpret_cast<uint16_t*>(at(Y.xh));
  p->ssq = reinterpret_cast<float*>(at(Y.ssq));
  p->ld_xd = Y.ld_xd; p->ld_xo = Y.ld_xo; p->ld_xh = Y.ld_xh;
  p->pxd = reinterpret_cast<uint16_t*>(at(Y.pxd));
  p->pxw = reinterpret_cast<uint16_t*>(at(Y.pxw));
  p->pq = reinterpret_cast<uint16_t*>(at(Y.pq));
  p->pqkv = reinterpret_cast<float*>(at(Y.pqkv));
  p->pr_mid = reinterpret_cast<float*>(at(Y.pr_mid));
  p->pr_io[0] = reinterpret_cast<float*>(at(Y.pr_io0));
  p->pr_io[1] = reinterpret_cast<float*>(at(Y.pr_io1));
  p->pssq = reinterpret_cast<float*>(at(Y.pssq));
  p->ppart = reinterpret_cast<float*>(at(Y.ppart));
  p->ppart_floats = Y.ppart_floats;
  p->pacnt = reinterpret_cast<int*>(at(Y.pacnt));
  p->pacnt_len = Y.pacnt_len;
  p->arg_part = reinterpret_cast<float*>(at(Y.arg_part));
  p->arg_cnt = reinterpret_cast<int*>(at(Y.arg_cnt));
  p->ld_xw = Y.ld_xw;
}

// The store view of one projection of a shared-store plan's layer (for the matrix-core kernels):
// 0 QKV (row map), 1 O (column map), 3 gate/up (row map, two matrices), 4 down (column map).
tasp::StoreView store_view(const tasp_plan_s* p, int l, int which) {
  const SharedLayer& Q = p->sl[l];
  const tasp_model_desc& d = p->desc;
  tasp::StoreView v{};
  switch (which) {
    case 0:
      v.w = Q.qkv; v.gs = Q.s_qkv; v.ld = d.d_model;
      v.store_rows = (d.n_q_heads + 2 * d.n_kv_heads) * d.head_dim; v.rows = Q.qkv_rows;
      break;
    case 1:
      v.w = Q.o; v.gs = Q.s_o; v.ld = d.n_q_heads * d.head_dim; v.store_rows = d.d_model;
      v.cols = Q.o_cols;
      break;
    case 3:
      v.w = Q.g; v.w2 = Q.u; v.gs = Q.s_g; v.gs2 = Q.s_u; v.ld = d.d_model; v.store_rows = d.d_ffn;
      v.rows = Q.ffn_rows;
      break;
    default:
      v.w = Q.d; v.gs = Q.s_d; v.ld = d.d_ffn; v.store_rows = d.d_model; v.cols = Q.down_cols;
      break;
  }
  return v;
}

struct Timer {
  std::vector<hipEvent_t> ev;
  std::vector<int> kinds;
};

template <class F>
tasp_status run_kernel(Timer* tm, int kind, hipStream_t s, F&& launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (tm) {
    HIP_TRY(hipEventCreate(&e0));
    HIP_TRY(hipEventCreate(&e1));
    tm->ev.push_back(e0);
    tm->ev.push_back(e1);
    tm->kinds.push_back(kind);
    HIP_TRY(hipEventRecord(e0, s));
  }
  const hipError_t e = launch();
  if (e != hipSuccess) return fail(TASP_ERR_HIP, "kernel launch (kind %d): %s", kind, hipGetErrorString(e));
  if (tm) HIP_TRY(hipEventRecord(e1, s));
  return TASP_OK;
}

// waits for the timed launches, reads their event pairs and releases the events
tasp_status finish_timed(tasp_status st, Timer* tm, hipStream_t s, float* kernel_ms, int32_t* kinds,
                         int32_t cap, int32_t* n, const char* what) {
  hipError_t h = hipStreamSynchronize(s);
  const int k = int(tm->kinds.size());
  if (st == TASP_OK && h == hipSuccess) {
    for (int i = 0; i < k && i < cap; ++i) {
      float ms = 0.0f;
      if (h == hipSuccess) h = hipEventElapsedTime(&ms, tm->ev[2 * i], tm->ev[2 * i + 1]);
      kernel_ms[i] = ms;
      kinds[i] = tm->kinds[i];
    }
    *n = k;
  }
  for (hipEvent_t e : tm->ev) (void)hipEventDestroy(e);
  if (st != TASP_OK) return st;
  if (h != hipSuccess) return fail(TASP_ERR_HIP, "%s: %s", what, hipGetErrorString(h));
  return TASP_OK;
}

tasp_status check_cache(const tasp_plan_s* p, const tasp_kv_cache* c) {
  if (!c) return fail(TASP_ERR_INVALID_ARG, "cache is NULL");
  if (!c->k || !c->v) return fail(TASP_ERR_INVALID_ARG, "cache k / v is NULL");
  if (c->batch < 1 || c->batch > p->desc.max_batch)
    return fail(TASP_ERR_SHAPE, "cache batch %d outside 1..%d", c->batch, p->desc.max_batch);
  if (c->max_seq < 1 || c->max_seq > p->desc.max_seq)
    return fail(TASP_ERR_SHAPE, "cache max_seq %d outside 1..%d", c->max_seq, p->desc.max_seq);
  return TASP_OK;
}

// gate/up GEMV of layer l: RMSNorm(r_mid) -> SwiGLU scratch
tasp::GemvArgs gateup_args(const tasp_plan_s* p, int l, int B) {
  const LayerPlan& P = p->layers[l];
  const int D = p->desc.d_model;
  tasp::GemvArgs a{};
  a.w = P.g; a.w2 = P.u; a.scale = P.s_g; a.scale2 = P.s_u; a.N = P.c; a.K = D; a.ld = D;
  a.x = p->r_mid; a.ldx = D; a.gamma = P.fn; a.eps = p->desc.rms_eps; a.y = p->h_buf;
  a.ldy = p->ld_h; a.B = B;
  return a;
}

// down GEMV of layer l: r_mid + Wd h -> y
tasp::GemvArgs down_args(const tasp_plan_s* p, int l, int B, float* y) {
  const LayerPlan& P = p->layers[l];
  const int D = p->desc.d_model;
  tasp::GemvArgs a{};
  a.w = P.dn; a.scale = P.s_d; a.N = D; a.K = P.c; a.ld = P.ld_d; a.x = p->h_buf;
  a.ldx = p->ld_h; a.resid = p->r_mid; a.y = y; a.ldy = D; a.B = B;
  return a;
}

// ---- shared-store plans (batch 1): the four projections through the plan's maps

tasp::SharedGemvArgs shared_qkv_args(const tasp_plan_s* p, int l, const float* in) {
  const LayerPlan& P = p->layers[l];
  const SharedLayer& Q = p->sl[l];
  const tasp_model_desc& d = p->desc;
  tasp::SharedGemvArgs a{};
  a.w = Q.qkv; a.s = Q.s_qkv; a.ld = d.d_model;
  a.store_rows = (d.n_q_heads + 2 * d.n_kv_heads) * d.head_dim;
  a.rows = Q.qkv_rows; a.N = P.n_qkv; a.K = d.d_model;
  a.x = in; a.gamma = P.an; a.eps = d.rms_eps; a.y = p->qkv_buf;
  return a;
}

tasp::SharedGemvArgs shared_o_args(const tasp_plan_s* p, int l, const float* in) {
  const LayerPlan& P = p->layers[l];
  const SharedLayer& Q = p->sl[l];
  const tasp_model_desc& d = p->desc;
  tasp::SharedGemvArgs a{};
  a.w = Q.o; a.s = Q.s_o; a.ld = d.n_q_heads * d.head_dim; a.store_rows = d.d_model;
  a.cols = Q.o_cols; a.N = d.d_model; a.K = P.m_q * d.head_dim;
  a.x = p->o_buf; a.resid = in; a.y = p->r_mid;
  return a;
}

tasp::SharedGemvArgs shared_gateup_args(const tasp_plan_s* p, int l) {
  const LayerPlan& P = p->layers[l];
  const SharedLayer& Q = p->sl[l];
  const tasp_model_desc& d = p->desc;
  tasp::SharedGemvArgs a{};
  a.w = Q.g; a.w2 = Q.u; a.s = Q.s_g; a.s2 = Q.s_u; a.ld = d.d_model; a.store_rows = d.d_ffn;
  a.rows = Q.ffn_rows; a.N = P.c; a.K = d.d_model;
  a.x = p->r_mid; a.gamma = P.fn; a.eps = d.rms_eps; a.y = p->h_buf;
  return a;
}

tasp::SharedGemvArgs shared_down_args(const tasp_plan_s* p, int l, float* y) {
  const LayerPlan& P = p->layers[l];
  const SharedLayer& Q = p->sl[l];
  const tasp_model_desc& d = p->desc;
  tasp::SharedGemvArgs a{};
  a.w = Q.d; a.s = Q.s_d; a.ld = d.d_ffn; a.store_rows = d.d_model;
  a.cols = Q.down_cols; a.N = d.d_model; a.K = P.c;
  a.x = p->h_buf; a.resid = p->r_mid; a.y = y;
  return a;
}

// decode attention of layer l over the retained groups; hl: write o as the batched operand
tasp::AttnArgs attn_args(const tasp_plan_s* p, int l, const tasp_kv_cache* cache, int pos, int B,
                         bool hl) {
  const LayerPlan& P = p->layers[l];
  const tasp_model_desc& d = p->desc;
  const size_t layer_cache = size_t(B) * d.n_kv_heads * cache->max_seq * d.head_dim;
  const int total = pos + 1;
  tasp::AttnArgs a{};
  a.qkv = p->qkv_buf; a.ld_qkv = p->ld_qkv; a.m_q = P.m_q; a.m_kv = P.m_kv; a.dh = d.head_dim;
  for (int q = 0; q < P.m_kv; ++q) a.kv_idx[q] = P.kv_idx[q];
  for (int q = 0; q <= P.m_kv; ++q) a.slot_start[q] = P.slot_start[q];
  a.kc = static_cast<uint16_t*>(cache->k) + l * layer_cache;
  a.vc = static_cast<uint16_t*>(cache->v) + l * layer_cache;
  a.Hkv = d.n_kv_heads; a.S = cache->max_seq; a.rope_cos = p->rope_cos;
  a.rope_sin = p->rope_sin; a.pos = pos; a.part = p->part; a.cnt = p->acnt;
  a.o = p->o_buf; a.ld_o = p->ld_obuf; a.B = B;
  if (hl) { a.o_hl = p->xo; a.ld_ohl = p->ld_xo; }
  // one sequence: short splits (many more workgroups than group slots); a batch: about one
  // workgroup per CU over its (sequence, group slot) units
  if (B == 1) tasp::attn_mfma_split(total, &a.chunk, &a.n_split);
  else tasp::attn_mfma_split_batched(total, B * P.m_kv, &a.chunk, &a.n_split);
  return a;
}

// ---- batched path (2..8 sequences): projections on the matrix cores over hi/lo operands

tasp::MfmaArgs mm_base(const tasp_plan_s* p, int B) {
  tasp::MfmaArgs a{};
  a.B = B;
  a.inv_d = 1.0f / float(p->desc.d_model);
  a.eps = p->desc.rms_eps;
  a.n_ssq = p->desc.d_model / 16;
  a.n_tiles_out = p->desc.d_model / 16;
  return a;
}

// gate/up of layer l: operand xd (x_mid * gamma_ffn, inverse RMS from ssq) -> SwiGLU into xh
tasp::MfmaArgs gateup_mm_args(const tasp_plan_s* p, int l, int B) {
  const LayerPlan& P = p->layers[l];
  tasp::MfmaArgs a = mm_base(p, B);
  a.w = P.g; a.w2_off = uint32_t(reinterpret_cast<const char*>(P.u) - reinterpret_cast<const char*>(P.g));
  a.scale = P.s_g; a.scale2 = P.s_u; a.N = P.c; a.K = p->desc.d_model; a.ld = p->desc.d_model;
  a.x = p->xd; a.ldx = p->ld_xd; a.ssq = p->ssq; a.xo = p->xh; a.ldxo = p->ld_xh;
  if (p->shared) a.sv = store_view(p, l, 3);
  return a;
}

// down of layer l: y = x_mid + Wd h, and the next operand (gain of the next RMSNorm, if any)
tasp::MfmaArgs down_mm_args(const tasp_plan_s* p, int l, int B, float* y) {
  const LayerPlan& P = p->layers[l];
  const tasp_model_desc& d = p->desc;
  tasp::MfmaArgs a = mm_base(p, B);
  a.w = P.dn; a.scale = P.s_d; a.N = d.d_model; a.K = P.c; a.ld = P.ld_d;
  a.x = p->xh; a.ldx = p->ld_xh; a.resid = p->r_mid; a.y = y; a.ldy = d.d_model;
  a.gamma_next = (l + 1 < d.n_layers) ? p->layers[l + 1].an : (d.vocab ? p->final_norm : nullptr);
  a.xo = p->xd; a.ldxo = p->ld_xd; a.ssq_out = p->ssq;
  if (p->shared) a.sv = store_view(p, l, 4);
  return a;
}

tasp_status decode_batched(tasp_plan p, const float* x, tasp_kv_cache* cache, int pos, float* out,
                           hipStream_t s, Timer* tm, int B) {
  const tasp_model_desc& d = p->desc;
  const int D = d.d_model, dh = d.head_dim, L = d.n_layers;
  tasp_status st;
  if ((st = run_kernel(tm, 6, s, [&] {
         return tasp::launch_mfma_prep(x, D, D, p->layers[0].an, p->xd, p->ld_xd, p->ssq, B, s);
       })))
    return st;
  for (int l = 0; l < L; ++l) {
    const LayerPlan& P = p->layers[l];
    const float* in = (l == 0) ? x : p->r_io[(l - 1) & 1];
    float* lo = (l == L - 1 && d.vocab == 0) ? out : p->r_io[l & 1];
    if (P.n_qkv > 0) {
      tasp::MfmaArgs a = mm_base(p, B);
      a.w = P.qkv; a.scale = P.s_qkv; a.N = P.n_qkv; a.K = D; a.ld = D;
      a.x = p->xd; a.ldx = p->ld_xd; a.ssq = p->ssq; a.y = p->qkv_buf; a.ldy = p->ld_qkv;
      if (p->shared) a.sv = store_view(p, l, 0);
      if ((st = run_kernel(tm, 0, s, [&] { return tasp::launch_mfma_gemv(tasp::MM_QKV, a, s); })))
        return st;
    }
    if (P.m_kv > 0) {
      const tasp::AttnArgs a = attn_args(p, l, cache, pos, B, true);
      if ((st = run_kernel(tm, 1, s, [&] { return tasp::launch_attn_decode(a, s); }))) return st;
    }
    {
      tasp::MfmaArgs a = mm_base(p, B);
      a.w = P.o; a.scale = P.s_o; a.N = D; a.K = P.m_q * dh; a.ld = P.ld_o;
      a.x = p->xo; a.ldx = p->ld_xo; a.resid = in; a.y = p->r_mid; a.ldy = D;
      a.gamma_next = P.fn; a.xo = p->xd; a.ldxo = p->ld_xd; a.ssq_out = p->ssq;
      if (p->shared) a.sv = store_view(p, l, 1);
      if ((st = run_kernel(tm, 2, s, [&] { return tasp::launch_mfma_gemv(tasp::MM_RESID, a, s); })))
        return st;
    }
    if (P.c > 0) {
      const tasp::MfmaArgs a = gateup_mm_args(p, l, B);
      if ((st = run_kernel(tm, 3, s, [&] { return tasp::launch_mfma_gemv(tasp::MM_GATEUP, a, s); })))
        return st;
    }
    {
      const tasp::MfmaArgs a = down_mm_args(p, l, B, lo);
      if ((st = run_kernel(tm, 4, s, [&] { return tasp::launch_mfma_gemv(tasp::MM_RESID, a, s); })))
        return st;
    }
  }
  if (d.vocab) {
    tasp::MfmaArgs a = mm_base(p, B);
    a.w = p->lm_head; a.N = d.vocab; a.K = D; a.ld = D; a.x = p->xd; a.ldx = p->ld_xd;
    a.ssq = p->ssq; a.y = out; a.ldy = d.vocab;
    if ((st = run_kernel(tm, 5, s, [&] { return tasp::launch_mfma_gemv(tasp::MM_LMHEAD, a, s); })))
      return st;
  }
  return TASP_OK;
}

// ---- prefill (T tokens of one sequence): projections and attention on the matrix cores

tasp::PfArgs pf_base(const tasp_plan_s* p, int T) {
  tasp::PfArgs a{};
  a.T = T;
  a.inv_d = 1.0f / float(p->desc.d_model);
  a.eps = p->desc.rms_eps;
  a.n_ssq = (p->desc.d_model + tasp::pf_ssq_block() - 1) / tasp::pf_ssq_block();
  a.n_ssq_out = a.n_ssq;
  a.part = p->ppart;
  a.part_floats = p->ppart_floats;
  return a;
}

// last_only: with an LM head, only the last token's logits (out [vocab]), by the decode LM head
// GEMV over that token's final residual (greedy decoding needs no other row)
tasp_status prefill_impl(tasp_plan p, const float* x, int T, tasp_kv_cache* cache, int pos0,
                         float* out, hipStream_t s, Timer* tm, bool last_only = false) {
  const tasp_model_desc& d = p->desc;
  const int D = d.d_model, dh = d.head_dim, L = d.n_layers, Pm = d.max_prefill;
  const uint32_t plane_d = uint32_t(size_t(Pm) * p->ld_xd);
  const uint32_t plane_w = uint32_t(size_t(Pm) * p->ld_xw);
  const uint32_t plane_q = uint32_t(size_t(d.n_q_heads) * Pm * dh);
  const size_t layer_cache = size_t(cache->batch) * d.n_kv_heads * cache->max_seq * dh;
  tasp_status st;
  if ((st = run_kernel(tm, 6, s, [&] {
         return tasp::launch_pf_prep(x, D, T, p->layers[0].an, p->pxd, plane_d, p->ld_xd, p->pssq, s);
       })))
    return st;
  for (int l = 0; l < L; ++l) {
    const LayerPlan& P = p->layers[l];
    const float* in = (l == 0) ? x : p->pr_io[(l - 1) & 1];
    float* lo = (l == L - 1 && d.vocab == 0) ? out : p->pr_io[l & 1];
    uint16_t* kc = static_cast<uint16_t*>(cache->k) + l * layer_cache;
    uint16_t* vc = static_cast<uint16_t*>(cache->v) + l * layer_cache;
    if (P.n_qkv > 0) {
      tasp::PfArgs a = pf_base(p, T);
      a.w = P.qkv; a.scale = P.s_qkv; a.N = P.n_qkv; a.K = D; a.ld = D;
      a.x = p->pxd; a.ldx = p->ld_xd; a.plane = plane_d; a.ssq = p->pssq;
      a.y = p->pqkv; a.ldy = p->ld_qkv;
      if (p->shared) a.sv = store_view(p, l, 0);
      if ((st = run_kernel(tm, 0, s, [&] { return tasp::launch_pf_gemm(tasp::MM_QKV, a, s); })))
        return st;
    }
    if (P.m_kv > 0) {
      tasp::PfRopeArgs r{};
      r.qkv = p->pqkv; r.ld_qkv = p->ld_qkv; r.m_q = P.m_q; r.m_kv = P.m_kv; r.dh = dh;
      for (int q = 0; q < P.m_kv; ++q) r.kv_idx[q] = P.kv_idx[q];
      r.kc = kc; r.vc = vc; r.S = cache->max_seq; r.rope_cos = p->rope_cos; r.rope_sin = p->rope_sin;
      r.pos0 = pos0; r.T = T; r.q_out = p->pq; r.q_plane = plane_q; r.T_ld = Pm;
      if ((st = run_kernel(tm, 7, s, [&] { return tasp::launch_pf_rope(r, s); }))) return st;
      tasp::PfAttnArgs a{};
      a.q = p->pq; a.q_plane = plane_q; a.T_ld = Pm; a.m_kv = P.m_kv; a.dh = dh;
      for (int q = 0; q < P.m_kv; ++q) a.kv_idx[q] = P.kv_idx[q];
      for (int q = 0; q <= P.m_kv; ++q) a.slot_start[q] = P.slot_start[q];
      a.kc = kc; a.vc = vc; a.S = cache->max_seq; a.pos0 = pos0; a.T = T;
      a.o = p->pxw; a.ldo = p->ld_xw; a.o_plane = plane_w;
      a.part = p->ppart; a.part_floats = p->ppart_floats; a.cnt = p->pacnt; a.cnt_len = p->pacnt_len;
      if ((st = run_kernel(tm, 1, s, [&] { return tasp::launch_pf_attn(a, s); }))) return st;
    }
    {
      tasp::PfArgs a = pf_base(p, T);
      a.w = P.o; a.scale = P.s_o; a.N = D; a.K = P.m_q * dh; a.ld = P.ld_o;
      a.x = p->pxw; a.ldx = p->ld_xw; a.plane = plane_w; a.resid = in; a.y = p->pr_mid; a.ldy = D;
      a.gamma_next = P.fn; a.xo = p->pxd; a.ldxo = p->ld_xd; a.plane_o = plane_d; a.ssq_out = p->pssq;
      if (p->shared) a.sv = store_view(p, l, 1);
      if ((st = run_kernel(tm, 2, s, [&] { return tasp::launch_pf_gemm(tasp::MM_RESID, a, s); })))
        return st;
    }
    if (P.c > 0) {
      tasp::PfArgs a = pf_base(p, T);
      if (p->shared) {
        a.sv = store_view(p, l, 3);
      } else {
        a.w = P.g;
        a.w2_off = uint32_t(reinterpret_cast<const char*>(P.u) - reinterpret_cast<const char*>(P.g));
      }
      a.scale = P.s_g; a.scale2 = P.s_u; a.N = P.c; a.K = D; a.ld = D;
      a.x = p->pxd; a.ldx = p->ld_xd; a.plane = plane_d; a.ssq = p->pssq;
      a.xo = p->pxw; a.ldxo = p->ld_xw; a.plane_o = plane_w;
      if ((st = run_kernel(tm, 3, s, [&] { return tasp::launch_pf_gemm(tasp::MM_GATEUP, a, s); })))
        return st;
    }
    {
      tasp::PfArgs a = pf_base(p, T);
      a.w = P.dn; a.scale = P.s_d; a.N = D; a.K = P.c; a.ld = P.ld_d;
      a.x = p->pxw; a.ldx = p->ld_xw; a.plane = plane_w; a.resid = p->pr_mid; a.y = lo; a.ldy = D;
      if (p->shared) a.sv = store_view(p, l, 4);
      a.gamma_next = (l + 1 < L) ? p->layers[l + 1].an : (d.vocab ? p->final_norm : nullptr);
      a.xo = p->pxd; a.ldxo = p->ld_xd; a.plane_o = plane_d; a.ssq_out = p->pssq;
      if ((st = run_kernel(tm, 4, s, [&] { return tasp::launch_pf_gemm(tasp::MM_RESID, a, s); })))
        return st;
    }
  }
  if (d.vocab && last_only) {
    tasp::GemvArgs a{};
    a.w = p->lm_head; a.N = d.vocab; a.K = D; a.ld = 2 * D;
    a.x = p->pr_io[(L - 1) & 1] + size_t(T - 1) * D; a.ldx = D;
    a.gamma = p->final_norm; a.eps = d.rms_eps; a.y = out; a.ldy = d.vocab;
    a.B = 1;
    if ((st = run_kernel(tm, 5, s, [&] { return tasp::launch_gemv(tasp::GEMV_LMHEAD, a, s); })))
      return st;
  } else if (d.vocab) {
    tasp::PfArgs a = pf_base(p, T);
    a.w = p->lm_head; a.N = d.vocab; a.K = D; a.ld = D; a.x = p->pxd; a.ldx = p->ld_xd;
    a.plane = plane_d; a.ssq = p->pssq; a.y = out; a.ldy = d.vocab;
    if ((st = run_kernel(tm, 5, s, [&] { return tasp::launch_pf_gemm(tasp::MM_LMHEAD, a, s); })))
      return st;
  }
  return TASP_OK;
}

tasp_status prefill_checked(tasp_plan p, const float* x, int32_t T, tasp_kv_cache* cache,
                            int32_t pos0, float* out, void* stream, Timer* tm,
                            bool last_only = false) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  if (!x || !out) return fail(TASP_ERR_INVALID_ARG, "x / out is NULL");
  tasp_status st = check_cache(p, cache);
  if (st != TASP_OK) return st;
  if (p->desc.max_prefill < 1) return fail(TASP_ERR_UNSUPPORTED, "plan compiled with max_prefill 0");
  if (cache->batch != 1) return fail(TASP_ERR_SHAPE, "prefill takes one sequence (cache batch %d)", cache->batch);
  if (T < 1 || T > p->desc.max_prefill) return fail(TASP_ERR_SHAPE, "T %d outside 1..%d", T, p->desc.max_prefill);
  if (pos0 < 0 || pos0 + T > cache->max_seq) return fail(TASP_ERR_POS_RANGE, "pos0 + T beyond the cache");
  if (pos0 > 0 && cache->plan_sig != p->sig)
    return fail(TASP_ERR_CACHE_PLAN_MISMATCH, "cache belongs to plan %016llx, not %016llx",
                (unsigned long long)cache->plan_sig, (unsigned long long)p->sig);
  if (last_only && p->desc.vocab < 1) return fail(TASP_ERR_UNSUPPORTED, "plan has no LM head");
  const size_t out_elems = last_only ? size_t(p->desc.vocab)
                                     : size_t(T) * (p->desc.vocab ? p->desc.vocab : p->desc.d_model);
  const char* xb = reinterpret_cast<const char*>(x);
  const char* ob = reinterpret_cast<const char*>(out);
  if (ob < xb + size_t(T) * p->desc.d_model * 4 && xb < ob + out_elems * 4)
    return fail(TASP_ERR_INVALID_ARG, "x and out overlap");
  if (pos0 == 0) cache->plan_sig = p->sig;             // a fresh sequence binds the cache
  return prefill_impl(p, x, T, cache, pos0, out, static_cast<hipStream_t>(stream), tm, last_only);
}

// one decode step of a shared-store plan (batch 1): the per-row kernels' sequence with the
// projections read from the store through the plan's maps; the LM head is the store's
tasp_status decode_shared(tasp_plan p, const float* x, tasp_kv_cache* cache, int pos, float* out,
                          hipStream_t s, Timer* tm) {
  const tasp_model_desc& d = p->desc;
  const int D = d.d_model, L = d.n_layers;
  tasp_status st = TASP_OK;
  for (int l = 0; l < L; ++l) {
    const LayerPlan& P = p->layers[l];
    const float* in = (l == 0) ? x : p->r_io[(l - 1) & 1];
    float* lo = (l == L - 1 && d.vocab == 0) ? out : p->r_io[l & 1];
    if (P.n_qkv > 0) {
      const tasp::SharedGemvArgs a = shared_qkv_args(p, l, in);
      if ((st = run_kernel(tm, 0, s, [&] { return tasp::launch_shared_gemv(tasp::GEMV_QKV, a, s); })))
        return st;
    }
    if (P.m_kv > 0) {
      const tasp::AttnArgs a = attn_args(p, l, cache, pos, 1, false);
      if ((st = run_kernel(tm, 1, s, [&] { return tasp::launch_attn_decode(a, s); }))) return st;
    }
    {
      const tasp::SharedGemvArgs a = shared_o_args(p, l, in);
      if ((st = run_kernel(tm, 2, s, [&] { return tasp::launch_shared_gemv(tasp::GEMV_RESID, a, s); })))
        return st;
    }
    if (P.c > 0) {
      const tasp::SharedGemvArgs a = shared_gateup_args(p, l);
      if ((st = run_kernel(tm, 3, s, [&] { return tasp::launch_shared_gemv(tasp::GEMV_GATEUP, a, s); })))
        return st;
    }
    {
      const tasp::SharedGemvArgs a = shared_down_args(p, l, lo);
      if ((st = run_kernel(tm, 4, s, [&] { return tasp::launch_shared_gemv(tasp::GEMV_RESID, a, s); })))
        return st;
    }
  }
  if (d.vocab) {
    tasp::GemvArgs a{};
    a.w = p->lm_head; a.N = d.vocab; a.K = D; a.ld = 2 * D; a.x = p->r_io[(L - 1) & 1];
    a.ldx = D; a.gamma = p->final_norm; a.eps = d.rms_eps; a.y = out; a.ldy = d.vocab; a.B = 1;
    if ((st = run_kernel(tm, 5, s, [&] { return tasp::launch_gemv(tasp::GEMV_LMHEAD, a, s); })))
      return st;
  }
  return TASP_OK;
}

tasp_status decode_impl(tasp_plan p, const float* x, tasp_kv_cache* cache, int32_t pos,
                        float* out, void* stream, Timer* tm) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  if (!x || !out) return fail(TASP_ERR_INVALID_ARG, "x / out is NULL");
  tasp_status st = check_cache(p, cache);
  if (st != TASP_OK) return st;
  if (cache->plan_sig != p->sig)
    return fail(TASP_ERR_CACHE_PLAN_MISMATCH, "cache belongs to plan %016llx, not %016llx",
                (unsigned long long)cache->plan_sig, (unsigned long long)p->sig);
  if (pos < 0 || pos >= cache->max_seq)
    return fail(TASP_ERR_POS_RANGE, "pos %d outside 0..%d", pos, cache->max_seq - 1);
  const tasp_model_desc& d = p->desc;
  const int B = cache->batch, D = d.d_model, dh = d.head_dim, L = d.n_layers;
  const size_t out_elems = size_t(B) * (d.vocab ? d.vocab : D);
  const char* xb = reinterpret_cast<const char*>(x);
  const char* ob = reinterpret_cast<const char*>(out);
  if (ob < xb + size_t(B) * D * 4 && xb < ob + out_elems * 4)
    return fail(TASP_ERR_INVALID_ARG, "x and out overlap");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (B > 1) return decode_batched(p, x, cache, pos, out, s, tm, B);
  if (p->shared) return decode_shared(p, x, cache, pos, out, s, tm);

  for (int l = 0; l < L; ++l) {
    const LayerPlan& P = p->layers[l];
    const float* in = (l == 0) ? x : p->r_io[(l - 1) & 1];
    float* lo = (l == L - 1 && d.vocab == 0) ? out : p->r_io[l & 1];
    if (P.n_qkv > 0) {
      tasp::GemvArgs a{};
      a.w = P.qkv; a.scale = P.s_qkv; a.N = P.n_qkv; a.K = D; a.ld = D;
      a.x = in; a.ldx = D; a.gamma = P.an; a.eps = d.rms_eps; a.y = p->qkv_buf;
      a.ldy = p->ld_qkv; a.B = B;
      if ((st = run_kernel(tm, 0, s, [&] { return tasp::launch_gemv(tasp::GEMV_QKV, a, s); })))
        return st;
    }
    if (P.m_kv > 0) {
      const tasp::AttnArgs a = attn_args(p, l, cache, pos, B, false);
      if ((st = run_kernel(tm, 1, s, [&] { return tasp::launch_attn_decode(a, s); }))) return st;
    }
    {
      tasp::GemvArgs a{};
      a.w = P.o; a.scale = P.s_o; a.N = D; a.K = P.m_q * dh; a.ld = P.ld_o; a.x = p->o_buf;
      a.ldx = p->ld_obuf; a.resid = in; a.y = p->r_mid; a.ldy = D; a.B = B;
      if ((st = run_kernel(tm, 2, s, [&] { return tasp::launch_gemv(tasp::GEMV_RESID, a, s); })))
        return st;
    }
    if (P.c > 0) {
      const tasp::GemvArgs a = gateup_args(p, l, B);
      if ((st = run_kernel(tm, 3, s, [&] { return tasp::launch_gemv(tasp::GEMV_GATEUP, a, s); })))
        return st;
    }
    {
      const tasp::GemvArgs a = down_args(p, l, B, lo);
      if ((st = run_kernel(tm, 4, s, [&] { return tasp::launch_gemv(tasp::GEMV_RESID, a, s); })))
        return st;
    }
  }
  if (d.vocab) {
    tasp::GemvArgs a{};
    a.w = p->lm_head; a.N = d.vocab; a.K = D; a.ld = 2 * D; a.x = p->r_io[(L - 1) & 1];
    a.ldx = D; a.gamma = p->final_norm; a.eps = d.rms_eps; a.y = out; a.ldy = d.vocab; a.B = B;
    if ((st = run_kernel(tm, 5, s, [&] { return tasp::launch_gemv(tasp::GEMV_LMHEAD, a, s); })))
      return st;
  }
  return TASP_OK;
}

}  // namespace

// ------------------------------------------------------------------------------- C ABI
// (every entry point below is declared extern "C" in tasp.h; helpers between them sit in
// anonymous namespaces and stay internal)

const char* tasp_status_string(tasp_status s) {
  switch (s) {
    case TASP_OK: return "ok";
    case TASP_ERR_INVALID_ARG: return "invalid argument";
    case TASP_ERR_SHAPE: return "unsupported or inconsistent shape";
    case TASP_ERR_MASK: return "mask byte not 0 or 1";
    case TASP_ERR_WORKSPACE: return "workspace too small or misaligned";
    case TASP_ERR_POS_RANGE: return "position out of range";
    case TASP_ERR_CACHE_PLAN_MISMATCH: return "KV cache belongs to another plan";
    case TASP_ERR_HIP: return "HIP runtime error";
    case TASP_ERR_UNSUPPORTED: return "unsupported";
    case TASP_ERR_INTERNAL: return "internal consistency check failed";
  }
  return "unknown status";
}

const char* tasp_last_error(void) { return g_err.c_str(); }

tasp_status tasp_plan_workspace_bytes(const tasp_model_desc* desc, const tasp_mask* mask,
                                      size_t* bytes) {
  tasp_status st = check_desc(desc);
  if (st != TASP_OK) return st;
  if (!bytes) return fail(TASP_ERR_INVALID_ARG, "bytes is NULL");
  Closed c;
  if ((st = host_close(desc, mask, &c)) != TASP_OK) return st;
  *bytes = make_layout(desc, c).total;
  return TASP_OK;
}

namespace {

// Signature of a plan: the model shape, the RMSNorm epsilon and RoPE base, the closed mask, the
// store format (0 per-row panels, 1 groupwise shared store) and the store's identity (a hash of
// every device address it names); equal signatures mean interchangeable cache contents. Two
// stores at distinct addresses, or one mask under another epsilon or RoPE base, never share a
// cache. (A store freed and re-filled at the same addresses keeps its identity: the caller owns
// that lifetime.)
uint64_t plan_signature(const tasp_model_desc& d, const Closed& c, int32_t format,
                        uint64_t store_id) {
  uint64_t sig = 1469598103934665603ull;
  const int32_t shape[7] = {d.n_layers, d.d_model, d.n_q_heads, d.n_kv_heads, d.head_dim, d.d_ffn, d.vocab};
  sig = fnv1a(sig, shape, sizeof shape);
  sig = fnv1a(sig, &d.rms_eps, sizeof d.rms_eps);
  sig = fnv1a(sig, &d.rope_theta, sizeof d.rope_theta);
  sig = fnv1a(sig, c.q.data(), c.q.size());
  sig = fnv1a(sig, c.kv.data(), c.kv.size());
  sig = fnv1a(sig, c.f.data(), c.f.size());
  sig = fnv1a(sig, &format, sizeof format);
  sig = fnv1a(sig, &store_id, sizeof store_id);
  return sig ? sig : 1;
}

uint64_t hash_ptrs(uint64_t h, std::initializer_list<const void*> ptrs) {
  for (const void* q : ptrs) {
    const uintptr_t v = reinterpret_cast<uintptr_t>(q);
    h = fnv1a(h, &v, sizeof v);
  }
  return h;
}

// identity of a per-row INT8 store: every weight, scale and gain address it names
uint64_t store_identity(const tasp_store& st, int n_layers) {
  uint64_t h = 1469598103934665603ull;
  for (int l = 0; l < n_layers; ++l) {
    const tasp_layer& S = st.layers[l];
    h = hash_ptrs(h, {S.wq.w, S.wq.scale, S.wk.w, S.wk.scale, S.wv.w, S.wv.scale, S.wo.w,
                      S.wo.scale, S.wg.w, S.wg.scale, S.wu.w, S.wu.scale, S.wd.w, S.wd.scale,
                      S.attn_norm, S.ffn_norm});
  }
  return hash_ptrs(h, {st.final_norm, st.lm_head});
}

// identity of a groupwise shared store
uint64_t store_identity(const tasp_gstore& st, int n_layers) {
  uint64_t h = 1099511628211ull;
  for (int l = 0; l < n_layers; ++l) {
    const tasp_glayer& S = st.layers[l];
    h = hash_ptrs(h, {S.wqkv.w, S.wqkv.scale, S.wo.w, S.wo.scale, S.wg.w, S.wg.scale, S.wu.w,
                      S.wu.scale, S.wd.w, S.wd.scale, S.attn_norm, S.ffn_norm});
  }
  return hash_ptrs(h, {st.final_norm, st.lm_head});
}

// A shared-store plan: its scale groups of 128 must tile every input dimension, and its widest
// batch-1 GEMV input (with the piece sums and the column map) must fit LDS.
tasp_status check_shared_desc(const tasp_model_desc* d) {
  tasp_status st = check_desc(d);
  if (st != TASP_OK) return st;
  if (d->d_model % 128 || (d->n_q_heads * d->head_dim) % 128 || d->d_ffn % 128)
    return fail(TASP_ERR_SHAPE, "the groupwise store needs d_model, n_q_heads*head_dim and d_ffn "
                "divisible by 128");
  const int widest = std::max({d->d_model, d->n_q_heads * d->head_dim, d->d_ffn});
  if (tasp::shared_gemv_lds_bytes(widest) > tasp::kMaxSharedGemvLds)
    return fail(TASP_ERR_UNSUPPORTED, "widest GEMV input exceeds LDS (%d)", widest);
  return TASP_OK;
}

// Reads the device index lists back (the compile's one synchronisation; `h` carries the status of
// the work enqueued before it), checks them against the host closure and keeps them in the plan.
tasp_status read_back_indices(tasp_plan_s* p, const Closed& c, const Layout& Y, char* ws,
                              hipStream_t s, hipError_t h) {
  const tasp_model_desc& d = p->desc;
  const int L = d.n_layers, Hq = d.n_q_heads, Hkv = d.n_kv_heads, F = d.d_ffn;
  auto at = [&](size_t off) { return ws + off; };
  int* dq = reinterpret_cast<int*>(at(Y.idx_q));
  int* dkv = reinterpret_cast<int*>(at(Y.idx_kv));
  int* dslot = reinterpret_cast<int*>(at(Y.idx_slot));
  int* dss = reinterpret_cast<int*>(at(Y.idx_slot_start));
  int* dffn = reinterpret_cast<int*>(at(Y.idx_ffn));
  int* dcnt = reinterpret_cast<int*>(at(Y.counts));
  // read the device index lists back (the one synchronisation) and check them
  std::vector<int> hq_idx(size_t(L) * Hq), hkv_idx(size_t(L) * Hkv), hslot(size_t(L) * Hq),
      hffn(size_t(L) * F), hcnt(size_t(L) * 4);
  if (h == hipSuccess) h = hipMemcpyAsync(hq_idx.data(), dq, hq_idx.size() * 4, hipMemcpyDeviceToHost, s);
  if (h == hipSuccess) h = hipMemcpyAsync(hkv_idx.data(), dkv, hkv_idx.size() * 4, hipMemcpyDeviceToHost, s);
  if (h == hipSuccess) h = hipMemcpyAsync(hslot.data(), dslot, hslot.size() * 4, hipMemcpyDeviceToHost, s);
  if (h == hipSuccess) h = hipMemcpyAsync(hffn.data(), dffn, hffn.size() * 4, hipMemcpyDeviceToHost, s);
  if (h == hipSuccess) h = hipMemcpyAsync(hcnt.data(), dcnt, hcnt.size() * 4, hipMemcpyDeviceToHost, s);
  if (h == hipSuccess) h = hipStreamSynchronize(s);
  if (h != hipSuccess) {
    (void)hipStreamSynchronize(s);
    return fail(TASP_ERR_HIP, "compile: %s", hipGetErrorString(h));
  }
  const int r = Hq / Hkv;
  for (int l = 0; l < L; ++l) {
    LayerPlan& P = p->layers[l];
    if (hcnt[l * 4] != P.m_q || hcnt[l * 4 + 1] != P.m_kv || hcnt[l * 4 + 2] != P.c) {
      return fail(TASP_ERR_INTERNAL, "layer %d: device counts (%d,%d,%d) != host (%d,%d,%d)", l,
                  hcnt[l * 4], hcnt[l * 4 + 1], hcnt[l * 4 + 2], P.m_q, P.m_kv, P.c);
    }
    P.q_idx.assign(hq_idx.begin() + size_t(l) * Hq, hq_idx.begin() + size_t(l) * Hq + P.m_q);
    P.q_kvslot.assign(hslot.begin() + size_t(l) * Hq, hslot.begin() + size_t(l) * Hq + P.m_q);
    P.kv_idx.assign(hkv_idx.begin() + size_t(l) * Hkv, hkv_idx.begin() + size_t(l) * Hkv + P.m_kv);
    P.ffn_idx.assign(hffn.begin() + size_t(l) * F, hffn.begin() + size_t(l) * F + P.c);
    bool ok = true;
    int k = 0;
    for (int hh = 0; hh < Hq; ++hh)
      if (c.q[size_t(l) * Hq + hh]) ok &= (k < P.m_q && P.q_idx[k++] == hh);
    k = 0;
    for (int g = 0; g < Hkv; ++g)
      if (c.kv[size_t(l) * Hkv + g]) ok &= (k < P.m_kv && P.kv_idx[k++] == g);
    k = 0;
    for (int j = 0; j < F; ++j)
      if (c.f[size_t(l) * F + j]) ok &= (k < P.c && P.ffn_idx[k++] == j);
    for (int i = 0; i < P.m_q && ok; ++i)
      ok &= P.q_kvslot[i] >= 0 && P.q_kvslot[i] < P.m_kv && P.kv_idx[P.q_kvslot[i]] == P.q_idx[i] / r;
    // slot j's heads are the run of the ascending head list whose slot is j
    P.slot_start.assign(size_t(P.m_kv) + 1, 0);
    for (int jj = 0; jj <= P.m_kv; ++jj)
      for (int i = 0; i < P.m_q; ++i) P.slot_start[jj] += (P.q_kvslot[i] < jj);
    for (int jj = 0; jj < P.m_kv && ok; ++jj) ok &= P.slot_start[jj + 1] > P.slot_start[jj];
    std::vector<int> dev_ss(size_t(Hkv) + 1);
    if (ok && hipMemcpy(dev_ss.data(), dss + size_t(l) * (Hkv + 1), (P.m_kv + 1) * sizeof(int),
                        hipMemcpyDeviceToHost) == hipSuccess) {
      for (int jj = 0; jj <= P.m_kv; ++jj) ok &= dev_ss[jj] == P.slot_start[jj];
    } else {
      ok = false;
    }
    if (!ok) return fail(TASP_ERR_INTERNAL, "layer %d: device index lists differ from the host closure", l);
  }
  return TASP_OK;
}

}  // namespace

tasp_status tasp_compile_plan(const tasp_model_desc* desc, const tasp_store* store,
                              const tasp_mask* mask, void* workspace, size_t workspace_bytes,
                              void* stream, tasp_plan* out) {
  tasp_status st = check_desc(desc);
  if (st != TASP_OK) return st;
  if (!store || !store->layers || !out) return fail(TASP_ERR_INVALID_ARG, "store / out is NULL");
  if (!workspace) return fail(TASP_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(TASP_ERR_WORKSPACE, "workspace not %zu-byte aligned", kAlign);
  const tasp_model_desc& d = *desc;
  for (int l = 0; l < d.n_layers; ++l) {
    const tasp_layer& S = store->layers[l];
    const tasp_qmat* mats[7] = {&S.wq, &S.wk, &S.wv, &S.wo, &S.wg, &S.wu, &S.wd};
    for (const tasp_qmat* m : mats)
      if (!m->w || !m->scale) return fail(TASP_ERR_INVALID_ARG, "layer %d: NULL weight", l);
    if (!S.attn_norm || !S.ffn_norm) return fail(TASP_ERR_INVALID_ARG, "layer %d: NULL gain", l);
    for (const tasp_qmat* m : mats)
      if (reinterpret_cast<uintptr_t>(m->w) % 16)
        return fail(TASP_ERR_INVALID_ARG, "layer %d: weight not 16-byte aligned", l);
  }
  if (d.vocab && (!store->final_norm || !store->lm_head))
    return fail(TASP_ERR_INVALID_ARG, "vocab > 0 but final_norm / lm_head is NULL");
  Closed c;
  if ((st = host_close(desc, mask, &c)) != TASP_OK) return st;
  const Layout Y = make_layout(desc, c);
  if (workspace_bytes < Y.total)
    return fail(TASP_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, Y.total);

  const int L = d.n_layers, D = d.d_model, Hq = d.n_q_heads, Hkv = d.n_kv_heads;
  const int dh = d.head_dim, F = d.d_ffn;
  char* ws = static_cast<char*>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto at = [&](size_t off) { return ws + off; };

  // device closure over the caller's (possibly not closed) mask bits
  std::vector<uint8_t> ones_q, ones_f;
  const uint8_t* hq = mask ? mask->q_keep : nullptr;
  const uint8_t* hf = mask ? mask->ffn_keep : nullptr;
  if (!hq) { ones_q.assign(size_t(L) * Hq, 1); hq = ones_q.data(); }
  if (!hf) { ones_f.assign(size_t(L) * F, 1); hf = ones_f.data(); }
  const bool has_kv = mask && mask->kv_keep;
  HIP_TRY(hipMemcpyAsync(at(Y.mask_q), hq, size_t(L) * Hq, hipMemcpyHostToDevice, s));
  if (has_kv)
    HIP_TRY(hipMemcpyAsync(at(Y.mask_kv), mask->kv_keep, size_t(L) * Hkv, hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(at(Y.mask_f), hf, size_t(L) * F, hipMemcpyHostToDevice, s));
  int* dq = reinterpret_cast<int*>(at(Y.idx_q));
  int* dkv = reinterpret_cast<int*>(at(Y.idx_kv));
  int* dslot = reinterpret_cast<int*>(at(Y.idx_slot));
  int* dss = reinterpret_cast<int*>(at(Y.idx_slot_start));
  int* dffn = reinterpret_cast<int*>(at(Y.idx_ffn));
  int* dcnt = reinterpret_cast<int*>(at(Y.counts));
  HIP_TRY(tasp::launch_closure(reinterpret_cast<uint8_t*>(at(Y.mask_q)),
                               has_kv ? reinterpret_cast<uint8_t*>(at(Y.mask_kv)) : nullptr,
                               reinterpret_cast<uint8_t*>(at(Y.mask_f)), L, Hq, Hkv, F, dq, dkv,
                               dslot, dss, dffn, dcnt, s));

  tasp_plan_s* p = new (std::nothrow) tasp_plan_s();
  if (!p) return fail(TASP_ERR_INTERNAL, "out of host memory");
  p->desc = d;
  p->layers.resize(L);
  for (int l = 0; l < L; ++l) {
    const LayerLayout& Q = Y.layers[l];
    const tasp_layer& S = store->layers[l];
    LayerPlan& P = p->layers[l];
    P.m_q = c.m_q[l]; P.m_kv = c.m_kv[l]; P.c = c.c[l];
    P.n_qkv = Q.n_qkv; P.ld_o = Q.ld_o; P.ld_d = Q.ld_d;
    P.qkv = reinterpret_cast<int8_t*>(at(Q.qkv)); P.s_qkv = reinterpret_cast<float*>(at(Q.s_qkv));
    P.o = reinterpret_cast<int8_t*>(at(Q.o)); P.s_o = reinterpret_cast<float*>(at(Q.s_o));
    P.g = reinterpret_cast<int8_t*>(at(Q.g)); P.u = reinterpret_cast<int8_t*>(at(Q.u));
    P.s_g = reinterpret_cast<float*>(at(Q.s_g)); P.s_u = reinterpret_cast<float*>(at(Q.s_u));
    P.dn = reinterpret_cast<int8_t*>(at(Q.dn)); P.s_d = reinterpret_cast<float*>(at(Q.s_d));
    P.an = reinterpret_cast<uint16_t*>(at(Q.an)); P.fn = reinterpret_cast<uint16_t*>(at(Q.fn));
    const int* lq = dq + size_t(l) * Hq;
    const int* lkv = dkv + size_t(l) * Hkv;
    const int* lf = dffn + size_t(l) * F;
    tasp_status e = TASP_OK;
    auto chk = [&](hipError_t h) {
      if (h != hipSuccess && e == TASP_OK) e = fail(TASP_ERR_HIP, "gather: %s", hipGetErrorString(h));
    };
    const int mq = P.m_q, mkv = P.m_kv;
    chk(tasp::launch_gather_head_rows(P.qkv, S.wq.w, lq, mq, dh, D, P.s_qkv, S.wq.scale, s));
    chk(tasp::launch_gather_head_rows(P.qkv + size_t(mq) * dh * D, S.wk.w, lkv, mkv, dh, D,
                                      P.s_qkv + mq * dh, S.wk.scale, s));
    chk(tasp::launch_gather_head_rows(P.qkv + size_t(mq + mkv) * dh * D, S.wv.w, lkv, mkv, dh, D,
                                      P.s_qkv + (mq + mkv) * dh, S.wv.scale, s));
    chk(tasp::launch_gather_head_cols(P.o, P.ld_o, S.wo.w, Hq * dh, lq, mq, dh, D, s));
    chk(tasp::launch_copy(P.s_o, S.wo.scale, size_t(D) * 4, s));
    chk(tasp::launch_gather_rows(P.g, S.wg.w, lf, P.c, D, P.s_g, S.wg.scale, s));
    chk(tasp::launch_gather_rows(P.u, S.wu.w, lf, P.c, D, P.s_u, S.wu.scale, s));
    chk(tasp::launch_gather_cols(P.dn, P.ld_d, S.wd.w, F, lf, P.c, D, s));
    chk(tasp::launch_copy(P.s_d, S.wd.scale, size_t(D) * 4, s));
    chk(tasp::launch_copy(P.an, S.attn_norm, size_t(D) * 2, s));
    chk(tasp::launch_copy(P.fn, S.ffn_norm, size_t(D) * 2, s));
    if (e != TASP_OK) { (void)hipStreamSynchronize(s); delete p; return e; }
  }
  if (d.vocab) {
    p->final_norm = reinterpret_cast<uint16_t*>(at(Y.final_norm));
    p->lm_head = reinterpret_cast<uint16_t*>(at(Y.lm_head));
    hipError_t h = tasp::launch_copy(p->final_norm, store->final_norm, size_t(D) * 2, s);
    if (h == hipSuccess) h = tasp::launch_copy(p->lm_head, store->lm_head, size_t(d.vocab) * D * 2, s);
    if (h != hipSuccess) {
      (void)hipStreamSynchronize(s);
      delete p;
      return fail(TASP_ERR_HIP, "LM head copy: %s", hipGetErrorString(h));
    }
  } else {
    p->final_norm = p->lm_head = nullptr;
  }
  // rotary table: angle pos * theta^(-2i/dh) evaluated in double, stored as float
  const int half = dh / 2;
  std::vector<float> tc(size_t(d.max_seq) * half), ts(size_t(d.max_seq) * half);
  for (int t = 0; t < d.max_seq; ++t)
    for (int i = 0; i < half; ++i) {
      const double ang = double(t) * std::pow(d.rope_theta, -2.0 * i / dh);
      tc[size_t(t) * half + i] = float(std::cos(ang));
      ts[size_t(t) * half + i] = float(std::sin(ang));
    }
  p->rope_cos = reinterpret_cast<float*>(at(Y.rope_cos));
  p->rope_sin = reinterpret_cast<float*>(at(Y.rope_sin));
  hipError_t h = hipMemcpyAsync(p->rope_cos, tc.data(), tc.size() * 4, hipMemcpyHostToDevice, s);
  if (h == hipSuccess) h = hipMemcpyAsync(p->rope_sin, ts.data(), ts.size() * 4, hipMemcpyHostToDevice, s);
  if (h == hipSuccess) h = tasp::launch_fill_zero(at(Y.zero_begin), Y.zero_end - Y.zero_begin, s);
  set_scratch(p, Y, ws);

  {
    const tasp_status rb = read_back_indices(p, c, Y, ws, s, h);
    if (rb != TASP_OK) {
      delete p;
      return rb;
    }
  }
  // ledger and signature
  double num = 0.0, den = 0.0;
  uint64_t wb = 0, sb = 0;
  for (int l = 0; l < L; ++l) {
    const LayerPlan& P = p->layers[l];
    num += layer_flops(desc, P.m_q, P.m_kv, P.c);
    den += layer_flops(desc, Hq, Hkv, F);
    wb += uint64_t(P.n_qkv) * D + uint64_t(D) * P.m_q * dh + 3ull * D * P.c;
    sb += 4ull * (uint64_t(P.n_qkv) + D + 2ull * P.c + D);
  }
  p->ratio = num / den;
  p->weight_bytes = wb;
  p->scale_bytes = sb;
  p->sig = plan_signature(d, c, 0, store_identity(*store, L));
  *out = p;
  return TASP_OK;
}

tasp_status tasp_shared_plan_workspace_bytes(const tasp_model_desc* desc, size_t* plan_bytes,
                                             size_t* scratch_bytes) {
  if (!plan_bytes || !scratch_bytes) return fail(TASP_ERR_INVALID_ARG, "plan_bytes / scratch_bytes is NULL");
  tasp_status st = check_shared_desc(desc);
  if (st != TASP_OK) return st;
  const Layout Y = make_shared_layout(desc);
  *plan_bytes = Y.total;
  *scratch_bytes = Y.scratch_total;
  return TASP_OK;
}

tasp_status tasp_compile_shared_plan(const tasp_model_desc* desc, const tasp_gstore* store,
                                     const tasp_mask* mask, void* workspace,
                                     size_t workspace_bytes, void* scratch, size_t scratch_bytes,
                                     void* stream, tasp_plan* out) {
  tasp_status st = check_shared_desc(desc);
  if (st != TASP_OK) return st;
  if (!store || !store->layers || !out) return fail(TASP_ERR_INVALID_ARG, "store / out is NULL");
  if (!workspace) return fail(TASP_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign || reinterpret_cast<uintptr_t>(scratch) % kAlign)
    return fail(TASP_ERR_WORKSPACE, "workspace / scratch not %zu-byte aligned", kAlign);
  const tasp_model_desc& d = *desc;
  for (int l = 0; l < d.n_layers; ++l) {
    const tasp_glayer& S = store->layers[l];
    const tasp_gqmat* mats[5] = {&S.wqkv, &S.wo, &S.wg, &S.wu, &S.wd};
    for (const tasp_gqmat* m : mats) {
      if (!m->w || !m->scale) return fail(TASP_ERR_INVALID_ARG, "layer %d: NULL weight", l);
      if (reinterpret_cast<uintptr_t>(m->w) % 16 || reinterpret_cast<uintptr_t>(m->scale) % 2)
        return fail(TASP_ERR_INVALID_ARG, "layer %d: weight not 16-byte / scale not 2-byte aligned", l);
    }
    if (!S.attn_norm || !S.ffn_norm) return fail(TASP_ERR_INVALID_ARG, "layer %d: NULL gain", l);
  }
  if (d.vocab && (!store->final_norm || !store->lm_head))
    return fail(TASP_ERR_INVALID_ARG, "vocab > 0 but final_norm / lm_head is NULL");
  Closed c;
  if ((st = host_close(desc, mask, &c)) != TASP_OK) return st;
  const int L = d.n_layers, Hq = d.n_q_heads, Hkv = d.n_kv_heads, dh = d.head_dim, F = d.d_ffn;
  // W_down columns are read 16 at a time: retained channels must come in aligned blocks of 16
  for (int l = 0; l < L; ++l)
    for (int j0 = 0; j0 < F; j0 += 16)
      for (int j = j0 + 1; j < j0 + 16; ++j)
        if (c.f[size_t(l) * F + j] != c.f[size_t(l) * F + j0])
          return fail(TASP_ERR_UNSUPPORTED,
                      "layer %d: channels %d..%d are partly retained (shared-store plans keep "
                      "channels in aligned blocks of 16)", l, j0, j0 + 15);
  const Layout Y = make_shared_layout(desc);
  // the scratch arena: the caller's (shareable), else the workspace's tail
  const size_t need = scratch ? Y.total : Y.total + Y.scratch_total;
  if (workspace_bytes < need)
    return fail(TASP_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, need);
  if (scratch && scratch_bytes < Y.scratch_total)
    return fail(TASP_ERR_WORKSPACE, "scratch %zu < %zu bytes", scratch_bytes, Y.scratch_total);
  char* ws = static_cast<char*>(workspace);
  char* sc = scratch ? static_cast<char*>(scratch) : ws + Y.total;
  hipStream_t s = static_cast<hipStream_t>(stream);
  auto at = [&](size_t off) { return ws + off; };

  std::vector<uint8_t> ones_q, ones_f;
  const uint8_t* hq = mask ? mask->q_keep : nullptr;
  const uint8_t* hf = mask ? mask->ffn_keep : nullptr;
  if (!hq) { ones_q.assign(size_t(L) * Hq, 1); hq = ones_q.data(); }
  if (!hf) { ones_f.assign(size_t(L) * F, 1); hf = ones_f.data(); }
  const bool has_kv = mask && mask->kv_keep;
  HIP_TRY(hipMemcpyAsync(at(Y.mask_q), hq, size_t(L) * Hq, hipMemcpyHostToDevice, s));
  if (has_kv)
    HIP_TRY(hipMemcpyAsync(at(Y.mask_kv), mask->kv_keep, size_t(L) * Hkv, hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(at(Y.mask_f), hf, size_t(L) * F, hipMemcpyHostToDevice, s));
  int* dq = reinterpret_cast<int*>(at(Y.idx_q));
  int* dkv = reinterpret_cast<int*>(at(Y.idx_kv));
  int* dffn = reinterpret_cast<int*>(at(Y.idx_ffn));
  int* dcnt = reinterpret_cast<int*>(at(Y.counts));
  HIP_TRY(tasp::launch_closure(reinterpret_cast<uint8_t*>(at(Y.mask_q)),
                               has_kv ? reinterpret_cast<uint8_t*>(at(Y.mask_kv)) : nullptr,
                               reinterpret_cast<uint8_t*>(at(Y.mask_f)), L, Hq, Hkv, F, dq, dkv,
                               reinterpret_cast<int*>(at(Y.idx_slot)),
                               reinterpret_cast<int*>(at(Y.idx_slot_start)), dffn, dcnt, s));
  tasp::SharedMapsArgs ma{Hq, Hkv, dh, F, dq, dkv, dffn, dcnt,
                          reinterpret_cast<int*>(at(Y.qkv_rows)), reinterpret_cast<int*>(at(Y.o_cols)),
                          reinterpret_cast<int*>(at(Y.down_cols))};
  HIP_TRY(tasp::launch_shared_maps(ma, L, s));

  tasp_plan_s* p = new (std::nothrow) tasp_plan_s();
  if (!p) return fail(TASP_ERR_INTERNAL, "out of host memory");
  p->desc = d;
  p->shared = true;
  p->layers.resize(L);
  p->sl.resize(L);
  for (int l = 0; l < L; ++l) {
    const tasp_glayer& S = store->layers[l];
    LayerPlan& P = p->layers[l];
    P.m_q = c.m_q[l]; P.m_kv = c.m_kv[l]; P.c = c.c[l];
    P.n_qkv = (P.m_q + 2 * P.m_kv) * dh; P.ld_o = P.m_q * dh; P.ld_d = P.c;
    P.qkv = P.o = P.g = P.u = P.dn = nullptr;
    P.s_qkv = P.s_o = P.s_g = P.s_u = P.s_d = nullptr;
    P.an = const_cast<uint16_t*>(S.attn_norm);
    P.fn = const_cast<uint16_t*>(S.ffn_norm);
    SharedLayer& Q = p->sl[l];
    Q.qkv = S.wqkv.w; Q.o = S.wo.w; Q.g = S.wg.w; Q.u = S.wu.w; Q.d = S.wd.w;
    Q.s_qkv = S.wqkv.scale; Q.s_o = S.wo.scale; Q.s_g = S.wg.scale; Q.s_u = S.wu.scale;
    Q.s_d = S.wd.scale;
    Q.qkv_rows = reinterpret_cast<int*>(at(Y.qkv_rows)) + size_t(l) * (Hq + 2 * Hkv) * dh;
    Q.o_cols = reinterpret_cast<int*>(at(Y.o_cols)) + size_t(l) * (Hq * dh / 16);
    Q.ffn_rows = dffn + size_t(l) * F;
    Q.down_cols = reinterpret_cast<int*>(at(Y.down_cols)) + size_t(l) * (F / 16);
  }
  p->final_norm = d.vocab ? const_cast<uint16_t*>(store->final_norm) : nullptr;
  p->lm_head = d.vocab ? const_cast<uint16_t*>(store->lm_head) : nullptr;
  const int half = dh / 2;
  std::vector<float> tc(size_t(d.max_seq) * half), ts(size_t(d.max_seq) * half);
  for (int t = 0; t < d.max_seq; ++t)
    for (int i = 0; i < half; ++i) {
      const double ang = double(t) * std::pow(d.rope_theta, -2.0 * i / dh);
      tc[size_t(t) * half + i] = float(std::cos(ang));
      ts[size_t(t) * half + i] = float(std::sin(ang));
    }
  p->rope_cos = reinterpret_cast<float*>(at(Y.rope_cos));
  p->rope_sin = reinterpret_cast<float*>(at(Y.rope_sin));
  hipError_t h = hipMemcpyAsync(p->rope_cos, tc.data(), tc.size() * 4, hipMemcpyHostToDevice, s);
  if (h == hipSuccess) h = hipMemcpyAsync(p->rope_sin, ts.data(), ts.size() * 4, hipMemcpyHostToDevice, s);
  if (h == hipSuccess) h = tasp::launch_fill_zero(sc + Y.zero_begin, Y.zero_end - Y.zero_begin, s);
  set_scratch(p, Y, sc);
  if ((st = read_back_indices(p, c, Y, ws, s, h)) != TASP_OK) {
    delete p;
    return st;
  }
  // the maps, checked against the host's reading of the index lists
  {
    std::vector<int> qr(size_t(L) * (Hq + 2 * Hkv) * dh), oc(size_t(L) * (Hq * dh / 16)),
        dc(size_t(L) * (F / 16));
    h = hipMemcpy(qr.data(), at(Y.qkv_rows), qr.size() * 4, hipMemcpyDeviceToHost);
    if (h == hipSuccess) h = hipMemcpy(oc.data(), at(Y.o_cols), oc.size() * 4, hipMemcpyDeviceToHost);
    if (h == hipSuccess) h = hipMemcpy(dc.data(), at(Y.down_cols), dc.size() * 4, hipMemcpyDeviceToHost);
    if (h != hipSuccess) {
      delete p;
      return fail(TASP_ERR_HIP, "compile: %s", hipGetErrorString(h));
    }
    for (int l = 0; l < L; ++l) {
      const LayerPlan& P = p->layers[l];
      bool ok = true;
      const int* lq = qr.data() + size_t(l) * (Hq + 2 * Hkv) * dh;
      for (int i = 0; i < P.m_q; ++i)
        for (int e = 0; e < dh; ++e) ok &= lq[i * dh + e] == P.q_idx[i] * dh + e;
      for (int j = 0; j < P.m_kv; ++j)
        for (int e = 0; e < dh; ++e) {
          ok &= lq[(P.m_q + j) * dh + e] == (Hq + P.kv_idx[j]) * dh + e;
          ok &= lq[(P.m_q + P.m_kv + j) * dh + e] == (Hq + Hkv + P.kv_idx[j]) * dh + e;
        }
      const int* lo = oc.data() + size_t(l) * (Hq * dh / 16);
      for (int q = 0; q < P.m_q * dh / 16; ++q) ok &= lo[q] == P.q_idx[q * 16 / dh] * dh + (q * 16) % dh;
      const int* ld = dc.data() + size_t(l) * (F / 16);
      for (int q = 0; q < P.c / 16; ++q) ok &= ld[q] == P.ffn_idx[q * 16];
      if (!ok) {
        delete p;
        return fail(TASP_ERR_INTERNAL, "layer %d: device maps differ from the index lists", l);
      }
    }
  }
  double num = 0.0, den = 0.0;
  uint64_t wb = 0, sb = 0;
  const int D = d.d_model;
  for (int l = 0; l < L; ++l) {
    const LayerPlan& P = p->layers[l];
    num += layer_flops(desc, P.m_q, P.m_kv, P.c);
    den += layer_flops(desc, Hq, Hkv, F);
    wb += uint64_t(P.n_qkv) * D + uint64_t(D) * P.m_q * dh + 3ull * D * P.c;
    // one BF16 scale per 128 weights read
    sb += 2ull * ((uint64_t(P.n_qkv) * D + uint64_t(D) * P.m_q * dh + 3ull * D * P.c) / 128);
  }
  p->ratio = num / den;
  p->weight_bytes = wb;
  p->scale_bytes = sb;
  p->sig = plan_signature(d, c, 1, store_identity(*store, L));
  *out = p;
  return TASP_OK;
}

tasp_status tasp_plan_counts(tasp_plan p, int32_t layer, int32_t* m_q, int32_t* m_kv,
                             int32_t* n_ffn) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  if (layer < 0 || layer >= p->desc.n_layers) return fail(TASP_ERR_INVALID_ARG, "bad layer %d", layer);
  const LayerPlan& P = p->layers[layer];
  if (m_q) *m_q = P.m_q;
  if (m_kv) *m_kv = P.m_kv;
  if (n_ffn) *n_ffn = P.c;
  return TASP_OK;
}

tasp_status tasp_plan_indices(tasp_plan p, int32_t layer, int32_t which, int32_t* dst,
                              int32_t cap, int32_t* n) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  if (layer < 0 || layer >= p->desc.n_layers) return fail(TASP_ERR_INVALID_ARG, "bad layer %d", layer);
  const LayerPlan& P = p->layers[layer];
  const std::vector<int>* v = nullptr;
  switch (which) {
    case TASP_IDX_Q: v = &P.q_idx; break;
    case TASP_IDX_KV: v = &P.kv_idx; break;
    case TASP_IDX_QKVSLOT: v = &P.q_kvslot; break;
    case TASP_IDX_FFN: v = &P.ffn_idx; break;
    default: return fail(TASP_ERR_INVALID_ARG, "bad index list %d", which);
  }
  if (n) *n = int32_t(v->size());
  if (!dst) return TASP_OK;
  if (cap < int32_t(v->size())) return fail(TASP_ERR_INVALID_ARG, "cap %d < %zu", cap, v->size());
  std::copy(v->begin(), v->end(), dst);
  return TASP_OK;
}

tasp_status tasp_plan_panel(tasp_plan p, int32_t layer, int32_t which, const int8_t** w,
                            const float** scale, int64_t* rows, int64_t* cols, int64_t* ld) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  if (layer < 0 || layer >= p->desc.n_layers) return fail(TASP_ERR_INVALID_ARG, "bad layer %d", layer);
  if (p->shared) return fail(TASP_ERR_UNSUPPORTED, "a shared-store plan owns no panels");
  const LayerPlan& P = p->layers[layer];
  const int D = p->desc.d_model;
  const int8_t* pw;
  const float* ps;
  int64_t r, c, l;
  switch (which) {
    case TASP_PANEL_QKV: pw = P.qkv; ps = P.s_qkv; r = P.n_qkv; c = D; l = D; break;
    case TASP_PANEL_O: pw = P.o; ps = P.s_o; r = D; c = int64_t(P.m_q) * p->desc.head_dim; l = P.ld_o; break;
    case TASP_PANEL_GATE: pw = P.g; ps = P.s_g; r = P.c; c = D; l = D; break;
    case TASP_PANEL_UP: pw = P.u; ps = P.s_u; r = P.c; c = D; l = D; break;
    case TASP_PANEL_DOWN: pw = P.dn; ps = P.s_d; r = D; c = P.c; l = P.ld_d; break;
    default: return fail(TASP_ERR_INVALID_ARG, "bad panel %d", which);
  }
  if (w) *w = pw;
  if (scale) *scale = ps;
  if (rows) *rows = r;
  if (cols) *cols = c;
  if (ld) *ld = l;
  return TASP_OK;
}

tasp_status tasp_plan_ledger(tasp_plan p, double* ratio, uint64_t* weight_bytes,
                             uint64_t* scale_bytes, uint64_t* signature) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  if (ratio) *ratio = p->ratio;
  if (weight_bytes) *weight_bytes = p->weight_bytes;
  if (scale_bytes) *scale_bytes = p->scale_bytes;
  if (signature) *signature = p->sig;
  return TASP_OK;
}

tasp_status tasp_plan_destroy(tasp_plan p) {
  delete p;
  return TASP_OK;
}

tasp_status tasp_kv_bind(tasp_plan p, tasp_kv_cache* cache) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  tasp_status st = check_cache(p, cache);
  if (st != TASP_OK) return st;
  cache->plan_sig = p->sig;
  return TASP_OK;
}

tasp_status tasp_decode_step(tasp_plan p, const float* x, tasp_kv_cache* cache, int32_t pos,
                             float* out, void* stream) {
  return decode_impl(p, x, cache, pos, out, stream, nullptr);
}

tasp_status tasp_decode_step_timed(tasp_plan p, const float* x, tasp_kv_cache* cache,
                                   int32_t pos, float* out, void* stream, float* kernel_ms,
                                   int32_t* kinds, int32_t cap, int32_t* n) {
  if (!kernel_ms || !kinds || !n) return fail(TASP_ERR_INVALID_ARG, "timing outputs are NULL");
  Timer tm;
  tasp_status st = decode_impl(p, x, cache, pos, out, stream, &tm);
  return finish_timed(st, &tm, static_cast<hipStream_t>(stream), kernel_ms, kinds, cap, n, "timed decode");
}

tasp_status tasp_prefill(tasp_plan p, const float* x, int32_t T, tasp_kv_cache* cache,
                         int32_t pos0, float* out, void* stream) {
  return prefill_checked(p, x, T, cache, pos0, out, stream, nullptr);
}

tasp_status tasp_prefill_last(tasp_plan p, const float* x, int32_t T, tasp_kv_cache* cache,
                              int32_t pos0, float* out, void* stream) {
  return prefill_checked(p, x, T, cache, pos0, out, stream, nullptr, true);
}

tasp_status tasp_prefill_timed(tasp_plan p, const float* x, int32_t T, tasp_kv_cache* cache,
                               int32_t pos0, float* out, void* stream, float* kernel_ms,
                               int32_t* kinds, int32_t cap, int32_t* n) {
  if (!kernel_ms || !kinds || !n) return fail(TASP_ERR_INVALID_ARG, "timing outputs are NULL");
  Timer tm;
  tasp_status st = prefill_checked(p, x, T, cache, pos0, out, stream, &tm);
  return finish_timed(st, &tm, static_cast<hipStream_t>(stream), kernel_ms, kinds, cap, n, "timed prefill");
}

tasp_status tasp_profile_stage(const tasp_plan* plans, const tasp_kv_cache* caches,
                               int32_t n_plans, int32_t layer, int32_t kind, int32_t pos,
                               int32_t reps, void* stream, float* ms_per_launch) {
  if (!plans || !caches || n_plans < 1 || reps < 1 || !ms_per_launch)
    return fail(TASP_ERR_INVALID_ARG, "plans / caches / n_plans / reps / ms_per_launch");
  if (kind != 1 && kind != 3 && kind != 4)
    return fail(TASP_ERR_UNSUPPORTED, "stage kind %d is not profiled", kind);
  // one launch per (layer, plan); layer -1 takes every layer that has the stage, in order
  struct Item {
    int plan, layer;
    bool shared;
    tasp::GemvArgs g;
    tasp::MfmaArgs m;
    tasp::AttnArgs at;
    tasp::SharedGemvArgs sg;
  };
  std::vector<Item> items;
  int batch = 0;
  for (int i = 0; i < n_plans; ++i) {
    const tasp_plan_s* p = plans[i];
    if (!p) return fail(TASP_ERR_INVALID_ARG, "plans[%d] is NULL", i);
    tasp_status st = check_cache(p, &caches[i]);
    if (st != TASP_OK) return st;
    if (caches[i].plan_sig != p->sig) return fail(TASP_ERR_CACHE_PLAN_MISMATCH, "caches[%d]", i);
    if (i > 0 && caches[i].batch != batch) return fail(TASP_ERR_SHAPE, "caches differ in batch");
    batch = caches[i].batch;
    if (layer < -1 || layer >= p->desc.n_layers) return fail(TASP_ERR_INVALID_ARG, "bad layer %d", layer);
    if (pos < 0 || pos >= caches[i].max_seq) return fail(TASP_ERR_POS_RANGE, "pos %d", pos);
    if (i > 0 && p->desc.n_layers != plans[0]->desc.n_layers)
      return fail(TASP_ERR_SHAPE, "plans differ in layer count");
  }
  const int L = plans[0]->desc.n_layers;
  for (int l = (layer < 0 ? 0 : layer); l < (layer < 0 ? L : layer + 1); ++l) {
    for (int i = 0; i < n_plans; ++i) {
      const tasp_plan_s* p = plans[i];
      const LayerPlan& P = p->layers[l];
      if ((kind == 3 && P.c == 0) || (kind == 1 && P.m_kv == 0)) {
        if (layer >= 0)
          return fail(TASP_ERR_SHAPE, kind == 3 ? "layer has no FFN channels"
                                                : "layer has no retained KV group");
        continue;
      }
      Item it{};
      it.plan = i;
      it.layer = l;
      it.shared = p->shared && batch == 1;
      if (kind == 1)
        it.at = attn_args(p, l, &caches[i], pos, batch, batch > 1);
      else if (p->shared && batch == 1)
        it.sg = (kind == 3) ? shared_gateup_args(p, l) : shared_down_args(p, l, p->r_io[l & 1]);
      else if (batch == 1)
        it.g = (kind == 3) ? gateup_args(p, l, batch) : down_args(p, l, batch, p->r_io[l & 1]);
      else
        it.m = (kind == 3) ? gateup_mm_args(p, l, batch) : down_mm_args(p, l, batch, p->r_io[l & 1]);
      items.push_back(it);
    }
  }
  if (items.empty()) return fail(TASP_ERR_SHAPE, "no layer has this stage");
  const tasp::GemvMode mode = (kind == 3) ? tasp::GEMV_GATEUP : tasp::GEMV_RESID;
  const tasp::MfmaMode mmode = (kind == 3) ? tasp::MM_GATEUP : tasp::MM_RESID;
  auto launch = [&](const Item& it, hipStream_t s) {
    if (kind == 1) return tasp::launch_attn_decode(it.at, s);
    if (it.shared) return tasp::launch_shared_gemv(mode, it.sg, s);
    return (batch == 1) ? tasp::launch_gemv(mode, it.g, s) : tasp::launch_mfma_gemv(mmode, it.m, s);
  };
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t e0, e1;
  HIP_TRY(hipEventCreate(&e0));
  HIP_TRY(hipEventCreate(&e1));
  hipError_t h = hipEventRecord(e0, s);
  for (int r = 0; r < reps && h == hipSuccess; ++r)
    for (size_t k = 0; k < items.size() && h == hipSuccess; ++k) h = launch(items[k], s);
  if (h == hipSuccess) h = hipEventRecord(e1, s);
  if (h == hipSuccess) h = hipEventSynchronize(e1);
  float ms = 0.0f;
  if (h == hipSuccess) h = hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (h != hipSuccess) return fail(TASP_ERR_HIP, "profile: %s", hipGetErrorString(h));
  *ms_per_launch = ms / float(size_t(reps) * items.size());
  return TASP_OK;
}

namespace {

// prompt ids pos0..T-1 are embedded and prefilled at those positions (pos0 == 0 binds the
// cache), then n_new greedy decode steps
tasp_status generate_impl(tasp_plan p, const int8_t* embed, const float* embed_scale,
                          const int32_t* prompt, int32_t T, int32_t pos0, int32_t n_new,
                          tasp_kv_cache* cache, int32_t* out_ids, float* x_scratch, float* logits,
                          void* stream) {
  if (!p) return fail(TASP_ERR_INVALID_ARG, "plan is NULL");
  const tasp_model_desc& d = p->desc;
  if (d.vocab < 1) return fail(TASP_ERR_UNSUPPORTED, "plan has no LM head");
  if (!embed || !embed_scale || !prompt || !out_ids || !x_scratch || !logits)
    return fail(TASP_ERR_INVALID_ARG, "embedding / prompt / outputs / scratch is NULL");
  if (n_new < 0) return fail(TASP_ERR_INVALID_ARG, "n_new < 0");
  if (pos0 < 0 || (pos0 > 0 && pos0 >= T))
    return fail(TASP_ERR_INVALID_ARG, "prefill start %d outside [0, %d)", pos0, T);
  tasp_status st = check_cache(p, cache);
  if (st != TASP_OK) return st;
  if (long(T) + n_new > cache->max_seq)
    return fail(TASP_ERR_POS_RANGE, "prompt + new tokens (%d + %d) beyond the cache", T, n_new);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = T - pos0;
  HIP_TRY(tasp::launch_embed(embed, embed_scale, d.vocab, d.d_model, prompt + pos0, n, x_scratch, s));
  if ((st = prefill_checked(p, x_scratch, n, cache, pos0, logits + size_t(n - 1) * d.vocab, stream,
                           nullptr, true)) != TASP_OK)
    return st;
  HIP_TRY(tasp::launch_argmax(logits + size_t(n - 1) * d.vocab, 1, d.vocab, out_ids, p->arg_part,
                              p->arg_cnt, s));
  for (int i = 0; i < n_new; ++i) {
    HIP_TRY(tasp::launch_embed(embed, embed_scale, d.vocab, d.d_model, out_ids + i, 1, x_scratch, s));
    if ((st = decode_impl(p, x_scratch, cache, T + i, logits, stream, nullptr)) != TASP_OK) return st;
    HIP_TRY(tasp::launch_argmax(logits, 1, d.vocab, out_ids + i + 1, p->arg_part, p->arg_cnt, s));
  }
  return TASP_OK;
}

}  // namespace

tasp_status tasp_generate(tasp_plan p, const int8_t* embed, const float* embed_scale,
                          const int32_t* prompt, int32_t T, int32_t n_new, tasp_kv_cache* cache,
                          int32_t* out_ids, float* x_scratch, float* logits, void* stream) {
  return generate_impl(p, embed, embed_scale, prompt, T, 0, n_new, cache, out_ids, x_scratch,
                       logits, stream);
}

// ---- routing

namespace {

struct RouterLayout {
  size_t tf, feats, h1, h2, probs1, choice1, total;
  int feat_dim;
};

tasp_status router_layout(const tasp_router* r, int n, RouterLayout* y) {
  if (!r) return fail(TASP_ERR_INVALID_ARG, "router is NULL");
  if (r->n_bins < 1 || r->n_bins > tasp::kMaxRouterBins)
    return fail(TASP_ERR_INVALID_ARG, "n_bins %d outside 1..%d", r->n_bins, tasp::kMaxRouterBins);
  if (r->n_tasks < 1 || r->n_tasks > tasp::kMaxRouterTasks)
    return fail(TASP_ERR_INVALID_ARG, "n_tasks %d outside 1..%d", r->n_tasks, tasp::kMaxRouterTasks);
  if (r->proj_dim < 1 || r->hidden1 < 1 || r->hidden2 < 1 || r->proj_dim > (1 << 20) ||
      r->hidden1 > (1 << 20) || r->hidden2 > (1 << 20))
    return fail(TASP_ERR_INVALID_ARG, "router widths outside 1..2^20");
  if (!(r->temperature > 0.0f) || !std::isfinite(r->temperature))
    return fail(TASP_ERR_INVALID_ARG, "temperature must be finite and > 0");
  if (!std::isfinite(r->tau)) return fail(TASP_ERR_INVALID_ARG, "tau is not finite");
  if (!r->proj || !r->w1 || !r->b1 || !r->w2 || !r->b2 || !r->w3 || !r->b3)
    return fail(TASP_ERR_INVALID_ARG, "router weight pointer is NULL");
  if (n < 1 || n > 65535) return fail(TASP_ERR_INVALID_ARG, "n_prompts %d outside 1..65535", n);
  y->feat_dim = r->proj_dim + tasp::kRouterScalars;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align_up(off + bytes, kAlign); return at; };
  y->tf = take(size_t(n) * r->n_bins * 4);
  y->feats = take(size_t(n) * y->feat_dim * 4);
  y->h1 = take(size_t(n) * r->hidden1 * 4);
  y->h2 = take(size_t(n) * r->hidden2 * 4);
  y->probs1 = take(size_t(tasp::kMaxRouterTasks) * 4);
  y->choice1 = take(4);
  y->total = off;
  return TASP_OK;
}

}  // namespace

tasp_status tasp_router_workspace_bytes(const tasp_router* r, int32_t n, size_t* bytes) {
  if (!bytes) return fail(TASP_ERR_INVALID_ARG, "bytes is NULL");
  RouterLayout y;
  tasp_status st = router_layout(r, n, &y);
  if (st != TASP_OK) return st;
  *bytes = y.total;
  return TASP_OK;
}

namespace {

// Arguments of a routing call other than its scratch, checked on the host.
tasp_status check_route_args(const tasp_router* r, const uint8_t* text, int32_t n_text,
                             const int32_t* offsets, int32_t n, const float* proxy_logprob,
                             const float* probs, const int32_t* choice, RouterLayout* y) {
  tasp_status st = router_layout(r, n, y);
  if (st != TASP_OK) return st;
  if (n_text < 0) return fail(TASP_ERR_INVALID_ARG, "n_text < 0");
  if ((!text && n_text > 0) || !proxy_logprob || !probs || !choice)
    return fail(TASP_ERR_INVALID_ARG, "text / proxy_logprob / probs / choice is NULL");
  if (!offsets && n != 1) return fail(TASP_ERR_INVALID_ARG, "offsets NULL with %d prompts", n);
  return TASP_OK;
}

// The five routing kernels over a scratch of at least y.total bytes at ws (device).
tasp_status route_launch(const tasp_router* r, const RouterLayout& y, const uint8_t* text,
                         int32_t n_text, const int32_t* offsets, int32_t n,
                         const float* proxy_logprob, char* ws, float* features, float* probs,
                         int32_t* choice, hipStream_t s) {
  float* tf = reinterpret_cast<float*>(ws + y.tf);
  float* feats = features ? features : reinterpret_cast<float*>(ws + y.feats);
  float* h1 = reinterpret_cast<float*>(ws + y.h1);
  float* h2 = reinterpret_cast<float*>(ws + y.h2);
  tasp::RouterFeatArgs fa{};
  fa.text = text; fa.n_text = n_text; fa.offsets = offsets; fa.logprob = proxy_logprob;
  fa.n_bins = r->n_bins; fa.proj_dim = r->proj_dim; fa.tf = tf; fa.feats = feats;
  fa.ld_feats = y.feat_dim;
  HIP_TRY(tasp::launch_router_features(fa, n, s));
  tasp::RouterDenseArgs pa{r->proj, nullptr, r->proj_dim, r->n_bins, tf, r->n_bins, feats,
                           y.feat_dim, n, 0};
  HIP_TRY(tasp::launch_router_dense(pa, s));
  tasp::RouterDenseArgs l1{r->w1, r->b1, r->hidden1, y.feat_dim, feats, y.feat_dim, h1, r->hidden1, n, 1};
  HIP_TRY(tasp::launch_router_dense(l1, s));
  tasp::RouterDenseArgs l2{r->w2, r->b2, r->hidden2, r->hidden1, h1, r->hidden1, h2, r->hidden2, n, 1};
  HIP_TRY(tasp::launch_router_dense(l2, s));
  tasp::RouterHeadArgs ha{r->w3, r->b3, r->n_tasks, r->hidden2, h2, r->temperature, r->tau, probs, choice};
  HIP_TRY(tasp::launch_router_head(ha, n, s));
  return TASP_OK;
}

// Scratch of tasp_route_noalloc: a fixed array in every GPU's memory (each device holds its own
// copy at its own address, from the library's load until the process ends). Host code never
// passes the array's name to a kernel or a copy: on the host that name is only a stand-in, so
// its device address is looked up once per device and kept in scratch_ptr[].
constexpr size_t kNoAllocScratchBytes = TASP_ROUTE_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up on the first call on that device.
tasp_status scratch_address(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(TASP_ERR_UNSUPPORTED, "device %d outside 0..%d", dev, kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(TASP_ERR_HIP, "hipGetSymbolAddress returned a null address");
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return TASP_OK;
}

}  // namespace

tasp_status tasp_route(const tasp_router* r, const uint8_t* text, int32_t n_text,
                       const int32_t* offsets, int32_t n, const float* proxy_logprob,
                       void* workspace, size_t workspace_bytes, float* features, float* probs,
                       int32_t* choice, void* stream) {
  RouterLayout y;
  tasp_status st = check_route_args(r, text, n_text, offsets, n, proxy_logprob, probs, choice, &y);
  if (st != TASP_OK) return st;
  if (!workspace) return fail(TASP_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(TASP_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (workspace_bytes < y.total)
    return fail(TASP_ERR_WORKSPACE, "workspace %zu < %zu bytes", workspace_bytes, y.total);
  return route_launch(r, y, text, n_text, offsets, n, proxy_logprob,
                      static_cast<char*>(workspace), features, probs, choice,
                      static_cast<hipStream_t>(stream));
}

tasp_status tasp_route_noalloc(const tasp_router* r, const uint8_t* text, int32_t n_text,
                               const int32_t* offsets, int32_t n, const float* proxy_logprob,
                               float* features, float* probs, int32_t* choice, void* stream) {
  RouterLayout y;
  tasp_status st = check_route_args(r, text, n_text, offsets, n, proxy_logprob, probs, choice, &y);
  if (st != TASP_OK) return st;
  if (y.total > kNoAllocScratchBytes)
    return fail(TASP_ERR_WORKSPACE,
                "routing %d prompts needs %zu bytes of scratch, more than the fixed %zu of "
                "tasp_route_noalloc (route fewer prompts per call, or use tasp_route)",
                n, y.total, kNoAllocScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_address(&ws)) != TASP_OK) return st;
  return route_launch(r, y, text, n_text, offsets, n, proxy_logprob, static_cast<char*>(ws),
                      features, probs, choice, static_cast<hipStream_t>(stream));
}

tasp_status tasp_serve_turn(const tasp_router* r, const tasp_plan* task_plans,
                            tasp_plan dense_plan, const uint8_t* text, int32_t n_text,
                            const float* proxy_logprob, const int8_t* embed,
                            const float* embed_scale, const int32_t* prompt, int32_t T,
                            int32_t n_cached, int32_t n_new, tasp_kv_cache* cache,
                            int32_t* out_ids, float* x_scratch, float* logits, void* workspace,
                            size_t workspace_bytes, int32_t* chosen, int32_t* reused,
                            void* stream) {
  RouterLayout y;
  tasp_status st = router_layout(r, 1, &y);
  if (st != TASP_OK) return st;
  if (!task_plans || !dense_plan || !chosen || !reused)
    return fail(TASP_ERR_INVALID_ARG, "plans / chosen / reused is NULL");
  const tasp_model_desc& d0 = dense_plan->desc;
  for (int t = 0; t < r->n_tasks; ++t) {
    const tasp_plan q = task_plans[t];
    if (!q) return fail(TASP_ERR_INVALID_ARG, "task plan %d is NULL", t);
    const tasp_model_desc& d = q->desc;
    if (d.n_layers != d0.n_layers || d.d_model != d0.d_model || d.n_q_heads != d0.n_q_heads ||
        d.n_kv_heads != d0.n_kv_heads || d.head_dim != d0.head_dim || d.d_ffn != d0.d_ffn ||
        d.vocab != d0.vocab)
      return fail(TASP_ERR_SHAPE, "task plan %d has another model shape than the dense plan", t);
  }
  if (n_cached < 0) return fail(TASP_ERR_INVALID_ARG, "n_cached < 0");
  if (!cache) return fail(TASP_ERR_INVALID_ARG, "cache is NULL");
  char* ws = static_cast<char*>(workspace);
  if (!ws) return fail(TASP_ERR_INVALID_ARG, "workspace is NULL");
  float* probs = reinterpret_cast<float*>(ws + y.probs1);
  int32_t* dchoice = reinterpret_cast<int32_t*>(ws + y.choice1);
  if ((st = tasp_route(r, text, n_text, nullptr, 1, proxy_logprob, workspace, workspace_bytes,
                       nullptr, probs, dchoice, stream)) != TASP_OK)
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t c = 0;
  HIP_TRY(hipMemcpyAsync(&c, dchoice, sizeof c, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (c < -1 || c >= r->n_tasks) return fail(TASP_ERR_INTERNAL, "router choice %d out of range", c);
  const tasp_plan p = (c >= 0) ? task_plans[c] : dense_plan;
  const bool keep = n_cached > 0 && n_cached < T && cache->plan_sig == p->sig;
  *chosen = c;
  *reused = keep ? 1 : 0;
  return generate_impl(p, embed, embed_scale, prompt, T, keep ? n_cached : 0, n_new, cache,
                       out_ids, x_scratch, logits, stream);
}

// ---- greedy mask construction

namespace {

struct MaskLayout {
  size_t status, keys_in, keys_out, idx_in, idx_out, temp, temp_bytes, total;
};

tasp_status mask_layout(const tasp_model_desc* d, int granule, MaskLayout* y) {
  tasp_status st = check_desc(d);
  if (st != TASP_OK) return st;
  if (granule < 1 || d->d_ffn % granule)
    return fail(TASP_ERR_SHAPE, "granule %d does not divide d_ffn %d", granule, d->d_ffn);
  const int nG = d->d_ffn / granule;
  const long n = long(d->n_layers) * (d->n_q_heads + nG);
  if (n > (1L << 30)) return fail(TASP_ERR_SHAPE, "too many candidates");
  if (tasp::mask_scan_lds_bytes(d->n_layers, d->n_q_heads, d->n_kv_heads, nG) > kLdsLimit)
    return fail(TASP_ERR_UNSUPPORTED, "candidate flags exceed LDS");
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align_up(off + bytes, kAlign); return at; };
  y->status = take(16);
  y->keys_in = take(size_t(n) * 8);
  y->keys_out = take(size_t(n) * 8);
  y->idx_in = take(size_t(n) * 4);
  y->idx_out = take(size_t(n) * 4);
  size_t tb = 0;
  const hipError_t e = tasp::mask_sort_temp_bytes(int(n), &tb);
  if (e != hipSuccess) return fail(TASP_ERR_HIP, "sort size query: %s", hipGetErrorString(e));
  y->temp_bytes = tb;
  y->temp = take(tb);
  y->total = off;
  return TASP_OK;
}

}  // namespace

tasp_status tasp_mask_workspace_bytes(const tasp_model_desc* desc, int32_t granule, size_t* bytes) {
  if (!bytes) return fail(TASP_ERR_INVALID_ARG, "bytes is NULL");
  MaskLayout y;
  tasp_status st = mask_layout(desc, granule, &y);
  if (st != TASP_OK) return st;
  *bytes = y.total;
  return TASP_OK;
}

tasp_status tasp_build_mask(const tasp_model_desc* desc, const float* head_scores,
                            const float* chan_scores, int32_t granule, double target,
                            void* workspace, size_t workspace_bytes, uint8_t* q_keep,
                            uint8_t* kv_keep, uint8_t* ffn_keep, uint64_t* flops_spent,
                            void* stream) {
  MaskLayout y;
  tasp_status st = mask_layout(desc, granule, &y);
  if (st != TASP_OK) return st;
  if (!head_scores || !chan_scores || !q_keep || !kv_keep || !ffn_keep)
    return fail(TASP_ERR_INVALID_ARG, "scores / outputs are NULL");
  if (!(target >= 0.0 && target <= 1.0)) return fail(TASP_ERR_INVALID_ARG, "target outside [0, 1]");
  if (!workspace) return fail(TASP_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
    return fail(TASP_ERR_WORKSPACE, "workspace not %zu-byte aligned", kAlign);
  if (workspace_bytes < y.total)
    return fail(TASP_ERR_WORKSPACE, "workspace %zu bytes, need %zu", workspace_bytes, y.total);
  const tasp_model_desc& d = *desc;
  char* base = static_cast<char*>(workspace);
  tasp::MaskArgs a{};
  a.head_scores = head_scores; a.chan_scores = chan_scores;
  a.L = d.n_layers; a.Hq = d.n_q_heads; a.Hkv = d.n_kv_heads; a.nG = d.d_ffn / granule;
  a.granule = granule; a.n_cand = a.L * (a.Hq + a.nG);
  const unsigned long long D = d.d_model, dh = d.head_dim;
  a.head_cost = 2 * D * dh + 2 * dh * D;
  a.group_cost = 2 * D * dh * 2;
  a.chan_cost = 6 * D * (unsigned long long)granule;
  a.head_rank_cost = double(a.head_cost) + double(a.group_cost) / double(a.Hq / a.Hkv);
  const unsigned long long full = (unsigned long long)d.n_layers *
      (2 * D * dh * (unsigned long long)(d.n_q_heads + 2 * d.n_kv_heads) +
       2 * dh * (unsigned long long)d.n_q_heads * D + 6 * D * (unsigned long long)d.d_ffn);
  a.budget = (unsigned long long)std::floor(target * double(full));
  a.q_keep = q_keep; a.kv_keep = kv_keep; a.ffn_keep = ffn_keep;
  a.status = reinterpret_cast<unsigned*>(base + y.status);
  a.spent = reinterpret_cast<unsigned long long*>(base + y.status + 8);
  hipStream_t s = static_cast<hipStream_t>(stream);
  HIP_TRY(hipMemsetAsync(base + y.status, 0, 16, s));
  HIP_TRY(tasp::launch_build_mask(a, base + y.temp, y.temp_bytes,
                                  reinterpret_cast<double*>(base + y.keys_in),
                                  reinterpret_cast<double*>(base + y.keys_out),
                                  reinterpret_cast<int*>(base + y.idx_in),
                                  reinterpret_cast<int*>(base + y.idx_out), s));
  uint64_t word[2] = {0, 0};
  HIP_TRY(hipMemcpyAsync(word, base + y.status, 16, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  if (word[0] & 1u) return fail(TASP_ERR_INVALID_ARG, "non-finite score");
  if (flops_spent) *flops_spent = word[1];
  return TASP_OK;
}

tasp_status tasp_copy_probe(void* dst, const void* src, size_t bytes, void* stream) {
  if (!dst || !src) return fail(TASP_ERR_INVALID_ARG, "dst / src is NULL");
  if (bytes % 16) return fail(TASP_ERR_INVALID_ARG, "bytes %% 16 != 0");
  HIP_TRY(tasp::launch_copy(dst, src, bytes, static_cast<hipStream_t>(stream)));
  return TASP_OK;
}

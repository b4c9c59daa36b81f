// Internal launcher interface between the host runtime and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tasp {

// ----------------------------------------------------------------- plan compilation

// Closure + ascending index lists for every layer (one workgroup per layer).
//   q_keep [L][Hq], kv_keep [L][Hkv] (nullable: all kept), ffn_keep [L][F]   (device bytes)
//   outputs per layer l (device int32): q_idx [l*Hq ..], kv_idx [l*Hkv ..], q_kvslot [l*Hq ..],
//   slot_start [l*(Hkv+1) ..] (first retained-head position of each retained group, then m_q),
//   ffn_idx [l*F ..], counts [l*4 ..] = {m_q, m_kv, c, 0}.
hipError_t launch_closure(const uint8_t* q_keep, const uint8_t* kv_keep, const uint8_t* ffn_keep,
                          int L, int Hq, int Hkv, int F, int* q_idx, int* kv_idx, int* q_kvslot,
                          int* slot_start, int* ffn_idx, int* counts, hipStream_t s);

// dst rows [i*dh + e] = src rows [idx[i]*dh + e] for i < n, e < dh; rows of K bytes (K % 16 == 0).
hipError_t launch_gather_head_rows(int8_t* dst, const int8_t* src, const int* idx, int n, int dh,
                                   int K, float* dst_scale, const float* src_scale, hipStream_t s);
// dst rows [i] = src rows [idx[i]] for i < n (rows of K bytes) and the matching scales.
hipError_t launch_gather_rows(int8_t* dst, const int8_t* src, const int* idx, int n, int K,
                              float* dst_scale, const float* src_scale, hipStream_t s);
// dst[r][i*dh + e] = src[r][idx[i]*dh + e] for r < rows; src row stride src_ld, dst stride dst_ld.
hipError_t launch_gather_head_cols(int8_t* dst, int dst_ld, const int8_t* src, int src_ld,
                                   const int* idx, int n, int dh, int rows, hipStream_t s);
// dst[r][j] = src[r][idx[j]] for j < n, zero for n <= j < dst_ld.
hipError_t launch_gather_cols(int8_t* dst, int dst_ld, const int8_t* src, int src_ld,
                              const int* idx, int n, int rows, hipStream_t s);
hipError_t launch_copy(void* dst, const void* src, size_t bytes, hipStream_t s);   // bytes % 16 == 0
hipError_t launch_fill_zero(void* dst, size_t bytes, hipStream_t s);              // bytes % 4 == 0

// ----------------------------------------------------------------- decode GEMVs

// GEMV_QKV: RMSNorm prologue, plain store; GEMV_RESID: residual add; GEMV_GATEUP: RMSNorm
// prologue, SwiGLU epilogue over paired gate / up rows; GEMV_LMHEAD: RMSNorm prologue, BF16
// weights (w holds BF16 rows of K elements), plain store.
enum GemvMode { GEMV_QKV = 0, GEMV_RESID = 1, GEMV_GATEUP = 2, GEMV_LMHEAD = 3 };

struct GemvArgs {
  const void* w;         // panel rows [N][ld] (gate/up: gate rows; LM head: BF16 [N][K])
  const void* w2;        // gate/up: up rows [N][ld]
  const float* scale;    // [N] (unused by the LM head)
  const float* scale2;   // gate/up: up scales [N]
  int N;                 // output rows (gate/up: channels)
  int K;                 // valid columns; INT8 columns K..ld-1 of a row are zero
  int ld;                // INT8 row stride in bytes, multiple of 16 and >= K
  const float* x;        // input rows [B][ldx]
  int ldx;
  const uint16_t* gamma; // RMSNorm gain (QKV, gate/up, LM head); null for GEMV_RESID
  float eps;
  const float* resid;    // residual rows [B][ldy] (GEMV_RESID)
  float* y;              // output rows [B][ldy]
  int ldy;
  int B;                 // batch rows (1; larger batches use the MFMA kernels)
};
hipError_t launch_gemv(GemvMode mode, const GemvArgs& a, hipStream_t s);
size_t gemv_lds_bytes(int B, int K);

// ----------------------------------------------------------------- shared-store decode GEMVs

// Batch-1 GEMVs over the groupwise store (INT8 [store_rows][ld], BF16 scales
// [store_rows][ld / 128]) through a plan's maps: plan row i reads store row rows[i] (null:
// i), plan columns 16 p .. 16 p + 15 read store columns cols[p] .. cols[p] + 15 (null: 16 p).
// Modes as for launch_gemv except the LM head. K % 16 == 0, ld % 128 == 0.
constexpr size_t kMaxSharedGemvLds = 159 * 1024;
struct SharedGemvArgs {
  const int8_t* w; const int8_t* w2;       // store matrix (gate/up: gate, up)
  const uint16_t* s; const uint16_t* s2;   // their scales
  int ld, store_rows;
  const int* rows; const int* cols;        // device maps (nullable)
  int N, K;                                // plan rows (gate/up: channels), plan columns
  const float* x;                          // input [K]
  const uint16_t* gamma; float eps;        // RMSNorm gain (QKV, gate/up)
  const float* resid;                      // GEMV_RESID: [N]
  float* y;                                // [N]
};
hipError_t launch_shared_gemv(GemvMode mode, const SharedGemvArgs& a, hipStream_t s);
size_t shared_gemv_lds_bytes(int K);

// Maps of every layer from the closure's index lists and counts: qkv_rows [L][(Hq + 2Hkv) dh]
// (store rows of the retained q heads, then K and V rows of the retained groups, for a store
// whose QKV matrix holds all q rows, then all K rows, then all V rows), o_cols [L][Hq dh / 16]
// (store columns of the retained heads' pieces), down_cols [L][F / 16] (first store column of
// each block of 16 retained channels; the retained channels must come in such blocks).
struct SharedMapsArgs {
  int Hq, Hkv, dh, F;
  const int* q_idx; const int* kv_idx; const int* ffn_idx; const int* counts;
  int* qkv_rows; int* o_cols; int* down_cols;
};
hipError_t launch_shared_maps(const SharedMapsArgs& a, int n_layers, hipStream_t s);

// ----------------------------------------------------------------- batched decode on MFMA

// Batch 2..8. Activations are a [16][ldx] BF16 operand: row 2b = bf16(v), row 2b+1 =
// bf16(v - bf16(v)) for sequence b (rows >= 2B unused); ldx % 64 == 0, ldx >= K.
// MM_QKV: plain store; MM_RESID: residual add, optionally writing the next operand (x * gamma_next)
// and per-16-row sums of squares; MM_GATEUP: SwiGLU of paired gate / up rows into the next operand;
// MM_LMHEAD: BF16 weights [N][ld], plain store. The inverse RMS of sequence b is
// rsqrt(inv_d * sum(ssq[b][0..n_ssq)) + eps) when ssq is given, else 1.
enum MfmaMode { MM_QKV = 0, MM_RESID = 1, MM_GATEUP = 2, MM_LMHEAD = 3 };

// A projection read from the groupwise shared store instead of a panel: INT8 rows [store_rows][ld]
// with one BF16 scale per row and 128 columns; plan row n is store row rows[n] (identity when
// rows is null), plan columns 16 p .. 16 p + 15 are store columns cols[p] .. cols[p] + 15
// (identity when cols is null). Gate/up use w / gs for the gate and w2 / gs2 for the up matrix.
struct StoreView {
  const int8_t* w; const int8_t* w2;
  const uint16_t* gs; const uint16_t* gs2;
  int ld, store_rows;
  const int* rows; const int* cols;
};

struct MfmaArgs {
  const void* w;              // panel rows [N][ld] (gate/up: gate rows)
  uint32_t w2_off;            // gate/up: byte offset of the up rows from w
  const float* scale;         // [N]
  const float* scale2;        // gate/up: up scales
  int N, K, ld;               // rows (gate/up: channels), valid columns, row stride (elements)
  const uint16_t* x; int ldx; // activation operand
  const float* ssq; int n_ssq; float inv_d, eps;
  const float* resid;         // MM_RESID: [B][ldy]
  float* y; int ldy;          // float32 output rows (not MM_GATEUP)
  uint16_t* xo; int ldxo;     // next operand (MM_GATEUP; MM_RESID when gamma_next is set)
  const uint16_t* gamma_next; // MM_RESID: gain of the next RMSNorm
  float* ssq_out; int n_tiles_out;  // MM_RESID with gamma_next: [B][n_tiles_out], n_tiles_out = ceil(N/16)
  int B;
  StoreView sv;               // gs set: weights read from a groupwise store (w, w2_off, scale unused)
};
hipError_t launch_mfma_gemv(MfmaMode mode, const MfmaArgs& a, hipStream_t s);
// The first operand of a step from float32 input rows x [B][ldx]: x * gamma as hi/lo and the
// sums of squares of x per 16 elements ([B][D/16]).
hipError_t launch_mfma_prep(const float* x, int ldx, int D, const uint16_t* gamma, uint16_t* xo,
                            int ldxo, float* ssq, int B, hipStream_t s);

// ----------------------------------------------------------------- prefill on MFMA

// T tokens of one sequence. Activation operands are two BF16 planes (hi, lo) of [T][ldx] each,
// `plane` elements apart; modes as for the batched decode. The inverse RMS of token t is
// rsqrt(inv_d * sum(ssq[t][0..n_ssq)) + eps) when ssq is given (partials per 64 rows).
struct PfArgs {
  const void* w; uint32_t w2_off;     // panel rows [N][ld] (gate/up: gate rows; up at w2_off bytes)
  const float* scale; const float* scale2;
  int N, K, ld;
  const uint16_t* x; int ldx; uint32_t plane;
  const float* ssq; int n_ssq; float inv_d, eps;
  const float* resid;                 // MM_RESID: [T][ldy]
  float* y; int ldy;                  // float32 output [T][ldy] (not MM_GATEUP)
  uint16_t* xo; int ldxo; uint32_t plane_o;   // next operand (MM_GATEUP; MM_RESID with gamma_next)
  const uint16_t* gamma_next;
  float* ssq_out; int n_ssq_out;      // MM_RESID with gamma_next: [T][ceil(N/64)]
  int T;
  float* part; size_t part_floats;    // MM_QKV / MM_RESID K-split partials [splits][T][N] (or null)
  StoreView sv;                       // gs set: weights read from a groupwise store
};
hipError_t launch_pf_gemm(MfmaMode mode, const PfArgs& a, hipStream_t s);
// floats of the K-split partial buffer of a plan (prompt chunks up to max_prefill tokens, panels
// of up to n_max rows)
size_t pf_split_buffer_floats(int max_prefill, int n_max);
// x float32 [T][D] -> hi/lo planes of x * gamma and sums of squares per 64 elements [T][D/64].
hipError_t launch_pf_prep(const float* x, int D, int T, const uint16_t* gamma, uint16_t* xo,
                          size_t plane, int ldxo, float* ssq, hipStream_t s);
int pf_ssq_block();

struct PfRopeArgs {
  const float* qkv; int ld_qkv;       // [T][ld_qkv]: raw q (m_q*dh), k (m_kv*dh), v (m_kv*dh)
  int m_q, m_kv, dh;
  int kv_idx[64];
  uint16_t* kc; uint16_t* vc;         // this layer's cache of sequence 0, [Hkv][S][dh]
  int S;
  const float* rope_cos; const float* rope_sin;
  int pos0, T;
  uint16_t* q_out; uint32_t q_plane; int T_ld;   // [2][m_q][T_ld][dh] hi/lo, q * log2(e)/sqrt(dh)
};
hipError_t launch_pf_rope(const PfRopeArgs& a, hipStream_t s);

struct PfAttnArgs {
  const uint16_t* q; uint32_t q_plane; int T_ld;   // as PfRopeArgs::q_out
  int m_kv, dh;
  int kv_idx[64];
  int slot_start[65];
  const uint16_t* kc; const uint16_t* vc;         // [Hkv][S][dh]
  int S, pos0, T;
  uint16_t* o; int ldo; uint32_t o_plane;         // hi/lo operand [2][T][ldo]
  // split query blocks: partial records (part_floats, nullable: no split) and one counter per
  // (retained head, query block), zero on entry and left zero
  float* part; size_t part_floats; int* cnt; int cnt_len;
  int split_sb;                                   // set by the launch: chunk length, 0 = none
};
hipError_t launch_pf_attn(const PfAttnArgs& a, hipStream_t s);
// floats of the partial records a prefill of up to max_prefill tokens may need (n_q_heads heads)
size_t pf_attn_record_floats(int max_prefill, int n_q_heads, int dh);

// ----------------------------------------------------------------- request loop

// x[t] = scale[ids[t]] * table[ids[t]] for t < n (NaN rows for ids outside [0, V)); d % 4 == 0
hipError_t launch_embed(const int8_t* table, const float* scale, int V, int d, const int* ids,
                        int n, float* x, hipStream_t s);
// ids_out[r] = argmax of logits row r of n rows of V (lowest id among equal maxima)
// with part (2 floats per chunk of kArgmaxChunk logits and row) and cnt (one per row, zero on
// entry and left zero) for n <= kArgmaxMaxRows rows of at most kArgmaxMaxChunks chunks, the rows
// are split over workgroups; otherwise one workgroup per row
constexpr int kArgmaxChunk = 4096;
constexpr int kArgmaxMaxChunks = 256;
constexpr int kArgmaxMaxRows = 8;
hipError_t launch_argmax(const float* logits, int n, int V, int* ids_out, float* part, int* cnt,
                         hipStream_t s);

// ----------------------------------------------------------------- mask construction

struct MaskArgs {
  const float* head_scores;           // device [L][Hq]
  const float* chan_scores;           // device [L][nG]
  int L, Hq, Hkv, nG, granule, n_cand;
  double head_rank_cost;              // own + group / r, the ranking denominator of a head
  unsigned long long head_cost, group_cost, chan_cost, budget;
  uint8_t* q_keep; uint8_t* kv_keep; uint8_t* ffn_keep;   // device outputs
  unsigned* status;                   // bit 0: a non-finite score
  unsigned long long* spent;          // FLOPs of the accepted set
};
size_t mask_scan_lds_bytes(int L, int Hq, int Hkv, int nG);
hipError_t mask_sort_temp_bytes(int n, size_t* bytes);
hipError_t launch_build_mask(const MaskArgs& a, void* temp, size_t temp_bytes, double* keys_in,
                             double* keys_out, int* idx_in, int* idx_out, hipStream_t s);

// ----------------------------------------------------------------- decode attention

struct AttnArgs {
  const float* qkv; int ld_qkv;    // [B][ld_qkv]: raw q (m_q*dh), k (m_kv*dh), v (m_kv*dh)
  int m_q, m_kv, dh;
  int kv_idx[64];                  // retained group ids (first m_kv entries)
  int slot_start[65];              // first retained-head position of each group slot, then m_q
  uint16_t* kc; uint16_t* vc;      // this layer's cache base, [B][Hkv][S][dh]
  int Hkv, S;
  const float* rope_cos; const float* rope_sin;  // [max_seq][dh/2]
  int pos, chunk, n_split;          // split s: rows [s chunk, (s+1) chunk), the last one to pos
  float* part;                     // [B][m_kv][n_split][8][dh + 4] when n_split > 1
  int* cnt;                        // [B][m_kv] split counters, zero before and after a launch
  float* o; int ld_o;              // [B][ld_o] retained heads in ascending order
  uint16_t* o_hl; int ld_ohl;      // when set: o as the hi/lo BF16 operand [16][ld_ohl] instead
  int B;
};
// Split-KV attention on the matrix cores; for n_split > 1 the last split of each (group slot,
// sequence) to finish merges the partials into o by log-sum-exp (n_split == 1 writes o directly).
hipError_t launch_attn_decode(const AttnArgs& a, hipStream_t s);
// split rows and count of the matrix-core kernel for total = pos + 1 attended rows: one sequence,
// and `units` (sequences x retained group slots) of a batch
void attn_mfma_split(int total, int* chunk, int* n_split);
void attn_mfma_split_batched(int total, int units, int* chunk, int* n_split);
int attn_mfma_max_split(int max_seq);   // largest split count it uses for up to max_seq rows

// ----------------------------------------------------------------- router

constexpr int kMaxRouterTasks = 16;
constexpr int kMaxRouterBins = 16384;
constexpr int kRouterScalars = 11;     // length, log-prob, 4 character counts, 5 descriptors

struct RouterFeatArgs {
  const uint8_t* text; int n_text;     // all prompts' bytes
  const int* offsets;                  // [n + 1] prompt bounds, clamped to [0, n_text]; null: one
                                       // prompt spanning the whole text
  const float* logprob;                // [n] proxy-LM mean token log-probabilities
  int n_bins, proj_dim;
  float* tf;                           // [n][n_bins] trigram term frequencies
  float* feats; int ld_feats;          // [n][ld_feats]; the scalars go to columns proj_dim ..
};
// y[b][j] = act(w[j] . x[b] + bias[j]) for j < N, b < B; w [N][K], bias [N] or null, act ReLU
// when relu != 0
struct RouterDenseArgs {
  const float* w; const float* bias; int N, K;
  const float* x; int ldx;
  float* y; int ldy;
  int B, relu;
};
struct RouterHeadArgs {
  const float* w; const float* bias; int n_tasks, K;   // w [n_tasks][K]
  const float* h;                                      // [n][K]
  float temperature, tau;
  float* probs; int* choice;                           // [n][n_tasks], [n]
};
size_t router_features_lds_bytes(int n_bins);
hipError_t launch_router_features(const RouterFeatArgs& a, int n_prompts, hipStream_t s);
hipError_t launch_router_dense(const RouterDenseArgs& a, hipStream_t s);
hipError_t launch_router_head(const RouterHeadArgs& a, int n_prompts, hipStream_t s);

}  // namespace tasp

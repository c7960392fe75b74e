// Internal declarations shared by the host orchestration (sbd_api.cpp) and the
// gfx950 kernels (*.hip).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "sbd.h"

namespace sbd {

typedef uint16_t bf16_t;            // raw IEEE bfloat16 bits
typedef uint8_t fp8_t;              // raw OCP e4m3 (fn) bits

constexpr int kWave = 64;           // CDNA wavefront width
constexpr int kMaxSplits = 64;      // split-KV partitions per (sequence, KV head, row block)
constexpr int kEbChunk = 4096;      // vocabulary entries per EB partial workgroup
constexpr int kEbInlineRows = 2048;  // masks of at most this many rows are passed by value
constexpr int kMaxBlock = 64;       // largest block size k
constexpr int kCounters = 65536;    // int32 words of arrival counters in the workspace
constexpr int kLayerCtr0 = 16384;    // first counter word of the per-XCD layer kernels (decode GEMMs below)
constexpr int kCtrStride = 32;      // int32 words between counters that live in one XCD's L2 (a 128-byte line each)

// Where a kernel is enqueued: the stream, plus optional start/stop events that the
// runtime records at the kernel's own start and end (per-kernel timing).
struct Exec {
  hipStream_t s;
  hipEvent_t start;
  hipEvent_t stop;
};

// Per-row parameters of one forward (row m = b * k + j).
struct RowParam {
  int32_t tok;   // token id
  int32_t pos;   // RoPE position
};

// Per-sequence parameters of one forward.
struct SeqParam {
  int32_t slot;       // cache slot
  int32_t cache_len;  // committed tokens before this forward
  int32_t n_causal;   // rows [0, n_causal) are causal
  int32_t pad;
};

// Where each buffer lives inside the caller's workspace (byte offsets).
struct Layout {
  int64_t cap;            // cache capacity per slot (max_seq_len rounded up to 64)
  int64_t m_max;          // rows per forward (max(max_batch*max_block, prefill_chunk))
  int64_t n_qkv;          // (n_q_heads + 2 n_kv_heads) * head_dim
  int64_t n_part;         // d_model / 16 sum-of-squares partials per row
  int64_t eb_chunks;      // ceil(vocab / kEbChunk)
  size_t kcache, vcache, rope, x, xn, sumsq, qkv, q, attn, act;
  size_t wpack;              // packed weights (see gemm.hip), element offsets below
  size_t wpack8;             // fp8 weights: the same packing, one byte per element
  size_t wscale;             // fp8 weights: per-row scales 2^e (floats), offsets below
  int64_t ws_layer, ws_o, ws_gu, ws_down, ws_lm;
  int64_t wp_layer;          // elements per layer: qkv, then o, then gate/up, then down
  int64_t wp_o, wp_gu, wp_down, wp_lm;
  size_t attn_ml, attn_o, rows, seqs, eb_mask, eb_part, eb_arg, gemv_part, counters;
  // sbd_block_step: the LM head's 64-column chunk statistics and the merged row values
  size_t eb_fpart, eb_farg, eb_rowstat, eb_rowtok;
  int64_t eb_frows, eb_fchunks;  // rows (min(max_batch * max_block, kStepMaxRows)), vocab / 64
  int64_t gemv_part_floats;  // split-K partial tiles of the decode GEMM
  size_t xn2, sumsq2;        // fused decode forward: second copy of xn (hi, lo) and its partials
  size_t fwd_gains, fwd_ctl, fwd_err;
  size_t lx_part, x64;        // per-XCD layer kernels: XCD-local partials, fixed-point residual
  int64_t fwd_ctl_ints;
  size_t total;
};

bool compute_layout(const sbd_model_config& c, Layout* out);

// Weight pointers of one layer (device bf16).
struct LayerW {
  const bf16_t *attn_norm, *wq, *wk, *wv, *wo, *q_norm, *k_norm, *mlp_norm;
  const bf16_t *w_gate, *w_up, *w_down;
};

// ---------------------------------------------------------------------------- GEMM
enum GemmEpi { EPI_SCALED_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3, EPI_LOGITS_EB = 4 };
// EPI_LOGITS_EB (LM head): EPI_SCALED_STORE (out_f32 may be null: nothing stored) plus the
// EB softmax statistics of every row's 64-column chunks (eb_stats.h) into eb_part / eb_arg.
constexpr int kEbFChunk = 64;
constexpr int kStepMaxRows = 512;  // batch * k of one sbd_block_step

// EPI_QKV (decode-sized GEMM only): the QKV projection's epilogue does the rest of the
// attention input — per-head RMSNorm of q and k (Qwen-3), rotate-half RoPE, q stored as
// scaled hi/lo, K and V written to the cache at position cache_len + j.
struct QkvEpi {
  const RowParam* rows;
  const SeqParam* seqs;
  int kblk, layer;
  int n_q, n_kv, d_h, qk_norm;
  float eps, q_scale;
  const float* rope;  // [cap][d_h/2][2]
  const bf16_t* q_norm;
  const bf16_t* k_norm;
  bf16_t* q;
  bf16_t* q_lo;
  void* kcache;       // KV cache: bf16, or e4m3 codes (kv_fp8) of value * kv_inv
  void* vcache;
  int kv_fp8;
  float kv_inv;
  int64_t cap;
  int n_slots;
};

// Activations travel as two bf16 arrays, hi = bf16(a) and lo = bf16(a - hi), which
// together carry about 16 significant bits; products with bf16 weights are exact in the
// fp32 accumulators, so a GEMM over (hi, lo) loses only the lo truncation.
//
// y[m][n] = sum_k A[m][k] * W[n][k] with W in the packed fragment order of gemm.hip.
struct GemmArgs {
  const bf16_t* A;     // hi part [M][K], row stride lda (a_mtiles == 0) or fragment order
  const bf16_t* A_lo;  // lo part, same layout
  int64_t lda;
  int M, K;
  int a_mtiles;        // A in fragment order with this many row tiles (0: row-major)
  int a_row0;          // first row of A used (fragment order only)
  int o_mtiles;        // xn (EPI_RESID) and act (EPI_SWIGLU) written in fragment order (0: row-major)
  const bf16_t* Wp;    // packed weights
  const fp8_t* Wp8;    // or (non-null) e4m3 weights in the same packing, with per-row scales
  const float* wscale; //   wscale[16 t + r] of packed tile t, row r
  int n_tiles;         // 16-row tiles of the packed matrix (a multiple of 8)
  // EPI_SCALED_STORE: out[m][n] = rinv[m] * y (rinv = 1 when sumsq_in == nullptr)
  float* out_f32;
  int64_t ldo;
  // EPI_LOGITS_EB: as EPI_SCALED_STORE (out_f32 nullable) plus the chunk statistics
  double* eb_part;
  int32_t* eb_arg;
  int eb_chunks, eb_mask_id;
  // row RMS from the producer's partial sums of squares [M][n_part] (EPI_SCALED_STORE,
  // EPI_SWIGLU)
  const float* sumsq_in;
  int n_part;
  float inv_d, eps;
  // EPI_RESID: x[m][n] += y; xn[m][n] = x * g_next[n] as hi/lo; sumsq_out[m][p] = sum of
  // x^2 over the columns of column block p (n_part_out = gemm_plan(...).n_cb partials)
  float* x;
  int64_t ldx;
  bf16_t* xn;
  bf16_t* xn_lo;
  const bf16_t* g_next;
  float* sumsq_out;
  int n_part_out;
  // EPI_SWIGLU: act[m][j] = silu(rinv*gate) * rinv*up as hi/lo
  bf16_t* act;
  bf16_t* act_lo;
  int64_t ld_act;
  // K split over workgroups: parked partial tiles (part_cap floats) and arrival counters
  // (zero between launches)
  float* part;
  int64_t part_cap;
  int* counters;
  // wait_ok: the device places workgroup i on XCD i % 8 and has 32 CUs per XCD, so in a plan
  // of one round every workgroup is resident at once and the K slices of a unit may wait for
  // each other (K is split only then): each slice then sums the slices of its own row tiles
  // and finishes them.  A wait that gives up after spin_limit polls raises the sticky error
  // err (device word, and its pinned host copy err_host).
  int wait_ok;
  int spin_limit;
  int* err;
  int* err_host;
  // set by launch_gemm from the plan
  int splits, m_blocks;
  int no_split;        // 1: one K slice per unit (no hand-off between workgroups)
};

// How launch_gemm cuts a product: mt 16-row tiles per row block (m_blocks row blocks),
// nt 16-column tiles per column block (n_cb blocks), K split `splits` ways.
struct GemmPlan {
  int mt, nt, splits, m_blocks, n_cb;
};
// nt12: 12-tile column blocks may be used (EPI_SWIGLU with bf16 weights: an epilogue
// without row reductions across the block's columns).  half_block: 16-tile blocks may be
// used when n_tiles % 16 == 8, the last one half full (EPI_SCALED_STORE / EPI_LOGITS_EB with
// bf16 weights; n_cb then counts it).
GemmPlan gemm_plan(int M, int n_tiles, int K, int64_t part_cap, bool nt12 = false, bool half_block = false);

hipError_t launch_gemm(GemmEpi epi, const GemmArgs& a, const Exec& ex);

// Decode-sized GEMM (M <= 16), gemv.hip: a workgroup owns C tiles of one packed group and
// a K range; its waves split the range, partial tiles meet in LDS, and K ranges split
// across workgroups are added by the last one to finish.
struct GemvArgs {
  const bf16_t* A;     // hi [M][K], row stride lda
  const bf16_t* A_lo;  // lo
  int64_t lda;
  int M, K;
  const bf16_t* Wp;    // packed weights
  const fp8_t* Wp8;    // the same in e4m3 (same packing), or null: then Wp is streamed
  const float* wscale; // with Wp8: per-row power-of-two scales [n_tiles * 16]
  int n_tiles;         // 16-row tiles of the packed matrix (a multiple of 8)
  // EPI_SCALED_STORE, SWIGLU, QKV: the input rows' RMSNorm scale 1/sqrt(mean(x^2) + eps)
  // is formed from the producer's partial sums of squares [M][n_part_in] (none: scale 1)
  const float* sumsq_in;
  int n_part_in;
  float* out_f32;        // EPI_SCALED_STORE, EPI_LOGITS_EB (nullable there)
  int64_t ldo;
  double* eb_part;       // EPI_LOGITS_EB: [M][eb_chunks][3] (max, Z, S) of 64-column chunks
  int32_t* eb_arg;       // [M][eb_chunks] argmax column or -1
  int eb_chunks, eb_mask_id;
  float* x;              // EPI_RESID
  int64_t ldx;
  bf16_t* xn;
  bf16_t* xn_lo;
  const bf16_t* g_next;
  float* sumsq;          // EPI_RESID: [M][n_part] partial sums of x^2, n_part = n_tiles / C
  int n_part;
  float inv_d, eps;
  bf16_t* act;           // EPI_SWIGLU
  bf16_t* act_lo;
  int64_t ld_act;
  QkvEpi qkv;            // EPI_QKV
  float* part;           // split K: partial tiles [splits][n_tiles][64 lanes][4]
  int64_t part_cap;      // floats available at part (bounds the split)
  int* counters;         // arrival counters (kCounters words), zero between launches
  int splits;            // K slices per unit (set by the launcher)
  int no_split;          // 1: one K slice per unit (no hand-off between workgroups)
};
// Launch shape of the decode GEMM; a zero field means "pick for the shape".
struct GemvShape {
  int C, NW, U, KS;
};
constexpr int kGemvMaxSplit = 16;
GemvShape gemv_pick(GemmEpi epi, int n_tiles, int K);
hipError_t launch_gemv(GemmEpi epi, const GemvArgs& a, GemvShape shape, const Exec& ex);
// Repack a row-major [rows][K] matrix (mode 0) or a gate/up pair (mode 1, rows = 2 * F
// packed rows) into the fragment order read by gemm_kernel.
hipError_t launch_pack(const bf16_t* src0, const bf16_t* src1, bf16_t* dst, int64_t rows, int K,
                       int mode, hipStream_t s);

// ---------------------------------------------------------------------------- misc kernels
struct EmbedArgs {
  const RowParam* rows;
  int M, d;
  const bf16_t* embed;
  const bf16_t* g;  // first attention-norm gain
  float* x;
  bf16_t* xn;
  bf16_t* xn_lo;
  float* sumsq;  // [M][d/16]
  int mtiles;    // xn, xn_lo in fragment order with this many row tiles (0: row-major)
  int64_t* x64;       // the same rows as fixed point (x * 2^32) for the per-XCD layer kernels, or null
  int64_t* x64_zero;  // with x64: the buffer the first layer kernel adds into, zeroed here
};
hipError_t launch_embed(const EmbedArgs& a, const Exec& ex);

struct RopeStageArgs {
  const RowParam* rows;
  const SeqParam* seqs;
  int M, k, layer;
  int n_q, n_kv, d_h;
  int qk_norm;
  float eps;
  float q_scale;  // folded into the stored queries
  const float* qkv;  // [M][(n_q + 2 n_kv) d_h]
  const bf16_t* q_norm;
  const bf16_t* k_norm;
  const float* rope;  // [cap][d_h/2][2] (cos, sin)
  bf16_t* q;     // [M][n_q][d_h] hi
  bf16_t* q_lo;  // lo
  void* kcache;  // bf16, or e4m3 codes (kv_fp8) of value * kv_inv
  void* vcache;
  int kv_fp8;
  float kv_inv;
  int64_t cap;
  int n_slots;
};
hipError_t launch_rope_stage(const RopeStageArgs& a, const Exec& ex);

hipError_t launch_rope_table(float* rope, int64_t cap, int d_h, double theta, hipStream_t s);

struct KvCopyArgs {
  void* kcache;        // bf16, or e4m3 codes (kv_fp8): imports round, exports widen
  void* vcache;
  int kv_fp8;
  float kv_scale, kv_inv;
  int64_t cap;
  int n_layers, n_slots, n_kv, d_h;
  int slot, pos0, n;
  const bf16_t* k_in;  // import source [n_layers][n][n_kv][d_h]
  const bf16_t* v_in;
  bf16_t* k_out;       // export destination
  bf16_t* v_out;
};
hipError_t launch_kv_import(const KvCopyArgs& a, hipStream_t s);
hipError_t launch_kv_export(const KvCopyArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------- attention
struct AttnArgs {
  const SeqParam* seqs;
  int B, k, layer;
  int n_q, n_kv, d_h;
  const bf16_t* q;     // [B*k][n_q][d_h] hi, pre-scaled by log2(e)/sqrt(d_h)
  const bf16_t* q_lo;  // lo
  const void* kcache;  // bf16, or e4m3 codes (kv_fp8) with the scale kv_scale
  const void* vcache;
  int kv_fp8;
  float kv_scale;
  int64_t cap;
  int n_slots;
  int n_rowblocks;  // ceil(group * k / 64)
  int n_splits;
  int blocks_per_split;  // 32-key blocks per split
  float* part_ml;   // [n_splits][B*k*n_q][2]
  float* part_o;    // [n_splits][B*k*n_q][d_h]
  bf16_t* out;     // [B*k][n_q*d_h] hi (row-major, or fragment order when out_mtiles > 0)
  bf16_t* out_lo;  // lo
  int out_mtiles;  // row tiles of the fragment-order output (0: row-major)
};
hipError_t launch_attention_split(const AttnArgs& a, const Exec& ex);
hipError_t launch_attention_merge(const AttnArgs& a, const Exec& ex);

// ---------------------------------------------------------------------------- fused decode forward
// The whole decode-sized forward (M <= 16 rows: every layer, then the LM head) as one launch
// of one persistent workgroup per CU (fused.hip); phases are separated by counters.
enum FwdPhase { PH_QKV = 0, PH_ATTN, PH_MERGE, PH_O, PH_GU, PH_DOWN, PH_N };
constexpr int kFwdMaxWorkgroups = 256;       // persistent workgroups (one per CU) at most
constexpr int kFwdMaxKw = 16;                // workgroups sharing one 128-column group at most
constexpr int kFwdPartFloats = 2048;         // parked partial of one workgroup: 16 rows x 128 columns
// Counters of one layer: phase counters, two per KV head, one per (sequence, KV head, row
// block) of the attention, one per group of each GEMM phase.
inline int64_t fused_counters_per_layer(int n_kv, int64_t n_qkv, int d, int ffn, int64_t n_attn_groups) {
  return 3 + 2 * n_kv + n_attn_groups + n_qkv / 128 + 2 * (d / 128) + 2 * (int64_t)ffn / 128;
}
struct FwdGains {
  const bf16_t *attn_norm, *mlp_norm, *q_norm, *k_norm;
};
struct FwdPlan {
  int groups[PH_N];    // 128-column groups of the GEMM phases
  int kw[PH_N];        // workgroups per group (each a 1/kw slice of K)
  int units[PH_N];     // groups x kw: completion count of a phase
  int attn_ready_target, merge_target;
  // counters (int32) of layer l start at ctl[ctr0 + l * ctr_stride]
  int ctr0, ctr_stride;
  int c_down_done, c_o_done, c_gu_done;
  int c_attn_ready;    // [n_kv] QKV units done per KV head
  int c_merge_done;    // [n_kv] merge tasks done per KV head
  int c_arr_attn;      // [B][n_kv][row blocks] split tasks done
  int c_arr_q, c_arr_o, c_arr_gu, c_arr_d;  // per-group arrival counters of the GEMM phases
  int n_ctl;           // int32 words to zero before a launch
};
struct FwdArgs {
  int M, B, k, n_layers;
  int d, n_q, n_kv, d_h, ffn, vocab, qk_norm;
  float eps, q_scale;
  const bf16_t* wpack;
  int64_t wp_layer, wp_o, wp_gu, wp_down, wp_lm;
  const FwdGains* gains;  // [n_layers], device
  const bf16_t* final_norm;
  const RowParam* rows;
  const SeqParam* seqs;
  float* x;               // residual stream [M][d]
  bf16_t *xn_d, *xn_d_lo; // x * g after the embedding or a down projection (QKV, LM head input)
  bf16_t *xn_o, *xn_o_lo; // x * g after an O projection (gate/up input)
  float *ssq_d, *ssq_o;   // their partial sums of x^2
  int n_part_embed;       // partials per row written by the embedding (later: one per group)
  bf16_t *q, *q_lo, *attn, *attn_lo, *act, *act_lo;
  bf16_t *kcache, *vcache;
  int64_t cap;
  int n_slots;
  const float* rope;
  int n_rowblocks, n_splits, blocks_per_split;
  float *part_ml, *part_o;
  float* part;            // split-K partial tiles
  float* logits;          // LM head output [lm_rows][vocab]
  int lm_row0, lm_rows;
  FwdPlan plan;
  int* ctl;               // dependency and arrival counters, zeroed before every launch
  int* err;               // [0] sticky error flag, [1] the task that gave up waiting
};
bool fused_plan(FwdArgs& f, int nwg, int64_t part_cap_floats);
hipError_t launch_fused_forward(const FwdArgs& f, int nwg, const Exec& ex);

// ---------------------------------------------------------------------------- per-XCD layer kernels
// A decode-sized layer (M <= 16 rows) as two launches of one workgroup per CU, each XCD
// owning one KV head's share of the work (layer_xcd.hip):
//   layer_attn_kernel: QKV projection (+ q/k norm, RoPE, K/V into the cache), attention,
//                      merge and O projection (+ residual, next norm's inputs)
//   layer_mlp_kernel:  gate/up (+ SwiGLU) and down projection (+ residual, next norm's inputs)
constexpr int kXcds = 8;        // XCDs of the chip; workgroup i runs on XCD i % 8
constexpr int kXcdWgs = 32;     // persistent workgroups (CUs) per XCD
constexpr int kLxQkvSlice = 2048 + 16;                    // parked QKV slice: 8 tiles + 16 row sums of x^2
constexpr int kLxQkvFloats = kXcdWgs * kLxQkvSlice;       // per XCD: parked QKV slices
constexpr int kLxAttnTasks = kXcdWgs;                     // attention tasks per XCD at most
constexpr int kLxRows = 64;                               // query rows per KV head at most
constexpr int kLxMaxRows = 16;                            // block rows (batch x k) of a forward at most
constexpr int64_t kLxXcdFloats = kLxQkvFloats + (int64_t)kLxAttnTasks * kLxRows * (128 + 2);
constexpr int64_t kLxPartFloats = (int64_t)kXcds * kLxXcdFloats;  // XCD-local partials
constexpr int kLxCtrLines = kXcds * 64 + 2;               // counter lines (kCtrStride words each)

// The residual stream of these kernels is int64 fixed point, x * 2^32 (x64): the O and down
// projections add their partial products into it with integer atomics (exact, in any order,
// so results do not depend on which XCD finishes first), and each consumer forms its
// normalised operand from it as it streams.
struct LayerXArgs {
  int M, B, k, layer;
  int d, n_q, n_kv, ffn, qk_norm;
  float eps, q_scale;
  int n_tasks;                       // attention key splits per sequence
  const void *wqkv, *wo, *wgu, *wdown;     // packed weights of the layer (bf16_t, or fp8_t)
  const float *sc_qkv, *sc_o, *sc_gu, *sc_down;  // fp8: per-row weight scales of each
  const bf16_t *q_norm, *k_norm;           // Qwen-3 per-head gains (qk_norm)
  const bf16_t* g_attn;              // attention norm gain of the layer
  const bf16_t* g_mlp;               // MLP norm gain of the layer
  const int64_t* x_src;              // residual stream [M][d], fixed point: read by this launch
  int64_t* x_dst;                    // the residual after this launch: zero on entry, atomics add into it
  int64_t* x_zero;                   // the third buffer: zeroed for the next launch
  bf16_t *q, *q_lo, *attn, *attn_lo, *act, *act_lo;
  void *kcache, *vcache;             // bf16, or e4m3 codes (kv_fp8)
  int kv_fp8;
  float kv_scale, kv_inv;
  int64_t cap;
  int n_slots;
  const float* rope;
  const RowParam* rows;
  const SeqParam* seqs;
  float* xpart;                      // kLxPartFloats
  int* ctr;                          // kLxCtrLines * kCtrStride words, zero at creation
  int* err;                          // sticky error word and the task code of a failed wait
  int* err_host;                     // pinned host copy of the same two words
  int spin_limit;                    // polls before a wait gives up
};
constexpr int kLxSpinDefault = 1 << 21;
// After the last layer: x (fp32), x * g (hi, lo) and per-16-column sums of squares of the
// fixed-point residual, the inputs of the LM head.
struct FinalizeArgs {
  int M, d;
  const int64_t* x64;
  const bf16_t* g;
  float* x;
  bf16_t *xn, *xn_lo;
  float* sumsq;  // [M][d/16]
};
// True when the per-XCD layer kernels implement this decode-sized forward on this device.
bool layer_xcd_fits(const sbd_model_config& c, int n_cu, int B, int k);
hipError_t launch_layer_attn(const LayerXArgs& a, bool fp8, const Exec& ex);
hipError_t launch_layer_mlp(const LayerXArgs& a, bool fp8, const Exec& ex);
hipError_t launch_layer_finalize(const FinalizeArgs& a, const Exec& ex);

// ---------------------------------------------------------------------------- EB sampler
struct EbArgs {
  int B, k, vocab, mask_id;
  const float* logits;      // [B][k][vocab]
  const uint8_t* is_mask;   // device [B][k]
  const double* entropy_in; // select-only mode: device [B][k]
  double gamma;
  int n_chunks;
  double* part;             // [B*k][n_chunks][3] (max, Z, S)
  int32_t* part_arg;        // [B*k][n_chunks]
  int32_t* n_accepted;      // [B]
  int32_t* accepted_pos;    // [B][k]
  int32_t* accepted_tok;    // [B][k] or null
  double* entropy_out;      // [B][k] or null
  int rule;                 // SBD_SELECT_*: the order and the stopping rule (gamma = its threshold)
  double* conf_out;         // [B][k] or null: max_v p_v of masked rows
  // Statistics from the LM head (sbd_block_step): eb_merge_kernel reduces the 64-column
  // chunks in part / part_arg (n_chunks per row) to these per-row values, which the select
  // kernel then takes (row_stats != null selects that mode).
  double* row_stats;        // [B*k][2]: entropy, confidence
  int32_t* row_tok;         // [B*k]
  // Masks of up to kEbInlineRows rows travel in the kernel arguments (bit r of mask_bits is
  // row r) instead of an upload on the stream; is_mask is then null.
  uint64_t mask_bits[kEbInlineRows / 64];
};
__device__ __forceinline__ bool eb_row_masked(const EbArgs& a, int64_t row) {
  return a.is_mask ? a.is_mask[row] != 0 : ((a.mask_bits[row >> 6] >> (row & 63)) & 1ull) != 0;
}
hipError_t launch_eb_partial(const EbArgs& a, const Exec& ex);
// Limits of sbd_eb_select_noalloc and the device address of its file-scope scratch on the
// current device (looked up once per device).
constexpr int kNoAllocRows = 1024;       // batch * k
constexpr int kNoAllocChunks = 64;       // vocab <= 64 * kEbChunk = 262144
constexpr int kNoAllocMaxDevices = 64;
hipError_t eb_noalloc_scratch(double** part, int32_t** part_arg);
hipError_t launch_eb_select(const EbArgs& a, bool select_only, const Exec& ex);
hipError_t launch_eb_merge(const EbArgs& a, const Exec& ex);
// Packing of e4m3 matrices (mode as launch_pack): into the fp8 packing, or widened to the
// bf16 packing with the scales 2^e0 (src0) and 2^e1 (src1).
hipError_t launch_pack_fp8(const fp8_t* src0, const fp8_t* src1, fp8_t* dst, int64_t rows, int K, int mode,
                           hipStream_t s);
hipError_t launch_pack_fp8_widen(const fp8_t* src0, const fp8_t* src1, int e0, int e1, bf16_t* dst, int64_t rows,
                                 int K, int mode, hipStream_t s);
hipError_t launch_xcd_probe(int* out, int n, hipStream_t s);
constexpr int kXcdProbeMax = 2048;  // largest probed grid
hipError_t launch_stream_probe(const void* buf, int64_t bytes, uint32_t* sink, int n_cu, hipStream_t s);

}  // namespace sbd

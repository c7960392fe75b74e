// C ABI of the SBD decode step: argument/state validation, KV-cache bookkeeping and the
// launch sequence of the block forward (eq. (hybrid_block) of Set Block Decoding) and of
// the EB-Sampler step (eq. (eb_sampler)).  Everything here runs on the host; all
// arithmetic happens in the kernels of gemm.hip, attention.hip, misc.hip and eb.hip.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "sbd_internal.h"

using namespace sbd;

namespace {

thread_local std::string g_err;  // last error of a context-less call

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

int effective_chunk(const sbd_model_config& c) { return c.prefill_chunk > 0 ? c.prefill_chunk : 256; }

// The KV cache's format as the kernels take it: e4m3 codes of value * inv, read back times
// scale (scale = 2^kv_scale_exp, exact), or bf16.
struct KvFmt {
  int fp8;
  float scale, inv;
};
KvFmt kv_fmt(const sbd_model_config& m) {
  if (m.kv_format != SBD_KV_FP8_E4M3) return KvFmt{0, 1.f, 1.f};
  return KvFmt{1, std::ldexp(1.f, m.kv_scale_exp), std::ldexp(1.f, -m.kv_scale_exp)};
}

const char* check_config(const sbd_model_config& c) {
  if (c.n_layers < 1) return "n_layers must be >= 1";
  if (c.d_model < 256 || c.d_model % 256) return "d_model must be a positive multiple of 256";
  if (c.head_dim != 64 && c.head_dim != 128) return "head_dim must be 64 or 128";
  if (c.n_q_heads < 1 || c.n_kv_heads < 1 || c.n_q_heads % c.n_kv_heads)
    return "n_q_heads must be a positive multiple of n_kv_heads";
  if ((c.n_q_heads * c.head_dim) % 256) return "n_q_heads*head_dim must be a multiple of 256";
  if (c.ffn_dim < 256 || c.ffn_dim % 256) return "ffn_dim must be a positive multiple of 256";
  if (c.vocab < 128 || c.vocab % 128) return "vocab must be a positive multiple of 128";
  if (((c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim) % 128)
    return "(n_q_heads + 2 n_kv_heads) * head_dim must be a multiple of 128";
  if (c.mask_id < 0 || c.mask_id >= c.vocab) return "mask_id must lie in [0, vocab)";
  if (c.qk_norm != 0 && c.qk_norm != 1) return "qk_norm must be 0 or 1";
  if (!(c.rms_eps > 0.f) || !std::isfinite(c.rms_eps)) return "rms_eps must be a positive number";
  if (!(c.rope_theta > 0.f) || !std::isfinite(c.rope_theta)) return "rope_theta must be a positive number";
  if (c.max_batch < 1 || c.max_batch > 4096) return "max_batch must lie in [1, 4096]";
  if (c.max_seq_len < 1 || c.max_seq_len > (1 << 24)) return "max_seq_len must lie in [1, 2^24]";
  if (c.max_block < 1 || c.max_block > kMaxBlock) return "max_block must lie in [1, 64]";
  if (c.prefill_chunk < 0 || c.prefill_chunk > 4096) return "prefill_chunk must lie in [0, 4096]";
  if (c.weight_format != SBD_WEIGHTS_BF16 && c.weight_format != SBD_WEIGHTS_FP8_E4M3)
    return "weight_format must be SBD_WEIGHTS_BF16 or SBD_WEIGHTS_FP8_E4M3";
  if (c.kv_format != SBD_KV_BF16 && c.kv_format != SBD_KV_FP8_E4M3)
    return "kv_format must be SBD_KV_BF16 or SBD_KV_FP8_E4M3";
  if (c.kv_format == SBD_KV_FP8_E4M3 && (c.kv_scale_exp < -100 || c.kv_scale_exp > 100))
    return "kv_scale_exp must lie in [-100, 100]";
  return nullptr;
}

}  // namespace

bool sbd::compute_layout(const sbd_model_config& c, Layout* L) {
  if (check_config(c)) return false;
  Layout o{};
  o.cap = ((int64_t)c.max_seq_len + 63) / 64 * 64;
  o.m_max = std::max<int64_t>((int64_t)c.max_batch * c.max_block, effective_chunk(c));
  o.m_max = (o.m_max + 15) / 16 * 16;  // whole row tiles: fragment-order activations
  o.n_qkv = (int64_t)(c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim;
  o.n_part = c.d_model / 16;
  o.eb_chunks = (c.vocab + kEbChunk - 1) / kEbChunk;
  const int64_t qd = (int64_t)c.n_q_heads * c.head_dim;
  const int64_t kv_elems = (int64_t)c.n_layers * c.max_batch * c.n_kv_heads * o.cap * c.head_dim;
  const int64_t eb_rows = (int64_t)c.max_batch * c.max_block;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  const int64_t kv_es = c.kv_format == SBD_KV_FP8_E4M3 ? 1 : 2;  // bytes per cached element
  o.kcache = take(kv_elems * kv_es);
  o.vcache = take(kv_elems * kv_es);
  o.rope = take(o.cap * (c.head_dim / 2) * 2 * sizeof(float));
  o.x = take(o.m_max * c.d_model * sizeof(float));
  o.xn = take(2 * o.m_max * c.d_model * 2);             // hi then lo
  o.sumsq = take(o.m_max * o.n_part * sizeof(float));
  o.qkv = take(o.m_max * o.n_qkv * sizeof(float));
  o.q = take(2 * o.m_max * qd * 2);
  o.attn = take(2 * o.m_max * qd * 2);
  o.act = take(2 * o.m_max * (int64_t)c.ffn_dim * 2);
  o.attn_ml = take((int64_t)kMaxSplits * o.m_max * c.n_q_heads * 2 * sizeof(float));
  o.attn_o = take((int64_t)kMaxSplits * o.m_max * qd * sizeof(float));
  o.rows = take(o.m_max * sizeof(RowParam));
  o.seqs = take((int64_t)c.max_batch * sizeof(SeqParam));
  o.eb_mask = take(eb_rows);
  o.eb_part = take(eb_rows * o.eb_chunks * 3 * sizeof(double));
  o.eb_arg = take(eb_rows * o.eb_chunks * sizeof(int32_t));
  o.eb_frows = std::min<int64_t>(eb_rows, kStepMaxRows);
  o.eb_fchunks = c.vocab / kEbFChunk;
  o.eb_fpart = take(o.eb_frows * o.eb_fchunks * 3 * sizeof(double));
  o.eb_farg = take(o.eb_frows * o.eb_fchunks * sizeof(int32_t));
  o.eb_rowstat = take(o.eb_frows * 2 * sizeof(double));
  o.eb_rowtok = take(o.eb_frows * sizeof(int32_t));
  // packed weights: per layer qkv [n_qkv][d], o [d][qd], gate/up [2F][d], down [d][F]
  o.wp_o = o.n_qkv * c.d_model;
  o.wp_gu = o.wp_o + (int64_t)c.d_model * qd;
  o.wp_down = o.wp_gu + 2 * (int64_t)c.ffn_dim * c.d_model;
  o.wp_layer = o.wp_down + (int64_t)c.d_model * c.ffn_dim;
  o.wp_lm = o.wp_layer * c.n_layers;
  o.wpack = take((o.wp_lm + (int64_t)c.vocab * c.d_model) * 2);
  if (c.weight_format == SBD_WEIGHTS_FP8_E4M3) {
    o.wpack8 = take(o.wp_lm + (int64_t)c.vocab * c.d_model);
    o.ws_o = o.n_qkv;
    o.ws_gu = o.ws_o + c.d_model;
    o.ws_down = o.ws_gu + 2 * (int64_t)c.ffn_dim;
    o.ws_layer = o.ws_down + c.d_model;
    o.ws_lm = o.ws_layer * c.n_layers;
    o.wscale = take((o.ws_lm + c.vocab) * sizeof(float));
  }
  const int64_t widest = std::max<int64_t>(std::max<int64_t>(o.n_qkv, 2 * (int64_t)c.ffn_dim), c.d_model);
  // split-K partials of the per-kernel path, or the parked partial tiles of the fused forward
  o.gemv_part_floats = std::max<int64_t>((int64_t)kGemvMaxSplit * 16 * widest, (int64_t)kFwdMaxWorkgroups * kFwdPartFloats);
  // M > 16: up to 8 K slices of every output of the QKV, O and down projections at 256 rows
  o.gemv_part_floats = std::max<int64_t>(o.gemv_part_floats, 8 * std::min<int64_t>(o.m_max, 256) *
                                                                 std::max<int64_t>(o.n_qkv, c.d_model));
  o.gemv_part = take(o.gemv_part_floats * sizeof(float));
  o.xn2 = take(2 * o.m_max * c.d_model * 2);
  o.sumsq2 = take(o.m_max * o.n_part * sizeof(float));
  o.fwd_gains = take((int64_t)c.n_layers * sizeof(FwdGains));
  const int64_t n_rb_max = ((int64_t)(c.n_q_heads / c.n_kv_heads) * c.max_block + 63) / 64;
  o.fwd_ctl_ints = (int64_t)c.n_layers *
                   fused_counters_per_layer(c.n_kv_heads, o.n_qkv, c.d_model, c.ffn_dim,
                                            (int64_t)c.max_batch * c.n_kv_heads * n_rb_max);
  o.fwd_ctl = take(o.fwd_ctl_ints * sizeof(int32_t));
  o.fwd_err = take(2 * sizeof(int32_t));
  o.lx_part = take(kLxPartFloats * sizeof(float));
  o.x64 = take(3 * kLxMaxRows * (int64_t)c.d_model * sizeof(int64_t));  // three residual buffers
  o.counters = take((int64_t)kCounters * sizeof(int32_t));
  o.total = off;
  *L = o;
  return true;
}

struct sbd_ctx {
  sbd_model_config cfg{};
  Layout lay{};
  std::vector<LayerW> layers;
  const bf16_t *embed = nullptr, *lm_head = nullptr, *final_norm = nullptr;
  char* ws = nullptr;
  hipStream_t stream = nullptr;
  std::vector<int32_t> cache_len, staged;
  static constexpr int kRing = 4;
  void* stage[kRing] = {};
  hipEvent_t ev[kRing] = {};
  bool ev_used[kRing] = {};
  int ring = 0;
  size_t stage_bytes = 0;
  std::string err;
  // per-kernel timing (sbd_profile_enable)
  bool prof = false;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  int32_t prof_count[SBD_KERNEL_COUNT] = {};
  double prof_ms[SBD_KERNEL_COUNT] = {};
  // decode path for M <= 16 (sbd_set_decode_path)
  int decode_path = SBD_DECODE_AUTO;
  int wait_limit = kLxSpinDefault;  // sbd_set_wait_limit
  int n_cu = 0;                 // workgroups of the fused forward: one per CU, at most kFwdMaxWorkgroups
  int n_cu_dev = 0;             // CUs of the device
  bool xcd_ok = false;          // workgroup i of a launch runs on XCD i % 8 (probed at creation)
  int32_t* err_host = nullptr;  // pinned copy of the fused forward's sticky error word

  template <class T>
  T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

namespace {

sbd_status fail(sbd_ctx* c, sbd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf; else g_err = buf;
  return st;
}

#define SBD_HIP(ctx, expr)                                                                  \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail(ctx, SBD_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

// Asynchronous faults of earlier work surface here.
sbd_status check_sticky(sbd_ctx* c) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(c, SBD_ERR_HIP, "earlier HIP error: %s", hipGetErrorString(e));
  // written by copies queued after each fused forward, or by a layer kernel or GEMM whose
  // wait gave up; it never goes back to zero
  if (c->err_host != nullptr && __atomic_load_n(c->err_host, __ATOMIC_ACQUIRE) != 0)
    return fail(c, SBD_ERR_HIP, "a forward gave up waiting for its inputs (task code %d: layer * 16 + phase "
                "of a per-XCD layer kernel, or 65536 + epilogue of a GEMM's K slices)",
                __atomic_load_n(c->err_host + 1, __ATOMIC_ACQUIRE));
  return SBD_OK;
}

// Copy host bytes to a device address on the context stream through a pinned ring slot.
sbd_status upload(sbd_ctx* c, void* dst, const void* src, size_t bytes) {
  if (bytes == 0) return SBD_OK;
  if (bytes > c->stage_bytes) return fail(c, SBD_ERR_INVALID_ARG, "upload of %zu bytes too large", bytes);
  const int i = c->ring;
  c->ring = (c->ring + 1) % sbd_ctx::kRing;
  if (c->ev_used[i]) SBD_HIP(c, hipEventSynchronize(c->ev[i]));
  std::memcpy(c->stage[i], src, bytes);
  SBD_HIP(c, hipMemcpyAsync(dst, c->stage[i], bytes, hipMemcpyHostToDevice, c->stream));
  SBD_HIP(c, hipEventRecord(c->ev[i], c->stream));
  c->ev_used[i] = true;
  return SBD_OK;
}

hipEvent_t take_event(sbd_ctx* c) {
  if (!c->pool.empty()) {
    hipEvent_t e = c->pool.back();
    c->pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Launch one kernel on the context stream: `expr` uses the Exec named `ex`.  When
// profiling, the runtime records a pair of events at the kernel's start and end.
#define SBD_LAUNCH(ctx, kind, expr)                                               \
  do {                                                                            \
    Exec ex{(ctx)->stream, nullptr, nullptr};                                     \
    if ((ctx)->prof) {                                                            \
      ex.start = take_event(ctx);                                                 \
      ex.stop = take_event(ctx);                                                  \
      if (!ex.start || !ex.stop) return fail(ctx, SBD_ERR_HIP, "hipEventCreate failed"); \
    }                                                                             \
    SBD_HIP(ctx, expr);                                                           \
    if ((ctx)->prof) (ctx)->recs.push_back(sbd_ctx::Rec{kind, ex.start, ex.stop}); \
  } while (0)

// K may be split over workgroups that hand their partials off through one XCD's L2, and
// the slices of a unit may wait for each other, only when the device places workgroup i on
// XCD i % 8 (probed at creation)
GemmArgs gemm_base(const bf16_t* A, const bf16_t* A_lo, int64_t lda, int M, int K, const bf16_t* Wp,
                   int n_tiles, float* part, int64_t part_cap, int* counters, const sbd_ctx* c) {
  GemmArgs g{};
  g.A = A; g.A_lo = A_lo; g.lda = lda; g.M = M; g.K = K; g.Wp = Wp; g.n_tiles = n_tiles;
  g.part = part; g.part_cap = part_cap; g.counters = counters; g.no_split = c->xcd_ok ? 0 : 1;
  g.wait_ok = c->xcd_ok ? 1 : 0;
  g.spin_limit = c->wait_limit;
  g.err = c->at<int>(c->lay.fwd_err);
  g.err_host = c->err_host;
  return g;
}

GemvArgs gemv_base(const bf16_t* A, const bf16_t* A_lo, int64_t lda, int M, int K, const bf16_t* Wp,
                   int n_tiles, float* part, int64_t part_cap, int* counters, bool split_ok) {
  GemvArgs v{};
  v.A = A; v.A_lo = A_lo; v.lda = lda; v.M = M; v.K = K; v.Wp = Wp; v.n_tiles = n_tiles;
  v.part = part; v.part_cap = part_cap; v.counters = counters; v.no_split = split_ok ? 0 : 1;
  return v;
}

// Key splits of the attention: enough workgroups for one round of one per CU (a workgroup
// takes 128 KB of LDS), as long as every split keeps a block.  More rounds cost a
// workgroup's start (queries, first stage of the ring, final combine and partial store)
// again on every CU: with ragged lengths (batch 32, 512 to 4096 positions) four splits
// instead of one took the attention from 92 to 105 us.
int pick_splits(int64_t work_groups_per_split, int nblocks, int n_cu) {
  const int64_t target = std::max(1, n_cu);
  int s = (int)std::max<int64_t>(1, (target + work_groups_per_split - 1) / work_groups_per_split);
  s = std::min(s, kMaxSplits);
  s = std::min(s, std::max(1, nblocks));
  return s;
}

// The LM head's EB statistics (sbd_block_step): 64-column chunk statistics of every row.
struct LmEb {
  double* part;
  int32_t* arg;
  int chunks, mask_id;
};

// One forward of B sequences x k rows whose per-row / per-sequence parameters are given.
// lm_row < 0: logits for all rows into `logits`; otherwise only for row lm_row.  eb: the LM
// head also writes the EB chunk statistics of all rows (logits may then be null).
sbd_status run_forward(sbd_ctx* c, int B, int k, const std::vector<RowParam>& rows,
                       const std::vector<SeqParam>& seqs, float* logits, int lm_row, const LmEb* eb = nullptr) {
  const sbd_model_config& m = c->cfg;
  const Layout& L = c->lay;
  const int M = B * k;
  const int d = m.d_model, dh = m.head_dim, nq = m.n_q_heads, nkv = m.n_kv_heads;
  const int qd = nq * dh;
  float* x = c->at<float>(L.x);
  bf16_t* xn = c->at<bf16_t>(L.xn);
  bf16_t* xn_lo = xn + L.m_max * d;
  float* sumsq = c->at<float>(L.sumsq);
  float* qkv = c->at<float>(L.qkv);
  bf16_t* q = c->at<bf16_t>(L.q);
  bf16_t* q_lo = q + L.m_max * qd;
  bf16_t* attn = c->at<bf16_t>(L.attn);
  bf16_t* attn_lo = attn + L.m_max * qd;
  bf16_t* act = c->at<bf16_t>(L.act);
  bf16_t* act_lo = act + L.m_max * (int64_t)m.ffn_dim;
  const RowParam* drows = c->at<RowParam>(L.rows);
  const SeqParam* dseqs = c->at<SeqParam>(L.seqs);
  float* vpart = c->at<float>(L.gemv_part);
  const int64_t vpart_cap = L.gemv_part_floats;
  int max_end = 0;
  for (const SeqParam& s : seqs) max_end = std::max(max_end, s.cache_len + k);
  const int G = nq / nkv;
  const int n_rb = (G * k + 63) / 64;
  const int nblocks = (max_end + 31) / 32;
  const bool small = M <= 16;  // decode-sized forward
  // fp8 weights: the GEMVs, layer kernels and GEMMs stream the bytes (the fused path the
  // widened bf16 copy)
  const bool f8 = m.weight_format == SBD_WEIGHTS_FP8_E4M3;
  auto w8 = [&](int64_t off, int64_t soff, GemvArgs& v) {
    if (f8) { v.Wp8 = c->at<fp8_t>(L.wpack8) + off; v.wscale = c->at<float>(L.wscale) + soff; }
  };
  auto g8 = [&](int64_t off, int64_t soff, GemmArgs& g) {  // the GEMM for more rows streams them too
    if (f8) { g.Wp8 = c->at<fp8_t>(L.wpack8) + off; g.wscale = c->at<float>(L.wscale) + soff; }
  };
  // forwards of more than 16 rows keep the GEMMs' activation operands in fragment order
  const int mt = small ? 0 : (M + 15) / 16;
  // the KV cache: bf16, or e4m3 codes of value * 2^-e
  const KvFmt kvf = kv_fmt(m);
  void* kcache = c->ws + L.kcache;
  void* vcache = c->ws + L.vcache;

  // The fused decode forward: checked before anything is enqueued.
  const bool fused = small && c->decode_path == SBD_DECODE_FUSED;
  FwdArgs f{};
  if (fused && kvf.fp8)
    return fail(c, SBD_ERR_UNSUPPORTED, "the fused decode forward reads a bf16 KV cache only");
  if (fused) {
    f.M = M; f.B = B; f.k = k; f.n_layers = m.n_layers;
    f.d = d; f.n_q = nq; f.n_kv = nkv; f.d_h = dh; f.ffn = m.ffn_dim; f.vocab = m.vocab; f.qk_norm = m.qk_norm;
    f.eps = m.rms_eps;
    f.q_scale = (float)(1.4426950408889634 / std::sqrt((double)dh));
    f.wpack = c->at<bf16_t>(L.wpack);
    f.wp_layer = L.wp_layer; f.wp_o = L.wp_o; f.wp_gu = L.wp_gu; f.wp_down = L.wp_down; f.wp_lm = L.wp_lm;
    f.gains = c->at<FwdGains>(L.fwd_gains); f.final_norm = c->final_norm;
    f.rows = drows; f.seqs = dseqs;
    f.x = x; f.xn_d = xn; f.xn_d_lo = xn_lo;
    f.xn_o = c->at<bf16_t>(L.xn2); f.xn_o_lo = f.xn_o + L.m_max * d;
    f.ssq_d = sumsq; f.ssq_o = c->at<float>(L.sumsq2); f.n_part_embed = d / 16;
    f.q = q; f.q_lo = q_lo; f.attn = attn; f.attn_lo = attn_lo; f.act = act; f.act_lo = act_lo;
    f.kcache = c->at<bf16_t>(L.kcache); f.vcache = c->at<bf16_t>(L.vcache); f.cap = L.cap;
    f.n_slots = m.max_batch; f.rope = c->at<float>(L.rope);
    // key splits: as many as fit one attention task per workgroup
    const int per = B * nkv * n_rb;
    const int fit = std::min(nblocks, std::max(1, std::min(kMaxSplits, std::max(1, c->n_cu) / per)));
    const int fbps = (nblocks + fit - 1) / fit;
    f.n_rowblocks = n_rb; f.blocks_per_split = fbps; f.n_splits = (nblocks + fbps - 1) / fbps;
    f.part_ml = c->at<float>(L.attn_ml); f.part_o = c->at<float>(L.attn_o);
    f.part = vpart;
    f.logits = logits; f.lm_row0 = lm_row < 0 ? 0 : lm_row; f.lm_rows = lm_row < 0 ? M : 1;
    f.ctl = c->at<int>(L.fwd_ctl); f.err = c->at<int>(L.fwd_err);
    if (c->n_cu < 1 || !fused_plan(f, c->n_cu, vpart_cap) || f.plan.n_ctl > L.fwd_ctl_ints)
      return fail(c, SBD_ERR_UNSUPPORTED, "the fused decode forward does not fit this model or device (%d CUs)",
                  c->n_cu);
  }

  // The per-XCD layer kernels: chosen by AUTO where they apply; checked before anything is
  // enqueued when asked for explicitly.
  const bool layers_fit = small && !fused && c->decode_path != SBD_DECODE_KERNELS &&
                          c->xcd_ok && layer_xcd_fits(m, c->n_cu_dev, B, k);
  if (small && c->decode_path == SBD_DECODE_LAYERS && !layers_fit)
    return fail(c, SBD_ERR_UNSUPPORTED, "the per-XCD layer kernels do not fit this forward or device (%d CUs%s)",
                c->n_cu_dev, c->xcd_ok ? "" : "; workgroup i does not run on XCD i % 8 here");

  sbd_status st = upload(c, c->ws + L.rows, rows.data(), rows.size() * sizeof(RowParam));
  if (st) return st;
  st = upload(c, c->ws + L.seqs, seqs.data(), seqs.size() * sizeof(SeqParam));
  if (st) return st;
  // the per-XCD layer kernels' residual buffers R0, R1, R2 (kLxMaxRows rows each)
  int64_t* xr[3];
  for (int i = 0; i < 3; ++i) xr[i] = c->at<int64_t>(L.x64) + (int64_t)i * kLxMaxRows * d;
  EmbedArgs ea{drows, M, d, c->embed, c->layers[0].attn_norm, x, xn, xn_lo, sumsq, mt,
               layers_fit ? xr[0] : nullptr, layers_fit ? xr[1] : nullptr};
  SBD_LAUNCH(c, SBD_KERNEL_EMBED, launch_embed(ea, ex));
  if (fused) {
    SBD_HIP(c, hipMemsetAsync(f.ctl, 0, (size_t)f.plan.n_ctl * sizeof(int32_t), c->stream));
    SBD_LAUNCH(c, SBD_KERNEL_FUSED, launch_fused_forward(f, c->n_cu, ex));
    SBD_HIP(c, hipMemcpyAsync(c->err_host, f.err, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, c->stream));
    return SBD_OK;
  }

  // Per-kernel path; for decode-sized forwards the QKV epilogue is fused and K is split.
  // Partial sums of x^2 per row handed from each RESID producer to the next consumer:
  // d/16 from the embedding, one per workgroup of the decode O and down projections.
  const int n_part_o = (d / 16) / gemv_pick(EPI_RESID, d / 16, qd).C;
  const int n_part_down = (d / 16) / gemv_pick(EPI_RESID, d / 16, m.ffn_dim).C;
  int n_part_cur = d / 16;
  int* counters = c->at<int>(L.counters);
  int n_splits = pick_splits((int64_t)B * nkv * n_rb, nblocks, c->n_cu_dev);
  const int bps = (nblocks + n_splits - 1) / n_splits;
  n_splits = (nblocks + bps - 1) / bps;

  if (layers_fit) {
    LayerXArgs lx{};
    lx.M = M; lx.B = B; lx.k = k; lx.d = d; lx.n_q = nq; lx.n_kv = nkv; lx.ffn = m.ffn_dim;
    lx.qk_norm = m.qk_norm; lx.eps = m.rms_eps;
    lx.q_scale = (float)(1.4426950408889634 / std::sqrt((double)dh));
    lx.n_tasks = kXcdWgs / B;
    lx.q = q; lx.q_lo = q_lo; lx.attn = attn; lx.attn_lo = attn_lo; lx.act = act; lx.act_lo = act_lo;
    lx.kcache = kcache; lx.vcache = vcache; lx.cap = L.cap;
    lx.kv_fp8 = kvf.fp8; lx.kv_scale = kvf.scale; lx.kv_inv = kvf.inv;
    lx.n_slots = m.max_batch; lx.rope = c->at<float>(L.rope); lx.rows = drows; lx.seqs = dseqs;
    lx.xpart = c->at<float>(L.lx_part);
    lx.ctr = c->at<int>(L.counters) + kLayerCtr0; lx.err = c->at<int>(L.fwd_err); lx.err_host = c->err_host;
    lx.spin_limit = c->wait_limit;
    for (int l = 0; l < m.n_layers; ++l) {
      const LayerW& w = c->layers[l];
      lx.layer = l;
      if (f8) {
        const fp8_t* wp8 = c->at<fp8_t>(L.wpack8) + (int64_t)l * L.wp_layer;
        const float* ws = c->at<float>(L.wscale) + (int64_t)l * L.ws_layer;
        lx.wqkv = wp8; lx.wo = wp8 + L.wp_o; lx.wgu = wp8 + L.wp_gu; lx.wdown = wp8 + L.wp_down;
        lx.sc_qkv = ws; lx.sc_o = ws + L.ws_o; lx.sc_gu = ws + L.ws_gu; lx.sc_down = ws + L.ws_down;
      } else {
        const bf16_t* wp = c->at<bf16_t>(L.wpack) + (int64_t)l * L.wp_layer;
        lx.wqkv = wp; lx.wo = wp + L.wp_o; lx.wgu = wp + L.wp_gu; lx.wdown = wp + L.wp_down;
      }
      lx.q_norm = w.q_norm; lx.k_norm = w.k_norm; lx.g_attn = w.attn_norm; lx.g_mlp = w.mlp_norm;
      // launch i = 2 l + h reads R[i % 3], adds into R[(i + 1) % 3], zeroes R[(i + 2) % 3]
      lx.x_src = xr[(2 * l) % 3]; lx.x_dst = xr[(2 * l + 1) % 3]; lx.x_zero = xr[(2 * l + 2) % 3];
      SBD_LAUNCH(c, SBD_KERNEL_LAYER_ATTN, launch_layer_attn(lx, f8, ex));
      lx.x_src = xr[(2 * l + 1) % 3]; lx.x_dst = xr[(2 * l + 2) % 3]; lx.x_zero = xr[(2 * l + 3) % 3];
      SBD_LAUNCH(c, SBD_KERNEL_LAYER_MLP, launch_layer_mlp(lx, f8, ex));
    }
    // the LM head's inputs (and the fp32 residual) from the fixed-point residual
    FinalizeArgs fa{M, d, xr[(2 * m.n_layers) % 3], c->final_norm, x, xn, xn_lo, sumsq};
    SBD_LAUNCH(c, SBD_KERNEL_LAYER_FINAL, launch_layer_finalize(fa, ex));
    n_part_cur = d / 16;
  }
  for (int l = 0; l < m.n_layers && !layers_fit; ++l) {
    const LayerW& w = c->layers[l];
    const bf16_t* wp = c->at<bf16_t>(L.wpack) + (int64_t)l * L.wp_layer;
    QkvEpi qe{};
    qe.rows = drows; qe.seqs = dseqs; qe.kblk = k; qe.layer = l;
    qe.n_q = nq; qe.n_kv = nkv; qe.d_h = dh; qe.qk_norm = m.qk_norm; qe.eps = m.rms_eps;
    qe.q_scale = (float)(1.4426950408889634 / std::sqrt((double)dh));
    qe.rope = c->at<float>(L.rope); qe.q_norm = w.q_norm; qe.k_norm = w.k_norm;
    qe.q = q; qe.q_lo = q_lo; qe.kcache = kcache; qe.vcache = vcache;
    qe.kv_fp8 = kvf.fp8; qe.kv_inv = kvf.inv;
    qe.cap = L.cap; qe.n_slots = m.max_batch;
    if (small) {
      // QKV + q/k norm + RoPE + KV staging in one kernel
      GemvArgs v = gemv_base(xn, xn_lo, d, M, d, wp, (int)(L.n_qkv / 16), vpart, vpart_cap, counters, c->xcd_ok);
      w8((int64_t)l * L.wp_layer, (int64_t)l * L.ws_layer, v);
      v.sumsq_in = sumsq; v.n_part_in = n_part_cur; v.inv_d = 1.0f / d; v.eps = m.rms_eps;
      v.qkv = qe;
      SBD_LAUNCH(c, SBD_KERNEL_QKV, launch_gemv(EPI_QKV, v, GemvShape{}, ex));
    } else {
      GemmArgs g = gemm_base(xn, xn_lo, d, M, d, wp, (int)(L.n_qkv / 16), vpart, vpart_cap, counters, c);
      g8((int64_t)l * L.wp_layer, (int64_t)l * L.ws_layer, g);
      g.a_mtiles = mt;
      g.out_f32 = qkv; g.ldo = L.n_qkv;
      g.sumsq_in = sumsq; g.n_part = n_part_cur; g.inv_d = 1.0f / d; g.eps = m.rms_eps;
      SBD_LAUNCH(c, SBD_KERNEL_QKV, launch_gemm(EPI_SCALED_STORE, g, ex));
      RopeStageArgs ra{};
      ra.rows = drows; ra.seqs = dseqs; ra.M = M; ra.k = k; ra.layer = l;
      ra.n_q = nq; ra.n_kv = nkv; ra.d_h = dh; ra.qk_norm = m.qk_norm; ra.eps = m.rms_eps;
      ra.q_scale = qe.q_scale;
      ra.qkv = qkv; ra.q_norm = w.q_norm; ra.k_norm = w.k_norm; ra.rope = c->at<float>(L.rope);
      ra.q = q; ra.q_lo = q_lo; ra.kcache = kcache; ra.vcache = vcache;
      ra.kv_fp8 = kvf.fp8; ra.kv_inv = kvf.inv;
      ra.cap = L.cap; ra.n_slots = m.max_batch;
      SBD_LAUNCH(c, SBD_KERNEL_ROPE, launch_rope_stage(ra, ex));
    }

    AttnArgs aa{};
    aa.seqs = dseqs; aa.B = B; aa.k = k; aa.layer = l; aa.n_q = nq; aa.n_kv = nkv; aa.d_h = dh;
    aa.q = q; aa.q_lo = q_lo; aa.kcache = kcache; aa.vcache = vcache; aa.cap = L.cap; aa.n_slots = m.max_batch;
    aa.kv_fp8 = kvf.fp8; aa.kv_scale = kvf.scale;
    aa.n_rowblocks = n_rb; aa.n_splits = n_splits; aa.blocks_per_split = bps;
    aa.part_ml = c->at<float>(L.attn_ml); aa.part_o = c->at<float>(L.attn_o); aa.out = attn;
    aa.out_lo = attn_lo;
    aa.out_mtiles = mt;
    SBD_LAUNCH(c, SBD_KERNEL_ATTENTION, launch_attention_split(aa, ex));
    if (n_splits > 1) SBD_LAUNCH(c, SBD_KERNEL_ATTN_MERGE, launch_attention_merge(aa, ex));

    if (small) {
      GemvArgs v = gemv_base(attn, attn_lo, qd, M, qd, wp + L.wp_o, d / 16, vpart, vpart_cap, counters, c->xcd_ok);
      w8((int64_t)l * L.wp_layer + L.wp_o, (int64_t)l * L.ws_layer + L.ws_o, v);
      v.x = x; v.ldx = d; v.xn = xn; v.xn_lo = xn_lo; v.g_next = w.mlp_norm;
      v.sumsq = sumsq; v.n_part = n_part_o;
      SBD_LAUNCH(c, SBD_KERNEL_O_PROJ, launch_gemv(EPI_RESID, v, GemvShape{}, ex));
    } else {
      GemmArgs go = gemm_base(attn, attn_lo, qd, M, qd, wp + L.wp_o, d / 16, vpart, vpart_cap, counters, c);
      g8((int64_t)l * L.wp_layer + L.wp_o, (int64_t)l * L.ws_layer + L.ws_o, go);
      go.a_mtiles = mt; go.o_mtiles = mt;
      go.x = x; go.ldx = d; go.xn = xn; go.xn_lo = xn_lo; go.g_next = w.mlp_norm; go.sumsq_out = sumsq;
      go.n_part_out = gemm_plan(M, d / 16, qd, c->xcd_ok ? vpart_cap : 0).n_cb;
      n_part_cur = go.n_part_out;
      SBD_LAUNCH(c, SBD_KERNEL_O_PROJ, launch_gemm(EPI_RESID, go, ex));
    }

    const bf16_t* g_after = (l + 1 < m.n_layers) ? c->layers[l + 1].attn_norm : c->final_norm;
    if (small) {
      GemvArgs vu = gemv_base(xn, xn_lo, d, M, d, wp + L.wp_gu, m.ffn_dim / 8, vpart, vpart_cap, counters, c->xcd_ok);
      w8((int64_t)l * L.wp_layer + L.wp_gu, (int64_t)l * L.ws_layer + L.ws_gu, vu);
      vu.sumsq_in = sumsq; vu.n_part_in = n_part_o; vu.inv_d = 1.0f / d; vu.eps = m.rms_eps;
      vu.act = act; vu.act_lo = act_lo; vu.ld_act = m.ffn_dim;
      SBD_LAUNCH(c, SBD_KERNEL_GATE_UP, launch_gemv(EPI_SWIGLU, vu, GemvShape{}, ex));
      GemvArgs vd = gemv_base(act, act_lo, m.ffn_dim, M, m.ffn_dim, wp + L.wp_down, d / 16, vpart, vpart_cap, counters, c->xcd_ok);
      w8((int64_t)l * L.wp_layer + L.wp_down, (int64_t)l * L.ws_layer + L.ws_down, vd);
      vd.x = x; vd.ldx = d; vd.xn = xn; vd.xn_lo = xn_lo; vd.g_next = g_after;
      vd.sumsq = sumsq; vd.n_part = n_part_down;
      n_part_cur = n_part_down;
      SBD_LAUNCH(c, SBD_KERNEL_DOWN, launch_gemv(EPI_RESID, vd, GemvShape{}, ex));
    } else {
      GemmArgs gu = gemm_base(xn, xn_lo, d, M, d, wp + L.wp_gu, m.ffn_dim / 8, vpart, vpart_cap, counters, c);
      g8((int64_t)l * L.wp_layer + L.wp_gu, (int64_t)l * L.ws_layer + L.ws_gu, gu);
      gu.a_mtiles = mt; gu.o_mtiles = mt;
      gu.sumsq_in = sumsq; gu.n_part = n_part_cur; gu.inv_d = 1.0f / d; gu.eps = m.rms_eps;
      gu.act = act; gu.act_lo = act_lo; gu.ld_act = m.ffn_dim;
      SBD_LAUNCH(c, SBD_KERNEL_GATE_UP, launch_gemm(EPI_SWIGLU, gu, ex));

      GemmArgs gd = gemm_base(act, act_lo, m.ffn_dim, M, m.ffn_dim, wp + L.wp_down, d / 16, vpart, vpart_cap,
                              counters, c);
      g8((int64_t)l * L.wp_layer + L.wp_down, (int64_t)l * L.ws_layer + L.ws_down, gd);
      gd.a_mtiles = mt; gd.o_mtiles = mt;
      gd.x = x; gd.ldx = d; gd.xn = xn; gd.xn_lo = xn_lo; gd.g_next = g_after;
      gd.sumsq_out = sumsq;
      gd.n_part_out = gemm_plan(M, d / 16, m.ffn_dim, c->xcd_ok ? vpart_cap : 0).n_cb;
      n_part_cur = gd.n_part_out;
      SBD_LAUNCH(c, SBD_KERNEL_DOWN, launch_gemm(EPI_RESID, gd, ex));
    }
  }

  if (logits != nullptr || eb != nullptr) {
    const int r0 = lm_row < 0 ? 0 : lm_row;
    const int Ml = lm_row < 0 ? M : 1;
    const GemmEpi lm_epi = eb ? EPI_LOGITS_EB : EPI_SCALED_STORE;
    if (mt == 0) {  // M <= 16: row-major inputs
      GemvArgs v = gemv_base(xn + (int64_t)r0 * d, xn_lo + (int64_t)r0 * d, d, Ml, d,
                             c->at<bf16_t>(L.wpack) + L.wp_lm, m.vocab / 16, vpart, vpart_cap, counters, c->xcd_ok);
      w8(L.wp_lm, L.ws_lm, v);
      v.sumsq_in = sumsq + (int64_t)r0 * n_part_cur; v.n_part_in = n_part_cur;
      v.inv_d = 1.0f / d; v.eps = m.rms_eps;
      v.out_f32 = logits; v.ldo = m.vocab;
      if (eb) { v.eb_part = eb->part; v.eb_arg = eb->arg; v.eb_chunks = eb->chunks; v.eb_mask_id = eb->mask_id; }
      SBD_LAUNCH(c, SBD_KERNEL_LM_HEAD, launch_gemv(lm_epi, v, GemvShape{}, ex));
    } else {
      // inputs in fragment order (also for one row of a prefill chunk: rows from a_row0)
      GemmArgs gl = gemm_base(xn, xn_lo, d, Ml, d, c->at<bf16_t>(L.wpack) + L.wp_lm, m.vocab / 16, vpart,
                              vpart_cap, counters, c);
      g8(L.wp_lm, L.ws_lm, gl);
      gl.a_mtiles = mt; gl.a_row0 = r0;
      gl.out_f32 = logits; gl.ldo = m.vocab;
      gl.sumsq_in = sumsq + (int64_t)r0 * n_part_cur; gl.n_part = n_part_cur;
      gl.inv_d = 1.0f / d; gl.eps = m.rms_eps;
      if (eb) { gl.eb_part = eb->part; gl.eb_arg = eb->arg; gl.eb_chunks = eb->chunks; gl.eb_mask_id = eb->mask_id; }
      SBD_LAUNCH(c, SBD_KERNEL_LM_HEAD, launch_gemm(lm_epi, gl, ex));
    }
  }
  return SBD_OK;
}

bool seq_ok(const sbd_ctx* c, int32_t seq) { return seq >= 0 && seq < c->cfg.max_batch; }

}  // namespace

extern "C" {

sbd_status sbd_workspace_bytes(const sbd_model_config* cfg, size_t* bytes) {
  if (!cfg || !bytes) return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  if (const char* why = check_config(*cfg)) return fail(nullptr, SBD_ERR_UNSUPPORTED, "%s", why);
  Layout L;
  compute_layout(*cfg, &L);
  *bytes = L.total;
  return SBD_OK;
}

sbd_status sbd_workspace_region(const sbd_model_config* cfg, const char* name, size_t* offset,
                                size_t* bytes) {
  if (!cfg || !name || !offset || !bytes) return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  if (const char* why = check_config(*cfg)) return fail(nullptr, SBD_ERR_UNSUPPORTED, "%s", why);
  Layout L;
  compute_layout(*cfg, &L);
  const int64_t qd = (int64_t)cfg->n_q_heads * cfg->head_dim;
  struct R { const char* n; size_t off, sz; } regions[] = {
      {"x", L.x, (size_t)(L.m_max * cfg->d_model * 4)},
      {"qkv", L.qkv, (size_t)(L.m_max * L.n_qkv * 4)},
      {"q", L.q, (size_t)(2 * L.m_max * qd * 2)},
      {"attn", L.attn, (size_t)(2 * L.m_max * qd * 2)},
      {"act", L.act, (size_t)(2 * L.m_max * cfg->ffn_dim * 2)},
      {"xn", L.xn, (size_t)(2 * L.m_max * cfg->d_model * 2)},
  };
  for (const R& r : regions)
    if (std::strcmp(r.n, name) == 0) {
      *offset = r.off;
      *bytes = r.sz;
      return SBD_OK;
    }
  return fail(nullptr, SBD_ERR_INVALID_ARG, "unknown region '%s'", name);
}

sbd_status sbd_create(const sbd_model_config* cfg, const sbd_weights* w, void* workspace,
                      size_t workspace_bytes, void* stream, sbd_ctx** out) {
  if (!cfg || !w || !out) return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  if (const char* why = check_config(*cfg)) return fail(nullptr, SBD_ERR_UNSUPPORTED, "%s", why);
  Layout L;
  compute_layout(*cfg, &L);
  if (!workspace) return fail(nullptr, SBD_ERR_INVALID_ARG, "workspace is null");
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (workspace_bytes < L.total)
    return fail(nullptr, SBD_ERR_OUT_OF_MEMORY, "workspace has %zu bytes, needs %zu", workspace_bytes, L.total);
  if (!w->embed || !w->lm_head || !w->final_norm || !w->attn_norm || !w->wq || !w->wk || !w->wv ||
      !w->wo || !w->mlp_norm || !w->w_gate || !w->w_up || !w->w_down)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "a weight pointer is null");
  if (cfg->qk_norm && (!w->q_norm || !w->k_norm))
    return fail(nullptr, SBD_ERR_INVALID_ARG, "qk_norm needs q_norm and k_norm");
  if (cfg->weight_format == SBD_WEIGHTS_FP8_E4M3) {
    if (!w->fp8_scale_exp) return fail(nullptr, SBD_ERR_INVALID_ARG, "fp8 weights need fp8_scale_exp");
    for (int64_t i = 0; i < (int64_t)cfg->n_layers * 7 + 1; ++i)
      if (w->fp8_scale_exp[i] < -100 || w->fp8_scale_exp[i] > 100)
        return fail(nullptr, SBD_ERR_INVALID_ARG, "fp8_scale_exp[%lld] = %d out of [-100, 100]", (long long)i,
                    w->fp8_scale_exp[i]);
  }
  for (int l = 0; l < cfg->n_layers; ++l) {
    if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] || !w->mlp_norm[l] ||
        !w->w_gate[l] || !w->w_up[l] || !w->w_down[l] ||
        (cfg->qk_norm && (!w->q_norm[l] || !w->k_norm[l])))
      return fail(nullptr, SBD_ERR_INVALID_ARG, "a weight pointer of layer %d is null", l);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(nullptr, SBD_ERR_HIP, "earlier HIP error: %s", hipGetErrorString(e));

  sbd_ctx* c = new sbd_ctx();
  c->cfg = *cfg;
  c->lay = L;
  c->ws = static_cast<char*>(workspace);
  c->stream = static_cast<hipStream_t>(stream);
  c->embed = static_cast<const bf16_t*>(w->embed);
  c->lm_head = static_cast<const bf16_t*>(w->lm_head);
  c->final_norm = static_cast<const bf16_t*>(w->final_norm);
  c->layers.resize(cfg->n_layers);
  for (int l = 0; l < cfg->n_layers; ++l) {
    LayerW& lw = c->layers[l];
    lw.attn_norm = static_cast<const bf16_t*>(w->attn_norm[l]);
    lw.wq = static_cast<const bf16_t*>(w->wq[l]);
    lw.wk = static_cast<const bf16_t*>(w->wk[l]);
    lw.wv = static_cast<const bf16_t*>(w->wv[l]);
    lw.wo = static_cast<const bf16_t*>(w->wo[l]);
    lw.q_norm = cfg->qk_norm ? static_cast<const bf16_t*>(w->q_norm[l]) : nullptr;
    lw.k_norm = cfg->qk_norm ? static_cast<const bf16_t*>(w->k_norm[l]) : nullptr;
    lw.mlp_norm = static_cast<const bf16_t*>(w->mlp_norm[l]);
    lw.w_gate = static_cast<const bf16_t*>(w->w_gate[l]);
    lw.w_up = static_cast<const bf16_t*>(w->w_up[l]);
    lw.w_down = static_cast<const bf16_t*>(w->w_down[l]);
  }
  c->cache_len.assign(cfg->max_batch, 0);
  c->staged.assign(cfg->max_batch, 0);
  c->stage_bytes = std::max<size_t>(L.m_max * sizeof(RowParam),
                                    std::max<size_t>((size_t)cfg->max_batch * sizeof(SeqParam),
                                                     (size_t)cfg->max_batch * cfg->max_block));
  auto cleanup = [&](sbd_status st) {
    for (int i = 0; i < sbd_ctx::kRing; ++i) {
      if (c->stage[i]) (void)hipHostFree(c->stage[i]);
      if (c->ev[i]) (void)hipEventDestroy(c->ev[i]);
    }
    g_err = c->err;
    delete c;
    return st;
  };
  for (int i = 0; i < sbd_ctx::kRing; ++i) {
    if (hipHostMalloc(&c->stage[i], c->stage_bytes, hipHostMallocDefault) != hipSuccess) {
      c->stage[i] = nullptr;
      c->err = "hipHostMalloc of the staging buffer failed";
      return cleanup(SBD_ERR_HIP);
    }
    if (hipEventCreateWithFlags(&c->ev[i], hipEventDisableTiming) != hipSuccess) {
      c->ev[i] = nullptr;
      c->err = "hipEventCreate failed";
      return cleanup(SBD_ERR_HIP);
    }
  }
  // Zero the KV cache once so never-written slots hold finite values; build the RoPE
  // table; repack every weight matrix into the GEMM's fragment order.
  const size_t kv_bytes = L.rope - L.kcache;
  bool ok = hipMemsetAsync(c->ws + L.kcache, 0, kv_bytes, c->stream) == hipSuccess &&
            hipMemsetAsync(c->ws + L.counters, 0, (size_t)kCounters * sizeof(int32_t), c->stream) ==
                hipSuccess &&
            launch_rope_table(c->at<float>(L.rope), L.cap, cfg->head_dim, (double)cfg->rope_theta,
                              c->stream) == hipSuccess;
  const int d = cfg->d_model, F = cfg->ffn_dim;
  const int qd = cfg->n_q_heads * cfg->head_dim, kvd = cfg->n_kv_heads * cfg->head_dim;
  const bool f8 = cfg->weight_format == SBD_WEIGHTS_FP8_E4M3;
  // fp8: the bytes in the fp8 packing, the widened values in the bf16 packing (for forwards of
  // more than 16 rows and the fused path), and per-row scales 2^e for the widening
  auto pk = [&](const bf16_t* s0, const bf16_t* s1, int e0, int e1, int64_t off, int64_t rows, int K, int mode) {
    if (!f8) return launch_pack(s0, s1, c->at<bf16_t>(L.wpack) + off, rows, K, mode, c->stream) == hipSuccess;
    const fp8_t* q0 = reinterpret_cast<const fp8_t*>(s0);
    const fp8_t* q1 = reinterpret_cast<const fp8_t*>(s1);
    return launch_pack_fp8(q0, q1, c->at<fp8_t>(L.wpack8) + off, rows, K, mode, c->stream) == hipSuccess &&
           launch_pack_fp8_widen(q0, q1, e0, e1, c->at<bf16_t>(L.wpack) + off, rows, K, mode, c->stream) ==
               hipSuccess;
  };
  std::vector<float> wscale;
  auto ex = [&](int l, int j) { return f8 ? w->fp8_scale_exp[(int64_t)l * 7 + j] : 0; };
  for (int l = 0; ok && l < cfg->n_layers; ++l) {
    const LayerW& lw = c->layers[l];
    const int64_t wp = (int64_t)l * L.wp_layer;
    ok = pk(lw.wq, nullptr, ex(l, 0), 0, wp, qd, d, 0) &&
         pk(lw.wk, nullptr, ex(l, 1), 0, wp + (int64_t)qd * d, kvd, d, 0) &&
         pk(lw.wv, nullptr, ex(l, 2), 0, wp + (int64_t)(qd + kvd) * d, kvd, d, 0) &&
         pk(lw.wo, nullptr, ex(l, 3), 0, wp + L.wp_o, d, qd, 0) &&
         pk(lw.w_gate, lw.w_up, ex(l, 4), ex(l, 5), wp + L.wp_gu, 2 * (int64_t)F, d, 1) &&
         pk(lw.w_down, nullptr, ex(l, 6), 0, wp + L.wp_down, d, F, 0);
    if (f8) {
      auto put = [&](int64_t rows, int e) { wscale.insert(wscale.end(), (size_t)rows, std::ldexp(1.0f, e)); };
      put(qd, ex(l, 0));
      put(kvd, ex(l, 1));
      put(kvd, ex(l, 2));
      put(d, ex(l, 3));
      for (int64_t t = 0; t < 2 * (int64_t)F / 16; ++t) {  // packed gate/up tile: 8 gate rows, then 8 up rows
        put(8, ex(l, 4));
        put(8, ex(l, 5));
      }
      put(d, ex(l, 6));
    }
  }
  const int e_lm = f8 ? w->fp8_scale_exp[(int64_t)cfg->n_layers * 7] : 0;
  ok = ok && pk(c->lm_head, nullptr, e_lm, 0, L.wp_lm, cfg->vocab, d, 0);
  if (ok && f8) {
    wscale.insert(wscale.end(), (size_t)cfg->vocab, std::ldexp(1.0f, e_lm));
    ok = (int64_t)wscale.size() == L.ws_lm + cfg->vocab &&
         hipMemcpy(c->ws + L.wscale, wscale.data(), wscale.size() * sizeof(float), hipMemcpyHostToDevice) == hipSuccess;
  }
  // fused decode forward: per-layer gains, error word (sticky) and its pinned host copy
  if (ok) {
    std::vector<FwdGains> gains(cfg->n_layers);
    for (int l = 0; l < cfg->n_layers; ++l)
      gains[l] = FwdGains{c->layers[l].attn_norm, c->layers[l].mlp_norm, c->layers[l].q_norm, c->layers[l].k_norm};
    ok = hipMemcpy(c->ws + L.fwd_gains, gains.data(), gains.size() * sizeof(FwdGains), hipMemcpyHostToDevice) ==
             hipSuccess &&
         hipMemsetAsync(c->ws + L.fwd_err, 0, 2 * sizeof(int32_t), c->stream) == hipSuccess &&
         hipHostMalloc((void**)&c->err_host, 2 * sizeof(int32_t), hipHostMallocDefault) == hipSuccess;
    if (ok) c->err_host[0] = c->err_host[1] = 0;
    else c->err_host = nullptr;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      c->n_cu = 0;
    c->n_cu_dev = c->n_cu;
    c->n_cu = std::min(c->n_cu, kFwdMaxWorkgroups);
    // which XCD each workgroup runs on, for grids of the layer kernels' size, of a split
    // GEMM's and the largest probed; the scratch is the attention partials' region, unused yet
    c->xcd_ok = c->n_cu_dev == kXcds * kXcdWgs &&
                (int64_t)kMaxSplits * L.m_max * cfg->n_q_heads * cfg->head_dim >= kXcdProbeMax;
    int* probe = c->at<int>(L.attn_o);
    std::vector<int32_t> ids(kXcdProbeMax);
    for (int n : {kXcds * kXcdWgs, 1000, kXcdProbeMax}) {
      if (!c->xcd_ok) break;
      int32_t good = 0;
      c->xcd_ok = launch_xcd_probe(probe, n, c->stream) == hipSuccess &&
                  hipMemcpyAsync(ids.data(), probe, (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost, c->stream) ==
                      hipSuccess &&
                  hipStreamSynchronize(c->stream) == hipSuccess &&
                  sbd_xcd_map_check(ids.data(), n, kXcds, &good) == SBD_OK && good == 1;
    }
    (void)hipGetLastError();
  }
  if (!ok) {
    c->err = "initialising the workspace failed";
    return cleanup(SBD_ERR_HIP);
  }
  *out = c;
  return SBD_OK;
}

sbd_status sbd_destroy(sbd_ctx* c) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  (void)hipStreamSynchronize(c->stream);
  for (auto& r : c->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
  for (int i = 0; i < sbd_ctx::kRing; ++i) {
    if (c->stage[i]) (void)hipHostFree(c->stage[i]);
    if (c->ev[i]) (void)hipEventDestroy(c->ev[i]);
  }
  if (c->err_host) (void)hipHostFree(c->err_host);
  delete c;
  return SBD_OK;
}

sbd_status sbd_set_stream(sbd_ctx* c, void* stream) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  c->stream = static_cast<hipStream_t>(stream);
  return SBD_OK;
}

sbd_status sbd_reset(sbd_ctx* c, int32_t seq) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  if (!seq_ok(c, seq)) return fail(c, SBD_ERR_INVALID_ARG, "seq %d out of range", seq);
  c->cache_len[seq] = 0;
  c->staged[seq] = 0;
  return SBD_OK;
}

sbd_status sbd_cache_len(const sbd_ctx* c, int32_t seq, int32_t* len) {
  if (!c || !len) return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  if (!seq_ok(c, seq)) return fail(const_cast<sbd_ctx*>(c), SBD_ERR_INVALID_ARG, "seq %d out of range", seq);
  *len = c->cache_len[seq];
  return SBD_OK;
}

sbd_status sbd_prefill(sbd_ctx* c, int32_t seq, const int32_t* tokens, int32_t n, float* last_logits) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  if (!seq_ok(c, seq)) return fail(c, SBD_ERR_INVALID_ARG, "seq %d out of range", seq);
  if (!tokens || n < 1) return fail(c, SBD_ERR_INVALID_ARG, "need n >= 1 tokens");
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= c->cfg.vocab || tokens[i] == c->cfg.mask_id)
      return fail(c, SBD_ERR_INVALID_ARG, "prompt token %d (=%d) out of range or the mask id", i, tokens[i]);
  if ((int64_t)c->cache_len[seq] + n > c->cfg.max_seq_len)
    return fail(c, SBD_ERR_CAPACITY, "cache_len %d + %d exceeds max_seq_len %d", c->cache_len[seq], n,
                c->cfg.max_seq_len);
  if (sbd_status st = check_sticky(c)) return st;
  const int chunk = effective_chunk(c->cfg);
  for (int off = 0; off < n; off += chunk) {
    const int kk = std::min(chunk, n - off);
    std::vector<RowParam> rows(kk);
    for (int j = 0; j < kk; ++j) rows[j] = RowParam{tokens[off + j], c->cache_len[seq] + j};
    std::vector<SeqParam> seqs{SeqParam{seq, c->cache_len[seq], kk, 0}};
    const bool last = off + kk == n;
    sbd_status st = run_forward(c, 1, kk, rows, seqs, last ? last_logits : nullptr, kk - 1);
    if (st) return st;
    c->cache_len[seq] += kk;
  }
  c->staged[seq] = 0;
  return SBD_OK;
}

}  // extern "C"

namespace {

// Validation of a block forward's arguments and state (nothing is changed or enqueued), and
// its per-row and per-sequence parameters.
sbd_status prepare_block(sbd_ctx* c, int32_t batch, const int32_t* seq_ids, int32_t k, const int32_t* tokens,
                         const uint8_t* is_mask, const int32_t* n_causal, const int32_t* pos_ids,
                         std::vector<RowParam>* rows, std::vector<SeqParam>* seqs) {
  const sbd_model_config& m = c->cfg;
  if (batch < 1 || batch > m.max_batch) return fail(c, SBD_ERR_INVALID_ARG, "batch %d out of [1, %d]", batch, m.max_batch);
  if (k < 1 || k > m.max_block) return fail(c, SBD_ERR_INVALID_ARG, "k %d out of [1, %d]", k, m.max_block);
  if (!seq_ids || !tokens) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  std::vector<char> seen(m.max_batch, 0);
  for (int b = 0; b < batch; ++b) {
    const int s = seq_ids[b];
    if (!seq_ok(c, s)) return fail(c, SBD_ERR_INVALID_ARG, "seq_ids[%d] = %d out of range", b, s);
    if (seen[s]) return fail(c, SBD_ERR_INVALID_ARG, "seq id %d appears twice", s);
    seen[s] = 1;
    const int nc = n_causal ? n_causal[b] : 1;
    if (nc < 0 || nc > k) return fail(c, SBD_ERR_INVALID_ARG, "n_causal[%d] = %d out of [0, k]", b, nc);
    const int Lb = c->cache_len[s];
    if ((int64_t)Lb + k > m.max_seq_len)
      return fail(c, SBD_ERR_CAPACITY, "seq %d: cache_len %d + k %d exceeds max_seq_len %d", s, Lb, k, m.max_seq_len);
    for (int j = 0; j < k; ++j) {
      const int t = tokens[b * k + j];
      if (t < 0 || t >= m.vocab) return fail(c, SBD_ERR_INVALID_ARG, "token[%d][%d] = %d out of range", b, j, t);
      if (is_mask && (is_mask[b * k + j] != 0) != (t == m.mask_id))
        return fail(c, SBD_ERR_INVALID_ARG, "is_mask[%d][%d] disagrees with the token", b, j);
      if (j < nc && t == m.mask_id) return fail(c, SBD_ERR_INVALID_ARG, "causal row %d of batch %d is a mask", j, b);
      if (pos_ids) {
        const int p = pos_ids[b * k + j];
        if (p < 0 || p >= m.max_seq_len) return fail(c, SBD_ERR_INVALID_ARG, "pos_ids[%d][%d] = %d out of range", b, j, p);
        if (j < nc && p != Lb + j)
          return fail(c, SBD_ERR_INVALID_ARG, "causal row %d of batch %d must have position %d", j, b, Lb + j);
      }
    }
  }
  rows->resize((size_t)batch * k);
  seqs->resize(batch);
  for (int b = 0; b < batch; ++b) {
    const int s = seq_ids[b];
    (*seqs)[b] = SeqParam{s, c->cache_len[s], n_causal ? n_causal[b] : 1, 0};
    for (int j = 0; j < k; ++j)
      (*rows)[b * k + j] = RowParam{tokens[b * k + j], pos_ids ? pos_ids[b * k + j] : c->cache_len[s] + j};
  }
  return SBD_OK;
}

// The masks of an EB selection into the kernel arguments (by value up to kEbInlineRows rows,
// else uploaded into the workspace).
sbd_status eb_masks(sbd_ctx* c, EbArgs* a, const uint8_t* is_mask, int64_t rows) {
  if (rows <= kEbInlineRows) {
    for (int64_t i = 0; i < rows; ++i)
      if (is_mask[i]) a->mask_bits[i >> 6] |= 1ull << (i & 63);
    return SBD_OK;
  }
  if (sbd_status st = upload(c, c->ws + c->lay.eb_mask, is_mask, (size_t)rows)) return st;
  a->is_mask = c->at<uint8_t>(c->lay.eb_mask);
  return SBD_OK;
}

}  // namespace

extern "C" {

sbd_status sbd_block_forward(sbd_ctx* c, int32_t batch, const int32_t* seq_ids, int32_t k,
                             const int32_t* tokens, const uint8_t* is_mask, const int32_t* n_causal,
                             const int32_t* pos_ids, float* logits) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  std::vector<RowParam> rows;
  std::vector<SeqParam> seqs;
  if (sbd_status st = prepare_block(c, batch, seq_ids, k, tokens, is_mask, n_causal, pos_ids, &rows, &seqs)) return st;
  if (!logits) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  if (sbd_status st = check_sticky(c)) return st;
  sbd_status st = run_forward(c, batch, k, rows, seqs, logits, -1);
  if (st) return st;
  for (int b = 0; b < batch; ++b) c->staged[seq_ids[b]] = seqs[b].n_causal;
  return SBD_OK;
}

sbd_status sbd_block_step(sbd_ctx* c, int32_t rule, int32_t batch, const int32_t* seq_ids, int32_t k,
                          const int32_t* tokens, const uint8_t* is_mask, const int32_t* n_causal,
                          const int32_t* pos_ids, double threshold, float* logits, int32_t* n_accepted,
                          int32_t* accepted_pos, int32_t* accepted_tok, double* entropy, double* confidence) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  std::vector<RowParam> rows;
  std::vector<SeqParam> seqs;
  if (sbd_status st = prepare_block(c, batch, seq_ids, k, tokens, is_mask, n_causal, pos_ids, &rows, &seqs)) return st;
  if (rule != SBD_SELECT_EB_ENTROPY && rule != SBD_SELECT_EB_CONFIDENCE && rule != SBD_SELECT_FACTOR)
    return fail(c, SBD_ERR_INVALID_ARG, "unknown selection rule %d", rule);
  if (std::isnan(threshold) || threshold < 0.0)
    return fail(c, SBD_ERR_INVALID_ARG, "threshold must be >= 0 (got %g)", threshold);
  if (!n_accepted || !accepted_pos || !accepted_tok) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  const sbd_model_config& m = c->cfg;
  const int64_t M = (int64_t)batch * k;
  if (M > c->lay.eb_frows)
    return fail(c, SBD_ERR_INVALID_ARG, "batch * k = %lld exceeds the %lld rows of one block step", (long long)M,
                (long long)c->lay.eb_frows);
  if (c->lay.eb_fchunks > 4096)
    return fail(c, SBD_ERR_UNSUPPORTED, "the block step merges at most 4096 chunks of 64 columns (vocab <= 262144)");
  // the fused decode forward has its own LM head: its statistics come from stored logits
  const bool stored = M <= 16 && c->decode_path == SBD_DECODE_FUSED;
  if (stored && !logits)
    return fail(c, SBD_ERR_UNSUPPORTED, "the fused decode path takes its statistics from stored logits: pass logits");
  if (sbd_status st = check_sticky(c)) return st;
  std::vector<uint8_t> msk((size_t)M);
  for (int64_t i = 0; i < M; ++i) msk[i] = is_mask ? (is_mask[i] != 0) : (tokens[i] == m.mask_id);
  LmEb eb{c->at<double>(c->lay.eb_fpart), c->at<int32_t>(c->lay.eb_farg), (int)c->lay.eb_fchunks, m.mask_id};
  sbd_status st = run_forward(c, batch, k, rows, seqs, logits, -1, stored ? nullptr : &eb);
  if (st) return st;
  for (int b = 0; b < batch; ++b) c->staged[seq_ids[b]] = seqs[b].n_causal;
  EbArgs a{};
  if ((st = eb_masks(c, &a, msk.data(), M))) return st;
  a.B = batch; a.k = k; a.vocab = m.vocab; a.mask_id = m.mask_id; a.logits = logits; a.gamma = threshold;
  a.n_accepted = n_accepted; a.accepted_pos = accepted_pos; a.accepted_tok = accepted_tok;
  a.entropy_out = entropy; a.rule = rule; a.conf_out = confidence;
  if (stored) {
    a.n_chunks = (m.vocab + kEbChunk - 1) / kEbChunk;
    a.part = c->at<double>(c->lay.eb_part); a.part_arg = c->at<int32_t>(c->lay.eb_arg);
    SBD_LAUNCH(c, SBD_KERNEL_EB_PARTIAL, launch_eb_partial(a, ex));
  } else {
    a.n_chunks = (int)c->lay.eb_fchunks;
    a.part = eb.part; a.part_arg = eb.arg;
    a.row_stats = c->at<double>(c->lay.eb_rowstat); a.row_tok = c->at<int32_t>(c->lay.eb_rowtok);
    SBD_LAUNCH(c, SBD_KERNEL_EB_PARTIAL, launch_eb_merge(a, ex));
  }
  SBD_LAUNCH(c, SBD_KERNEL_EB_SELECT, launch_eb_select(a, false, ex));
  return SBD_OK;
}

sbd_status sbd_commit(sbd_ctx* c, int32_t batch, const int32_t* seq_ids, const int32_t* n_commit) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  if (batch < 1 || batch > c->cfg.max_batch || !seq_ids || !n_commit)
    return fail(c, SBD_ERR_INVALID_ARG, "bad batch or null argument");
  std::vector<char> seen(c->cfg.max_batch, 0);
  for (int b = 0; b < batch; ++b) {
    const int s = seq_ids[b];
    if (!seq_ok(c, s)) return fail(c, SBD_ERR_INVALID_ARG, "seq_ids[%d] = %d out of range", b, s);
    if (seen[s]) return fail(c, SBD_ERR_INVALID_ARG, "seq id %d appears twice", s);
    seen[s] = 1;
    if (n_commit[b] < 0) return fail(c, SBD_ERR_INVALID_ARG, "n_commit[%d] < 0", b);
    if (n_commit[b] > c->staged[s])
      return fail(c, SBD_ERR_STATE, "seq %d: commit of %d rows but only %d causal rows are staged", s,
                  n_commit[b], c->staged[s]);
  }
  for (int b = 0; b < batch; ++b) {
    c->cache_len[seq_ids[b]] += n_commit[b];
    c->staged[seq_ids[b]] = 0;
  }
  return SBD_OK;
}

static sbd_status eb_common(sbd_ctx* c, int32_t batch, int32_t k, const uint8_t* is_mask, double gamma,
                            int32_t* n_accepted, int32_t* accepted_pos) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  if (batch < 1 || batch > c->cfg.max_batch) return fail(c, SBD_ERR_INVALID_ARG, "batch %d out of range", batch);
  if (k < 1 || k > c->cfg.max_block) return fail(c, SBD_ERR_INVALID_ARG, "k %d out of range", k);
  if (!is_mask || !n_accepted || !accepted_pos) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  if (std::isnan(gamma) || gamma < 0.0) return fail(c, SBD_ERR_INVALID_ARG, "gamma must be >= 0 (got %g)", gamma);
  return SBD_OK;
}

sbd_status sbd_eb_select(sbd_ctx* c, int32_t batch, int32_t k, int32_t vocab, const float* logits,
                         const uint8_t* is_mask, double gamma, int32_t mask_id, int32_t* n_accepted,
                         int32_t* accepted_pos, int32_t* accepted_tok, double* entropy) {
  return sbd_select(c, SBD_SELECT_EB_ENTROPY, batch, k, vocab, logits, is_mask, gamma, mask_id, n_accepted,
                    accepted_pos, accepted_tok, entropy, nullptr);
}

sbd_status sbd_select(sbd_ctx* c, int32_t rule, int32_t batch, int32_t k, int32_t vocab, const float* logits,
                      const uint8_t* is_mask, double gamma, int32_t mask_id, int32_t* n_accepted,
                      int32_t* accepted_pos, int32_t* accepted_tok, double* entropy, double* confidence) {
  if (sbd_status st = eb_common(c, batch, k, is_mask, gamma, n_accepted, accepted_pos)) return st;
  if (rule != SBD_SELECT_EB_ENTROPY && rule != SBD_SELECT_EB_CONFIDENCE && rule != SBD_SELECT_FACTOR)
    return fail(c, SBD_ERR_INVALID_ARG, "unknown selection rule %d", rule);
  if (!logits || !accepted_tok) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  if (vocab < 1 || vocab > c->cfg.vocab) return fail(c, SBD_ERR_INVALID_ARG, "vocab %d out of [1, %d]", vocab, c->cfg.vocab);
  if (mask_id < -1 || mask_id >= vocab) return fail(c, SBD_ERR_INVALID_ARG, "mask_id %d out of [-1, vocab)", mask_id);
  if (sbd_status st = check_sticky(c)) return st;
  EbArgs a{};
  // masks by value where they fit: no copy on the stream ahead of the kernels
  if (sbd_status st = eb_masks(c, &a, is_mask, (int64_t)batch * k)) return st;
  a.B = batch; a.k = k; a.vocab = vocab; a.mask_id = mask_id; a.logits = logits;
  a.gamma = gamma;
  a.n_chunks = (vocab + kEbChunk - 1) / kEbChunk;
  a.part = c->at<double>(c->lay.eb_part); a.part_arg = c->at<int32_t>(c->lay.eb_arg);
  a.n_accepted = n_accepted; a.accepted_pos = accepted_pos; a.accepted_tok = accepted_tok;
  a.entropy_out = entropy; a.rule = rule; a.conf_out = confidence;
  SBD_LAUNCH(c, SBD_KERNEL_EB_PARTIAL, launch_eb_partial(a, ex));
  SBD_LAUNCH(c, SBD_KERNEL_EB_SELECT, launch_eb_select(a, false, ex));
  return SBD_OK;
}

sbd_status sbd_eb_select_noalloc(void* stream, int32_t batch, int32_t k, int32_t vocab, const float* logits,
                                 const uint8_t* is_mask, double gamma, int32_t mask_id, int32_t* n_accepted,
                                 int32_t* accepted_pos, int32_t* accepted_tok, double* entropy) {
  if (batch < 1 || k < 1 || k > kMaxBlock)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "batch %d or k %d out of range (k <= %d)", batch, k, kMaxBlock);
  if ((int64_t)batch * k > kNoAllocRows)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "batch * k = %lld exceeds the %d rows of the static scratch",
                (long long)batch * k, kNoAllocRows);
  if (vocab < 1 || vocab > kNoAllocChunks * kEbChunk)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "vocab %d out of [1, %d] (the static scratch's limit)", vocab,
                kNoAllocChunks * kEbChunk);
  if (!logits || !is_mask || !n_accepted || !accepted_pos || !accepted_tok)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  if (mask_id < -1 || mask_id >= vocab) return fail(nullptr, SBD_ERR_INVALID_ARG, "mask_id %d out of [-1, vocab)", mask_id);
  if (std::isnan(gamma) || gamma < 0.0) return fail(nullptr, SBD_ERR_INVALID_ARG, "gamma must be >= 0 (got %g)", gamma);
  EbArgs a{};
  hipError_t e = eb_noalloc_scratch(&a.part, &a.part_arg);
  if (e != hipSuccess)
    return fail(nullptr, SBD_ERR_HIP, "device address of the static scratch: %s", hipGetErrorString(e));
  const int64_t rows = (int64_t)batch * k;  // <= kNoAllocRows <= kEbInlineRows: masks by value
  for (int64_t i = 0; i < rows; ++i)
    if (is_mask[i]) a.mask_bits[i >> 6] |= 1ull << (i & 63);
  a.B = batch; a.k = k; a.vocab = vocab; a.mask_id = mask_id; a.logits = logits; a.gamma = gamma;
  a.n_chunks = (vocab + kEbChunk - 1) / kEbChunk;
  a.n_accepted = n_accepted; a.accepted_pos = accepted_pos; a.accepted_tok = accepted_tok;
  a.entropy_out = entropy; a.rule = SBD_SELECT_EB_ENTROPY;
  const Exec ex{static_cast<hipStream_t>(stream), nullptr, nullptr};
  if ((e = launch_eb_partial(a, ex)) != hipSuccess || (e = launch_eb_select(a, false, ex)) != hipSuccess)
    return fail(nullptr, SBD_ERR_HIP, "EB launch failed: %s", hipGetErrorString(e));
  return SBD_OK;
}

sbd_status sbd_stream_probe(void* stream, const void* buf, size_t bytes, uint32_t* sink) {
  if (!buf || !sink || bytes < 16 || bytes % 16)
    return fail(nullptr, SBD_ERR_INVALID_ARG, "need a buffer of a positive multiple of 16 bytes and a sink");
  int dev = 0, n_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = launch_stream_probe(buf, (int64_t)bytes, sink, n_cu, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(nullptr, SBD_ERR_HIP, "stream probe: %s", hipGetErrorString(e));
  return SBD_OK;
}

sbd_status sbd_eb_select_entropies(sbd_ctx* c, int32_t batch, int32_t k, const double* entropy,
                                   const uint8_t* is_mask, double gamma, int32_t* n_accepted,
                                   int32_t* accepted_pos) {
  if (sbd_status st = eb_common(c, batch, k, is_mask, gamma, n_accepted, accepted_pos)) return st;
  if (!entropy) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  if (sbd_status st = check_sticky(c)) return st;
  if (sbd_status st = upload(c, c->ws + c->lay.eb_mask, is_mask, (size_t)batch * k)) return st;
  EbArgs a{};
  a.B = batch; a.k = k; a.is_mask = c->at<uint8_t>(c->lay.eb_mask); a.entropy_in = entropy;
  a.gamma = gamma; a.n_accepted = n_accepted; a.accepted_pos = accepted_pos;
  SBD_LAUNCH(c, SBD_KERNEL_EB_SELECT, launch_eb_select(a, true, ex));
  return SBD_OK;
}

static sbd_status kv_common(sbd_ctx* c, int32_t seq, int32_t pos0, int32_t n, const void* kp, const void* vp,
                            bool import) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  if (!seq_ok(c, seq)) return fail(c, SBD_ERR_INVALID_ARG, "seq %d out of range", seq);
  if (!kp || !vp || n < 1 || pos0 < 0) return fail(c, SBD_ERR_INVALID_ARG, "bad pointer, n or pos0");
  if ((int64_t)pos0 + n > c->cfg.max_seq_len)
    return fail(c, SBD_ERR_CAPACITY, "pos0 %d + n %d exceeds max_seq_len %d", pos0, n, c->cfg.max_seq_len);
  if (import && pos0 > c->cache_len[seq])
    return fail(c, SBD_ERR_INVALID_ARG, "pos0 %d beyond cache_len %d", pos0, c->cache_len[seq]);
  return check_sticky(c);
}

static KvCopyArgs kv_copy_base(sbd_ctx* c, int32_t seq, int32_t pos0, int32_t n) {
  const KvFmt kvf = kv_fmt(c->cfg);
  KvCopyArgs a{};
  a.kcache = c->ws + c->lay.kcache; a.vcache = c->ws + c->lay.vcache; a.cap = c->lay.cap;
  a.kv_fp8 = kvf.fp8; a.kv_scale = kvf.scale; a.kv_inv = kvf.inv;
  a.n_layers = c->cfg.n_layers; a.n_slots = c->cfg.max_batch; a.n_kv = c->cfg.n_kv_heads;
  a.d_h = c->cfg.head_dim; a.slot = seq; a.pos0 = pos0; a.n = n;
  return a;
}

sbd_status sbd_kv_import(sbd_ctx* c, int32_t seq, int32_t pos0, int32_t n, const void* k, const void* v) {
  if (sbd_status st = kv_common(c, seq, pos0, n, k, v, true)) return st;
  KvCopyArgs a = kv_copy_base(c, seq, pos0, n);
  a.k_in = static_cast<const bf16_t*>(k); a.v_in = static_cast<const bf16_t*>(v);
  SBD_HIP(c, launch_kv_import(a, c->stream));
  c->cache_len[seq] = pos0 + n;
  c->staged[seq] = 0;
  return SBD_OK;
}

sbd_status sbd_kv_export(sbd_ctx* c, int32_t seq, int32_t pos0, int32_t n, void* k, void* v) {
  if (sbd_status st = kv_common(c, seq, pos0, n, k, v, false)) return st;
  KvCopyArgs a = kv_copy_base(c, seq, pos0, n);
  a.k_out = static_cast<bf16_t*>(k); a.v_out = static_cast<bf16_t*>(v);
  SBD_HIP(c, launch_kv_export(a, c->stream));
  return SBD_OK;
}

sbd_status sbd_set_decode_path(sbd_ctx* c, int32_t path) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  if (path != SBD_DECODE_AUTO && path != SBD_DECODE_FUSED && path != SBD_DECODE_KERNELS &&
      path != SBD_DECODE_LAYERS)
    return fail(c, SBD_ERR_INVALID_ARG, "unknown decode path %d", path);
  c->decode_path = path;
  return SBD_OK;
}

sbd_status sbd_set_wait_limit(sbd_ctx* c, int32_t polls) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  c->wait_limit = polls < 0 ? kLxSpinDefault : polls;
  return SBD_OK;
}

sbd_status sbd_decode_path_fits(const sbd_ctx* c, int32_t path, int32_t batch, int32_t k, int32_t* fits) {
  if (!c || !fits) return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  switch (path) {
    case SBD_DECODE_AUTO:
    case SBD_DECODE_KERNELS: *fits = 1; return SBD_OK;
    case SBD_DECODE_FUSED: {
      const sbd_model_config& m = c->cfg;
      *fits = c->n_cu >= 1 && m.d_model % 128 == 0 && (m.head_dim == 64 || m.head_dim == 128) &&
              m.kv_format == SBD_KV_BF16 ? 1 : 0;
      return SBD_OK;
    }
    case SBD_DECODE_LAYERS: *fits = c->xcd_ok && layer_xcd_fits(c->cfg, c->n_cu_dev, batch, k) ? 1 : 0; return SBD_OK;
    default: return fail(nullptr, SBD_ERR_INVALID_ARG, "unknown decode path %d", path);
  }
}

sbd_status sbd_xcd_map_check(const int32_t* xcc_ids, int32_t n, int32_t n_xcd, int32_t* ok) {
  if (!xcc_ids || !ok || n < 1 || n_xcd < 1) return fail(nullptr, SBD_ERR_INVALID_ARG, "bad argument");
  *ok = 1;
  for (int32_t i = 0; i < n; ++i)
    if (xcc_ids[i] != i % n_xcd) {
      *ok = 0;
      break;
    }
  return SBD_OK;
}

sbd_status sbd_xcd_map_ok(const sbd_ctx* c, int32_t* ok) {
  if (!c || !ok) return fail(nullptr, SBD_ERR_INVALID_ARG, "null argument");
  *ok = c->xcd_ok ? 1 : 0;
  return SBD_OK;
}

sbd_status sbd_profile_enable(sbd_ctx* c, int32_t enable) {
  if (!c) return fail(nullptr, SBD_ERR_INVALID_ARG, "null context");
  c->prof = enable != 0;
  return SBD_OK;
}

sbd_status sbd_profile_read(sbd_ctx* c, int32_t kernel, int32_t* launches, double* total_ms) {
  if (!c || !launches || !total_ms) return fail(c, SBD_ERR_INVALID_ARG, "null argument");
  if (kernel < 0 || kernel >= SBD_KERNEL_COUNT) return fail(c, SBD_ERR_INVALID_ARG, "kernel %d out of range", kernel);
  if (!c->recs.empty()) {
    SBD_HIP(c, hipEventSynchronize(c->recs.back().b));
    for (auto& r : c->recs) {
      float ms = 0.f;
      SBD_HIP(c, hipEventElapsedTime(&ms, r.a, r.b));
      c->prof_count[r.kind] += 1;
      c->prof_ms[r.kind] += ms;
      c->pool.push_back(r.a);
      c->pool.push_back(r.b);
    }
    c->recs.clear();
  }
  *launches = c->prof_count[kernel];
  *total_ms = c->prof_ms[kernel];
  c->prof_count[kernel] = 0;
  c->prof_ms[kernel] = 0.0;
  return SBD_OK;
}

const char* sbd_status_string(sbd_status s) {
  switch (s) {
    case SBD_OK: return "ok";
    case SBD_ERR_INVALID_ARG: return "invalid argument";
    case SBD_ERR_STATE: return "invalid state";
    case SBD_ERR_CAPACITY: return "capacity exceeded";
    case SBD_ERR_OUT_OF_MEMORY: return "workspace too small";
    case SBD_ERR_HIP: return "HIP error";
    case SBD_ERR_UNSUPPORTED: return "unsupported shape";
  }
  return "unknown status";
}

const char* sbd_last_error(const sbd_ctx* c) { return c ? c->err.c_str() : g_err.c_str(); }

}  // extern "C"

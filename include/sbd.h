/*
 * sbd.h - C ABI of the MI355X (gfx950) Set Block Decoding decode step.
 *
 * One decode step of Set Block Decoding (SBD, arXiv 2509.04185) is one forward pass
 * of the SBD network f_theta over a block of k rows against an exact KV cache
 * (Sec. 2.3, eq. (hybrid_block); Alg. 3), followed by one step of the entropy-bounded
 * (EB) sampler (Sec. 2.2, eq. (eb_sampler)).  This library runs both on one GPU with
 * hand-written HIP kernels.
 *
 * Conventions shared by every entry point
 *  - Every function returns an sbd_status; no exception crosses the ABI.
 *  - Arguments and state are validated on the host before anything is enqueued; on
 *    any error nothing is enqueued and no state changes.  sbd_last_error() then gives
 *    a one-line reason.
 *  - "device" pointers are GPU global memory (e.g. torch CUDA tensors); "host"
 *    pointers are ordinary CPU memory that is read before the call returns.
 *  - All GPU work is enqueued on the context's stream and is asynchronous: outputs are
 *    valid once that stream has been synchronised.  An asynchronous device fault is
 *    reported as SBD_ERR_HIP by a later call.
 *  - Row-major layouts throughout; bf16 means IEEE bfloat16 (1/8/7 bits).
 *  - A context is used by one host thread at a time.  The library keeps no global
 *    state other than the thread-local error text of context-less calls.
 */
#ifndef SBD_H_
#define SBD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SBD_OK = 0,
  SBD_ERR_INVALID_ARG = 1,   /* a pointer, size, id or value is out of its documented range */
  SBD_ERR_STATE = 2,         /* the call is not allowed in the context's current state */
  SBD_ERR_CAPACITY = 3,      /* a sequence would exceed max_seq_len */
  SBD_ERR_OUT_OF_MEMORY = 4, /* the workspace is smaller than sbd_workspace_bytes() */
  SBD_ERR_HIP = 5,           /* a HIP runtime call or an earlier kernel failed */
  SBD_ERR_UNSUPPORTED = 6    /* the model shape is outside what the kernels implement */
} sbd_status;

typedef struct sbd_ctx sbd_ctx; /* opaque, created by sbd_create */

/* Selection rules of one sampling step (sbd_select, sbd_block_step). */
enum { SBD_SELECT_EB_ENTROPY = 0, SBD_SELECT_EB_CONFIDENCE = 1, SBD_SELECT_FACTOR = 2 };

/*
 * Decoder shape (Llama-3.1 / Qwen-3 style; the SBD network has no architectural
 * changes, Sec. 1) plus capacity limits.
 *   n_q_heads % n_kv_heads == 0; query head h reads KV head h / (n_q_heads/n_kv_heads).
 *   head_dim is 64 or 128.  d_model, n_q_heads*head_dim and ffn_dim are multiples of 256;
 *   vocab and (n_q_heads + 2 n_kv_heads) * head_dim are multiples of 128.  mask_id in
 *   [0, vocab) is the input-only mask token 'm'.
 *   qk_norm != 0 enables the per-head RMSNorm of q and k before RoPE (Qwen-3).
 *   max_batch: number of sequence slots (ids 0..max_batch-1).
 *   max_seq_len: tokens per slot, including the k rows staged by a block forward.
 *   max_block: largest k accepted by sbd_block_forward / sbd_eb_select (<= 64).
 *   prefill_chunk: rows per forward inside sbd_prefill (0 selects 256).
 */
typedef struct {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab, mask_id;
  int32_t qk_norm;
  float rms_eps, rope_theta;
  int32_t max_batch, max_seq_len, max_block, prefill_chunk;
  int32_t weight_format;  /* SBD_WEIGHTS_BF16 (0) or SBD_WEIGHTS_FP8_E4M3 (1), see sbd_weights */
  int32_t kv_format;      /* SBD_KV_BF16 (0) or SBD_KV_FP8_E4M3 (1), see below */
  int32_t kv_scale_exp;   /* SBD_KV_FP8_E4M3 only (else ignored): scale exponent e in [-100, 100] */
} sbd_model_config;

/*
 * Formats of the projection and LM-head matrices (wq, wk, wv, wo, w_gate, w_up, w_down,
 * lm_head).  The embedding and every norm gain are bf16 in both.
 *   SBD_WEIGHTS_BF16      bf16 values.
 *   SBD_WEIGHTS_FP8_E4M3  OCP e4m3 bytes (1 sign, 4 exponent bits of bias 7, 3 mantissa
 *                         bits; no infinities, 0x7f / 0xff NaN) with a power-of-two scale per
 *                         matrix: the weight is e4m3(q) * 2^e (the FP8 weights of the
 *                         paper's timing model, Sec. 4.1).  Every forward streams the bytes
 *                         and widens them to bf16 in registers (exactly), except the fused
 *                         decode path, which streams a bf16 copy of the same values made in
 *                         sbd_create.
 */
enum { SBD_WEIGHTS_BF16 = 0, SBD_WEIGHTS_FP8_E4M3 = 1 };

/*
 * Formats of the KV cache (the cache of exact KV caching, Sec. 1 and Alg. 3).
 *   SBD_KV_BF16      each cached key (after RoPE) and value is the bf16 rounding (nearest,
 *                    ties to even) of the float the forward computes.
 *   SBD_KV_FP8_E4M3  one byte per element (the 1-byte KV of the paper's timing model,
 *                    Sec. 4.1): the e4m3 code of v * 2^-e, e = kv_scale_exp, rounded to the
 *                    nearest code with ties to even and saturated at +-448 (NaN stays NaN),
 *                    read back as e4m3 * 2^e.  The rows a forward stages are rounded so
 *                    before its own attention reads them.  sbd_kv_import rounds its bf16
 *                    input the same way; sbd_kv_export returns the stored values, which
 *                    bf16 holds exactly.  The fused decode path reads bf16 caches only
 *                    (UNSUPPORTED here); the other paths read both formats.
 */
enum { SBD_KV_BF16 = 0, SBD_KV_FP8_E4M3 = 1 };

/*
 * Weights: device memory, borrowed (they must outlive the context and not change); bf16,
 * or for the projection and LM-head matrices the format of cfg->weight_format.
 * Matrices are logical [out][in] row-major.  Per-layer fields are host arrays of
 * n_layers device pointers.  q_norm / k_norm may be NULL when qk_norm == 0.
 *   embed [vocab][d_model], lm_head [vocab][d_model], final_norm [d_model]
 *   attn_norm [d_model], wq [n_q_heads*head_dim][d_model], wk, wv [n_kv_heads*head_dim][d_model],
 *   wo [d_model][n_q_heads*head_dim], q_norm, k_norm [head_dim], mlp_norm [d_model],
 *   w_gate, w_up [ffn_dim][d_model], w_down [d_model][ffn_dim]
 */
typedef struct {
  const void *embed, *lm_head, *final_norm;
  const void *const *attn_norm, *const *wq, *const *wk, *const *wv, *const *wo;
  const void *const *q_norm, *const *k_norm, *const *mlp_norm;
  const void *const *w_gate, *const *w_up, *const *w_down;
  /* SBD_WEIGHTS_FP8_E4M3 only (else ignored): host int32 [n_layers * 7 + 1], the scale
   * exponents e of wq, wk, wv, wo, w_gate, w_up, w_down of layer 0, of layer 1, ..., then
   * of lm_head; each in [-100, 100]. */
  const int32_t* fp8_scale_exp;
} sbd_weights;

/* Bytes of device workspace sbd_create needs for this config (KV cache, activations,
 * partial results, RoPE table, and a copy of every weight matrix repacked into the
 * order the GEMM kernels stream).  *bytes is set only on SBD_OK. */
sbd_status sbd_workspace_bytes(const sbd_model_config* cfg, size_t* bytes);

/*
 * Create a context on the current HIP device.  workspace: device memory of at least
 * sbd_workspace_bytes() bytes, 256-byte aligned, caller-owned, not touched by anyone
 * else while the context lives.  stream: a hipStream_t (NULL = the null stream).
 * Every sequence slot starts empty.  The weights are read here once, to repack them into
 * the workspace (the originals must still outlive the context: the embedding and norm
 * gains are read from them).  The library allocates no device memory itself; it
 * allocates a small pinned host staging buffer here.
 */
sbd_status sbd_create(const sbd_model_config* cfg, const sbd_weights* w, void* workspace,
                      size_t workspace_bytes, void* stream, sbd_ctx** out);
sbd_status sbd_destroy(sbd_ctx* ctx);
/* Replace the stream later calls enqueue on (e.g. torch's current stream). */
sbd_status sbd_set_stream(sbd_ctx* ctx, void* stream);

/* Empty one sequence slot (cache length 0, nothing staged). */
sbd_status sbd_reset(sbd_ctx* ctx, int32_t seq);
/* Number of committed tokens in a slot. */
sbd_status sbd_cache_len(const sbd_ctx* ctx, int32_t seq, int32_t* len);

/*
 * Prefill (Alg. 2, first step): a causal forward f_theta(x;) over n prompt tokens
 * (host int32 ids in [0, vocab), mask id excluded) appended after the slot's cache,
 * committing all n rows.  Runs in forwards of at most prefill_chunk rows.
 * last_logits: device fp32 [vocab] receiving the logits of the last prompt row, or NULL.
 * Errors: CAPACITY if cache_len + n > max_seq_len.
 */
sbd_status sbd_prefill(sbd_ctx* ctx, int32_t seq, const int32_t* tokens, int32_t n,
                       float* last_logits);

/*
 * Block forward (eq. (hybrid_block); one iteration of Alg. 3) for `batch` sequences.
 *   seq_ids  host [batch], distinct slot ids.
 *   tokens   host [batch][k] ids in [0, vocab); mask rows hold mask_id.
 *   is_mask  host [batch][k] or NULL; when given it must equal (tokens == mask_id).
 *   n_causal host [batch] or NULL (= all 1).  Rows j < n_causal[b] are committed but
 *            not yet cached tokens and attend causally; rows j >= n_causal[b] form the
 *            prediction block and see every row (App. A inference mask: key kv is
 *            visible to query q iff kv <= q or q >= the first prediction index).
 *            Causal rows may not be masks.
 *   pos_ids  host [batch][k] or NULL (= cache_len + j).  RoPE positions; causal rows
 *            must keep cache_len + j.  Values in [0, max_seq_len).
 *   logits   device fp32 [batch][k][vocab], all rows, all vocab columns (row j's
 *            logits predict the token at its own position, eq. (p_theta_masked)).
 * The K/V of all k rows are staged in cache slots [cache_len, cache_len + k); the
 * first n_causal of them become permanent with sbd_commit.
 * Errors: CAPACITY if cache_len + k > max_seq_len for some sequence.
 */
sbd_status sbd_block_forward(sbd_ctx* ctx, int32_t batch, const int32_t* seq_ids, int32_t k,
                             const int32_t* tokens, const uint8_t* is_mask,
                             const int32_t* n_causal, const int32_t* pos_ids, float* logits);

/*
 * One decode step in one call: sbd_block_forward followed by the selection rule `rule`
 * (SBD_SELECT_*, threshold as for sbd_select) over the masked rows, with the selection's
 * softmax statistics taken from the LM head itself (Sec. 2.2, eq. (eb_sampler): only each
 * row's entropy, confidence and argmax are needed, not its logits).  The LM head's epilogue
 * reduces every 64-column chunk of every row to (max, argmax, Z, S) in float64; a merge
 * forms each row's entropy, confidence and token; the logits are written only when
 * `logits` is not NULL, and never read back.
 *   Arguments as sbd_block_forward and sbd_select; is_mask may be NULL (then the masked
 *   set is tokens == mask_id); the column mask_id of the config is excluded.
 *   logits    device fp32 [batch][k][vocab] or NULL.
 *   outputs   n_accepted [batch], accepted_pos [batch][k] (row indices of the block,
 *             ascending, then -1), accepted_tok [batch][k], entropy and confidence
 *             [batch][k] (nullable): as sbd_select.
 * The entropies equal sbd_select's on the same logits up to float64 summation order (the
 * chunks differ; ~1e-12 relative); the accepted rows and tokens are the same except where
 * a decision is that close.  Limits: batch * k <= 512 (INVALID_ARG beyond).  On the fused
 * decode path (SBD_DECODE_FUSED) the statistics come from the stored logits, which must
 * then be given (UNSUPPORTED otherwise).  The staged K/V and sbd_commit are as for
 * sbd_block_forward.
 */
sbd_status sbd_block_step(sbd_ctx* ctx, int32_t rule, int32_t batch, const int32_t* seq_ids, int32_t k,
                          const int32_t* tokens, const uint8_t* is_mask, const int32_t* n_causal,
                          const int32_t* pos_ids, double threshold, float* logits, int32_t* n_accepted,
                          int32_t* accepted_pos, int32_t* accepted_tok, double* entropy,
                          double* confidence);

/*
 * Exact KV caching (Sec. 1, advantages; Alg. 3): make the K/V staged by the last block
 * forward of each listed sequence permanent for its first n_commit[b] rows
 * (cache_len += n_commit[b]).  n_commit[b] <= that forward's n_causal[b], else STATE.
 * Host arrays seq_ids, n_commit [batch].  Bookkeeping only: no data moves.
 */
sbd_status sbd_commit(sbd_ctx* ctx, int32_t batch, const int32_t* seq_ids,
                      const int32_t* n_commit);

/*
 * EB-Sampler step (Sec. 2.2, eq. (eb_sampler)) on fp32 logits.
 *   logits   device fp32 [batch][k][vocab] (any logits; vocab <= the config's vocab).
 *   is_mask  host [batch][k]: the masked set M of each block.
 *   gamma    >= 0, may be +INFINITY; NaN is rejected.
 *   mask_id  column excluded from the distribution, or -1 for none.
 * For each masked row: H = entropy (nats, float64) of softmax over the vocabulary
 * without mask_id, tok = smallest id attaining the maximum logit.  Masked rows are
 * ordered by (H, row) ascending; with c_r the float64 running sum of the first r
 * entropies (c_0 = 0), s = largest r in [1, |M|] with c_{r-1} <= gamma.
 * Outputs (device): n_accepted [batch] = s (0 if M is empty); accepted_pos
 * [batch][k] = the s rows ascending, then -1; accepted_tok [batch][k] = their tokens,
 * then -1; entropy [batch][k] (nullable) = H for masked rows, NaN otherwise.
 * A masked row whose softmax is undefined (no finite logit outside mask_id, or a NaN or
 * infinite logit) has H = NaN (tok = -1 when no logit is finite), is ordered after every
 * other row and is never accepted: s runs over the other masked rows only, and is 0 when
 * there are none.
 */
sbd_status sbd_eb_select(sbd_ctx* ctx, int32_t batch, int32_t k, int32_t vocab,
                         const float* logits, const uint8_t* is_mask, double gamma,
                         int32_t mask_id, int32_t* n_accepted, int32_t* accepted_pos,
                         int32_t* accepted_tok, double* entropy);

/*
 * One sampling step under a selection rule (Sec. 2.2 and App. B), on fp32 logits.
 * Arguments and outputs as sbd_eb_select, plus:
 *   rule       SBD_SELECT_EB_ENTROPY: exactly sbd_eb_select (threshold = gamma).
 *              SBD_SELECT_EB_CONFIDENCE: App. B, EB-Sampler with the confidence error
 *              proxy: masked rows ordered by (confidence descending, row); s = largest r
 *              in [1, |M|] with sum_{j<=r} H - max_{j<=r} H <= threshold (float64,
 *              summed in that order).
 *              SBD_SELECT_FACTOR: App. B, Factor parallel decoding: the same order; s =
 *              largest r with (r + 1) * (1 - c_r) < threshold, at least 1 (c_r the r-th
 *              confidence; App. B prints the condition without the 1 -, which would
 *              reveal fewer rows the more confident they are).
 *   threshold  gamma (EB rules) or f (Factor): >= 0, may be +INFINITY; NaN is rejected.
 *   confidence device float64 [batch][k] (nullable) = max_v p_v = 1 / Z of each masked
 *              row (the softmax without mask_id), NaN otherwise.
 * As for sbd_eb_select, a row with NaN statistics is never accepted.
 * Errors: INVALID_ARG for an unknown rule, otherwise as sbd_eb_select.
 */
sbd_status sbd_select(sbd_ctx* ctx, int32_t rule, int32_t batch, int32_t k, int32_t vocab,
                      const float* logits, const uint8_t* is_mask, double threshold, int32_t mask_id,
                      int32_t* n_accepted, int32_t* accepted_pos, int32_t* accepted_tok, double* entropy,
                      double* confidence);

/*
 * sbd_eb_select for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, hosts that forbid hipMalloc): no context and no workspace.
 * The chunk statistics live in a fixed scratch array of the library (1.75 MiB per device,
 * held until the process ends; its device address is looked up on the first call on each
 * device).  No hipMalloc, hipFree or other allocating call is made.
 *   stream   hipStream_t to enqueue on (NULL = the null stream); the current device's
 *            scratch is used.
 *   Other arguments, outputs and the selection rule exactly as sbd_eb_select, with
 *   is_mask a host array [batch][k].
 * Limits: batch * k <= 1024, k <= 64, vocab <= 262144; beyond them INVALID_ARG (and
 * nothing is enqueued).  Errors are reported through sbd_last_error(NULL).
 * All calls on one device share its scratch: two calls that overlap in time on one device
 * (different streams, or different host threads) race and give wrong results.
 */
sbd_status sbd_eb_select_noalloc(void* stream, int32_t batch, int32_t k, int32_t vocab,
                                 const float* logits, const uint8_t* is_mask, double gamma,
                                 int32_t mask_id, int32_t* n_accepted, int32_t* accepted_pos,
                                 int32_t* accepted_tok, double* entropy);

/*
 * The selection part of sbd_eb_select alone, on given entropies (device float64
 * [batch][k]); same ordering, rule and outputs (no tokens); a NaN entropy is never accepted.
 */
sbd_status sbd_eb_select_entropies(sbd_ctx* ctx, int32_t batch, int32_t k,
                                   const double* entropy, const uint8_t* is_mask, double gamma,
                                   int32_t* n_accepted, int32_t* accepted_pos);

/*
 * Write n cached rows of a slot from device bf16 K, V [n_layers][n][n_kv_heads][head_dim]
 * (K after RoPE), starting at position pos0 <= cache_len; the slot's cache length
 * becomes pos0 + n and nothing stays staged.  Restores a saved cache, or installs a
 * cache produced elsewhere.  An SBD_KV_FP8_E4M3 cache stores the rounding of the values
 * described with that format.  Errors: CAPACITY if pos0 + n > max_seq_len.
 */
sbd_status sbd_kv_import(sbd_ctx* ctx, int32_t seq, int32_t pos0, int32_t n, const void* k,
                         const void* v);
/* Read rows [pos0, pos0 + n) of a slot (committed or staged) into the same layout. */
sbd_status sbd_kv_export(sbd_ctx* ctx, int32_t seq, int32_t pos0, int32_t n, void* k, void* v);

/*
 * Byte offset and size inside the workspace of a named internal buffer, for
 * inspection by tests: "x" (fp32 residual [rows][d_model]), "qkv" (fp32 projections),
 * "q" (rotated, scaled queries), "attn" (attention output), "act" (SwiGLU output), "xn"
 * (gain-scaled residual).  The last four hold bf16 pairs: [2][rows][width], the value
 * being hi + lo.  rows is the workspace's row capacity, max(max_batch * max_block,
 * prefill chunk).  Values are those of the last layer of the last forward.  INVALID_ARG
 * for an unknown name.
 */
sbd_status sbd_workspace_region(const sbd_model_config* cfg, const char* name, size_t* offset,
                                size_t* bytes);

/*
 * Which kernels run a decode-sized forward (at most 16 rows: sbd_block_forward with
 * batch * k <= 16, and prefill chunks that small).
 *   SBD_DECODE_AUTO     the library's choice (the default): SBD_DECODE_LAYERS where it
 *                       applies, otherwise one kernel per step.
 *   SBD_DECODE_FUSED    the fused forward: every layer and the LM head in one launch of one
 *                       persistent workgroup per CU.  A forward it cannot take fails with
 *                       SBD_ERR_UNSUPPORTED: it needs d_model a multiple of 128 and head_dim
 *                       64 or 128.
 *   SBD_DECODE_KERNELS  one kernel per step.
 *   SBD_DECODE_LAYERS   two launches per layer (QKV + attention + O projection; gate/up +
 *                       down), each XCD of the chip owning one KV head's share.  Needs a
 *                       device of 256 CUs in 8 XCDs, n_kv_heads 8, head_dim 128, d_model
 *                       4096, ffn_dim 12288, 14336 or 16384, batch * k <= 16 and
 *                       (n_q_heads / n_kv_heads) * k <= 64; a forward it cannot take fails
 *                       with SBD_ERR_UNSUPPORTED.
 * All give the same results up to float summation order.  Larger forwards always run one
 * kernel per step.  INVALID_ARG for another value.
 */
typedef enum {
  SBD_DECODE_AUTO = 0,
  SBD_DECODE_FUSED = 1,
  SBD_DECODE_KERNELS = 2,
  SBD_DECODE_LAYERS = 3
} sbd_decode_path;
sbd_status sbd_set_decode_path(sbd_ctx* ctx, int32_t path);
/*
 * Testing aid: the number of polls after which a dependency wait inside a launch gives up:
 * those of the per-XCD layer kernels (decode-sized forwards), and the wait of a split GEMM's
 * K slices for each other (forwards and prefill chunks of more than 16 rows).  A negative
 * value restores the default of about two million, which no correct launch comes near.  A
 * wait that gives up raises the sticky error that every later call on the context reports
 * as SBD_ERR_HIP, with a task code (layer * 16 + phase for a layer kernel, 65536 + the
 * epilogue for GEMM slices); the launch still runs to its end (on wrong data), it never
 * hangs.  With a small limit a test can take that path on purpose.  INVALID_ARG for a null
 * context.
 */
sbd_status sbd_set_wait_limit(sbd_ctx* ctx, int32_t polls);
/*
 * *fits = 1 when `path` can run a decode-sized forward of `batch` sequences of `k` rows on
 * this context's model and device, else 0 (SBD_DECODE_AUTO and SBD_DECODE_KERNELS always
 * can).  INVALID_ARG for a null pointer or an unknown path.
 */
sbd_status sbd_decode_path_fits(const sbd_ctx* ctx, int32_t path, int32_t batch, int32_t k, int32_t* fits);

/*
 * The per-XCD layer kernels and the K-split GEMMs hand partial results between workgroups
 * through one XCD's L2 and rely on workgroup i of a launch running on XCD i % 8 (256 CUs in
 * 8 XCDs).  sbd_create checks this with a probe kernel that reads each workgroup's XCC_ID
 * register (grids of 256, 1000 and 2048 workgroups); where it does not hold, the layer
 * kernels are not used (SBD_DECODE_LAYERS fails with UNSUPPORTED, AUTO takes one kernel per
 * step) and no GEMM splits K, so no hand-off between XCDs is needed.
 *   sbd_xcd_map_ok: *ok = 1 when the probe found the mapping.
 *   sbd_xcd_map_check: the decision itself on given per-workgroup XCD ids (host only):
 *   *ok = 1 iff xcc_ids[i] == i % n_xcd for every i < n.
 */
sbd_status sbd_xcd_map_ok(const sbd_ctx* ctx, int32_t* ok);
sbd_status sbd_xcd_map_check(const int32_t* xcc_ids, int32_t n, int32_t n_xcd, int32_t* ok);

/*
 * Per-kernel timing, for measurement tools.  While enabled, every kernel launch the
 * context makes is bracketed by a pair of HIP events on its stream (this adds a little
 * time between kernels).  sbd_profile_read waits for the recorded work, adds up the
 * elapsed times of all launches of one kernel kind since the previous read of that kind,
 * and returns the launch count and the total in milliseconds.
 */
typedef enum {
  SBD_KERNEL_EMBED = 0,      /* embedding gather + first RMSNorm inputs */
  SBD_KERNEL_QKV = 1,        /* QKV projection */
  SBD_KERNEL_ROPE = 2,       /* q/k norm, RoPE, KV staging */
  SBD_KERNEL_ATTENTION = 3,  /* split-KV block-hybrid attention */
  SBD_KERNEL_ATTN_MERGE = 4, /* merge of the attention splits */
  SBD_KERNEL_O_PROJ = 5,     /* output projection + residual */
  SBD_KERNEL_GATE_UP = 6,    /* gate/up projection + SwiGLU */
  SBD_KERNEL_DOWN = 7,       /* down projection + residual */
  SBD_KERNEL_LM_HEAD = 8,    /* final norm + LM head */
  SBD_KERNEL_EB_PARTIAL = 9, /* EB per-chunk softmax statistics */
  SBD_KERNEL_EB_SELECT = 10, /* EB merge, sort and select */
  SBD_KERNEL_FUSED = 11,     /* fused decode forward: all layers + LM head in one launch */
  SBD_KERNEL_LAYER_ATTN = 12,/* per-XCD layer kernel: QKV + attention + O projection */
  SBD_KERNEL_LAYER_MLP = 13, /* per-XCD layer kernel: gate/up + down projection */
  SBD_KERNEL_LAYER_FINAL = 14, /* per-XCD layer kernels: final norm inputs from the residual */
  SBD_KERNEL_COUNT = 15
} sbd_kernel;
sbd_status sbd_profile_enable(sbd_ctx* ctx, int32_t enable);
/*
 * Measurement aid: one read of `bytes` of device memory at `buf` (a positive multiple of
 * 16) by a plain streaming kernel on `stream` (NULL = the null stream), the device's
 * achievable read rate to compare the block forward's weight streams with.  sink: device
 * uint32 [64], written practically never (it keeps the loads from being dropped).  No
 * context needed; errors through sbd_last_error(NULL).
 */
sbd_status sbd_stream_probe(void* stream, const void* buf, size_t bytes, uint32_t* sink);
sbd_status sbd_profile_read(sbd_ctx* ctx, int32_t kernel, int32_t* launches, double* total_ms);

const char* sbd_status_string(sbd_status s);
/* Reason for the last failed call on ctx; ctx == NULL gives the calling thread's last
 * context-less failure (e.g. of sbd_create). */
const char* sbd_last_error(const sbd_ctx* ctx);

#ifdef __cplusplus
}
#endif
#endif /* SBD_H_ */

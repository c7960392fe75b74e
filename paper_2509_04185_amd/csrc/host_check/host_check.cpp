// sbd_host_check: the C ABI's argument validation and state machine, on the CPU, built with
// AddressSanitizer and UndefinedBehaviorSanitizer (hip_stub.cpp stands in for the runtime and
// the kernels).  Every forced error must be reported with its status and a reason, and must
// leave the context's state unchanged; the state machine (prefill, block forward, commit,
// reset, KV import) must move the cache lengths as documented.  Exit status 0 when every
// check holds.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "sbd.h"

static int g_failed = 0, g_checks = 0;
#define CHECK(cond)                                                    \
  do {                                                                 \
    ++g_checks;                                                        \
    if (!(cond)) {                                                     \
      ++g_failed;                                                      \
      std::fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond);   \
    }                                                                  \
  } while (0)
// a call that must fail with `want`, leave a reason, and not change the cache length of slot 0
#define FAILS(want, ctx, call)                                         \
  do {                                                                 \
    int32_t l0_ = -1, l1_ = -1;                                        \
    sbd_cache_len(ctx, 0, &l0_);                                       \
    const sbd_status st_ = (call);                                     \
    CHECK(st_ == (want));                                              \
    CHECK(std::strlen(sbd_last_error(ctx)) > 0);                       \
    sbd_cache_len(ctx, 0, &l1_);                                       \
    CHECK(l0_ == l1_);                                                 \
  } while (0)

static sbd_model_config tiny_config() {
  sbd_model_config c{};
  c.n_layers = 2; c.d_model = 256; c.n_q_heads = 4; c.n_kv_heads = 2; c.head_dim = 64; c.ffn_dim = 768;
  c.vocab = 1024; c.mask_id = 1023; c.qk_norm = 0; c.rms_eps = 1e-5f; c.rope_theta = 1e4f;
  c.max_batch = 4; c.max_seq_len = 96; c.max_block = 8; c.prefill_chunk = 0; c.weight_format = SBD_WEIGHTS_BF16;
  return c;
}

int main() {
  // ---- configuration and workspace
  sbd_model_config cfg = tiny_config();
  size_t bytes = 0;
  CHECK(sbd_workspace_bytes(nullptr, &bytes) == SBD_ERR_INVALID_ARG);
  CHECK(sbd_workspace_bytes(&cfg, nullptr) == SBD_ERR_INVALID_ARG);
  {
    sbd_model_config b = cfg;
    b.head_dim = 96;
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_ERR_UNSUPPORTED);
    b = cfg;
    b.mask_id = 1024;
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_ERR_UNSUPPORTED);
    b = cfg;
    b.rms_eps = NAN;
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_ERR_UNSUPPORTED);
    b = cfg;
    b.weight_format = 7;
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_ERR_UNSUPPORTED);
    b = cfg;
    b.kv_format = 2;
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_ERR_UNSUPPORTED);
    b = cfg;
    b.kv_format = SBD_KV_FP8_E4M3;
    b.kv_scale_exp = 101;
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_ERR_UNSUPPORTED);
    b.kv_scale_exp = -100;
    size_t b8 = 0, b16 = 0;
    CHECK(sbd_workspace_bytes(&b, &b8) == SBD_OK && sbd_workspace_bytes(&cfg, &b16) == SBD_OK);
    CHECK(b8 < b16);  // one byte per cached element instead of two
    b = cfg;
    b.kv_scale_exp = 1000;  // ignored with a bf16 cache
    CHECK(sbd_workspace_bytes(&b, &bytes) == SBD_OK);
  }
  CHECK(sbd_workspace_bytes(&cfg, &bytes) == SBD_OK && bytes > 0);

  // ---- weights ("device" pointers: never dereferenced by the host code)
  static char dummy[256];
  std::vector<const void*> per_layer(cfg.n_layers, dummy);
  sbd_weights w{};
  w.embed = w.lm_head = w.final_norm = dummy;
  w.attn_norm = w.wq = w.wk = w.wv = w.wo = w.mlp_norm = w.w_gate = w.w_up = w.w_down = per_layer.data();

  void* ws = std::aligned_alloc(256, (bytes + 255) / 256 * 256);
  sbd_ctx* ctx = nullptr;
  CHECK(sbd_create(&cfg, &w, nullptr, bytes, nullptr, &ctx) == SBD_ERR_INVALID_ARG && ctx == nullptr);
  CHECK(sbd_create(&cfg, &w, static_cast<char*>(ws) + 16, bytes, nullptr, &ctx) == SBD_ERR_INVALID_ARG);
  CHECK(sbd_create(&cfg, &w, ws, bytes - 1, nullptr, &ctx) == SBD_ERR_OUT_OF_MEMORY);
  {
    sbd_weights b = w;
    b.lm_head = nullptr;
    CHECK(sbd_create(&cfg, &b, ws, bytes, nullptr, &ctx) == SBD_ERR_INVALID_ARG);
    std::vector<const void*> holed = per_layer;
    holed[1] = nullptr;
    b = w;
    b.wo = holed.data();
    CHECK(sbd_create(&cfg, &b, ws, bytes, nullptr, &ctx) == SBD_ERR_INVALID_ARG);
    sbd_model_config q = cfg;
    q.qk_norm = 1;
    size_t qb = 0;
    CHECK(sbd_workspace_bytes(&q, &qb) == SBD_OK);
    void* qws = std::aligned_alloc(256, (qb + 255) / 256 * 256);
    CHECK(sbd_create(&q, &w, qws, qb, nullptr, &ctx) == SBD_ERR_INVALID_ARG);  // no q/k norm gains
    std::free(qws);
    sbd_model_config f8 = cfg;
    f8.weight_format = SBD_WEIGHTS_FP8_E4M3;
    size_t fb = 0;
    CHECK(sbd_workspace_bytes(&f8, &fb) == SBD_OK && fb > bytes);
    void* fws = std::aligned_alloc(256, (fb + 255) / 256 * 256);
    CHECK(sbd_create(&f8, &w, fws, fb, nullptr, &ctx) == SBD_ERR_INVALID_ARG);  // no scale exponents
    std::vector<int32_t> exps(cfg.n_layers * 7 + 1, -12);
    exps[3] = 200;
    b = w;
    b.fp8_scale_exp = exps.data();
    CHECK(sbd_create(&f8, &b, fws, fb, nullptr, &ctx) == SBD_ERR_INVALID_ARG);  // exponent out of range
    exps[3] = -11;
    CHECK(sbd_create(&f8, &b, fws, fb, nullptr, &ctx) == SBD_OK && ctx != nullptr);
    CHECK(sbd_destroy(ctx) == SBD_OK);
    ctx = nullptr;
    std::free(fws);
  }
  CHECK(sbd_create(&cfg, &w, ws, bytes, nullptr, &ctx) == SBD_OK && ctx != nullptr);
  if (!ctx) {
    std::fprintf(stderr, "no context: stopping\n");
    return 1;
  }
  int32_t ok = -1;
  CHECK(sbd_xcd_map_ok(ctx, &ok) == SBD_OK && ok == 0);  // the stand-in device has no CUs
  int32_t fits = -1;
  CHECK(sbd_decode_path_fits(ctx, SBD_DECODE_LAYERS, 1, 4, &fits) == SBD_OK && fits == 0);

  // ---- prefill
  std::vector<int32_t> prompt(40);
  for (int i = 0; i < 40; ++i) prompt[i] = (i * 37) % 1000;
  int32_t len = -1;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_prefill(ctx, 9, prompt.data(), 40, nullptr));   // slot out of range
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_prefill(ctx, 0, prompt.data(), 0, nullptr));    // no tokens
  prompt[5] = 1023;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_prefill(ctx, 0, prompt.data(), 40, nullptr));   // the mask id
  prompt[5] = 1024;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_prefill(ctx, 0, prompt.data(), 40, nullptr));   // out of range
  prompt[5] = 5;
  std::vector<int32_t> longp(97, 3);
  FAILS(SBD_ERR_CAPACITY, ctx, sbd_prefill(ctx, 0, longp.data(), 97, nullptr));
  CHECK(sbd_prefill(ctx, 0, prompt.data(), 40, nullptr) == SBD_OK);
  CHECK(sbd_cache_len(ctx, 0, &len) == SBD_OK && len == 40);
  CHECK(sbd_prefill(ctx, 1, prompt.data(), 10, nullptr) == SBD_OK);

  // ---- block forward: each argument check of sbd_block_forward, forced one at a time
  const int k = 4;
  static float logits_buf[2 * 8 * 1024];
  float* logits = logits_buf;
  int32_t seqs[2] = {0, 1};
  int32_t toks[8] = {7, 1023, 1023, 1023, 8, 1023, 1023, 1023};
  uint8_t msk[8] = {0, 1, 1, 1, 0, 1, 1, 1};
  int32_t nc[2] = {1, 1};
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, 9, toks, msk, nc, nullptr, logits));  // k > max_block
  nc[0] = 5;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, nullptr, logits));  // n_causal > k
  nc[0] = 2;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, nullptr, logits));  // causal mask row
  nc[0] = 1;
  msk[2] = 0;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, nullptr, logits));  // inconsistent
  msk[2] = 1;
  toks[4] = 5000;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, nullptr, logits));  // token range
  toks[4] = 8;
  int32_t dup[2] = {1, 1};
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, dup, k, toks, msk, nc, nullptr, logits));   // duplicated
  int32_t bad_seq[2] = {0, 4};
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, bad_seq, k, toks, msk, nc, nullptr, logits));
  int32_t pos[8] = {40, 41, 42, 43, 10, 11, 12, 13};
  pos[0] = 41;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, pos, logits));  // causal position
  pos[0] = 40;
  pos[7] = 96;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, pos, logits));  // position range
  pos[7] = 13;
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, pos, nullptr));   // no logits
  // commit before any forward of slot 0
  int32_t one[1] = {0}, n1[1] = {1};
  FAILS(SBD_ERR_STATE, ctx, sbd_commit(ctx, 1, one, n1));
  CHECK(sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, pos, logits) == SBD_OK);
  int32_t n2[2] = {2, 1};
  FAILS(SBD_ERR_STATE, ctx, sbd_commit(ctx, 2, seqs, n2));  // more than the forward's causal rows
  int32_t n_neg[2] = {-1, 0};
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_commit(ctx, 2, seqs, n_neg));
  int32_t n_ok[2] = {1, 0};
  CHECK(sbd_commit(ctx, 2, seqs, n_ok) == SBD_OK);
  CHECK(sbd_cache_len(ctx, 0, &len) == SBD_OK && len == 41);
  CHECK(sbd_cache_len(ctx, 1, &len) == SBD_OK && len == 10);
  FAILS(SBD_ERR_STATE, ctx, sbd_commit(ctx, 1, one, n1));  // staged rows were consumed
  // capacity: 41 + k > 96 once the slot is nearly full
  std::vector<int32_t> fill(52, 9);
  CHECK(sbd_prefill(ctx, 0, fill.data(), 52, nullptr) == SBD_OK);  // 93 now
  FAILS(SBD_ERR_CAPACITY, ctx, sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, nullptr, logits));
  CHECK(sbd_reset(ctx, 0) == SBD_OK);
  CHECK(sbd_cache_len(ctx, 0, &len) == SBD_OK && len == 0);
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_reset(ctx, -1));

  // ---- selection
  int32_t n_acc[2], acc_pos[8], acc_tok[8];
  double H[8], C[8];
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select(ctx, 2, k, 1024, logits, msk, NAN, 1023, n_acc, acc_pos, acc_tok, H));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select(ctx, 2, k, 1024, logits, msk, -0.5, 1023, n_acc, acc_pos, acc_tok, H));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select(ctx, 2, k, 2048, logits, msk, 1.0, 1023, n_acc, acc_pos, acc_tok, H));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select(ctx, 2, k, 1024, logits, msk, 1.0, 1024, n_acc, acc_pos, acc_tok, H));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select(ctx, 5, k, 1024, logits, msk, 1.0, 1023, n_acc, acc_pos, acc_tok, H));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select(ctx, 2, k, 1024, logits, nullptr, 1.0, 1023, n_acc, acc_pos, acc_tok, H));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_select(ctx, 3, 2, k, 1024, logits, msk, 1.0, 1023, n_acc, acc_pos, acc_tok, H, C));
  CHECK(sbd_eb_select(ctx, 2, k, 1024, logits, msk, INFINITY, 1023, n_acc, acc_pos, acc_tok, H) == SBD_OK);
  CHECK(sbd_select(ctx, SBD_SELECT_FACTOR, 2, k, 1024, logits, msk, 2.0, -1, n_acc, acc_pos, acc_tok, H, C) == SBD_OK);
  CHECK(sbd_eb_select_entropies(ctx, 2, k, H, msk, 1.0, n_acc, acc_pos) == SBD_OK);
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_eb_select_entropies(ctx, 2, k, nullptr, msk, 1.0, n_acc, acc_pos));

  // ---- block step
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_step(ctx, 9, 2, seqs, k, toks, msk, nc, nullptr, 1.0, nullptr, n_acc,
                                                 acc_pos, acc_tok, H, C));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_step(ctx, 0, 2, seqs, k, toks, msk, nc, nullptr, NAN, nullptr, n_acc,
                                                 acc_pos, acc_tok, H, C));
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_block_step(ctx, 0, 2, seqs, k, toks, msk, nc, nullptr, 1.0, nullptr, nullptr,
                                                 acc_pos, acc_tok, H, C));
  CHECK(sbd_set_decode_path(ctx, SBD_DECODE_FUSED) == SBD_OK);
  FAILS(SBD_ERR_UNSUPPORTED, ctx, sbd_block_step(ctx, 0, 2, seqs, k, toks, msk, nc, nullptr, 1.0, nullptr, n_acc,
                                                 acc_pos, acc_tok, H, C));
  CHECK(sbd_set_decode_path(ctx, SBD_DECODE_AUTO) == SBD_OK);
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_set_decode_path(ctx, 9));
  CHECK(sbd_block_step(ctx, 0, 2, seqs, k, toks, nullptr, nc, nullptr, 1.0, nullptr, n_acc, acc_pos, acc_tok, H, C) ==
        SBD_OK);
  CHECK(sbd_commit(ctx, 2, seqs, n_ok) == SBD_OK);
  CHECK(sbd_cache_len(ctx, 0, &len) == SBD_OK && len == 1);

  // ---- KV import / export
  static uint16_t kv[2 * 8 * 2 * 64];
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_kv_import(ctx, 0, 5, 4, kv, kv));  // beyond cache_len
  FAILS(SBD_ERR_CAPACITY, ctx, sbd_kv_import(ctx, 0, 0, 97, kv, kv));
  CHECK(sbd_kv_import(ctx, 0, 0, 8, kv, kv) == SBD_OK);
  CHECK(sbd_cache_len(ctx, 0, &len) == SBD_OK && len == 8);
  CHECK(sbd_kv_export(ctx, 0, 0, 8, kv, kv) == SBD_OK);

  // ---- the allocation-free EB step: its limits
  CHECK(sbd_eb_select_noalloc(nullptr, 17, 64, 128, logits, msk, 1.0, -1, n_acc, acc_pos, acc_tok, nullptr) ==
        SBD_ERR_INVALID_ARG);
  CHECK(sbd_eb_select_noalloc(nullptr, 1, 4, 262145, logits, msk, 1.0, -1, n_acc, acc_pos, acc_tok, nullptr) ==
        SBD_ERR_INVALID_ARG);
  CHECK(sbd_eb_select_noalloc(nullptr, 2, 4, 1024, logits, msk, 1.0, 1023, n_acc, acc_pos, acc_tok, H) == SBD_OK);

  // ---- profiling, status strings, teardown
  CHECK(sbd_profile_enable(ctx, 1) == SBD_OK);
  CHECK(sbd_block_forward(ctx, 2, seqs, k, toks, msk, nc, nullptr, logits) == SBD_OK);
  int32_t launches = 0;
  double ms = 0.0;
  CHECK(sbd_profile_read(ctx, SBD_KERNEL_LM_HEAD, &launches, &ms) == SBD_OK && launches == 1);
  FAILS(SBD_ERR_INVALID_ARG, ctx, sbd_profile_read(ctx, SBD_KERNEL_COUNT, &launches, &ms));
  for (int s = 0; s <= 6; ++s) CHECK(std::strlen(sbd_status_string(static_cast<sbd_status>(s))) > 0);
  CHECK(sbd_destroy(ctx) == SBD_OK);
  CHECK(sbd_destroy(nullptr) == SBD_ERR_INVALID_ARG);
  std::free(ws);

  std::printf("%d of %d host checks %s\n", g_checks - g_failed, g_checks, g_failed ? "passed, some FAILED" : "passed");
  return g_failed ? 1 : 0;
}

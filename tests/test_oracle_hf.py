"""Pins of the oracle's decoder body against an independent implementation (CPU only).

The paper states that the SBD network is the unchanged Llama-3.1 / Qwen-3 decoder (Sec. 1,
advantages list; Sec. 3.1 names Llama-3.1-8B and Qwen-3-8B), and defines no numbers for
its body.  The oracle composes that body itself (pre-norm residual blocks, SwiGLU with the
gate inside the SiLU, per-head q/k RMSNorm before rotate-half RoPE, untied LM head).  Here
the same bf16 weights go into the ``transformers`` implementations of both families, in
float64 on the CPU, and the oracle's causal forward (causal point at the end, which is a
plain next-token-prediction forward over every row) and its prefill cache must agree with
them.  The library routines compute their RMSNorm in float32, so the agreement is at
float32 level.

Planted mistakes in the oracle's composition (gate and up exchanged, post-norm blocks,
q/k-norm after RoPE, a norm without its gain, a GELU in place of SiLU) are each shown to
fail the comparison.
"""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import sbd_oracle as O

transformers = pytest.importorskip("transformers")

REL_L2 = 1e-5     # float32-level agreement (the library's RMSNorm runs in float32)
T = 24            # tokens of the compared sequence


def _hf_model(shape, w):
    """A transformers model of `shape` holding the weights `w` (bf16 torch tensors), float64."""
    common = dict(vocab_size=shape.vocab, hidden_size=shape.d_model, intermediate_size=shape.ffn_dim,
                  num_hidden_layers=shape.n_layers, num_attention_heads=shape.n_q_heads,
                  num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                  rms_norm_eps=shape.rms_eps, rope_theta=shape.rope_theta, tie_word_embeddings=False,
                  attention_bias=False, max_position_embeddings=4096, attn_implementation="eager")
    if shape.qk_norm:
        cfg = transformers.Qwen3Config(**common)
        model = transformers.Qwen3ForCausalLM(cfg)
    else:
        cfg = transformers.LlamaConfig(mlp_bias=False, **common)
        model = transformers.LlamaForCausalLM(cfg)
    model = model.double().eval()
    sd = {"model.embed_tokens.weight": w["embed"], "model.norm.weight": w["final_norm"],
          "lm_head.weight": w["lm_head"]}
    names = {"attn_norm": "input_layernorm", "mlp_norm": "post_attention_layernorm",
             "wq": "self_attn.q_proj", "wk": "self_attn.k_proj", "wv": "self_attn.v_proj",
             "wo": "self_attn.o_proj", "w_gate": "mlp.gate_proj", "w_up": "mlp.up_proj",
             "w_down": "mlp.down_proj"}
    if shape.qk_norm:
        names.update(q_norm="self_attn.q_norm", k_norm="self_attn.k_norm")
    for li, lw in enumerate(w["layers"]):
        for key, hf in names.items():
            sd[f"model.layers.{li}.{hf}.weight"] = lw[key]
    sd = {k: v.to(torch.float64) for k, v in sd.items()}
    missing, unexpected = model.load_state_dict(sd, strict=False)
    # rotary buffers are not parameters; every parameter must have been given
    assert not unexpected and not [m for m in missing if "rotary" not in m], (missing, unexpected)
    return model


@pytest.fixture(scope="module", params=["tiny", "tiny_qk"])
def pair(request):
    shape = synth.SHAPES[request.param]
    w = synth.make_weights(shape, 31)
    model = O.Model(shape, synth.weights_to_host(w), dtype=np.float64)
    hf = _hf_model(shape, w)
    tokens = synth.make_tokens(31, T, shape)
    with torch.no_grad():
        out = hf(input_ids=torch.from_numpy(tokens.astype(np.int64))[None], use_cache=True)
    return shape, model, tokens, out


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def test_causal_logits_match_transformers(pair):
    shape, model, tokens, out = pair
    ref = out.logits[0].numpy()
    got = model.full_forward(tokens, causal_point=T)
    assert got.shape == ref.shape == (T, shape.vocab)
    assert _rel(got, ref) <= REL_L2


def test_prefill_cache_matches_transformers(pair):
    """Post-RoPE keys and the values of every layer (the exact KV cache of Sec. 1)."""
    shape, model, tokens, out = pair
    cache, last = model.prefill(tokens)
    for li in range(shape.n_layers):
        layer = out.past_key_values.layers[li]
        k_ref = layer.keys[0].permute(1, 0, 2).numpy()       # [T][H_kv][d_h]
        v_ref = layer.values[0].permute(1, 0, 2).numpy()
        assert _rel(cache.K[li], k_ref) <= REL_L2
        assert _rel(cache.V[li], v_ref) <= REL_L2
    assert _rel(last, out.logits[0, -1].numpy()) <= REL_L2


def test_block_forward_rows_match_transformers(pair):
    """A cached block of causal rows (k = 4 after a 20-token prefix) gives the library's
    logits of those positions: the cached path composes the same body."""
    shape, model, tokens, out = pair
    cache, _ = model.prefill(tokens[:T - 4])
    res = model.block_forward([cache], tokens[None, T - 4:], [4])
    assert _rel(res.logits[0], out.logits[0, T - 4:].numpy()) <= REL_L2


def test_decode_weight_matches_torch_bf16():
    """decode_weight reads raw bf16 bit patterns; torch's bf16 -> float32 conversion is the
    definition.  All 65536 patterns, NaNs compared as NaN."""
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):
        got = O.decode_weight(bits, np.float32)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32))  # -0.0 and denormals too
    assert O.decode_weight(bits, np.float64).dtype == np.float64


# ------------------------------------------------------------------ planted mistakes


def _fails(pair):
    shape, model, tokens, out = pair
    fresh = O.Model(shape, model.w, dtype=np.float64)
    return _rel(fresh.full_forward(tokens, causal_point=T), out.logits[0].numpy()) > 100 * REL_L2


def test_planted_gate_up_swap_is_caught(pair, monkeypatch):
    def mlp(self, x, li):
        s = self.s
        h2 = O.rms_norm(x, self.W("mlp_norm", li), s.rms_eps)
        a = O.silu(h2 @ self.W("w_up", li).T) * (h2 @ self.W("w_gate", li).T)
        return a @ self.W("w_down", li).T
    monkeypatch.setattr(O.Model, "_mlp", mlp)
    assert _fails(pair)


def test_planted_gelu_for_silu_is_caught(pair, monkeypatch):
    monkeypatch.setattr(O, "silu", lambda z: 0.5 * z * (1.0 + np.tanh(0.7978845608 * (z + 0.044715 * z ** 3))))
    assert _fails(pair)


def test_planted_norm_without_gain_is_caught(pair, monkeypatch):
    plain = O.rms_norm
    monkeypatch.setattr(O, "rms_norm", lambda x, g, eps: plain(x, np.ones_like(g), eps))
    assert _fails(pair)


def test_planted_post_norm_blocks_are_caught(pair, monkeypatch):
    def full_forward(self, tokens, causal_point, pos=None):
        s = self.s
        tokens = np.asarray(tokens).reshape(-1)
        n = tokens.shape[0]
        vis = np.arange(n)[None, :] <= np.arange(n)[:, None]
        x = self.W("embed")[tokens]
        for li in range(s.n_layers):
            q, kk, vv = self._qkv(x, li, np.arange(n))
            x = O.rms_norm(x + O.attention(q, kk, vv, vis).reshape(n, -1) @ self.W("wo", li).T,
                           self.W("attn_norm", li), s.rms_eps)
            a = O.silu(x @ self.W("w_gate", li).T) * (x @ self.W("w_up", li).T)
            x = O.rms_norm(x + a @ self.W("w_down", li).T, self.W("mlp_norm", li), s.rms_eps)
        return x @ self.W("lm_head").T
    monkeypatch.setattr(O.Model, "full_forward", full_forward)
    assert _fails(pair)


def test_planted_qk_norm_after_rope_is_caught(monkeypatch):
    shape = synth.TINY_QK
    w = synth.make_weights(shape, 31)
    hf = _hf_model(shape, w)
    tokens = synth.make_tokens(31, T, shape)
    with torch.no_grad():
        ref = hf(input_ids=torch.from_numpy(tokens.astype(np.int64))[None]).logits[0].numpy()

    def qkv(self, h, li, pos):
        s = self.s
        rows = h.shape[0]
        q = (h @ self.W("wq", li).T).reshape(rows, s.n_q_heads, s.head_dim)
        k = (h @ self.W("wk", li).T).reshape(rows, s.n_kv_heads, s.head_dim)
        v = (h @ self.W("wv", li).T).reshape(rows, s.n_kv_heads, s.head_dim)
        cos, sin = O.rope_cos_sin(pos, s.head_dim, s.rope_theta, self.dtype)
        q, k = O.apply_rope(q, cos, sin), O.apply_rope(k, cos, sin)
        return O.rms_norm(q, self.W("q_norm", li), s.rms_eps), O.rms_norm(k, self.W("k_norm", li), s.rms_eps), v
    monkeypatch.setattr(O.Model, "_qkv", qkv)
    model = O.Model(shape, synth.weights_to_host(w), dtype=np.float64)
    assert _rel(model.full_forward(tokens, causal_point=T), ref) > 100 * REL_L2


def test_planted_tied_head_is_caught(pair):
    shape, model, tokens, out = pair
    w = dict(model.w)
    w["lm_head"] = w["embed"]
    tied = O.Model(shape, w, dtype=np.float64)
    assert _rel(tied.full_forward(tokens, causal_point=T), out.logits[0].numpy()) > 100 * REL_L2


def test_eight_b_layer_shape_matches_transformers():
    """One layer at the 8B Llama shape (GQA 32/8, d_h 128, F 14336, theta 5e5) with a small
    vocabulary: the shape-dependent parts (head grouping, the RoPE frequencies of d_h = 128)
    agree too."""
    shape = dataclasses.replace(synth.LLAMA8B, n_layers=1, vocab=256, mask_id=255)
    w = synth.make_weights(shape, 5)
    hf = _hf_model(shape, w)
    tokens = synth.make_tokens(5, 6, shape)
    with torch.no_grad():
        ref = hf(input_ids=torch.from_numpy(tokens.astype(np.int64))[None]).logits[0].numpy()
    model = O.Model(shape, synth.weights_to_host(w), dtype=np.float64)
    assert _rel(model.full_forward(tokens, causal_point=6), ref) <= REL_L2


def test_decode_e4m3_matches_torch_float8():
    """The oracle's e4m3 decoder against torch's float8_e4m3fn, all 256 patterns, and the
    format's landmarks (1, the largest 448, the smallest subnormal 2^-9, -0)."""
    bits = np.arange(256, dtype=np.uint8)
    got = O.decode_e4m3(bits)
    ref = torch.from_numpy(bits).view(torch.float8_e4m3fn).to(torch.float32).numpy().astype(np.float64)
    nan = np.isnan(ref)
    assert nan.sum() == 2 and np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert O.decode_e4m3([0x38, 0x7E, 0x01, 0x80]).tolist() == [1.0, 448.0, 2.0 ** -9, 0.0]
    assert np.signbit(O.decode_e4m3([0x80]))[0]


def test_fp8_weights_model_uses_scaled_values():
    """An FP8 model's matrices are the decoded bytes times 2^e of their matrix; the causal
    forward then matches transformers run on those same values."""
    shape = synth.TINY
    w8 = synth.make_weights_fp8(shape, 32)
    host = synth.weights_to_host(w8)
    model = O.Model(shape, host, dtype=np.float64)
    exps = w8["fp8_scale_exp"]
    assert len(exps) == shape.n_layers * 7 + 1 and all(-20 <= e <= 0 for e in exps)
    wq = model.W("wq", 1)
    ref = torch.from_numpy(host["layers"][1]["wq"]).view(torch.float8_e4m3fn).double().numpy() * 2.0 ** exps[7]
    assert np.array_equal(wq, ref)
    assert np.array_equal(model.W("lm_head"),
                          torch.from_numpy(host["lm_head"]).view(torch.float8_e4m3fn).double().numpy() * 2.0 ** exps[-1])
    # the widened values in bf16 (exact: at most 4 significant bits) into the library model
    wide = {k: v for k, v in w8.items() if k not in ("layers", "fp8_scale_exp")}
    wide["layers"] = [dict(lw) for lw in w8["layers"]]
    for li, lw in enumerate(wide["layers"]):
        for j, key in enumerate(synth.FP8_KEYS):
            lw[key] = (lw[key].view(torch.float8_e4m3fn).float() * 2.0 ** exps[li * 7 + j]).to(torch.bfloat16)
    wide["lm_head"] = (w8["lm_head"].view(torch.float8_e4m3fn).float() * 2.0 ** exps[-1]).to(torch.bfloat16)
    hf = _hf_model(shape, wide)
    tokens = synth.make_tokens(32, T, shape)
    with torch.no_grad():
        out = hf(input_ids=torch.from_numpy(tokens.astype(np.int64))[None]).logits[0].numpy()
    assert _rel(model.full_forward(tokens, causal_point=T), out) <= REL_L2

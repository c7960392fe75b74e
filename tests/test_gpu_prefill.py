"""The KV cache a long real prefill leaves on the GPU, pinned position by position.

Alg. 2 starts with a prefill of the prompt and every later block attends to that cache, so
the cache must be the exact one (Sec. 1): the post-RoPE keys and the values a causal
forward produces at every position.  At 32768 (Llama-3.1-8B shape) and 8192 (Qwen-3-8B
shape, q/k norm) positions a full CPU prefill is too slow, but layer 0's keys and values
depend only on the prompt's embeddings, so the oracle recomputes them at every position,
and layer 1's at sampled positions p from the oracle's own layer 0 (one causal row at p
over the recomputed layer-0 cache: its layer-1 K/V need nothing else).  This covers RoPE
at large positions and the prefill's split attention over long prefixes.  Two-layer
decoders of the real layer shapes; both caches hold bf16 values, so a difference of one
bf16 unit where the two sides round differently is allowed (max-abs 0.07 at magnitudes up
to ~8).
"""
import dataclasses

import numpy as np
import pytest
import torch

import parity
import synth
from oracle import sbd_oracle as O

pytestmark = pytest.mark.gpu

CASES = {"llama8b_l32768": (synth.LLAMA8B, 32768, 1201), "qwen8b_l8192": (synth.QWEN8B, 8192, 1202)}


@pytest.mark.parametrize("name", list(CASES))
def test_long_prefill_cache(name):
    from paper_2509_04185_amd import Sbd
    base, T, seed = CASES[name]
    shape = dataclasses.replace(base, name=base.name + "_2layers", n_layers=2)
    torch.cuda.empty_cache()
    print(f"[gpu] {name}: prefill of {T} tokens", flush=True)
    w = synth.make_weights(shape, seed, device="cuda")
    lib = Sbd(shape, w, max_batch=1, max_seq_len=T + 64, max_block=16)
    prompt = synth.make_tokens(seed, T, shape, stream=7)
    lib.prefill(0, prompt, want_logits=False)
    assert lib.cache_len(0) == T
    kk, vv = lib.kv_export(0, 0, T)
    torch.cuda.synchronize()
    gk = kk.float().cpu().numpy()              # [2][T][H_kv][d_h]
    gv = vv.float().cpu().numpy()
    del kk, vv
    lib.close()

    model = O.Model(shape, synth.weights_to_host(w), dtype=np.float32, kv_bf16=True)
    print("    oracle: layer 0 at every position", flush=True)
    x = model.W("embed")[prompt]
    h = O.rms_norm(x, model.W("attn_norm", 0), shape.rms_eps)
    _, k0, v0 = model._qkv(h, 0, np.arange(T))
    del x, h
    # measured: max-abs 3.1e-2 (one bf16 unit), rel-L2 4.2e-5 (layer 0); 5.4e-4 (layer 1)
    parity.close(gk[0], k0, max_abs=0.07, regress=(0.07, 5e-4), label="K layer 0: ")
    parity.close(gv[0], v0, max_abs=0.07, regress=(0.07, 5e-4), label="V layer 0: ")

    rng = np.random.default_rng(seed)
    positions = sorted({0, 1, 255, 256, 257, 4095, T // 2 + 3, T - 1} |
                       {int(p) for p in rng.integers(0, T, 4)})
    print(f"    oracle: layer 1 at positions {positions}", flush=True)
    got_k, got_v, ref_k, ref_v = [], [], [], []
    for p in positions:
        c = O.SeqCache.__new__(O.SeqCache)
        empty = np.zeros((p, shape.n_kv_heads, shape.head_dim), np.float32)
        c.K = [k0[:p], empty]                  # layer 1's cache does not enter its K/V at p
        c.V = [v0[:p], empty]
        res = model.block_forward([c], prompt[None, p:p + 1], [1])
        ref_k.append(res.K_new[0][1][0])
        ref_v.append(res.V_new[0][1][0])
        got_k.append(gk[1][p])
        got_v.append(gv[1][p])
    parity.close(np.stack(got_k), np.stack(ref_k), max_abs=0.07, regress=(0.07, 4e-3), label="K layer 1: ")
    parity.close(np.stack(got_v), np.stack(ref_v), max_abs=0.07, regress=(0.07, 4e-3), label="V layer 1: ")

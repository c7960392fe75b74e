"""FP8 (e4m3) KV cache, the 1-byte KV of the paper's timing model (Sec. 4.1), on the GPU.

The cache holds the e4m3 code of v * 2^-e for every key (after RoPE) and value, rounded to
the nearest code with ties to even and saturated at +-448; the rows a forward stages are
rounded before its own attention reads them.  The oracle (Model(kv_fp8_exp=e)) rounds its
keys and values the same way (round_to_e4m3, pinned against brute force and torch's cast).

* import then export: bit-exact against the oracle's rounding of the same bf16 inputs,
  with every tie of the e4m3 grid, saturation, subnormals, infinities and NaN planted;
* caches written by forwards: the two sides round floats that agree to float precision,
  so a value at a rounding midpoint may land one code apart (parity.kv8_close);
* logits: the contract bound and a regression bound against the oracle with the same
  cache format, on every path that reads an fp8 cache: the per-kernel path (one kernel per
  step for at most 16 rows, the GEMM, RoPE-staging and split-attention kernels for more
  rows and for prefill), the per-XCD layer kernels at the Llama-3.1-8B layer shape, and
  FP8 weights with an FP8 cache (the paper's timing assumption) at the benched size.
The fused decode path reads bf16 caches only: asking for it is UNSUPPORTED.
"""
import dataclasses

import numpy as np
import pytest
import torch

import parity
import synth
from oracle import sbd_oracle as O

pytestmark = pytest.mark.gpu

REGRESS = (5e-3, 6e-4)
KV8 = "fp8_e4m3"


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def planted_values(e):
    """bf16 values that probe the rounding: every midpoint of neighbouring e4m3 values (ties:
    at most 5 significant bits, exact in bf16), the values themselves, saturation, infinities,
    NaN, signed zeros, values below half the smallest subnormal; all times 2^e."""
    vals = O.decode_e4m3(np.arange(256))
    u = np.unique(vals[~np.isnan(vals)])
    x = np.concatenate([u, (u[1:] + u[:-1]) / 2, [450.0, 464.0, 480.0, 8192.0, 2.0 ** -11, -0.0]])
    x = x * 2.0 ** e
    x = np.concatenate([x, [np.inf, -np.inf, np.nan, 3e38, -3e38]])
    t = torch.from_numpy(x).float().to(torch.bfloat16)
    assert np.array_equal(t.double().numpy()[:-5], x[:-5])       # planted exactly
    return t


@pytest.mark.parametrize("e", [0, -3, 2])
def test_kv8_import_export_rounds_like_the_oracle(e):
    from paper_2509_04185_amd import Sbd
    shape = synth.TINY
    print(f"[gpu] e4m3 KV import/export, scale 2^{e}", flush=True)
    w = synth.make_weights(shape, 9300, device="cuda")
    lib = Sbd(shape, w, max_batch=2, max_seq_len=160, max_block=16, kv_format=KV8, kv_scale_exp=e)
    kk, vv = synth.make_kv(shape, 9300 + e, 1, 150, device="cuda")
    p = planted_values(e).cuda()
    kk.view(-1)[:p.numel()] = p
    vv.view(-1)[-p.numel():] = p.flip(0)
    lib.kv_import(1, 0, kk, vv)
    k2, v2 = lib.kv_export(1, 0, 150)
    torch.cuda.synchronize()
    assert np.array_equal(host(k2), O.round_to_e4m3(host(kk), e), equal_nan=True)
    assert np.array_equal(host(v2), O.round_to_e4m3(host(vv), e), equal_nan=True)
    # a second import over part of the range rounds again; the rest is kept
    lib.kv_import(1, 20, kk[:, :30].contiguous(), vv[:, :30].contiguous())
    assert lib.cache_len(1) == 50
    k3, _ = lib.kv_export(1, 0, 50)
    torch.cuda.synchronize()
    assert np.array_equal(host(k3[:, 20:]), O.round_to_e4m3(host(kk[:, :30]), e), equal_nan=True)
    assert np.array_equal(host(k3[:, :20]), host(k2[:, :20]), equal_nan=True)
    lib.close()


@pytest.mark.parametrize("shape,e", [(synth.TINY, 0), (synth.TINY_QK, -2)], ids=["tiny", "tiny_qk"])
def test_kv8_tiny_prefill_blocks_commit(shape, e):
    """Prefill (GEMM path, RoPE staging, split attention), block forwards of 4, 16 and 32
    rows, commit, against the oracle with an e4m3 cache; the fused path is refused."""
    from paper_2509_04185_amd import Sbd
    from paper_2509_04185_amd.binding import SbdError
    print(f"[gpu] {shape.name} with an e4m3 KV cache, scale 2^{e}", flush=True)
    w = synth.make_weights(shape, 9310, device="cuda")
    lib = Sbd(shape, w, max_batch=4, max_seq_len=128, max_block=16, prefill_chunk=24,
              kv_format=KV8, kv_scale_exp=e)
    model = O.Model(shape, synth.weights_to_host(w), dtype=np.float64, kv_fp8_exp=e)
    caches = []
    for b in range(4):
        prompt = synth.make_tokens(9311 + b, 20 + 9 * b, shape)  # up to 47 rows: two chunks
        got = lib.prefill(b, prompt)
        cache, ref_last = model.prefill(prompt)
        caches.append(cache)
        parity.close(got.cpu().numpy(), ref_last, regress=REGRESS, label=f"prefill {b}: ")
        kx, vx = lib.kv_export(b, 0, len(prompt))
        torch.cuda.synchronize()
        for li in range(shape.n_layers):
            parity.kv8_close(host(kx[li]), caches[b].K[li], e, label=f"prefill {b} K layer {li}: ")
            parity.kv8_close(host(vx[li]), caches[b].V[li], e, label=f"prefill {b} V layer {li}: ")
    assert not lib.decode_path_fits("fused", 1, 4)
    for B, k in ((1, 4), (2, 8), (4, 8)):
        toks, is_mask = synth.block_rows(9320 + B, shape, B, k, n_causal=2)
        got = lib.block_forward(list(range(B)), toks, is_mask=is_mask, n_causal=[2] * B).cpu().numpy()
        ref = model.block_forward(caches[:B], toks, [2] * B).logits
        parity.close(got, ref, regress=REGRESS, label=f"{B}x{k}: ")
    # commit the two causal rows of the last forward; the staged keys/values enter the cache
    res = model.block_forward(caches, toks, [2] * 4)
    lib.commit(list(range(4)), [2] * 4)
    O.Model.commit(caches, res, [2] * 4)
    for b in range(4):
        L = caches[b].length
        assert lib.cache_len(b) == L
        kx, vx = lib.kv_export(b, L - 2, 2)
        torch.cuda.synchronize()
        for li in range(shape.n_layers):
            parity.kv8_close(host(kx[li]), caches[b].K[li][L - 2:], e, max_frac=0.01, label=f"commit {b} K {li}: ")
            parity.kv8_close(host(vx[li]), caches[b].V[li][L - 2:], e, max_frac=0.01, label=f"commit {b} V {li}: ")
    toks, is_mask = synth.block_rows(9330, shape, 2, 4, n_causal=1)
    got = lib.block_forward([0, 1], toks, is_mask=is_mask).cpu().numpy()
    parity.close(got, model.block_forward(caches[:2], toks, [1, 1]).logits, regress=REGRESS, label="after commit: ")
    lib.set_decode_path("fused")
    with pytest.raises(SbdError, match="UNSUPPORTED"):
        lib.block_forward([0], toks[:1], is_mask=is_mask[:1])
    lib.set_decode_path("auto")
    lib.close()


@pytest.mark.parametrize("family", ["llama", "qwen"])
@pytest.mark.parametrize("weights", ["bf16", "fp8"])
def test_kv8_8b_layer_shape(weights, family):
    """Two layers of the Llama-3.1-8B or Qwen-3-8B shape (head_dim 128; Qwen: per-head q/k
    RMSNorm, ffn 12288), synthetic 700-position cache in e4m3, 16 rows on the per-XCD layer
    kernels and on the per-kernel path, 4 x 8 rows on the GEMM path; also the block step's
    selection."""
    from paper_2509_04185_amd import Sbd
    base = synth.LLAMA8B if family == "llama" else synth.QWEN8B
    shape = dataclasses.replace(base, name=f"{family}8b_2layers", n_layers=2)
    e = 0
    torch.cuda.empty_cache()
    print(f"[gpu] 2-layer {family} 8B shape, {weights} weights, e4m3 KV cache", flush=True)
    if weights == "fp8":
        w = synth.make_weights_fp8(shape, 9400, device="cuda")
    else:
        w = synth.make_weights(shape, 9400, device="cuda")
    lib = Sbd(shape, w, max_batch=4, max_seq_len=1024, max_block=16, kv_format=KV8, kv_scale_exp=e)
    model = O.Model(shape, synth.weights_to_host(w), dtype=np.float32, kv_fp8_exp=e)
    caches = []
    for b in range(4):
        kk, vv = synth.make_kv(shape, 9400, b, 700 - 150 * b, device="cuda")
        lib.kv_import(b, 0, kk, vv)
        caches.append(O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32).to_e4m3(e))
    toks, is_mask = synth.block_rows(9401, shape, 1, 16, n_causal=1)
    ref = model.block_forward(caches[:1], toks, [1]).logits
    paths = [p for p in ("layers", "kernels") if lib.decode_path_fits(p, 1, 16)]
    for p in paths:
        lib.set_decode_path(p)
        got = lib.block_forward([0], toks, is_mask=is_mask, n_causal=[1]).cpu().numpy()
        parity.close(got, ref, regress=REGRESS, label=f"1x16 {p}: ")
        n, pos, tok, H, C, logits = lib.block_step([0], toks, "eb_entropy", 1.0, is_mask=is_mask, n_causal=[1],
                                                   want_logits=True)
        acc, rtok, rH = O.eb_select(logits.cpu().numpy(), is_mask, 1.0, shape.mask_id)
        parity.eb_compare(n, pos, tok, acc, rtok, rH, is_mask, 1.0, label=f"block step {p}: ")
    lib.set_decode_path("auto")
    toks, is_mask = synth.block_rows(9402, shape, 4, 8, n_causal=1)
    got = lib.block_forward([0, 1, 2, 3], toks, is_mask=is_mask, n_causal=[1] * 4).cpu().numpy()
    parity.close(got, model.block_forward(caches, toks, [1] * 4).logits, regress=REGRESS, label="4x8: ")
    lib.close()


@pytest.mark.parametrize("name,sample,weights", [("llama8b_b1_l2048_k16", [0], "fp8"),
                                                 ("llama8b_b4_l32768_k16", [0, 3], "bf16")])
def test_kv8_fullsize(name, sample, weights):
    """The benched configuration with FP8 weights and an e4m3 cache (the paper's timing
    assumption; per-XCD layer kernels), and the batch-4 32768-position configuration with
    an e4m3 cache (64 rows: GEMM, RoPE staging, split attention over 1024 key blocks)."""
    from paper_2509_04185_amd import Sbd
    wl = synth.WORKLOADS[name]
    s = wl.shape
    e = 0
    torch.cuda.empty_cache()
    print(f"[gpu] {name}, {weights} weights, e4m3 KV cache", flush=True)
    w = synth.make_weights_fp8(s, wl.seed, device="cuda") if weights == "fp8" else \
        synth.make_weights(s, wl.seed, device="cuda")
    lens = wl.cache_lens()
    lib = Sbd(s, w, max_batch=wl.batch, max_seq_len=max(lens) + wl.k + 64, max_block=wl.k,
              kv_format=KV8, kv_scale_exp=e)
    for b, L in enumerate(lens):
        kk, vv = synth.make_kv(s, wl.seed, b, L, device="cuda")
        lib.kv_import(b, 0, kk, vv)
        del kk, vv
    toks, is_mask = synth.block_rows(wl.seed, s, wl.batch, wl.k, n_causal=1)
    got = lib.block_forward(list(range(wl.batch)), toks, is_mask=is_mask, n_causal=[1] * wl.batch)
    got = got.cpu().numpy()[sample]
    lib.close()
    model = O.Model(s, synth.weights_to_host(w), dtype=np.float32, cache_decoded=False, kv_fp8_exp=e)
    caches = []
    for b in sample:
        kk, vv = synth.make_kv(s, wl.seed, b, lens[b], device="cuda")
        caches.append(O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32).to_e4m3(e))
        del kk, vv
    print(f"    oracle on sequences {sample}", flush=True)
    ref = model.block_forward(caches, toks[sample], [1] * len(sample)).logits
    parity.close(got, ref, regress=REGRESS, label=f"{name}: ")

"""FP8 (e4m3) weights, the paper's timing assumption (Sec. 4.1: FP8 weights), on the GPU.

Every projection matrix and the LM head are OCP e4m3 bytes with a power-of-two scale per
matrix (synth.make_weights_fp8).  The per-XCD layer kernels, the one-kernel-per-step GEMVs
and the GEMM for more than 16 rows stream the bytes and widen them to bf16 in registers; the
fused path streams a bf16 copy of the same values.  The widening is exact, so:
* an FP8 context gives the same logits, bit for bit, as a bf16 context holding the widened
  values on the one-kernel-per-step and fused paths and the GEMM for more rows (the MFMAs
  see the same operands in the same order); on the per-XCD layer kernels to float rounding
  (the compiler contracts a few multiply-adds differently in the two instantiations);
* against the oracle (which decodes the bytes itself) the contract and regression bounds of
  the bf16 path apply unchanged (the weights are the model; their rounding is not error).
Cases: the tiny decoder on every path, two layers of the Llama-3.1-8B shape on the per-XCD
layer kernels, the benched configuration (32 layers, k = 16, 2048 cached positions) and the
batch-4 32768-position configuration (64 rows: the GEMM for more rows on the e4m3 bytes).
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


def widened(w8):
    """The bf16 weights holding exactly the FP8 model's values."""
    exps = w8["fp8_scale_exp"]
    out = {k: v for k, v in w8.items() if k not in ("layers", "fp8_scale_exp")}
    out["layers"] = []
    for li, lw in enumerate(w8["layers"]):
        lw2 = dict(lw)
        for j, key in enumerate(synth.FP8_KEYS):
            lw2[key] = (lw[key].view(torch.float8_e4m3fn).float() * 2.0 ** exps[li * 7 + j]).to(torch.bfloat16)
        out["layers"].append(lw2)
    out["lm_head"] = (w8["lm_head"].view(torch.float8_e4m3fn).float() * 2.0 ** exps[-1]).to(torch.bfloat16)
    return out


def paths_of(lib, B, k):
    if B * k > 16:
        return ["auto"]
    return [p for p in ("layers", "fused", "kernels") if lib.decode_path_fits(p, B, k)]


def forward_all(lib, paths, seq_ids, toks, is_mask, n_causal):
    out = {}
    for p in paths:
        lib.set_decode_path(p)
        out[p] = lib.block_forward(seq_ids, toks, is_mask=is_mask, n_causal=n_causal).cpu().numpy()
    lib.set_decode_path("auto")
    return out


def test_fp8_tiny_every_path():
    from paper_2509_04185_amd import Sbd
    shape = synth.TINY
    print("[gpu] tiny decoder with FP8 weights", flush=True)
    w8 = synth.make_weights_fp8(shape, 9001, device="cuda")
    wb = widened(w8)
    lib8 = Sbd(shape, w8, max_batch=4, max_seq_len=128, max_block=16)
    libb = Sbd(shape, wb, max_batch=4, max_seq_len=128, max_block=16)
    model = O.Model(shape, synth.weights_to_host(w8), dtype=np.float64, kv_bf16=True)
    prompts = [synth.make_tokens(9002 + b, 20 + 7 * b, shape) for b in range(4)]
    caches = []
    for b, p in enumerate(prompts):
        l8 = lib8.prefill(b, p)
        lb = libb.prefill(b, p)
        cache, ref_last = model.prefill(p)
        caches.append(cache)
        parity.close(l8.cpu().numpy(), ref_last, regress=REGRESS, label=f"prefill {b}: ")
        assert torch.equal(l8, lb), "FP8 prefill differs from the widened bf16 model"
    for B, k in ((1, 4), (2, 8), (4, 8)):           # 32 rows: the GEMM path
        toks, is_mask = synth.block_rows(9010 + B, shape, B, k, n_causal=1)
        paths = paths_of(lib8, B, k)
        g8 = forward_all(lib8, paths, list(range(B)), toks, is_mask, [1] * B)
        gb = forward_all(libb, paths, list(range(B)), toks, is_mask, [1] * B)
        ref = model.block_forward(caches[:B], toks, [1] * B).logits
        for p in paths:
            assert np.array_equal(g8[p], gb[p]), f"{B}x{k} {p}: FP8 differs from the widened bf16 model"
            parity.close(g8[p], ref, regress=REGRESS, label=f"{B}x{k} {p}: ")
        # the staged K/V are not committed: the caches stay the prompts'
    lib8.close()
    libb.close()


@pytest.mark.parametrize("family", ["llama", "qwen"])
def test_fp8_8b_layer_kernels(family):
    """Two layers of the Llama-3.1-8B or Qwen-3-8B shape, 16 rows, synthetic 700-position
    cache: the per-XCD layer kernels streaming e4m3 against the same kernels on the widened
    values and against the oracle; also n_causal = 0 and the block step's statistics."""
    from paper_2509_04185_amd import Sbd
    base = synth.LLAMA8B if family == "llama" else synth.QWEN8B
    shape = dataclasses.replace(base, name=f"{family}8b_2layers", n_layers=2)
    torch.cuda.empty_cache()
    print(f"[gpu] 2-layer {family} 8B shape with FP8 weights", flush=True)
    w8 = synth.make_weights_fp8(shape, 9100, device="cuda")
    lib8 = Sbd(shape, w8, max_batch=1, max_seq_len=1024, max_block=16)
    libb = Sbd(shape, widened(w8), max_batch=1, max_seq_len=1024, max_block=16)
    kk, vv = synth.make_kv(shape, 9100, 0, 700, device="cuda")
    lib8.kv_import(0, 0, kk, vv)
    libb.kv_import(0, 0, kk, vv)
    cache = O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32)
    model = O.Model(shape, synth.weights_to_host(w8), dtype=np.float32, kv_bf16=True)
    if not lib8.decode_path_fits("layers", 1, 16):
        pytest.skip("the per-XCD layer kernels need a device of 256 CUs in 8 XCDs")
    for nc in (1, 0):
        toks, is_mask = synth.block_rows(9101 + nc, shape, 1, 16, n_causal=nc)
        if nc == 0:
            toks[0, 5] = 77
            is_mask[0, 5] = 0
        paths = paths_of(lib8, 1, 16)
        g8 = forward_all(lib8, paths, [0], toks, is_mask, [nc])
        gb = forward_all(libb, paths, [0], toks, is_mask, [nc])
        ref = model.block_forward([cache], toks, [nc]).logits
        for p in paths:
            if p == "layers":
                # the two instantiations of the layer kernels contract different multiply-adds
                # into FMAs (measured: 227 of 229K SwiGLU outputs one bf16 unit apart)
                parity.close(g8[p], gb[p], regress=(1e-4, 1e-5), label=f"n_causal {nc} {p} vs widened: ")
            else:
                assert np.array_equal(g8[p], gb[p]), f"n_causal {nc} {p}: FP8 differs from the widened bf16 model"
            parity.close(g8[p], ref, regress=REGRESS, label=f"n_causal {nc} {p}: ")
    n, pos, tok, H, C, logits = lib8.block_step([0], toks, "eb_entropy", 1.0, is_mask=is_mask, n_causal=[0],
                                                want_logits=True)
    acc, rtok, rH = O.eb_select(logits.cpu().numpy(), is_mask, 1.0, shape.mask_id)
    parity.eb_compare(n, pos, tok, acc, rtok, rH, is_mask, 1.0, label="block step: ")
    lib8.close()
    libb.close()


@pytest.mark.parametrize("name,sample", [("llama8b_b1_l2048_k16", [0]), ("llama8b_b4_l32768_k16", [0, 3])])
def test_fp8_fullsize(name, sample):
    """The benched configuration (per-XCD layer kernels on e4m3) and the batch-4 long-context
    one (64 rows: the GEMM for more rows), on synthetic caches, against the oracle."""
    from paper_2509_04185_amd import Sbd
    wl = synth.WORKLOADS[name]
    s = wl.shape
    torch.cuda.empty_cache()
    print(f"[gpu] {name} with FP8 weights", flush=True)
    w8 = synth.make_weights_fp8(s, wl.seed, device="cuda")
    lens = wl.cache_lens()
    lib = Sbd(s, w8, max_batch=wl.batch, max_seq_len=max(lens) + wl.k + 64, max_block=wl.k)
    for b, L in enumerate(lens):
        kk, vv = synth.make_kv(s, wl.seed, b, L, device="cuda")
        lib.kv_import(b, 0, kk, vv)
        del kk, vv
    toks, is_mask = synth.block_rows(wl.seed, s, wl.batch, wl.k, n_causal=1)
    paths = paths_of(lib, wl.batch, wl.k)
    got = {p: g[sample] for p, g in forward_all(lib, paths, list(range(wl.batch)), toks, is_mask,
                                                 [1] * wl.batch).items()}
    lib.close()
    model = O.Model(s, synth.weights_to_host(w8), dtype=np.float32, cache_decoded=False, kv_bf16=True)
    caches = []
    for b in sample:
        kk, vv = synth.make_kv(s, wl.seed, b, lens[b], device="cuda")
        caches.append(O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32))
        del kk, vv
    print(f"    oracle on sequences {sample}", flush=True)
    ref = model.block_forward(caches, toks[sample], [1] * len(sample)).logits
    for p in paths:
        parity.close(got[p], ref, regress=REGRESS, label=f"{p}: ")

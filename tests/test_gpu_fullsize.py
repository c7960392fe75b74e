"""GPU parity at the full 8B shapes of the four decode workloads.

The GPU runs the whole batch in the launch configuration of each workload; the fp32
oracle recomputes sampled sequences one by one (sequences are independent) from the same
bf16 weights and the same synthetic KV cache, installed on the GPU through sbd_kv_import.
The benchmark's own configuration (Llama-3.1-8B shape, batch 1, 2048-token prompt, k=16)
is also checked end to end with a real prefill on both sides.

Tolerance: max-abs <= 5e-2 and rel-L2 <= 1e-2 on the logits of the compared rows (the
contract), plus a regression bound at about ten times the measured error (synthetic caches:
max-abs 5e-3, rel-L2 6e-4; measured up to 4.9e-4 / 6.2e-5); EB selections bit-exact on
identical fp32 logits, with the decision margins printed (a flip at a margin below 1e-9
would be reported as degenerate).  Sequences compared: every sequence of the batch-4 and
batch-8 workloads, the shortest, the two middle and the longest of the ragged batch-32 one.
"""
import math

import numpy as np
import pytest
import torch

import parity
import synth
from oracle import sbd_oracle as O

pytestmark = pytest.mark.gpu

MAX_ABS, REL_L2 = 5e-2, 1e-2
REGRESS = (5e-3, 6e-4)          # about ten times the error measured on synthetic caches


def close(got, ref, max_abs=MAX_ABS, rel_l2=REL_L2, regress=REGRESS):
    return parity.close(got, ref, regress=regress, max_abs=max_abs, rel_l2=rel_l2)


def eb_bit_exact(lib, logits_np, is_mask, gammas, mask_id):
    for gamma in gammas:
        acc, rtok, rH = O.eb_select(logits_np, is_mask, gamma, mask_id)
        n_acc, pos, tok, H = lib.eb_select(torch.from_numpy(logits_np).cuda(), is_mask, gamma, mask_id)
        parity.eb_compare(n_acc, pos, tok, acc, rtok, rH, is_mask, gamma)
        m = is_mask.astype(bool)
        np.testing.assert_allclose(H.cpu().numpy()[m], rH[m], rtol=1e-12, atol=1e-14)


def make_ctx(wl, import_cache=True):
    from paper_2509_04185_amd import Sbd
    torch.cuda.empty_cache()
    s = wl.shape
    w = synth.make_weights(s, wl.seed, device="cuda")
    lens = wl.cache_lens()
    lib = Sbd(s, w, max_batch=wl.batch, max_seq_len=max(lens) + wl.k + 64, max_block=wl.k)
    if import_cache:
        for b, L in enumerate(lens):
            kk, vv = synth.make_kv(s, wl.seed, b, L, device="cuda")
            lib.kv_import(b, 0, kk, vv)
            del kk, vv
    return w, lib, lens


SAMPLES = {"llama8b_b1_l2048_k16": [0], "llama8b_b32_ragged_k8": "spread",
           "llama8b_b4_l32768_k16": [0, 1, 2, 3], "qwen8b_b8_l8192_k16": list(range(8))}

# Extra decode-sized cases for the per-XCD layer kernels (at most 16 rows): the Qwen-3-8B
# shape (q/k norm, ffn 12288) at batch 1, and two sequences of different lengths in one
# block forward.  Parity cases only, not benchmark workloads.
EXTRA = {
    "qwen8b_b1_l2048_k16": (synth.Workload("qwen8b_b1_l2048_k16", synth.QWEN8B, 1006, 1, 16, (1.0,),
                                           prompt_lens=(2048,)), [0]),
    "llama8b_b2_ragged_k8": (synth.Workload("llama8b_b2_ragged_k8", synth.LLAMA8B, 1007, 2, 8, (0.5,),
                                            prompt_lens=(1500, 700)), [0, 1]),
    # forwards of 32 and 48 rows: the GEMM for more than 16 rows with blocks of 2 and 4 row
    # tiles (48 rows: the last block's fourth tile repeats row 47), activations in fragment order
    "llama8b_b2_l1024_k16": (synth.Workload("llama8b_b2_l1024_k16", synth.LLAMA8B, 1009, 2, 16, (1.0,),
                                            prompt_lens=(1024, 1024)), [1]),
    "llama8b_b3_ragged_k16": (synth.Workload("llama8b_b3_ragged_k16", synth.LLAMA8B, 1010, 3, 16, (1.0,),
                                             prompt_lens=(900, 1600, 300)), [2]),
}


def workload(name):
    return EXTRA[name][0] if name in EXTRA else synth.WORKLOADS[name]


def decode_paths(lib, batch, k):
    """The decode paths a forward of batch x k rows runs on: every one that takes it."""
    if batch * k > 16:
        return ["auto"]
    return [p for p in ("layers", "fused", "kernels") if lib.decode_path_fits(p, batch, k)]


@pytest.mark.parametrize("name", list(SAMPLES) + list(EXTRA))
def test_fullsize_block_forward(name):
    wl = workload(name)
    s = wl.shape
    print(f"[gpu] {name}: B={wl.batch} k={wl.k}", flush=True)
    w, lib, lens = make_ctx(wl)
    sample = EXTRA[name][1] if name in EXTRA else SAMPLES[name]
    if sample == "spread":  # shortest, the two middle and the longest cache
        order = [int(i) for i in np.argsort(lens, kind="stable")]
        sample = sorted({order[0], order[len(order) // 2 - 1], order[len(order) // 2], order[-1]})
    toks, is_mask = synth.block_rows(wl.seed, s, wl.batch, wl.k, n_causal=1)
    # a decode-sized forward (<= 16 rows) is checked on every path that takes it
    paths = decode_paths(lib, wl.batch, wl.k)
    got = {}
    for path in paths:
        lib.set_decode_path(path)
        logits = lib.block_forward(list(range(wl.batch)), toks, is_mask=is_mask)
        n_acc, _, _, _ = lib.eb_select(logits, is_mask, wl.gammas[0], s.mask_id)
        # every path adds its partial sums in a fixed order (or exactly, in integers): the
        # same forward again gives the same bits
        again = lib.block_forward(list(range(wl.batch)), toks, is_mask=is_mask)
        torch.cuda.synchronize()
        assert (n_acc >= 1).all()
        assert torch.equal(logits, again), f"decode path {path} is not reproducible"
        got[path] = logits[sample].cpu().numpy()
        del logits, again
    host = synth.weights_to_host(w)
    model = O.Model(s, host, dtype=np.float32, cache_decoded=False, kv_bf16=True)
    caches = []
    for b in sample:
        kk, vv = synth.make_kv(s, wl.seed, b, lens[b], device="cuda")
        caches.append(O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32))
        del kk, vv
    print(f"    oracle on sequences {sample} (cache {[lens[b] for b in sample]})", flush=True)
    ref = model.block_forward(caches, toks[sample], [1] * len(sample)).logits
    for path in paths:
        print(f"    decode path {path}", flush=True)
        close(got[path], ref)
    eb_bit_exact(lib, ref.astype(np.float32), is_mask[sample], wl.gammas, s.mask_id)


@pytest.mark.parametrize("name", list(SAMPLES))
def test_fullsize_eb_ladder(name):
    """EB at each workload's (batch, k, vocab) on logits that spread the entropies."""
    wl = synth.WORKLOADS[name]
    s = wl.shape
    from paper_2509_04185_amd import Sbd
    import dataclasses
    one = dataclasses.replace(s, n_layers=1)
    torch.cuda.empty_cache()
    w = synth.make_weights(one, wl.seed, device="cuda")
    lib = Sbd(one, w, max_batch=wl.batch, max_seq_len=64, max_block=wl.k)
    logits = synth.entropy_ladder_logits(wl.seed, wl.batch, wl.k, s.vocab).numpy()
    _, is_mask = synth.block_rows(wl.seed, s, wl.batch, wl.k, n_causal=1)
    eb_bit_exact(lib, logits, is_mask, sorted(set(wl.gammas) | {0.0, 1.0, 4.0, math.inf}), s.mask_id)


def test_benched_configuration_with_real_prefill():
    """Llama-3.1-8B shape, batch 1, 2048-token prompt prefilled on both sides, k = 16."""
    wl = synth.WORKLOADS["llama8b_b1_l2048_k16"]
    s = wl.shape
    print("[gpu] benched configuration: prefill 2048 + block forward", flush=True)
    w, lib, lens = make_ctx(wl, import_cache=False)
    prompt = synth.make_tokens(wl.seed, lens[0], s, stream=100)
    last = lib.prefill(0, prompt)
    toks, is_mask = synth.block_rows(wl.seed, s, 1, wl.k, n_causal=1)
    got_paths = {}
    for path in decode_paths(lib, 1, wl.k):
        lib.set_decode_path(path)
        got_paths[path] = lib.block_forward([0], toks, is_mask=is_mask).cpu().numpy()
    logits = lib.block_forward([0], toks, is_mask=is_mask)
    k_gpu, v_gpu = lib.kv_export(0, 0, lens[0])
    torch.cuda.synchronize()
    got, got_last = logits.cpu().numpy(), last.cpu().numpy()
    kl = k_gpu[-1].float().cpu().numpy()
    vl = v_gpu[-1].float().cpu().numpy()
    del k_gpu, v_gpu, logits
    model = O.Model(s, synth.weights_to_host(w), dtype=np.float32, cache_decoded=False, kv_bf16=True)
    print("    oracle prefill of 2048 tokens", flush=True)
    cache, ref_last = model.prefill(prompt)
    # a real prefill on both sides: cache errors add up over 2048 positions (measured rel-L2
    # ~7e-4 on the block logits), so the regression bound is looser here
    real = (5e-2, 7e-3)
    close(got_last, ref_last, regress=real)
    # both caches hold bf16 values; allow a bf16 ulp at magnitude ~8 where roundings differ
    # (last layer after 2048 real positions: measured max-abs 3.1e-2, rel-L2 2.0e-3)
    close(kl, cache.K[-1], max_abs=0.07, regress=(0.07, 6e-3))
    close(vl, cache.V[-1], max_abs=0.07, regress=(0.07, 6e-3))
    ref = model.block_forward([cache], toks, [1]).logits
    close(got, ref, regress=real)
    for path, g in got_paths.items():
        print(f"    decode path {path}", flush=True)
        close(g, ref, regress=real)


def test_layer_kernel_wait_that_gives_up_is_reported():
    """A dependency wait inside the per-XCD layer kernels that gives up - forced from the host
    with a poll limit of 0, so the launch itself stays in bounds and ends - is reported by the
    next call on the context as SBD_ERR_HIP; a fresh context then gives the same logits as
    before.  One layer of the Llama-3.1-8B shape, 128 cached positions, k = 16."""
    import dataclasses
    from paper_2509_04185_amd import Sbd
    from paper_2509_04185_amd.binding import SbdError
    s = dataclasses.replace(synth.LLAMA8B, n_layers=1)
    torch.cuda.empty_cache()
    w = synth.make_weights(s, 1008, device="cuda")

    def fresh_ctx():
        lib = Sbd(s, w, max_batch=1, max_seq_len=256, max_block=16)
        kk, vv = synth.make_kv(s, 1008, 0, 128, device="cuda")
        lib.kv_import(0, 0, kk, vv)
        return lib

    lib = fresh_ctx()
    if not lib.decode_path_fits("layers", 1, 16):
        pytest.skip("the per-XCD layer kernels need a device of 256 CUs in 8 XCDs")
    print("[gpu] layer kernels: forced wait failure", flush=True)
    lib.set_decode_path("layers")
    toks, is_mask = synth.block_rows(1008, s, 1, 16, n_causal=1)
    ref = lib.block_forward([0], toks, is_mask=is_mask)
    torch.cuda.synchronize()
    lib.set_wait_limit(0)
    lib.block_forward([0], toks, is_mask=is_mask)  # its waits give up; the launch still ends
    torch.cuda.synchronize()
    with pytest.raises(SbdError) as err:
        lib.block_forward([0], toks, is_mask=is_mask)
    assert "SBD_ERR_HIP" in str(err.value) and "gave up waiting" in str(err.value), str(err.value)
    del lib
    lib2 = fresh_ctx()
    lib2.set_decode_path("layers")
    got = lib2.block_forward([0], toks, is_mask=is_mask)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)

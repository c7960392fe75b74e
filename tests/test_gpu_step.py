"""sbd_block_step: the block forward with the selection's softmax statistics taken from the
LM head's epilogue (Sec. 2.2, eq. (eb_sampler) needs each masked row's entropy,
confidence and argmax, not its logits), against sbd_block_forward + sbd_select on the same
inputs and against the oracle's selection on those logits.

The step's own stored logits are the reference for its selection: sbd_select on them gives
entropies that agree to float64 summation order (the step merges 64-column chunks,
sbd_select 4096-column ones) and the same accepted rows and tokens, a flip being allowed
only at a decision margin below 1e-9; the oracle's selection on them agrees the same way.
The stored logits equal sbd_block_forward's up to the summation order of the LM head's
launch shape (the step always takes whole 128-column groups in one wave).  Paths: the
decode GEMM (at most 16 rows), the GEMM for more rows, and at the 8B layer shape the
per-XCD layer kernels; the tiny decoder's LM head is scaled by 16 (exact in bf16) so that
the entropies spread and every rule accepts varying numbers of rows.  At the Qwen-3-8B
vocabulary (9496 tiles) the LM head of more than 64 rows ends in a half-full 16-tile block.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import parity
import synth
from oracle import sbd_oracle as O

pytestmark = pytest.mark.gpu

RULES = {"eb_entropy": O.RULE_EB_ENTROPY, "eb_confidence": O.RULE_EB_CONFIDENCE, "factor": O.RULE_FACTOR}
CASES = [("eb_entropy", 0.0), ("eb_entropy", 1.0), ("eb_entropy", math.inf), ("eb_confidence", 1.0),
         ("factor", 2.0)]


def to_dev(w, dev):
    return {k: (v.to(dev) if k != "layers" else [{kk: vv.to(dev) for kk, vv in lw.items()}
                                                 for lw in v]) for k, v in w.items()}


def check_step(lib, shape, seq_ids, toks, is_mask, n_causal, label, logits_optional=True):
    """block_step (with and, where allowed, without logits) against block_forward + select,
    every rule."""
    for rule, thr in CASES:
        fwd_logits = lib.block_forward(seq_ids, toks, is_mask=is_mask, n_causal=n_causal)
        n, p, t, H, C, ref_logits = lib.block_step(seq_ids, toks, rule, thr, is_mask=is_mask, n_causal=n_causal,
                                                   want_logits=True)
        rn, rp, rt, rH, rC = lib.select(ref_logits, is_mask, rule, thr, shape.mask_id)
        if logits_optional:
            n2, p2, t2, H2, C2, none = lib.block_step(seq_ids, toks, rule, thr, is_mask=is_mask, n_causal=n_causal)
            assert none is None
        else:
            n2, p2, t2 = n, p, t
        torch.cuda.synchronize()
        # the LM head of the step may take another launch shape (other summation order)
        parity.close(ref_logits.cpu().numpy(), fwd_logits.cpu().numpy(), regress=(1e-4, 1e-5),
                     label=f"{label} step vs forward logits: ")
        for a, b in ((n, n2), (p, p2), (t, t2)):
            assert torch.equal(a, b), "storing the logits changed the step's selection"
        m = is_mask.astype(bool)
        Hn, rHn = H.cpu().numpy(), rH.cpu().numpy()
        np.testing.assert_allclose(Hn[m], rHn[m], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(C.cpu().numpy()[m], rC.cpu().numpy()[m], rtol=1e-12, atol=1e-15)
        assert np.isnan(Hn[~m]).all()
        # the library's own selection on the stored logits, and the oracle's
        acc, rtok, oH, oC = O.select(ref_logits.cpu().numpy(), is_mask, RULES[rule], thr, shape.mask_id)
        if rule == "eb_entropy":
            parity.eb_compare(n, p, t, acc, rtok, oH, is_mask, thr, label=f"{label} {rule}: ")
            parity.eb_compare(n, p, t, [rp[b, :int(rn[b])].tolist() for b in range(len(acc))],
                              [rt[b, :int(rn[b])].tolist() for b in range(len(acc))], rHn, is_mask, thr,
                              label=f"{label} {rule} vs select: ")
        else:
            for b in range(len(acc)):
                k_ = int(n[b])
                assert p[b, :k_].tolist() == acc[b] and t[b, :k_].tolist() == rtok[b], (label, rule, thr, b)
                assert p[b, :k_].tolist() == rp[b, :int(rn[b])].tolist()
        print(f"    {label} {rule} {thr}: accepted {n.tolist()}", flush=True)


@pytest.fixture(scope="module")
def tiny():
    from paper_2509_04185_amd import Sbd
    shape = synth.TINY
    w = synth.make_weights(shape, 8008)
    w["lm_head"] = (w["lm_head"].float() * 16.0).to(torch.bfloat16)
    print("[gpu] tiny decoder for the block step", flush=True)
    lib = Sbd(shape, to_dev(w, "cuda"), max_batch=40, max_seq_len=128, max_block=16)
    for b in range(8):
        lib.prefill(b, synth.make_tokens(8100 + b, 20 + 3 * b, shape), want_logits=False)
    return shape, lib


@pytest.mark.parametrize("path", ["kernels", "fused"])
def test_block_step_decode_sized(tiny, path):
    shape, lib = tiny
    lib.set_decode_path(path)
    toks, is_mask = synth.block_rows(8200, shape, 2, 8, n_causal=1)
    is_mask[1, 3] = 0
    toks[1, 3] = 17                    # a row revealed by an earlier step
    check_step(lib, shape, [0, 1], toks, is_mask, [1, 0], f"{path} 2x8", logits_optional=path != "fused")
    lib.set_decode_path("auto")


def test_block_step_fused_path_needs_logits(tiny):
    from paper_2509_04185_amd.binding import SbdError
    shape, lib = tiny
    lib.set_decode_path("fused")
    toks, is_mask = synth.block_rows(8201, shape, 1, 4, n_causal=1)
    with pytest.raises(SbdError, match="UNSUPPORTED"):
        lib.block_step([0], toks, "eb_entropy", 1.0, is_mask=is_mask)
    lib.set_decode_path("auto")


def test_block_step_more_than_16_rows(tiny):
    """32 and 48 rows: the LM head on the GEMM for more than 16 rows; every sequence of
    the batch, mixed n_causal, the mask taken from the tokens (is_mask omitted)."""
    shape, lib = tiny
    for B, k in ((4, 8), (3, 16)):
        toks, is_mask = synth.block_rows(8300 + B, shape, B, k, n_causal=2)
        nc = [2] * B
        nc[-1] = 0
        toks[-1, :2] = shape.mask_id
        is_mask = (toks == shape.mask_id).astype(np.uint8)
        check_step(lib, shape, list(range(B)), toks, is_mask, nc, f"{B}x{k}")
        n, p, t, H, C, _ = lib.block_step(list(range(B)), toks, "eb_entropy", 1.0, n_causal=nc)
        n1, p1, t1, H1, C1, _ = lib.block_step(list(range(B)), toks, "eb_entropy", 1.0, is_mask=is_mask, n_causal=nc)
        assert torch.equal(n, n1) and torch.equal(p, p1) and torch.equal(t, t1)


def test_block_step_row_limit(tiny):
    from paper_2509_04185_amd.binding import SbdError
    shape, lib = tiny
    toks, is_mask = synth.block_rows(8400, shape, 40, 16, n_causal=0)
    with pytest.raises(SbdError, match="block step"):
        lib.block_step(list(range(40)), toks, "eb_entropy", 1.0, is_mask=is_mask, n_causal=[0] * 40)


def test_block_step_8b_layer_shape():
    """Two layers of the Llama-3.1-8B shape, full vocabulary (2004 chunks per row): the
    per-XCD layer kernels (16 rows) and the GEMM path (4 x 8 rows)."""
    from paper_2509_04185_amd import Sbd
    shape = dataclasses.replace(synth.LLAMA8B, name="llama8b_2layers", n_layers=2)
    torch.cuda.empty_cache()
    print("[gpu] 2-layer 8B shape for the block step", flush=True)
    w = synth.make_weights(shape, 8500, device="cuda")
    lib = Sbd(shape, w, max_batch=4, max_seq_len=1024, max_block=16)
    for b in range(4):
        kk, vv = synth.make_kv(shape, 8500, b, 300 + 100 * b, device="cuda")
        lib.kv_import(b, 0, kk, vv)
    toks, is_mask = synth.block_rows(8501, shape, 1, 16, n_causal=1)
    paths = [p for p in ("layers", "kernels") if lib.decode_path_fits(p, 1, 16)]
    for path in paths:
        lib.set_decode_path(path)
        check_step(lib, shape, [0], toks, is_mask, [1], f"8B {path} 1x16")
    lib.set_decode_path("auto")
    toks, is_mask = synth.block_rows(8502, shape, 4, 8, n_causal=1)
    check_step(lib, shape, [0, 1, 2, 3], toks, is_mask, [1] * 4, "8B 4x8")
    lib.close()


def test_block_step_qwen_vocab_half_block():
    """Two layers of the Qwen-3-8B shape, 8 x 16 rows on the GEMM path: its 9496 vocabulary
    tiles (8 mod 16) run as 16-tile blocks, the last one half full, both in the LM head that
    stores logits and in the one that hands the EB statistics to the selection (the last 128
    columns come from that block)."""
    from paper_2509_04185_amd import Sbd
    shape = dataclasses.replace(synth.QWEN8B, name="qwen8b_2layers", n_layers=2)
    torch.cuda.empty_cache()
    print("[gpu] 2-layer Qwen 8B shape for the block step (half-full last LM-head block)", flush=True)
    w = synth.make_weights(shape, 8600, device="cuda")
    lib = Sbd(shape, w, max_batch=8, max_seq_len=512, max_block=16)
    for b in range(8):
        kk, vv = synth.make_kv(shape, 8600, b, 100 + 37 * b, device="cuda")
        lib.kv_import(b, 0, kk, vv)
    toks, is_mask = synth.block_rows(8601, shape, 8, 16, n_causal=1)
    check_step(lib, shape, list(range(8)), toks, is_mask, [1] * 8, "Qwen 8x16")
    lib.close()

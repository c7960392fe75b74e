"""GPU parity of the per-XCD layer kernels (the decode path the library picks for every
forward of at most 16 rows at the 8B shapes) in the states the Alg. 3 loop puts them in.

A 2-layer decoder of the real Llama-3.1-8B layer shape (d 4096, 32/8 heads, d_h 128,
F 14336, full vocabulary) runs on the GPU; the fp32 oracle computes the same forwards from
the same bf16 weights and caches.  Cases:
* n_causal = 0: every iteration of Alg. 3 after a block's first feeds the block alone,
  each row seeing every other (App. A mask with the causal point at the cache end);
* a batch whose sequences carry different n_causal and cache lengths;
* an empty cache (no prompt), n_causal 1 and 0;
* blocks of 1, 2 and 5 rows (k = 1: the next-token forward of the speedup model);
* permuted positions: moving the prediction rows together with their pos_ids permutes
  their logits (the block is bidirectional, Fig. 3);
* n_causal = 2 after a real prefill: the cached block equals a full recompute without a
  cache under the App. A mask (exact KV caching, Sec. 1), and the committed rows hold the
  recompute's K/V;
* the generation loop of Alg. 2 / Alg. 3 for two blocks of 16: the first forward of the
  second block carries 32 rows (previous block causal) and runs on the GEMM path for more
  than 16 rows, every later forward on the layer kernels.  The oracle replays every step on
  the tokens the GPU fed; selections and tokens must agree unless the oracle's own margin
  for that decision is within the measured error (reported as degenerate).
Bounds: the contract (max-abs 5e-2, rel-L2 1e-2) and a regression bound of max-abs 5e-3,
rel-L2 6e-4 (about ten times the error measured at these shapes).
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

REGRESS = (5e-3, 6e-4)
SHAPE = dataclasses.replace(synth.LLAMA8B, name="llama8b_2layers", n_layers=2)
SEED = 1101


class Setup:
    def __init__(self):
        from paper_2509_04185_amd import Sbd
        torch.cuda.empty_cache()
        print(f"[gpu] building {SHAPE.name}", flush=True)
        self.w = synth.make_weights(SHAPE, SEED, device="cuda")
        self.lib = Sbd(SHAPE, self.w, max_batch=2, max_seq_len=2048, max_block=32)
        self.model = O.Model(SHAPE, synth.weights_to_host(self.w), dtype=np.float32, kv_bf16=True)

    def install(self, seq, n, stream=0):
        """Synthetic cache of n positions in slot seq on both sides."""
        kk, vv = synth.make_kv(SHAPE, SEED + stream, seq, n, device="cuda")
        self.lib.reset(seq)
        self.lib.kv_import(seq, 0, kk, vv)
        return O.SeqCache.from_arrays(synth.to_host_bits(kk), synth.to_host_bits(vv), np.float32)

    def paths(self, batch, k):
        return [p for p in ("layers", "fused", "kernels") if self.lib.decode_path_fits(p, batch, k)]


@pytest.fixture(scope="module")
def setup():
    s = Setup()
    if not s.lib.decode_path_fits("layers", 1, 16):
        pytest.skip("the per-XCD layer kernels need a device of 256 CUs in 8 XCDs")
    yield s
    s.lib.close()


def revealed_block(seed, k, n_causal, frac_revealed):
    """Block rows of one sequence as Alg. 3 leaves them: n_causal real rows, then a
    prediction block in which some rows were already revealed by earlier steps."""
    rng = np.random.default_rng(seed)
    toks = synth.make_tokens(seed, k, SHAPE, stream=3).astype(np.int32)
    pred = np.arange(k) >= n_causal
    masked = pred & (rng.random(k) >= frac_revealed)
    if pred.any() and not masked.any():
        masked[np.nonzero(pred)[0][-1]] = True
    toks[masked] = SHAPE.mask_id
    return toks, masked.astype(np.uint8)


def run_paths(setup, seq_ids, toks, is_mask, n_causal, pos=None):
    out = {}
    for path in setup.paths(len(seq_ids), toks.shape[1]):
        setup.lib.set_decode_path(path)
        out[path] = setup.lib.block_forward(seq_ids, toks, is_mask=is_mask, n_causal=n_causal,
                                            pos_ids=pos).cpu().numpy()
    setup.lib.set_decode_path("auto")
    return out


def test_n_causal_zero_on_layer_kernels(setup):
    """Alg. 3 after a block's first iteration: the block alone, all rows bidirectional."""
    cache = setup.install(0, 700)
    toks, is_mask = revealed_block(11, 16, 0, 0.4)
    got = run_paths(setup, [0], toks[None], is_mask[None], [0])
    assert "layers" in got
    ref = setup.model.block_forward([cache], toks[None], [0]).logits
    for path, g in got.items():
        parity.close(g, ref, regress=REGRESS, label=f"{path}: ")


def test_mixed_n_causal_batch_on_layer_kernels(setup):
    """Two sequences of different cache lengths in one forward, n_causal 0 and 3 (k = 8)."""
    caches = [setup.install(0, 1500, stream=1), setup.install(1, 333, stream=1)]
    t0, m0 = revealed_block(21, 8, 0, 0.3)
    t1, m1 = revealed_block(22, 8, 3, 0.3)
    toks, is_mask = np.stack([t0, t1]), np.stack([m0, m1])
    got = run_paths(setup, [0, 1], toks, is_mask, [0, 3])
    assert "layers" in got
    ref = setup.model.block_forward(caches, toks, [0, 3]).logits
    for path, g in got.items():
        parity.close(g, ref, regress=REGRESS, label=f"{path}: ")


def test_empty_cache_on_layer_kernels(setup):
    """Nothing cached (a sequence without a prompt): 31 of each XCD's 32 attention tasks get
    an empty key range and the merge takes the one that holds the block; n_causal 1 and 0."""
    for nc in (1, 0):
        setup.lib.reset(0)
        toks, is_mask = revealed_block(41 + nc, 16, nc, 0.2)
        got = run_paths(setup, [0], toks[None], is_mask[None], [nc])
        assert "layers" in got
        ref = setup.model.block_forward([setup.model.new_cache()], toks[None], [nc]).logits
        for path, g in got.items():
            parity.close(g, ref, regress=REGRESS, label=f"{path}, n_causal {nc}: ")


@pytest.mark.parametrize("k", [1, 2, 5])
def test_small_blocks_on_layer_kernels(setup, k):
    """The small blocks the speedup model times (k = 1 is the next-token forward, Sec. 4.2):
    one causal row, then k - 1 masks, on a 1000-position cache."""
    cache = setup.install(0, 1000, stream=4)
    toks, is_mask = revealed_block(50 + k, k, 1, 0.0)
    got = run_paths(setup, [0], toks[None], is_mask[None], [1])
    assert "layers" in got
    ref = setup.model.block_forward([cache], toks[None], [1]).logits
    for path, g in got.items():
        parity.close(g, ref, regress=REGRESS, label=f"{path}, k {k}: ")


def test_permuted_positions_on_layer_kernels(setup):
    """Prediction rows moved together with their pos_ids: their logits move with them."""
    cache = setup.install(0, 900, stream=2)
    L = 900
    toks, is_mask = revealed_block(31, 16, 1, 0.3)
    perm = np.concatenate([[0], 1 + np.random.default_rng(32).permutation(15)])
    pos = L + np.arange(16)
    tp, mp, pp = toks[perm], is_mask[perm], pos[perm]
    setup.lib.set_decode_path("layers")
    base = setup.lib.block_forward([0], toks[None], is_mask=is_mask[None], n_causal=[1]).cpu().numpy()
    moved = setup.lib.block_forward([0], tp[None], is_mask=mp[None], n_causal=[1],
                                    pos_ids=pp[None]).cpu().numpy()
    setup.lib.set_decode_path("auto")
    ref = setup.model.block_forward([cache], tp[None], [1], pos=pp[None]).logits
    parity.close(moved, ref, regress=REGRESS, label="layers, permuted: ")
    # the GPU's own two forwards: the same rows up to the summation order of the block keys
    parity.close(moved[0], base[0][perm], regress=(2e-3, 2e-4), label="permuted vs unpermuted: ")


def test_cached_block_equals_full_recompute_after_prefill(setup):
    """n_causal = 2 after a real 300-token prefill; logits equal the oracle's full recompute
    over prompt + block with the App. A mask, and commit(2) leaves the recompute's K/V."""
    lib, model = setup.lib, setup.model
    P = 300
    prompt = synth.make_tokens(41, P, SHAPE, stream=4)
    lib.reset(0)
    lib.prefill(0, prompt, want_logits=False)
    toks, is_mask = revealed_block(42, 16, 2, 0.25)
    got = run_paths(setup, [0], toks[None], is_mask[None], [2])
    assert "layers" in got
    full_toks = np.concatenate([prompt, toks])
    print("    oracle full recompute of 316 rows", flush=True)
    ref = model.full_forward(full_toks, causal_point=P + 2)[P:]
    for path, g in got.items():
        parity.close(g[0], ref, regress=(5e-3, 1e-3), label=f"{path}: ")
    # commit the two causal rows of the last forward (the auto path's): the cache now holds
    # the K/V of prompt + 2 tokens, which a prefill of those tokens gives too
    setup.lib.block_forward([0], toks[None], is_mask=is_mask[None], n_causal=[2])
    lib.commit([0], [2])
    assert lib.cache_len(0) == P + 2
    kk, vv = lib.kv_export(0, P, 2)
    cache, _ = model.prefill(full_toks[:P + 2])
    for li in range(SHAPE.n_layers):
        parity.close(kk[li].float().cpu().numpy(), cache.K[li][P:P + 2], max_abs=0.07, regress=(0.07, 4e-3),
                     label=f"K layer {li}: ")
        parity.close(vv[li].float().cpu().numpy(), cache.V[li][P:P + 2], max_abs=0.07, regress=(0.07, 4e-3),
                     label=f"V layer {li}: ")


class Recorder:
    """The library with its block forwards' logits and the selections' entropies kept, for
    the step-by-step replay (attribute access goes to the library)."""

    def __init__(self, lib):
        self._lib = lib
        self.logits = None
        self.H = None

    def __getattr__(self, name):
        return getattr(self._lib, name)

    def block_forward(self, *a, **kw):
        self.logits = self._lib.block_forward(*a, **kw)
        return self.logits

    def select(self, *a, **kw):
        out = self._lib.select(*a, **kw)
        self.H = out[3]
        return out


def test_generation_loop_two_blocks_of_16(setup):
    from paper_2509_04185_amd import sample_blocks
    lib, model = setup.lib, setup.model
    k, gamma = 16, 1.0
    prompt = synth.make_tokens(51, 200, SHAPE, stream=5)
    lib.reset(0)
    lib.prefill(0, prompt, want_logits=False)
    cache, _ = model.prefill(prompt)
    rec = Recorder(lib)
    steps = []

    def on_forward(toks, nc, n_acc, pos, tok):
        # the oracle takes the same step on the same fed rows, from its own cache
        res = model.block_forward([cache], toks, [nc])
        if nc:
            O.Model.commit([cache], res, [nc])
        rows = res.logits[:, nc:]
        is_mask = (toks[:, nc:] == SHAPE.mask_id).astype(np.uint8)
        acc, rtok, rH = O.eb_select(rows, is_mask, gamma, SHAPE.mask_id)
        err, _ = parity.close(rec.logits.cpu().numpy(), res.logits, regress=REGRESS,
                              label=f"step {len(steps)} ({toks.shape[1]} rows): ")
        gH = rec.H.cpu().numpy()[:, nc:]    # the selection ran over all fed rows
        m = is_mask.astype(bool)
        h_err = float(np.abs(gH[m] - rH[m]).max())
        n = int(n_acc[0])
        got_rows = (pos[0, :n] - nc).tolist()
        got_tok = tok[0, :n].tolist()
        if got_rows != acc[0] or got_tok != rtok[0]:
            # allowed only where the oracle's decision is within the measured error
            rws = [j for j in range(k) if m[0, j]]
            h_margin = parity.eb_margin(rH[0], rws, gamma, len(acc[0]))
            cand = rows[0][acc[0]].copy()
            cand[:, SHAPE.mask_id] = -np.inf
            tops = np.sort(cand, axis=-1)[:, -2:]
            t_margin = float((tops[:, 1] - tops[:, 0]).min())
            assert h_margin < 20 * h_err or t_margin < 20 * err, \
                (len(steps), got_rows, acc[0], got_tok, rtok[0], h_margin, h_err, t_margin, err)
            print(f"    step {len(steps)}: degenerate decision (entropy margin {h_margin:.2e}, "
                  f"token margin {t_margin:.2e})", flush=True)
        steps.append((toks.shape[1], nc))

    out = sample_blocks(rec, [0], 2, k, "eb_entropy", gamma, on_forward=on_forward)
    print(f"    {len(steps)} forwards: {steps}", flush=True)
    assert steps[0] == (16, 0)
    second = [i for i, (rows, nc) in enumerate(steps) if nc == k]
    assert len(second) == 1 and steps[second[0]][0] == 2 * k      # the 32-row forward
    assert all(rows == k for i, (rows, nc) in enumerate(steps) if i != second[0])
    assert len(out[0]) == 2 * k and SHAPE.mask_id not in out[0]
    assert lib.cache_len(0) == 200 + k
    # the committed first block equals the oracle's cache, which followed the GPU's tokens
    kk, vv = lib.kv_export(0, 200, k)
    for li in range(SHAPE.n_layers):
        parity.close(kk[li].float().cpu().numpy(), cache.K[li][200:], max_abs=0.07, regress=(0.07, 4e-3),
                     label=f"K layer {li}: ")
        parity.close(vv[li].float().cpu().numpy(), cache.V[li][200:], max_abs=0.07, regress=(0.07, 4e-3),
                     label=f"V layer {li}: ")


def test_xcd_placement_probe(setup):
    """The probe at context creation found workgroup i on XCD i % 8 (the placement the layer
    kernels and the split GEMMs hand partials off under), so AUTO takes the layer kernels."""
    assert setup.lib.xcd_map_ok()
    assert setup.lib.decode_path_fits("layers", 1, 16)

"""GPU parity of the HIP path against the CPU oracle on the tiny decoder (and its qk-norm
variant), plus the SBD invariants and the ABI's state machine on the device.

Tolerance for logits (bf16 weights/activations on the GPU vs the float64 oracle on the
same bf16 weights): max-abs <= 5e-2 and rel-L2 <= 1e-2 over the whole logits tensor.
"""
import math
import sys

import numpy as np
import pytest
import torch

import parity
import synth
from oracle import sbd_oracle as O

pytestmark = pytest.mark.gpu

MAX_ABS, REL_L2 = 5e-2, 1e-2


def close(got, ref, max_abs=MAX_ABS, rel_l2=REL_L2):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref).max()
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    print(f"    max-abs {err:.3e}  rel-L2 {rel:.3e}", flush=True)
    assert err <= max_abs and rel <= rel_l2, f"max-abs {err:.3e} rel-L2 {rel:.3e}"
    return err, rel


def to_dev(w, dev):
    return {k: (v.to(dev) if k != "layers" else [{kk: vv.to(dev) for kk, vv in lw.items()}
                                                 for lw in v]) for k, v in w.items()}


class Tiny:
    def __init__(self, shape, seed, max_batch=4, max_seq_len=256, max_block=16, chunk=0, path="auto"):
        from paper_2509_04185_amd import Sbd
        print(f"[gpu] building {shape.name} seed={seed} batch={max_batch} decode path {path}", flush=True)
        self.shape = shape
        self.path = path
        self.w_cpu = synth.make_weights(shape, seed)
        self.lib = Sbd(shape, to_dev(self.w_cpu, "cuda"), max_batch=max_batch,
                       max_seq_len=max_seq_len, max_block=max_block, prefill_chunk=chunk)
        self.lib.set_decode_path(path)
        # The KV cache stores bf16: the oracle rounds K/V the same way (activations stay fp64).
        self.model = O.Model(shape, synth.weights_to_host(self.w_cpu), dtype=np.float64, kv_bf16=True)


# Decode-sized forwards (<= 16 rows) run either as the fused single launch or as one kernel
# per step; every forward test runs on both.  "fused" makes a forward the fused launch cannot
# take an error, so these tests cannot pass on the other path by accident.
PATHS = ["fused", "kernels"]


@pytest.fixture(scope="module", params=PATHS)
def tiny(request):
    return Tiny(synth.TINY, 1001, path=request.param)


@pytest.fixture(scope="module", params=PATHS)
def tiny_qk(request):
    return Tiny(synth.TINY_QK, 2002, chunk=24, path=request.param)


def fresh(t, seqs=(0, 1, 2, 3)):
    for s in seqs:
        t.lib.reset(s)


# ------------------------------------------------------------------ the tiny workload


def test_tiny_workload_block_forward(tiny):
    """Batch 1, 64-token prompt in the cache, k = 4 (1 real + 3 masks)."""
    wl = synth.WORKLOADS["tiny_b1_l64_k4"]
    fresh(tiny)
    prompt = synth.make_tokens(wl.seed, 64, tiny.shape)
    last = tiny.lib.prefill(0, prompt)
    toks, is_mask = synth.block_rows(wl.seed, tiny.shape, 1, 4, n_causal=1)
    logits = tiny.lib.block_forward([0], toks, is_mask=is_mask)
    torch.cuda.synchronize()
    cache, ref_last = tiny.model.prefill(prompt)
    ref = tiny.model.block_forward([cache], toks, [1]).logits
    close(last.cpu().numpy(), ref_last)
    close(logits.cpu().numpy(), ref)
    assert tiny.lib.cache_len(0) == 64


@pytest.mark.parametrize("gamma", [0.0, 0.5, math.inf])
def test_tiny_workload_eb_select_bit_exact(tiny, gamma):
    """EB on the oracle's own fp32 logits (x4): identical accepted set and tokens."""
    wl = synth.WORKLOADS["tiny_b1_l64_k4"]
    prompt = synth.make_tokens(wl.seed, 64, tiny.shape)
    cache, _ = tiny.model.prefill(prompt)
    toks, is_mask = synth.block_rows(wl.seed, tiny.shape, 1, 4, n_causal=1)
    ref_logits = (tiny.model.block_forward([cache], toks, [1]).logits * wl.logit_scale).astype(np.float32)
    acc, rtok, rH = O.eb_select(ref_logits, is_mask, gamma, tiny.shape.mask_id)
    n_acc, pos, tok, H = tiny.lib.eb_select(torch.from_numpy(ref_logits).cuda(), is_mask, gamma,
                                            tiny.shape.mask_id)
    parity.eb_compare(n_acc, pos, tok, acc, rtok, rH, is_mask, gamma)
    Hg = H.cpu().numpy()
    for j in range(4):
        if is_mask[0, j]:
            assert abs(Hg[0, j] - rH[0, j]) <= 1e-12 * max(1.0, abs(rH[0, j]))
        else:
            assert math.isnan(Hg[0, j])


# ------------------------------------------------------------------ EB on ladder logits


@pytest.fixture(scope="module")
def wide():
    """A context whose vocabulary and block size cover the EB cases (one layer suffices)."""
    import dataclasses
    shape = dataclasses.replace(synth.TINY, name="tiny_v16k", vocab=16384, mask_id=16383, n_layers=1)
    return Tiny(shape, 3003, max_batch=4, max_seq_len=64, max_block=64)


@pytest.mark.parametrize("B,k,V,mask_id", [(1, 16, 1024, 1023), (3, 8, 4096, 0), (2, 5, 5000, -1),
                                           (4, 16, 12000, 11999), (1, 64, 2048, 7),
                                           (2, 64, 16384, 16383), (3, 9, 4097, 4096)])
def test_eb_select_ladder_bit_exact(wide, B, k, V, mask_id):
    """EB on entropy-ladder logits: identical accepted sets and tokens at every gamma."""
    logits = synth.entropy_ladder_logits(B * 100 + k, B, k, V)
    rng = np.random.default_rng(B * 7 + k)
    is_mask = (rng.random((B, k)) < 0.8).astype(np.uint8)
    is_mask[:, 0] = 0
    if k > 1:
        is_mask[:, 1] = 1
    for gamma in (0.0, 0.1, 1.0, 4.0, math.inf):
        acc, rtok, rH = O.eb_select(logits.numpy(), is_mask, gamma, mask_id)
        n_acc, pos, tok, H = wide.lib.eb_select(logits.cuda(), is_mask, gamma, mask_id)
        parity.eb_compare(n_acc, pos, tok, acc, rtok, rH, is_mask, gamma)
        Hg = H.cpu().numpy()
        m = is_mask.astype(bool)
        np.testing.assert_allclose(Hg[m], rH[m], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("B,k,V,mask_id", [(1, 16, 1024, 1023), (3, 8, 4096, 0), (2, 64, 16384, 16383),
                                           (3, 9, 4097, 4096)])
def test_select_rules_ladder_bit_exact(wide, B, k, V, mask_id):
    """The App. B rules (EB with the confidence proxy, Factor) on ladder logits: identical
    accepted sets and tokens; confidences to float64 rounding; the entropy rule through
    sbd_select equals sbd_eb_select."""
    logits = synth.entropy_ladder_logits(B * 100 + k + 1, B, k, V)
    rng = np.random.default_rng(B * 11 + k)
    is_mask = (rng.random((B, k)) < 0.8).astype(np.uint8)
    is_mask[:, 0] = 0
    if k > 1:
        is_mask[:, 1] = 1
    m = is_mask.astype(bool)
    cases = [("eb_confidence", O.RULE_EB_CONFIDENCE, g) for g in (0.0, 0.1, 1.0, 4.0, math.inf)]
    cases += [("factor", O.RULE_FACTOR, f) for f in (0.0, 0.05, 0.5, 2.0, 8.0, math.inf)]
    cases += [("eb_entropy", O.RULE_EB_ENTROPY, 1.0)]
    for name, rule, thr in cases:
        acc, rtok, rH, rC = O.select(logits.numpy(), is_mask, rule, thr, mask_id)
        n_acc, pos, tok, H, C = wide.lib.select(logits.cuda(), is_mask, name, thr, mask_id)
        for b in range(B):
            n = int(n_acc[b])
            assert pos[b, :n].tolist() == acc[b], (name, thr, b)
            assert tok[b, :n].tolist() == rtok[b], (name, thr, b)
            assert (pos[b, n:] == -1).all()
        np.testing.assert_allclose(H.cpu().numpy()[m], rH[m], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(C.cpu().numpy()[m], rC[m], rtol=1e-12, atol=1e-15)
        assert np.isnan(C.cpu().numpy()[~m]).all()
    n1, p1, t1, _ = wide.lib.eb_select(logits.cuda(), is_mask, 1.0, mask_id)
    n2, p2, t2, _, _ = wide.lib.select(logits.cuda(), is_mask, "eb_entropy", 1.0, mask_id)
    assert torch.equal(n1, n2) and torch.equal(p1, p2) and torch.equal(t1, t2)


@pytest.mark.parametrize("name,rule", [("eb_entropy", O.RULE_EB_ENTROPY),
                                       ("eb_confidence", O.RULE_EB_CONFIDENCE),
                                       ("factor", O.RULE_FACTOR)])
def test_select_sequences_with_no_or_one_masked_row(wide, name, rule):
    """Degenerate masked sets: a sequence with no masked row accepts nothing (n = 0, every
    slot -1) at any threshold; one with a single masked row accepts it at every threshold,
    0 included (the rule keeps at least one row); a full sequence beside them as usual."""
    B, k, V, mask_id = 3, 16, 4096, 4095
    logits = synth.entropy_ladder_logits(78, B, k, V)
    is_mask = np.zeros((B, k), np.uint8)
    is_mask[1, 9] = 1
    is_mask[2, 1:] = 1
    m = is_mask.astype(bool)
    for thr in (0.0, 1.0, math.inf):
        acc, rtok, rH, rC = O.select(logits.numpy(), is_mask, rule, thr, mask_id)
        assert acc[0] == [] and acc[1] == [9]
        n_acc, pos, tok, H, C = wide.lib.select(logits.cuda(), is_mask, name, thr, mask_id)
        for b in range(B):
            n = int(n_acc[b])
            assert pos[b, :n].tolist() == acc[b], (name, thr, b)
            assert tok[b, :n].tolist() == rtok[b], (name, thr, b)
            assert (pos[b, n:] == -1).all()
        assert int(n_acc[0]) == 0 and int(n_acc[1]) == 1
        np.testing.assert_allclose(H.cpu().numpy()[m], rH[m], rtol=1e-12, atol=1e-13)
        assert np.isnan(H.cpu().numpy()[~m]).all()


@pytest.mark.parametrize("name,rule,thr", [("eb_entropy", O.RULE_EB_ENTROPY, 0.5),
                                           ("eb_entropy", O.RULE_EB_ENTROPY, math.inf),
                                           ("eb_confidence", O.RULE_EB_CONFIDENCE, 1.0),
                                           ("eb_confidence", O.RULE_EB_CONFIDENCE, math.inf),
                                           ("factor", O.RULE_FACTOR, 2.0),
                                           ("factor", O.RULE_FACTOR, math.inf)])
def test_select_rows_with_undefined_softmax(wide, name, rule, thr):
    """Masked rows whose softmax is undefined: all -inf outside the mask column (vocabulary
    of three chunks), a NaN logit, an infinite logit.  Their entropy and confidence are NaN,
    they are never accepted (not even at an infinite threshold), and the other rows are
    selected as the oracle selects them; a sequence whose only masked rows are such rows
    accepts nothing."""
    B, k, V, mask_id = 3, 8, 9000, 8999
    logits = synth.entropy_ladder_logits(77, B, k, V)
    logits[0, 3, :] = -math.inf
    logits[0, 3, mask_id] = 5.0  # the excluded column is finite, and must stay excluded
    logits[0, 5, 4321] = math.nan
    logits[1, 2, 8000] = math.inf
    logits[2, 1, :] = -math.inf
    is_mask = np.ones((B, k), np.uint8)
    is_mask[:, 0] = 0
    is_mask[2, 2:] = 0             # sequence 2: its only masked row has no finite logit
    m = is_mask.astype(bool)
    bad = np.zeros((B, k), bool)
    bad[0, 3] = bad[0, 5] = bad[1, 2] = bad[2, 1] = True
    n_acc, pos, tok, H, C = wide.lib.select(logits.cuda(), is_mask, name, thr, mask_id)
    H, C = H.cpu().numpy(), C.cpu().numpy()
    assert np.isnan(H[bad]).all() and np.isnan(C[bad]).all()
    with np.errstate(invalid="ignore"):
        acc, rtok, rH, rC = O.select(logits.numpy(), is_mask, rule, thr, mask_id)
    ok = m & ~bad
    np.testing.assert_allclose(H[ok], rH[ok], rtol=1e-12, atol=1e-13)
    for b in range(B):
        n = int(n_acc[b])
        assert pos[b, :n].tolist() == acc[b], (b, name, thr)
        assert tok[b, :n].tolist() == rtok[b], (b, name, thr)
        assert not any(bad[b, j] for j in acc[b])
        assert (pos[b, n:] == -1).all()
    assert int(n_acc[2]) == 0
    if thr == math.inf:
        assert sorted(acc[0]) == [j for j in range(k) if ok[0, j]]


def test_eb_select_many_rows_mask_upload():
    """More rows than the masks passed by value (2048): the mask goes through the stream
    upload instead; same accepted sets and tokens as the oracle."""
    import dataclasses
    shape = dataclasses.replace(synth.TINY, name="tiny_b40", n_layers=1)
    t = Tiny(shape, 4004, max_batch=40, max_seq_len=64, max_block=64)
    B, k, V, mask_id = 40, 64, shape.vocab, shape.mask_id
    logits = synth.entropy_ladder_logits(4040, B, k, V)
    rng = np.random.default_rng(4041)
    is_mask = (rng.random((B, k)) < 0.7).astype(np.uint8)
    is_mask[:, 0] = 0
    is_mask[:, 1] = 1
    for gamma in (0.5, math.inf):
        acc, rtok, rH = O.eb_select(logits.numpy(), is_mask, gamma, mask_id)
        n_acc, pos, tok, H = t.lib.eb_select(logits.cuda(), is_mask, gamma, mask_id)
        for b in range(B):
            n = int(n_acc[b])
            assert pos[b, :n].tolist() == acc[b], (b, gamma)
            assert tok[b, :n].tolist() == rtok[b], (b, gamma)
        m = is_mask.astype(bool)
        np.testing.assert_allclose(H.cpu().numpy()[m], rH[m], rtol=1e-12, atol=1e-13)


def test_eb_select_entropies_hand_cases(tiny):
    H = torch.tensor([[0.0, 0.25, 0.125, 0.375, 0.125]], dtype=torch.float64, device="cuda")
    is_mask = np.array([[0, 1, 1, 1, 1]], np.uint8)
    for gamma, want in ((0.0, [2]), (0.125, [2, 4]), (0.25, [1, 2, 4]), (0.4999, [1, 2, 4]),
                        (0.5, [1, 2, 3, 4]), (math.inf, [1, 2, 3, 4])):
        n, pos = tiny.lib.eb_select_entropies(H, is_mask, gamma)
        assert pos[0, :int(n[0])].tolist() == want
    n, pos = tiny.lib.eb_select_entropies(H, np.zeros((1, 5), np.uint8), 1.0)
    assert int(n[0]) == 0 and (pos == -1).all()


# ------------------------------------------------------------------ SBD invariants on the GPU


def test_k1_is_next_token_prediction(tiny):
    fresh(tiny)
    prompt = synth.make_tokens(5, 40, tiny.shape)
    tiny.lib.prefill(0, prompt[:-1], want_logits=False)
    got = tiny.lib.block_forward([0], prompt[-1:].reshape(1, 1))
    tiny.lib.prefill(1, prompt)
    last = tiny.lib.prefill(2, prompt)
    torch.cuda.synchronize()
    ntp = tiny.model.full_forward(prompt, causal_point=len(prompt))[-1]
    close(got[0, 0].cpu().numpy(), ntp)
    close(last.cpu().numpy(), ntp)


def test_row0_independent_of_prediction_rows(tiny):
    fresh(tiny)
    tiny.lib.prefill(0, synth.make_tokens(6, 30, tiny.shape), want_logits=False)
    toks, _ = synth.block_rows(7, tiny.shape, 1, 6, n_causal=1)
    a = tiny.lib.block_forward([0], toks).clone()
    toks2 = toks.copy()
    toks2[0, 3] = 11
    b = tiny.lib.block_forward([0], toks2)
    torch.cuda.synchronize()
    assert torch.equal(a[0, 0], b[0, 0])
    assert (a[0, 1] - b[0, 1]).abs().max() > 1e-4


def test_prediction_rows_permutation_equivariant(tiny_qk):
    t = tiny_qk
    fresh(t)
    t.lib.prefill(0, synth.make_tokens(8, 33, t.shape), want_logits=False)
    L = t.lib.cache_len(0)
    toks = np.array([[3, 77, t.shape.mask_id, 500, t.shape.mask_id, 9]], np.int32)
    pos = np.array([[L + j for j in range(6)]], np.int32)
    perm = [0, 4, 1, 5, 3, 2]
    a = t.lib.block_forward([0], toks, pos_ids=pos).clone()
    b = t.lib.block_forward([0], toks[:, perm], pos_ids=pos[:, perm])
    torch.cuda.synchronize()
    close(b[0].cpu().numpy(), a[0, perm].cpu().numpy(), max_abs=1e-2, rel_l2=1e-3)


def test_cached_block_equals_full_recompute(tiny_qk):
    t = tiny_qk
    fresh(t)
    prompt = synth.make_tokens(9, 50, t.shape)      # prefill chunk 24: three chunks
    t.lib.prefill(0, prompt, want_logits=False)
    toks, _ = synth.block_rows(10, t.shape, 1, 8, n_causal=2)
    got = t.lib.block_forward([0], toks, n_causal=[2])
    torch.cuda.synchronize()
    full = t.model.full_forward(np.concatenate([prompt, toks[0]]), causal_point=len(prompt) + 2)
    close(got[0].cpu().numpy(), full[len(prompt):])


def test_commit_is_exact(tiny_qk):
    t = tiny_qk
    fresh(t)
    prompt = synth.make_tokens(11, 20, t.shape)
    nxt = synth.make_tokens(12, 3, t.shape)
    t.lib.prefill(0, np.concatenate([prompt, nxt]), want_logits=False)
    t.lib.prefill(1, prompt, want_logits=False)
    toks = np.array([[nxt[0], nxt[1], nxt[2], t.shape.mask_id, t.shape.mask_id]], np.int32)
    t.lib.block_forward([1], toks, n_causal=[3])
    t.lib.commit([1], [3])
    assert t.lib.cache_len(1) == 23
    k0, v0 = t.lib.kv_export(0, 0, 23)
    k1, v1 = t.lib.kv_export(1, 0, 23)
    torch.cuda.synchronize()
    # Layer 0 depends only on the token and position: bit-identical.  Later layers went
    # through attention splits of different shapes, so allow bf16 rounding differences.
    assert torch.equal(k0[0], k1[0]) and torch.equal(v0[0], v1[0])
    close(k1.float().cpu().numpy(), k0.float().cpu().numpy(), max_abs=5e-2, rel_l2=1e-2)
    close(v1.float().cpu().numpy(), v0.float().cpu().numpy(), max_abs=5e-2, rel_l2=1e-2)
    # and the cache matches the oracle's exact cache
    c, _ = t.model.prefill(np.concatenate([prompt, nxt]))
    for li in range(t.shape.n_layers):
        close(k0[li].float().cpu().numpy(), c.K[li], max_abs=5e-2, rel_l2=1e-2)
        close(v0[li].float().cpu().numpy(), c.V[li], max_abs=5e-2, rel_l2=1e-2)


def test_kv_import_roundtrip_and_parity(tiny):
    fresh(tiny)
    s = tiny.shape
    k, v = synth.make_kv(s, 13, 0, 70, device="cuda")
    tiny.lib.kv_import(0, 0, k, v)
    assert tiny.lib.cache_len(0) == 70
    k2, v2 = tiny.lib.kv_export(0, 0, 70)
    torch.cuda.synchronize()
    assert torch.equal(k, k2) and torch.equal(v, v2)
    toks, is_mask = synth.block_rows(14, s, 1, 4, n_causal=1)
    got = tiny.lib.block_forward([0], toks, is_mask=is_mask)
    torch.cuda.synchronize()
    cache = O.SeqCache.from_arrays(synth.to_host_bits(k), synth.to_host_bits(v), np.float64)
    ref = tiny.model.block_forward([cache], toks, [1]).logits
    close(got.cpu().numpy(), ref)


def test_split_gemm_wait_gives_up_then_recovers():
    """The K slices of a split GEMM wait for each other with a bounded wait.  A forward of 64
    rows on the tiny model runs its down projection (K = 768) as 4 K slices; with a limit of
    zero polls the slices that arrive first give up, the launch still ends, and the next call
    reports the sticky error (task code 65536 + the residual epilogue, 1); a fresh context then
    computes the same logits as before, to the bit."""
    from paper_2509_04185_amd import SbdError
    s = synth.TINY
    B, k = 4, 16

    def make():
        t = Tiny(s, 5105, max_batch=B, max_seq_len=128, max_block=k)
        for b in range(B):
            t.lib.prefill(b, synth.make_tokens(80 + b, 20 + 7 * b, s), want_logits=False)
        return t

    toks, is_mask = synth.block_rows(81, s, B, k, n_causal=1)
    seqs = list(range(B))
    t = make()
    print("[gpu] split GEMM: forced wait failure, 4 x 16 rows", flush=True)
    ref = t.lib.block_forward(seqs, toks, is_mask=is_mask).clone()
    torch.cuda.synchronize()
    t.lib.set_wait_limit(0)
    t.lib.block_forward(seqs, toks, is_mask=is_mask)  # its waits give up; the launch still ends
    torch.cuda.synchronize()
    with pytest.raises(SbdError) as e:
        t.lib.block_forward(seqs, toks, is_mask=is_mask)
    assert "gave up waiting" in str(e.value) and "task code 65537" in str(e.value), str(e.value)
    t.lib.close()
    t2 = make()
    got = t2.lib.block_forward(seqs, toks, is_mask=is_mask)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    t2.lib.close()


def test_ragged_batch_matches_single_sequences(tiny):
    fresh(tiny)
    s = tiny.shape
    lens = [5, 37, 64, 100]
    prompts = [synth.make_tokens(20 + i, n, s) for i, n in enumerate(lens)]
    for i, p in enumerate(prompts):
        tiny.lib.prefill(i, p, want_logits=False)
    toks, _ = synth.block_rows(30, s, 4, 8, n_causal=2)
    nc = np.array([1, 2, 0, 1], np.int32)
    toks[[0, 3], 1] = s.mask_id            # one causal row, then masks
    toks[2, 0] = s.mask_id                 # no causal row; row 1 is an unmasked block row
    is_mask = (toks == s.mask_id).astype(np.uint8)
    both = tiny.lib.block_forward([3, 1, 0, 2], toks[[3, 1, 0, 2]], is_mask=is_mask[[3, 1, 0, 2]],
                                  n_causal=nc[[3, 1, 0, 2]]).cpu().numpy()
    caches = [tiny.model.prefill(p)[0] for p in prompts]
    ref = tiny.model.block_forward(caches, toks, nc).logits
    close(both, ref[[3, 1, 0, 2]])


@pytest.mark.parametrize("nc", [0, 1])
def test_block_forward_on_an_empty_cache(tiny_qk, nc):
    """Nothing cached (a sequence without a prompt): the App. A mask with L = 0, so row 0
    attends to itself alone when causal (nc = 1) and every row to the whole block when
    nc = 0.  A decode-sized forward on each decode path, then one of 32 rows (4 sequences x
    8 rows, two of them with empty caches, two after prefills) on the kernels for more rows."""
    t = tiny_qk
    s = t.shape
    fresh(t)
    toks, is_mask = synth.block_rows(90 + nc, s, 1, 6, n_causal=1)
    assert t.lib.cache_len(0) == 0
    got = t.lib.block_forward([0], toks, is_mask=is_mask, n_causal=[nc]).cpu().numpy()
    ref = t.model.block_forward([t.model.new_cache()], toks, [nc]).logits
    close(got, ref)

    fresh(t)
    prompts = {1: synth.make_tokens(95, 20, s), 3: synth.make_tokens(96, 45, s)}
    for b, p in prompts.items():
        t.lib.prefill(b, p, want_logits=False)
    toks4, is_mask4 = synth.block_rows(97 + nc, s, 4, 8, n_causal=1)
    ncs = [nc, 1, 1 - nc, 1]
    got4 = t.lib.block_forward([0, 1, 2, 3], toks4, is_mask=is_mask4, n_causal=ncs).cpu().numpy()
    caches = [t.model.prefill(prompts[b])[0] if b in prompts else t.model.new_cache() for b in range(4)]
    ref4 = t.model.block_forward(caches, toks4, ncs).logits
    close(got4, ref4)


def test_largest_block_at_full_capacity():
    """k = 64 (the largest block) on a cache filled to max_seq_len by the block (cache_len +
    k = max_seq_len = 200: 128 query rows per KV head, two row blocks of the split attention)
    beside a short sequence, against the oracle; one position more is refused."""
    from paper_2509_04185_amd import SbdError
    s = synth.TINY
    t = Tiny(s, 5005, max_batch=2, max_seq_len=200, max_block=64)
    k = 64
    prompts = [synth.make_tokens(70, 200 - k, s), synth.make_tokens(71, 9, s)]
    for b, p in enumerate(prompts):
        t.lib.prefill(b, p, want_logits=False)
    toks, is_mask = synth.block_rows(72, s, 2, k, n_causal=3)
    nc = [3, 1]
    got = t.lib.block_forward([0, 1], toks, is_mask=is_mask, n_causal=nc).cpu().numpy()
    caches = [t.model.prefill(p)[0] for p in prompts]
    ref = t.model.block_forward(caches, toks, nc).logits
    close(got, ref)
    t.lib.commit([0, 1], [3, 1])
    assert t.lib.cache_len(0) == 200 - k + 3
    with pytest.raises(SbdError) as e:
        t.lib.block_forward([0], toks[:1], is_mask=is_mask[:1], n_causal=[1])
    assert e.value.name == "SBD_ERR_CAPACITY", str(e.value)
    t.lib.close()


def test_qk_norm_model_block_forward(tiny_qk):
    t = tiny_qk
    fresh(t)
    prompt = synth.make_tokens(40, 77, t.shape)
    last = t.lib.prefill(0, prompt)
    toks, is_mask = synth.block_rows(41, t.shape, 1, 16, n_causal=1)
    got = t.lib.block_forward([0], toks, is_mask=is_mask)
    torch.cuda.synchronize()
    cache, ref_last = t.model.prefill(prompt)
    close(last.cpu().numpy(), ref_last)
    close(got.cpu().numpy(), t.model.block_forward([cache], toks, [1]).logits)


def test_intermediate_buffers_last_layer(tiny):
    """The rotated queries and attention output of the last layer against the oracle's steps."""
    fresh(tiny)
    s = tiny.shape
    prompt = synth.make_tokens(50, 31, s)
    tiny.lib.prefill(0, prompt, want_logits=False)
    toks, _ = synth.block_rows(51, s, 1, 4, n_causal=1)
    tiny.lib.block_forward([0], toks)
    torch.cuda.synchronize()
    m = tiny.model
    cache, _ = m.prefill(prompt)
    # replay the oracle's forward up to the last layer's attention
    x = m.W("embed")[toks[0]]
    L = cache.length
    li_last = s.n_layers - 1
    for li in range(s.n_layers):
        h = O.rms_norm(x, m.W("attn_norm", li), s.rms_eps)
        q, kk, vv = m._qkv(h, li, [L + j for j in range(4)])
        Kall = np.concatenate([cache.K[li], kk])
        Vall = np.concatenate([cache.V[li], vv])
        o = O.attention(q, Kall, Vall, O.inference_mask(L, 4, 1))
        if li == li_last:
            break
        x = x + o.reshape(4, -1) @ m.W("wo", li).T
        x = x + m._mlp(x, li)
    qd = s.n_q_heads * s.head_dim
    scale = math.log2(math.e) / math.sqrt(s.head_dim)

    def pair(name):   # [2][rows][width] bf16 -> hi + lo of the first 4 rows
        t = tiny.lib.region(name).float().cpu().numpy().reshape(2, -1, qd)
        return (t[0, :4] + t[1, :4]).reshape(4, s.n_q_heads, s.head_dim)

    close(pair("q") / scale, q, max_abs=1e-3, rel_l2=1e-4)
    close(pair("attn"), o, max_abs=1e-3, rel_l2=1e-4)


def test_decode_path_kernels_launched(tiny):
    """The selected decode path is the one that runs: one fused launch, or none."""
    fresh(tiny)
    s = tiny.shape
    tiny.lib.prefill(0, synth.make_tokens(70, 20, s), want_logits=False)
    toks, is_mask = synth.block_rows(71, s, 1, 16, n_causal=1)
    tiny.lib.profile(True)
    try:
        tiny.lib.profile_read()
        tiny.lib.block_forward([0], toks, is_mask=is_mask)
        stats = tiny.lib.profile_read()
    finally:
        tiny.lib.profile(False)
    launches = {k: n for k, (n, _) in stats.items() if n}
    print(f"    launches {launches}", flush=True)
    if tiny.path == "fused":
        assert launches.get("fused") == 1 and "qkv" not in launches and "lm_head" not in launches
    else:
        assert "fused" not in launches and launches.get("qkv") == s.n_layers


# ------------------------------------------------------------------ state machine and errors


def test_state_and_argument_errors(tiny):
    from paper_2509_04185_amd import SbdError
    fresh(tiny)
    s = tiny.shape
    lib = tiny.lib
    lib.prefill(0, synth.make_tokens(60, 10, s), want_logits=False)
    toks, is_mask = synth.block_rows(61, s, 1, 4, n_causal=1)

    def err(fn, name):
        with pytest.raises(SbdError) as e:
            fn()
        assert e.value.name == name, str(e.value)

    err(lambda: lib.commit([0], [1]), "SBD_ERR_STATE")                    # nothing staged
    lib.block_forward([0], toks)
    err(lambda: lib.commit([0], [2]), "SBD_ERR_STATE")                    # only 1 causal row
    lib.commit([0], [1])
    err(lambda: lib.commit([0], [1]), "SBD_ERR_STATE")                    # already committed
    assert lib.cache_len(0) == 11
    bad = is_mask.copy()
    bad[0, 1] = 0
    err(lambda: lib.block_forward([0], toks, is_mask=bad), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.block_forward([0], np.full((1, 4), s.mask_id, np.int32)), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.block_forward([0, 0], np.vstack([toks, toks])), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.block_forward([9], toks), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.block_forward([0], toks, pos_ids=[[0, 12, 13, 14]]), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.prefill(1, synth.make_tokens(62, 300, s)), "SBD_ERR_CAPACITY")
    logits = torch.zeros((1, 4, s.vocab), device="cuda")
    err(lambda: lib.eb_select(logits, is_mask, float("nan"), s.mask_id), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.eb_select(logits, is_mask, -0.1, s.mask_id), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.select(logits, is_mask, "factor", float("nan"), s.mask_id), "SBD_ERR_INVALID_ARG")
    dummy = torch.empty((1, 4), dtype=torch.int32, device="cuda")
    err(lambda: lib._call("sbd_select", 7, 1, 4, logits.shape[2], logits.data_ptr(),
                          is_mask.astype(np.uint8).ctypes.data, 1.0, s.mask_id, dummy.data_ptr(),
                          dummy.data_ptr(), dummy.data_ptr(), None, None), "SBD_ERR_INVALID_ARG")
    err(lambda: lib.eb_select(torch.zeros((1, 4, 2048), device="cuda"), is_mask, 1.0, -1),
        "SBD_ERR_INVALID_ARG")
    assert lib.lib.sbd_set_decode_path(lib.ctx, 4) == 1                     # unknown path
    # the per-XCD layer kernels need the 8B layer shape: the tiny decoder is refused before
    # anything is enqueued
    assert not lib.decode_path_fits("layers", 1, 4)
    lib.set_decode_path("layers")
    err(lambda: lib.block_forward([0], toks), "SBD_ERR_UNSUPPORTED")
    lib.set_decode_path(tiny.path)
    # a failed call changes nothing
    assert lib.cache_len(0) == 11
    lib.block_forward([0], toks, n_causal=[1])
    lib.commit([0], [1])
    assert lib.cache_len(0) == 12

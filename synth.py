"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle's callers.

This module holds no arithmetic of the method: it only draws random weights,
prompts, KV-cache contents and logits of the shapes the paper's workloads have
(8B Llama-3.1 / Qwen-3 decoders, Sec. 3.1; block sizes up to 16 and contexts
up to 32k tokens, Sec. 3.1 and Sec. 4.1), plus the tiny decoder used for the
small parity cases.  Both sides of a parity test (the HIP library and the CPU
oracle) receive the very same arrays from here.

Weights are returned as torch ``bfloat16`` tensors on the requested device;
``to_host_bits`` gives the raw bf16 bit patterns as numpy ``uint16`` so the
oracle can decode them itself.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Decoder shape.  Names follow the usual Llama/Qwen notation."""
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    mask_id: int
    qk_norm: bool
    rms_eps: float
    rope_theta: float


TINY = ModelShape("tiny", n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                  ffn_dim=768, vocab=1024, mask_id=1023, qk_norm=False, rms_eps=1e-5,
                  rope_theta=1e4)
# Same as TINY with the per-head q/k RMSNorm switched on (exercises the Qwen-3 path).
TINY_QK = dataclasses.replace(TINY, name="tiny_qk", qk_norm=True)
LLAMA8B = ModelShape("llama3.1-8b", n_layers=32, d_model=4096, n_q_heads=32, n_kv_heads=8,
                     head_dim=128, ffn_dim=14336, vocab=128256, mask_id=128255, qk_norm=False,
                     rms_eps=1e-5, rope_theta=5e5)
QWEN8B = ModelShape("qwen3-8b", n_layers=36, d_model=4096, n_q_heads=32, n_kv_heads=8,
                    head_dim=128, ffn_dim=12288, vocab=151936, mask_id=151935, qk_norm=True,
                    rms_eps=1e-6, rope_theta=1e6)

SHAPES = {s.name: s for s in (TINY, TINY_QK, LLAMA8B, QWEN8B)}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One decode-step workload: a model shape, a batch of cached prompts, a block."""
    name: str
    shape: ModelShape
    seed: int
    batch: int
    k: int
    gammas: tuple
    prompt_lens: Optional[tuple] = None      # fixed lengths (None -> ragged draw)
    ragged: Optional[tuple] = None           # (lo, hi) inclusive, drawn per sequence
    logit_scale: float = 1.0                 # EB runs on logits * scale (tiny case)

    def cache_lens(self) -> List[int]:
        if self.prompt_lens is not None:
            return list(self.prompt_lens)
        rng = np.random.default_rng([self.seed, 7])
        lo, hi = self.ragged
        return [int(v) for v in rng.integers(lo, hi + 1, self.batch)]


WORKLOADS = {
    "tiny_b1_l64_k4": Workload("tiny_b1_l64_k4", TINY, 1001, 1, 4, (0.0, 0.5, math.inf),
                               prompt_lens=(64,), logit_scale=4.0),
    "llama8b_b1_l2048_k16": Workload("llama8b_b1_l2048_k16", LLAMA8B, 1002, 1, 16, (1.0,),
                                     prompt_lens=(2048,)),
    "llama8b_b32_ragged_k8": Workload("llama8b_b32_ragged_k8", LLAMA8B, 1003, 32, 8, (0.5,),
                                      ragged=(512, 4096)),
    "llama8b_b4_l32768_k16": Workload("llama8b_b4_l32768_k16", LLAMA8B, 1004, 4, 16, (1.0,),
                                      prompt_lens=(32768,) * 4),
    "qwen8b_b8_l8192_k16": Workload("qwen8b_b8_l8192_k16", QWEN8B, 1005, 8, 16,
                                    (0.1, 1.0, 4.0), prompt_lens=(8192,) * 8),
}

LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "q_norm", "k_norm", "mlp_norm",
              "w_gate", "w_up", "w_down")


def _tensor_shapes(s: ModelShape) -> Dict[str, tuple]:
    qd, kvd = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim
    return {
        "attn_norm": (s.d_model,), "wq": (qd, s.d_model), "wk": (kvd, s.d_model),
        "wv": (kvd, s.d_model), "wo": (s.d_model, qd), "q_norm": (s.head_dim,),
        "k_norm": (s.head_dim,), "mlp_norm": (s.d_model,), "w_gate": (s.ffn_dim, s.d_model),
        "w_up": (s.ffn_dim, s.d_model), "w_down": (s.d_model, s.ffn_dim),
    }


def _gen(seed: int, idx: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 100003 + int(idx))
    return g


def make_weights(shape: ModelShape, seed: int, device="cpu", std: float = 0.02,
                 gain_std: float = 0.1, layers: Optional[Sequence[int]] = None) -> dict:
    """Random-init bf16 weights, N(0, std) per matrix, drawn per tensor from its own stream.

    Norm gains are 1 + N(0, gain_std) (gain_std=0 gives the plain all-ones gains); a
    non-trivial gain makes any mis-indexed gain visible in a parity test.  Every
    tensor is drawn from a generator seeded by (seed, tensor index), so a subset of
    layers can be regenerated alone.  Matrices use the [out][in] row-major layout.
    """
    dev = torch.device(device)
    shapes = _tensor_shapes(shape)

    def draw(idx, shp, is_gain):
        g = _gen(seed, idx, dev)
        t = torch.randn(shp, generator=g, device=dev, dtype=torch.float32)
        if is_gain:
            t = 1.0 + gain_std * t
        else:
            t = t * std
        return t.to(torch.bfloat16)

    w = {
        "embed": draw(0, (shape.vocab, shape.d_model), False),
        "lm_head": draw(1, (shape.vocab, shape.d_model), False),
        "final_norm": draw(2, (shape.d_model,), True),
        "layers": [],
    }
    for li in (range(shape.n_layers) if layers is None else layers):
        lw = {}
        for ki, key in enumerate(LAYER_KEYS):
            lw[key] = draw(1000 + 100 * li + ki, shapes[key], key.endswith("norm"))
        w["layers"].append(lw)
    return w


FP8_KEYS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def make_weights_fp8(shape: ModelShape, seed: int, device="cpu", std: float = 0.02,
                     gain_std: float = 0.1, layers: Optional[Sequence[int]] = None) -> dict:
    """make_weights with every projection matrix and the LM head held as OCP e4m3 bytes
    (torch.uint8) with a power-of-two scale per matrix, the FP8 weights of the paper's
    timing model (Sec. 4.1): e is the smallest exponent with max|w| / 2^e <= 448 (the
    largest e4m3 value) and the bytes are torch's float8_e4m3fn conversion of w / 2^e.
    "fp8_scale_exp" lists e for wq, wk, wv, wo, w_gate, w_up, w_down of each layer, then the
    LM head's.  The embedding and the norm gains stay bf16."""
    w = make_weights(shape, seed, device, std, gain_std, layers)
    exps = []

    def q(t):
        a = t.float()
        top = float(a.abs().max())
        e = math.ceil(math.log2(top / 448.0)) if top > 0 else 0
        return (a * 2.0 ** -e).to(torch.float8_e4m3fn).view(torch.uint8), e

    for lw in w["layers"]:
        for key in FP8_KEYS:
            lw[key], e = q(lw[key])
            exps.append(e)
    w["lm_head"], e = q(w["lm_head"])
    exps.append(e)
    w["fp8_scale_exp"] = exps
    return w


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """Raw bit patterns of a tensor as a host numpy array: bf16 as uint16, e4m3 bytes as uint8."""
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.uint8:
        return t.numpy()
    return t.view(torch.int16).numpy().view(np.uint16)


def weights_to_host(w: dict) -> dict:
    out = {k: (to_host_bits(v) if k != "fp8_scale_exp" else list(v)) for k, v in w.items() if k != "layers"}
    out["layers"] = [{k: to_host_bits(v) for k, v in lw.items()} for lw in w["layers"]]
    return out


def make_tokens(seed: int, n: int, shape: ModelShape, stream: int = 0) -> np.ndarray:
    """Uniform token ids on [0, V) excluding the mask id."""
    rng = np.random.default_rng([seed, 11, stream])
    t = rng.integers(0, shape.vocab - 1, n).astype(np.int32)
    t[t >= shape.mask_id] += 1          # skip mask_id (a no-op when mask_id == V-1)
    return t


def make_kv(shape: ModelShape, seed: int, seq: int, n: int, device="cpu",
            std: float = 1.25) -> tuple:
    """Synthetic cache contents for one sequence: K and V as bf16 [n_layers][n][H_kv][d_h].

    The scale matches what a random-init decoder of the 8B shape produces for its
    projected keys and values (unit-variance RMS-normalised inputs times N(0, 0.02)
    weights over d_model = 4096 inputs gives a standard deviation near 1.28).
    """
    dev = torch.device(device)
    shp = (shape.n_layers, n, shape.n_kv_heads, shape.head_dim)
    gk = _gen(seed, 500000 + 2 * seq, dev)
    gv = _gen(seed, 500001 + 2 * seq, dev)
    k = (torch.randn(shp, generator=gk, device=dev) * std).to(torch.bfloat16)
    v = (torch.randn(shp, generator=gv, device=dev) * std).to(torch.bfloat16)
    return k, v


def entropy_ladder_logits(seed: int, batch: int, k: int, vocab: int, device="cpu",
                          lo: float = 0.25, hi: float = 32.0) -> torch.Tensor:
    """fp32 logits [batch][k][vocab]; row j is sigma_j * N(0,1), sigma_j log-uniform on [lo, hi].

    Spreads per-row entropies from near 0 to near ln(vocab) so that intermediate
    thresholds accept intermediate numbers of rows.
    """
    dev = torch.device(device)
    g = _gen(seed, 900000, dev)
    z = torch.randn((batch, k, vocab), generator=g, device=dev, dtype=torch.float32)
    rng = np.random.default_rng([seed, 13])
    sig = np.exp(rng.uniform(math.log(lo), math.log(hi), (batch, k))).astype(np.float32)
    return z * torch.from_numpy(sig).to(dev)[:, :, None]


def block_rows(seed: int, shape: ModelShape, batch: int, k: int, n_causal: int = 1,
               stream: int = 1) -> tuple:
    """Block tokens and mask flags: rows < n_causal are real ids, the rest are the mask id."""
    toks = np.full((batch, k), shape.mask_id, dtype=np.int32)
    real = make_tokens(seed, batch * max(n_causal, 1), shape, stream=stream)
    real = real.reshape(batch, max(n_causal, 1))
    toks[:, :n_causal] = real[:, :n_causal]
    is_mask = (toks == shape.mask_id).astype(np.uint8)
    return toks, is_mask

"""Python binding of libsbd.so: argument marshalling over the C ABI declared in sbd.h.

Every computation runs in the HIP library; this module only converts arguments
(torch CUDA tensors -> device pointers, numpy/int sequences -> host arrays), owns the
device workspace tensor, and turns non-OK statuses into ``SbdError``.  If the library
has not been built it raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_size_t, c_void_p
from typing import Optional

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsbd.so")

STATUS = {0: "SBD_OK", 1: "SBD_ERR_INVALID_ARG", 2: "SBD_ERR_STATE", 3: "SBD_ERR_CAPACITY",
          4: "SBD_ERR_OUT_OF_MEMORY", 5: "SBD_ERR_HIP", 6: "SBD_ERR_UNSUPPORTED"}

LAYER_FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "q_norm", "k_norm", "mlp_norm",
                "w_gate", "w_up", "w_down")

# sbd_kernel values, in order.
KERNEL_NAMES = ("embed", "qkv", "rope", "attention", "attn_merge", "o_proj", "gate_up", "down",
                "lm_head", "eb_partial", "eb_select", "fused", "layer_attn", "layer_mlp", "layer_final")
DECODE_PATHS = {"auto": 0, "fused": 1, "kernels": 2, "layers": 3}  # sbd_decode_path
SELECT_RULES = {"eb_entropy": 0, "eb_confidence": 1, "factor": 2}  # SBD_SELECT_*

# Every entry point of sbd.h with its argument types.
SIGNATURES = {
    "sbd_workspace_bytes": [c_void_p, POINTER(c_size_t)],
    "sbd_workspace_region": [c_void_p, c_char_p, POINTER(c_size_t), POINTER(c_size_t)],
    "sbd_create": [c_void_p, c_void_p, c_void_p, c_size_t, c_void_p, POINTER(c_void_p)],
    "sbd_destroy": [c_void_p],
    "sbd_set_stream": [c_void_p, c_void_p],
    "sbd_reset": [c_void_p, c_int32],
    "sbd_cache_len": [c_void_p, c_int32, POINTER(c_int32)],
    "sbd_prefill": [c_void_p, c_int32, c_void_p, c_int32, c_void_p],
    "sbd_block_forward": [c_void_p, c_int32, c_void_p, c_int32, c_void_p, c_void_p, c_void_p,
                          c_void_p, c_void_p],
    "sbd_commit": [c_void_p, c_int32, c_void_p, c_void_p],
    "sbd_block_step": [c_void_p, c_int32, c_int32, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                       c_double, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p],
    "sbd_eb_select": [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_double, c_int32,
                      c_void_p, c_void_p, c_void_p, c_void_p],
    "sbd_select": [c_void_p, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_double, c_int32,
                   c_void_p, c_void_p, c_void_p, c_void_p, c_void_p],
    "sbd_eb_select_entropies": [c_void_p, c_int32, c_int32, c_void_p, c_void_p, c_double,
                                c_void_p, c_void_p],
    "sbd_eb_select_noalloc": [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_double, c_int32,
                              c_void_p, c_void_p, c_void_p, c_void_p],
    "sbd_kv_import": [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p],
    "sbd_kv_export": [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p],
    "sbd_set_decode_path": [c_void_p, c_int32],
    "sbd_decode_path_fits": [c_void_p, c_int32, c_int32, c_int32, POINTER(c_int32)],
    "sbd_set_wait_limit": [c_void_p, c_int32],
    "sbd_profile_enable": [c_void_p, c_int32],
    "sbd_xcd_map_ok": [c_void_p, POINTER(c_int32)],
    "sbd_xcd_map_check": [c_void_p, c_int32, c_int32, POINTER(c_int32)],
    "sbd_stream_probe": [c_void_p, c_void_p, c_size_t, c_void_p],
    "sbd_profile_read": [c_void_p, c_int32, POINTER(c_int32), POINTER(c_double)],
    "sbd_status_string": [c_int32],
    "sbd_last_error": [c_void_p],
}


class ModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_q_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("ffn_dim", c_int32),
                ("vocab", c_int32), ("mask_id", c_int32), ("qk_norm", c_int32),
                ("rms_eps", c_float), ("rope_theta", c_float), ("max_batch", c_int32),
                ("max_seq_len", c_int32), ("max_block", c_int32), ("prefill_chunk", c_int32),
                ("weight_format", c_int32), ("kv_format", c_int32), ("kv_scale_exp", c_int32)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("lm_head", c_void_p), ("final_norm", c_void_p)] + \
               [(f, POINTER(c_void_p)) for f in LAYER_FIELDS] + [("fp8_scale_exp", POINTER(c_int32))]

WEIGHT_FORMATS = {"bf16": 0, "fp8_e4m3": 1}  # SBD_WEIGHTS_*
KV_FORMATS = {"bf16": 0, "fp8_e4m3": 1}      # SBD_KV_*


class SbdError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")
        self.status = status
        self.name = STATUS.get(status, str(status))


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libsbd.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (paper_2509_04185_amd/build.py "
                           "or __graft_entry__.build()); there is no fallback path")
    lib = ctypes.CDLL(path)
    for name, args in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = c_char_p if name in ("sbd_status_string", "sbd_last_error") else c_int32
    _lib = lib
    return lib


def make_config(shape, max_batch: int, max_seq_len: int, max_block: int,
                prefill_chunk: int = 0, weight_format: str = "bf16", kv_format: str = "bf16",
                kv_scale_exp: int = 0) -> ModelConfig:
    return ModelConfig(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                       shape.head_dim, shape.ffn_dim, shape.vocab, shape.mask_id,
                       int(bool(shape.qk_norm)), float(shape.rms_eps), float(shape.rope_theta),
                       max_batch, max_seq_len, max_block, prefill_chunk, WEIGHT_FORMATS[weight_format],
                       KV_FORMATS[kv_format], int(kv_scale_exp))


def _check(lib, st: int, where: str, ctx=None):
    if st != 0:
        raise SbdError(st, where, lib.sbd_last_error(ctx).decode(errors="replace"))


def workspace_bytes(cfg: ModelConfig) -> int:
    lib = load_library()
    n = c_size_t(0)
    _check(lib, lib.sbd_workspace_bytes(ctypes.byref(cfg), ctypes.byref(n)), "sbd_workspace_bytes")
    return n.value


def _host(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(c_void_p)


def _dev(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous CUDA tensor")
    return c_void_p(t.data_ptr())


class Sbd:
    """One library context: model weights (borrowed), KV cache and scratch (owned workspace)."""

    REGION_DTYPES = {"x": torch.float32, "qkv": torch.float32, "q": torch.bfloat16,
                     "attn": torch.bfloat16, "act": torch.bfloat16, "xn": torch.bfloat16}

    def __init__(self, shape, weights: dict, max_batch: int, max_seq_len: int, max_block: int,
                 prefill_chunk: int = 0, device="cuda", kv_format: str = "bf16", kv_scale_exp: int = 0):
        """weights: bf16 tensors, or with an "fp8_scale_exp" entry (synth.make_weights_fp8) the
        projection and LM-head matrices as e4m3 bytes (uint8) with those scale exponents.
        kv_format "fp8_e4m3": the KV cache holds e4m3 codes of value * 2^-kv_scale_exp."""
        self.lib = load_library()
        self.shape = shape
        self.weight_format = "fp8_e4m3" if "fp8_scale_exp" in weights else "bf16"
        self.kv_format = kv_format
        self.cfg = make_config(shape, max_batch, max_seq_len, max_block, prefill_chunk, self.weight_format,
                               kv_format, kv_scale_exp)
        self.device = torch.device(device)
        self.weights = weights                       # keep the borrowed tensors alive
        nbytes = workspace_bytes(self.cfg)
        self.workspace = torch.zeros(nbytes, dtype=torch.uint8, device=self.device)
        nl = shape.n_layers
        self._arrays = {}
        w = Weights()
        w.embed = _dev(weights["embed"])
        w.lm_head = _dev(weights["lm_head"])
        w.final_norm = _dev(weights["final_norm"])
        for f in LAYER_FIELDS:
            arr = (c_void_p * nl)(*[weights["layers"][l][f].data_ptr() for l in range(nl)])
            self._arrays[f] = arr
            setattr(w, f, ctypes.cast(arr, POINTER(c_void_p)))
        if self.weight_format == "fp8_e4m3":
            exps = [int(e) for e in weights["fp8_scale_exp"]]
            self._exps = (c_int32 * len(exps))(*exps)
            w.fp8_scale_exp = ctypes.cast(self._exps, POINTER(c_int32))
        self._w = w
        ctx = c_void_p()
        st = self.lib.sbd_create(ctypes.byref(self.cfg), ctypes.byref(w),
                                 c_void_p(self.workspace.data_ptr()), nbytes, self._stream(),
                                 ctypes.byref(ctx))
        _check(self.lib, st, "sbd_create")
        self.ctx = ctx

    # -- plumbing ---------------------------------------------------------------------
    def _stream(self):
        return c_void_p(torch.cuda.current_stream(self.device).cuda_stream)

    def _call(self, name: str, *args):
        self.lib.sbd_set_stream(self.ctx, self._stream())
        _check(self.lib, getattr(self.lib, name)(self.ctx, *args), name, self.ctx)

    def close(self):
        if getattr(self, "ctx", None):
            self.lib.sbd_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- entry points -----------------------------------------------------------------
    def reset(self, seq: int):
        self._call("sbd_reset", int(seq))

    def cache_len(self, seq: int) -> int:
        n = c_int32(0)
        _check(self.lib, self.lib.sbd_cache_len(self.ctx, int(seq), ctypes.byref(n)),
               "sbd_cache_len", self.ctx)
        return n.value

    def prefill(self, seq: int, tokens, want_logits: bool = True) -> Optional[torch.Tensor]:
        toks = _host(tokens, np.int32).reshape(-1)
        out = torch.empty(self.shape.vocab, dtype=torch.float32, device=self.device) \
            if want_logits else None
        self._call("sbd_prefill", int(seq), _ptr(toks), int(toks.size), _dev(out))
        return out

    def block_forward(self, seq_ids, tokens, is_mask=None, n_causal=None, pos_ids=None,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
        seq = _host(seq_ids, np.int32).reshape(-1)
        toks = _host(tokens, np.int32)
        B, k = toks.shape
        msk = None if is_mask is None else _host(is_mask, np.uint8)
        nc = None if n_causal is None else _host(n_causal, np.int32)
        pos = None if pos_ids is None else _host(pos_ids, np.int32)
        if out is None:
            out = torch.empty((B, k, self.shape.vocab), dtype=torch.float32, device=self.device)
        self._call("sbd_block_forward", B, _ptr(seq), k, _ptr(toks), _ptr(msk), _ptr(nc),
                   _ptr(pos), _dev(out))
        return out

    def block_step(self, seq_ids, tokens, rule: str = "eb_entropy", threshold: float = 1.0, is_mask=None,
                   n_causal=None, pos_ids=None, want_logits: bool = False):
        """sbd_block_step: block forward + selection with the statistics from the LM head.
        Returns (n_accepted, accepted_pos, accepted_tok, entropy, confidence, logits or None)."""
        seq = _host(seq_ids, np.int32).reshape(-1)
        toks = _host(tokens, np.int32)
        B, k = toks.shape
        msk = None if is_mask is None else _host(is_mask, np.uint8)
        nc = None if n_causal is None else _host(n_causal, np.int32)
        pos = None if pos_ids is None else _host(pos_ids, np.int32)
        dev = self.device
        logits = torch.empty((B, k, self.shape.vocab), dtype=torch.float32, device=dev) if want_logits else None
        n_acc = torch.empty(B, dtype=torch.int32, device=dev)
        acc_pos = torch.empty((B, k), dtype=torch.int32, device=dev)
        acc_tok = torch.empty((B, k), dtype=torch.int32, device=dev)
        H = torch.empty((B, k), dtype=torch.float64, device=dev)
        C = torch.empty((B, k), dtype=torch.float64, device=dev)
        self._call("sbd_block_step", SELECT_RULES[rule], B, _ptr(seq), k, _ptr(toks), _ptr(msk), _ptr(nc), _ptr(pos),
                   float(threshold), _dev(logits), _dev(n_acc), _dev(acc_pos), _dev(acc_tok), _dev(H), _dev(C))
        return n_acc, acc_pos, acc_tok, H, C, logits

    def commit(self, seq_ids, n_commit):
        seq = _host(seq_ids, np.int32).reshape(-1)
        n = _host(n_commit, np.int32).reshape(-1)
        self._call("sbd_commit", int(seq.size), _ptr(seq), _ptr(n))

    def eb_select(self, logits: torch.Tensor, is_mask, gamma: float, mask_id: int,
                  want_entropy: bool = True):
        B, k, V = logits.shape
        msk = _host(is_mask, np.uint8)
        n_acc = torch.empty(B, dtype=torch.int32, device=logits.device)
        pos = torch.empty((B, k), dtype=torch.int32, device=logits.device)
        tok = torch.empty((B, k), dtype=torch.int32, device=logits.device)
        H = torch.empty((B, k), dtype=torch.float64, device=logits.device) if want_entropy else None
        self._call("sbd_eb_select", B, k, V, _dev(logits), _ptr(msk), float(gamma), int(mask_id),
                   _dev(n_acc), _dev(pos), _dev(tok), _dev(H))
        return n_acc, pos, tok, H

    def select(self, logits: torch.Tensor, is_mask, rule: str, threshold: float, mask_id: int):
        """One sampling step under a selection rule (sbd_select): "eb_entropy", "eb_confidence" or
        "factor".  Returns (n_accepted, accepted_pos, accepted_tok, entropy, confidence)."""
        B, k, V = logits.shape
        msk = _host(is_mask, np.uint8)
        dev = logits.device
        n_acc = torch.empty(B, dtype=torch.int32, device=dev)
        pos = torch.empty((B, k), dtype=torch.int32, device=dev)
        tok = torch.empty((B, k), dtype=torch.int32, device=dev)
        H = torch.empty((B, k), dtype=torch.float64, device=dev)
        C = torch.empty((B, k), dtype=torch.float64, device=dev)
        self._call("sbd_select", SELECT_RULES[rule], B, k, V, _dev(logits), _ptr(msk), float(threshold),
                   int(mask_id), _dev(n_acc), _dev(pos), _dev(tok), _dev(H), _dev(C))
        return n_acc, pos, tok, H, C

    def eb_select_entropies(self, entropy: torch.Tensor, is_mask, gamma: float):
        B, k = entropy.shape
        msk = _host(is_mask, np.uint8)
        n_acc = torch.empty(B, dtype=torch.int32, device=entropy.device)
        pos = torch.empty((B, k), dtype=torch.int32, device=entropy.device)
        self._call("sbd_eb_select_entropies", B, k, _dev(entropy), _ptr(msk), float(gamma),
                   _dev(n_acc), _dev(pos))
        return n_acc, pos

    def kv_import(self, seq: int, pos0: int, k: torch.Tensor, v: torch.Tensor):
        n = k.shape[1]
        self._call("sbd_kv_import", int(seq), int(pos0), int(n), _dev(k), _dev(v))

    def kv_export(self, seq: int, pos0: int, n: int):
        s = self.shape
        shp = (s.n_layers, n, s.n_kv_heads, s.head_dim)
        k = torch.empty(shp, dtype=torch.bfloat16, device=self.device)
        v = torch.empty(shp, dtype=torch.bfloat16, device=self.device)
        self._call("sbd_kv_export", int(seq), int(pos0), int(n), _dev(k), _dev(v))
        return k, v

    def set_decode_path(self, path: str):
        """Kernels of decode-sized forwards: "auto", "fused", "kernels" or "layers" (sbd_set_decode_path)."""
        code = DECODE_PATHS[path]
        _check(self.lib, self.lib.sbd_set_decode_path(self.ctx, code), "sbd_set_decode_path", self.ctx)

    def set_wait_limit(self, polls: int):
        """Polls before a wait inside a layer-kernel or split-GEMM launch gives up; negative: the default."""
        _check(self.lib, self.lib.sbd_set_wait_limit(self.ctx, polls), "sbd_set_wait_limit", self.ctx)

    def decode_path_fits(self, path: str, batch: int, k: int) -> bool:
        """Whether `path` can run a forward of `batch` x `k` rows here (sbd_decode_path_fits)."""
        fits = c_int32(0)
        _check(self.lib, self.lib.sbd_decode_path_fits(self.ctx, DECODE_PATHS[path], batch, k, ctypes.byref(fits)),
               "sbd_decode_path_fits", self.ctx)
        return bool(fits.value)

    def xcd_map_ok(self) -> bool:
        """Whether the probe at creation found workgroup i on XCD i % 8 (sbd_xcd_map_ok)."""
        ok = c_int32(0)
        _check(self.lib, self.lib.sbd_xcd_map_ok(self.ctx, ctypes.byref(ok)), "sbd_xcd_map_ok", self.ctx)
        return bool(ok.value)

    def profile(self, enable: bool):
        _check(self.lib, self.lib.sbd_profile_enable(self.ctx, int(bool(enable))),
               "sbd_profile_enable", self.ctx)

    def profile_read(self) -> dict:
        """{kernel name: (launches, total ms)} since the previous read."""
        out = {}
        for i, name in enumerate(KERNEL_NAMES):
            n, ms = c_int32(0), c_double(0.0)
            _check(self.lib, self.lib.sbd_profile_read(self.ctx, i, ctypes.byref(n), ctypes.byref(ms)),
                   "sbd_profile_read", self.ctx)
            out[name] = (n.value, ms.value)
        return out

    def region(self, name: str) -> torch.Tensor:
        """View of an internal buffer of the workspace (values of the last layer / forward)."""
        off, nb = c_size_t(0), c_size_t(0)
        _check(self.lib, self.lib.sbd_workspace_region(ctypes.byref(self.cfg), name.encode(),
                                                       ctypes.byref(off), ctypes.byref(nb)),
               "sbd_workspace_region")
        return self.workspace[off.value: off.value + nb.value].view(self.REGION_DTYPES[name])


def eb_select_noalloc(logits: torch.Tensor, is_mask, gamma: float, mask_id: int, out=None):
    """sbd_eb_select_noalloc on torch's current stream: the EB step without a context or a
    workspace.  out: optional preallocated (n_accepted, accepted_pos, accepted_tok, entropy)."""
    lib = load_library()
    B, k, V = logits.shape
    msk = _host(is_mask, np.uint8)
    dev = logits.device
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, k), dtype=torch.int32, device=dev),
               torch.empty((B, k), dtype=torch.int32, device=dev), torch.empty((B, k), dtype=torch.float64, device=dev))
    n_acc, pos, tok, H = out
    stream = c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    _check(lib, lib.sbd_eb_select_noalloc(stream, B, k, V, _dev(logits), _ptr(msk), float(gamma), int(mask_id),
                                          _dev(n_acc), _dev(pos), _dev(tok), _dev(H)), "sbd_eb_select_noalloc")
    return n_acc, pos, tok, H


def stream_probe(buf: torch.Tensor, sink: torch.Tensor):
    """sbd_stream_probe on torch's current stream: one streaming read of the whole tensor."""
    lib = load_library()
    stream = c_void_p(torch.cuda.current_stream(buf.device).cuda_stream)
    _check(lib, lib.sbd_stream_probe(stream, _dev(buf), buf.numel() * buf.element_size(), _dev(sink)),
           "sbd_stream_probe")


def status_string(status: int) -> str:
    return load_library().sbd_status_string(status).decode()

"""CPU oracle for one Set Block Decoding (SBD) step.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke entry point and the benchmark's CPU-baseline leg may
import this module.  The product path (the HIP library and its Python binding) never
calls it, and it shares no code with that path: it takes plain numpy arrays (weights
as floats or as raw bf16 bit patterns in uint16) and computes everything itself.

What it computes, following the paper (Set Block Decoding, arXiv 2509.04185):

* The SBD network f_theta of eq. (hybrid): a standard decoder in which the tokens left
  of ';' (the committed prefix) use causal attention and the k block tokens right of
  ';' use bidirectional attention (Sec. 2.3, Fig. 3).  The inference attention mask is
  the one of App. A (inference mask): key kv is visible to query q iff kv <= q, or q is
  at or after the first index of the prediction block.
* The block logits z_hat_{t+i} predict the token at their own position t+i (Sec. 2.3,
  eq. (p_theta_masked)); all block rows share the positions of the tokens they stand
  for (App. A, training code: one position id per token location).
* Exact KV caching (Sec. 1, advantages list; Alg. 3): the cache only ever receives the
  keys/values of causal rows.  ``commit`` appends those rows.
* The EB-Sampler of Sec. 2.2, eq. (eb_sampler): sort masked positions by ascending
  entropy of their predicted distributions; reveal the first s, s >= 1 the largest
  integer with sum_{j<s} H_(j) <= gamma.

The decoder body (RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU MLP,
optional per-head q/k RMSNorm of Qwen-3) is the standard Llama-3.1 / Qwen-3 block;
the paper states there are no architectural changes (Sec. 1, advantages list).

Readings where the paper is silent (each is listed with its reason in the design notes):
* the mask token is excluded from the entropy and the argmax (the output distribution
  lives on V, Sec. 2 notation; the mask token is an input-only symbol);
* entropies are in nats of softmax(z) at temperature 1; tokens are argmax (Sec. 3.1
  uses temperature 0 for tokens);
* equal entropies are ordered by row index; argmax ties go to the smallest token id;
* gamma may be 0 (used in Sec. 3.2) or +inf.

Weights are bf16 bit patterns, or (FP8 weights, the paper's timing assumption of Sec. 4.1)
e4m3 bytes with a power-of-two scale per matrix, decoded here from the format's definition.

Precision: everything runs in the dtype given to ``Model`` (float64 by default);
EB statistics are always float64.  With ``kv_bf16`` the keys and values are held in
bfloat16, the storage format of the KV cache, with ``kv_fp8_exp`` in e4m3 with a
power-of-two scale (the 1-byte KV of Sec. 4.1); activations stay in the working dtype.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np

# ----------------------------------------------------------------------------- helpers


def decode_weight(a, dtype=np.float64) -> np.ndarray:
    """Float view of a weight array; uint16 arrays are raw bf16 bit patterns."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        bits = np.empty(a.shape, dtype=np.uint32)
        np.left_shift(a, 16, out=bits, dtype=np.uint32)
        a = bits.view(np.float32)
    return a.astype(dtype, copy=False)


def decode_e4m3(bits, dtype=np.float64) -> np.ndarray:
    """Values of OCP FP8 E4M3 bytes (the "fn" variant): 1 sign bit, 4 exponent bits of bias
    7, 3 mantissa bits; exponent field 0 holds the subnormals m/8 * 2^-6; the two patterns
    with every exponent and mantissa bit set are NaN; there are no infinities."""
    return _E4M3_VALUES.astype(dtype)[np.asarray(bits, dtype=np.uint8)]


def _e4m3_table() -> np.ndarray:
    """The value of each of the 256 e4m3 codes, from the format's definition."""
    b = np.arange(256)
    sign = (b >> 7) & 1
    e = (b >> 3) & 15
    m = (b & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0))
    mag = np.where((e == 15) & (b & 7 == 7), np.nan, mag)
    return np.where(sign == 1, -mag, mag)


_E4M3_VALUES = _e4m3_table()


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (8 significant bits, ties to even), same dtype out.

    Written with frexp/ldexp: a = m * 2^e with 0.5 <= |m| < 1, so m * 2^8 holds the 8
    kept bits before the point; rint rounds half to even.  Values are assumed to be in
    the normal range of bfloat16 (the exponent range of float32).
    """
    a = np.asarray(a)
    m, e = np.frexp(a.astype(np.float64))
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8).astype(a.dtype)


def round_to_e4m3(a: np.ndarray, scale_exp: int = 0) -> np.ndarray:
    """What a KV cache of e4m3 bytes with the scale 2^e holds for a (the 1-byte KV of the
    paper's timing model, Sec. 4.1): x = a * 2^-e rounded to the nearest e4m3 value, ties to
    even, saturated at +-448 (the largest finite code), times 2^e; NaN stays NaN.

    The e4m3 values (decode_e4m3): from 2^-6 up they carry 4 significant bits; below 2^-6
    they are the multiples of 2^-9.  With x = m * 2^q, 0.5 <= |m| < 1 (frexp), |x| >= 2^-6
    is q >= -5 and keeps rint(m * 2^4) * 2^(q - 4); below, rint(x * 2^9) * 2^-9 (rint rounds
    half to even; a carry to 2^q, or from the subnormals to 2^-6, is the next code up).
    """
    a = np.asarray(a)
    x = np.ldexp(a.astype(np.float64), -int(scale_exp))
    m, q = np.frexp(x)
    r = np.where(q >= -5, np.ldexp(np.rint(np.ldexp(m, 4)), q - 4), np.ldexp(np.rint(np.ldexp(x, 9)), -9))
    return np.ldexp(np.clip(r, -448.0, 448.0), int(scale_exp)).astype(a.dtype)


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis (Llama/Qwen RMSNorm)."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def rope_cos_sin(pos: Sequence[int], head_dim: int, theta: float, dtype) -> tuple:
    """cos/sin of the rotate-half RoPE angles p * theta^(-2i/d_h), i < d_h/2.

    Angles are formed in float64 and then cast to the working dtype.
    """
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / head_dim)
    phi = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(phi).astype(dtype), np.sin(phi).astype(dtype)


def apply_rope(u: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate the pairs (u_i, u_{i+d/2}) of every head by the row's angles.

    u: [rows, heads, d_h]; cos, sin: [rows, d_h/2].
    """
    half = u.shape[-1] // 2
    a, b = u[..., :half], u[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def inference_mask(n_prefix: int, k: int, n_causal: int) -> np.ndarray:
    """Visibility [k, n_prefix + k] of the block rows over prefix + block keys.

    The App. A inference mask with query index q = n_prefix + j, key index kv and
    causal point = n_prefix + n_causal (the first index of the prediction block):
    visible iff kv <= q or causal_point <= q.
    """
    q_idx = n_prefix + np.arange(k)[:, None]
    kv_idx = np.arange(n_prefix + k)[None, :]
    causal_point = n_prefix + n_causal
    return (kv_idx <= q_idx) | (causal_point <= q_idx)


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, visible: np.ndarray) -> np.ndarray:
    """Grouped-query softmax attention.

    q: [rows, H_q, d_h]; K, V: [keys, H_kv, d_h]; visible: [rows, keys] bool.
    Query head h reads key/value head floor(h * H_kv / H_q).
    """
    rows, n_q, d_h = q.shape
    n_kv = K.shape[1]
    out = np.zeros_like(q)
    scale = 1.0 / math.sqrt(d_h)
    for h in range(n_q):
        g = h * n_kv // n_q
        s = (q[:, h, :] @ K[:, g, :].T) * scale
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ V[:, g, :]
    return out


# ----------------------------------------------------------------------------- model


class SeqCache:
    """Exact KV cache of one sequence: per layer K, V as [L][H_kv][d_h] arrays."""

    def __init__(self, n_layers: int, n_kv: int, d_h: int, dtype):
        self.K = [np.zeros((0, n_kv, d_h), dtype) for _ in range(n_layers)]
        self.V = [np.zeros((0, n_kv, d_h), dtype) for _ in range(n_layers)]

    @property
    def length(self) -> int:
        return self.K[0].shape[0]

    def copy(self) -> "SeqCache":
        c = SeqCache.__new__(SeqCache)
        c.K = [a.copy() for a in self.K]
        c.V = [a.copy() for a in self.V]
        return c

    def to_e4m3(self, scale_exp: int) -> "SeqCache":
        """A copy holding what an e4m3 cache with the scale 2^scale_exp stores (round_to_e4m3)."""
        c = SeqCache.__new__(SeqCache)
        c.K = [round_to_e4m3(a, scale_exp) for a in self.K]
        c.V = [round_to_e4m3(a, scale_exp) for a in self.V]
        return c

    @classmethod
    def from_arrays(cls, K, V, dtype) -> "SeqCache":
        """K, V: [n_layers][L][H_kv][d_h] (float or bf16 bits)."""
        c = cls.__new__(cls)
        c.K = [decode_weight(K[i], dtype) for i in range(len(K))]
        c.V = [decode_weight(V[i], dtype) for i in range(len(V))]
        return c


class BlockResult:
    """Output of one block forward: logits per row plus the staged K/V of every row."""

    def __init__(self, logits, K_new, V_new, n_causal):
        self.logits = logits          # [B][k][V]
        self.K_new = K_new            # per sequence: per layer [k][H_kv][d_h]
        self.V_new = V_new
        self.n_causal = n_causal      # per sequence


class Model:
    """The SBD network f_theta on plain arrays.

    ``shape`` needs the attributes n_layers, d_model, n_q_heads, n_kv_heads, head_dim,
    ffn_dim, vocab, qk_norm, rms_eps, rope_theta.  ``weights`` is a dict with embed,
    lm_head, final_norm and a list ``layers`` of dicts (attn_norm, wq, wk, wv, wo,
    q_norm, k_norm, mlp_norm, w_gate, w_up, w_down); matrices are [out][in].
    """

    def __init__(self, shape, weights: dict, dtype=np.float64, cache_decoded: bool = True,
                 kv_bf16: bool = False, kv_fp8_exp: Optional[int] = None):
        """kv_bf16: keys/values are stored in bfloat16 (the KV-cache storage format of the
        GPU path): every K/V row is rounded to bf16 when it is produced, before it is used
        by attention or appended to the cache.  kv_fp8_exp = e: they are stored as e4m3
        bytes with the scale 2^e instead (round_to_e4m3), rounded the same way."""
        self.s = shape
        self.w = weights
        self.dtype = np.dtype(dtype)
        self._memo = {} if cache_decoded else None
        self.kv_bf16 = kv_bf16
        self.kv_fp8_exp = kv_fp8_exp

    # FP8 weights (uint8 arrays): the order of the per-matrix scale exponents in
    # weights["fp8_scale_exp"], per layer; the LM head's comes after every layer's
    FP8_ORDER = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")

    def W(self, name: str, layer: Optional[int] = None) -> np.ndarray:
        key = (name, layer)
        if self._memo is not None and key in self._memo:
            return self._memo[key]
        src = self.w[name] if layer is None else self.w["layers"][layer][name]
        if np.asarray(src).dtype == np.uint8:
            # e4m3 bytes times the matrix's power-of-two scale (exact)
            i = self.s.n_layers * 7 if layer is None else layer * 7 + self.FP8_ORDER.index(name)
            a = decode_e4m3(src, self.dtype) * self.dtype.type(2.0 ** int(self.w["fp8_scale_exp"][i]))
        else:
            a = decode_weight(src, self.dtype)
        if self._memo is not None:
            self._memo[key] = a
        return a

    def new_cache(self) -> SeqCache:
        s = self.s
        return SeqCache(s.n_layers, s.n_kv_heads, s.head_dim, self.dtype)

    # -- the network ---------------------------------------------------------------
    def _qkv(self, h, li, pos):
        s = self.s
        rows = h.shape[0]
        q = (h @ self.W("wq", li).T).reshape(rows, s.n_q_heads, s.head_dim)
        k = (h @ self.W("wk", li).T).reshape(rows, s.n_kv_heads, s.head_dim)
        v = (h @ self.W("wv", li).T).reshape(rows, s.n_kv_heads, s.head_dim)
        if s.qk_norm:
            q = rms_norm(q, self.W("q_norm", li), s.rms_eps)
            k = rms_norm(k, self.W("k_norm", li), s.rms_eps)
        cos, sin = rope_cos_sin(pos, s.head_dim, s.rope_theta, self.dtype)
        q, k = apply_rope(q, cos, sin), apply_rope(k, cos, sin)
        if self.kv_fp8_exp is not None:
            k, v = round_to_e4m3(k, self.kv_fp8_exp), round_to_e4m3(v, self.kv_fp8_exp)
        elif self.kv_bf16:
            k, v = round_to_bf16(k), round_to_bf16(v)
        return q, k, v

    def _mlp(self, x, li):
        s = self.s
        h2 = rms_norm(x, self.W("mlp_norm", li), s.rms_eps)
        a = silu(h2 @ self.W("w_gate", li).T) * (h2 @ self.W("w_up", li).T)
        return a @ self.W("w_down", li).T

    def block_forward(self, caches: List[SeqCache], tokens, n_causal, pos=None) -> BlockResult:
        """Eq. (hybrid_block) for a batch of independent sequences.

        tokens: [B][k] ids (mask id allowed); n_causal: [B], rows < n_causal[b] are the
        committed-but-uncached causal rows, the rest form the prediction block;
        pos: [B][k] position ids, default cache length + row.
        Returns logits [B][k][V] and the post-RoPE K and the V of every block row.
        """
        s = self.s
        tokens = np.asarray(tokens)
        B, k = tokens.shape
        n_causal = [int(n) for n in np.broadcast_to(np.asarray(n_causal), (B,))]
        L = [c.length for c in caches]
        if pos is None:
            pos = np.array([[L[b] + j for j in range(k)] for b in range(B)])
        pos = np.asarray(pos)
        E = self.W("embed")
        x = E[tokens.reshape(-1)].astype(self.dtype)           # [B*k][d]
        K_new = [[None] * s.n_layers for _ in range(B)]
        V_new = [[None] * s.n_layers for _ in range(B)]
        for li in range(s.n_layers):
            h = rms_norm(x, self.W("attn_norm", li), s.rms_eps)
            o = np.zeros((B * k, s.n_q_heads, s.head_dim), self.dtype)
            for b in range(B):
                r = slice(b * k, (b + 1) * k)
                q, kk, vv = self._qkv(h[r], li, pos[b])
                K_new[b][li], V_new[b][li] = kk, vv
                Kall = np.concatenate([caches[b].K[li], kk], axis=0)
                Vall = np.concatenate([caches[b].V[li], vv], axis=0)
                vis = inference_mask(L[b], k, n_causal[b])
                o[r] = attention(q, Kall, Vall, vis)
            x = x + o.reshape(B * k, -1) @ self.W("wo", li).T
            x = x + self._mlp(x, li)
        hf = rms_norm(x, self.W("final_norm"), s.rms_eps)
        logits = hf @ self.W("lm_head").T
        return BlockResult(logits.reshape(B, k, s.vocab), K_new, V_new, n_causal)

    @staticmethod
    def commit(caches: List[SeqCache], res: BlockResult, n_commit) -> None:
        """Append the staged K/V of rows [0, n) of the last forward (exact caching)."""
        for b, c in enumerate(caches):
            n = int(n_commit[b])
            if n > res.n_causal[b]:
                raise ValueError("only causal rows can be committed")
            for li in range(len(c.K)):
                c.K[li] = np.concatenate([c.K[li], res.K_new[b][li][:n]], axis=0)
                c.V[li] = np.concatenate([c.V[li], res.V_new[b][li][:n]], axis=0)

    def prefill(self, tokens) -> tuple:
        """NTP forward over a prompt (all rows causal), then commit every row.

        Returns (cache, logits of the last prompt row).
        """
        tokens = np.asarray(tokens).reshape(1, -1)
        c = self.new_cache()
        res = self.block_forward([c], tokens, [tokens.shape[1]])
        self.commit([c], res, [tokens.shape[1]])
        return c, res.logits[0, -1]

    def full_forward(self, tokens, causal_point: int, pos=None) -> np.ndarray:
        """All rows at once, no cache, with the App. A inference mask over the whole sequence.

        Used to check that cached decoding is exact.  Returns logits [T][V].
        """
        s = self.s
        tokens = np.asarray(tokens).reshape(-1)
        T = tokens.shape[0]
        pos = np.arange(T) if pos is None else np.asarray(pos)
        q_idx = np.arange(T)[:, None]
        kv_idx = np.arange(T)[None, :]
        vis = (kv_idx <= q_idx) | (causal_point <= q_idx)
        x = self.W("embed")[tokens].astype(self.dtype)
        for li in range(s.n_layers):
            h = rms_norm(x, self.W("attn_norm", li), s.rms_eps)
            q, kk, vv = self._qkv(h, li, pos)
            o = attention(q, kk, vv, vis)
            x = x + o.reshape(T, -1) @ self.W("wo", li).T
            x = x + self._mlp(x, li)
        return rms_norm(x, self.W("final_norm"), s.rms_eps) @ self.W("lm_head").T


# ----------------------------------------------------------------------------- EB sampler


def row_entropy(logits_row, mask_id: int) -> tuple:
    """Entropy (nats) and argmax of softmax over the vocabulary without the mask token.

    With m the row maximum and t_v = l_v - m (float64): Z = sum e^t, S = sum e^t * t,
    H = log Z - S / Z, which equals -sum p log p for p = e^t / Z.
    The argmax is the smallest token id reaching the maximum.
    """
    l = np.asarray(logits_row, dtype=np.float32)
    keep = np.ones(l.shape[0], dtype=bool)
    if 0 <= mask_id < l.shape[0]:
        keep[mask_id] = False
    ids = np.nonzero(keep)[0]
    lv = l[ids]
    m = lv.max()
    tok = int(ids[np.argmax(lv == m)])
    t = lv.astype(np.float64) - np.float64(m)
    e = np.exp(t)
    Z = e.sum()
    S = (e * t).sum()
    return math.log(Z) - S / Z, tok


def row_confidence(logits_row, mask_id: int) -> float:
    """Confidence of a masked row (App. B): the largest probability of softmax over the
    vocabulary without the mask token, c = max_v p_v = e^0 / Z = 1 / Z with Z as in
    row_entropy (float64)."""
    l = np.asarray(logits_row, dtype=np.float32)
    keep = np.ones(l.shape[0], dtype=bool)
    if 0 <= mask_id < l.shape[0]:
        keep[mask_id] = False
    lv = l[keep]
    t = lv.astype(np.float64) - np.float64(lv.max())
    return 1.0 / np.exp(t).sum()


# Selection rules of one sampling step (Sec. 2.2 and App. B).
RULE_EB_ENTROPY, RULE_EB_CONFIDENCE, RULE_FACTOR = 0, 1, 2


def select_from_stats(H: Sequence[float], conf: Sequence[float], masked_rows: Sequence[int], rule: int,
                      threshold: float) -> List[int]:
    """Rows to reveal under one of the three rules, given per-row entropies and confidences.

    RULE_EB_ENTROPY: eq. (eb_sampler), threshold = gamma (eb_select_from_entropy).
    RULE_EB_CONFIDENCE: App. B, EB-Sampler with the confidence error proxy: the masked rows
      ordered by (confidence descending, row) as i_1..i_n; s is the largest r in [1, n] with
      sum_{j<=r} H_{i_j} - max_{j<=r} H_{i_j} <= gamma (sum left to right in float64).
    RULE_FACTOR: App. B, Factor parallel decoding: the same order; n is the largest r with
      (r + 1) * (1 - c_{i_r}) < f, at least 1 (the printed condition lacks the 1 - c; see
      the design notes).
    A row whose entropy or confidence is NaN (its softmax is undefined: no finite logit, a
    NaN or an infinite one) is never revealed and is left out of the order; with no other
    masked row nothing is revealed.  Returns the revealed rows sorted by row.
    """
    if rule == RULE_EB_ENTROPY:
        return eb_select_from_entropy(H, masked_rows, threshold)
    usable = [j for j in masked_rows if not (math.isnan(float(H[j])) or math.isnan(float(conf[j])))]
    order = sorted(usable, key=lambda j: (-float(conf[j]), int(j)))
    if not order:
        return []
    s = 1
    if rule == RULE_EB_CONFIDENCE:
        c = 0.0
        top = -math.inf
        for r, j in enumerate(order, start=1):
            c = c + float(H[j])
            top = max(top, float(H[j]))
            if c - top <= threshold:
                s = r
    elif rule == RULE_FACTOR:
        for r, j in enumerate(order, start=1):
            if (r + 1) * (1.0 - float(conf[j])) < threshold:
                s = r
    else:
        raise ValueError(f"unknown rule {rule}")
    return sorted(int(j) for j in order[:s])


def select(logits, is_mask, rule: int, threshold: float, mask_id: int) -> tuple:
    """One sampling step under `rule` on a batch of blocks.  Returns (accepted, tokens, H,
    conf): revealed rows (ascending), their argmax ids, and the entropies and confidences of
    the masked rows (nan elsewhere)."""
    logits = np.asarray(logits, dtype=np.float32)
    is_mask = np.asarray(is_mask).astype(bool)
    B, k, _ = logits.shape
    accepted, tokens = [], []
    H = np.full((B, k), np.nan)
    C = np.full((B, k), np.nan)
    for b in range(B):
        rows = [j for j in range(k) if is_mask[b, j]]
        toks = {}
        for j in rows:
            H[b, j], toks[j] = row_entropy(logits[b, j], mask_id)
            C[b, j] = row_confidence(logits[b, j], mask_id)
        acc = select_from_stats(H[b], C[b], rows, rule, threshold)
        accepted.append(acc)
        tokens.append([toks[j] for j in acc])
    return accepted, tokens, H, C


def eb_select_from_entropy(H: Sequence[float], masked_rows: Sequence[int], gamma: float) -> List[int]:
    """Eq. (eb_sampler): rows to reveal, given per-row entropies.

    Masked rows are ordered by (H, row) ascending as i_1..i_n; c_0 = 0 and
    c_r = c_{r-1} + H_{i_r}, summed left to right in float64; s is the largest
    r in [1, n] with c_{r-1} <= gamma (so s >= 1 whenever n >= 1).  Returns the first
    s rows of the order, sorted by row.  A row with a NaN entropy (undefined softmax) is
    left out of the order and never revealed.
    """
    usable = [j for j in masked_rows if not math.isnan(float(H[j]))]
    order = sorted(usable, key=lambda j: (float(H[j]), int(j)))
    s = 0
    c = 0.0
    for r, j in enumerate(order, start=1):
        if c <= gamma:
            s = r
        c = c + float(H[j])
    return sorted(int(j) for j in order[:s])


def eb_select(logits, is_mask, gamma: float, mask_id: int) -> tuple:
    """One EB-Sampler step on a batch of blocks (Sec. 2.2 and Alg. 3).

    logits: [B][k][V] float32; is_mask: [B][k].  Returns (accepted, tokens, H):
    accepted[b] = rows revealed (ascending), tokens[b] = their argmax ids,
    H[b][j] = entropy of masked rows (nan for unmasked rows).
    """
    logits = np.asarray(logits, dtype=np.float32)
    is_mask = np.asarray(is_mask).astype(bool)
    B, k, _ = logits.shape
    accepted, tokens = [], []
    H = np.full((B, k), np.nan)
    for b in range(B):
        rows = [j for j in range(k) if is_mask[b, j]]
        toks = {}
        for j in rows:
            H[b, j], toks[j] = row_entropy(logits[b, j], mask_id)
        acc = eb_select_from_entropy(H[b], rows, gamma)
        accepted.append(acc)
        tokens.append([toks[j] for j in acc])
    return accepted, tokens, H


def sample_blocks(model: "Model", caches: List[SeqCache], n_blocks: int, k: int, rule: int, threshold: float,
                  mask_id: int) -> tuple:
    """Alg. 2 after its prefill: n_blocks calls of Alg. 3 (Sample block) for every sequence.

    A block starts as k mask tokens.  While it holds masks: one forward of the network; in
    the first iteration of every block but the first, the previous block's k tokens enter
    as causal rows ahead of the block (the f(x_<t-k, x_t-k:t-1; x_hat) form of Alg. 3) and
    are committed to the cache afterwards; later iterations feed the block alone.  The
    block's rows are then unmasked by the selection rule (eq. (eb_sampler), or App. B), with
    argmax tokens (temperature 0, Sec. 3.1).  Sequences run in lockstep.
    Returns (tokens [B][n_blocks*k], trace): trace lists, per forward, the fed tokens,
    n_causal and the (accepted rows, tokens) of every sequence.
    """
    B = len(caches)
    out = [[] for _ in range(B)]
    trace = []
    prev = None
    for _ in range(n_blocks):
        xh = np.full((B, k), mask_id, dtype=np.int64)
        first = True
        while (xh == mask_id).any():
            if first and prev is not None:
                toks, nc, off = np.concatenate([prev, xh], axis=1), k, k
            else:
                toks, nc, off = xh.copy(), 0, 0
            res = model.block_forward(caches, toks, [nc] * B)
            if nc:
                Model.commit(caches, res, [k] * B)
            is_mask = (xh == mask_id).astype(np.uint8)
            acc, tk, _, _ = select(res.logits[:, off:off + k], is_mask, rule, threshold, mask_id)
            if any(is_mask[b].any() and not acc[b] for b in range(B)):
                raise RuntimeError("a block with masks left revealed nothing (no usable softmax in any masked row)")
            trace.append((toks.copy(), nc, acc, tk))
            for b in range(B):
                for j, t in zip(acc[b], tk[b]):
                    xh[b, j] = t
            first = False
        prev = xh.copy()
        for b in range(B):
            out[b].extend(int(t) for t in xh[b])
    return out, trace

"""Comparison helpers shared by the GPU parity tests (no test functions here).

Two bounds apply to every logits comparison:
* the contract: max-abs <= 5e-2 and rel-L2 <= 1e-2 of the fp32 oracle (bf16 path);
* a regression bound, about ten times the error the path is measured to have at that
  case, so that a change which makes the kernels much less accurate fails even while it
  stays inside the contract.

EB decisions on identical fp32 logits must agree exactly.  Both sides compute the
entropies in float64 with different summation orders (they agree to ~1e-12), so a
decision can only flip where the oracle's own margin is below that level; such cases are
reported as degenerate instead of failing: the margin of a selection is the smallest of
|c_{s-1} - gamma| (s >= 2), |c_s - gamma| and H_(s+1) - H_(s) (sorted entropies, running
sums c).
"""
import math

import numpy as np

CONTRACT_MAX_ABS, CONTRACT_REL_L2 = 5e-2, 1e-2
DEGENERATE_MARGIN = 1e-9


def errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = float(np.abs(got - ref).max())
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    return err, rel


def close(got, ref, regress=None, max_abs=CONTRACT_MAX_ABS, rel_l2=CONTRACT_REL_L2, label=""):
    """Assert the contract bound and, when given, the regression bound (max_abs, rel_l2)."""
    err, rel = errors(got, ref)
    print(f"    {label}max-abs {err:.3e}  rel-L2 {rel:.3e}", flush=True)
    assert err <= max_abs and rel <= rel_l2, f"{label}max-abs {err:.3e} rel-L2 {rel:.3e} (contract)"
    if regress is not None:
        assert err <= regress[0] and rel <= regress[1], \
            f"{label}max-abs {err:.3e} rel-L2 {rel:.3e} above the regression bound {regress}"
    return err, rel


def eb_margin(H, rows, gamma, s):
    """Decision margin of an EB selection that accepted s rows (see the module docstring)."""
    usable = sorted((j for j in rows if not math.isnan(H[j])), key=lambda j: (H[j], j))
    n = len(usable)
    c = [0.0]
    for j in usable:
        c.append(c[-1] + float(H[j]))
    m = math.inf
    if n == 0:
        return m
    if math.isfinite(gamma) and s >= 2:      # c_0 = 0 is exact: the first row needs no margin
        m = min(m, abs(c[s - 1] - gamma))
    if s < n:
        if math.isfinite(gamma):
            m = min(m, abs(c[s] - gamma))
        m = min(m, float(H[usable[s]]) - float(H[usable[s - 1]]))
    return m


def eb_compare(n_acc, pos, tok, ref_acc, ref_tok, ref_H, is_mask, gamma, label=""):
    """Compare the library's EB outputs with the oracle's, sequence by sequence; a mismatch is
    accepted only at a degenerate margin.  Returns the smallest margin seen."""
    n_acc, pos, tok = (np.asarray(a.cpu() if hasattr(a, "cpu") else a) for a in (n_acc, pos, tok))
    worst = math.inf
    for b in range(len(ref_acc)):
        rows = [j for j in range(is_mask.shape[1]) if is_mask[b, j]]
        n = int(n_acc[b])
        margin = eb_margin(ref_H[b], rows, gamma, len(ref_acc[b]))
        worst = min(worst, margin)
        same = pos[b, :n].tolist() == ref_acc[b] and tok[b, :n].tolist() == ref_tok[b]
        if not same:
            assert margin < DEGENERATE_MARGIN, (label, b, gamma, pos[b, :n].tolist(), ref_acc[b], margin)
            print(f"    {label}sequence {b} gamma {gamma}: degenerate decision (margin {margin:.2e})", flush=True)
        assert (pos[b, n:] == -1).all()
    print(f"    {label}gamma {gamma}: smallest EB decision margin {worst:.3e}", flush=True)
    return worst


def kv8_close(got, ref, scale_exp, max_frac=3e-3, label=""):
    """Keys/values of an e4m3 cache against the oracle's (both on the grid e4m3 * 2^e).

    The two sides round floats that agree to float precision, not bit for bit, so a value
    near the midpoint of two codes may land on either: at most max_frac of the elements may
    differ, each by one step of the grid (the larger spacing at a binade edge).  With the
    inputs agreeing to a relative 5e-5 (hi/lo activations), a flip has a chance of about
    2 * 5e-5 / 2^-3 = 8e-4 per element; layers whose inputs are bit-identical on both sides
    (layer 0) show none."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    s = 2.0 ** scale_exp
    mag = np.maximum(np.abs(got), np.abs(ref)) / s
    step = np.where(mag >= 2.0 ** -6, np.exp2(np.floor(np.log2(np.maximum(mag, 2.0 ** -6))) - 3), 2.0 ** -9) * s
    diff = got != ref
    n = int(diff.sum())
    print(f"    {label}{n} of {got.size} values one code apart", flush=True)
    assert n <= max_frac * got.size, f"{label}{n} of {got.size} e4m3 values differ"
    assert (np.abs(got - ref)[diff] <= step[diff]).all(), f"{label}values differ by more than one e4m3 step"

"""Set Block Decoding generation loop (Alg. 2 and Alg. 3 of the paper) over the C ABI.

Host control flow only: every forward, selection and cache update is a call into
libsbd.so (sbd_block_forward, sbd_select, sbd_commit); this module moves token ids and the
accepted rows between the host and those calls.
"""
from typing import Callable, List, Optional, Sequence

import numpy as np


def sample_blocks(lib, seq_ids: Sequence[int], n_blocks: int, k: int, rule: str = "eb_entropy",
                  threshold: float = 1.0, on_forward: Optional[Callable] = None) -> List[List[int]]:
    """Generate n_blocks blocks of k tokens for each sequence after its prefill (Alg. 2).

    Each block is Alg. 3: it starts as k mask tokens; while masks remain, one block
    forward, then the selection rule (`rule`, `threshold`: see sbd_select) reveals rows with
    their argmax tokens.  The first forward of every block but the first carries the
    previous block's k tokens as causal rows (n_causal = k, 2k rows) and commits them to
    the cache right after; later forwards feed the block alone (n_causal = 0).  Sequences
    run in lockstep.  on_forward(tokens, n_causal, n_accepted, accepted_pos, accepted_tok),
    if given, sees every step (host arrays).  Returns the generated ids per sequence.
    """
    s = lib.shape
    mask = s.mask_id
    ids = [int(b) for b in seq_ids]
    B = len(ids)
    out = [[] for _ in range(B)]
    prev = None
    for _ in range(n_blocks):
        xh = np.full((B, k), mask, dtype=np.int32)
        first = True
        while (xh == mask).any():
            if first and prev is not None:
                toks, nc = np.concatenate([prev, xh], axis=1), k
            else:
                toks, nc = xh.copy(), 0
            is_mask = (toks == mask).astype(np.uint8)
            logits = lib.block_forward(ids, toks, is_mask=is_mask, n_causal=[nc] * B)
            if nc:
                lib.commit(ids, [k] * B)
            # the causal rows are not masks, so only the block's rows are candidates
            n_acc, pos, tok, _, _ = lib.select(logits, is_mask, rule, threshold, mask)
            n_acc, pos, tok = n_acc.cpu().numpy(), pos.cpu().numpy(), tok.cpu().numpy()
            if on_forward is not None:
                on_forward(toks.copy(), nc, n_acc.copy(), pos.copy(), tok.copy())
            for b in range(B):
                if int(n_acc[b]) < 1 and (xh[b] == mask).any():
                    raise RuntimeError(f"sequence {ids[b]}: no masked row of the block has a usable softmax "
                                       "(every logit non-finite); nothing can be revealed")
                for i in range(int(n_acc[b])):
                    if int(tok[b, i]) < 0:
                        raise RuntimeError(f"sequence {ids[b]}: accepted row {int(pos[b, i])} has no token")
                    xh[b, int(pos[b, i]) - nc] = tok[b, i]
            first = False
        prev = xh.copy()
        for b in range(B):
            out[b].extend(int(t) for t in xh[b])
    return out

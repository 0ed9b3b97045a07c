"""Block partition and the block pairs the token predicate makes active
(oracle; test only).

Blocks follow the appendix's frame-aligned partition: each region (system
prefix, visual tokens, query tokens) of each video is cut into consecutive
blocks of B tokens counted from the region's start; a region's last block may
be short. A (query block, key block) pair is active when at least one token
pair in it is allowed. Blocks are listed in token order; the CSR lists each
query block's active key blocks in increasing order.
"""
from __future__ import annotations

import numpy as np

from .layout import Layout, Rule


def partition(lay: Layout, rule: Rule):
    """(start, length, region, video) of every block, in token order."""
    out = []
    for n in range(lay.n_seq):
        for a, e, reg in ((lay.tok0[n], lay.vis0[n], 0),
                          (lay.vis0[n], lay.txt0[n], 1),
                          (lay.txt0[n], lay.end[n], 2)):
            for s in range(int(a), int(e), rule.block):
                out.append((s, min(rule.block, int(e) - s), reg, n))
    return np.asarray(out, np.int64).reshape(-1, 4)


def active_csr(lay: Layout, rule: Rule, brute: bool = False):
    """CSR (row_ptr, col) of active block pairs.

    ``brute=True`` evaluates the predicate on every token pair of every
    video (small layouts only); otherwise each query token's allowed keys are
    enumerated and mapped to blocks.
    """
    blk = partition(lay, rule)
    tok2blk = np.zeros(lay.S, np.int64)
    for j, (s, ln, _, _) in enumerate(blk):
        tok2blk[s:s + ln] = j
    sets = [set() for _ in range(len(blk))]
    if brute:
        for n in range(lay.n_seq):
            t = np.arange(lay.tok0[n], lay.end[n])
            ok = lay.allowed(t[:, None], t[None, :], rule)
            ii, mm = np.nonzero(ok)
            for a, b in set(zip(tok2blk[t[ii]].tolist(),
                                tok2blk[t[mm]].tolist())):
                sets[a].add(b)
    else:
        for i in range(lay.S):
            sets[tok2blk[i]].update(
                np.unique(tok2blk[lay.allowed_keys(i, rule)]).tolist())
    row_ptr = np.zeros(len(blk) + 1, np.int64)
    cols = []
    for j, st in enumerate(sets):
        c = sorted(st)
        cols.extend(c)
        row_ptr[j + 1] = row_ptr[j] + len(c)
    return blk, row_ptr, np.asarray(cols, np.int64)

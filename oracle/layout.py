"""Token layout and visibility predicate (oracle; test infrastructure only).

Follows the appendix section "Detailed Sparse Prefilling":

* The context of one video is X = [X_sys; X_vis; X_Q]. The system prefix is
  visible to every later token and never takes part in block selection.
* Visual tokens are grouped per anchor frame (N_v consecutive tokens each) and
  partitioned into blocks of B tokens counted from the start of the visual
  region; the query tokens are partitioned on their own, the last block may be
  short. Blocks never mix videos ("belongs to the same input sample").
* The current block's causal prefix is always visible (the set E_i).

The block-sparse rule of the workloads replaces the paper's adaptive top-p
retention by a static one: a visual row in block b sees the first
``sink_blocks`` visual blocks, the ``window`` visual blocks before b and its
own block b (causally); a query row sees every visual block and the query
tokens up to itself. ``window = -1`` means all preceding visual blocks (plain
causal attention).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

SYS, VIS, TXT = 0, 1, 2


@dataclass(frozen=True)
class Rule:
    block: int
    sink_blocks: int
    window: int      # -1: unlimited


class Layout:
    """Per-token bookkeeping for a packed batch of videos."""

    def __init__(self, n_sys, n_frames, n_text, tokens_per_frame: int):
        self.n_sys = np.asarray(n_sys, np.int64)
        self.n_frames = np.asarray(n_frames, np.int64)
        self.n_text = np.asarray(n_text, np.int64)
        self.Nv = int(tokens_per_frame)
        self.n_seq = len(self.n_frames)
        self.n_vis = self.n_frames * self.Nv
        lens = self.n_sys + self.n_vis + self.n_text
        self.tok0 = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
        self.vis0 = self.tok0 + self.n_sys
        self.txt0 = self.vis0 + self.n_vis
        self.end = self.tok0 + lens
        self.S = int(self.end[-1]) if self.n_seq else 0
        self.frame0 = np.concatenate(
            [[0], np.cumsum(self.n_frames)[:-1]]).astype(np.int64)
        self.T = int(self.n_frames.sum())
        self.textrow0 = np.concatenate(
            [[0], np.cumsum(self.n_text)[:-1]]).astype(np.int64)
        # per-token tables
        seq = np.zeros(self.S, np.int64)
        region = np.zeros(self.S, np.int64)
        rpos = np.zeros(self.S, np.int64)
        frame = np.full(self.S, -1, np.int64)
        for n in range(self.n_seq):
            a, v, t, e = self.tok0[n], self.vis0[n], self.txt0[n], self.end[n]
            seq[a:e] = n
            region[a:v] = SYS
            region[v:t] = VIS
            region[t:e] = TXT
            rpos[a:v] = np.arange(v - a)
            rpos[v:t] = np.arange(t - v)
            rpos[t:e] = np.arange(e - t)
            frame[v:t] = self.frame0[n] + np.arange(t - v) // self.Nv
        self.seq, self.region, self.rpos, self.frame = seq, region, rpos, frame

    # ------------------------------------------------------------------
    def allowed(self, i, m, rule: Rule):
        """Token predicate: may query token i attend to key token m?

        Vectorised over broadcastable integer arrays ``i`` and ``m``.
        """
        i = np.asarray(i)
        m = np.asarray(m)
        same = self.seq[i] == self.seq[m]
        causal = m <= i
        ri, rm = self.region[i], self.region[m]
        key_sys = rm == SYS
        qb = self.rpos[i] // rule.block
        kb = self.rpos[m] // rule.block
        in_sink = kb < rule.sink_blocks
        if rule.window < 0:
            in_win = np.ones_like(kb, dtype=bool)
        else:
            in_win = (kb >= qb - rule.window) & (kb <= qb)
        vis_row = (ri == VIS) & (rm == VIS) & (in_sink | in_win)
        txt_row = (ri == TXT) & ((rm == VIS) | (rm == TXT))
        return same & causal & (key_sys | vis_row | txt_row)

    def allowed_keys(self, i: int, rule: Rule) -> np.ndarray:
        """Sorted key tokens visible to query token i, enumerated from the
        rule's definition (not from the predicate; tests check they agree)."""
        n = self.seq[i]
        keys = [np.arange(self.tok0[n], min(self.vis0[n], i + 1))]
        if self.region[i] == VIS:
            qb = self.rpos[i] // rule.block
            nb = -(-int(self.n_vis[n]) // rule.block)
            blocks = set(range(min(rule.sink_blocks, nb)))
            lo = 0 if rule.window < 0 else max(0, qb - rule.window)
            blocks.update(range(lo, qb + 1))
            for b in sorted(blocks):
                a = self.vis0[n] + b * rule.block
                e = min(self.txt0[n], a + rule.block, i + 1)
                if e > a:
                    keys.append(np.arange(a, e))
        elif self.region[i] == TXT:
            keys.append(np.arange(self.vis0[n], i + 1))
        return np.concatenate(keys).astype(np.int64)

    def text_rows(self, n=None) -> np.ndarray:
        if n is None:
            return np.concatenate([np.arange(self.txt0[k], self.end[k])
                                   for k in range(self.n_seq)]).astype(np.int64)
        return np.arange(self.txt0[n], self.end[n], dtype=np.int64)

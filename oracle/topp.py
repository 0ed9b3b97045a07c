"""Adaptive top-p block retention and the attention it induces (oracle; test
infrastructure only).

Follows the appendix section "Detailed Sparse Prefilling", step by step:

1. Blocks. The visual tokens and the query tokens of a video are cut into
   region-relative blocks of B tokens (``layout``); the system prefix takes
   no part in selection. A video's selectable blocks are numbered 0, 1, ...
   in token order (visual blocks, then query-token blocks): the *local*
   block index used below.
2. Block representative (mean-key equation): kbar_j = (1/|K_j|) sum of the
   block's key vectors, per kv head.
3. History H_i (definition after the mean-key equation): the blocks of the
   same video that end before position i. For a row in local block b these
   are exactly the local blocks 0 .. b-1; the row's own block is not in
   H_i.
4. Block affinity g_ij = q_i . kbar_j / sqrt(d) over H_i (affinity
   equation), normalised by a softmax over H_i (probability equation).
5. Retention: rank H_i by p_ij, descending, and keep the smallest subset
   whose cumulative probability reaches tau_p; every other history block is
   masked out.
6. Attention of row i then runs over the causally valid system-prefix
   tokens, the causal prefix of its own block (the set E_i of the coarse-map
   equation) and every token of the retained blocks, with exact logits
   q_i . k_m / sqrt(d).

Readings where the text leaves a choice (each is listed with the design
notes):

* Equal probabilities are ranked by ascending block index (a stable sort).
* If rounding keeps the cumulative probability of the whole history below
  tau_p, the whole history is retained.
* H_i counts the query-token blocks before the row's block as well as the
  visual blocks: both are blocks of the same sample that end before i.
* Selection is per query head (q_i is the head's projected query) against
  the kbar of that head's kv head.

Everything is float64 unless a caller passes ``dtype=np.float32`` for the
probability arithmetic of step 4-5.
"""
from __future__ import annotations

import numpy as np

from .layout import Layout, SYS, VIS, TXT
from .attention import _softmax


class Blocks:
    """Selectable (non-system) blocks of every video, in token order."""

    def __init__(self, lay: Layout, block: int):
        self.lay = lay
        self.B = int(block)
        self.start, self.len, self.region, self.seq = [], [], [], []
        self.first = np.zeros(lay.n_seq, np.int64)   # first block of video n
        self.count = np.zeros(lay.n_seq, np.int64)
        for n in range(lay.n_seq):
            self.first[n] = len(self.start)
            for a, e, reg in ((lay.vis0[n], lay.txt0[n], VIS),
                              (lay.txt0[n], lay.end[n], TXT)):
                for s in range(int(a), int(e), self.B):
                    self.start.append(s)
                    self.len.append(min(self.B, int(e) - s))
                    self.region.append(reg)
                    self.seq.append(n)
            self.count[n] = len(self.start) - self.first[n]
        self.start = np.asarray(self.start, np.int64)
        self.len = np.asarray(self.len, np.int64)
        self.region = np.asarray(self.region, np.int64)
        self.seq = np.asarray(self.seq, np.int64)
        # local block index of every token (-1 for system-prefix tokens)
        self.local = np.full(lay.S, -1, np.int64)
        for gb in range(self.start.size):
            n = self.seq[gb]
            a = self.start[gb]
            self.local[a:a + self.len[gb]] = gb - self.first[n]

    @property
    def max_count(self) -> int:
        return int(self.count.max()) if self.count.size else 0

    def history(self, i: int) -> np.ndarray:
        """Local indices of H_i: blocks of i's video whose last token comes
        before i (system tokens have no selectable history)."""
        if self.local[i] < 0:
            return np.zeros(0, np.int64)
        return np.arange(self.local[i], dtype=np.int64)

    def tokens(self, n: int, j: int) -> np.ndarray:
        gb = self.first[n] + j
        return np.arange(self.start[gb], self.start[gb] + self.len[gb])


def mean_keys(k: np.ndarray, blk: Blocks) -> np.ndarray:
    """kbar [n_blocks_total, Hkv, d]: mean of each selectable block's keys."""
    out = np.zeros((blk.start.size, k.shape[1], k.shape[2]))
    for gb in range(blk.start.size):
        a, ln = blk.start[gb], blk.len[gb]
        out[gb] = k[a:a + ln].sum(axis=0) / ln
    return out


def retain(g: np.ndarray, tau: float, dtype=np.float64):
    """Top-p retention of one or more rows of affinities ``g [R, n]``.

    Returns ``(keep [R, n] bool, info)`` where ``info`` holds, per row, the
    probabilities ``p``, the retained count ``k``, the cumulative mass just
    before and at the cut (``c_before``, ``c_at``) and the probabilities of
    the last retained and first dropped block (``p_last``, ``p_next``).
    """
    g = np.asarray(g, dtype)
    R, n = g.shape
    keep = np.zeros((R, n), bool)
    info = {"p": np.zeros((R, n), dtype), "k": np.zeros(R, np.int64),
            "c_before": np.zeros(R), "c_at": np.zeros(R),
            "p_last": np.zeros(R), "p_next": np.zeros(R)}
    if n == 0:
        return keep, info
    mx = g.max(axis=1, keepdims=True)
    e = np.exp(g - mx)
    p = e / e.sum(axis=1, keepdims=True)
    info["p"] = p
    tau = dtype(tau)
    for r in range(R):
        order = np.argsort(-p[r], kind="stable")   # ties: lower index first
        c = np.cumsum(p[r, order])
        hit = np.nonzero(c >= tau)[0]
        kk = int(hit[0]) + 1 if hit.size else n
        keep[r, order[:kk]] = True
        info["k"][r] = kk
        info["c_before"][r] = c[kk - 2] if kk >= 2 else 0.0
        info["c_at"][r] = c[kk - 1]
        info["p_last"][r] = p[r, order[kk - 1]]
        info["p_next"][r] = p[r, order[kk]] if kk < n else -1.0
    return keep, info


def select(q: np.ndarray, k: np.ndarray, lay: Layout, blk: Blocks,
           tau: float, scale: float, rows=None, dtype=np.float64):
    """Retained history blocks of every (query head, row).

    Returns ``(keep [Hq, R, max_count] bool, info)``; ``info`` holds the
    per-(head, row) arrays of ``retain`` (``k``, ``c_before``, ``c_at``,
    ``p_last``, ``p_next``) and ``nh`` (= |H_i|). Rows without history
    (system tokens, a video's first block) retain nothing.
    """
    if rows is None:
        rows = np.arange(lay.S, dtype=np.int64)
    rows = np.asarray(rows, np.int64)
    hq, hkv = q.shape[1], k.shape[1]
    grp = hq // hkv
    kbar = mean_keys(k, blk)
    keep = np.zeros((hq, rows.size, max(blk.max_count, 1)), bool)
    names = ("k", "c_before", "c_at", "p_last", "p_next")
    info = {nm: np.zeros((hq, rows.size)) for nm in names}
    info["nh"] = np.zeros(rows.size, np.int64)
    # rows of one local block share H_i: handle them together
    key = [(int(lay.seq[i]), int(blk.local[i])) for i in rows]
    groups = {}
    for j, kk in enumerate(key):
        groups.setdefault(kk, []).append(j)
    for (n, lb), idx in groups.items():
        idx = np.asarray(idx)
        info["nh"][idx] = max(lb, 0)
        if lb <= 0:
            continue
        hist = kbar[blk.first[n]:blk.first[n] + lb]          # [lb, Hkv, d]
        for h in range(hq):
            gmat = (q[rows[idx], h, :] @ hist[:, h // grp, :].T) * scale
            kp, inf = retain(gmat, tau, dtype)
            keep[h, idx, :lb] = kp
            for nm in names:
                info[nm][h, idx] = inf[nm]
    return keep, info


def allowed_keys(lay: Layout, blk: Blocks, i: int, kept_local) -> np.ndarray:
    """Keys of row i under retention: causal system prefix, the causal
    prefix of the row's own block and all tokens of the retained blocks."""
    n = lay.seq[i]
    parts = [np.arange(lay.tok0[n], min(lay.vis0[n], i + 1))]
    lb = blk.local[i]
    if lb >= 0:
        for j in sorted(int(x) for x in kept_local):
            assert j < lb
            parts.append(blk.tokens(n, j))
        gb = blk.first[n] + lb
        parts.append(np.arange(blk.start[gb], i + 1))
    return np.concatenate(parts).astype(np.int64)


def attend(q, k, v, lay: Layout, blk: Blocks, keep, rows, scale: float,
           want_p: bool = False):
    """Attention output and LSE of ``rows`` with per-(head, row) retention
    ``keep [Hq, R, max_count]`` (rows in the same order as ``rows``).

    Rows of one video and one local block share their candidate keys (the
    video's tokens up to the last of them); each (head, row) keeps the keys
    ``allowed_keys`` names, the others get logit -inf. Returns
    ``O [R, Hq, d]``, ``LSE [Hq, R]`` and, if ``want_p``, per group the
    triple (row indices into ``rows``, keys, P [Hq, r, keys])."""
    rows = np.asarray(rows, np.int64)
    hq, hkv, d = q.shape[1], k.shape[1], q.shape[2]
    grp = hq // hkv
    O = np.zeros((rows.size, hq, d))
    LSE = np.zeros((hq, rows.size))
    plist = []
    groups = {}
    for j, i in enumerate(rows):
        groups.setdefault((int(lay.seq[i]), int(blk.local[i])), []).append(j)
    for (n, lb), idx in groups.items():
        idx = np.asarray(idx)
        ri = rows[idx]
        keys = np.arange(lay.tok0[n], ri.max() + 1, dtype=np.int64)
        lk = blk.local[keys]
        causal = keys[None, :] <= ri[:, None]
        base = causal & ((lk[None, :] < 0) | (lk[None, :] == lb))
        hist = (lk >= 0) & (lk < max(lb, 0))
        ps = []
        for h in range(hq):
            ok = base.copy()
            if lb > 0:
                kept = keep[h][idx][:, lk[hist]]        # [r, n_hist_keys]
                ok[:, hist] |= kept & causal[:, hist]
            s = (q[ri, h, :] @ k[keys, h // grp, :].T) * scale
            s = np.where(ok, s, -np.inf)
            p, lse = _softmax(s)
            O[idx, h] = p @ v[keys, h // grp, :]
            LSE[h, idx] = lse
            if want_p:
                ps.append(p)
        if want_p:
            plist.append((idx, keys, ps))
    return O, LSE, plist


def evidence(q, k, v, lay: Layout, blk: Blocks, keep_txt, rows_txt,
             scale: float):
    """Query-frame evidence under retention (same definition as the static
    path: per frame, the raw sum over the video's query rows of their
    softmax mass on the frame's visual keys; text_mass takes the rest)."""
    hq = q.shape[1]
    E = np.zeros((hq, lay.T))
    tm = np.zeros((hq, lay.n_seq))
    O, LSE, plist = attend(q, k, v, lay, blk, keep_txt, rows_txt, scale,
                           want_p=True)
    for idx, keys, ps in plist:
        n = lay.seq[rows_txt[idx[0]]]
        vis = lay.region[keys] == VIS
        for h in range(hq):
            col = ps[h].sum(axis=0)                  # sum over query rows
            E[h] += np.bincount(lay.frame[keys[vis]], weights=col[vis],
                                minlength=lay.T)
            tm[h, n] += col[~vis].sum()
    return E, tm, O, LSE


def run_layer(q, k, v, lay: Layout, block: int, tau: float, scale: float,
              rows=None, dtype=np.float64):
    """Oracle for one layer under adaptive top-p retention.

    Returns a dict with the retention of the requested rows (``keep``,
    ``info``), ``O``/``LSE`` of those rows, and ``E``/``text_mass`` from all
    query rows (whose retention is ``keep_txt``/``info_txt``)."""
    blk = Blocks(lay, block)
    if rows is None:
        rows = np.arange(lay.S, dtype=np.int64)
    rows = np.asarray(rows, np.int64)
    txt = lay.text_rows()
    keep_t, info_t = select(q, k, lay, blk, tau, scale, txt, dtype)
    E, tm, _, _ = evidence(q, k, v, lay, blk, keep_t, txt, scale)
    keep, info = select(q, k, lay, blk, tau, scale, rows, dtype)
    O, LSE, _ = attend(q, k, v, lay, blk, keep, rows, scale)
    return {"rows": rows, "keep": keep, "info": info, "O": O, "LSE": LSE,
            "E": E, "text_mass": tm, "rows_txt": txt, "keep_txt": keep_t,
            "info_txt": info_t, "blocks": blk}

"""Masked-softmax attention and query-frame evidence (oracle; test only).

Definitions followed:

* Attention logits are q_i . k_m / sqrt(d) (appendix, block-affinity
  equation: the scale is the head dimension's square root; the same scale
  applies to the exact logits of the coarse map).
* A row's softmax runs over exactly the keys the visibility predicate allows
  (block-sparse attention with the retained blocks plus the exact causal
  prefix of the current block; appendix, coarse-map equation, first case).
* Grouped-query attention: q head h reads kv head floor(h / (Hq / Hkv)).
* Query-frame evidence (Evidence Decomposition): the complete query-token
  group's attention to each anchor frame's visual tokens. Here E[h, f] is the
  raw sum over the query rows i of video(f) of the softmax mass P_im over the
  visual keys m of frame f; ``text_mass[h, n]`` is the same rows' mass on the
  non-visual keys (system prefix and query tokens). Per row, the two add up
  to one.

Everything is float64. Rows are processed in small groups for vectorisation;
the grouping has no effect on the result because every logit is masked by the
token predicate before the softmax.
"""
from __future__ import annotations

import numpy as np

from .layout import Layout, Rule, SYS, VIS, TXT


def _softmax(s: np.ndarray):
    """Row softmax of logits with -inf for masked keys; returns (P, LSE)."""
    mx = s.max(axis=1, keepdims=True)
    p = np.exp(s - mx)
    z = p.sum(axis=1, keepdims=True)
    return p / z, (mx + np.log(z))[:, 0]


def _row_groups(lay: Layout, rows: np.ndarray, group: int):
    """Split ``rows`` into runs of consecutive tokens of one video and one
    region, at most ``group`` long."""
    rows = np.asarray(rows, np.int64)
    if rows.size == 0:
        return
    start = 0
    for j in range(1, rows.size + 1):
        brk = (j == rows.size or rows[j] != rows[j - 1] + 1
               or lay.seq[rows[j]] != lay.seq[rows[start]]
               or lay.region[rows[j]] != lay.region[rows[start]]
               or j - start >= group)
        if brk:
            yield rows[start:j]
            start = j


def _candidates(lay: Layout, grp: np.ndarray, rule: Rule, mode: str):
    n = lay.seq[grp[0]]
    if mode == "dense":
        return np.arange(lay.tok0[n], grp[-1] + 1, dtype=np.int64)
    keys = np.unique(np.concatenate([lay.allowed_keys(int(i), rule)
                                     for i in grp]))
    return keys


def attend(q, k, v, lay: Layout, rule: Rule, scale: float, rows,
           mode: str = "allowed", group: int = 64, want_p: bool = False):
    """Attention output and log-sum-exp for query tokens ``rows``.

    q: [S, Hq, d], k/v: [S, Hkv, d] (float64). Returns ``O [R, Hq, d]``,
    ``LSE [Hq, R]`` and, if ``want_p``, a list of (row_group, keys, P[Hq])
    triples holding each group's normalised probabilities.
    """
    rows = np.asarray(rows, np.int64)
    hq, hkv, d = q.shape[1], k.shape[1], q.shape[2]
    grp_size = hq // hkv
    O = np.zeros((rows.size, hq, d))
    LSE = np.zeros((hq, rows.size))
    where = {int(r): j for j, r in enumerate(rows)}
    plist = []
    for grp in _row_groups(lay, rows, group):
        keys = _candidates(lay, grp, rule, mode)
        ok = lay.allowed(grp[:, None], keys[None, :], rule)
        idx = np.array([where[int(r)] for r in grp])
        ps = []
        for h in range(hq):
            g = h // grp_size
            s = (q[grp, h, :] @ k[keys, g, :].T) * scale
            s = np.where(ok, s, -np.inf)
            p, lse = _softmax(s)
            O[idx, h, :] = p @ v[keys, g, :]
            LSE[h, idx] = lse
            if want_p:
                ps.append(p)
        if want_p:
            plist.append((grp, keys, ps))
    return O, LSE, plist


def evidence(q, k, v, lay: Layout, rule: Rule, scale: float,
             mode: str = "allowed"):
    """Query-frame evidence of one layer.

    Returns ``(E [Hq, T], text_mass [Hq, n_seq], O_txt, LSE_txt, rows_txt)``
    where the last three are the query rows' outputs (computed on the way).
    """
    hq = q.shape[1]
    E = np.zeros((hq, lay.T))
    tm = np.zeros((hq, lay.n_seq))
    rows = lay.text_rows() if lay.n_seq else np.zeros(0, np.int64)
    O, LSE, plist = attend(q, k, v, lay, rule, scale, rows, mode=mode,
                           group=1 << 30, want_p=True)
    for grp, keys, ps in plist:
        n = lay.seq[grp[0]]
        vis = lay.region[keys] == VIS
        fr = lay.frame[keys[vis]]
        for h in range(hq):
            colmass = ps[h].sum(axis=0)            # sum over the query rows
            E[h] += np.bincount(fr, weights=colmass[vis], minlength=lay.T)
            tm[h, n] += colmass[~vis].sum()
    return E, tm, O, LSE, rows


def run_layer(q, k, v, lay: Layout, rule: Rule, scale: float, rows=None,
              mode: str = "allowed"):
    """Oracle for one layer.

    Returns a dict with ``rows``, ``O [R, Hq, d]``, ``LSE [Hq, R]`` for the
    requested rows (all rows if None), and ``E [Hq, T]``, ``text_mass
    [Hq, n_seq]`` from all query rows.
    """
    if rows is None:
        rows = np.arange(lay.S, dtype=np.int64)
    rows = np.asarray(rows, np.int64)
    E, tm, _, _, _ = evidence(q, k, v, lay, rule, scale, mode=mode)
    O, LSE, _ = attend(q, k, v, lay, rule, scale, rows, mode=mode)
    return {"rows": rows, "O": O, "LSE": LSE, "E": E, "text_mass": tm}


def dense_reference(q, k, v, lay: Layout, rule: Rule, scale: float):
    """Whole-matrix form for small inputs: all S x S logits per head, masked
    by the predicate, row softmax, P V, and the evidence sums read off P."""
    S, hq, d = q.shape
    hkv = k.shape[1]
    i = np.arange(S)
    ok = lay.allowed(i[:, None], i[None, :], rule)
    O = np.zeros((S, hq, d))
    LSE = np.zeros((hq, S))
    E = np.zeros((hq, lay.T))
    tm = np.zeros((hq, lay.n_seq))
    txt = lay.region == TXT
    vis = lay.region == VIS
    for h in range(hq):
        g = h // (hq // hkv)
        s = np.where(ok, (q[:, h, :] @ k[:, g, :].T) * scale, -np.inf)
        p, LSE[h] = _softmax(s)
        O[:, h, :] = p @ v[:, g, :]
        for n in range(lay.n_seq):
            rows = txt & (lay.seq == n)
            col = p[rows].sum(axis=0)
            E[h] += np.bincount(lay.frame[vis], weights=col[vis],
                                minlength=lay.T)
            tm[h, n] = col[~vis].sum()
    return {"O": O, "LSE": LSE, "E": E, "text_mass": tm}

"""The paper's coarse attention map and the sparse-vs-dense alignment
metrics (oracle; test infrastructure only).

Coarse map (appendix, coarse-map equation and the row normalisation after
it): for query token i,
    a_im = q_i . k_m / sqrt(d)  for m in E_i (the causally valid system
                                 prefix and the causal prefix of i's block),
    a_im = g_ij                 for m in a retained block j in S_i (g the
                                 block affinity of the top-p step),
    a_im = -inf                 otherwise,
and A~_im = exp(a_im) / sum_n exp(a_in). Heads are averaged and the cues are
sliced from it exactly as from the exact map (``cues``, ``attention``):
A_qf from the query rows, A_ff between frames, A_if inside frames.

Alignment metrics (Reliability of Sparse Attention Maps; the paper names
them without formulas, the readings are listed with the design notes): a
sparse map s and a dense map t over the same positions, both non-negative:
* Pearson and Spearman correlation of the flattened maps;
* JS: Jensen-Shannon divergence (natural log) of s / sum s and t / sum t;
* Top-10 %: |top-k(s) & top-k(t)| / k with k = ceil(0.1 n) (ties broken by
  position);
* Keep: fraction of positions the sparse map keeps (s > 0);
* Mass-rec: the dense mass on the kept positions, sum_{s>0} t / sum t.
"""
from __future__ import annotations

import math

import numpy as np

from .layout import Layout, SYS, VIS, TXT
from . import topp


def coarse_probs(q, k, lay: Layout, blk, keep, rows, scale: float):
    """A~ rows of ``rows`` per head: a list of (row tokens, keys,
    P [Hq, r, m]) groups; ``keep [Hq, R, max_count]`` is the top-p
    retention of ``rows`` (in ``rows`` order)."""
    rows = np.asarray(rows, np.int64)
    hq, hkv = q.shape[1], k.shape[1]
    grp = hq // hkv
    kbar = topp.mean_keys(k, blk)
    groups = {}
    for j, i in enumerate(rows):
        groups.setdefault((int(lay.seq[i]), int(blk.local[i])), []).append(j)
    out = []
    for (n, lb), idx in groups.items():
        idx = np.asarray(idx)
        ri = rows[idx]
        keys = np.arange(lay.tok0[n], ri.max() + 1, dtype=np.int64)
        lk = blk.local[keys]
        causal = keys[None, :] <= ri[:, None]
        exact = causal & ((lk[None, :] < 0) | (lk[None, :] == lb))
        hist = (lk >= 0) & (lk < max(lb, 0))
        ps = []
        for h in range(hq):
            s = (q[ri, h, :] @ k[keys, h // grp, :].T) * scale
            a = np.where(exact, s, -np.inf)
            if lb > 0:
                gj = (q[ri, h, :] @ kbar[blk.first[n]:blk.first[n] + lb,
                                         h // grp, :].T) * scale   # [r, lb]
                kept = keep[h][idx][:, :lb]                          # [r, lb]
                g_tok = gj[:, lk[hist]]                              # [r, m]
                a[:, hist] = np.where(kept[:, lk[hist]], g_tok, -np.inf)
            mx = a.max(axis=1, keepdims=True)
            e = np.exp(a - mx)
            ps.append(e / e.sum(axis=1, keepdims=True))
        out.append((ri, keys, np.stack(ps)))
    return out


def query_frame(lay: Layout, groups, hq: int):
    """E[h, f]: raw sums over the query rows of their mass on each frame
    (the kernel's evidence slice), from (row tokens, keys, P) groups; other
    rows are ignored."""
    E = np.zeros((hq, lay.T))
    for ri, keys, P in groups:
        txt = lay.region[ri] == TXT
        if not txt.any():
            continue
        vis = lay.region[keys] == VIS
        for h in range(hq):
            col = P[h][txt][:, vis].sum(axis=0)
            E[h] += np.bincount(lay.frame[keys[vis]], weights=col,
                                minlength=lay.T)
    return E


def dense_groups(q, k, v, lay: Layout, rows, scale: float):
    """Dense causal attention (every earlier key of the video) of ``rows``
    as (rows, keys, P) groups: the reference the sparse maps are compared
    with."""
    from .attention import attend
    from .layout import Rule
    rule = Rule(1 << 30, 0, -1)      # one block per region: causal
    _, _, plist = attend(q, k, v, lay, rule, scale, rows, mode="dense",
                         want_p=True)
    for grp, keys, ps in plist:
        yield grp, keys, np.stack(ps)


# ---------------------------------------------------------------------------
# alignment metrics

def _ranks(x):
    """Average ranks (1-based) with ties sharing their mean rank."""
    order = np.argsort(x, kind="stable")
    r = np.empty(len(x))
    xs = x[order]
    i = 0
    while i < len(x):
        j = i
        while j + 1 < len(x) and xs[j + 1] == xs[i]:
            j += 1
        r[order[i:j + 1]] = (i + j) / 2.0 + 1.0
        i = j + 1
    return r


def pearson(s, t):
    s = np.asarray(s, np.float64).ravel()
    t = np.asarray(t, np.float64).ravel()
    sc, tc = s - s.mean(), t - t.mean()
    den = math.sqrt(float((sc * sc).sum()) * float((tc * tc).sum()))
    return float((sc * tc).sum() / den) if den > 0 else 0.0


def spearman(s, t):
    return pearson(_ranks(np.asarray(s, np.float64).ravel()),
                   _ranks(np.asarray(t, np.float64).ravel()))


def js_divergence(s, t):
    p = np.asarray(s, np.float64).ravel()
    q = np.asarray(t, np.float64).ravel()
    p, q = p / p.sum(), q / q.sum()
    m = 0.5 * (p + q)

    def kl(a, b):
        nz = a > 0
        return float((a[nz] * np.log(a[nz] / b[nz])).sum())
    return 0.5 * kl(p, m) + 0.5 * kl(q, m)


def top_overlap(s, t, frac=0.1):
    s = np.asarray(s, np.float64).ravel()
    t = np.asarray(t, np.float64).ravel()
    kk = max(1, int(math.ceil(frac * s.size)))
    ts = set(np.argsort(-s, kind="stable")[:kk].tolist())
    tt = set(np.argsort(-t, kind="stable")[:kk].tolist())
    return len(ts & tt) / kk


def keep_ratio(s):
    s = np.asarray(s, np.float64).ravel()
    return float((s > 0).mean())


def mass_recovery(s, t):
    s = np.asarray(s, np.float64).ravel()
    t = np.asarray(t, np.float64).ravel()
    return float(t[s > 0].sum() / t.sum())


def alignment(s, t):
    """All six metrics of a sparse map ``s`` against a dense map ``t``."""
    return {"pearson": pearson(s, t), "spearman": spearman(s, t),
            "js": js_divergence(s, t), "top10": top_overlap(s, t),
            "keep": keep_ratio(s), "mass_rec": mass_recovery(s, t)}

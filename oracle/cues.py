"""Cross-frame and intra-frame evidence cues (oracle; test infrastructure only).

Evidence Decomposition: attention maps are averaged over heads with the layer
kept; the visual blocks of each anchor frame are located in them, and

* the cross-frame cue A_ff holds, for every frame a and every earlier frame
  b of the same video, the averaged attention from a's visual tokens to b's.
  Reading taken: A_ff[a, b] = (1 / (Hq N_v)) sum_h sum_{i in a} sum_{m in b}
  P^h_im, i.e. the mean over a's query rows (and heads) of the row's total
  probability on b's keys (keys summed, as for the query-frame cue);
* the timestamp-aligned cross-frame evidence E_ff averages, per frame t, the
  attention t assigns to its preceding frames, out(t) = mean_{b < t}
  A_ff[t, b], and the attention it receives from its subsequent frames,
  in(t) = mean_{a > t} A_ff[a, t]; a video's first frame has only in(t),
  its last only out(t), and a single-frame video has E_ff = 0;
* the intra-frame cue A_if keeps, per frame t, the token-level causal
  attention among its own visual tokens: A_if[t][i][m] = (1 / Hq) sum_h
  P^h_{i m} for query token i and key token m of frame t (0 for m > i);
  E_if is A_if flattened per timestamp.

P^h is the attention of the sparse pass itself (the exact masked softmax of
whichever rule produced it), so pairs outside the pattern are 0.
"""
from __future__ import annotations

import numpy as np

from .layout import Layout, VIS


def accumulate(lay: Layout, groups, hq: int):
    """Sum head-summed probabilities into frame-pair and intra-frame maps.

    ``groups`` yields ``(rows, keys, P)`` with P [Hq, len(rows), len(keys)]
    the normalised probabilities of visual query rows. Returns
    ``(A_ff [T, T], A_if [T, N_v, N_v])``, already averaged (A_ff over heads
    and the N_v rows of the query frame, A_if over heads). A_ff is filled
    for b < a within a video only.
    """
    T, Nv = lay.T, lay.Nv
    aff = np.zeros((T, T))
    aif = np.zeros((T, Nv, Nv))
    for rows, keys, P in groups:
        Ps = np.asarray(P).sum(axis=0)                  # [r, m]
        kfr = lay.frame[keys]
        vis = lay.region[keys] == VIS
        kv = keys[vis]
        for j, i in enumerate(rows):
            if lay.region[i] != VIS:
                continue
            a = lay.frame[i]
            aff[a] += np.bincount(kfr[vis], weights=Ps[j, vis], minlength=T)
            same = kfr[vis] == a
            ii = (i - lay.vis0[lay.seq[i]]) % Nv
            mm = (kv[same] - lay.vis0[lay.seq[i]]) % Nv
            aif[a, ii, mm] += Ps[j, vis][same]
    aff /= hq * Nv
    aif /= hq
    tri = np.zeros((T, T), bool)
    for n in range(lay.n_seq):
        f0, F = int(lay.frame0[n]), int(lay.n_frames[n])
        tri[f0:f0 + F, f0:f0 + F] = np.tril(np.ones((F, F), bool), -1)
    return np.where(tri, aff, 0.0), aif


def e_ff(lay: Layout, A_ff: np.ndarray) -> np.ndarray:
    """Timestamp-aligned cross-frame evidence [T] from A_ff [T, T]."""
    out = np.zeros(lay.T)
    for n in range(lay.n_seq):
        f0, F = int(lay.frame0[n]), int(lay.n_frames[n])
        A = A_ff[f0:f0 + F, f0:f0 + F]
        for t in range(F):
            sides = []
            if t > 0:
                sides.append(A[t, :t].sum() / t)
            if t < F - 1:
                sides.append(A[t + 1:, t].sum() / (F - 1 - t))
            out[f0 + t] = np.mean(sides) if sides else 0.0
    return out


def static_groups(q, k, v, lay: Layout, rule, scale: float, rows=None):
    """(rows, keys, P) groups of the static-rule oracle for visual rows."""
    from .attention import attend
    if rows is None:
        rows = np.nonzero(lay.region == VIS)[0]
    _, _, plist = attend(q, k, v, lay, rule, scale, rows, want_p=True)
    for grp, keys, ps in plist:
        yield grp, keys, np.stack(ps)


def topp_groups(q, k, v, lay: Layout, blk, keep, rows, scale: float):
    """(rows, keys, P) groups of the top-p oracle for ``rows`` (visual),
    whose retention ``keep [Hq, R, max_count]`` is given in ``rows`` order."""
    from .topp import attend
    _, _, plist = attend(q, k, v, lay, blk, keep, rows, scale, want_p=True)
    for idx, keys, ps in plist:
        yield rows[idx], keys, np.stack(ps)

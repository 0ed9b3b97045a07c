"""Pins of the coarse-map oracle (appendix, coarse-map equation: exact
logits on E_i, the block affinity on retained blocks, row softmax) and of
the sparse-vs-dense alignment metrics.

Pins: with one-token blocks and tau_p = 1 every block keeps its exact logit
and everything is retained, so the coarse map is dense causal attention
(torch SDPA); with keys constant inside each block the block affinity is
the exact logit, so the coarse map equals the top-p oracle's exact
attention; pure-Python loops with subset enumeration on a tiny case; the
metrics against scipy routines and closed forms.
"""
import itertools
import math

import numpy as np
import pytest
import scipy.stats
from scipy.spatial.distance import jensenshannon

from oracle import coarse, topp
from oracle.layout import Layout, SYS, VIS


def _rand(S, hq, hkv, d, seed, qs=1.0):
    r = np.random.default_rng(seed)
    return (r.standard_normal((S, hq, d)) * qs, r.standard_normal((S, hkv, d)),
            r.standard_normal((S, hkv, d)))


def _dense_map(q, k, lay, scale):
    """Row softmax over every earlier key of the same video (loops over
    heads, numpy per row; no oracle code)."""
    S, hq, _ = q.shape
    grp = hq // k.shape[1]
    P = np.zeros((hq, S, S))
    for h in range(hq):
        for i in range(S):
            m = np.nonzero((lay.seq == lay.seq[i]) & (np.arange(S) <= i))[0]
            s = k[m, h // grp] @ q[i, h] * scale
            e = np.exp(s - s.max())
            P[h, i, m] = e / e.sum()
    return P


def _coarse_full(q, k, lay, B, tau, scale):
    blk = topp.Blocks(lay, B)
    rows = np.arange(lay.S)
    keep, _ = topp.select(q, k, lay, blk, tau, scale, rows)
    P = np.zeros((q.shape[1], lay.S, lay.S))
    for ri, keys, Pg in coarse.coarse_probs(q, k, lay, blk, keep, rows,
                                            scale):
        for h in range(q.shape[1]):
            P[h][np.ix_(ri, keys)] = Pg[h]
    return P, keep, blk


def test_one_token_blocks_tau_one_is_dense_causal():
    lay = Layout((2, 0), (3, 2), (4, 3), 2)
    q, k, _ = _rand(lay.S, 4, 2, 6, 3)
    P, _, _ = _coarse_full(q, k, lay, 1, 1.0, 0.4)
    np.testing.assert_allclose(P, _dense_map(q, k, lay, 0.4), rtol=0,
                               atol=1e-13)


def test_block_constant_keys_give_exact_retained_attention():
    lay = Layout((3,), (6,), (10,), 4)
    blk = topp.Blocks(lay, 4)
    q, k, v = _rand(lay.S, 2, 1, 5, 8, qs=2.0)
    for gb in range(blk.start.size):           # one key vector per block
        a = blk.start[gb]
        k[a:a + blk.len[gb]] = k[a]
    P, keep, _ = _coarse_full(q, k, lay, 4, 0.8, 0.5)
    rows = np.arange(lay.S)
    _, _, plist = topp.attend(q, k, v, lay, blk, keep, rows, 0.5,
                              want_p=True)
    for idx, keys, ps in plist:
        for h in range(2):
            np.testing.assert_allclose(P[h][np.ix_(rows[idx], keys)], ps[h],
                                       rtol=0, atol=1e-13)


def test_coarse_map_loops():
    ns, nf, nt, Nv, B = (2,), (4,), (6,), 4, 4
    lay = Layout(ns, nf, nt, Nv)
    q, k, _ = _rand(lay.S, 2, 1, 4, 21, qs=2.0)
    tau, scale = 0.75, 0.5
    P, keep, blk = _coarse_full(q, k, lay, B, tau, scale)
    nb = int(blk.count[0])
    # query-frame evidence of the coarse map, looped: the query rows
    # (tokens past the system prefix and the frames) summed per frame
    vis0, txt0 = ns[0], ns[0] + nf[0] * Nv
    E = np.zeros((2, nf[0]))
    for h in range(2):
        for i in range(lay.S):
            lb = int(blk.local[i])
            means = [[math.fsum(k[t, 0, c] for t in blk.tokens(0, j)) /
                      blk.len[j] for c in range(4)] for j in range(nb)]
            g = [math.fsum(q[i, h, c] * means[j][c] for c in range(4)) *
                 scale for j in range(max(lb, 0))]
            kept = set()
            if g:
                mx = max(g)
                p = [math.exp(x - mx) for x in g]
                z = math.fsum(p)
                p = [x / z for x in p]
                for size in range(1, len(p) + 1):
                    best = None
                    for sub in itertools.combinations(range(len(p)), size):
                        m = math.fsum(p[j] for j in sub)
                        if m >= tau and (best is None or m > best[0]):
                            best = (m, set(sub))
                    if best:
                        kept = best[1]
                        break
            logits = {}
            for m in range(i + 1):
                if lay.region[m] == SYS or blk.local[m] == lb:
                    logits[m] = math.fsum(q[i, h, c] * k[m, 0, c]
                                          for c in range(4)) * scale
                elif blk.local[m] in kept:
                    logits[m] = g[int(blk.local[m])]
            mx = max(logits.values())
            z = math.fsum(math.exp(x - mx) for x in logits.values())
            want = np.zeros(lay.S)
            for m, x in logits.items():
                want[m] = math.exp(x - mx) / z
            np.testing.assert_allclose(P[h, i], want, rtol=0, atol=1e-13)
            if i >= txt0:
                for m in range(vis0, txt0):
                    E[h, (m - vis0) // Nv] += want[m]
    # the oracle's query_frame from the groups of every row (rows that are
    # not query tokens must contribute nothing)
    rows = np.arange(lay.S)
    groups = coarse.coarse_probs(q, k, lay, blk, keep, rows, scale)
    np.testing.assert_allclose(coarse.query_frame(lay, groups, 2), E,
                               rtol=0, atol=1e-12)


def test_metrics_against_scipy_and_closed_forms():
    r = np.random.default_rng(4)
    s = r.random(200) ** 3
    s[r.random(200) < 0.4] = 0.0
    t = s + 0.05 * r.random(200)
    assert abs(coarse.pearson(s, t) - scipy.stats.pearsonr(s, t)[0]) < 1e-12
    assert abs(coarse.spearman(s, t) -
               scipy.stats.spearmanr(s, t)[0]) < 1e-12   # ties at zero
    assert abs(coarse.js_divergence(s, t) - jensenshannon(s, t) ** 2) < 1e-12
    assert coarse.js_divergence(t, t) == 0.0
    assert abs(coarse.js_divergence([1, 0, 0, 0], [0, 0, 1, 1]) -
               math.log(2)) < 1e-15
    assert coarse.top_overlap(t, t) == 1.0
    assert coarse.top_overlap(np.arange(50.0), -np.arange(50.0)) == 0.0
    assert coarse.keep_ratio(s) == float((s > 0).mean())
    assert coarse.mass_recovery(np.ones(9), t[:9]) == 1.0
    assert abs(coarse.mass_recovery(s, t) - t[s > 0].sum() / t.sum()) < 1e-15

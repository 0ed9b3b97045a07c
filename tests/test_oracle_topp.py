"""Pins of the top-p retention oracle (appendix "Detailed Sparse Prefilling":
mean-key, affinity and probability equations, smallest subset reaching
tau_p, attention over E_i and the retained blocks).

Each pin is independent of the oracle's code path: subset enumeration
instead of sort + cumulative sum, token-by-token history enumeration, a
closed-form block mean, exact rationals for the tie case, torch's
scaled_dot_product_attention for tau_p = 1, and pure-Python loops for the
attention under a given retention.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle.layout import Layout, SYS, VIS, TXT
from oracle import topp


def _rand_layer(S, hq, hkv, d, seed):
    r = np.random.default_rng(seed)
    return (r.standard_normal((S, hq, d)), r.standard_normal((S, hkv, d)),
            r.standard_normal((S, hkv, d)))


# ---------------------------------------------------------------------------
# retention rule

def _brute_min_subset(p, tau):
    """All subsets: the minimal size reaching tau and the largest mass of a
    subset of that size."""
    n = len(p)
    for size in range(1, n + 1):
        best = None
        for sub in itertools.combinations(range(n), size):
            m = math.fsum(p[j] for j in sub)
            if m >= tau and (best is None or m > best[0]):
                best = (m, set(sub))
        if best is not None:
            return size, best
    return n, (math.fsum(p), set(range(n)))


def _py_softmax(g):
    mx = max(g)
    e = [math.exp(x - mx) for x in g]
    z = math.fsum(e)
    return [x / z for x in e]


@pytest.mark.parametrize("tau", [0.3, 0.5, 0.9, 0.97, 0.999])
def test_retain_matches_subset_enumeration(tau):
    r = np.random.default_rng(11)
    for n in range(1, 10):
        g = r.standard_normal((6, n)) * 1.5
        keep, info = topp.retain(g, tau)
        for row in range(6):
            p = _py_softmax(list(g[row]))
            size, (mass, best) = _brute_min_subset(p, tau)
            got = set(np.nonzero(keep[row])[0].tolist())
            assert len(got) == size
            assert got == best          # distinct p: the heaviest set is unique


def test_retain_boundary_is_inclusive_and_ties_go_to_lower_index():
    # four equal probabilities of exactly 1/4: 1/4 + 1/4 reaches 1/2
    keep, info = topp.retain(np.zeros((1, 4)), 0.5)
    assert np.nonzero(keep[0])[0].tolist() == [0, 1]
    keep, _ = topp.retain(np.zeros((1, 4)), 0.5 + 1e-12)
    assert np.nonzero(keep[0])[0].tolist() == [0, 1, 2]
    # a dominant block alone covers the threshold
    g = np.array([[0.0, 40.0, 0.0, 1.0]])
    keep, _ = topp.retain(g, 0.97)
    assert np.nonzero(keep[0])[0].tolist() == [1]


def test_retain_tau_one_keeps_every_block():
    g = np.random.default_rng(3).standard_normal((20, 37)) * 3
    keep, _ = topp.retain(g, 1.0)
    assert keep.all()


# ---------------------------------------------------------------------------
# blocks, history, mean keys

LAYOUTS = [
    ((0,), (8,), (20,), 16, 16),
    ((3, 0, 5), (5, 7, 2), (9, 20, 3), 16, 32),
    ((2,), (9,), (33,), 8, 16),          # two frames per block, odd frames
]


@pytest.mark.parametrize("li", range(len(LAYOUTS)))
def test_history_matches_token_enumeration(li):
    ns, nf, nt, Nv, B = LAYOUTS[li]
    lay = Layout(ns, nf, nt, Nv)
    blk = topp.Blocks(lay, B)
    # enumerate the blocks from the region definition, token by token
    blocks = []
    for n in range(lay.n_seq):
        for a, e in ((lay.vis0[n], lay.txt0[n]), (lay.txt0[n], lay.end[n])):
            t = a
            while t < e:
                blocks.append((n, t, min(t + B, e) - 1))
                t += B
    for i in range(lay.S):
        if lay.region[i] == SYS:
            assert blk.history(i).size == 0
            continue
        mine = [(n, a, z) for (n, a, z) in blocks if n == lay.seq[i]]
        want = [j for j, (n, a, z) in enumerate(mine) if z < i and
                not (a <= i <= z)]
        assert blk.history(i).tolist() == want
        own = [j for j, (n, a, z) in enumerate(mine) if a <= i <= z]
        assert own == [blk.local[i]]


@pytest.mark.parametrize("li", range(len(LAYOUTS)))
def test_mean_keys_closed_form(li):
    ns, nf, nt, Nv, B = LAYOUTS[li]
    lay = Layout(ns, nf, nt, Nv)
    blk = topp.Blocks(lay, B)
    a = np.array([[0.5, -1.0, 2.0]])
    b = np.array([[0.25, 0.125, -0.5]])
    pos = np.arange(lay.S, dtype=np.float64)[:, None, None]
    k = a[None] + b[None] * pos                       # affine in position
    kbar = topp.mean_keys(k, blk)
    for gb in range(blk.start.size):
        centre = blk.start[gb] + (blk.len[gb] - 1) / 2.0
        np.testing.assert_allclose(kbar[gb], a + b * centre, rtol=0,
                                   atol=1e-12)


# ---------------------------------------------------------------------------
# whole selection chain against loops + subset enumeration

def test_select_chain_bruteforce():
    ns, nf, nt, Nv, B = (3,), (6,), (20,), 16, 16
    lay = Layout(ns, nf, nt, Nv)
    blk = topp.Blocks(lay, B)
    hq, hkv, d = 4, 2, 8
    q, k, _ = _rand_layer(lay.S, hq, hkv, d, 5)
    q *= 2.5                                           # spread the affinities
    tau, scale = 0.9, 1.0 / math.sqrt(d)
    keep, info = topp.select(q, k, lay, blk, tau, scale)
    nblk = blk.count[0]
    for h in range(hq):
        g = h // (hq // hkv)
        # block means by loops
        means = []
        for j in range(nblk):
            toks = blk.tokens(0, j)
            means.append([math.fsum(k[t, g, c] for t in toks) / len(toks)
                          for c in range(d)])
        for i in range(lay.S):
            hist = [j for j in range(nblk)
                    if blk.start[j] + blk.len[j] - 1 < i
                    and not (blk.start[j] <= i < blk.start[j] + blk.len[j])]
            got = set(np.nonzero(keep[h, i])[0].tolist())
            if not hist:
                assert got == set()
                continue
            aff = [math.fsum(q[i, h, c] * means[j][c] for c in range(d)) *
                   scale for j in hist]
            p = _py_softmax(aff)
            size, (mass, best) = _brute_min_subset(p, tau)
            assert got == {hist[x] for x in best}, (h, i)


def test_uniform_affinity_keeps_first_ceil_tau_n_blocks():
    ns, nf, nt, Nv, B = (0,), (30,), (40,), 16, 16
    lay = Layout(ns, nf, nt, Nv)
    blk = topp.Blocks(lay, B)
    q = np.zeros((lay.S, 2, 16))
    _, k, _ = _rand_layer(lay.S, 2, 1, 16, 9)
    tau = 0.97
    keep, info = topp.select(q, k, lay, blk, tau, 0.25)
    checked = 0
    for i in range(lay.S):
        n = int(blk.local[i])
        if n <= 0:
            continue
        t = Fraction(tau) * n
        if t.denominator == 1:
            continue                       # exact boundary: rounding decides
        want = list(range(math.ceil(t)))
        for h in range(2):
            assert np.nonzero(keep[h, i])[0].tolist() == want
        checked += 1
    assert checked > 500


# ---------------------------------------------------------------------------
# attention under retention

def _sdpa_causal(q, k, v, lay, scale):
    """torch SDPA in float64 with a same-video causal mask (GQA expanded)."""
    S, hq, d = q.shape
    hkv = k.shape[1]
    i = torch.arange(S)
    seq = torch.from_numpy(lay.seq)
    mask = (i[None, :] <= i[:, None]) & (seq[None, :] == seq[:, None])
    rep = hq // hkv
    Q = torch.from_numpy(q).permute(1, 0, 2)
    K = torch.from_numpy(k).repeat_interleave(rep, dim=1).permute(1, 0, 2)
    V = torch.from_numpy(v).repeat_interleave(rep, dim=1).permute(1, 0, 2)
    O = torch.nn.functional.scaled_dot_product_attention(
        Q, K.contiguous(), V.contiguous(), attn_mask=mask, scale=scale)
    return O.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("li", range(len(LAYOUTS)))
def test_tau_one_equals_causal_attention(li):
    ns, nf, nt, Nv, B = LAYOUTS[li]
    lay = Layout(ns, nf, nt, Nv)
    q, k, v = _rand_layer(lay.S, 4, 2, 16, 21 + li)
    res = topp.run_layer(q, k, v, lay, B, 1.0, 0.25)
    assert all(res["keep"][:, j, :res["info"]["nh"][j]].all()
               for j in range(lay.S))
    want = _sdpa_causal(q, k, v, lay, 0.25)
    np.testing.assert_allclose(res["O"], want, rtol=0, atol=1e-12)


def test_attention_under_retention_bruteforce():
    ns, nf, nt, Nv, B = (2, 1), (4, 3), (7, 5), 8, 8
    lay = Layout(ns, nf, nt, Nv)
    blk = topp.Blocks(lay, B)
    hq, hkv, d = 2, 1, 4
    q, k, v = _rand_layer(lay.S, hq, hkv, d, 33)
    q *= 3.0
    tau, scale = 0.6, 0.5
    res = topp.run_layer(q, k, v, lay, B, tau, scale)
    keep = res["keep"]
    # token roles from the layout numbers alone: (video, region, global
    # frame) of every token, region 0 system, 1 visual, 2 query
    role = []
    f0 = 0
    for n in range(len(ns)):
        role += [(n, 0, -1)] * ns[n]
        role += [(n, 1, f0 + t // Nv) for t in range(nf[n] * Nv)]
        role += [(n, 2, -1)] * nt[n]
        f0 += nf[n]
    E = [[0.0] * f0 for _ in range(hq)]
    tm = [[0.0] * len(ns) for _ in range(hq)]
    for h in range(hq):
        for i in range(lay.S):
            kept = set(np.nonzero(keep[h, i])[0].tolist())
            keys = []
            for m in range(lay.S):
                if lay.seq[m] != lay.seq[i] or m > i:
                    continue
                if (lay.region[m] == SYS or blk.local[m] == blk.local[i]
                        or blk.local[m] in kept):
                    keys.append(m)
            s = [math.fsum(q[i, h, c] * k[m, 0, c] for c in range(d)) * scale
                 for m in keys]
            p = _py_softmax(s)
            o = [math.fsum(p[x] * v[m, 0, c] for x, m in enumerate(keys))
                 for c in range(d)]
            np.testing.assert_allclose(res["O"][i, h], o, rtol=0, atol=1e-12)
            lse = max(s) + math.log(math.fsum(math.exp(x - max(s)) for x in s))
            assert abs(res["LSE"][h, i] - lse) < 1e-12
            # evidence (Evidence Decomposition, query-frame cue): a query
            # row's mass on each frame's visual keys, the rest to text_mass
            if role[i][1] == 2:
                for x, m in enumerate(keys):
                    if role[m][1] == 1:
                        E[h][role[m][2]] += p[x]
                    else:
                        tm[h][role[i][0]] += p[x]
    np.testing.assert_allclose(res["E"], E, rtol=0, atol=1e-12)
    np.testing.assert_allclose(res["text_mass"], tm, rtol=0, atol=1e-12)
    # per head, frame masses plus the rest = number of query rows
    tot = res["E"].sum(axis=1) + res["text_mass"].sum(axis=1)
    np.testing.assert_allclose(tot, lay.n_text.sum(), rtol=0, atol=1e-12)


def test_dominant_block_is_retained_alone():
    ns, nf, nt, Nv, B = (0,), (8,), (16,), 16, 16
    lay = Layout(ns, nf, nt, Nv)
    blk = topp.Blocks(lay, B)
    d = 16
    q, k, v = _rand_layer(lay.S, 1, 1, d, 44)
    u = np.zeros(d)
    u[3] = 1.0
    j0 = 2
    toks = blk.tokens(0, j0)
    k[toks, 0, :] = 30.0 * u
    q[:, 0, :] += 30.0 * u
    keep, info = topp.select(q, k, lay, blk, 0.97, 1.0 / math.sqrt(d))
    for i in range(lay.S):
        lb = blk.local[i]
        got = np.nonzero(keep[0, i])[0].tolist()
        if lb > j0:
            assert got == [j0], i


def test_retention_invariants_on_workload_rows():
    import workloads as wl
    w = wl.get(2)
    ns, nf, nt = wl.layout_arrays(w)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    blk = topp.Blocks(lay, w.block)
    q, k, _ = wl.gen_layer(w, 0).as_f64()
    rows = np.concatenate([np.arange(64 * b, 64 * b + 64) for b in (3, 77)] +
                          [lay.text_rows()])
    keep, info = topp.select(q, k, lay, blk, 0.97, w.softmax_scale, rows)
    kbar = topp.mean_keys(k, blk)
    for h in (0, 13, 27):
        for j, i in enumerate(rows):
            nh = info["nh"][j]
            g = q[i, h] @ kbar[:nh, h // 7].T * w.softmax_scale
            p = np.exp(g - g.max())
            p /= p.sum()
            kept = keep[h, j, :nh]
            assert p[kept].sum() >= 0.97
            assert p[kept].sum() - p[kept].min() < 0.97
            if (~kept).any():
                assert p[kept].min() >= p[~kept].max()

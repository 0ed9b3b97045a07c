"""Pins of the cross-frame and intra-frame cue oracle (Evidence
Decomposition: heads averaged with the layer kept; A_ff from each frame to
its preceding frames, averaged between their visual blocks; E_ff the mean of
the attention a frame assigns backwards and receives forwards; A_if the
token-level causal attention inside each frame).

Pins: pure-Python loops over the brute-force probabilities, the closed form
of uniform attention (Q = 0, all-causal), the per-frame mass balance, and
E_ff's one-sided ends on a hand-built matrix.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import brute, cues
from oracle.layout import Layout, Rule

CASES = [
    # n_sys, n_frames, n_text, Nv, B, sink, window
    ((0,), (5,), (3,), 4, 4, 1, 1),
    ((2, 0), (4, 3), (2, 5), 4, 8, 1, 0),      # two frames per block
    ((0,), (6,), (2,), 8, 8, 0, -1),           # all-causal
    ((3,), (3,), (4,), 2, 4, 2, 1),
]


def _rand(S, hq, hkv, d, seed):
    r = np.random.default_rng(seed)
    return (r.standard_normal((S, hq, d)) * 1.5, r.standard_normal((S, hkv, d)),
            r.standard_normal((S, hkv, d)))


def _loops(P, toks, hq, T, Nv):
    """A_ff [T][T] (b < a) and A_if [T][Nv][Nv] by loops over P."""
    aff = [[0.0] * T for _ in range(T)]
    aif = [[[0.0] * Nv for _ in range(Nv)] for _ in range(T)]
    for h in range(hq):
        for i, ti in enumerate(toks):
            if ti[1] != "vis":
                continue
            a = ti[3]
            for m, p in P[h][i].items():
                tm = toks[m]
                if tm[1] != "vis":
                    continue
                b = tm[3]
                if b < a:
                    aff[a][b] += p / (hq * Nv)
                elif b == a:
                    aif[a][ti[2] % Nv][tm[2] % Nv] += p / hq
    return np.array(aff), np.array(aif)


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_cues_match_loops(ci):
    ns, nf, nt, Nv, B, sink, win = CASES[ci]
    lay = Layout(ns, nf, nt, Nv)
    hq, hkv, d = 4, 2, 6
    q, k, v = _rand(lay.S, hq, hkv, d, 50 + ci)
    scale = 0.4
    P, toks = brute.probabilities(q.tolist(), k.tolist(), list(ns), list(nf),
                                  list(nt), Nv, B, sink, win, scale)
    want_ff, want_if = _loops(P, toks, hq, lay.T, Nv)
    A_ff, A_if = cues.accumulate(lay, cues.static_groups(
        q, k, v, lay, Rule(B, sink, win), scale), hq)
    np.testing.assert_allclose(A_ff, want_ff, rtol=0, atol=1e-13)
    np.testing.assert_allclose(A_if, want_if, rtol=0, atol=1e-13)


def test_uniform_attention_closed_form():
    # Q = 0, all-causal, one video without system prefix: row i (position
    # i in the video) spreads 1/(i+1) over keys 0..i.
    Nv, F = 4, 6
    lay = Layout((0,), (F,), (3,), Nv)
    q = np.zeros((lay.S, 2, 4))
    _, k, v = _rand(lay.S, 2, 1, 4, 7)
    A_ff, A_if = cues.accumulate(lay, cues.static_groups(
        q, k, v, lay, Rule(Nv, 0, -1), 0.5), 2)
    for a in range(F):
        for b in range(F):
            want = (float(sum(Fraction(1, i + 1)
                              for i in range(a * Nv, (a + 1) * Nv)))
                    if b < a else 0.0)
            assert abs(A_ff[a, b] - want) < 1e-14
        for ii in range(Nv):
            for mm in range(Nv):
                i = a * Nv + ii
                want = 1.0 / (i + 1) if mm <= ii else 0.0
                assert abs(A_if[a, ii, mm] - want) < 1e-14


@pytest.mark.parametrize("ci", [0, 2])
def test_frame_mass_balance(ci):
    # no system prefix: a visual row's mass is all on visual keys of its own
    # or earlier frames, so N_v sum_{b<a} A_ff[a,b] + sum A_if[a] = N_v
    ns, nf, nt, Nv, B, sink, win = CASES[ci]
    lay = Layout(ns, nf, nt, Nv)
    q, k, v = _rand(lay.S, 4, 1, 5, 90 + ci)
    A_ff, A_if = cues.accumulate(lay, cues.static_groups(
        q, k, v, lay, Rule(B, sink, win), 0.3), 4)
    tot = Nv * A_ff.sum(axis=1) + A_if.sum(axis=(1, 2))
    np.testing.assert_allclose(tot, Nv, rtol=0, atol=1e-12)


def test_e_ff_sides():
    lay = Layout((0, 0, 0), (4, 1, 2), (1, 1, 1), 2)
    A = np.zeros((lay.T, lay.T))
    # video 0: frames 0..3
    A[1, 0], A[2, 0], A[2, 1], A[3, 0], A[3, 1], A[3, 2] = 1, 2, 3, 4, 5, 6
    A[6, 5] = 7                              # video 2: frames 5, 6
    e = cues.e_ff(lay, A)
    want = [
        (1 + 2 + 4) / 3,                     # frame 0: received only
        ((1) / 1 + (3 + 5) / 2) / 2,
        ((2 + 3) / 2 + (6) / 1) / 2,
        (4 + 5 + 6) / 3,                     # last frame: assigned only
        0.0,                                 # single-frame video
        7.0, 7.0,
    ]
    np.testing.assert_allclose(e, want, rtol=0, atol=1e-15)

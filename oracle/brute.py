"""Pure-Python brute force for tiny inputs (oracle pin; test only).

Written without NumPy and without the ``layout`` module: it re-derives each
token's video, region and block with explicit loops, applies the visibility
rule token by token and evaluates the softmax with ``math.exp``. It is the
independent pin for the vectorised oracle on inputs of a few dozen tokens.
"""
from __future__ import annotations

import math


def _tokens(n_sys, n_frames, n_text, Nv):
    """List of (video, region, pos_in_region, global_frame) per token."""
    toks = []
    frame_base = 0
    for n in range(len(n_frames)):
        for p in range(n_sys[n]):
            toks.append((n, "sys", p, None))
        for p in range(n_frames[n] * Nv):
            toks.append((n, "vis", p, frame_base + p // Nv))
        for p in range(n_text[n]):
            toks.append((n, "txt", p, None))
        frame_base += n_frames[n]
    return toks


def _visible(ti, tm, i, m, B, sink, window):
    if ti[0] != tm[0] or m > i:
        return False
    if tm[1] == "sys":
        return True
    if ti[1] == "vis" and tm[1] == "vis":
        qb, kb = ti[2] // B, tm[2] // B
        if kb < sink:
            return True
        return window < 0 or (qb - window <= kb <= qb)
    if ti[1] == "txt":
        return tm[1] in ("vis", "txt")
    return False


def attention(q, k, v, n_sys, n_frames, n_text, Nv, B, sink, window, scale):
    """q[S][Hq][d], k/v[S][Hkv][d] nested lists of floats.

    Returns (O[S][Hq][d], LSE[Hq][S], E[Hq][T], text_mass[Hq][n_videos]).
    """
    toks = _tokens(n_sys, n_frames, n_text, Nv)
    S = len(toks)
    hq, hkv, d = len(q[0]), len(k[0]), len(q[0][0])
    T = sum(n_frames)
    O = [[[0.0] * d for _ in range(hq)] for _ in range(S)]
    LSE = [[0.0] * S for _ in range(hq)]
    E = [[0.0] * T for _ in range(hq)]
    tm = [[0.0] * len(n_frames) for _ in range(hq)]
    for h in range(hq):
        g = h // (hq // hkv)
        for i in range(S):
            keys = [m for m in range(S)
                    if _visible(toks[i], toks[m], i, m, B, sink, window)]
            logits = []
            for m in keys:
                dot = 0.0
                for c in range(d):
                    dot += q[i][h][c] * k[m][g][c]
                logits.append(dot * scale)
            mx = max(logits)
            ex = [math.exp(x - mx) for x in logits]
            z = math.fsum(ex)
            LSE[h][i] = mx + math.log(z)
            for c in range(d):
                O[i][h][c] = math.fsum(ex[j] / z * v[m][g][c]
                                       for j, m in enumerate(keys))
            if toks[i][1] == "txt":
                for j, m in enumerate(keys):
                    if toks[m][1] == "vis":
                        E[h][toks[m][3]] += ex[j] / z
                    else:
                        tm[h][toks[i][0]] += ex[j] / z
    return O, LSE, E, tm


def probabilities(q, k, n_sys, n_frames, n_text, Nv, B, sink, window, scale):
    """Per (head, query token) the softmax probabilities over its visible
    keys, as {key token: probability} dicts: P[h][i]. Also returns the token
    table of ``_tokens`` (video, region, position in region, global frame)."""
    toks = _tokens(n_sys, n_frames, n_text, Nv)
    S = len(toks)
    hq, hkv, d = len(q[0]), len(k[0]), len(q[0][0])
    P = [[None] * S for _ in range(hq)]
    for h in range(hq):
        g = h // (hq // hkv)
        for i in range(S):
            keys = [m for m in range(S)
                    if _visible(toks[i], toks[m], i, m, B, sink, window)]
            logits = [math.fsum(q[i][h][c] * k[m][g][c] for c in range(d)) *
                      scale for m in keys]
            mx = max(logits)
            ex = [math.exp(x - mx) for x in logits]
            z = math.fsum(ex)
            P[h][i] = {m: ex[j] / z for j, m in enumerate(keys)}
    return P, toks

"""Pins for the fp64 oracle: brute force, closed forms, a library attention
routine, invariants, block sets. CPU only."""
import math

import numpy as np
import pytest

import oracle
from oracle import blocks as oblocks
from oracle.layout import Layout, Rule, VIS, TXT
import workloads as wl


def _rand_case(seed, n_sys, n_frames, n_text, Nv, hq, hkv, d):
    rng = np.random.default_rng(seed)
    lay = Layout(n_sys, n_frames, n_text, Nv)
    q = rng.standard_normal((lay.S, hq, d))
    k = rng.standard_normal((lay.S, hkv, d))
    v = rng.standard_normal((lay.S, hkv, d))
    return lay, q, k, v


TINY = [
    # n_sys, n_frames, n_text, Nv, B, sink, window, hq, hkv, d
    ((0,), (6,), (5,), 4, 4, 1, 2, 2, 1, 6),
    ((3,), (5,), (4,), 4, 8, 1, 1, 4, 2, 5),
    ((2, 0), (3, 4), (3, 2), 4, 4, 2, 1, 2, 2, 4),
    ((0,), (4,), (7,), 3, 3, 1, -1, 2, 1, 3),    # all-causal
    ((1, 2), (2, 3), (2, 5), 2, 4, 0, 1, 3, 1, 4),  # no sink, B spans frames
]


@pytest.mark.parametrize("case", range(len(TINY)))
@pytest.mark.parametrize("mode", ["allowed", "dense"])
def test_oracle_matches_brute_force(case, mode):
    ns, nf, nt, Nv, B, sink, win, hq, hkv, d = TINY[case]
    lay, q, k, v = _rand_case(100 + case, ns, nf, nt, Nv, hq, hkv, d)
    rule = Rule(B, sink, win)
    scale = 1.0 / math.sqrt(d)
    ref = oracle.run_layer(q, k, v, lay, rule, scale, mode=mode)
    O, LSE, E, tm = oracle.brute.attention(
        q.tolist(), k.tolist(), v.tolist(), list(ns), list(nf), list(nt),
        Nv, B, sink, win, scale)
    np.testing.assert_allclose(ref["O"], np.array(O), atol=1e-12, rtol=0)
    np.testing.assert_allclose(ref["LSE"], np.array(LSE), atol=1e-12, rtol=0)
    np.testing.assert_allclose(ref["E"], np.array(E), atol=1e-12, rtol=0)
    np.testing.assert_allclose(ref["text_mass"], np.array(tm), atol=1e-12,
                               rtol=0)
    dense = oracle.attention.dense_reference(q, k, v, lay, rule, scale)
    for key in ("O", "LSE", "E", "text_mass"):
        np.testing.assert_allclose(ref[key], dense[key], atol=1e-12, rtol=0)


def test_allowed_keys_equal_predicate():
    rng = np.random.default_rng(7)
    for trial in range(6):
        nseq = int(rng.integers(1, 3))
        ns = rng.integers(0, 3, nseq)
        nf = rng.integers(1, 9, nseq)
        nt = rng.integers(1, 7, nseq)
        Nv = int(rng.choice([2, 4, 8]))
        B = int(rng.choice([2, 4, 8, 16]))
        rule = Rule(B, int(rng.integers(0, 3)), int(rng.choice([-1, 0, 1, 3])))
        lay = Layout(ns, nf, nt, Nv)
        allm = np.arange(lay.S)
        for i in range(lay.S):
            want = np.nonzero(lay.allowed(i, allm, rule))[0]
            np.testing.assert_array_equal(lay.allowed_keys(i, rule), want)


def test_block_csr_enumerated_equals_brute():
    rng = np.random.default_rng(11)
    for trial in range(5):
        nseq = int(rng.integers(1, 3))
        lay = Layout(rng.integers(0, 5, nseq), rng.integers(1, 12, nseq),
                     rng.integers(1, 20, nseq), int(rng.choice([4, 8])))
        rule = Rule(int(rng.choice([4, 8])), int(rng.integers(0, 3)),
                    int(rng.choice([-1, 1, 2])))
        a = oblocks.active_csr(lay, rule, brute=True)
        b = oblocks.active_csr(lay, rule, brute=False)
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)


def _closed_form_pairs(n_vis_blocks, n_txt_blocks, sink, W):
    """Active pairs per head: visual block i keeps its own block, the
    preceding min(i, W) blocks and the sink blocks below that window; text
    block t keeps every visual block and text blocks 0..t."""
    tot = 0
    for i in range(n_vis_blocks):
        w = i if W < 0 else min(i, W)
        tot += w + 1 + min(sink, i - w)
    for t in range(n_txt_blocks):
        tot += n_vis_blocks + t + 1
    return tot


@pytest.mark.parametrize("cid,expect", [(1, 45), (2, 1364), (3, 3030)])
def test_active_pairs_closed_form(cid, expect):
    w = wl.get(cid)
    ns, nf, nt = wl.layout_arrays(w)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    nvb = -(-int(nf[0]) * w.tokens_per_frame // w.block)
    ntb = -(-int(nt[0]) // w.block)
    assert _closed_form_pairs(nvb, ntb, w.sink_blocks, w.window) == expect
    if cid <= 2:
        _, rp, _ = oblocks.active_csr(lay, Rule(w.block, w.sink_blocks,
                                                w.window))
        assert int(rp[-1]) == expect


def _allowed_count_and_sum(lay, rule, i):
    """Closed-form size and index sum of query i's visible set."""
    n = lay.seq[i]
    a, v0, t0 = int(lay.tok0[n]), int(lay.vis0[n]), int(lay.txt0[n])
    ns = v0 - a
    cnt, tot = ns, (a + v0 - 1) * ns // 2
    p = int(lay.rpos[i])
    if i < v0:                              # system-prefix row: causal
        return p + 1, (a + i) * (p + 1) // 2
    B, sink, W = rule.block, rule.sink_blocks, rule.window
    if lay.region[i] == VIS:
        qb = p // B
        lo = 0 if W < 0 else max(0, qb - W)
        ranges = [(lo, qb)]                 # full blocks lo..qb-1 + own
        if min(sink, lo) > 0:
            ranges.append((0, min(sink, lo)))
        for b0, b1 in ranges:
            for b in range(b0, b1):
                s = v0 + b * B
                cnt += B
                tot += (2 * s + B - 1) * B // 2
        s = v0 + qb * B
        m = p - qb * B + 1
        cnt += m
        tot += (2 * s + m - 1) * m // 2
    elif lay.region[i] == TXT:
        m = i - v0 + 1
        cnt += m
        tot += (v0 + i) * m // 2
    return cnt, tot


LAYOUTS = [
    ((0,), (32,), (32,), 16, Rule(64, 1, -1)),
    ((0,), (40,), (70,), 64, Rule(64, 1, 8)),
    ((5,), (23,), (9,), 16, Rule(32, 2, 3)),
    ((3, 0, 7), (9, 14, 5), (4, 64, 17), 32, Rule(64, 1, 2)),
]


@pytest.mark.parametrize("li", range(len(LAYOUTS)))
def test_uniform_logits_closed_form(li):
    ns, nf, nt, Nv, rule = LAYOUTS[li]
    lay = Layout(ns, nf, nt, Nv)
    S, d = lay.S, 3
    q = np.zeros((S, 2, d))
    k = np.random.default_rng(li).standard_normal((S, 1, d))
    m = np.arange(S, dtype=np.float64)
    v = np.stack([np.ones(S), m / S, (m / S) ** 2], axis=1)[:, None, :]
    res = oracle.run_layer(q, k, v, lay, rule, 1.0)
    for j, i in enumerate(res["rows"]):
        cnt, tot = _allowed_count_and_sum(lay, rule, int(i))
        assert abs(res["O"][j, 0, 0] - 1.0) < 1e-12
        assert abs(res["O"][j, 1, 1] * cnt * S - tot) < 1e-7 * max(1, tot)
        assert abs(res["LSE"][0, j] - math.log(cnt)) < 1e-12
    # evidence: each query row r of video n puts 1/(n_sys+n_vis+r+1) on
    # every visual key, so a frame receives N_v * sum_r 1/(...).
    for n in range(lay.n_seq):
        nsys, nvis = int(ns[n]), int(nf[n]) * Nv
        ef = sum(Nv / (nsys + nvis + r + 1) for r in range(int(nt[n])))
        tmf = sum((nsys + r + 1) / (nsys + nvis + r + 1)
                  for r in range(int(nt[n])))
        f0 = int(lay.frame0[n])
        np.testing.assert_allclose(res["E"][:, f0:f0 + int(nf[n])], ef,
                                   rtol=1e-12)
        np.testing.assert_allclose(res["text_mass"][:, n], tmf, rtol=1e-12)


def test_causal_attention_matches_torch_sdpa():
    """All-causal single video (the tiny fp32 workload's rule) equals the
    library's causal scaled-dot-product attention, K/V repeated per group."""
    torch = pytest.importorskip("torch")
    w = wl.get(1)
    layer = wl.gen_layer(w, 0)
    q, k, v = layer.as_f64()
    ns, nf, nt = wl.layout_arrays(w)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    rule = Rule(w.block, w.sink_blocks, w.window)
    res = oracle.run_layer(q, k, v, lay, rule, w.softmax_scale)
    g = w.hq // w.hkv
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, 0)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, 0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, is_causal=True)[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(res["O"], ref, atol=1e-12, rtol=0)


def test_lse_from_library_probabilities():
    """With one-hot values (d >= S) the library's causal attention returns
    the probabilities themselves; LSE_i = s_im - ln P_im for every allowed m."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    lay = Layout((0,), (6,), (8,), 4)            # S = 32, all-causal
    rule = Rule(8, 1, -1)
    S, d = lay.S, 32
    q = rng.standard_normal((S, 2, d))
    k = rng.standard_normal((S, 1, d))
    v = np.eye(S)[:, None, :]
    res = oracle.run_layer(q, k, v, lay, rule, 0.3)
    tq = torch.from_numpy(q).permute(1, 0, 2)[None]
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(2, 0)[None]
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(2, 0)[None]
    P = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, is_causal=True, scale=0.3)[0].numpy()   # [H, S, S]
    for h in range(2):
        s = (q[:, h, :] @ k[:, 0, :].T) * 0.3
        for i in range(S):
            lse = s[i, : i + 1] - np.log(P[h, i, : i + 1])
            np.testing.assert_allclose(lse, res["LSE"][h, i], atol=1e-10)


def test_invariants_and_isolation():
    lay, q, k, v = _rand_case(3, (2, 0, 4), (7, 5, 9), (6, 3, 11), 4, 4, 2, 8)
    rule = Rule(8, 1, 2)
    res = oracle.run_layer(q, k, v, lay, rule, 0.4)
    # each query row's mass sums to one: frames + non-visual = N_q per video
    for n in range(lay.n_seq):
        f0, F = int(lay.frame0[n]), int(lay.n_frames[n])
        tot = res["E"][:, f0:f0 + F].sum(axis=1) + res["text_mass"][:, n]
        np.testing.assert_allclose(tot, lay.n_text[n], atol=1e-12)
    assert (res["E"] >= 0).all()
    # constant values pass through every softmax unchanged
    vc = np.broadcast_to(np.arange(8.0), v.shape).copy()
    rc = oracle.run_layer(q, k, vc, lay, rule, 0.4)
    np.testing.assert_allclose(rc["O"], np.broadcast_to(np.arange(8.0),
                                                        rc["O"].shape),
                               atol=1e-12)
    # permuting keys inside one frame leaves the evidence unchanged
    f = 3
    toks = np.nonzero(lay.frame == f)[0]
    perm = np.arange(lay.S)
    perm[toks] = toks[::-1]
    rp = oracle.run_layer(q, k[perm], v[perm], lay, rule, 0.4)
    np.testing.assert_allclose(rp["E"], res["E"], atol=1e-12)
    # no leakage across videos: perturbing video 2 leaves videos 0, 1 as is
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    sl = slice(int(lay.tok0[2]), int(lay.end[2]))
    q2[sl] += 1.0
    k2[sl] *= -2.0
    v2[sl] += 3.0
    r2 = oracle.run_layer(q2, k2, v2, lay, rule, 0.4)
    keep = lay.seq[res["rows"]] < 2
    assert np.array_equal(r2["O"][keep], res["O"][keep])
    assert np.array_equal(r2["LSE"][:, keep], res["LSE"][:, keep])
    fk = lay.frame0[2]
    assert np.array_equal(r2["E"][:, :fk], res["E"][:, :fk])


def _evidence_layer(w, layer=0, seed=0):
    ns, nf, nt = wl.layout_arrays(w, seed)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    rule = Rule(w.block, w.sink_blocks, w.window)
    q, k, v = wl.gen_layer(w, layer, seed).as_f64()
    E, tm, _, _, _ = oracle.attention.evidence(q, k, v, lay, rule,
                                               w.softmax_scale)
    return lay, E, tm


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_planted_frames_rank_first(cid):
    w = wl.get(cid)
    lay, E, tm = _evidence_layer(w)
    _, core, _ = wl.plant_table(w)
    e_qf, pooled = oracle.frame_evidence(E[None], lay.n_frames, lay.n_text)
    top = oracle.topk_per_video(pooled, lay.n_frames, [len(core)])[0]
    assert sorted(top.tolist()) == sorted(core.tolist())


@pytest.mark.slow
def test_planted_frames_rank_first_ragged():
    w = wl.get(5)
    lay, E, tm = _evidence_layer(w)
    _, core, _ = wl.plant_table(w)
    _, pooled = oracle.frame_evidence(E[None], lay.n_frames, lay.n_text)
    ks = []
    for n in range(lay.n_seq):
        f0, F = int(lay.frame0[n]), int(lay.n_frames[n])
        ks.append(int(((core >= f0) & (core < f0 + F)).sum()))
    tops = oracle.topk_per_video(pooled, lay.n_frames, ks)
    for n in range(lay.n_seq):
        f0, F = int(lay.frame0[n]), int(lay.n_frames[n])
        want = core[(core >= f0) & (core < f0 + F)] - f0
        assert sorted(tops[n].tolist()) == sorted(want.tolist())


@pytest.mark.slow
def test_segment_core_outranks_unplanted():
    w = wl.get(4)
    lay, E, tm = _evidence_layer(w)
    strength, core, _ = wl.plant_table(w)
    _, pooled = oracle.frame_evidence(E[None], lay.n_frames, lay.n_text)
    assert pooled[core].min() > pooled[strength == 0].max()


def test_aggregation_and_topk_by_hand():
    E = np.zeros((2, 2, 5))
    E[0, 0] = [1, 2, 3, 0, 4]
    E[0, 1] = [1, 0, 1, 0, 0]
    E[1, 0] = [0, 0, 2, 2, 2]
    E[1, 1] = [2, 2, 0, 2, 0]
    e_qf, pooled = oracle.frame_evidence(E, [3, 2], [2, 4])
    # video 0 (frames 0-2) has 2 query rows, video 1 (frames 3-4) has 4
    np.testing.assert_allclose(e_qf[0], [0.5, 0.5, 1.0, 0.0, 0.5])
    np.testing.assert_allclose(e_qf[1], [0.5, 0.5, 0.5, 0.5, 0.25])
    np.testing.assert_allclose(pooled, [0.5, 0.5, 0.75, 0.25, 0.375])
    tops = oracle.topk_per_video(pooled, [3, 2], [2, 1])
    assert tops[0].tolist() == [2, 0]      # tie 0/1 broken by index
    assert tops[1].tolist() == [1]

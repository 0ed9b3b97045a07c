"""Host-side checks of libevisel.so (no GPU): exported symbols, the plan's
block partition and active pairs against the oracle's token predicate, the
work list's coverage, and the documented error codes."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from oracle import blocks as oblocks
from oracle.layout import Layout, Rule
import workloads as wl
import paper_2608_05780_amd as ev

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ev.LIB_PATH):
        pytest.skip("libevisel.so not built (run __graft_entry__.build())")
    return ev.load()


def test_exports_every_declared_symbol(lib):
    hdr = open(os.path.join(ROOT, "include", "evisel.h")).read()
    declared = set(re.findall(r"\b(evisel_[a-z_]+)\s*\(", hdr))
    assert declared == set(ev.EXPORTED)
    raw = ctypes.CDLL(ev.LIB_PATH)
    for name in declared:
        assert hasattr(raw, name), name


def _plan(n_frames, n_text, Nv, rule, hq=4, hkv=2, n_sys=None, tau_p=0.0):
    return ev.build_block_mask(n_frames, n_text, Nv, rule.block,
                               rule.sink_blocks, rule.window, hq, hkv,
                               n_sys=n_sys, host_only=True, tau_p=tau_p)


CASES = [
    ((0,), (32,), (32,), 16, Rule(64, 1, -1)),
    ((0,), (128,), (64,), 64, Rule(64, 1, 8)),
    ((3, 0, 70), (9, 14, 5), (4, 64, 130), 32, Rule(64, 1, 2)),
    ((5,), (23,), (9,), 16, Rule(32, 2, 3)),
    ((0, 1), (7, 3), (3, 3), 4, Rule(8, 0, 1)),
]


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_plan_matches_oracle_blocks(lib, ci):
    ns, nf, nt, Nv, rule = CASES[ci]
    m = _plan(nf, nt, Nv, rule, n_sys=ns)
    lay = Layout(ns, nf, nt, Nv)
    blk, rp, col = oblocks.active_csr(lay, rule, brute=lay.S < 3000)
    got = ev.mask_export(m)
    np.testing.assert_array_equal(got["start"], blk[:, 0])
    np.testing.assert_array_equal(got["len"], blk[:, 1])
    np.testing.assert_array_equal(got["region"], blk[:, 2])
    np.testing.assert_array_equal(got["video"], blk[:, 3])
    np.testing.assert_array_equal(got["row_ptr"], rp)
    np.testing.assert_array_equal(got["col"], col)
    st = m.stats
    assert st["n_tokens"] == lay.S and st["n_frames_total"] == lay.T
    assert st["n_text_rows"] == int(np.sum(nt))


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_workload_plans(lib, cid):
    w = wl.get(cid)
    ns, nf, nt = wl.layout_arrays(w)
    rule = Rule(w.block, w.sink_blocks, w.window)
    m = _plan(nf, nt, w.tokens_per_frame, rule, hq=w.hq, hkv=w.hkv, n_sys=ns)
    got = ev.mask_export(m)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    if cid <= 3:
        blk, rp, col = oblocks.active_csr(lay, rule)
        np.testing.assert_array_equal(got["row_ptr"], rp)
        np.testing.assert_array_equal(got["col"], col)
    expect = {1: 45, 2: 1364, 3: 3030, 4: 20330}
    if cid in expect:
        assert m.stats["n_active_pairs"] == expect[cid]
    _check_work(m, got, w.hq)


@pytest.mark.parametrize("hq,hkv", [(28, 4), (6, 2), (2, 2), (8, 2)])
def test_odd_heads_are_paired(lib, hq, hkv):
    """With an odd number of query heads per kv head, the odd head of each
    group runs as paired items (two query blocks per work-group): every
    region with two or more blocks pairs them, query-token tiles pair chunk
    by chunk, and only a region's last odd block stays alone. Even groups
    have no paired items. Top-p masks pair the same way over their
    all-causal candidate rows."""
    ns, nf, nt, Nv, rule = CASES[2]
    m = _plan(nf, nt, Nv, rule, hq=hq, hkv=hkv, n_sys=ns)
    got = ev.mask_export(m)
    _check_work(m, got, hq)
    wk = ev.mask_export_work(m)
    group = hq // hkv
    n_paired = int((wk["qblock2"] >= 0).sum())
    if group % 2 == 0:
        assert n_paired == 0 and m.stats["n_paired_tiles"] == 0
    else:
        region, video = got["region"], got["video"]
        odd = {}
        for idx, qb, h0, nh, run, s in _work_units(m, got, hq):
            if h0 % group == group - 1:
                odd.setdefault((qb, h0), []).append(idx)
        paired_blocks = {}
        for qb, q2, h0 in zip(wk["qblock"], wk["qblock2"], wk["head"]):
            if q2 >= 0:
                paired_blocks.setdefault(int(h0), set()).update(
                    (int(qb), int(q2)))
        for g in range(hkv):
            h = g * group + group - 1
            for n in range(len(nf)):
                for r in (0, 1, 2):
                    ids = np.nonzero((video == n) & (region == r))[0]
                    lone = set(ids.tolist()) - paired_blocks.get(h, set())
                    assert len(lone) == len(ids) % 2, (h, n, r, lone)
                    if lone:
                        assert lone == {int(ids[-1])}
        assert n_paired > 0
    mt = _plan(nf, nt, Nv, rule, hq=hq, hkv=hkv, n_sys=ns, tau_p=0.97)
    _check_work(mt, ev.mask_export(mt), hq)
    n_paired_topp = int((ev.mask_export_work(mt)["qblock2"] >= 0).sum())
    assert (n_paired_topp > 0) == (group % 2 == 1)


def _work_units(m, csr, hq):
    """The work list as (launch index, query block, first head, heads, CSR
    run, slot) units: an ordinary item is one unit; a paired item (the odd
    head of a kv group over two query blocks of one video and region) is
    one unit per query block, whose CSR run is read back from its tiles.
    Checks that a paired item's tiles are the two runs merged by key block."""
    wk = ev.mask_export_work(m)
    pt = ev.mask_export_paired(m)
    region, col = csr["region"], csr["col"]
    group = hq // m.stats["hkv"]
    units = []
    for idx, (qb, h0, nh, a, e, s, q2, s2) in enumerate(zip(
            wk["qblock"], wk["head"], wk["nheads"], wk["kb_begin"],
            wk["kb_end"], wk["slot"], wk["qblock2"], wk["slot2"])):
        if qb < 0:
            continue
        if q2 < 0:
            assert s2 == -1
            units.append((idx, int(qb), int(h0), int(nh), (int(a), int(e)),
                          int(s)))
            continue
        assert nh == 1 and group % 2 == 1 and h0 % group == group - 1
        assert csr["video"][qb] == csr["video"][q2]
        assert region[qb] == region[q2] and qb != q2
        assert (s2 >= 0) == (s >= 0) == (region[qb] == 2)
        blocks = pt["block"][a:e]
        assert len(blocks) > 0 and np.all(np.diff(blocks) > 0)
        pa, pb = pt["pos_a"][a:e], pt["pos_b"][a:e]
        assert np.all((pa >= 0) | (pb >= 0))
        for q, pos, sl in ((qb, pa, s), (q2, pb, s2)):
            p = pos[pos >= 0]
            assert len(p) > 0 and np.all(np.diff(p) == 1)   # one run
            np.testing.assert_array_equal(col[p], blocks[pos >= 0])
            units.append((idx, int(q), int(h0), 1, (int(p[0]), int(p[-1]) + 1),
                          int(sl)))
    return units


def _check_work(m, csr, hq):
    """Every (query block, head) is covered exactly once by contiguous runs of
    its CSR row; heads of an item share a kv head; query-token items use
    distinct slots that exactly fill [0, n_chunk_slots); the query-token
    chunks that read the same key range (same video, kv head and chunk
    index) are launched on one XCD (work-group i runs on XCD i mod 8)."""
    region, rp = csr["region"], csr["row_ptr"]
    group = hq // m.stats["hkv"]
    seen, text_items = {}, []
    xcd_of = {}
    for idx, qb, h0, nh, (a, e), s in _work_units(m, csr, hq):
        if region[qb] == 2:
            xcd_of[(qb, h0, a)] = idx % 8
        assert rp[qb] <= a < e <= rp[qb + 1]
        assert 1 <= nh <= 4 and h0 // group == (h0 + nh - 1) // group
        for i in range(nh):
            seen.setdefault((qb, h0 + i), []).append((a, e))
        if region[qb] == 2:
            text_items.append((qb, h0, nh, s))
        else:
            assert s == -1 and (a, e) == (rp[qb], rp[qb + 1])
    assert len(seen) == len(region) * hq
    for (qb, h), runs in seen.items():
        runs.sort()
        assert runs[0][0] == rp[qb] and runs[-1][1] == rp[qb + 1]
        for (a0, e0), (a1, e1) in zip(runs, runs[1:]):
            assert e0 == a1
    slots = []
    for qb, h0, nh, s in text_items:
        nch = len(seen[(qb, h0)])
        slots.extend(s + i * nch for i in range(nh))
    assert sorted(slots) == list(range(m.stats["n_chunk_slots"]))
    groups = {}
    for qb, h0, nh, s in text_items:
        runs = sorted(seen[(qb, h0)])
        for c, (a, e) in enumerate(runs):
            if (qb, h0, a) in xcd_of:
                key = (int(csr["video"][qb]), h0 // group, c)
                groups.setdefault(key, set()).add(xcd_of[(qb, h0, a)])
    assert all(len(x) == 1 for x in groups.values()), groups


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_topp_plan_is_all_causal_candidates(lib, ci):
    """Top-p masks take every causal block as a candidate (the retained
    subset is decided on the device): the CSR equals the all-causal rule's,
    and the history word count covers the longest selectable history."""
    ns, nf, nt, Nv, rule = CASES[ci]
    m = _plan(nf, nt, Nv, rule, n_sys=ns, tau_p=0.97)
    causal = Rule(rule.block, 0, -1)
    lay = Layout(ns, nf, nt, Nv)
    blk, rp, col = oblocks.active_csr(lay, causal, brute=lay.S < 3000)
    got = ev.mask_export(m)
    np.testing.assert_array_equal(got["row_ptr"], rp)
    np.testing.assert_array_equal(got["col"], col)
    from oracle import topp
    b = topp.Blocks(lay, rule.block)
    assert m.stats["hist_words"] == max(1, -(-(b.max_count - 1) // 32))
    assert abs(m.stats["tau_p"] - 0.97) < 1e-7
    _check_work(m, got, 4)


def _status(fn):
    with pytest.raises(ev.EviselError) as ei:
        fn()
    return ei.value.status


def test_error_codes(lib):
    r = Rule(64, 1, 8)
    assert _status(lambda: _plan([4], [2], 64, r, hq=6, hkv=4)) == \
        ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([0], [2], 64, r)) == ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [0], 64, r)) == ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 0, r)) == ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 64, Rule(0, 1, 8))) == \
        ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 64, Rule(64, -1, 8))) == \
        ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 64, Rule(64, 1, -2))) == \
        ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 64, r, n_sys=[-1])) == \
        ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 64, r, tau_p=1.5)) == \
        ev.ERR_INVALID_ARG
    assert _status(lambda: _plan([3], [2], 64, r, tau_p=-0.25)) == \
        ev.ERR_INVALID_ARG
    # more candidate key blocks per query block than the kernel's list holds
    assert _status(lambda: _plan([2100], [2], 64, r, tau_p=0.9)) == \
        ev.ERR_UNSUPPORTED
    # compute calls refuse a host-only plan before touching the device
    m = _plan([3], [2], 64, r)
    st = lib.evisel_sparse_prefill(m.handle, 0, 1, None, None, None, 128, 0,
                                   0.1, None, None, None, None, None, None,
                                   None, 0, None)
    assert st == ev.ERR_INVALID_ARG
    assert b"device" in lib.evisel_last_error()
    st = lib.evisel_frame_evidence(m.handle, None, 1, None, None, None, None,
                                   None, None, None)
    assert st == ev.ERR_INVALID_ARG
    assert lib.evisel_sparse_prefill_workspace(m.handle, 96) == 0
    assert lib.evisel_sparse_prefill_workspace(m.handle, 128) > 0
    assert lib.evisel_mask_info(None, None) == ev.ERR_INVALID_ARG
    st = lib.evisel_select_blocks(m.handle, None, None, 128, 0, 0.1, None,
                                  None, None, 0, None)
    assert st == ev.ERR_INVALID_ARG
    lib.evisel_mask_free(None)                   # ignored
    # kernel-timing sessions: argument errors come before any HIP call
    assert lib.evisel_profile_begin(0, 0, 1) == ev.ERR_INVALID_ARG
    assert lib.evisel_profile_begin(4, 0, 0) == ev.ERR_INVALID_ARG
    assert lib.evisel_profile_end(None, None) == ev.ERR_INVALID_ARG

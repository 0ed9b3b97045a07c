"""GPU parity of the adaptive top-p retention path (evisel_select_blocks and
evisel_sparse_prefill with tau_p > 0) against the oracle (appendix "Detailed
Sparse Prefilling").

Retention is an integer result decided by floating point, and the kernel
takes it in fp32 while the oracle works in fp64. A (head, row) is
"ambiguous" when the oracle's decision is within the kernel's rounding of
flipping: the cumulative probability just before or at the cut lies within
eps_c of tau_p, or the last retained and first dropped probabilities differ
by less than 2 eps_e relative. eps_e bounds the kernel's relative error in
exp(g_j - g_max): twice the affinity error bound, scale * sum_c |q_c|
|kbar_jc| * (2^-16 + (2d + 70) 2^-24) (bf16 hi/lo split of kbar, the fp32
block-mean sum and the MFMA accumulation), plus 1e-6; eps_c = 2 eps_e +
|H| 2^-23. Every non-ambiguous (head, row) must retain exactly the oracle's
set; an ambiguous one may differ but must still be a valid top-p set within
those bounds. Outputs and LSE are compared on the (head, row) pairs whose
sets agree, evidence on the frames that no disagreeing query row changes;
tolerances as for the static rule.
"""
import numpy as np
import pytest

from oracle.layout import Layout
from oracle import topp
import workloads as wl
from gpu_harness import run_gpu, sample_rows, to_device, say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    pytest.ev = gpu_lib

O_TOL, E_TOL, LSE_TOL = 2e-2, 1e-3, 2e-3
TAU = float(np.float32(0.97))


def _layout(w, seed=0):
    ns, nf, nt = wl.layout_arrays(w, seed)
    return Layout(ns, nf, nt, w.tokens_per_frame)


def _gpu_bits(ev, mask, w, layer, seed=0, inputs=None):
    import torch
    inputs = inputs if inputs is not None else wl.gen_layer(w, layer, seed)
    q, k, _ = to_device(inputs, w, torch)
    st = mask.stats
    nb, W = st["n_blocks"], st["hist_words"]
    rb = torch.full((w.hq, nb, W, 64), -1, dtype=torch.int32, device="cuda")
    ub = torch.full((w.hq, nb, W), -1, dtype=torch.int32, device="cuda")
    ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d),
                     dtype=torch.uint8, device="cuda")
    ev.select_blocks(mask, q, k, rb, ub, ws, softmax_scale=w.softmax_scale)
    torch.cuda.synchronize()
    return rb.cpu().numpy(), ub.cpu().numpy()


def _keep_of_rows(ev, rb, mask, blk, rows, max_count):
    """GPU retention of token ``rows`` in the oracle's layout
    [Hq, R, max_count]."""
    ex = ev.mask_export(mask)
    bid = np.searchsorted(ex["start"], rows, side="right") - 1
    r = rows - ex["start"][bid]
    words = rb[:, bid, :, r].view(np.uint32)        # [R, Hq, W]
    words = np.moveaxis(words, 0, 1)                 # [Hq, R, W]
    j = np.arange(min(max_count, 32 * words.shape[2]))
    bits = ((words[:, :, j // 32] >> (j % 32).astype(np.uint32)) & 1).astype(
        bool)
    nh = np.maximum(blk.local[rows], 0)
    inside = j[None, None, :] < nh[None, :, None]
    # bits past the history must be zero
    assert not (bits & ~inside).any(), "bits set past a row's history"
    keep = np.zeros(words.shape[:2] + (max_count,), bool)
    keep[:, :, :j.size] = bits
    return keep


def _classify(q, k, lay, blk, rows, keep_o, keep_g, info, scale, tau, d,
              kbar=None):
    """(match [Hq, R], ambiguous [Hq, R]); asserts that every mismatch is
    ambiguous and still a valid top-p set. ``kbar``: the oracle's mean keys
    when ``k`` is not at hand."""
    if kbar is None:
        kbar = topp.mean_keys(k, blk)
    hq, hkv = q.shape[1], kbar.shape[1]
    grp = hq // hkv
    nh = info["nh"]
    match = (keep_o == keep_g).all(axis=2)
    amb = np.zeros_like(match)
    u_aff = 2.0 ** -16 + (2 * d + 70) * 2.0 ** -24
    groups = {}
    for j, i in enumerate(rows):
        groups.setdefault((int(lay.seq[i]), int(blk.local[i])), []).append(j)
    n_bad = 0
    for (n, lb), idx in groups.items():
        if lb <= 0:
            continue
        idx = np.asarray(idx)
        hist = kbar[blk.first[n]:blk.first[n] + lb]
        for h in range(hq):
            qa = np.abs(q[rows[idx], h, :])
            bound = (qa @ np.abs(hist[:, h // grp, :]).T).max(axis=1) * scale
            eps_e = 2 * bound * u_aff + 1e-6
            eps_c = 2 * eps_e + lb * 2.0 ** -23
            cb, ca = info["c_before"][h, idx], info["c_at"][h, idx]
            pl, pn = info["p_last"][h, idx], info["p_next"][h, idx]
            a = ((cb > tau - eps_c) | (ca < tau + eps_c) |
                 ((pn >= 0) & (pl - pn < 2 * eps_e * pl)))
            amb[h, idx] = a
            for t in np.nonzero(~match[h, idx])[0]:
                jj = idx[t]
                assert a[t], (f"head {h} row {rows[jj]}: retention differs "
                              "outside the rounding margin")
                g = q[rows[jj], h] @ hist[:, h // grp].T * scale
                p = np.exp(g - g.max())
                p /= p.sum()
                kept = keep_g[h, jj, :lb]
                m = p[kept].sum()
                assert m >= tau - eps_c[t]
                assert m - p[kept].min() < tau + eps_c[t]
                if (~kept).any():
                    assert p[kept].min() >= p[~kept].max() * (1 - 2 * eps_e[t])
                n_bad += 1
    say(f"  retention: {match.size} (head, row) pairs, {int(amb.sum())} "
        f"ambiguous, {n_bad} differ")
    return match, amb


def _run_case(w, rows_budget=None, seed=0, layers=None, transform=None):
    ev = pytest.ev
    lay = _layout(w, seed)
    blk = topp.Blocks(lay, w.block)
    layers = layers if layers is not None else list(range(w.n_layers))
    keeps = {}
    inputs = {l: wl.gen_layer(w, l, seed) for l in layers}
    if transform is not None:
        inputs = {l: transform(x, lay, blk) for l, x in inputs.items()}
    res = run_gpu(ev, w, layers, seed, layer_inputs=lambda l: inputs[l])
    for j, l in enumerate(layers):
        q, k, v = inputs[l].as_f64()
        rows = (np.arange(lay.S) if rows_budget is None else
                sample_rows(lay, rows_budget, seed + 17 * l))
        ref = topp.run_layer(q, k, v, lay, w.block, w.tau_p,
                             w.softmax_scale, rows)
        rb, ub = _gpu_bits(ev, res.mask, w, l, seed, inputs=inputs[l])
        mc = ref["keep"].shape[2]
        kg = _keep_of_rows(ev, rb, res.mask, blk, rows, mc)
        match, _ = _classify(q, k, lay, blk, rows, ref["keep"], kg,
                             ref["info"], w.softmax_scale, w.tau_p, w.d)
        # outputs on agreeing (head, row) pairs
        Og = res.O[j][rows].astype(np.float64)          # [R, Hq, d]
        sel = match.T                                    # [R, Hq]
        scale_o = max(np.abs(ref["O"]).max(), 1e-30)
        o_err = np.abs(Og - ref["O"])[sel].max() / scale_o
        lse_err = np.abs(res.LSE[j][:, rows] - ref["LSE"])[match].max()
        # evidence: drop frames touched by disagreeing query rows
        txt = ref["rows_txt"]
        kt = _keep_of_rows(ev, rb, res.mask, blk, txt, mc)
        mt, _ = _classify(q, k, lay, blk, txt, ref["keep_txt"], kt,
                          ref["info_txt"], w.softmax_scale, w.tau_p, w.d)
        okf = np.ones((w.hq, lay.T), bool)
        for h, jj in zip(*np.nonzero(~mt)):
            i = txt[jj]
            n = lay.seq[i]
            diff = np.nonzero(kt[h, jj] != ref["keep_txt"][h, jj])[0]
            for b in diff:
                toks = blk.tokens(n, int(b))
                fr = lay.frame[toks]
                okf[h, fr[fr >= 0]] = False
        e_err = np.abs(res.E[j] - ref["E"])[okf].max()
        t_err = np.abs(res.text_mass[j] - ref["text_mass"]).max()
        say(f"  layer {l}: O rel err {o_err:.2e}  LSE {lse_err:.2e}  "
            f"E {e_err:.2e} ({int((~okf).sum())} frames excluded)  "
            f"text_mass {t_err:.2e}")
        assert o_err <= O_TOL and lse_err <= LSE_TOL
        assert e_err <= E_TOL
        if mt.all():
            assert t_err <= E_TOL
        if w.dtype == "fp32":
            # fp32 LSE error grows with the logits' magnitude (large under
            # the structured keys): 2^-24 per operation on |LSE|-sized terms
            lse_tight = 1e-5 + 1e-6 * np.abs(ref["LSE"]).max()
            assert o_err <= 1e-4 and e_err <= 1e-5 and lse_err <= lse_tight
        keeps[l] = (ref, kg, rb, ub)
    return res, keeps


def _small(name, **kw):
    base = dict(name=name, config_id=900, n_layers=1, hq=4, hkv=2, d=128,
                dtype="bf16", tokens_per_frame=32, block=64, sink_blocks=1,
                window=8, plant="choose", tau_p=0.9,
                plant_args={"count": 2, "s_frame": (2.0, 2.0),
                            "s_query": 2.0})
    base.update(kw)
    return wl.Workload(**base)


SMALL = {
    "ragged_sys_struct": _small(
        "ragged-sys-struct", n_frames=(9, 14, 5), n_text=(64, 32, 130),
        n_sys=(5, 0, 70), n_videos=3, key_struct=(2.0, 2.0, 0.8)),
    "struct_d64_fp32": _small(
        "struct-d64-fp32", dtype="fp32", d=64, hq=4, hkv=1,
        tokens_per_frame=16, n_frames=(40,), n_text=(48,), n_sys=(3,),
        key_struct=(2.0, 2.0, 0.8), tau_p=TAU),
    "plain_d64": _small(
        "plain-d64", d=64, hq=8, hkv=2, tokens_per_frame=64,
        n_frames=(24,), n_text=(100,), n_sys=(0,), tau_p=TAU),
    "tau_one": _small(
        "tau-one", tokens_per_frame=64, n_frames=(20,), n_text=(64,),
        n_sys=(0,), tau_p=1.0),
    # three query heads per kv head: the odd head runs as paired items
    # (two visual blocks, or the same chunk of two query-token blocks, per
    # work-group), each half skipping what its own rows did not retain
    "odd_group_struct": _small(
        "odd-group-struct", hq=6, hkv=2, n_frames=(9, 40, 5),
        n_text=(64, 70, 130), n_sys=(5, 0, 70), n_videos=3,
        key_struct=(2.0, 2.0, 0.8)),
    "odd_group_fp32": _small(
        "odd-group-fp32", dtype="fp32", d=64, hq=3, hkv=1,
        tokens_per_frame=16, n_frames=(48,), n_text=(100,), n_sys=(3,),
        key_struct=(2.0, 2.0, 0.8), tau_p=TAU),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_topp_small(name):
    w = SMALL[name]
    say(f"case {name}")
    _run_case(w)


def test_topp_tiny_fp32_config():
    w = wl.get(1, tau_p=TAU)
    say("case config-1 top-p")
    _run_case(w)


def test_topp_uniform_affinity_ties():
    # Q = 0: every affinity is exactly 0, so retention is decided by the tie
    # rule (lower block index first)
    w = _small("uniform-q0", d=64, hq=2, hkv=1, tokens_per_frame=16,
               n_frames=(96, 30), n_text=(70, 9), n_sys=(0, 4), n_videos=2,
               tau_p=TAU)
    ev = pytest.ev
    lay = _layout(w)
    blk = topp.Blocks(lay, w.block)
    ns, nf, nt = wl.layout_arrays(w)
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, tau_p=w.tau_p)
    import torch
    lay_in = wl.gen_layer(w, 0, q_override="zero")
    q, k, _ = to_device(lay_in, w, torch)
    st = mask.stats
    rb = torch.full((w.hq, st["n_blocks"], st["hist_words"], 64), -1,
                    dtype=torch.int32, device="cuda")
    ub = torch.full((w.hq, st["n_blocks"], st["hist_words"]), -1,
                    dtype=torch.int32, device="cuda")
    ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d),
                     dtype=torch.uint8, device="cuda")
    ev.select_blocks(mask, q, k, rb, ub, ws)
    torch.cuda.synchronize()
    rows = np.arange(lay.S)
    kg = _keep_of_rows(ev, rb.cpu().numpy(), mask, blk, rows,
                       blk.max_count)
    q64, k64, _ = lay_in.as_f64()
    ko, info = topp.select(q64, k64, lay, blk, w.tau_p, w.softmax_scale)
    from fractions import Fraction
    checked = 0
    for j, i in enumerate(rows):
        n = int(blk.local[i])
        if n <= 0:
            assert not kg[:, j].any()
            continue
        t = Fraction(w.tau_p) * n
        if abs(t - round(t)) < Fraction(1, 1000):
            continue               # the cut sits on a rounding boundary
        want = np.zeros(blk.max_count, bool)
        want[:int(np.ceil(float(t)))] = True
        for h in range(w.hq):
            np.testing.assert_array_equal(kg[h, j], want)
            np.testing.assert_array_equal(ko[h, j], want)
        checked += 1
    assert checked > 1000


def _dup_key_blocks(x, lay, blk):
    """Every third visual block takes block 1's keys (bit for bit), so those
    blocks share one mean key and every row sees a run of exactly equal
    affinities, which some rows' cuts fall inside."""
    k = x.k.copy()
    starts = [s for s in range(lay.S) if lay.frame[s] >= 0 and
              (s == 0 or lay.frame[s - 1] != lay.frame[s])]
    src = starts[1]
    for j, s in enumerate(starts):
        if j >= 3 and j % 3 == 0 and s + 64 <= lay.S and \
                (lay.frame[s:s + 64] >= 0).all():
            k[s:s + 64] = k[src:src + 64]
    return wl.Layer(q=x.q, k=k, v=x.v, u=x.u)


def _scale_queries(x, lay, blk, f=200.0):
    """Queries scaled so that a row's affinities span a few hundred log2
    units: most probabilities underflow to +0 in fp32 and rows keep one or
    two blocks."""
    q = wl.bf16_bits(wl.bf16_bits_to_f32(x.q) * np.float32(f))
    return wl.Layer(q=q, k=x.k, v=x.v, u=x.u)


def test_topp_equal_affinity_runs():
    w = _small("dup-keys", tokens_per_frame=64, n_frames=(150,),
               n_text=(64,), n_sys=(0,), tau_p=TAU)
    say("case duplicated key blocks")
    _, keeps = _run_case(w, rows_budget=512, transform=_dup_key_blocks)
    # equal probabilities sit inside the rounding margin, but the rule that
    # takes them in block order is exact: every row keeps the oracle's set
    ref, kg, _, _ = keeps[0]
    np.testing.assert_array_equal(kg, ref["keep"])


def test_topp_equal_affinity_runs_long_register_form():
    # the same tie rule in the long register form (600-block histories, 38
    # entries per lane, three mask words per lane)
    w = _small("dup-keys-long", d=64, hq=2, hkv=1, tokens_per_frame=64,
               n_frames=(600,), n_text=(40,), n_sys=(0,), tau_p=TAU)
    say("case duplicated key blocks, long register form")
    _, keeps = _run_case(w, rows_budget=256, transform=_dup_key_blocks)
    ref, kg, _, _ = keeps[0]
    np.testing.assert_array_equal(kg, ref["keep"])


def test_topp_underflowing_probabilities():
    w = _small("scaled-q", tokens_per_frame=64, n_frames=(120,),
               n_text=(64,), n_sys=(2,), tau_p=TAU)
    say("case queries x200")
    _, keeps = _run_case(w, rows_budget=512, transform=_scale_queries)
    ref, kg, _, _ = keeps[0]
    np.testing.assert_array_equal(kg, ref["keep"])


def test_topp_skips_tiles_and_is_deterministic():
    w = SMALL["ragged_sys_struct"]
    ev = pytest.ev
    lay = _layout(w)
    blk = topp.Blocks(lay, w.block)
    res, keeps = _run_case(w)
    ref, kg, rb, ub = keeps[0]
    # the union over a block's rows leaves some history blocks out
    ex = ev.mask_export(res.mask)
    nh = np.array([max(int(blk.local[s]), 0) for s in ex["start"]])
    pop = np.array([[bin(int(x) & 0xFFFFFFFF).count("1") for x in row.ravel()]
                    for row in ub.reshape(w.hq, -1)]).reshape(ub.shape).sum(2)
    assert (pop < nh[None, :]).sum() > 0
    say(f"  union keeps {pop.sum()} of {nh.sum() * w.hq} history blocks")
    # union = OR of the rows, and a second call gives identical bits
    rb2, ub2 = _gpu_bits(ev, res.mask, w, 0)
    np.testing.assert_array_equal(rb, rb2)
    np.testing.assert_array_equal(ub, ub2)
    orr = np.bitwise_or.reduce(rb.view(np.uint32), axis=3)
    np.testing.assert_array_equal(orr, ub.view(np.uint32))
    res2 = run_gpu(ev, w, [0])
    np.testing.assert_array_equal(res.O[0], res2.O[0])
    np.testing.assert_array_equal(res.E, res2.E)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_topp_long_history_register_form(dtype):
    # 600 visual blocks: a row's share of its history (38 entries at 16
    # lanes per row) exceeds the common register form, so the long form
    # (up to 72 entries per lane, two waves per SIMD) runs it
    w = _small("long-history", d=64, hq=2, hkv=1, tokens_per_frame=64,
               n_frames=(600,), n_text=(40,), n_sys=(6,), tau_p=TAU,
               key_struct=(1.0, 1.0, 0.9), dtype=dtype)
    say(f"case long history, long register form, {dtype}")
    _run_case(w, rows_budget=256)


def test_topp_very_long_history_streams_from_lds():
    # 1,200 visual blocks: 76 entries per lane exceed the long register
    # form too, so the retention streams each row's share from LDS (one
    # work-group per CU)
    w = _small("very-long-history", d=64, hq=2, hkv=1, tokens_per_frame=64,
               n_frames=(1200,), n_text=(40,), n_sys=(6,), tau_p=TAU,
               key_struct=(1.0, 1.0, 0.9))
    say("case very long history, LDS-streaming retention")
    _run_case(w, rows_budget=256)


def test_topp_register_rows_of_sixteen_lanes():
    # 340 visual blocks (d = 64): a row's share of the longest history fits
    # the registers only at 16 lanes per row (24 entries each). Rows whose
    # history holds 321-340 blocks (every query row among them) also get a
    # whole 32-column tile of -inf padding past the end of their affinity
    # row, which the register variant then loads as zero probabilities.
    w = _small("sixteen-lanes", d=64, hq=2, hkv=1, tokens_per_frame=64,
               n_frames=(340,), n_text=(40,), n_sys=(6,), tau_p=TAU,
               key_struct=(1.0, 1.0, 0.9))
    say("case sixteen lanes per row, register variant")
    _run_case(w, rows_budget=256)


def test_topp_config2_layer():
    w = wl.get(2, tau_p=TAU)
    say("case config-2 top-p")
    _run_case(w, rows_budget=512)


def test_topp_config4_long_video():
    # 1,026 selectable blocks: 33 history words, LDS-streaming retention
    w = wl.get(4, tau_p=TAU)
    say("case config-4 top-p, layer 0")
    _run_case(w, rows_budget=256, layers=[0])


def test_topp_config5_ragged_batch():
    # eight videos of 64-512 frames x 32 tokens, two frames per block
    w = wl.get(5, tau_p=TAU)
    say("case config-5 top-p, layer 0")
    _run_case(w, rows_budget=512, layers=[0])


@pytest.mark.timeout(900)
def test_topp_config3_all_layers_query_rows():
    """All 28 layers of the bench workload under top-p: every query row's
    retention against the oracle (differences only inside the rounding
    margin), the evidence per (head, frame) on the frames no disagreeing row
    touches, and the per-video ranking of the 28-layer pooled score. The
    oracle runs in worker processes, fed the layer the GPU ran."""
    import concurrent.futures as cf
    import multiprocessing as mp
    import torch
    from gpu_harness import oracle_topp_query_rows, _limit_threads
    from test_gpu_parity import _check_ranking
    w = wl.get(3, tau_p=TAU)
    seed = 0
    ev = pytest.ev
    lay = _layout(w, seed)
    blk = topp.Blocks(lay, w.block)
    txt = lay.text_rows()
    ns, nf, nt = wl.layout_arrays(w, seed)
    # a mask of its own for the per-layer retention bits
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, tau_p=w.tau_p)
    st = mask.stats
    rb = torch.empty((w.hq, st["n_blocks"], st["hist_words"], 64),
                     dtype=torch.int32, device="cuda")
    ub = torch.empty((w.hq, st["n_blocks"], st["hist_words"]),
                     dtype=torch.int32, device="cuda")
    ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d),
                     dtype=torch.uint8, device="cuda")
    _, core, _ = wl.plant_table(w, seed)
    planted = [int(((core >= f0) & (core < f0 + F)).sum())
               for f0, F in zip(lay.frame0, lay.n_frames)]
    ks = [int(F) for F in lay.n_frames]
    cache, futs, kept = {}, {}, {}
    ex = cf.ProcessPoolExecutor(3, mp_context=mp.get_context("spawn"),
                                initializer=_limit_threads, initargs=(5,))

    def layer_inputs(l):
        cache.clear()
        cache[l] = wl.gen_layer(w, l, seed)
        return cache[l]

    def on_layer(j, l, out, lse):
        x = cache[l]
        futs[j] = ex.submit(oracle_topp_query_rows, w, seed, x.q[txt], x.k,
                            x.v)
        q, k, _ = to_device(x, w, torch)
        ev.select_blocks(mask, q, k, rb, ub, ws, softmax_scale=w.softmax_scale)
        torch.cuda.synchronize()
        kept[j] = _keep_of_rows(ev, rb.cpu().numpy(), mask, blk, txt,
                                blk.max_count)

    try:
        layers = list(range(w.n_layers))
        res = run_gpu(ev, w, layers, seed, k_per_video=ks, keep_o=False,
                      layer_inputs=layer_inputs, on_layer=on_layer)
        E_ref_all, n_differ = [], 0
        for j in layers:
            keep, info, E_ref, tm_ref, kbar, q_txt = futs[j].result()
            qf = np.zeros((lay.S, w.hq, w.d))
            qf[txt] = q_txt
            mt, _ = _classify(qf, None, lay, blk, txt, keep, kept[j], info,
                              w.softmax_scale, w.tau_p, w.d, kbar=kbar)
            okf = np.ones((w.hq, lay.T), bool)
            for h, jj in zip(*np.nonzero(~mt)):
                i = txt[jj]
                for b in np.nonzero(kept[j][h, jj] != keep[h, jj])[0]:
                    fr = lay.frame[blk.tokens(lay.seq[i], int(b))]
                    okf[h, fr[fr >= 0]] = False
            e_err = np.abs(res.E[j] - E_ref)[okf].max()
            say(f"  layer {j}: E {e_err:.2e} "
                f"({int((~mt).sum())} (head, row) pairs differ)")
            assert e_err <= E_TOL
            if mt.all():
                assert np.abs(res.text_mass[j] - tm_ref).max() <= E_TOL
            n_differ += int((~mt).sum())
            E_ref_all.append(E_ref)
    finally:
        ex.shutdown(cancel_futures=True)
    _check_ranking(res, np.stack(E_ref_all), lay, planted)


def test_topp_config3_two_layers():
    w = wl.get(3, tau_p=TAU)
    say("case config-3 top-p, layers 0 and 1")
    _run_case(w, rows_budget=256, layers=[0, 1])

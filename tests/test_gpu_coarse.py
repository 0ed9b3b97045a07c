"""GPU parity of the paper's coarse query-frame evidence
(evisel_coarse_evidence: appendix, coarse-map equation) and a synthetic
analogue of the sparse-vs-dense alignment table (Reliability of Sparse
Attention Maps) computed from the GPU's maps.

Coarse evidence is compared with the oracle on the (head, query row) pairs
whose retention agrees with the oracle's (see the top-p tests for the
rounding-margin rule); frames that a disagreeing row's differing blocks
cover are left out. Tolerance 1e-3 (fp32: 1e-4).

The alignment test computes Pearson, Spearman, JS, Top-10 %, Keep and
Mass-recovery of the exact sparse cues (A_qf, A_ff, A_if) and of the coarse
A_qf against dense causal attention, once from the GPU's maps and once from
the oracle's sparse maps, and requires the two to agree; it prints the
table.
"""
import numpy as np
import pytest

from oracle import coarse, cues, topp
from oracle.layout import Layout, VIS
import workloads as wl
from gpu_harness import run_gpu, to_device, say
from test_gpu_topp import _gpu_bits, _keep_of_rows, TAU

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    pytest.ev = gpu_lib


def _w(name, **kw):
    base = dict(name=name, config_id=901, n_layers=1, hq=4, hkv=2, d=128,
                dtype="bf16", tokens_per_frame=32, block=64, sink_blocks=1,
                window=8, plant="choose", tau_p=TAU,
                plant_args={"count": 3, "s_frame": (2.0, 3.0),
                            "s_query": 2.0})
    base.update(kw)
    return wl.Workload(**base)


CASES = {
    "ragged_struct": _w("ragged-struct", n_frames=(9, 14, 5),
                        n_text=(64, 32, 130), n_sys=(5, 0, 70), n_videos=3,
                        key_struct=(2.0, 2.0, 0.8)),
    "fp32_d64": _w("fp32-d64", dtype="fp32", d=64, hq=4, hkv=1,
                   tokens_per_frame=16, n_frames=(40,), n_text=(48,),
                   n_sys=(3,), key_struct=(2.0, 2.0, 0.8)),
    "plain_d64": _w("plain-d64", d=64, hq=8, hkv=2, tokens_per_frame=64,
                    n_frames=(24,), n_text=(100,), n_sys=(0,)),
    "config2": wl.get(2, tau_p=TAU),
}


def _layout(w):
    ns, nf, nt = wl.layout_arrays(w)
    return Layout(ns, nf, nt, w.tokens_per_frame)


def _gpu_coarse(w, mask, l=0):
    import torch
    ev = pytest.ev
    q, k, _ = to_device(wl.gen_layer(w, l), w, torch)
    T = mask.stats["n_frames_total"]
    out = torch.full((w.hq, T), float("nan"), device="cuda")
    ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d),
                     dtype=torch.uint8, device="cuda")
    ev.coarse_evidence(mask, q, k, out, ws, softmax_scale=w.softmax_scale)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("name", list(CASES))
def test_coarse_evidence(name):
    w = CASES[name]
    ev = pytest.ev
    say(f"case {name}")
    lay = _layout(w)
    blk = topp.Blocks(lay, w.block)
    ns, nf, nt = wl.layout_arrays(w)
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, tau_p=w.tau_p)
    Eg = _gpu_coarse(w, mask)
    q, k, _ = wl.gen_layer(w, 0).as_f64()
    txt = lay.text_rows()
    keep, info = topp.select(q, k, lay, blk, w.tau_p, w.softmax_scale, txt)
    Eo = coarse.query_frame(lay, coarse.coarse_probs(
        q, k, lay, blk, keep, txt, w.softmax_scale), w.hq)
    rb, _ = _gpu_bits(ev, mask, w, 0)
    kg = _keep_of_rows(ev, rb, mask, blk, txt, keep.shape[2])
    okf = np.ones_like(Eo, bool)
    for h, j in zip(*np.nonzero((kg != keep).any(axis=2))):
        n = lay.seq[txt[j]]
        for b in np.nonzero(kg[h, j] != keep[h, j])[0]:
            fr = lay.frame[blk.tokens(n, int(b))]
            okf[h, fr[fr >= 0]] = False
    err = np.abs(Eg - Eo)[okf].max()
    say(f"  coarse evidence err {err:.2e} ({int((~okf).sum())} excluded)")
    assert err <= (1e-4 if w.dtype == "fp32" else 1e-3)
    assert np.isfinite(Eg).all()


def test_alignment_table():
    w = _w("align", n_frames=(48,), n_text=(64,), n_sys=(0,), hq=4, hkv=2,
           key_struct=(2.0, 2.0, 0.8))
    ev = pytest.ev
    lay = _layout(w)
    blk = topp.Blocks(lay, w.block)
    res = run_gpu(ev, w, [0], cues=True, keep_o=False)
    E_coarse = _gpu_coarse(w, res.mask)
    q, k, v = wl.gen_layer(w, 0).as_f64()
    rows = np.arange(lay.S)
    vis = np.nonzero(lay.region == VIS)[0]
    keep, _ = topp.select(q, k, lay, blk, w.tau_p, w.softmax_scale, rows)
    # oracle sparse (exact), coarse and dense maps
    sp = list(cues.topp_groups(q, k, v, lay, blk, keep, rows,
                               w.softmax_scale))
    co = coarse.coarse_probs(q, k, lay, blk, keep, rows, w.softmax_scale)
    de = list(coarse.dense_groups(q, k, v, lay, rows, w.softmax_scale))

    def maps(groups):
        g = list(groups)
        E = coarse.query_frame(lay, g, w.hq).sum(axis=0)
        A_ff, A_if = cues.accumulate(
            lay, [(r[lay.region[r] == VIS], kk, P[:, lay.region[r] == VIS])
                  for r, kk, P in g], w.hq)
        return E, A_ff, A_if
    Es, FFs, IFs = maps(sp)
    Ec, _, _ = maps(co)
    Ed, FFd, IFd = maps(de)
    tri = np.tril(np.ones((lay.T, lay.T), bool), -1)
    low = np.tril(np.ones((w.tokens_per_frame,) * 2, bool))[None]
    low = np.broadcast_to(low, IFd.shape)
    # the GPU's maps
    A_ff_g = np.zeros((lay.T, lay.T))
    pr = ev.mask_export_pairs(res.mask)
    A_ff_g[pr["a"], pr["b"]] = res.pairs[0]
    gpu = {"A_qf": res.E[0].sum(axis=0), "A_ff": A_ff_g[tri],
           "A_if": res.intra[0][low], "A_qf coarse": E_coarse.sum(axis=0)}
    ora = {"A_qf": Es, "A_ff": FFs[tri], "A_if": IFs[low], "A_qf coarse": Ec}
    dense = {"A_qf": Ed, "A_ff": FFd[tri], "A_if": IFd[low],
             "A_qf coarse": Ed}
    say("  cue          Pear.   Spear.  JS       Top-10%  Keep    Mass-rec")
    for name in gpu:
        mg = coarse.alignment(gpu[name], dense[name])
        mo = coarse.alignment(ora[name], dense[name])
        say(f"  {name:12s} {mg['pearson']:.3f}   {mg['spearman']:.3f}   "
            f"{mg['js']:.4f}   {mg['top10']:.3f}    {mg['keep']:.3f}   "
            f"{mg['mass_rec']:.4f}")
        for key in ("pearson", "spearman", "mass_rec"):
            assert abs(mg[key] - mo[key]) <= 5e-3, (name, key)
        assert abs(mg["js"] - mo["js"]) <= 1e-3
        assert abs(mg["keep"] - mo["keep"]) <= 2.0 / gpu[name].size
        assert abs(mg["top10"] - mo["top10"]) <= 0.1

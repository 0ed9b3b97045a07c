"""Runs the HIP probe through the C ABI and the oracle on the same seeded
inputs (shared by the GPU tests, smoke() and the benchmark's checks)."""
from __future__ import annotations

import sys
from dataclasses import dataclass

import numpy as np

import workloads as wl


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@dataclass
class GpuRun:
    O: list          # per layer numpy [S, Hq, d] float32
    LSE: list        # per layer numpy [Hq, S]
    E: np.ndarray    # [L, Hq, T]
    text_mass: np.ndarray
    e_qf: np.ndarray
    e_qf_layer: np.ndarray
    topk: list       # per video int arrays (local frame ids)
    mask: object
    pairs: object = None      # [L, n_pairs] A_ff of the exported pairs
    intra: object = None      # [L, T, N_v, N_v] A_if
    e_ff: object = None       # [L, T]


def to_device(layer: wl.Layer, w: wl.Workload, torch):
    if w.dtype == "bf16":
        cv = lambda a: torch.from_numpy(a.view(np.int16)).view(
            torch.bfloat16).cuda()
    else:
        cv = lambda a: torch.from_numpy(a).cuda()
    return cv(layer.q), cv(layer.k), cv(layer.v)


def run_gpu(ev, w: wl.Workload, layers, seed=0, k_per_video=None,
            keep_o=True, layer_inputs=None, on_layer=None, cues=False,
            work_order=None):
    """Run ``layers`` (list of layer ids) of workload ``w`` on the GPU.

    ``on_layer(j, layer_id, out, lse)`` (torch tensors on the GPU) is called
    after each layer; with ``keep_o`` the outputs are also copied to host.
    ``work_order(n_items)`` returns a permutation of the attention work list
    to launch it in (default: the plan's order)."""
    import torch
    ns, nf, nt = wl.layout_arrays(w, seed)
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, tau_p=w.tau_p)
    st = mask.stats
    if work_order is not None:
        ev.mask_permute_work(mask, work_order(st["n_work_items"]))
    S, T, nseq = st["n_tokens"], st["n_frames_total"], len(nf)
    L = len(layers)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    out = torch.empty((S, w.hq, w.d), dtype=dt, device="cuda")
    lse = torch.empty((w.hq, S), dtype=torch.float32, device="cuda")
    evid = torch.full((L, w.hq, T), float("nan"), device="cuda")
    tm = torch.full((L, w.hq, nseq), float("nan"), device="cuda")
    ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d, cues=cues),
                     dtype=torch.uint8, device="cuda")
    pairs = intra = None
    if cues:
        npair = st["n_frame_pairs"]
        pairs = torch.full((L, max(npair, 1)), float("nan"), device="cuda")
        intra = torch.full((L, T, w.tokens_per_frame, w.tokens_per_frame),
                           float("nan"), device="cuda")
    Os, LSEs = [], []
    for j, l in enumerate(layers):
        lay = layer_inputs(l) if layer_inputs else wl.gen_layer(w, l, seed)
        q, k, v = to_device(lay, w, torch)
        say(f"  gpu: {w.name} layer {l} S={S} hq={w.hq} d={w.d}")
        ev.sparse_prefill(mask, j, L, q, k, v, out, evid, ws, lse=lse,
                          text_mass=tm, softmax_scale=w.softmax_scale,
                          frame_pairs=pairs, intra_frame=intra)
        torch.cuda.synchronize()
        if on_layer is not None:
            on_layer(j, l, out, lse)
        if keep_o:
            Os.append(out.float().cpu().numpy())
            LSEs.append(lse.cpu().numpy())
    e_qf = torch.empty(T, device="cuda")
    e_qf_layer = torch.empty((L, T), device="cuda")
    topk = []
    if k_per_video is not None:
        kk = torch.tensor(list(k_per_video), dtype=torch.int32, device="cuda")
        tk = torch.full((max(1, int(sum(k_per_video))),), -1,
                        dtype=torch.int32, device="cuda")
        ev.frame_evidence(mask, evid, L, e_qf, e_qf_layer=e_qf_layer,
                          k_per_seq=kk, topk=tk)
        torch.cuda.synchronize()
        flat = tk.cpu().numpy()
        off = 0
        for k in k_per_video:
            topk.append(flat[off:off + int(k)].astype(np.int64))
            off += int(k)
    else:
        ev.frame_evidence(mask, evid, L, e_qf, e_qf_layer=e_qf_layer)
        torch.cuda.synchronize()
    e_ff = None
    if cues:
        e_ff = torch.full((L, T), float("nan"), device="cuda")
        ev.frame_evidence(mask, evid, L, e_qf, frame_pairs=pairs, e_ff=e_ff)
        torch.cuda.synchronize()
        e_ff = e_ff.cpu().numpy().astype(np.float64)
        pairs = pairs.cpu().numpy().astype(np.float64)[:, :st["n_frame_pairs"]]
        intra = intra.cpu().numpy().astype(np.float64)
    return GpuRun(Os, LSEs, evid.cpu().numpy().astype(np.float64),
                  tm.cpu().numpy().astype(np.float64),
                  e_qf.cpu().numpy().astype(np.float64),
                  e_qf_layer.cpu().numpy().astype(np.float64), topk, mask,
                  pairs, intra, e_ff)


def sample_rows(lay, n_rows, seed, run=64):
    """All query-token rows plus about ``n_rows`` other rows, drawn as
    seeded runs of ``run`` consecutive tokens at random offsets (so they
    straddle block boundaries)."""
    rng = np.random.default_rng(seed)
    txt = lay.text_rows()
    other = np.setdiff1d(np.arange(lay.S), txt)
    if other.size <= n_rows:
        return np.union1d(other, txt)
    starts = rng.choice(other.size - run, size=max(1, n_rows // run),
                        replace=False)
    pick = np.unique(np.concatenate([other[s:s + run] for s in starts]))
    return np.union1d(pick, txt)


def output_error(O_gpu, O_ref, rows):
    """max |O_gpu - O_ref| / max |O_ref| over ``rows``."""
    g = O_gpu[rows].astype(np.float64)
    return float(np.abs(g - O_ref).max() / max(np.abs(O_ref).max(), 1e-30))


def oracle_query_rows(w: wl.Workload, seed: int, qt, k, v):
    """The oracle's evidence, non-visual mass, O and LSE of one layer's query
    rows. ``qt`` holds q of those rows only (the oracle reads q at the rows
    it computes and nowhere else); k and v are whole. Inputs are bf16 bit
    patterns or fp32, as ``wl.gen_layer`` returns them. Runs in a worker
    process: it imports neither torch nor the HIP library."""
    from oracle.attention import evidence
    from oracle.layout import Layout, Rule
    ns, nf, nt = wl.layout_arrays(w, seed)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    rule = Rule(w.block, w.sink_blocks, w.window)
    if qt.dtype == np.uint16:
        cv = lambda a: wl.bf16_bits_to_f32(a).astype(np.float64)
    else:
        cv = lambda a: a.astype(np.float64)
    q = np.zeros((lay.S,) + qt.shape[1:])
    q[lay.text_rows()] = cv(qt)
    E, tm, O, LSE, _ = evidence(q, cv(k), cv(v), lay, rule, w.softmax_scale)
    return E, tm, O, LSE


def oracle_topp_query_rows(w: wl.Workload, seed: int, qt, k, v):
    """The oracle's top-p retention of one layer's query rows (``keep``,
    ``info``), their evidence and non-visual mass, the mean keys the
    retention used, and the rows' q (float64). ``qt`` holds q of those rows
    only; k and v are whole (bf16 bit patterns or fp32). Runs in a worker
    process: it imports neither torch nor the HIP library."""
    from oracle import topp
    from oracle.layout import Layout
    ns, nf, nt = wl.layout_arrays(w, seed)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    blk = topp.Blocks(lay, w.block)
    if qt.dtype == np.uint16:
        cv = lambda a: wl.bf16_bits_to_f32(a).astype(np.float64)
    else:
        cv = lambda a: a.astype(np.float64)
    txt = lay.text_rows()
    q = np.zeros((lay.S,) + qt.shape[1:])
    q[txt] = cv(qt)
    k64, v64 = cv(k), cv(v)
    keep, info = topp.select(q, k64, lay, blk, w.tau_p, w.softmax_scale, txt)
    E, tm, _, _ = topp.evidence(q, k64, v64, lay, blk, keep, txt,
                                w.softmax_scale)
    return keep, info, E, tm, topp.mean_keys(k64, blk), q[txt]


def _limit_threads(n):
    from threadpoolctl import threadpool_limits
    threadpool_limits(n)


#!/usr/bin/env python3
"""Benchmark of the sparse-prefill evidence probe on one MI355X.

Workload: 28 independent layers (fresh seeded Q, K, V per layer), 28 query
heads / 4 kv heads, head dim 128, bf16; one video of 256 frames x 64 visual
tokens followed by 128 query tokens (16,512 tokens); block-sparse rule: sink
block + 8 preceding blocks + own block for visual rows, query rows dense over
all visual blocks; 16 planted frames.

One step = the whole probe: for each of the 28 layers one
evisel_sparse_prefill call (attention with fused evidence partials, split-row
combine, evidence reduction), then one evisel_frame_evidence call (head/layer
aggregation and top-16 frames). Inputs are resident in HBM before timing.

Prints one JSON line: probe tokens/s (value), ms per step, the attention
kernel's roofline against the bf16 MFMA peak (active-block FLOPs over the
kernel's HIP-event time, measured over the timed region, where only that
kernel is bracketed by events, on every 27th prefill call), the other
kernels' times from two further untimed steps, and the fp64 CPU oracle's
throughput on a bounded sample (whole layers, at least 10 s) as a
baseline.

``--tau-p P`` runs the same workload under the paper's adaptive top-p
retention instead of the static rule: every layer first selects each row's
history blocks on the GPU (that time is part of the step), and the
attention's active-block FLOPs are those of the key tiles actually computed
(after dropping tiles no row of a work item retained), counted per layer
from the retention bits after the timed region.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # 256 CU x 2.4 GHz x 4096 flop/clk (dense)
PEAK_HBM_GBS = 8000.0


# Sources whose change invalidates the committed counter figures: the
# attention kernel and the plan that orders its work (launch order decides
# how much of the key/value traffic each XCD's L2 absorbs).
TRAFFIC_SOURCES = ("attn.hip", "attn_pipe.hip", "attn_tiles.h", "plan.cpp",
                   "plan.h")


def traffic_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2608_05780_amd", "csrc", f),
                      "rb").read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per attention launch from the committed counter summary,
    or None when the attention kernel or the plan changed since it was
    measured."""
    summ = os.path.join(ROOT, "profiles",
                        "attn_pipe_kernel_16k28L_hbm_counters.md")
    try:
        sha = traffic_source_sha()
        for line in open(summ):
            if line.startswith("traffic_per_launch"):
                kv = dict(x.split("=") for x in line.split()[1:])
                if kv["source_sha256"] == sha:
                    return float(kv["fetch_bytes"]) + float(kv["write_bytes"])
    except (OSError, KeyError, ValueError):
        pass
    return None


def attention_kernel_name(w, args):
    """The attention kernel the library launches for this run: the
    pipelined kernel for bf16 inputs under the static rule (its frame-cue
    form with the cues, for frames of 32 or 64 keys), attn_kernel
    otherwise."""
    if w.dtype == "bf16" and w.tau_p == 0 and (not args.cues or
                                               w.tokens_per_frame >= 32):
        return f"attn_pipe_kernel<{w.d}, {'true' if args.cues else 'false'}>"
    path = "Bf16Path" if w.dtype == "bf16" else "F32Path"
    return f"attn_kernel<{path}<{w.d}>, {w.d}, {'true' if w.tau_p > 0 else 'false'}>"


def measured_sq():
    """MFMA busy, co-execution and VALU/MFMA ratio of the attention kernel
    from the committed SQ counter summary, or None when the attention kernel
    or the plan changed since it was measured."""
    summ = os.path.join(ROOT, "profiles", "attn_pipe_kernel_16k28L_sq_counters.md")
    try:
        sha = traffic_source_sha()
        for line in open(summ):
            if line.startswith("sq_per_launch"):
                kv = dict(x.split("=") for x in line.split()[1:])
                if kv.pop("source_sha256") == sha:
                    return {k: float(v) for k, v in kv.items()}
    except (OSError, KeyError, ValueError):
        pass
    return None


def allowed_token_pairs(ev, mask):
    """Token pairs (query, key) the static rule allows, per head and layer:
    a key block before the query block is visible whole, the diagonal block
    causally (len * (len + 1) / 2 pairs)."""
    import numpy as np
    ex = ev.mask_export(mask)
    ln = ex["len"].astype(np.int64)
    rows = np.repeat(np.arange(len(ln)), np.diff(ex["row_ptr"]))
    col = ex["col"].astype(np.int64)
    diag = rows == col
    return float(np.where(diag, ln[rows] * (ln[rows] + 1) // 2,
                          ln[rows] * ln[col]).sum())


def work_units(ev, mask):
    """The attention work list as (query block, first head, heads, CSR run)
    units: an ordinary item is one unit; a paired item (one head over two
    query blocks) is one unit per query block, its run read back from the
    paired-tile list."""
    import numpy as np
    wk = ev.mask_export_work(mask)
    pt = ev.mask_export_paired(mask)
    units = []
    for qb, h0, nh, a, e, q2 in zip(wk["qblock"], wk["head"], wk["nheads"],
                                    wk["kb_begin"], wk["kb_end"],
                                    wk["qblock2"]):
        if qb < 0:
            continue
        if q2 < 0:
            units.append((int(qb), int(h0), int(nh), int(a), int(e)))
            continue
        for q, pos in ((qb, pt["pos_a"][a:e]), (q2, pt["pos_b"][a:e])):
            p = pos[pos >= 0]
            units.append((int(q), int(h0), 1, int(p[0]), int(p[-1]) + 1))
    return units


def topp_computed_pairs(ev, mask, w, qs, kks, ws):
    """Key tiles the top-p attention computes per layer (mean over
    layers), summed over query heads, and the mean fraction of its history
    a row retains. Recomputes each layer's retention (same kernels). A unit
    of work computes a candidate tile when it is always visible or some row
    of the unit's heads retained it."""
    import numpy as np
    import torch
    st = mask.stats
    nb, W = st["n_blocks"], st["hist_words"]
    ex = ev.mask_export(mask)
    units = work_units(ev, mask)
    col = ex["col"]
    # local history index of every block (-1: system prefix)
    local = np.full(nb, -1, np.int64)
    for n in np.unique(ex["video"]):
        ids = np.nonzero((ex["video"] == n) & (ex["region"] != 0))[0]
        local[ids] = np.arange(ids.size)
    rb = torch.empty((w.hq, nb, W, 64), dtype=torch.int32, device="cuda")
    ub = torch.empty((w.hq, nb, W), dtype=torch.int32, device="cuda")
    total, kept, hist = 0.0, 0.0, 0.0
    for l in range(len(qs)):
        ev.select_blocks(mask, qs[l], kks[l], rb, ub, ws,
                         softmax_scale=w.softmax_scale)
        u = ub.cpu().numpy().view(np.uint32)
        for qb, h0, nh, a, e in units:
            c = col[a:e]
            loc = local[c]
            always = (loc < 0) | (c == qb)
            lc = np.maximum(loc, 0)
            word = np.bitwise_or.reduce(u[h0:h0 + nh, qb][:, lc // 32], axis=0)
            keep = always | (((word >> (lc % 32).astype(np.uint32)) & 1) > 0)
            total += float(keep.sum()) * nh
        bits = rb.cpu().numpy().view(np.uint32)
        pc = np.unpackbits(bits.view(np.uint8)).reshape(-1).sum()
        kept += float(pc)
        lens = ex["len"].astype(np.int64)
        hist += float((np.maximum(local, 0) * lens).sum() * w.hq)
    return total / len(qs), kept / max(hist, 1.0)


def cue_record(w, st, S, T, prof):
    """Frame-cue kernels per layer: their HIP-event time and the bytes the
    two kernels must move at least (the intra-frame pass reads the visual
    rows' Q, the K of their blocks and their LSE and writes the maps; the
    pair pass reads one partial and one LSE per (head, pair row))."""
    Nv, calls = w.tokens_per_frame, max(1, prof["calls"])
    s_vis = T * Nv
    esz = 2 if w.dtype == "bf16" else 4
    intra_bytes = (s_vis * (w.hq + w.hkv) * w.d * esz + w.hq * s_vis * 4 +
                   T * Nv * Nv * 4)
    pair_bytes = st["n_frame_pairs"] * w.hq * Nv * 8 + st["n_frame_pairs"] * 4
    ms = prof["cues_ms"] / calls
    return {"ms_per_layer": ms, "frame_pairs": st["n_frame_pairs"],
            "algorithmic_bytes_per_layer": intra_bytes + pair_bytes,
            "achieved_GBps": (intra_bytes + pair_bytes) / (ms * 1e-3) / 1e9}


def coarse_work(ev, mask, w):
    """Algorithmic work of one layer of coarse evidence: the block
    affinities of every row against its history (MFMA on the mean keys'
    bf16 hi and lo parts), the exact logits of its own block's causal prefix
    and the video's system prefix (MFMA), and the bytes it must move at least
    (Q read by the retention and by the coarse pass, K read by the mean-key
    pooling, the evidence row written)."""
    import numpy as np
    ex = ev.mask_export(mask)
    flop = 0.0
    parts = 2 if w.dtype == "bf16" else 1
    for n in np.unique(ex["video"]):
        ids = np.nonzero(ex["video"] == n)[0]
        sys_len = int(ex["len"][ids][ex["region"][ids] == 0].sum())
        sel = ids[ex["region"][ids] != 0]
        for i, b in enumerate(sel):
            rows = int(ex["len"][b])
            # history: the selectable blocks before b; exact part: the
            # system prefix and the causal prefix of b (rows x (rows+1)/2)
            flop += 2.0 * w.d * w.hq * (parts * rows * i + rows * sys_len +
                                        rows * (rows + 1) / 2)
    esz = 2 if w.dtype == "bf16" else 4
    S, T = mask.stats["n_tokens"], mask.stats["n_frames_total"]
    nbytes = (2 * S * w.hq * w.d * esz + S * w.hkv * w.d * esz +
              w.hq * T * 4)
    return flop, nbytes


def coarse_main(args, ev, w, mask, qs, kks, evid, e_qf, kk, topk, ws,
                stream, S, T, L, ks, core):
    """--coarse: the paper's coarse query-frame evidence of every layer
    (the retention kernels plus the coarse pass), then the frame
    aggregation and top-k; timed like the exact probe, with HIP events
    around every layer's coarse call on the caller's stream."""
    import numpy as np
    import torch

    def step(evs=None):
        for l in range(L):
            if evs is not None:
                evs[l][0].record(stream)
            ev.coarse_evidence(mask, qs[l], kks[l], evid[l], ws,
                               softmax_scale=w.softmax_scale, stream=stream)
            if evs is not None:
                evs[l][1].record(stream)
        ev.frame_evidence(mask, evid, L, e_qf, k_per_seq=kk, topk=topk,
                          stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    # per-layer times of the coarse call from one further, bracketed step
    evs = [(torch.cuda.Event(enable_timing=True),
            torch.cuda.Event(enable_timing=True)) for _ in range(L)]
    step(evs)
    torch.cuda.synchronize()
    layer_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    # the retention alone (mean keys + per-row selection) per layer, from
    # one further pass of evisel_select_blocks calls, each bracketed
    st = mask.stats
    rb = torch.empty((w.hq, st["n_blocks"], st["hist_words"], 64),
                     dtype=torch.int32, device="cuda")
    ub = torch.empty((w.hq, st["n_blocks"], st["hist_words"]),
                     dtype=torch.int32, device="cuda")
    for l in range(L):
        evs[l][0].record(stream)
        ev.select_blocks(mask, qs[l], kks[l], rb, ub, ws,
                         softmax_scale=w.softmax_scale, stream=stream)
        evs[l][1].record(stream)
    torch.cuda.synchronize()
    sel_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    flop, nbytes = coarse_work(ev, mask, w)
    found = sorted(topk[:sum(ks)].cpu().numpy().tolist())
    rec = {
        "metric": "coarse-evidence probe tokens/sec (top-p retention + "
                  "coarse query-frame evidence)",
        "value": S / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) Q/K/V, planted frames)",
        "config": {"workload": w.name, "layers": L, "tokens": S,
                   "frames": T, "tokens_per_frame": w.tokens_per_frame,
                   "hq": w.hq, "hkv": w.hkv, "head_dim": w.d,
                   "block": w.block, "tau_p": w.tau_p,
                   "parallelism": "single-gpu"},
        "coarse": {"ms_per_layer": layer_ms,
                   "retention_ms_per_layer": sel_ms,
                   "algorithmic_flop_per_layer": flop,
                   "algorithmic_bytes_per_layer": nbytes,
                   "achieved_TFLOPs": flop / (layer_ms * 1e-3) / 1e12,
                   "achieved_GBps": nbytes / (layer_ms * 1e-3) / 1e9},
        "topk_planted_recovered": found == sorted(core.tolist()),
    }
    print(json.dumps(rec), flush=True)


def _world():
    return int(os.environ.get("WORLD_SIZE", "1")), int(os.environ.get("RANK",
                                                                      "0"))


def cpu_baseline(w, seed=0, min_seconds=10.0):
    """The fp64 oracle (as it stands) on whole layers, taken in order until
    at least ``min_seconds`` have passed: all rows' output and LSE plus the
    evidence of all query rows. Scaled to probe tokens/s for the whole
    L-layer probe."""
    import numpy as np
    import oracle
    from oracle.layout import Layout, Rule
    import workloads as wl
    try:
        from threadpoolctl import threadpool_info
        threads = max(i["num_threads"] for i in threadpool_info())
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    ns, nf, nt = wl.layout_arrays(w, seed)
    lay = Layout(ns, nf, nt, w.tokens_per_frame)
    rule = Rule(w.block, w.sink_blocks, w.window)
    dt, done = 0.0, 0
    while done < w.n_layers and (done == 0 or dt < min_seconds):
        q, k, v = wl.gen_layer(w, done, seed).as_f64()
        t0 = time.perf_counter()
        oracle.run_layer(q, k, v, lay, rule, w.softmax_scale)
        dt += time.perf_counter() - t0
        done += 1
    per_layer = dt / done
    return {"value": lay.S / (per_layer * w.n_layers), "unit": "tokens/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"layers 0-{done - 1} of {w.n_layers}, all {lay.S} rows "
                      f"x {w.hq} heads + evidence ({dt:.1f} s), scaled to "
                      f"{w.n_layers} layers",
            "host_cpus": os.cpu_count()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cues", action="store_true",
                    help="also produce the cross-frame (A_ff, E_ff) and "
                         "intra-frame (A_if) cues in every step")
    ap.add_argument("--tau-p", type=float, default=0.0,
                    help="adaptive top-p retention threshold (0: the "
                         "workload's static rule)")
    ap.add_argument("--coarse", action="store_true",
                    help="with --tau-p: the paper's coarse query-frame "
                         "evidence instead of the exact sparse pass (no "
                         "attention output); one step = the coarse evidence "
                         "of every layer plus the frame aggregation")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes "
                         "(3 times), to scale HBM byte counters")
    args = ap.parse_args()
    world, rank = _world()
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the probe is not sharded "
              "across GPUs in this library (run with --gpus 1).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import workloads as wl
    import paper_2608_05780_amd as ev

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "launches": 3}))
        return
    ev.load()
    if args.coarse and (args.tau_p <= 0 or args.cues):
        print("--coarse needs --tau-p > 0 and no --cues", file=sys.stderr)
        sys.exit(2)
    w = wl.get(args.config, tau_p=args.tau_p) if args.tau_p > 0 else \
        wl.get(args.config)
    L = w.n_layers
    ns, nf, nt = wl.layout_arrays(w, args.seed)
    _, core, _ = wl.plant_table(w, args.seed)
    ks = []
    off = 0
    for F in nf:
        ks.append(int(((core >= off) & (core < off + F)).sum()))
        off += int(F)

    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv, n_sys=ns,
                               tau_p=w.tau_p)
    st = mask.stats
    S, T = st["n_tokens"], st["n_frames_total"]
    print(f"# {w.name}: S={S} T={T} active pairs/head/layer="
          f"{st['n_active_pairs']} items={st['n_work_items']}",
          file=sys.stderr, flush=True)

    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    qs, kks, vs = [], [], []
    t0 = time.time()
    for l in range(L):
        lay = wl.gen_layer(w, l, args.seed)
        cv = (lambda a: torch.from_numpy(a.view(np.int16)).view(dt).cuda()) \
            if w.dtype == "bf16" else (lambda a: torch.from_numpy(a).cuda())
        qs.append(cv(lay.q))
        kks.append(cv(lay.k))
        vs.append(cv(lay.v))
    print(f"# inputs generated and uploaded in {time.time() - t0:.1f} s",
          file=sys.stderr, flush=True)
    out = torch.empty((S, w.hq, w.d), dtype=dt, device="cuda")
    lse = torch.empty((w.hq, S), dtype=torch.float32, device="cuda")
    evid = torch.empty((L, w.hq, T), dtype=torch.float32, device="cuda")
    tmass = torch.empty((L, w.hq, len(nf)), dtype=torch.float32, device="cuda")
    e_qf = torch.empty(T, dtype=torch.float32, device="cuda")
    kk = torch.tensor(ks, dtype=torch.int32, device="cuda")
    topk = torch.empty(max(1, sum(ks)), dtype=torch.int32, device="cuda")
    ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d, cues=args.cues),
                     dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    pairs = intra = e_ff = None
    if args.cues:
        Nv = w.tokens_per_frame
        pairs = torch.empty((L, max(1, st["n_frame_pairs"])),
                            dtype=torch.float32, device="cuda")
        intra = torch.empty((L, T, Nv, Nv), dtype=torch.float32,
                            device="cuda")
        e_ff = torch.empty((L, T), dtype=torch.float32, device="cuda")

    def step():
        for l in range(L):
            ev.sparse_prefill(mask, l, L, qs[l], kks[l], vs[l], out, evid, ws,
                              lse=lse, text_mass=tmass,
                              softmax_scale=w.softmax_scale, stream=stream,
                              frame_pairs=pairs, intra_frame=intra)
        ev.frame_evidence(mask, evid, L, e_qf, k_per_seq=kk, topk=topk,
                          stream=stream, frame_pairs=pairs, e_ff=e_ff)

    if args.coarse:
        coarse_main(args, ev, w, mask, qs, kks, evid, e_qf, kk, topk, ws,
                    stream, S, T, L, ks, core)
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Timed region: HIP events around the attention kernel only, and only
    # on every `stride`-th prefill call: each event is a dependency packet
    # that idles the GPU for several microseconds, so bracketing every
    # launch would lengthen the step by about 5 %. The per-kernel breakdown
    # comes from two further, untimed steps.
    calls = args.steps * L
    stride = max(1, min(27, calls // 4))
    ev.profile_begin(-(-calls // stride), all_kernels=False, stride=stride)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof_attn = ev.profile_end()
    ms_step = (t1 - t0) * 1e3 / args.steps
    n_detail = 2
    ev.profile_begin(n_detail * L, all_kernels=True)
    for _ in range(n_detail):
        step()
    torch.cuda.synchronize()
    prof = ev.profile_end()

    found = sorted(topk[:sum(ks)].cpu().numpy().tolist())
    planted_ok = found == sorted(core.tolist())
    tile_flop = 4.0 * w.block * w.block * w.d
    if w.tau_p > 0:
        pairs, kept_frac = topp_computed_pairs(ev, mask, w, qs, kks, ws)
        flop_layer = tile_flop * pairs
    else:
        flop_layer = tile_flop * w.hq * st["n_active_pairs"]
    attn_ms = prof_attn["attention_ms"] / max(1, prof_attn["calls"])
    achieved = flop_layer / (attn_ms * 1e-3) / 1e12
    # strict count: 4 d flop per allowed (query, key) token pair and head
    strict_flop = (4.0 * w.d * w.hq * allowed_token_pairs(ev, mask)
                   if w.tau_p == 0 else None)
    # combine + evidence kernel: the query rows' per-frame partial masses
    # and the evidence row, the chunk partials (O, reference max, row sum,
    # non-visual mass), the merged O and LSE of the query rows
    ev_ms = prof["combine_ms"] / max(1, prof["calls"])
    segtot = int(np.sum(np.asarray(nt, np.int64) * np.asarray(nf, np.int64)))
    ev_bytes = (4.0 * w.hq * (segtot + T)
                + st["n_chunk_slots"] * 64.0 * (4 * w.d + 12)
                + st["n_text_rows"] * w.hq * (2.0 * w.d + 4))
    rec = {
        "metric": "probe prefill tokens/sec + active-block attention TFLOP/s "
                  "(% bf16 MFMA peak)",
        "value": S / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) Q/K/V, planted frames)",
        "config": {"workload": w.name, "layers": L, "tokens": S,
                   "frames": T, "tokens_per_frame": w.tokens_per_frame,
                   "query_tokens": int(sum(nt)), "hq": w.hq, "hkv": w.hkv,
                   "head_dim": w.d, "block": w.block,
                   "sink_blocks": w.sink_blocks, "window": w.window,
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "mfma", "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS,
                     # counters cover the static-rule kernel without cues
                     "traffic": (measured_traffic() if args.config == 3 and
                                 w.tau_p == 0 and not args.cues else None),
                     "kernel": attention_kernel_name(w, args),
                     # SQ counters of the same kernel and workload (null when
                     # stale or for another workload)
                     "sq_counters": (measured_sq() if args.config == 3 and
                                     w.tau_p == 0 and not args.cues
                                     else None),
                     "flop_per_launch": flop_layer,
                     "avg_launch_ms": attn_ms,
                     "timed_launches": prof_attn["calls"]},
        "strict_allowed_pairs": (None if strict_flop is None else {
            "flop_per_launch": strict_flop,
            "achieved_TFLOPs": strict_flop / (attn_ms * 1e-3) / 1e12,
            "frac": strict_flop / (attn_ms * 1e-3) / 1e12 /
                    PEAK_BF16_TFLOPS}),
        # kernels the step does not launch are null, not the empty span
        # between their events
        "kernels_ms_per_layer": {
            "cues": (prof["cues_ms"] / max(1, prof["calls"])
                     if args.cues else None),
            "retention": (prof["select_ms"] / max(1, prof["calls"])
                          if w.tau_p > 0 else None),
            "attention": attn_ms,
            "combine_evidence": ev_ms},
        "evidence_reduce_GBps": ev_bytes / (ev_ms * 1e-3) / 1e9,
        **({"cues": cue_record(w, st, S, T, prof)} if args.cues else {}),
        "topk_planted_recovered": planted_ok,
    }
    if w.tau_p > 0:
        rec["config"]["tau_p"] = w.tau_p
        rec["config"]["sink_blocks"] = rec["config"]["window"] = None

        rec["topp"] = {"computed_tile_pairs_per_layer": flop_layer / tile_flop,
                       "candidate_tile_pairs_per_layer":
                           float(w.hq * st["n_active_pairs"]),
                       "row_retained_fraction": kept_frac}
        args.no_cpu_baseline = True    # the oracle baseline is the static one
    if not args.no_cpu_baseline and rank == 0:
        print("# timing the CPU oracle on whole layers (>= 10 s) ...", file=sys.stderr,
              flush=True)
        rec["cpu_baseline"] = cpu_baseline(w, args.seed)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()

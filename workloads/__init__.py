"""Seeded synthetic workloads for the sparse-prefill evidence probe.

This module only draws inputs. It holds none of the probe's arithmetic: no
masking, no softmax, no evidence reduction. Both the fp64 oracle and the HIP
path take their inputs from here, and nothing else is shared between them.

A workload is a packed batch of videos. Video n contributes, in order,
``n_sys[n]`` system-prompt tokens, ``n_frames[n] * tokens_per_frame`` visual
tokens (one group of ``tokens_per_frame`` tokens per anchor frame) and
``n_text[n]`` query tokens: the prefill context X = [X_sys; X_vis; X_Q] of the
paper's appendix on sparse prefilling.

Draw protocol (fixed, so the oracle and the GPU see bit-identical inputs):

* ``SeedSequence([seed, config_id]).spawn(n_layers + 1)``: child 0 draws the
  plant table (and, for the ragged batch, the frame counts); child l+1 is
  spawned again into 3 * CHUNKS + 1 streams for layer l: the token range is
  cut into CHUNKS equal parts, and part c of Q, K and V is filled from
  streams c, CHUNKS + c and 2 * CHUNKS + c; the last stream draws u. Each
  stream is a ``Generator(PCG64)``; the parts are filled by a thread pool,
  which does not change any value.
* Q ``[S, Hq, d]``, K and V ``[S, Hkv, d]`` are i.i.d. N(0, 1) float32; u is a
  unit vector in R^d (float32).
* Optional frame structure (``key_struct = (beta, gamma, rho)``, off in the
  paper-shaped configs): per video and kv head an AR(1) sequence of frame
  content vectors c_0 = xi_0, c_f = rho c_{f-1} + sqrt(1 - rho^2) xi_f
  (xi ~ N(0, I_d), drawn from stream 3 * CHUNKS + 1, videos in order, then
  frames, kv heads, dimensions); the K rows of frame f get ``+ beta c_f``
  and the visual Q rows of frame f (every q head of the kv head) get
  ``+ gamma c_f``. It gives the keys the block-level content and the queries
  the locality that make a block-affinity selection sparse.
* Planting: every kv head's K rows of a planted frame f get ``+ s_f * u`` and
  every q head's query-token rows get ``+ s_Q * u`` (float32 arithmetic).
* bf16 workloads are then rounded to bf16 with round-to-nearest-even; the
  result is carried as the raw uint16 bit patterns.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNKS = 8

__all__ = ["Workload", "CONFIGS", "get", "layout_arrays", "plant_table",
           "gen_layer", "bf16_bits", "bf16_bits_to_f32", "Layer"]


@dataclass(frozen=True)
class Workload:
    """Shape and sparsity rule of one synthetic probe workload."""
    name: str
    config_id: int
    n_layers: int
    hq: int
    hkv: int
    d: int
    dtype: str                      # "fp32" or "bf16"
    tokens_per_frame: int           # N_v
    block: int                      # B
    sink_blocks: int
    window: int                     # preceding visual blocks; -1 = all-causal
    plant: str                      # plant recipe name
    n_frames: tuple = ()            # per video (empty: drawn, ragged batch)
    n_text: tuple = ()
    n_sys: tuple = ()
    n_videos: int = 1
    ragged_frames: tuple = ()       # (lo, hi) inclusive, ragged batch only
    plant_args: dict = field(default_factory=dict)
    tau_p: float = 0.0              # > 0: adaptive top-p retention rule
    key_struct: tuple = ()          # (beta, gamma, rho) frame structure

    @property
    def softmax_scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))


CONFIGS = {
    1: Workload(
        name="tiny-fp32-1L-32f16-32q", config_id=1, n_layers=1, hq=4, hkv=1,
        d=64, dtype="fp32", tokens_per_frame=16, block=64, sink_blocks=1,
        window=-1, plant="fixed", n_frames=(32,), n_text=(32,), n_sys=(0,),
        plant_args={"frames": (5, 20), "s_frame": 3.0, "s_query": 3.0}),
    2: Workload(
        name="qwen2vl7b-1L-128f64-64q", config_id=2, n_layers=1, hq=28,
        hkv=4, d=128, dtype="bf16", tokens_per_frame=64, block=64,
        sink_blocks=1, window=8, plant="choose", n_frames=(128,),
        n_text=(64,), n_sys=(0,),
        plant_args={"count": 6, "s_frame": (2.0, 2.0), "s_query": 2.0}),
    3: Workload(
        name="qwen2vl7b-28L-256f64-128q", config_id=3, n_layers=28, hq=28,
        hkv=4, d=128, dtype="bf16", tokens_per_frame=64, block=64,
        sink_blocks=1, window=8, plant="choose", n_frames=(256,),
        n_text=(128,), n_sys=(0,),
        plant_args={"count": 16, "s_frame": (1.0, 3.0), "s_query": 2.0}),
    4: Workload(
        name="qwen2vl7b-28L-1024f64-128q", config_id=4, n_layers=28, hq=28,
        hkv=4, d=128, dtype="bf16", tokens_per_frame=64, block=64,
        sink_blocks=1, window=16, plant="segments", n_frames=(1024,),
        n_text=(128,), n_sys=(0,),
        plant_args={"segments": 3, "fraction": 0.10, "s_frame": (1.5, 3.0),
                    "sigma": 4.0, "shoulder": 12, "s_query": 2.0}),
    5: Workload(
        name="qwen2vl7b-28L-ragged8x(64-512)f32-64q", config_id=5,
        n_layers=28, hq=28, hkv=4, d=128, dtype="bf16", tokens_per_frame=32,
        block=64, sink_blocks=1, window=8, plant="ragged", n_videos=8,
        ragged_frames=(64, 512),
        plant_args={"fraction": 0.05, "s_frame": (1.0, 3.0), "s_query": 2.0,
                    "text": 64}),
}


def get(cid: int, **overrides) -> Workload:
    """Return workload ``cid``, optionally with fields replaced."""
    w = CONFIGS[cid]
    if overrides:
        kw = dict(w.__dict__)
        kw.update(overrides)
        w = Workload(**kw)
    return w


def _streams(w: Workload, seed: int):
    ss = np.random.SeedSequence([int(seed), int(w.config_id)])
    return ss.spawn(w.n_layers + 1)


def layout_arrays(w: Workload, seed: int = 0):
    """Per-video (n_sys, n_frames, n_text) int32 arrays.

    The ragged batch draws its frame counts from the plant stream, uniformly
    over the inclusive range, before anything else is drawn from it.
    """
    if w.plant == "ragged":
        rng = np.random.Generator(np.random.PCG64(_streams(w, seed)[0]))
        lo, hi = w.ragged_frames
        nf = rng.integers(lo, hi + 1, size=w.n_videos).astype(np.int32)
        nt = np.full(w.n_videos, w.plant_args["text"], np.int32)
        ns = np.zeros(w.n_videos, np.int32)
        return ns, nf, nt
    return (np.asarray(w.n_sys, np.int32), np.asarray(w.n_frames, np.int32),
            np.asarray(w.n_text, np.int32))


def plant_table(w: Workload, seed: int = 0):
    """Planted frames and strengths.

    Returns ``(strength, core, s_query)``: ``strength`` is float32 over all
    frames of the batch (global frame ids, videos in order), ``core`` is the
    sorted array of "planted" global frame ids (the frames a correct probe
    must rank first), ``s_query`` the query-row strength.
    """
    ns, nf, nt = layout_arrays(w, seed)
    total = int(nf.sum())
    strength = np.zeros(total, np.float32)
    a = w.plant_args
    rng = np.random.Generator(np.random.PCG64(_streams(w, seed)[0]))
    if w.plant == "ragged":
        rng.integers(w.ragged_frames[0], w.ragged_frames[1] + 1,
                     size=w.n_videos)               # replay the count draw
    core = []
    if w.plant == "fixed":
        for f in a["frames"]:
            strength[f] = a["s_frame"]
            core.append(f)
    elif w.plant == "choose":
        picks = np.sort(rng.choice(total, size=a["count"], replace=False))
        lo, hi = a["s_frame"]
        s = rng.uniform(lo, hi, size=a["count"]).astype(np.float32)
        strength[picks] = s
        core = list(picks)
    elif w.plant == "segments":
        # Three contiguous core segments covering ``fraction`` of the
        # frames, each with i.i.d. core strengths and Gaussian shoulders of
        # width sigma outside the core.
        T = total
        nseg = a["segments"]
        per = int(round(a["fraction"] * T)) // nseg
        sig, sh = a["sigma"], a["shoulder"]
        margin = int(np.ceil(3 * sig))
        gap = 2 * sh + 1
        while True:
            starts = np.sort(rng.integers(margin, T - margin - per + 1,
                                          size=nseg))
            ok = all(starts[i + 1] - (starts[i] + per) >= gap
                     for i in range(nseg - 1))
            if ok:
                break
        lo, hi = a["s_frame"]
        for st in starts:
            s = rng.uniform(lo, hi, size=per).astype(np.float32)
            strength[st:st + per] = s
            core.extend(range(st, st + per))
            for dlt in range(1, sh + 1):
                fall = np.float32(np.exp(-dlt * dlt / (2.0 * sig * sig)))
                if st - dlt >= 0:
                    strength[st - dlt] = max(strength[st - dlt], s[0] * fall)
                if st + per - 1 + dlt < T:
                    strength[st + per - 1 + dlt] = max(
                        strength[st + per - 1 + dlt], s[-1] * fall)
    elif w.plant == "ragged":
        off = 0
        lo, hi = a["s_frame"]
        for n in range(w.n_videos):
            F = int(nf[n])
            k = max(1, int(round(a["fraction"] * F)))
            picks = np.sort(rng.choice(F, size=k, replace=False)) + off
            strength[picks] = rng.uniform(lo, hi, size=k).astype(np.float32)
            core.extend(picks)
            off += F
    else:
        raise ValueError(w.plant)
    return strength, np.asarray(sorted(core), np.int64), np.float32(a["s_query"])


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even.

    Uses torch's (multithreaded, round-to-nearest-even) conversion when
    available; ``bf16_bits_numpy`` is the same rounding written out."""
    try:
        import torch
    except ImportError:
        return bf16_bits_numpy(x)
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_numpy(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns by integer round-to-nearest-even."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32)
    r = ((u + np.uint32(0x7FFF) + ((u >> 16) & np.uint32(1))) >> 16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exactly equal float32 values."""
    return (np.ascontiguousarray(b, np.uint16).astype(np.uint32) << 16).view(
        np.float32)


@dataclass
class Layer:
    """One layer's inputs: float32 arrays or bf16 bit patterns (uint16)."""
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    u: np.ndarray

    def as_f64(self):
        """(q, k, v) widened exactly to float64."""
        if self.q.dtype == np.uint16:
            cv = lambda a: bf16_bits_to_f32(a).astype(np.float64)
        else:
            cv = lambda a: a.astype(np.float64)
        return cv(self.q), cv(self.k), cv(self.v)


def token_ranges(w: Workload, seed: int = 0):
    """Per-video token offsets: (tok0, vis0, txt0, end) int64 arrays."""
    ns, nf, nt = layout_arrays(w, seed)
    lens = ns.astype(np.int64) + nf.astype(np.int64) * w.tokens_per_frame + nt
    tok0 = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    vis0 = tok0 + ns
    txt0 = vis0 + nf.astype(np.int64) * w.tokens_per_frame
    return tok0, vis0, txt0, tok0 + lens


def gen_layer(w: Workload, layer: int, seed: int = 0,
              q_override: Optional[str] = None) -> Layer:
    """Draw layer ``layer``'s Q, K, V (planted, then rounded if bf16).

    ``q_override="zero"`` replaces Q by zeros after drawing (used by the
    closed-form tests; the draw order is unchanged).
    """
    ns, nf, nt = layout_arrays(w, seed)
    tok0, vis0, txt0, end = token_ranges(w, seed)
    S = int(end[-1])
    kids = _streams(w, seed)[layer + 1].spawn(3 * CHUNKS + 2)
    q = np.empty((S, w.hq, w.d), np.float32)
    k = np.empty((S, w.hkv, w.d), np.float32)
    v = np.empty((S, w.hkv, w.d), np.float32)
    cuts = [S * c // CHUNKS for c in range(CHUNKS + 1)]

    def fill(job):
        arr, c, kid = job
        a, b = cuts[c], cuts[c + 1]
        if b > a:
            np.random.Generator(np.random.PCG64(kid)).standard_normal(
                dtype=np.float32, out=arr[a:b])

    jobs = [(arr, c, kids[t * CHUNKS + c])
            for t, arr in enumerate((q, k, v)) for c in range(CHUNKS)]
    with ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(fill, jobs))
    rng = np.random.Generator(np.random.PCG64(kids[3 * CHUNKS]))
    u = rng.standard_normal(w.d, dtype=np.float32).astype(np.float64)
    u = (u / np.linalg.norm(u)).astype(np.float32)
    Nv = w.tokens_per_frame
    if w.key_struct:
        beta, gamma, rho = (float(x) for x in w.key_struct)
        srng = np.random.Generator(np.random.PCG64(kids[3 * CHUNKS + 1]))
        grp = w.hq // w.hkv
        for n in range(len(nf)):
            F = int(nf[n])
            xi = srng.standard_normal((F, w.hkv, w.d), dtype=np.float32)
            c = np.empty_like(xi)
            c[0] = xi[0]
            a_r = np.float32(rho)
            b_r = np.float32(np.sqrt(1.0 - rho * rho))
            for f in range(1, F):
                c[f] = a_r * c[f - 1] + b_r * xi[f]
            toks = c.repeat(Nv, axis=0)                  # [F * Nv, hkv, d]
            a, e = int(vis0[n]), int(vis0[n]) + F * Nv
            k[a:e] += np.float32(beta) * toks
            q[a:e] += np.float32(gamma) * np.repeat(toks, grp, axis=1)
    strength, _, s_q = plant_table(w, seed)
    foff = 0
    for n in range(len(nf)):
        F = int(nf[n])
        s = strength[foff:foff + F]
        for f in np.nonzero(s)[0]:
            a = int(vis0[n]) + int(f) * Nv
            k[a:a + Nv] += np.float32(s[f]) * u
        q[int(txt0[n]):int(end[n])] += s_q * u
        foff += F
    if q_override == "zero":
        q[:] = 0.0
    if w.dtype == "bf16":
        return Layer(bf16_bits(q), bf16_bits(k), bf16_bits(v), u)
    return Layer(q, k, v, u)

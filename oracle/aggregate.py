"""Head/layer aggregation and per-video top-k (oracle; test only).

Evidence Decomposition: attention is averaged over heads with the layer
dimension kept, and the query-frame cue averages the query-token group's
attention per anchor frame; E_qf is that cue per timestamp (one anchor frame
per timestamp). Here:

* E_qf[l, t] = sum_h E[l, h, t] / (Hq * N_q(video(t))), the mean over heads
  and over the video's query rows of the per-frame softmax mass;
* the layer-pooled score is the mean over layers of E_qf[l, t];
* top-k per video orders frames by (score descending, frame index ascending).
"""
from __future__ import annotations

import numpy as np


def frame_evidence(E_all: np.ndarray, n_frames, n_text):
    """E_all [L, Hq, T] -> (E_qf [L, T], pooled [T])."""
    E_all = np.asarray(E_all, np.float64)
    L, hq, T = E_all.shape
    nq = np.repeat(np.asarray(n_text, np.float64), np.asarray(n_frames))
    e_qf = E_all.sum(axis=1) / (hq * nq[None, :])
    return e_qf, e_qf.mean(axis=0)


def topk_per_video(score: np.ndarray, n_frames, k_per_video):
    """Per video, the k local frame indices with the largest score, ties
    broken by the smaller index. Returns a list of int arrays."""
    out = []
    off = 0
    for F, k in zip(np.asarray(n_frames), np.asarray(k_per_video)):
        s = np.asarray(score[off:off + int(F)])
        order = sorted(range(int(F)), key=lambda t: (-s[t], t))
        out.append(np.asarray(order[:int(k)], np.int64))
        off += int(F)
    return out


def boundary_gap(score: np.ndarray, n_frames, k_per_video):
    """Per video, score[rank k-1] - score[rank k] (inf when k == F)."""
    gaps = []
    off = 0
    for F, k in zip(np.asarray(n_frames), np.asarray(k_per_video)):
        s = np.sort(np.asarray(score[off:off + int(F)]))[::-1]
        gaps.append(np.inf if int(k) >= int(F) else s[int(k) - 1] - s[int(k)])
        off += int(F)
    return np.asarray(gaps)

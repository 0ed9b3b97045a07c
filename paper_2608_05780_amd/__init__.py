"""MI355X (gfx950) sparse-prefill evidence probe -- Python binding.

Argument marshalling over ``libevisel.so`` (C ABI in ``include/evisel.h``);
every step of the probe runs in the library's HIP kernels. PyTorch supplies
device memory and streams only. Importing this package does not load the
library; the first call does, and raises if it has not been built.

Entry points (same names as the C ABI):
    build_block_mask       layout + rule + head counts -> Mask (plan on device)
    select_blocks          top-p masks: per-row retained history blocks
    sparse_prefill         one layer: attention output, LSE, evidence slice
    frame_evidence         head/layer aggregation and per-video top-k frames
    sparse_prefill_workspace, mask_info, mask_export, mask_export_work,
    mask_export_paired     plan inspection (host tables)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

__all__ = ["load", "EviselError", "Mask", "build_block_mask",
           "sparse_prefill_workspace", "sparse_prefill", "frame_evidence",
           "select_blocks", "unpack_row_bits", "mask_export_pairs",
           "coarse_evidence",
           "mask_info", "mask_export", "mask_export_work",
           "mask_export_paired", "mask_permute_work", "profile_begin",
           "sparse_prefill_noalloc", "NOALLOC_WORKSPACE_BYTES",
           "profile_end", "LIB_PATH"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)),
                        "libevisel.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_NOMEM = range(6)
BF16, FP32 = 0, 1

_i32p = ctypes.POINTER(ctypes.c_int32)


class _Layout(ctypes.Structure):
    _fields_ = [("n_seq", ctypes.c_int32), ("n_sys", _i32p),
                ("n_frames", _i32p), ("n_text", _i32p),
                ("tokens_per_frame", ctypes.c_int32)]


class _Rule(ctypes.Structure):
    _fields_ = [("block", ctypes.c_int32), ("sink_blocks", ctypes.c_int32),
                ("window", ctypes.c_int32), ("tau_p", ctypes.c_float)]


class _Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "n_tokens", "n_frames_total", "n_text_rows", "n_blocks",
        "n_active_pairs", "n_work_items", "n_text_tiles", "n_chunk_slots")] + \
        [(n, ctypes.c_int32) for n in ("hq", "hkv", "block",
                                       "tokens_per_frame", "hist_words")] + \
        [("tau_p", ctypes.c_float), ("n_frame_pairs", ctypes.c_int64),
         ("n_paired_tiles", ctypes.c_int64)]


_lib = None

_SIGS = {
    "evisel_build_block_mask": (ctypes.c_int, [ctypes.POINTER(_Layout),
                                               ctypes.POINTER(_Rule),
                                               ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_void_p,
                                               ctypes.POINTER(ctypes.c_void_p)]),
    "evisel_build_block_mask_host": (ctypes.c_int, [
        ctypes.POINTER(_Layout), ctypes.POINTER(_Rule), ctypes.c_int32,
        ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p)]),
    "evisel_mask_free": (None, [ctypes.c_void_p]),
    "evisel_mask_permute_work": (ctypes.c_int, [ctypes.c_void_p, _i32p,
                                                ctypes.c_void_p]),
    "evisel_mask_info": (ctypes.c_int, [ctypes.c_void_p,
                                        ctypes.POINTER(_Stats)]),
    "evisel_mask_export": (ctypes.c_int, [ctypes.c_void_p] + [_i32p] * 6),
    "evisel_mask_export_work": (ctypes.c_int, [ctypes.c_void_p] + [_i32p] * 8),
    "evisel_mask_export_paired": (ctypes.c_int, [ctypes.c_void_p] + [_i32p] * 3),
    "evisel_sparse_prefill_workspace": (ctypes.c_size_t, [ctypes.c_void_p,
                                                          ctypes.c_int32]),
    "evisel_sparse_prefill": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_size_t, ctypes.c_void_p]),
    "evisel_sparse_prefill_noalloc": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int,
        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "evisel_cue_workspace": (ctypes.c_size_t, [ctypes.c_void_p,
                                               ctypes.c_int32]),
    "evisel_mask_export_pairs": (ctypes.c_int, [ctypes.c_void_p, _i32p,
                                                _i32p]),
    "evisel_select_blocks": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "evisel_coarse_evidence": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
        ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_size_t, ctypes.c_void_p]),
    "evisel_frame_evidence": (ctypes.c_int, [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p]),
    "evisel_profile_begin": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32]),
    "evisel_profile_end": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double),
                                          ctypes.POINTER(ctypes.c_int64)]),
    "evisel_last_error": (ctypes.c_char_p, []),
}

EXPORTED = tuple(_SIGS)


class EviselError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"evisel status {status}: {msg}")
        self.status = status


def load(path: Optional[str] = None):
    """Load libevisel.so (in-tree build). Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(
            f"{p} is not built; run `python -m paper_2608_05780_amd.build`")
    lib = ctypes.CDLL(p)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != OK:
        raise EviselError(status, _lib.evisel_last_error().decode())


def _arr(vals):
    a = (ctypes.c_int32 * len(vals))(*[int(x) for x in vals])
    return a


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


class Mask:
    """Owns an ``evisel_mask``; freed when garbage-collected."""

    def __init__(self, handle: ctypes.c_void_p, n_frames, n_text, n_sys):
        self._h = handle
        self.n_frames = list(n_frames)
        self.n_text = list(n_text)
        self.n_sys = list(n_sys)
        self.stats = mask_info(self)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.evisel_mask_free(self._h)
            self._h = None


def build_block_mask(n_frames: Sequence[int], n_text: Sequence[int],
                     tokens_per_frame: int, block: int, sink_blocks: int,
                     window: int, hq: int, hkv: int,
                     n_sys: Optional[Sequence[int]] = None, stream=None,
                     host_only: bool = False, tau_p: float = 0.0) -> Mask:
    """``tau_p`` > 0 selects the adaptive top-p retention rule (sink_blocks
    and window are then ignored)."""
    lib = load()
    ns = list(n_sys) if n_sys is not None else [0] * len(n_frames)
    a_f, a_t, a_s = _arr(n_frames), _arr(n_text), _arr(ns)
    lay = _Layout(len(n_frames), ctypes.cast(a_s, _i32p),
                  ctypes.cast(a_f, _i32p), ctypes.cast(a_t, _i32p),
                  tokens_per_frame)
    rule = _Rule(block, sink_blocks, window, float(tau_p))
    h = ctypes.c_void_p()
    if host_only:
        _check(lib.evisel_build_block_mask_host(ctypes.byref(lay),
                                                ctypes.byref(rule), hq, hkv,
                                                ctypes.byref(h)))
    else:
        _check(lib.evisel_build_block_mask(ctypes.byref(lay),
                                           ctypes.byref(rule), hq, hkv,
                                           _stream(stream), ctypes.byref(h)))
    return Mask(h, n_frames, n_text, ns)


def mask_info(mask: Mask) -> dict:
    st = _Stats()
    _check(load().evisel_mask_info(mask.handle, ctypes.byref(st)))
    return {n: getattr(st, n) for n, _ in _Stats._fields_}


def mask_export(mask: Mask) -> dict:
    import numpy as np
    nb, nnz = mask.stats["n_blocks"], mask.stats["n_active_pairs"]
    out = {k: np.zeros(nb, np.int32) for k in ("start", "len", "region",
                                               "video")}
    out["row_ptr"] = np.zeros(nb + 1, np.int32)
    out["col"] = np.zeros(max(nnz, 1), np.int32)
    p = lambda a: a.ctypes.data_as(_i32p)
    _check(load().evisel_mask_export(mask.handle, p(out["start"]),
                                     p(out["len"]), p(out["region"]),
                                     p(out["video"]), p(out["row_ptr"]),
                                     p(out["col"])))
    out["col"] = out["col"][:nnz]
    return out


def mask_export_work(mask: Mask) -> dict:
    import numpy as np
    n = mask.stats["n_work_items"]
    keys = ("qblock", "head", "nheads", "kb_begin", "kb_end", "slot",
            "qblock2", "slot2")
    out = {k: np.zeros(max(n, 1), np.int32) for k in keys}
    p = lambda a: a.ctypes.data_as(_i32p)
    _check(load().evisel_mask_export_work(mask.handle,
                                          *[p(out[k]) for k in keys]))
    return {k: v[:n] for k, v in out.items()}


def mask_permute_work(mask: Mask, perm, stream=None):
    """New launch order of the attention work list: item i is the current
    item perm[i] (a permutation of range(n_work_items))."""
    import numpy as np
    p = np.ascontiguousarray(np.asarray(perm, np.int32))
    if p.size != mask.stats["n_work_items"]:
        raise ValueError("perm needs one entry per work item")
    _check(load().evisel_mask_permute_work(mask.handle, p.ctypes.data_as(_i32p),
                                           _stream(stream)))


def mask_export_paired(mask: Mask) -> dict:
    """Key tiles of paired work items: key block and its CSR position in
    the first / second query block's row (-1: not active there)."""
    import numpy as np
    n = mask.stats["n_paired_tiles"]
    keys = ("block", "pos_a", "pos_b")
    out = {k: np.zeros(max(n, 1), np.int32) for k in keys}
    p = lambda a: a.ctypes.data_as(_i32p)
    _check(load().evisel_mask_export_paired(mask.handle,
                                            *[p(out[k]) for k in keys]))
    return {k: v[:n] for k, v in out.items()}


def sparse_prefill_workspace(mask: Mask, d: int, cues: bool = False) -> int:
    """Workspace bytes of a prefill call (``cues``: with frame-cue
    outputs)."""
    n = int(load().evisel_sparse_prefill_workspace(mask.handle, d))
    if cues:
        n += int(load().evisel_cue_workspace(mask.handle, d))
    return n


def mask_export_pairs(mask: Mask) -> dict:
    """Frame pairs (a, b) of the cross-frame cue, in output order."""
    import numpy as np
    n = mask.stats["n_frame_pairs"]
    a = np.zeros(max(n, 1), np.int32)
    b = np.zeros(max(n, 1), np.int32)
    p = lambda x: x.ctypes.data_as(_i32p)
    _check(load().evisel_mask_export_pairs(mask.handle, p(a), p(b)))
    return {"a": a[:n], "b": b[:n]}


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return FP32
    raise TypeError(f"unsupported dtype {t.dtype}")


def sparse_prefill(mask: Mask, layer: int, n_layers: int, q, k, v, out,
                   evidence, workspace, lse=None, text_mass=None,
                   softmax_scale: Optional[float] = None, stream=None,
                   frame_pairs=None, intra_frame=None):
    """One probe layer. Tensors are contiguous torch tensors on the GPU:
    q/out [S, Hq, d], k/v [S, Hkv, d] (bf16 or fp32), evidence
    [n_layers, Hq, T] fp32, lse [Hq, S] fp32, text_mass [n_layers, Hq, n_seq]
    fp32, frame_pairs [n_layers, n_frame_pairs] fp32, intra_frame
    [n_layers, T, N_v, N_v] fp32, workspace a uint8 tensor of
    sparse_prefill_workspace(mask, d, cues) bytes."""
    d = int(q.shape[-1])
    scale = float(softmax_scale) if softmax_scale is not None else d ** -0.5
    _check(load().evisel_sparse_prefill(
        mask.handle, layer, n_layers, _ptr(q), _ptr(k), _ptr(v), d,
        _dtype_code(q), scale, _ptr(out), _ptr(lse), _ptr(evidence),
        _ptr(text_mass), _ptr(frame_pairs), _ptr(intra_frame), _ptr(workspace),
        0 if workspace is None else workspace.numel() * workspace.element_size(),
        _stream(stream)))


# bytes of the library's static workspace per GPU (EVISEL_NOALLOC_WORKSPACE_BYTES)
NOALLOC_WORKSPACE_BYTES = 64 << 20


def sparse_prefill_noalloc(mask: Mask, layer: int, n_layers: int, q, k, v,
                           out, evidence, lse=None, text_mass=None,
                           softmax_scale: Optional[float] = None, stream=None,
                           frame_pairs=None, intra_frame=None):
    """sparse_prefill with the library's static per-GPU workspace instead of
    a caller's (allocates nothing; calls that overlap on one GPU race)."""
    d = int(q.shape[-1])
    scale = float(softmax_scale) if softmax_scale is not None else d ** -0.5
    _check(load().evisel_sparse_prefill_noalloc(
        mask.handle, layer, n_layers, _ptr(q), _ptr(k), _ptr(v), d,
        _dtype_code(q), scale, _ptr(out), _ptr(lse), _ptr(evidence),
        _ptr(text_mass), _ptr(frame_pairs), _ptr(intra_frame),
        _stream(stream)))


def select_blocks(mask: Mask, q, k, row_bits, block_bits, workspace,
                  softmax_scale: Optional[float] = None, stream=None):
    """Top-p retention of one layer. ``row_bits`` is a device int32 tensor
    [Hq, n_blocks, W, 64], ``block_bits`` [Hq, n_blocks, W] (W =
    ``mask.stats["hist_words"]``); bit j % 32 of word j // 32 marks local
    history block j."""
    d = int(q.shape[-1])
    scale = float(softmax_scale) if softmax_scale is not None else d ** -0.5
    _check(load().evisel_select_blocks(
        mask.handle, _ptr(q), _ptr(k), d, _dtype_code(q), scale,
        _ptr(row_bits), _ptr(block_bits), _ptr(workspace),
        0 if workspace is None else workspace.numel() * workspace.element_size(),
        _stream(stream)))


def coarse_evidence(mask: Mask, q, k, evidence, workspace,
                    softmax_scale: Optional[float] = None, stream=None):
    """The paper's coarse query-frame evidence of one layer (top-p masks):
    ``evidence`` is a device fp32 tensor [Hq, T]."""
    d = int(q.shape[-1])
    scale = float(softmax_scale) if softmax_scale is not None else d ** -0.5
    _check(load().evisel_coarse_evidence(
        mask.handle, _ptr(q), _ptr(k), d, _dtype_code(q), scale,
        _ptr(evidence), _ptr(workspace),
        0 if workspace is None else workspace.numel() * workspace.element_size(),
        _stream(stream)))


def unpack_row_bits(bits, n_hist: int):
    """[..., W, 64] int32 words (numpy) -> bool [..., 64, n_hist]."""
    import numpy as np
    w = np.ascontiguousarray(bits).view(np.uint32)
    j = np.arange(n_hist)
    words = np.take(w, j // 32, axis=-2)              # [..., n_hist, 64]
    return ((words >> (j % 32).astype(np.uint32)[:, None]) & 1).astype(
        bool).swapaxes(-1, -2)


def frame_evidence(mask: Mask, evidence, n_layers: int, e_qf,
                   e_qf_layer=None, k_per_seq=None, topk=None, stream=None,
                   frame_pairs=None, e_ff=None):
    """Head/layer aggregation and top-k. ``k_per_seq`` is a device int32
    tensor [n_seq]; ``topk`` a device int32 tensor [sum k]; ``e_ff``
    [n_layers, T] needs the prefill's ``frame_pairs``."""
    _check(load().evisel_frame_evidence(
        mask.handle, _ptr(evidence), n_layers, _ptr(e_qf_layer), _ptr(e_qf),
        _ptr(k_per_seq), _ptr(topk), _ptr(frame_pairs), _ptr(e_ff),
        _stream(stream)))


def profile_begin(capacity: int, all_kernels: bool = True, stride: int = 1):
    """Start timing the kernels of up to ``capacity`` of the following
    prefill calls: calls 0, stride, 2*stride, ... of the session
    (``all_kernels`` False: the attention kernel only, so that the others
    run back to back)."""
    _check(load().evisel_profile_begin(int(capacity), int(bool(all_kernels)),
                                       int(stride)))


def profile_end() -> dict:
    """Finish the timing session: summed ms per kernel and the call count."""
    ms = (ctypes.c_double * 4)()
    n = ctypes.c_int64()
    _check(load().evisel_profile_end(ms, ctypes.byref(n)))
    return {"select_ms": ms[0], "attention_ms": ms[1], "combine_ms": ms[2],
            "cues_ms": ms[3], "calls": n.value}

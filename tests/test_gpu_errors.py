"""Error paths of the compute calls on a real device mask: every rejected
call returns its documented status code and launches nothing (the outputs,
filled with a sentinel beforehand, are unchanged after the stream syncs).
No kernel is reached: these are the argument checks in front of the
launches."""
import ctypes

import numpy as np
import pytest

import workloads as wl
from gpu_harness import say

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    pytest.ev = gpu_lib


def _setup(d=128):
    import torch
    ev = pytest.ev
    w = wl.get(2, name="errors", config_id=301, hq=4, hkv=1, n_frames=(12,),
               n_text=(40,), tokens_per_frame=64, window=2,
               plant_args={"count": 1, "s_frame": (2.0, 2.0), "s_query": 2.0})
    ns, nf, nt = wl.layout_arrays(w)
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv, n_sys=ns)
    st = mask.stats
    S, T = st["n_tokens"], st["n_frames_total"]
    bf = torch.bfloat16

    def buf(*shape, dtype=bf):
        return torch.randn(*shape, device="cuda").to(dtype)

    t = {
        "q": buf(S, w.hq, d), "k": buf(S, w.hkv, d), "v": buf(S, w.hkv, d),
        "out": torch.full((S, w.hq, d), 7.0, dtype=bf, device="cuda"),
        "lse": torch.full((w.hq, S), 7.0, device="cuda"),
        "evid": torch.full((1, w.hq, T), 7.0, device="cuda"),
        "tm": torch.full((1, w.hq, 1), 7.0, device="cuda"),
    }
    n_ws = ev.sparse_prefill_workspace(mask, 128)
    t["ws"] = torch.empty(n_ws + 512, dtype=torch.uint8, device="cuda")
    return ev, w, mask, t, n_ws


def _call(ev, mask, t, d, ws_ptr, ws_bytes, q=None, out=None, layer=0,
          frame_pairs=None):
    """The C entry point itself, with raw pointers."""
    import torch
    lib = ev.load()
    q = t["q"].data_ptr() if q is None else q
    out = t["out"].data_ptr() if out is None else out
    stream = torch.cuda.current_stream().cuda_stream
    return lib.evisel_sparse_prefill(
        mask.handle, layer, 1, ctypes.c_void_p(q),
        ctypes.c_void_p(t["k"].data_ptr()), ctypes.c_void_p(t["v"].data_ptr()),
        d, ev.BF16, 1.0 / np.sqrt(d), ctypes.c_void_p(out),
        ctypes.c_void_p(t["lse"].data_ptr()),
        ctypes.c_void_p(t["evid"].data_ptr()),
        ctypes.c_void_p(t["tm"].data_ptr()),
        ctypes.c_void_p(frame_pairs), None, ctypes.c_void_p(ws_ptr), ws_bytes,
        ctypes.c_void_p(stream))


def _untouched(t):
    import torch
    torch.cuda.synchronize()
    for name in ("out", "lse", "evid", "tm"):
        assert bool((t[name].float() == 7.0).all()), name


def test_rejected_calls_launch_nothing():
    import torch
    ev, w, mask, t, n_ws = _setup()
    ws = t["ws"].data_ptr()
    assert ws % 256 == 0
    lib = ev.load()
    cases = []
    # head dim 96: unsupported (the tensors really have d = 96)
    _, _, mask96, t96, _ = _setup(d=96)
    cases.append(("d = 96", lambda: _call(ev, mask96, t96, 96,
                                         t96["ws"].data_ptr(), n_ws),
                  ev.ERR_UNSUPPORTED, t96))
    # one byte short of the workspace the mask needs
    cases.append(("workspace - 1", lambda: _call(ev, mask, t, 128, ws,
                                                n_ws - 1),
                  ev.ERR_WORKSPACE, t))
    # workspace not 256-byte aligned
    cases.append(("workspace misaligned", lambda: _call(ev, mask, t, 128,
                                                       ws + 16, n_ws),
                  ev.ERR_WORKSPACE, t))
    # q two bytes past a 16-byte boundary
    cases.append(("q misaligned", lambda: _call(ev, mask, t, 128, ws, n_ws,
                                               q=t["q"].data_ptr() + 2),
                  ev.ERR_INVALID_ARG, t))
    cases.append(("out misaligned", lambda: _call(ev, mask, t, 128, ws, n_ws,
                                                 out=t["out"].data_ptr() + 8),
                  ev.ERR_INVALID_ARG, t))
    # layer outside [0, n_layers)
    cases.append(("layer 1 of 1", lambda: _call(ev, mask, t, 128, ws, n_ws,
                                               layer=1),
                  ev.ERR_INVALID_ARG, t))
    # frame cues requested without their extra workspace
    fp = torch.full((4,), 7.0, device="cuda")
    cases.append(("cues without cue workspace",
                  lambda: _call(ev, mask, t, 128, ws, n_ws,
                                frame_pairs=fp.data_ptr()),
                  ev.ERR_WORKSPACE, t))
    for name, fn, want, tt in cases:
        say(f"case {name}")
        st = fn()
        msg = lib.evisel_last_error().decode()
        say(f"  status {st}: {msg}")
        assert st == want, (name, st, msg)
        assert msg
        _untouched(tt)
    torch.cuda.synchronize()
    assert bool((fp == 7.0).all())
    # the same mask and buffers still work afterwards
    st = _call(ev, mask, t, 128, ws, n_ws)
    assert st == ev.OK, lib.evisel_last_error().decode()
    torch.cuda.synchronize()
    assert bool(torch.isfinite(t["out"].float()).all())


def test_host_only_mask_is_rejected():
    import torch
    ev, w, _, t, n_ws = _setup()
    ns, nf, nt = wl.layout_arrays(w)
    host = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, host_only=True)
    st = _call(ev, host, t, 128, t["ws"].data_ptr(), n_ws)
    assert st == ev.ERR_INVALID_ARG
    _untouched(t)

"""The no-allocation prefill entry point (evisel_sparse_prefill_noalloc)
against the ordinary one (evisel_sparse_prefill with a caller workspace),
both through the C ABI: same mask, same inputs, and the outputs (O, LSE,
evidence, non-visual mass) bitwise equal. Two calls in a row, the second on
a smaller workload, so that the second starts with the first call's data
in the shared device workspace. A mask needing more workspace than the
static array holds is refused with WORKSPACE and nothing written."""
import numpy as np
import pytest

import workloads as wl
from gpu_harness import say, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    pytest.ev = gpu_lib


def _small():
    # 5 system tokens, 7 frames of 16 tokens, 37 query tokens: ragged blocks
    return wl.get(2, name="ragged-sys-noalloc", config_id=402, hq=4, hkv=1,
                  n_frames=(7,), n_text=(37,), n_sys=(5,),
                  tokens_per_frame=16, window=1,
                  plant_args={"count": 2, "s_frame": (2.0, 2.0),
                              "s_query": 2.0})


def _both(w, seed=0):
    """Outputs of layer 0 of ``w`` from the ordinary call, then from the
    no-allocation call."""
    import torch
    ev = pytest.ev
    ns, nf, nt = wl.layout_arrays(w, seed)
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, tau_p=w.tau_p)
    st = mask.stats
    S, T, nseq = st["n_tokens"], st["n_frames_total"], len(nf)
    q, k, v = to_device(wl.gen_layer(w, 0, seed), w, torch)
    res = []
    for mode in ("workspace", "noalloc"):
        out = torch.full((S, w.hq, w.d), float("nan"), dtype=q.dtype,
                         device="cuda")
        lse = torch.full((w.hq, S), float("nan"), device="cuda")
        evid = torch.full((1, w.hq, T), float("nan"), device="cuda")
        tm = torch.full((1, w.hq, nseq), float("nan"), device="cuda")
        say(f"  {mode}: {w.name} S={S} hq={w.hq} d={w.d} tau={w.tau_p}")
        if mode == "workspace":
            ws = torch.empty(ev.sparse_prefill_workspace(mask, w.d),
                             dtype=torch.uint8, device="cuda")
            ev.sparse_prefill(mask, 0, 1, q, k, v, out, evid, ws, lse=lse,
                              text_mass=tm, softmax_scale=w.softmax_scale)
        else:
            ev.sparse_prefill_noalloc(mask, 0, 1, q, k, v, out, evid,
                                      lse=lse, text_mass=tm,
                                      softmax_scale=w.softmax_scale)
        torch.cuda.synchronize()
        res.append([x.float().cpu().numpy() for x in (out, lse, evid, tm)])
    return res


def _assert_same(a, b):
    for name, x, y in zip(("O", "LSE", "evidence", "text_mass"), a, b):
        assert np.isfinite(x).all(), name
        assert np.array_equal(x, y), (name, float(np.abs(x - y).max()))


def test_noalloc_matches_workspace_call_twice():
    big = wl.get(2)        # one layer of the 8k-token probe, 28 heads
    small = _small()
    assert big.d == 128
    say("call 1: the one-layer probe workload")
    a, b = _both(big)
    _assert_same(a, b)
    say("call 2: a smaller ragged workload, after call 1")
    a, b = _both(small)
    _assert_same(a, b)


def test_noalloc_top_p_matches():
    w = wl.get(2, name="topp-noalloc", config_id=403, tau_p=0.97)
    a, b = _both(w)
    _assert_same(a, b)


def test_noalloc_refuses_oversize_mask():
    import torch
    ev = pytest.ev
    w = wl.get(5)          # 8 ragged videos, 78912 tokens, top-p retention
    ns, nf, nt = wl.layout_arrays(w)
    mask = ev.build_block_mask(nf, nt, w.tokens_per_frame, w.block,
                               w.sink_blocks, w.window, w.hq, w.hkv,
                               n_sys=ns, tau_p=0.97)
    need = ev.sparse_prefill_workspace(mask, w.d)
    assert need > ev.NOALLOC_WORKSPACE_BYTES
    # the call is refused before any buffer is read: small stand-ins
    q = torch.zeros((64, w.hq, w.d), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((64, w.hkv, w.d), dtype=torch.bfloat16, device="cuda")
    out = torch.full_like(q, 7.0)
    evid = torch.full((1, w.hq, 8), 7.0, device="cuda")
    with pytest.raises(ev.EviselError) as ei:
        ev.sparse_prefill_noalloc(mask, 0, 1, q, kv, kv, out, evid)
    say(f"  refused: {ei.value}")
    assert ei.value.status == ev.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out.float() == 7.0).all()) and bool((evid == 7.0).all())

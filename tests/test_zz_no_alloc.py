"""The no-allocation entry point vkv_step_run_static against vkv_step_run.

Both run the same kernels; the static entry point uses the library's own
per-device workspace.  Two calls in a row (the second on a smaller input, so
stale contents of the shared array from the first call would show), each
compared with vkv_step_run on a caller workspace: selected and admitted sets,
theta, outputs and lse identical.  Also: a step whose workspace exceeds the
static array is refused before anything runs."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

from _harness import gpu_index

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[no-alloc] {msg}", flush=True)


def _run_both(ctx, wl, two_tier, k, cm=1.0):
    index, has_rope, eta, eps, gam = gpu_index(ctx, wl, two_tier)
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"],
                    wl["r"] if wl["mode"] != synth.MODE_ROPE else 0, index=index,
                    index_has_rope=has_rope, P=wl["P"], eta=eta, eps=eps, gam=gam)
    res = []
    for static in (False, True):
        bufs = vkv.Buffers(step, k, two_tier=two_tier, cert_mult=cm)
        bufs.sel.fill_(-3)
        bufs.out.fill_(7)
        if static:
            # through the C ABI directly (the binding adds nothing)
            rc = ctx.lib.vkv_step_run_static(
                ctx.handle, step.ref, int(k), ctypes.c_void_p(bufs.key.data_ptr()),
                ctypes.c_void_p(bufs.ub.data_ptr()) if bufs.ub is not None else None,
                ctypes.c_void_p(bufs.sel.data_ptr()), ctypes.c_void_p(bufs.theta.data_ptr()),
                ctypes.c_void_p(bufs.adm.data_ptr()) if bufs.adm is not None else None,
                ctypes.c_void_p(bufs.adm_count.data_ptr()) if bufs.adm_count is not None else None,
                int(bufs.cap), ctypes.c_float(cm), ctypes.c_float(wl["scale"]),
                ctypes.c_void_p(bufs.out.data_ptr()), ctypes.c_void_p(bufs.lse.data_ptr()),
                ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            ctx.check(rc)
        else:
            bufs.run(ctx, step, wl["scale"])
        torch.cuda.synchronize()
        r = {"sel": bufs.sel.cpu().numpy(), "theta": bufs.theta.cpu().numpy(),
             "out": bufs.out.view(torch.int16).cpu().numpy(), "lse": bufs.lse.cpu().numpy()}
        if two_tier:
            r["adm_count"] = bufs.adm_count.cpu().numpy()
            r["adm"] = [bufs.adm[b, :int(r["adm_count"][b])].cpu().numpy() for b in range(wl["B"])]
        res.append(r)
    return res


def _same(a, b, two_tier):
    assert np.array_equal(a["sel"], b["sel"])
    assert np.array_equal(a["theta"], b["theta"])
    assert np.array_equal(a["out"], b["out"])
    assert np.array_equal(a["lse"], b["lse"])
    if two_tier:
        assert np.array_equal(a["adm_count"], b["adm_count"])
        for x, y in zip(a["adm"], b["adm"]):
            assert np.array_equal(x, y)


def test_static_workspace_matches_caller_workspace_twice():
    ctx = vkv.Context(0)
    # first call: a two-tier step of 3 x 30000 rows; second: a smaller one-tier step
    cases = [
        (synth.CONFIGS["cfg3"].with_(H=64), 3, 30000, 500, True),
        (synth.CONFIGS["cfg0"].with_(H=16), 1, 6000, 700, False),
    ]
    for cfg, B, T, k, two_tier in cases:
        _say(f"B={B} T={T} k={k} two_tier={two_tier} H={cfg.H}")
        wl = synth.make_workload(cfg, "cuda", B=B, T=T)
        ref, got = _run_both(ctx, wl, two_tier, k)
        _same(ref, got, two_tier)
        assert np.all(got["sel"][:, :k] >= 0)
    ctx.close()


def test_static_workspace_refuses_oversized_steps():
    ctx = vkv.Context(0)
    cfg = synth.CONFIGS["cfg4"]
    wl = synth.make_workload(cfg, "cuda", B=2, T=4096)   # inputs only; the shape below is what is checked
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], synth.MODE_ROPE, 0)
    step.c.B, step.c.T = 64, 65536                      # a workspace far above the static array
    step.c.cache_batch_stride = 65536 * 576
    need = vkv.workspace_size(step, 2048)
    assert need > (64 << 20)
    with pytest.raises(vkv.VkvError) as ei:
        vkv.step_run_static(ctx, step, 2048, wl["q_lat"], None, wl["q_lat"], wl["q_lat"], None, None, 0,
                            0.1, wl["q_lat"], wl["q_lat"])
    assert ei.value.code == -7 and "static" in str(ei.value)
    ctx.close()

"""GPU parity of the calibrated trigger (Sec. 4.2, Eq. (trigger) against the
tier-1 maximum logit; the conformal z; the optional top-j cap).

Bar: the tier-1 maxima s*_h and their rows bit-exact (fp64), the fired sets
bit-exact, the calibration statistics (hard flags, z_q) exact, the conformal
z equal, attention outputs within 2e-2 and lse within 1e-3.
"""
import sys

import numpy as np
import pytest
import torch

import _checks
import oracle
import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

from _harness import gpu_index, host_inputs, index_cols

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-trigger] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = vkv.Context(0)
    yield c
    c.close()


def _step_of(wl, pack):
    index, has_rope, eta, eps, gam = pack
    return vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"], index=index,
                    index_has_rope=has_rope, P=wl["P"], eta=eta, eps=eps, gam=gam)


@pytest.mark.parametrize("H,T,W", [(20, 3000, 40), (128, 5000, 256), (7, 600, 0)])
def test_row_max_is_exact(ctx, H, T, W):
    """vkv_row_max over lists (with and without the recent window) and over the
    whole context, against the oracle: maxima equal in fp64, rows equal
    (duplicated rows make ties, which go to the lower row)."""
    say(f"row max H={H} T={T} W={W}")
    cfg = synth.CONFIGS["cfg3"].with_(H=H, W=W)
    wl = synth.make_workload(cfg, "cuda", B=2, T=T)
    wl["cache"][1, 500] = wl["cache"][1, 77]           # ties in sequence 1
    wl["cache"][0, T - 1] = wl["cache"][0, 3]
    pack = gpu_index(ctx, wl, True)
    step = _step_of(wl, pack)
    A = wl["A"]
    g = torch.Generator().manual_seed(H)
    lists = torch.stack([torch.randperm(A, generator=g)[:min(A, 900)].sort().values for _ in range(2)])
    lists[1, 0] = 77
    lists[1, 1:] = lists[1, 1:].clamp(min=78)
    lists = lists.sort(dim=1).values.to(torch.int32).cuda().contiguous()
    cache, q_lat, q_rope, _ = host_inputs(wl, [0, 1])
    for rows, add_recent in ((lists, True), (lists, False), (None, True)):
        smax = torch.empty(2, H, dtype=torch.float64, device="cuda")
        arg = torch.empty(2, H, dtype=torch.int32, device="cuda")
        vkv.row_max(ctx, step, rows, add_recent, smax, arg)
        torch.cuda.synchronize()
        for b in range(2):
            lst = np.arange(A, dtype=np.int32) if rows is None else rows[b].cpu().numpy()
            if add_recent:
                lst = np.concatenate([lst, np.arange(A, wl["T"], dtype=np.int32)])
            osm, oarg = oracle.row_max(q_lat[b], q_rope[b], cache[b], lst)
            assert np.array_equal(smax[b].cpu().numpy(), osm), (b, rows is None, add_recent)
            assert np.array_equal(arg[b].cpu().numpy(), oarg), (b, rows is None, add_recent)


@pytest.mark.parametrize("nsplit_ws", [False, True])
def test_row_max_all_rows_tied(ctx, nsplit_ws):
    """Heads whose query is zero score every row 0: every row is a candidate,
    the per-head lists overflow and the kernel scores the whole range exactly;
    the maximum is 0 at the lowest listed row.  The other heads are ordinary.
    Through vkv_row_max (one range) and through the kept-tier step (several
    ranges merged)."""
    H, T, W = 20, 6000, 64
    say(f"row max with all rows tied, ranges={'several' if nsplit_ws else 'one'}")
    cfg = synth.CONFIGS["cfg3"].with_(H=H, W=W)
    wl = synth.make_workload(cfg, "cuda", B=2, T=T)
    wl["q_lat"][:, :3] = 0      # bf16 bits of +0
    wl["q_rope"][:, :3] = 0
    pack = gpu_index(ctx, wl, True)
    step = _step_of(wl, pack)
    A = wl["A"]
    g = torch.Generator().manual_seed(11)
    lists = torch.stack([torch.randperm(A, generator=g)[:1500].sort().values for _ in range(2)])
    lists = lists.to(torch.int32).cuda().contiguous()
    smax = torch.empty(2, H, dtype=torch.float64, device="cuda")
    arg = torch.empty(2, H, dtype=torch.int32, device="cuda")
    if nsplit_ws:
        k = lists.shape[1]
        ws = vkv.alloc_workspace(step, k, A)
        d = dict(dtype=torch.float32, device="cuda")
        ub = torch.empty(2, A, **d)
        fired = torch.empty(2, A, dtype=torch.int32, device="cuda")
        cnt = torch.empty(2, dtype=torch.int32, device="cuda")
        out = torch.empty(2, H, 512, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(2, H, **d)
        vkv.step_run_kept(ctx, step, ws, k, lists, None, ub, 0.1, smax, arg, 0, fired, cnt, A, wl["scale"], out, lse)
    else:
        vkv.row_max(ctx, step, lists, True, smax, arg)
    torch.cuda.synchronize()
    cache, q_lat, q_rope, _ = host_inputs(wl, [0, 1])
    for b in range(2):
        lst = np.concatenate([lists[b].cpu().numpy(), np.arange(A, wl["T"], dtype=np.int32)])
        osm, oarg = oracle.row_max(q_lat[b], q_rope[b], cache[b], lst)
        assert np.all(osm[:3] == 0.0) and np.all(oarg[:3] == lst.min())
        assert np.array_equal(smax[b].cpu().numpy(), osm), b
        assert np.array_equal(arg[b].cpu().numpy(), oarg), b


def _trigger_step(ctx, wl, k, cm, topj):
    pack = gpu_index(ctx, wl, True)
    step = _step_of(wl, pack)
    B, H, A = wl["B"], wl["H"], wl["A"]
    ws = vkv.alloc_workspace(step, k, A)
    d = dict(dtype=torch.float32, device="cuda")
    key = torch.empty(B, A, **d)
    ub = torch.empty(B, A, **d)
    sel = torch.empty(B, max(k, 1), dtype=torch.int32, device="cuda")
    theta = torch.empty(B, dtype=torch.float64, device="cuda")
    smax = torch.empty(B, H, dtype=torch.float64, device="cuda")
    arg = torch.empty(B, H, dtype=torch.int32, device="cuda")
    fired = torch.empty(B, A, dtype=torch.int32, device="cuda")
    cnt = torch.empty(B, dtype=torch.int32, device="cuda")
    out = torch.empty(B, H, 512, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, H, **d)
    vkv.step_run_trigger(ctx, step, ws, k, key, ub, sel, theta, cm, smax, arg, topj, fired, cnt, A,
                         wl["scale"], out, lse)
    torch.cuda.synchronize()
    return dict(sel=sel.cpu().numpy()[:, :k], theta=theta.cpu().numpy(), smax=smax.cpu().numpy(),
                fired=fired.cpu().numpy(), cnt=cnt.cpu().numpy(), out=out.float().cpu().numpy().astype(np.float64),
                lse=lse.cpu().numpy().astype(np.float64)), (step, ws, sel, ub, smax)


@pytest.mark.parametrize("cm,topj", [(1.0, 0), (0.12, 0), (0.12, 16), (0.0, 3)])
def test_trigger_step_against_the_oracle(ctx, cm, topj):
    say(f"trigger step cert_mult={cm} topj={topj}")
    cfg = synth.CONFIGS["cfg3"].with_(H=64)
    wl = synth.make_workload(cfg, "cuda", B=2, T=9000)
    k = 280
    g, _ = _trigger_step(ctx, wl, k, cm, topj)
    cache, q_lat, q_rope, P = host_inputs(wl, [0, 1])
    idx, eta, eps, gam = oracle.digest_build(cache, P, wl["r"], with_rope=True)
    o = oracle.step_trigger(cache, q_lat, q_rope, idx, P, wl["r"], wl["mode"], wl["W"], k, wl["scale"],
                           eta, eps, gam, cm, topj)
    for b in range(2):
        assert np.array_equal(g["sel"][b], o["sel"][b])
        assert np.array_equal(g["smax"][b], o["smax"][b]), b
        assert int(g["cnt"][b]) == o["fired_count"][b], (b, int(g["cnt"][b]), o["fired_count"][b])
        assert np.array_equal(g["fired"][b, :o["fired_count"][b]], o["fired"][b]), b
        assert _checks.rel_l2(g["out"][b], o["out"][b]) < _checks.OUT_TOL
        assert np.all(np.abs(g["lse"][b] - o["lse"][b]) < _checks.LSE_TOL)
    say(f"  fired per sequence: {[int(c) for c in g['cnt']]} of {wl['A'] - k} outside S")


def test_trigger_repeated_on_one_workspace(ctx):
    """vkv_trigger twice after one step (another cap the second time): each
    equals the oracle (the candidate list is emptied by its consumer)."""
    say("trigger repeated")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=5000)
    k = 150
    g, (step, ws, sel, ub, smax) = _trigger_step(ctx, wl, k, 0.15, 0)
    cache, q_lat, q_rope, P = host_inputs(wl, [0, 1])
    idx, eta, eps, gam = oracle.digest_build(cache, P, wl["r"], with_rope=True)
    A = wl["A"]
    for topj in (5, 0):
        fired = torch.empty(2, A, dtype=torch.int32, device="cuda")
        cnt = torch.empty(2, dtype=torch.int32, device="cuda")
        vkv.trigger(ctx, step, ws, k, sel, ub, 0.15, smax, topj, fired, cnt, A)
        torch.cuda.synchronize()
        o = oracle.step_trigger(cache, q_lat, q_rope, idx, P, wl["r"], wl["mode"], wl["W"], k, wl["scale"],
                               eta, eps, gam, 0.15, topj)
        for b in range(2):
            n = o["fired_count"][b]
            assert int(cnt[b]) == n and np.array_equal(fired[b, :n].cpu().numpy(), o["fired"][b])


def test_calibration_statistic_and_conformal_z(ctx):
    """Calibration queries of one request against its context (the context
    replicated per query): hard flags and z_q from the GPU equal the
    oracle's, and the library's conformal z of them equals the oracle's."""
    say("calibration")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    nq = 24
    base = synth.make_workload(cfg, "cuda", B=1, T=4000)
    qs = synth.make_workload(cfg, "cuda", B=nq, T=64, seed=11)       # fresh queries
    wl = dict(base)
    wl["B"] = nq
    wl["cache"] = base["cache"].expand(nq, -1, -1).contiguous()
    wl["q_lat"], wl["q_rope"] = qs["q_lat"], qs["q_rope"]
    pack = gpu_index(ctx, wl, True)
    step = _step_of(wl, pack)
    A, T, H, k, r = wl["A"], wl["T"], wl["H"], 120, wl["r"]
    ws = vkv.alloc_workspace(step, k, A)
    sel = torch.empty(nq, k, dtype=torch.int32, device="cuda")
    theta = torch.empty(nq, dtype=torch.float64, device="cuda")
    vkv.query_prep(ctx, step, ws)
    vkv.score(ctx, step, ws, None, None)
    vkv.select(ctx, step, ws, k, sel, theta)
    d64 = dict(dtype=torch.float64, device="cuda")
    s1, a1 = torch.empty(nq, H, **d64), torch.empty(nq, H, dtype=torch.int32, device="cuda")
    s2, a2 = torch.empty(nq, H, **d64), torch.empty(nq, H, dtype=torch.int32, device="cuda")
    vkv.row_max(ctx, step, sel, True, s1, a1)
    vkv.row_max(ctx, step, None, True, s2, a2)
    hard = torch.empty(nq, H, dtype=torch.int32, device="cuda")
    zq = torch.empty(nq, H, **d64)
    vkv.required_inflation(ctx, step, ws, k, sel, s1, a2, hard, zq)
    torch.cuda.synchronize()
    cache, q_lat, q_rope, P = host_inputs(wl, [0])
    idx, eta, eps, gam = oracle.digest_build(cache, P, r, with_rope=True)
    ql = synth.to_numpy_bits(wl["q_lat"])
    qr = synth.to_numpy_bits(wl["q_rope"])
    qt, a, n_, e = oracle.query_prep(ql, qr, P, r, wl["mode"])
    x = oracle.index_rows(cache[0], idx[0], wl["mode"], r, True)
    zs = []
    for b in range(nq):
        key, _ = oracle.index_keys(qt[b], x, A)
        osel, _ = oracle.select(key, k)
        assert np.array_equal(sel[b].cpu().numpy(), osel)
        t1 = np.concatenate([osel, np.arange(A, T, dtype=np.int32)])
        sm, _ = oracle.row_max(ql[b], qr[b], cache[0], t1)
        _, am = oracle.row_max(ql[b], qr[b], cache[0], np.arange(T, dtype=np.int32))
        oh, oz = oracle.required_inflation(qt[b], a[b], n_[b], e[b], x, eta[0], eps[0], gam[0], A, osel, r, sm, am)
        assert np.array_equal(hard[b].cpu().numpy().astype(bool), oh), b
        assert np.array_equal(zq[b].cpu().numpy()[oh], oz[oh]), b
        zs.extend(oz[oh].tolist())
    hz = zq.cpu().numpy()[hard.cpu().numpy().astype(bool)]
    assert len(zs) >= 18, len(zs)
    assert vkv.conformal_z(hz) == oracle.conformal_z(np.array(zs))
    z, mh, kk = vkv.conformal_z(hz)
    say(f"  hard pairs {len(zs)} of {nq * H}; z = {z:.4f} (rank {kk}, min_hard {mh})")

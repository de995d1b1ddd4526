"""Serving integration (Sec. 4.3, the decode step inside the model's graph):
the step captured in a HIP graph with worst-case buffers, several layers per
graph with the model's own work between them, and the all-layer CSR pack of
the fired rows.

Every graph is replayed several times with eager work and synchronisations
between replays; the inputs are refreshed in place between replays, and every
replay must reproduce the eager results of the same inputs bit for bit (the
same kernels run in both, and every step result is order-independent).
"""
import sys

import numpy as np
import pytest
import torch

import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

from _harness import gpu_index

pytestmark = pytest.mark.gpu
NB = vkv.SIGMA_BLOCK


def say(msg):
    print(f"[gpu-graph] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = vkv.Context(0)
    yield c
    c.close()


def _capture(fn):
    """Warm up on a side stream, then capture fn() into a graph."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _snapshot(tensors):
    return [t.clone() for t in tensors]


def _eager_noise():
    """The program's own eager work between replays."""
    a = torch.randn(512, 512, device="cuda")
    (a @ a).sum().item()
    torch.cuda.synchronize()


def _new_queries(wl, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    wl["q_lat"].copy_(torch.randn(wl["q_lat"].shape, generator=g, device="cuda").to(torch.bfloat16))
    wl["q_rope"].copy_(torch.randn(wl["q_rope"].shape, generator=g, device="cuda").to(torch.bfloat16))


@pytest.mark.parametrize("two_tier", [False, True])
def test_step_graph_replays_match_eager(ctx, two_tier):
    """vkv_step_run captured once, replayed on refreshed queries."""
    say(f"step graph two_tier={two_tier}")
    cfg = synth.CONFIGS["cfg3"].with_(H=32)
    wl = synth.make_workload(cfg, "cuda", B=3, T=6000)
    pack = gpu_index(ctx, wl, two_tier)
    index, has_rope, eta, eps, gam = pack
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"], index=index,
                    index_has_rope=has_rope, P=wl["P"], eta=eta, eps=eps, gam=gam)
    k = 500
    bufs = vkv.Buffers(step, k, two_tier=two_tier, cert_mult=0.15)
    outs = [bufs.sel, bufs.theta, bufs.out, bufs.lse] + ([bufs.adm, bufs.adm_count] if two_tier else [])
    g = _capture(lambda: bufs.run(ctx, step, wl["scale"]))
    ref_bufs = vkv.Buffers(step, k, two_tier=two_tier, cert_mult=0.15)
    ref_outs = [ref_bufs.sel, ref_bufs.theta, ref_bufs.out, ref_bufs.lse] + (
        [ref_bufs.adm, ref_bufs.adm_count] if two_tier else [])
    for rep in range(4):
        _new_queries(wl, 100 + rep)
        for t in outs:
            t.fill_(0) if t.dtype != torch.float64 else t.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(outs)
        _eager_noise()
        ref_bufs.run(ctx, step, wl["scale"])
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(got, ref_outs)):
            if two_tier and i == 4:      # adm: only the first adm_count rows are defined
                for s in range(wl["B"]):
                    n = int(min(ref_bufs.adm_count[s].item(), bufs.cap))
                    assert torch.equal(a[s, :n], b[s, :n]), (rep, s)
            else:
                assert torch.equal(a, b), (rep, i)
        say(f"  replay {rep} equal to eager")


def test_static_step_under_capture(ctx):
    """The no-allocation entry point captured: replays equal eager vkv_step_run."""
    say("static step graph")
    cfg = synth.CONFIGS["cfg3"].with_(H=16)
    wl = synth.make_workload(cfg, "cuda", B=2, T=5000)
    pack = gpu_index(ctx, wl, True)
    index, has_rope, eta, eps, gam = pack
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"], index=index,
                    index_has_rope=has_rope, P=wl["P"], eta=eta, eps=eps, gam=gam)
    k, A = 400, wl["A"]
    st = vkv.Buffers(step, k, two_tier=True, cert_mult=0.2)
    g = _capture(lambda: vkv.step_run_static(ctx, step, k, st.key, st.ub, st.sel, st.theta, st.adm, st.adm_count,
                                             A, wl["scale"], st.out, st.lse, cert_mult=0.2))
    ref = vkv.Buffers(step, k, two_tier=True, cert_mult=0.2)
    for rep in range(3):
        _new_queries(wl, 300 + rep)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot([st.sel, st.theta, st.out, st.lse, st.adm_count])
        _eager_noise()
        ref.run(ctx, step, wl["scale"])
        torch.cuda.synchronize()
        for a, b in zip(got, [ref.sel, ref.theta, ref.out, ref.lse, ref.adm_count]):
            assert torch.equal(a, b), rep


def test_multi_layer_decode_graph_with_csr_pack(ctx):
    """L layers of the deployed per-step path (sigma tier + trigger + top-j +
    attention, vkv_step_run_kept) in one graph; layer l + 1's query is made
    from layer l's output by the model's own (torch) work inside the graph;
    the fired rows of all layers and sequences are packed CSR at the end."""
    L, B, H, W = 3, 2, 16, 200
    T = 2 * NB + W
    cfg = synth.CONFIGS["cfg3"].with_(H=H, W=W)
    layers = []
    for layer in range(L):
        wl = synth.make_workload(cfg, "cuda", B=B, T=T, seed=50 + layer)
        index, has_rope, eta, eps, gam = gpu_index(ctx, wl, True)
        sig = torch.empty(B, 2 * NB, dtype=torch.float64, device="cuda")
        ws = torch.empty(vkv.sigma_workspace_size(B, 2), dtype=torch.uint8, device="cuda")
        vkv.sigma_close(ctx, wl["cache"], 0, 2, 16, ws, sig)
        K = vkv.sigma_tier_size(2 * NB, 380)
        kept = torch.empty(B, K, dtype=torch.int32, device="cuda")
        vkv.sigma_select(ctx, sig, 2 * NB, 380, 4, kept)
        layers.append(dict(wl=wl, index=index, has_rope=has_rope, eta=eta, eps=eps, gam=gam, kept=kept, K=K))
    A = 2 * NB
    q_lat = [layers[0]["wl"]["q_lat"]] + [torch.empty_like(layers[0]["wl"]["q_lat"]) for _ in range(L - 1)]
    q_rope = layers[0]["wl"]["q_rope"]
    fired = torch.empty(L, B, A, dtype=torch.int32, device="cuda")
    cnt = torch.empty(L, B, dtype=torch.int32, device="cuda")
    offsets = torch.empty(L * B + 1, dtype=torch.int32, device="cuda")
    packed = torch.empty(L * B * A, dtype=torch.int32, device="cuda")

    def build(outs):
        steps = []
        for layer, d in enumerate(layers):
            wl = d["wl"]
            step = vkv.Step(wl["cache"], q_lat[layer], q_rope, W, wl["mode"], wl["r"], index=d["index"],
                            index_has_rope=d["has_rope"], P=wl["P"], eta=d["eta"], eps=d["eps"], gam=d["gam"])
            f32 = dict(dtype=torch.float32, device="cuda")
            bufs = dict(ws=vkv.alloc_workspace(step, d["K"], A), key=torch.empty(B, A, **f32),
                        ub=torch.empty(B, A, **f32),
                        smax=torch.empty(B, H, dtype=torch.float64, device="cuda"),
                        arg=torch.empty(B, H, dtype=torch.int32, device="cuda"),
                        out=torch.empty(B, H, 512, dtype=torch.bfloat16, device="cuda"), lse=torch.empty(B, H, **f32))
            steps.append((step, bufs))
            outs.extend([bufs["smax"], bufs["arg"], bufs["out"], bufs["lse"]])
        return steps

    def run(steps, fired_t, cnt_t, offsets_t, packed_t):
        for layer, (step, b) in enumerate(steps):
            d = layers[layer]
            vkv.step_run_kept(ctx, step, b["ws"], d["K"], d["kept"], b["key"], b["ub"], 0.12, b["smax"], b["arg"],
                              16, fired_t[layer], cnt_t[layer], A, d["wl"]["scale"], b["out"], b["lse"])
            if layer + 1 < L:       # the model's work between layers
                q_lat[layer + 1].copy_((q_lat[layer].float() + 0.25 * b["out"].float()).to(torch.bfloat16))
        vkv.pack_rows(ctx, fired_t.view(L * B, A), cnt_t.view(L * B), offsets_t, packed_t)

    outs_g = []
    steps_g = build(outs_g)
    g = _capture(lambda: run(steps_g, fired, cnt, offsets, packed))
    outs_e = []
    steps_e = build(outs_e)
    fired_e, cnt_e = torch.empty_like(fired), torch.empty_like(cnt)
    offsets_e, packed_e = torch.empty_like(offsets), torch.empty_like(packed)
    for rep in range(3):
        _new_queries(dict(q_lat=q_lat[0], q_rope=q_rope), 700 + rep)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(outs_g + [cnt, offsets])
        got_fired = fired.clone()
        got_packed = packed.clone()
        _eager_noise()
        run(steps_e, fired_e, cnt_e, offsets_e, packed_e)
        torch.cuda.synchronize()
        for a, b in zip(got, outs_e + [cnt_e, offsets_e]):
            assert torch.equal(a, b), rep
        c = cnt_e.cpu().numpy().reshape(-1)
        off = offsets_e.cpu().numpy()
        assert off[0] == 0 and np.array_equal(np.diff(off), np.minimum(c, A))
        fe = fired_e.view(L * B, A).cpu().numpy()
        pk = packed_e.cpu().numpy()
        for i in range(L * B):
            n = min(int(c[i]), A)
            assert np.array_equal(got_fired.view(L * B, A)[i, :n].cpu().numpy(), fe[i, :n])
            assert np.array_equal(pk[off[i]:off[i] + n], fe[i, :n])
        assert torch.equal(got_packed[:off[-1]], packed_e[:off[-1]])
        say(f"  replay {rep}: fired per (layer, seq) {c.tolist()}")


def test_pack_rows_edge_cases(ctx):
    """Counts above cap pack cap rows, negative and zero counts none."""
    n, cap = 7, 5
    lists = torch.arange(n * cap, dtype=torch.int32, device="cuda").view(n, cap)
    counts = torch.tensor([0, 5, 9, -3, 2, 1, 5], dtype=torch.int32, device="cuda")
    offsets = torch.full((n + 1,), -1, dtype=torch.int32, device="cuda")
    packed = torch.full((n * cap,), -1, dtype=torch.int32, device="cuda")
    vkv.pack_rows(ctx, lists, counts, offsets, packed)
    torch.cuda.synchronize()
    lens = [0, 5, 5, 0, 2, 1, 5]
    assert offsets.cpu().tolist() == list(np.concatenate([[0], np.cumsum(lens)]))
    want = np.concatenate([np.arange(i * cap, i * cap + m) for i, m in enumerate(lens)])
    assert np.array_equal(packed.cpu().numpy()[:len(want)], want)


def test_page_bound_under_capture(ctx):
    """Query prep, page boxes and page bounds captured in one graph: replays on
    refreshed queries equal the eager calls (they allocate nothing and never
    synchronise)."""
    say("page bound graph")
    cfg = synth.CONFIGS["cfg3"].with_(H=32)
    wl = synth.make_workload(cfg, "cuda", B=2, T=7000)
    index, has_rope, *_ = gpu_index(ctx, wl, False)
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"], index=index,
                    index_has_rope=has_rope, P=wl["P"])
    page = 48
    npg = (wl["A"] + page - 1) // page
    n = synth.D_ROPE + wl["r"]
    ws = vkv.alloc_workspace(step, 0)
    box = torch.empty(2, npg, 2, n, dtype=torch.bfloat16, device="cuda")
    bound = torch.empty(2, npg, dtype=torch.float64, device="cuda")

    def run(w, bx, bd):
        s = torch.cuda.current_stream()
        vkv.query_prep(ctx, step, w, s)
        vkv.page_box(ctx, step, page, bx, s)
        vkv.page_bound(ctx, step, w, page, bx, bd, s)

    g = _capture(lambda: run(ws, box, bound))
    ws2 = vkv.alloc_workspace(step, 0)
    box2, bound2 = torch.empty_like(box), torch.empty_like(bound)
    for rep in range(3):
        _new_queries(wl, 300 + rep)
        bound.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        got = bound.clone()
        _eager_noise()
        run(ws2, box2, bound2)
        torch.cuda.synchronize()
        assert torch.equal(box, box2) and torch.equal(got, bound2), rep
        say(f"  replay {rep} equal to eager")

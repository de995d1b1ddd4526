"""GPU parity of the page-box bound (the page-bound pruning paragraph of the
appendix on prior algorithms) against the fp64 oracle: the boxes and the
bounds bit for bit, then the soundness of pruning by the bound against the
tier-1 set of the same step, with the fraction of pages it would skip."""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

from _harness import gpu_index, gpu_step, host_inputs, index_cols

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-page] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    vkv.load()
    c = vkv.Context(0)
    yield c
    c.close()


def _width(wl):
    cols, has_rope = index_cols(wl["mode"], wl["r"])
    return cols if cols else synth.D_ROPE


def gpu_pages(ctx, wl, page, index_pack=None):
    """Boxes and bounds through vkv_page_box / vkv_page_bound (after the query prep)."""
    if index_pack is None:
        index_pack = gpu_index(ctx, wl, False)
    index, has_rope, *_ = index_pack
    B, T, _ = wl["cache"].shape
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"],
                    wl["r"] if wl["mode"] != synth.MODE_ROPE else 0, index=index, index_has_rope=has_rope, P=wl["P"])
    ws = vkv.alloc_workspace(step, 0)
    vkv.query_prep(ctx, step, ws)
    A = T - wl["W"]
    npg = (A + page - 1) // page
    n = _width(wl)
    box = torch.empty(B, max(npg, 1), 2, n, dtype=torch.bfloat16, device="cuda")
    bound = torch.empty(B, max(npg, 1), dtype=torch.float64, device="cuda")
    vkv.page_box(ctx, step, page, box)
    vkv.page_bound(ctx, step, ws, page, box, bound)
    torch.cuda.synchronize()
    return (box.view(torch.int16).cpu().numpy().view(np.uint16)[:, :npg], bound.cpu().numpy()[:, :npg])


def oracle_pages(wl, seqs, page):
    """The oracle's boxes and bounds from the generator's inputs (its own index and query prep)."""
    cache, q_lat, q_rope, P = host_inputs(wl, seqs)
    mode, r, W = wl["mode"], wl["r"], wl["W"]
    cols, has_rope = index_cols(mode, r)
    rr = r if mode != synth.MODE_ROPE else 0
    index = None
    if cols:
        index = oracle.digest_build(cache, P, rr, with_rope=has_rope, scalars=False)[0]
    qt = oracle.query_prep(q_lat, q_rope, P, rr, mode)[0]
    A = cache.shape[1] - W
    out = []
    for j in range(len(seqs)):
        x = oracle.index_rows(cache[j], index[j] if index is not None else None, mode, rr, has_rope)
        box = oracle.page_box(x, A, page)
        out.append((box, oracle.page_bound(qt[j], box)))
    return out


def _wide(rng, shape, lo, hi):
    m = rng.integers(0, 128, shape)
    e = rng.integers(lo, hi, shape)
    sg = rng.choice([-1.0, 1.0], shape)
    return torch.from_numpy((sg * np.ldexp(1.0 + m / 128.0, e)).astype(np.float32)).to(torch.bfloat16)


@pytest.mark.parametrize("mode,r,page,T,W", [
    (synth.MODE_ROPE_DIGEST, 64, 64, 3000, 64),     # several pages, a ragged last one
    (synth.MODE_ROPE_DIGEST, 64, 1, 700, 20),       # one-row pages: the bound is the key
    (synth.MODE_DIGEST, 128, 37, 2500, 100),
    (synth.MODE_ROPE, 0, 100, 2100, 0),
    (synth.MODE_ROPE_DIGEST, 256, 5000, 3000, 10),  # one page holds every row
])
def test_page_box_and_bound_bit_exact(ctx, mode, r, page, T, W):
    say(f"page box/bound mode={mode} r={r} page={page} T={T} W={W}")
    cfg = synth.CONFIGS["cfg2_r64"].with_(H=24, mode=mode, r=r, W=W,
                                          basis="none" if mode == synth.MODE_ROPE else "orthonormal")
    wl = synth.make_workload(cfg, "cuda", B=2, T=T)
    box, bound = gpu_pages(ctx, wl, page)
    for b, (obox, obound) in enumerate(oracle_pages(wl, [0, 1], page)):
        assert np.array_equal(box[b], obox), f"box of sequence {b}"
        assert np.array_equal(bound[b], obound), f"bound of sequence {b}"


def test_page_bound_bit_exact_under_rounding(ctx):
    """Queries and rows spread over 2^40: the fp64 sums round at many steps,
    so any order other than d ascending changes some bounds."""
    say("page bound, wide inputs")
    rng = np.random.default_rng(7)
    cfg = synth.CONFIGS["cfg2_r64"].with_(H=16, mode=synth.MODE_ROPE, r=0, W=0, basis="none")
    wl = synth.make_workload(cfg, "cuda", B=2, T=1500)
    wl["cache"] = _wide(rng, (2, 1500, synth.D_ROW), -20, 20).cuda()
    wl["q_rope"] = _wide(rng, (2, 16, synth.D_ROPE), -20, 20).cuda()
    box, bound = gpu_pages(ctx, wl, 48)
    for b, (obox, obound) in enumerate(oracle_pages(wl, [0, 1], 48)):
        assert np.array_equal(box[b], obox) and np.array_equal(bound[b], obound)


def test_page_bound_without_archived_rows(ctx):
    cfg = synth.CONFIGS["cfg2_r64"].with_(H=8, W=256)
    wl = synth.make_workload(cfg, "cuda", B=1, T=256)
    box, bound = gpu_pages(ctx, wl, 64)
    assert box.shape[1] == 0 and bound.shape[1] == 0


def test_page_entry_points_refuse_bad_arguments(ctx):
    cfg = synth.CONFIGS["cfg2_r64"].with_(H=8)
    wl = synth.make_workload(cfg, "cuda", B=1, T=600)
    index, has_rope, *_ = gpu_index(ctx, wl, False)
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"], wl["r"], index=index,
                    index_has_rope=has_rope, P=wl["P"])
    ws = vkv.alloc_workspace(step, 0)
    box = torch.empty(1, 6, 2, wl["r"], dtype=torch.bfloat16, device="cuda")
    bound = torch.empty(1, 6, dtype=torch.float64, device="cuda")
    for bad in (0, -3):
        with pytest.raises(vkv.VkvError) as e:
            vkv.page_box(ctx, step, bad, box)
        assert e.value.code == -1
        with pytest.raises(vkv.VkvError) as e:
            vkv.page_bound(ctx, step, ws, bad, box, bound)
        assert e.value.code == -1
    with pytest.raises(vkv.VkvError) as e:
        vkv.page_bound(ctx, step, ws, 64, box, torch.empty(0, dtype=torch.float64, device="cuda"))
    assert e.value.code == -1
    with pytest.raises(vkv.VkvError) as e:   # a workspace too small for the query prep's outputs
        vkv.page_bound(ctx, step, ws[:16], 64, box, bound)
    assert e.value.code == -7


@pytest.mark.parametrize("name,page", [("cfg0", 8), ("cfg1", 16), ("cfg2_r64", 32), ("cfg3", 64), ("cfg4", 64)])
def test_pruning_by_the_page_bound_is_sound_at_full_size(ctx, name, page):
    """At the full configuration: the bounds of sampled sequences against the
    oracle bit for bit, and on every sequence no page whose bound is below
    the step's theta holds a tier-1 row; reports the share of pages such a
    scan would skip (the paper measures under 0.2% on its checkpoint)."""
    cfg = synth.CONFIGS[name]
    say(f"page pruning {name} page={page}")
    wl = synth.make_workload(cfg, "cuda")
    B = wl["cache"].shape[0]
    index_pack = gpu_index(ctx, wl, False)
    res, _ = gpu_step(ctx, wl, index_pack=index_pack)
    box, bound = gpu_pages(ctx, wl, page, index_pack)
    A, k = wl["A"], wl["k"]
    skipped = 0
    for b in range(B):
        prunable = bound[b] < res["theta"][b]
        skipped += int(prunable.sum())
        pages_of_sel = np.unique(res["sel"][b] // page)
        assert not np.any(prunable[pages_of_sel]), f"sequence {b}: a pruned page holds a tier-1 row"
    seqs = [0, B - 1]
    for j, (obox, obound) in zip(seqs, oracle_pages(wl, seqs, page)):
        assert np.array_equal(box[j], obox) and np.array_equal(bound[j], obound)
    frac = skipped / (B * bound.shape[1])
    say(f"{name} page={page}: {skipped} of {B * bound.shape[1]} pages below theta ({100 * frac:.3f}%)")

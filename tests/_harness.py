"""Shared drivers for the GPU parity tests: run one decode step through the
C ABI and the same step on the fp64 oracle, from the same seeded inputs."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

from _checks import rel_l2  # noqa: F401  (re-exported for the tests)


def index_cols(mode: int, r: int) -> tuple[int, bool]:
    """(columns, has_rope) of the packed index used for a mode."""
    if mode == synth.MODE_ROPE:
        return 0, True
    if mode == synth.MODE_DIGEST:
        return r, False
    return synth.D_ROPE + r, True


def gpu_index(ctx, wl, two_tier: bool):
    """Index (and certificate scalars) built on the GPU by vkv_digest_build."""
    cache, P, r, mode = wl["cache"], wl["P"], wl["r"], wl["mode"]
    B, T, _ = cache.shape
    cols, has_rope = index_cols(mode, r)
    index = None
    if cols:
        index = torch.empty(B, T, cols, dtype=torch.bfloat16, device=cache.device)
    eta = eps = gam = None
    if two_tier:
        eta = torch.empty(B, T, dtype=torch.float32, device=cache.device)
        eps = torch.empty_like(eta)
        gam = torch.empty_like(eta)
    if index is not None or two_tier:
        vkv.digest_build(ctx, cache, P, r if mode != synth.MODE_ROPE else 0, has_rope, index,
                         eta, eps, gam)
    return index, has_rope, eta, eps, gam


def gpu_step(ctx, wl, k=None, two_tier=False, cap=None, index_pack=None, cert_mult=1.0):
    """One full step through vkv_step_run.  Returns (host results, device bufs)."""
    k = wl["k"] if k is None else k
    if index_pack is None:
        index_pack = gpu_index(ctx, wl, two_tier)
    index, has_rope, eta, eps, gam = index_pack
    step = vkv.Step(wl["cache"], wl["q_lat"], wl["q_rope"], wl["W"], wl["mode"],
                    wl["r"] if wl["mode"] != synth.MODE_ROPE else 0, index=index,
                    index_has_rope=has_rope, P=wl["P"], eta=eta, eps=eps, gam=gam)
    bufs = vkv.Buffers(step, k, two_tier=two_tier, cap=cap, cert_mult=cert_mult)
    bufs.run(ctx, step, wl["scale"])
    torch.cuda.synchronize()
    res = {
        "key": bufs.key.cpu().numpy(),
        "sel": bufs.sel.cpu().numpy()[:, :k],
        "theta": bufs.theta.cpu().numpy(),
        "out": bufs.out.float().cpu().numpy().astype(np.float64),
        "out_bits": bufs.out.view(torch.int16).cpu().numpy().view(np.uint16),
        "lse": bufs.lse.cpu().numpy().astype(np.float64),
    }
    if two_tier:
        res["ub"] = bufs.ub.cpu().numpy()
        res["adm_count"] = bufs.adm_count.cpu().numpy()
        res["adm"] = bufs.adm.cpu().numpy()
    return res, (step, bufs, index_pack)


def host_inputs(wl, seqs):
    """Host bit copies of the inputs of the sequences ``seqs`` (the oracle's view)."""
    idx = list(seqs)
    t = torch.tensor(idx, device=wl["cache"].device)
    cache = synth.to_numpy_bits(wl["cache"].index_select(0, t))
    q_lat = synth.to_numpy_bits(wl["q_lat"].index_select(0, t))
    q_rope = synth.to_numpy_bits(wl["q_rope"].index_select(0, t))
    P = synth.to_numpy_bits(wl["P"]) if wl["P"] is not None else None
    return cache, q_lat, q_rope, P


def oracle_step(wl, seqs, k=None, two_tier=False, cap=None, nthreads=0, cert_mult=1.0):
    """The same step on the oracle for the listed sequences (inputs rebuilt
    from the generator's tensors; the index is built by the oracle itself)."""
    k = wl["k"] if k is None else k
    cache, q_lat, q_rope, P = host_inputs(wl, seqs)
    mode, r, W = wl["mode"], wl["r"], wl["W"]
    cols, has_rope = index_cols(mode, r)
    rr = r if mode != synth.MODE_ROPE else 0
    index = eta = eps = gam = None
    if cols or two_tier:
        index, eta, eps, gam = oracle.digest_build(cache, P, rr, with_rope=has_rope,
                                                   scalars=two_tier, nthreads=nthreads)
        if not cols:
            index = None
    res = oracle.step(cache, q_lat, q_rope, index, P, rr, mode, W, k, wl["scale"],
                      two_tier=two_tier, eta=eta, eps=eps, gam=gam, cap=cap,
                      index_has_rope=has_rope, nthreads=nthreads, cert_mult=cert_mult)
    out = {}
    for j, b in enumerate(seqs):
        out[b] = {key: res[key][j] for key in ("sel", "theta", "out", "lse", "key")}
        if two_tier:
            out[b]["adm"] = res["adm"][j]
            out[b]["adm_count"] = res["adm_count"][j]
    return out, (cache, q_lat, q_rope, P, index, eta, eps, gam)


def bf16_bits_of(x: np.ndarray) -> np.ndarray:
    """fp64 -> bf16 bits (one RNE, via the oracle's rounding)."""
    f = np.vectorize(oracle.round_bf16, otypes=[np.uint16])
    return f(x)

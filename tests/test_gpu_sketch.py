"""GPU parity of the data-driven sketch basis (Sec. 4.2, the index entry: V_r
from the context's own prefix queries) and of a certified step that uses it.

The oracle takes V_r as the top-r eigenvectors of the prefix queries' second
moment (a dense symmetric eigensolver); the GPU finds the same subspace by
subspace iteration.  Only the subspace is unique (any orthonormal basis of it
gives the same index scores and residual norms), so the bar is on
subspace-level quantities:
  * each row m_j of the GPU basis (bf16, divided by the 1 - 2^-6 factor) lies
    in the oracle's subspace up to its own bf16 rounding: the component
    outside is at most 2^-8 ||m_j|| (RNE's relative bound) plus 1e-6;
  * the rows are orthonormal up to that rounding (Gram within 3 * 2^-8 of I);
  * the captured second moment trace(V^T C V) equals the sum of the oracle's
    top-r eigenvalues to 1e-9 relative, the total trace(C) to 1e-12;
  * the rounded basis passes the contractivity check of the index build;
  * a two-tier step on that basis matches the oracle given the same basis
    (the standard step bar), and under an inflation z admits fewer rows than
    a random orthonormal basis of the same rank on queries concentrated near
    a subspace.
"""
import sys

import numpy as np
import pytest
import torch

import _checks
import oracle
import paper_2609_03949_amd as vkv
from paper_2609_03949_amd import synth

from _harness import gpu_step, oracle_step

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[gpu-sketch] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = vkv.Context(0)
    yield c
    c.close()


def _dec(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _gpu_basis(ctx, q: torch.Tensor, r: int, iters: int = 8):
    ws = torch.empty(vkv.sketch_workspace_size(r), dtype=torch.uint8, device=q.device)
    P = torch.empty(r, synth.D_LAT, dtype=torch.bfloat16, device=q.device)
    energy = torch.empty(2, dtype=torch.float64, device=q.device)
    vkv.sketch_basis(ctx, q, r, iters, ws, P, energy)
    torch.cuda.synchronize()
    return P, energy.cpu().numpy()


def _check_against_oracle(P_gpu: torch.Tensor, energy: np.ndarray, q_bits: np.ndarray, r: int):
    P_o, V_o, w_o = oracle.sketch_basis(q_bits, r)
    M = _dec(synth.to_numpy_bits(P_gpu)) / oracle.SKETCH_SCALE          # [r, 512]
    norms = np.linalg.norm(M, axis=1)
    outside = np.linalg.norm(M - (M @ V_o) @ V_o.T, axis=1)
    assert np.all(outside <= 2.0 ** -8 * norms + 1e-6), float(np.max(outside / norms))
    inside = M @ V_o
    assert np.max(np.abs(inside @ inside.T - np.eye(r))) < 3 * 2.0 ** -8
    C = oracle.content_second_moment(q_bits)
    assert abs(energy[0] - w_o.sum()) <= 1e-9 * w_o.sum(), (energy[0], w_o.sum())
    assert abs(energy[1] - np.trace(C)) <= 1e-12 * np.trace(C)
    return P_o, V_o, w_o


@pytest.mark.parametrize("r,m", [(64, 4096), (32, 1000), (256, 6000)])
def test_sketch_basis_spans_the_oracle_subspace(ctx, r, m):
    """Queries near an r-dim planted subspace: the top-r eigenspace is
    separated by a wide gap, so the GPU's subspace is the oracle's."""
    say(f"sketch r={r} m={m}")
    cfg = synth.CONFIGS["cfg0"].with_(queries="lowrank")
    q = synth.prefix_queries(cfg, m, "cuda", rank=r)
    P, energy = _gpu_basis(ctx, q, r)
    _check_against_oracle(P, energy, synth.to_numpy_bits(q), r)


def test_sketch_basis_beyond_the_gap(ctx):
    """r = 64 over queries near a 48-dim subspace: the 16 directions past the
    gap come from the isotropic noise, where the eigenvalues are not
    separated and no solver's subspace is unique.  The GPU basis still holds
    the planted 48 dimensions (to its rounding) and captures the optimal
    second moment up to the noise's share of it."""
    cfg = synth.CONFIGS["cfg0"].with_(queries="lowrank")
    q = synth.prefix_queries(cfg, 4096, "cuda")
    P, energy = _gpu_basis(ctx, q, 64)
    qb = synth.to_numpy_bits(q)
    _, V_o, w_o = oracle.sketch_basis(qb, 64)
    M = _dec(synth.to_numpy_bits(P)) / oracle.SKETCH_SCALE
    Qm, _ = np.linalg.qr(M.T)                       # orthonormal basis of the GPU's span
    top = V_o[:, :synth.QUERY_RANK]
    miss = np.linalg.norm(top - Qm @ (Qm.T @ top), axis=0)
    assert np.all(miss < 2.0 ** -7), float(miss.max())
    assert energy[0] <= w_o.sum() * (1 + 1e-12)
    assert energy[0] >= w_o[:synth.QUERY_RANK].sum() + 0.5 * w_o[synth.QUERY_RANK:].sum()


def test_sketch_basis_is_contractive_for_the_index_build(ctx):
    cfg = synth.CONFIGS["cfg0"].with_(queries="lowrank")
    q = synth.prefix_queries(cfg, 2048, "cuda")
    P, _ = _gpu_basis(ctx, q, 64)
    wl = synth.make_workload(cfg.with_(two_tier=True), device="cuda", T=1024)
    B, T, _ = wl["cache"].shape
    index = torch.empty(B, T, 64 + 64, dtype=torch.bfloat16, device="cuda")
    eta = torch.empty(B, T, dtype=torch.float32, device="cuda")
    eps, gam = torch.empty_like(eta), torch.empty_like(eta)
    vkv.digest_build(ctx, wl["cache"], P, 64, True, index, eta, eps, gam)   # raises if not contractive
    torch.cuda.synchronize()
    assert oracle.gershgorin(synth.to_numpy_bits(P)) < 1.0


def test_sketch_rejects_queries_of_too_low_rank(ctx):
    """Queries supported on 16 coordinates cannot give a 32-dim basis: the
    factorisation's pivot test reports it instead of returning noise."""
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    x = torch.zeros(512, synth.D_LAT, device="cuda")
    x[:, :16] = torch.randn(512, 16, generator=g, device="cuda")
    q = x.to(torch.bfloat16).contiguous()
    with pytest.raises(vkv.VkvError) as ei:
        _gpu_basis(ctx, q, 32)
    assert ei.value.code == -4
    # too few queries is the same defect
    q2 = synth.prefix_queries(synth.CONFIGS["cfg0"].with_(queries="lowrank"), 20, "cuda")
    with pytest.raises(vkv.VkvError):
        _gpu_basis(ctx, q2, 32)


def test_sketch_argument_errors(ctx):
    q = synth.prefix_queries(synth.CONFIGS["cfg0"], 64, "cuda")
    for r in (0, 16, 48, 544):
        with pytest.raises(vkv.VkvError):
            vkv.sketch_workspace_size(r)
    ws = torch.empty(vkv.sketch_workspace_size(64) - 256, dtype=torch.uint8, device="cuda")
    P = torch.empty(64, synth.D_LAT, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(vkv.VkvError) as ei:
        vkv.sketch_basis(ctx, q, 64, 4, ws, P)
    assert ei.value.code == -7


def test_step_on_the_sketch_basis_matches_the_oracle_and_admits_less(ctx):
    """A two-tier step (Sec. 4.2 with Lemma (Index certificate)) on the GPU's
    data-driven basis against the oracle on the same basis, under the sound
    bound and under an inflation z = 4 (multiplier z / sqrt(512 - r)).  The
    basis fitted to the queries' subspace leaves a small query residual a_h,
    so at z = 4 it admits far fewer rows than a random orthonormal basis of
    rank 64, which admits the whole archive."""
    cfg = synth.CONFIGS["cfg0"].with_(queries="lowrank", two_tier=True, basis="orthonormal")
    q = synth.prefix_queries(cfg, 4096, "cuda")
    P, _ = _gpu_basis(ctx, q, cfg.r)
    wl = synth.make_workload(cfg, device="cuda")
    k = wl["k"]
    cap = wl["A"] - k
    counts = {}
    for cm in (1.0, 4.0 / np.sqrt(512 - cfg.r)):
        for name, basis in (("random", wl["P"]), ("sketch", P)):
            w = dict(wl, P=basis)
            say(f"step basis={name} cert_mult={cm:.4f}")
            got, _ = gpu_step(ctx, w, two_tier=True, cap=cap, cert_mult=cm)
            want, _ = oracle_step(w, range(wl["B"]), two_tier=True, cap=cap, cert_mult=cm)
            _checks.check_step(got, want, range(wl["B"]), two_tier=True)
            counts[(name, cm)] = int(got["adm_count"].sum())
    say(f"admitted rows of the {wl['B'] * cap} outside S: {counts}")
    z4 = 4.0 / np.sqrt(512 - cfg.r)
    assert counts[("random", z4)] == wl["B"] * cap
    assert counts[("sketch", z4)] < 0.6 * counts[("random", z4)]

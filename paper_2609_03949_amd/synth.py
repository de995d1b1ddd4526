"""Seeded synthetic MLA-shaped decode workloads.

This module only draws inputs; it holds none of the method's arithmetic and is
the one piece shared by the HIP path's tests/bench and the oracle.  Every
tensor is drawn in fp32 from a torch generator seeded per (config seed,
sequence), so any sequence can be regenerated on its own, then rounded once
to bf16 (round-to-nearest-even).

Workloads follow the paper's decode setting (arXiv 2609.03949, Sec. 3
Eq. (setup)): cache rows of 576 bf16 = 512 content latent + 64 decoupled
branch; absorbed queries q_lat [H,512] and q_rope [H,64].
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

D_LAT, D_ROPE, D_ROW = 512, 64, 576
MODE_ROPE, MODE_DIGEST, MODE_ROPE_DIGEST = 1, 2, 3
MODE_NAMES = {MODE_ROPE: "rope", MODE_DIGEST: "digest", MODE_ROPE_DIGEST: "rope+digest"}


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    B: int
    H: int
    T: int
    W: int                 # recent window (always attended, never scored)
    k: int                 # per-sequence budget, rho * T
    mode: int              # index scoring mode
    r: int                 # digest rank (0 = none)
    basis: str             # "gaussian" (N(0,1/r)), "orthonormal" (0.97 * Q^T), "none"
    needles: int           # planted rows per sequence
    rows: str = "gaussian"  # "gaussian", "mixture", "lognormal"
    two_tier: bool = False  # certified admission on top of the top-k
    seed: int = 0
    queries: str = "gaussian"  # content queries: "gaussian" N(0, I), "lowrank" (QUERY_RANK-dim subspace + noise)

    @property
    def A(self) -> int:
        return self.T - self.W

    @property
    def n_index(self) -> int:
        return (D_ROPE if self.mode & 1 else 0) + (self.r if self.mode & 2 else 0)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(192.0)

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# The five decode workloads (shapes of the paper's 8k-128k needle/serving
# contexts at rho = 1/8, 1/32, 1/128 and the rank sweep r = 64..256).
CONFIGS = {
    "cfg0": Config("cfg0", B=1, H=16, T=8192, W=128, k=1024, mode=MODE_ROPE_DIGEST, r=64,
                   basis="gaussian", needles=8),
    "cfg1": Config("cfg1", B=8, H=128, T=32768, W=256, k=1024, mode=MODE_ROPE, r=0,
                   basis="none", needles=32),
    "cfg2_r64": Config("cfg2_r64", B=4, H=64, T=65536, W=256, k=512, mode=MODE_DIGEST, r=64,
                       basis="orthonormal", needles=32, rows="mixture"),
    "cfg2_r128": Config("cfg2_r128", B=4, H=64, T=65536, W=256, k=512, mode=MODE_DIGEST, r=128,
                        basis="orthonormal", needles=32, rows="mixture"),
    "cfg2_r192": Config("cfg2_r192", B=4, H=64, T=65536, W=256, k=512, mode=MODE_DIGEST, r=192,
                        basis="orthonormal", needles=32, rows="mixture"),
    "cfg2_r256": Config("cfg2_r256", B=4, H=64, T=65536, W=256, k=512, mode=MODE_DIGEST, r=256,
                        basis="orthonormal", needles=32, rows="mixture"),
    "cfg3": Config("cfg3", B=16, H=128, T=32768, W=256, k=1024, mode=MODE_ROPE_DIGEST, r=64,
                   basis="orthonormal", needles=32, rows="lognormal", two_tier=True),
    "cfg4": Config("cfg4", B=32, H=128, T=131072, W=512, k=4096, mode=MODE_ROPE_DIGEST, r=64,
                   basis="orthonormal", needles=256),
}

BASIS_SEED = 20260903
NEEDLE_SIGMAS = 6.0    # planted needle score, in standard deviations of a branch score


def describe(cfg: Config) -> str:
    return (f"{cfg.name}: B={cfg.B} H={cfg.H} T={cfg.T} W={cfg.W} k={cfg.k} "
            f"mode={MODE_NAMES[cfg.mode]} r={cfg.r} basis={cfg.basis} rows={cfg.rows} "
            f"needles={cfg.needles} two_tier={cfg.two_tier} queries={cfg.queries}")


# ------------------------------------------------------------------ helpers

def bf16_bits(x: torch.Tensor) -> torch.Tensor:
    """fp32 tensor -> bf16 tensor (round to nearest even)."""
    return x.to(torch.bfloat16)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def rope_rotate(x: torch.Tensor, pos0: int = 0, base: float = 1e4) -> torch.Tensor:
    """NeoX half-split rotary embedding of x [T, 64] at positions pos0.. (fp64 angles)."""
    T, d = x.shape
    half = d // 2
    i = torch.arange(half, device=x.device, dtype=torch.float64)
    theta = base ** (-2.0 * i / d)
    t = torch.arange(pos0, pos0 + T, device=x.device, dtype=torch.float64)
    ang = t[:, None] * theta[None, :]
    cos, sin = torch.cos(ang).float(), torch.sin(ang).float()
    x1, x2 = x[:, :half], x[:, half:]
    return torch.cat([x1 * cos - x2 * sin, x1 * sin + x2 * cos], dim=1)


def make_basis(kind: str, r: int, seed: int = BASIS_SEED, scale: float = 0.97) -> Optional[torch.Tensor]:
    """Digest basis P [r, 512] as bf16 (CPU).

    gaussian:    entries N(0, 1/r) so that E[(Pq).(Pc)] = q.c.
    orthonormal: scale * Q^T with Q from the QR of a seeded fp64 Gaussian
                 [512, r]; the 0.97 keeps the rounded basis contractive.
    identity:    P = I (r = 512); coordinate selectors for r < 512."""
    if kind == "none" or r == 0:
        return None
    g = _gen("cpu", seed + r)
    if kind == "gaussian":
        P = torch.randn(r, D_LAT, generator=g, dtype=torch.float64) / math.sqrt(r)
    elif kind == "orthonormal":
        G = torch.randn(D_LAT, r, generator=g, dtype=torch.float64)
        Q, _ = torch.linalg.qr(G)
        P = scale * Q.T
    elif kind == "identity":
        P = torch.eye(D_LAT, dtype=torch.float64)[:r]
    elif kind == "zero":
        P = torch.zeros(r, D_LAT, dtype=torch.float64)
    else:
        raise ValueError(kind)
    return bf16_bits(P.float()).contiguous()


def _plant(x: torch.Tensor, qdir: torch.Tensor, target: float) -> torch.Tensor:
    """Move x so that qdir.x = target (qdir unit): x + (target - qdir.x) qdir."""
    return x + (target - (x * qdir).sum(-1, keepdim=True)) * qdir


QUERY_RANK = 48       # dimension of the planted content-query subspace ("lowrank" queries)
QUERY_NOISE = 0.05    # isotropic noise per coordinate around it (signal: 3 per subspace coordinate)


def query_subspace(rank: int = QUERY_RANK, seed: int = BASIS_SEED + 1) -> torch.Tensor:
    """Orthonormal [512, rank] fp64 basis of the planted content-query subspace (CPU)."""
    g = _gen("cpu", seed + rank)
    U, _ = torch.linalg.qr(torch.randn(D_LAT, rank, generator=g, dtype=torch.float64))
    return U


def lowrank_content(n: int, g: torch.Generator, device, rank: int = QUERY_RANK,
                    noise: float = QUERY_NOISE) -> torch.Tensor:
    """n content queries [n, 512] fp32: 3 N(0, I_rank) coordinates in the planted
    subspace plus noise N(0, noise^2 I_512) (queries concentrated near a subspace,
    the regime the data-driven sketch basis is for)."""
    U = query_subspace(rank).float().to(device)
    coef = 3.0 * torch.randn(n, rank, generator=g, device=device)
    return coef @ U.T + noise * torch.randn(n, D_LAT, generator=g, device=device)


def prefix_queries(cfg: Config, m: int, device, seed: Optional[int] = None,
                   rank: int = QUERY_RANK) -> torch.Tensor:
    """m prefix content queries [m, 512] bf16 from the same law as the decode
    queries of ``cfg`` (another stream of the generator): the sample the sketch
    basis is computed from."""
    seed = cfg.seed if seed is None else seed
    g = _gen(device, 9_100_003 + 1013 * seed)
    if cfg.queries == "lowrank":
        x = lowrank_content(m, g, device, rank)
    else:
        x = torch.randn(m, D_LAT, generator=g, device=device)
    return bf16_bits(x).contiguous()


def make_queries(cfg: Config, device, seed: Optional[int] = None, B: Optional[int] = None):
    B = cfg.B if B is None else B
    seed = cfg.seed if seed is None else seed
    g = _gen(device, 7_000_003 + 1009 * seed)
    if cfg.queries == "lowrank":
        q_lat = lowrank_content(B * cfg.H, g, device).view(B, cfg.H, D_LAT)
    else:
        q_lat = torch.randn(B, cfg.H, D_LAT, generator=g, device=device)
    q_rope = torch.randn(B, cfg.H, D_ROPE, generator=g, device=device)
    return q_lat, q_rope


def make_sequence(cfg: Config, b: int, q_lat_b: torch.Tensor, q_rope_b: torch.Tensor, device,
                  T: Optional[int] = None, seed: Optional[int] = None):
    """One sequence's cache rows [T, 576] (fp32, before rounding) and needle rows."""
    T = cfg.T if T is None else T
    W = min(cfg.W, T)
    A = T - W
    seed = cfg.seed if seed is None else seed
    g = _gen(device, 1_000_003 * (seed + 1) + 7919 * b)
    if cfg.rows == "mixture":
        gc = _gen(device, 55_001 + seed)
        mu = torch.randn(64, D_LAT, generator=gc, device=device)
        assign = torch.randint(0, 64, (T,), generator=g, device=device)
        lat = mu[assign] + 0.5 * torch.randn(T, D_LAT, generator=g, device=device)
    else:
        lat = torch.randn(T, D_LAT, generator=g, device=device)
    rope = rope_rotate(torch.randn(T, D_ROPE, generator=g, device=device))
    gcpu = _gen("cpu", 31_337 + 104_729 * seed + b)
    n_needle = min(cfg.needles, A)
    pos = torch.randperm(A, generator=gcpu)[:n_needle].sort().values if A > 0 else torch.zeros(0, dtype=torch.long)
    if n_needle:
        heads = torch.arange(n_needle) % cfg.H
        pd = pos.to(device)
        hd = heads.to(device)
        qr = q_rope_b[hd].float()
        ql = q_lat_b[hd].float()
        qr_n = qr.norm(dim=-1, keepdim=True)
        ql_n = ql.norm(dim=-1, keepdim=True)
        # +6 sigma per branch: for rows ~ N(0, I) the score q.x of a branch has
        # sigma = ||q||, so the unit-direction component q^.x is set to 6,
        # which makes q.x = 6 ||q|| = 6 sigma
        rope[pd] = _plant(rope[pd], qr / qr_n, NEEDLE_SIGMAS)
        lat[pd] = _plant(lat[pd], ql / ql_n, NEEDLE_SIGMAS)
    row = torch.cat([lat, rope], dim=1)
    if cfg.rows == "lognormal":
        row = row * torch.exp(0.5 * torch.randn(T, 1, generator=g, device=device))
    return row, pos


def make_workload(cfg: Config, device="cpu", B: Optional[int] = None, T: Optional[int] = None,
                  seed: Optional[int] = None, basis: Optional[str] = None):
    """All inputs of one decode step for ``cfg`` (optionally with fewer
    sequences B or a shorter context T), as bf16 tensors on ``device``.

    Returns a dict: cache [B,T,576], q_lat [B,H,512], q_rope [B,H,64], P [r,512]
    or None, needles (list of LongTensor positions), plus the config values."""
    B = cfg.B if B is None else B
    T = cfg.T if T is None else T
    seed = cfg.seed if seed is None else seed
    q_lat32, q_rope32 = make_queries(cfg, device, seed, B)
    q_lat = bf16_bits(q_lat32)
    q_rope = bf16_bits(q_rope32)
    cache = torch.empty(B, T, D_ROW, dtype=torch.bfloat16, device=device)
    needles = []
    for b in range(B):
        row, pos = make_sequence(cfg, b, q_lat[b], q_rope[b], device, T, seed)
        cache[b] = bf16_bits(row)
        needles.append(pos)
        del row
    P = make_basis(basis or cfg.basis, cfg.r)
    if P is not None:
        P = P.to(device)
    W = min(cfg.W, T)
    return {
        "cfg": cfg, "B": B, "H": cfg.H, "T": T, "W": W, "A": T - W,
        "k": min(cfg.k, T - W), "mode": cfg.mode, "r": cfg.r, "scale": cfg.scale,
        "cache": cache, "q_lat": q_lat, "q_rope": q_rope, "P": P, "needles": needles,
    }


def to_numpy_bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)

"""Checkers shared by the GPU parity tests and their known-bad tests.

Each checker raises AssertionError when a result of the HIP path does not meet
the parity bar against the fp64 oracle: selected and admitted index sets
bit-exact, theta equal in fp64, attention outputs within 2e-2 relative L2 per
(b, h) and lse within 1e-3 (natural log), and fp32 index keys within their
certified band.  They take plain numpy arrays, so the CPU known-bad tests
drive them with oracle results into which a mistake has been planted.
"""
from __future__ import annotations

import numpy as np

OUT_TOL = 2e-2
LSE_TOL = 1e-3


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    """Relative L2 error per row (last axis), max over rows."""
    num = np.linalg.norm(a - b, axis=-1)
    den = np.maximum(np.linalg.norm(b, axis=-1), 1e-30)
    return float(np.max(num / den))


def check_step(g: dict, o: dict, seqs, two_tier: bool = False) -> bool:
    """g: the GPU step's host copies ("sel" [B,k], "theta" [B], "out" [B,H,512],
    "lse" [B,H], with two_tier also "adm" [B,cap] and "adm_count" [B]); o: the
    oracle's per-sequence results keyed by sequence index."""
    for b in seqs:
        ob = o[b]
        assert np.array_equal(g["sel"][b], ob["sel"]), f"sel differs for sequence {b}"
        if len(ob["sel"]):
            assert g["theta"][b] == ob["theta"], (b, g["theta"][b], ob["theta"])
        if two_tier:
            assert int(g["adm_count"][b]) == ob["adm_count"], (b, g["adm_count"][b], ob["adm_count"])
            m = min(ob["adm_count"], g["adm"].shape[1])
            assert np.array_equal(g["adm"][b, :m], ob["adm"][:m]), f"admitted set differs for {b}"
        err = rel_l2(g["out"][b], ob["out"])
        assert err < OUT_TOL, (b, err)
        fin = np.isfinite(ob["lse"])
        assert np.array_equal(fin, np.isfinite(g["lse"][b])), f"lse finiteness differs for {b}"
        assert np.all(np.abs(g["lse"][b][fin] - ob["lse"][fin]) < LSE_TOL), f"lse differs for {b}"
    return True


def check_keys_in_band(key_tilde: np.ndarray, key_exact: np.ndarray, E) -> float:
    """Every fp32 key within its certified band E (scalar or per row) of the
    exact fp64 key; returns the largest ratio error / E."""
    err = np.abs(np.asarray(key_tilde, np.float64) - np.asarray(key_exact, np.float64))
    E = np.broadcast_to(np.asarray(E, np.float64), err.shape)
    bad = err > E
    assert not np.any(bad), f"{int(bad.sum())} keys outside the band (first at row {int(np.argmax(bad))})"
    return float(np.max(err / E)) if err.size else 0.0

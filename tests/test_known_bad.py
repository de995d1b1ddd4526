"""Every parity gate first driven with a known-bad input (the discipline of
the paper's Sec. 6 and appendix "Measurement integrity: full protocol": a
check is trusted only after it has been shown to refuse a broken result).

The mistakes are planted on the CPU, in copies of the oracle's own results,
and fed to the same checkers the GPU parity tests use.
"""
import copy

import numpy as np
import pytest

import _checks
from paper_2609_03949_amd import synth


@pytest.fixture(scope="module")
def clean(oracle_mod):
    """One small two-tier step on the oracle, in the GPU result layout."""
    cfg = synth.CONFIGS["cfg3"].with_(H=8, r=64, rows="gaussian", needles=4)
    wl = synth.make_workload(cfg, "cpu", B=2, T=1200)
    cache = synth.to_numpy_bits(wl["cache"])
    q_lat = synth.to_numpy_bits(wl["q_lat"])
    q_rope = synth.to_numpy_bits(wl["q_rope"])
    P = synth.to_numpy_bits(wl["P"])
    index, eta, eps, gam = oracle_mod.digest_build(cache, P, cfg.r, with_rope=True)
    k = 40
    res = oracle_mod.step(cache, q_lat, q_rope, index, P, cfg.r, cfg.mode, wl["W"], k, cfg.scale,
                          two_tier=True, eta=eta, eps=eps, gam=gam, cert_mult=0.05)
    B, A = 2, wl["A"]
    o = {b: {key: res[key][b] for key in ("sel", "theta", "out", "lse", "key", "adm", "adm_count")}
         for b in range(B)}
    cap = A
    g = {
        "sel": np.stack([res["sel"][b] for b in range(B)]),
        "theta": np.array([res["theta"][b] for b in range(B)]),
        "out": np.stack([res["out"][b] for b in range(B)]),
        "lse": np.stack([res["lse"][b] for b in range(B)]),
        "adm_count": np.array([res["adm_count"][b] for b in range(B)], np.int32),
        "adm": np.zeros((B, cap), np.int32),
    }
    for b in range(B):
        g["adm"][b, :res["adm_count"][b]] = res["adm"][b]
    assert all(0 < res["adm_count"][b] < A - k for b in range(B))   # a partial admission
    return g, o


def _fails(g, o):
    with pytest.raises(AssertionError):
        _checks.check_step(g, o, [0, 1], two_tier=True)


def test_clean_result_passes(clean):
    g, o = clean
    assert _checks.check_step(g, o, [0, 1], two_tier=True)


def test_flipped_selected_index_is_refused(clean):
    g, o = copy.deepcopy(clean)
    sel = g["sel"][1]
    outside = np.setdiff1d(np.arange(sel.max() + 2), sel)
    sel[7] = outside[0]                       # one selected row replaced by another row
    g["sel"][1] = np.sort(sel)
    _fails(g, o)


def test_swapped_selected_order_is_refused(clean):
    g, o = copy.deepcopy(clean)
    g["sel"][0, [3, 4]] = g["sel"][0, [4, 3]]  # same set, not ascending
    _fails(g, o)


def test_theta_off_by_one_ulp_is_refused(clean):
    g, o = copy.deepcopy(clean)
    g["theta"][0] = np.nextafter(g["theta"][0], np.inf)
    _fails(g, o)


def test_dropped_or_replaced_admitted_row_is_refused(clean):
    g, o = copy.deepcopy(clean)
    g["adm_count"][0] -= 1                    # one admitted row missing from the count
    _fails(g, o)
    g, o = copy.deepcopy(clean)
    n = int(g["adm_count"][1])
    taken = set(g["adm"][1, :n]) | set(g["sel"][1])
    other = next(u for u in range(10 ** 6) if u not in taken)
    adm = np.sort(np.concatenate([np.delete(g["adm"][1, :n], n // 2), [other]]))
    g["adm"][1, :n] = adm                     # same count, one row replaced
    _fails(g, o)


def test_output_perturbed_beyond_tolerance_is_refused(clean):
    g, o = copy.deepcopy(clean)
    row = g["out"][1, 3]
    row += 2.5e-2 * np.linalg.norm(row) * np.eye(1, row.size, 11)[0]   # one element, rel-L2 2.5e-2
    _fails(g, o)
    # and a perturbation inside the tolerance passes
    g, o = copy.deepcopy(clean)
    row = g["out"][1, 3]
    row += 1.5e-2 * np.linalg.norm(row) * np.eye(1, row.size, 11)[0]
    assert _checks.check_step(g, o, [0, 1], two_tier=True)


def test_lse_perturbed_beyond_tolerance_is_refused(clean):
    g, o = copy.deepcopy(clean)
    g["lse"][0, 2] += 2e-3
    _fails(g, o)
    g, o = copy.deepcopy(clean)
    g["lse"][0, 2] = -np.inf
    _fails(g, o)


def test_band_shrunk_below_measured_error_is_refused(oracle_mod):
    """fp32 keys (the scorer's precision, here a plain float32 dot product)
    pass the certified band E = 2 (n + n/32) 2^-23 max ||qt|| max ||x||; the
    same keys fail once E is shrunk below the error actually measured."""
    rng = np.random.default_rng(3)
    n, H, A = 128, 16, 3000
    q = rng.standard_normal((H, n)).astype(np.float32)
    x = rng.standard_normal((A, n)).astype(np.float32)
    to_bits = lambda v: ((v.view(np.uint32).astype(np.uint64) + 0x7FFF
                          + ((v.view(np.uint32) >> 16) & 1)) >> 16).astype(np.uint16)
    qb, xb = to_bits(q), to_bits(x)
    key, _ = oracle_mod.index_keys(qb, xb, A)
    qd, xd = oracle_mod.decode_bf16(qb), oracle_mod.decode_bf16(xb)
    key32 = (xd.astype(np.float32) @ qd.astype(np.float32).T).max(axis=1)
    E = 2 * (n + n / 32) * 2.0 ** -23 * np.linalg.norm(qd, axis=1).max() * np.linalg.norm(xd, axis=1).max()
    ratio = _checks.check_keys_in_band(key32, key, E)
    assert 0 < ratio < 1
    measured = np.max(np.abs(key32.astype(np.float64) - key))
    with pytest.raises(AssertionError):
        _checks.check_keys_in_band(key32, key, 0.5 * measured)
    # a single key moved just outside the band is caught too
    bad = key32.astype(np.float64).copy()
    bad[1234] = key[1234] + 1.01 * E
    with pytest.raises(AssertionError):
        _checks.check_keys_in_band(bad, key, E)

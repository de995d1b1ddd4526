"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Every check here compares the oracle with something other than itself: exact
rational arithmetic, closed forms, textbook special cases, invariants the
paper states (Lemma (Index certificate), Lemma (Bounded leakage), Lemma
(Exchangeability), the Eq. (reads) byte budget) or brute force on tiny inputs.
CPU only.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2609_03949_amd import budget, synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(12345)


# ----------------------------------------------------------------- helpers

def bits_of(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits by exact rational RNE (independent of the oracle)."""
    return np.array([exact_rne_bf16(Fraction(float(v))) for v in np.ravel(x)],
                    np.uint16).reshape(np.shape(x))


def exact_rne_bf16(q: Fraction) -> int:
    """Round an exact rational to the nearest bf16 (ties to even); bits."""
    if q == 0:
        return 0
    sign = 0x8000 if q < 0 else 0
    a = abs(q)
    # exponent E with 2^E <= a < 2^(E+1)
    E = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** E > a:
        E -= 1
    if Fraction(2) ** (E + 1) <= a:
        E += 1
    qexp = E - 7 if E >= -126 else -133
    scaled = a / Fraction(2) ** qexp
    fl = scaled.numerator // scaled.denominator
    frac = scaled - fl
    if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    val = Fraction(fl) * Fraction(2) ** qexp
    if val >= Fraction(2) ** 128:
        return sign | 0x7F80
    f = np.float32(float(val))
    return sign | int(np.array([f], np.float32).view(np.uint32)[0] >> 16)


def dec(bits) -> np.ndarray:
    b = np.asarray(bits, np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def frac_of_bits(b: int) -> Fraction:
    return Fraction(float(dec(np.array([b], np.uint16))[0]))


def small_int_bf16(shape, lo=-8, hi=8) -> np.ndarray:
    """bf16 bits of small integers: every fp64 dot product of these is exact."""
    v = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def rand_bf16(shape, scale=1.0) -> np.ndarray:
    v = (rng.standard_normal(shape) * scale).astype(np.float32)
    # torch-independent RNE fp32 -> bf16
    u = v.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def exact_dot(a_bits, b_bits) -> Fraction:
    return sum((frac_of_bits(int(x)) * frac_of_bits(int(y)) for x, y in zip(a_bits, b_bits)),
               Fraction(0))


def fsqrt_upper(x: Fraction) -> float:
    return math.sqrt(float(x)) if x > 0 else 0.0


# ----------------------------------------------------------- bf16 rounding

def test_round_bf16_matches_exact_rational_rne(oracle_mod):
    vals = list(rng.standard_normal(400) * np.exp(rng.uniform(-60, 60, 400)))
    # exact halfway cases between adjacent bf16 values, both parities
    for m in (0x3F80, 0x3F81, 0x4000, 0x4001, 0x0080, 0x0081, 0x7F7D, 0x7F7E, 0x0001, 0x0002):
        lo = frac_of_bits(m)
        hi = frac_of_bits(m + 1)
        vals += [float((lo + hi) / 2), float(-(lo + hi) / 2)]
        vals += [float((lo + hi) / 2) * (1 + 2 ** -40), float((lo + hi) / 2) * (1 - 2 ** -40)]
    # subnormal range, overflow, values that double-round through fp32
    vals += [1e-39, -3e-40, 2e-45, 1e38, 3.3e38, 3.4e38]
    half_to_inf = float((Fraction(2) - Fraction(1, 256)) * Fraction(2) ** 127)
    vals += [half_to_inf * (1 - 2 ** -40)]
    vals += [1.0 + 2 ** -8 + 2 ** -30, 1.0 + 2 ** -8 - 2 ** -30, 1.0 + 2 ** -9 + 2 ** -35]
    for v in vals:
        want = exact_rne_bf16(Fraction(v))
        got = oracle_mod.round_bf16(v)
        assert got == want, (v, hex(got), hex(want))
    assert oracle_mod.round_bf16(0.0) == 0 and oracle_mod.round_bf16(-0.0) == 0x8000
    assert oracle_mod.round_bf16(half_to_inf) == 0x7F80      # ties to even -> overflow
    assert oracle_mod.round_bf16(-1e39) == 0xFF80


def test_ru_f32_and_ru_sqrt_are_tight_upper_roundings(oracle_mod):
    xs = list(np.abs(rng.standard_normal(300)) * np.exp(rng.uniform(-30, 30, 300)))
    xs += [0.0, 1.0, 2.0, 4.0, 1e-30, 123456789.123]
    for x in xs:
        f = oracle_mod.ru_f32(x)
        assert Fraction(f) >= Fraction(x)
        prev = np.nextafter(np.float32(f), np.float32(-np.inf))
        assert Fraction(float(prev)) < Fraction(x) or f == 0.0
        s = oracle_mod.ru_sqrt_f32(x)
        assert Fraction(s) ** 2 >= Fraction(x)
        sp = np.nextafter(np.float32(s), np.float32(0))
        assert s == 0.0 or Fraction(float(sp)) ** 2 < Fraction(x)


# ------------------------------------------------------------ digest / index

def _cache_from_latent(lat_bits, rope_bits=None):
    T = lat_bits.shape[0]
    if rope_bits is None:
        rope_bits = rand_bf16((T, 64))
    return np.concatenate([lat_bits, rope_bits], axis=1)[None].copy()


def test_digest_identity_basis_reproduces_latent_bits(oracle_mod):
    lat = rand_bf16((24, 512))
    cache = _cache_from_latent(lat)
    P = np.eye(512, dtype=np.float32)
    Pb = (P.view(np.uint32) >> 16).astype(np.uint16)
    index, eta, eps, gam = oracle_mod.digest_build(cache, Pb, 512, with_rope=True)
    assert np.array_equal(index[0, :, :64], cache[0, :, 512:])
    assert np.array_equal(index[0, :, 64:], lat)
    cn = np.linalg.norm(dec(lat), axis=1)
    # nothing is left outside the sketch: eta and eps are at the margin level
    assert np.all(eta[0] < 1e-3 * cn) and np.all(eps[0] < 1e-8 * cn)
    assert np.all(gam[0] >= cn) and np.all(gam[0] <= cn * (1 + 1e-6))


def test_digest_coordinate_selector_and_residual_norm(oracle_mod):
    lat = rand_bf16((16, 512))
    cache = _cache_from_latent(lat)
    cols = np.sort(rng.choice(512, 64, replace=False))
    P = np.zeros((64, 512), np.float32)
    P[np.arange(64), cols] = 1.0
    Pb = (P.view(np.uint32) >> 16).astype(np.uint16)
    index, eta, eps, gam = oracle_mod.digest_build(cache, Pb, 64, with_rope=False)
    assert np.array_equal(index[0], lat[:, cols])
    c = dec(lat)
    rest = np.delete(c, cols, axis=1)
    want_eta = np.linalg.norm(rest, axis=1)
    want_gam = np.linalg.norm(c[:, cols], axis=1)
    assert np.all(eta[0] >= want_eta * (1 - 1e-12))
    assert np.allclose(eta[0], want_eta, rtol=1e-6)
    assert np.allclose(gam[0], want_gam, rtol=1e-6) and np.all(gam[0] >= want_gam * (1 - 1e-12))
    assert np.all(eps[0] < 1e-8 * np.linalg.norm(c, axis=1))


def _f32_up_sqrt(x: Fraction) -> float:
    """Smallest float f with f * f >= x (exact rational search)."""
    f = np.float32(math.sqrt(float(x))) if x > 0 else np.float32(0)
    while Fraction(float(f)) ** 2 < x:
        f = np.nextafter(f, np.float32(np.inf))
    while f > 0:
        p = np.nextafter(f, np.float32(0))
        if Fraction(float(p)) ** 2 >= x:
            f = p
        else:
            break
    return float(f)


def test_digest_zero_basis_gives_exact_margin_values(oracle_mod):
    """P = 0: the sketch is empty, so w = P c = 0 exactly and the only nonzero
    parts of eps and gamma are the rounding margin of the bound on ||P c - w||,
    2^-40 * sqrt(r * ||c||^2) rounded up (exact values below, from rational
    arithmetic); eta is a tight upper bound of ||c||.  Small-integer latents
    make ||c||^2 an exact fp64 integer."""
    r = 64
    lat = small_int_bf16((8, 512), -6, 6)
    cache = _cache_from_latent(lat)
    Pb = np.zeros((r, 512), np.uint16)
    index, eta, eps, gam = oracle_mod.digest_build(cache, Pb, r, with_rope=True)
    assert np.all(index[0, :, 64:] == 0)
    for u in range(8):
        N = sum((frac_of_bits(int(b)) ** 2 for b in lat[u]), Fraction(0))
        margin = Fraction(2) ** -40 * Fraction(_f32_up_sqrt(r * N))
        assert Fraction(float(eps[0, u])) == margin and Fraction(float(gam[0, u])) == margin
        e = Fraction(float(eta[0, u]))
        assert e * e >= N
        prev = Fraction(float(np.nextafter(np.float32(eta[0, u]), np.float32(0))))
        assert prev * prev < N * (1 + Fraction(1, 2 ** 36))


def test_query_prep_head_scalars_against_exact_rationals(oracle_mod):
    """Head side of Lemma (Index certificate) with the bf16 rounding of the
    query digest: a_h, n_h = ||qd_h||, e_h = ||qd_h - P q_h|| are valid upper
    bounds of the exact quantities and tight (exact rational arithmetic);
    qd_h = RNE(P q_h) of the exact sum."""
    r, H = 8, 3
    q_lat = rand_bf16((1, H, 512))
    q_rope = rand_bf16((1, H, 64))
    Pb = synth.to_numpy_bits(synth.make_basis("orthonormal", r))
    qt, a, nq, e = oracle_mod.query_prep(q_lat, q_rope, Pb, r, oracle_mod.MODE_ROPE_DIGEST)
    assert np.array_equal(qt[0, :, :64], q_rope[0])
    for h in range(H):
        q = [frac_of_bits(int(b)) for b in q_lat[0, h]]
        w = [sum((frac_of_bits(int(Pb[j, i])) * q[i] for i in range(512)), Fraction(0))
             for j in range(r)]
        d = [exact_rne_bf16(v) for v in w]
        assert list(qt[0, h, 64:]) == d
        Nq = sum((v * v for v in q), Fraction(0))
        Nw = sum((v * v for v in w), Fraction(0))
        Nd = sum((frac_of_bits(dj) ** 2 for dj in d), Fraction(0))
        Ne = sum(((frac_of_bits(d[j]) - w[j]) ** 2 for j in range(r)), Fraction(0))
        qn = math.sqrt(float(Nq))
        # n_h: the smallest float above ||qd|| up to the 2^-40 margin -- tight to ~1 ulp
        nh = Fraction(float(nq[0, h]))
        assert nh * nh >= Nd
        prev = Fraction(float(np.nextafter(np.float32(nq[0, h]), np.float32(0))))
        assert prev * prev < Nd * (1 + Fraction(1, 2 ** 36))
        for got, ex in ((a[0, h], Nq - Nw), (e[0, h], Ne)):
            assert Fraction(float(got)) ** 2 >= ex
            assert float(got) <= fsqrt_upper(ex) * (1 + 1e-6) + 1e-9 * qn


def test_digest_random_basis_against_exact_rationals(oracle_mod):
    """d = RNE(P c) of the exact sum; eta/eps/gamma are valid and tight upper
    bounds of sqrt(c^T (I-P^T P) c), ||d - P c||, ||P c|| (exact arithmetic)."""
    r = 8
    lat = rand_bf16((3, 512))
    cache = _cache_from_latent(lat)
    P = synth.make_basis("orthonormal", r)
    Pb = synth.to_numpy_bits(P)
    index, eta, eps, gam = oracle_mod.digest_build(cache, Pb, r, with_rope=False)
    for u in range(3):
        c = [frac_of_bits(int(b)) for b in lat[u]]
        y = [sum((frac_of_bits(int(Pb[j, i])) * c[i] for i in range(512)), Fraction(0))
             for j in range(r)]
        d = [exact_rne_bf16(v) for v in y]
        assert list(index[0, u]) == d
        cc = sum((v * v for v in c), Fraction(0))
        yy = sum((v * v for v in y), Fraction(0))
        ee = sum(((frac_of_bits(d[j]) - y[j]) ** 2 for j in range(r)), Fraction(0))
        for got, ex in ((eta[0, u], cc - yy), (eps[0, u], ee), (gam[0, u], yy)):
            assert Fraction(float(got)) ** 2 >= ex          # valid upper bound
            assert float(got) <= fsqrt_upper(ex) * (1 + 1e-6) + 1e-6  # and tight


def test_basis_used_by_configs_is_certified_contractive(oracle_mod):
    for r in (64, 128, 192, 256):
        Pb = synth.to_numpy_bits(synth.make_basis("orthonormal", r))
        assert oracle_mod.gershgorin(Pb) < 1.0
        s = np.linalg.svd(dec(Pb), compute_uv=False)
        assert s[0] <= 1.0 and s[0] ** 2 <= oracle_mod.gershgorin(Pb)


# --------------------------------------------------------------- index keys

def test_keys_single_head_is_plain_dot_product(oracle_mod):
    q = small_int_bf16((1, 96))
    x = small_int_bf16((50, 96))
    key, bad = oracle_mod.index_keys(q, x, 50, check_exact=True)
    want = dec(x) @ dec(q)[0]
    assert bad == 0
    assert np.array_equal(key, want)


def test_keys_zero_query_gives_zero_and_first_k_selected(oracle_mod):
    q = np.zeros((4, 128), np.uint16)
    x = rand_bf16((300, 128))
    key, _ = oracle_mod.index_keys(q, x, 300)
    assert np.all(key == 0.0)
    sel, theta = oracle_mod.select(key, 37)
    assert np.array_equal(sel, np.arange(37)) and theta == 0.0


def test_keys_are_max_over_heads(oracle_mod):
    q = rand_bf16((16, 128))
    x = rand_bf16((500, 128))
    key, bad = oracle_mod.index_keys(q, x, 500, check_exact=True)
    per_head = np.stack([oracle_mod.index_keys(q[h:h + 1], x, 500)[0] for h in range(16)], 1)
    assert np.array_equal(key, per_head.max(1))
    assert np.allclose(key, (dec(x) @ dec(q).T).max(1), rtol=1e-12, atol=1e-12)


def test_full_rank_identity_digest_gives_exact_latent_and_full_scores(oracle_mod):
    H, T, W = 3, 40, 8
    lat = small_int_bf16((T, 512), -3, 3)
    rope = small_int_bf16((T, 64), -3, 3)
    cache = np.concatenate([lat, rope], 1)[None].copy()
    q_lat = small_int_bf16((1, H, 512), -3, 3)
    q_rope = small_int_bf16((1, H, 64), -3, 3)
    Pb = (np.eye(512, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)
    index, *_ = oracle_mod.digest_build(cache, Pb, 512, with_rope=True, scalars=False)
    A = T - W
    lat_scores = dec(lat[:A]) @ dec(q_lat[0]).T
    full = lat_scores + dec(rope[:A]) @ dec(q_rope[0]).T
    for mode, want in ((oracle_mod.MODE_DIGEST, lat_scores.max(1)),
                       (oracle_mod.MODE_ROPE_DIGEST, full.max(1))):
        qt, *_ = oracle_mod.query_prep(q_lat, q_rope, Pb, 512, mode)
        x = oracle_mod.index_rows(cache[0], index[0], mode, 512)
        key, bad = oracle_mod.index_keys(qt[0], x, A, check_exact=True)
        assert bad == 0 and np.array_equal(key, want)
    s = oracle_mod.full_scores(q_lat[0], q_rope[0], cache[0], A)
    assert np.array_equal(s, full)


@pytest.mark.parametrize("name", sorted(synth.CONFIGS))
def test_keys_are_exact_on_every_workload(oracle_mod, name):
    """The exactness self-check on a reduced shape of every workload (one
    sequence, 1536 rows, the workload's own heads, mode and basis): every
    sequential fp64 key sum equals the exact real dot product, so on these
    inputs the sequential definition is the exact one."""
    cfg = synth.CONFIGS[name]
    wl = synth.make_workload(cfg, "cpu", B=1, T=1536)
    cache = synth.to_numpy_bits(wl["cache"])
    Pb = synth.to_numpy_bits(wl["P"]) if wl["P"] is not None else None
    q_lat = synth.to_numpy_bits(wl["q_lat"])
    q_rope = synth.to_numpy_bits(wl["q_rope"])
    rr = cfg.r if cfg.mode != oracle_mod.MODE_ROPE else 0
    has_rope = cfg.mode != oracle_mod.MODE_DIGEST
    index = None
    if cfg.mode != oracle_mod.MODE_ROPE:
        index, *_ = oracle_mod.digest_build(cache, Pb, rr, with_rope=has_rope, scalars=False)
    qt, *_ = oracle_mod.query_prep(q_lat, q_rope, Pb, rr, cfg.mode)
    x = oracle_mod.index_rows(cache[0], None if index is None else index[0], cfg.mode, rr, has_rope)
    key, bad = oracle_mod.index_keys(qt[0], x, wl["A"], check_exact=True)
    assert bad == 0


# ------------------------------------------------------------------ select

def test_select_matches_brute_force_sort_with_ties(oracle_mod):
    for A, k in ((1, 1), (10, 3), (257, 64), (1000, 999), (1000, 1000), (50, 0)):
        key = rng.integers(-4, 5, size=A).astype(np.float64)
        sel, theta = oracle_mod.select(key, k)
        order = sorted(range(A), key=lambda u: (-key[u], u))[:k]
        assert list(sel) == sorted(order)
        assert theta == (min(key[order]) if k else -math.inf)


def test_select_all_ties_takes_lowest_indices(oracle_mod):
    key = np.full(100, 2.5)
    sel, theta = oracle_mod.select(key, 10)
    assert np.array_equal(sel, np.arange(10)) and theta == 2.5


# --------------------------------------------------------- bound / admission

def _tiny_two_tier(oracle_mod, basis="orthonormal", r=32, T=300, W=20, H=4, lognormal=True,
                   needles=32):
    cfg = synth.CONFIGS["cfg3"].with_(H=H, r=r, basis=basis, needles=needles,
                                      rows="lognormal" if lognormal else "gaussian")
    wl = synth.make_workload(cfg, "cpu", B=1, T=T)
    cache = synth.to_numpy_bits(wl["cache"])
    Pb = synth.to_numpy_bits(wl["P"]) if wl["P"] is not None else None
    q_lat = synth.to_numpy_bits(wl["q_lat"])
    q_rope = synth.to_numpy_bits(wl["q_rope"])
    index, eta, eps, gam = oracle_mod.digest_build(cache, Pb, r, with_rope=True)
    qt, a, nq, e = oracle_mod.query_prep(q_lat, q_rope, Pb, r, oracle_mod.MODE_ROPE_DIGEST)
    x = oracle_mod.index_rows(cache[0], index[0], oracle_mod.MODE_ROPE_DIGEST, r)
    return wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x


def test_certificate_bounds_every_head_and_row(oracle_mod):
    """Lemma (Index certificate): |s_h(u) - s^_h(u)| <= B_h(u) for all (u, h)."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(oracle_mod)
    A = wl["A"]
    s = oracle_mod.full_scores(q_lat[0], q_rope[0], cache[0], A)
    H = qt.shape[1]
    for h in range(H):
        sh_hat, _ = oracle_mod.index_keys(qt[0, h:h + 1], x, A)
        Bh = a[0, h].astype(np.float64) * eta[0, :A] + nq[0, h] * eps[0, :A].astype(np.float64) \
            + e[0, h] * gam[0, :A].astype(np.float64)
        gap = np.abs(s[:, h] - sh_hat)
        assert np.all(gap <= Bh * (1 + 1e-9))
        # the bound is Cauchy-Schwarz, so it is loose but not absurdly so
        assert np.all(Bh <= 2.0 * (np.linalg.norm(dec(q_lat[0, h])) *
                                   np.linalg.norm(dec(cache[0, :A, :512]), axis=1)) + 1e-6)


def test_admission_invariant_on_every_skipped_row(oracle_mod):
    """Every archived row that is neither selected nor admitted has
    max_h s_h(u) <= UB_u <= theta (s exact), i.e. it could not beat S."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="identity", r=448, lognormal=False)
    A = wl["A"]
    key, _ = oracle_mod.index_keys(qt[0], x, A)
    sel, theta = oracle_mod.select(key, 30)
    ub = oracle_mod.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A)
    adm, cnt = oracle_mod.admit(ub, sel, theta)
    s = oracle_mod.full_scores(q_lat[0], q_rope[0], cache[0], A).max(1)
    assert np.all(s <= ub * (1 + 1e-12) + 1e-9)
    skipped = np.setdiff1d(np.arange(A), np.concatenate([sel, adm]))
    assert np.all(ub[skipped] <= theta) and np.all(s[skipped] <= theta + 1e-9)
    assert np.all(ub[adm] > theta) and len(np.intersect1d(adm, sel)) == 0
    assert 0 < cnt < A - 30   # a partial sketch admits some rows, not all


def test_identity_basis_admits_nothing(oracle_mod):
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="identity", r=512, lognormal=False)
    A = wl["A"]
    key, _ = oracle_mod.index_keys(qt[0], x, A)
    sel, theta = oracle_mod.select(key, 40)
    ub = oracle_mod.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A)
    adm, cnt = oracle_mod.admit(ub, sel, theta)
    assert cnt == 0
    assert np.all(ub - key < 1e-6)   # B = 0 up to the rounding margin


def test_zero_basis_bound_is_norm_product(oracle_mod):
    """P = 0: B_h(u) = ||q_lat_h|| * ||c_u||, the config's literal bound."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="zero", r=64)
    A = wl["A"]
    qn = np.linalg.norm(dec(q_lat[0]), axis=1)
    cn = np.linalg.norm(dec(cache[0, :A, :512]), axis=1)
    ub = oracle_mod.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A)
    rope_s = dec(cache[0, :A, 512:]) @ dec(q_rope[0]).T
    want = (rope_s + qn[None, :] * cn[:, None]).max(1)
    assert np.allclose(ub, want, rtol=1e-6) and np.all(ub >= want * (1 - 1e-12) - 1e-9)


def test_sound_bound_admits_almost_everything_on_config3_data(oracle_mod):
    """Context for config 3: with i.i.d. rows the sound Cauchy-Schwarz bound
    admits nearly every archived row (the paper reports the sound trigger
    firing on almost every step)."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="orthonormal", r=64, T=2048, W=32, H=16, needles=2)
    A = wl["A"]
    key, _ = oracle_mod.index_keys(qt[0], x, A)
    sel, theta = oracle_mod.select(key, A // 32)
    ub = oracle_mod.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A)
    adm, cnt = oracle_mod.admit(ub, sel, theta)
    assert cnt > 0.9 * (A - len(sel))


# ------------------------------------------------------------------ attend

def _dense_numpy(q_lat, q_rope, cache_rows, scale):
    """Textbook dense attention in numpy (independent of the oracle's loops)."""
    K = dec(cache_rows)
    Q = np.concatenate([dec(q_lat), dec(q_rope)], axis=1)
    S = scale * (Q @ K.T)
    m = S.max(1, keepdims=True)
    w = np.exp(S - m)
    Z = w.sum(1, keepdims=True)
    return (w @ K[:, :512]) / Z, (m + np.log(Z))[:, 0], S


def test_attend_with_full_budget_equals_dense(oracle_mod):
    H, T = 6, 200
    cache = rand_bf16((T, 576))
    q_lat = rand_bf16((H, 512), 0.2)
    q_rope = rand_bf16((H, 64), 0.2)
    rows = np.arange(T, dtype=np.int32)
    out, lse = oracle_mod.attend(q_lat, q_rope, cache, rows, 0.07)
    o2, l2, _ = _dense_numpy(q_lat, q_rope, cache, 0.07)
    assert np.allclose(out, o2, rtol=1e-10, atol=1e-12) and np.allclose(lse, l2, rtol=1e-12)


def test_attend_single_row_returns_that_row_exactly(oracle_mod):
    cache = rand_bf16((50, 576))
    q_lat = rand_bf16((3, 512))
    q_rope = rand_bf16((3, 64))
    out, lse = oracle_mod.attend(q_lat, q_rope, cache, np.array([17], np.int32), 0.1)
    assert np.array_equal(out, np.repeat(dec(cache[17:18, :512]), 3, 0))
    s = 0.1 * (dec(q_lat) @ dec(cache[17, :512]) + dec(q_rope) @ dec(cache[17, 512:]))
    assert np.allclose(lse, s, rtol=1e-14, atol=1e-14)


def test_attend_zero_query_is_mean_of_values(oracle_mod):
    cache = rand_bf16((64, 576))
    rows = np.array([3, 9, 9, 40, 63], np.int32)
    out, lse = oracle_mod.attend(np.zeros((2, 512), np.uint16), np.zeros((2, 64), np.uint16),
                                 cache, rows, 0.5)
    assert np.allclose(out[0], dec(cache[rows, :512]).mean(0), rtol=1e-13, atol=1e-14)
    assert np.allclose(lse, math.log(5))


def test_attend_is_permutation_invariant_and_multiset(oracle_mod):
    """Lemma (Exchangeability): the output depends only on the multiset."""
    cache = rand_bf16((120, 576))
    q_lat = rand_bf16((4, 512), 0.3)
    q_rope = rand_bf16((4, 64), 0.3)
    rows = rng.choice(120, 60, replace=False).astype(np.int32)
    o1, l1 = oracle_mod.attend(q_lat, q_rope, cache, rows, 0.09)
    o2, l2 = oracle_mod.attend(q_lat, q_rope, cache, rng.permutation(rows).astype(np.int32), 0.09)
    assert np.allclose(o1, o2, rtol=1e-12, atol=1e-14) and np.allclose(l1, l2, rtol=1e-13)
    # a duplicated row counts twice: compare with explicit weights
    dup = np.concatenate([rows, rows[:1]])
    o3, l3 = oracle_mod.attend(q_lat, q_rope, cache, dup, 0.09)
    _, _, S = _dense_numpy(q_lat, q_rope, cache[rows], 0.09)
    w = np.exp(S - S.max(1, keepdims=True))
    w[:, 0] *= 2
    want = (w @ dec(cache[rows, :512])) / w.sum(1, keepdims=True)
    assert np.allclose(o3, want, rtol=1e-10, atol=1e-12)


def test_empty_attended_set(oracle_mod):
    cache = rand_bf16((4, 576))
    out, lse = oracle_mod.attend(rand_bf16((2, 512)), rand_bf16((2, 64)), cache,
                                 np.zeros(0, np.int32), 0.1)
    assert np.all(out == 0) and np.all(np.isneginf(lse))


def test_bounded_leakage_lemma(oracle_mod):
    """Lemma (Bounded leakage), rigorous form for two convex combinations:
    ||o_F - o_all|| <= 2 * (Z_excluded / Z_all) * max ||v||."""
    T, H = 400, 5
    cache = rand_bf16((T, 576))
    q_lat = rand_bf16((H, 512), 0.25)
    q_rope = rand_bf16((H, 64), 0.25)
    o_all, _, S = _dense_numpy(q_lat, q_rope, cache, 0.1)
    for frac in (0.1, 0.5, 0.9):
        F = np.sort(rng.choice(T, int(frac * T), replace=False)).astype(np.int32)
        oF, _ = oracle_mod.attend(q_lat, q_rope, cache, F, 0.1)
        E = np.setdiff1d(np.arange(T), F)
        w = np.exp(S - S.max(1, keepdims=True))
        mass = w[:, E].sum(1) / w.sum(1)
        vmax = np.linalg.norm(dec(cache[:, :512]), axis=1).max()
        gap = np.linalg.norm(oF - o_all, axis=1)
        assert np.all(gap <= 2 * mass * vmax + 1e-12)


def test_oracle_step_dense_when_budget_covers_archive(oracle_mod):
    """The kill-switch identity: with k = A the step attends every row, so it
    reproduces dense attention over the whole cache."""
    cfg = synth.CONFIGS["cfg0"].with_(H=4)
    wl = synth.make_workload(cfg, "cpu", T=512)
    cache = synth.to_numpy_bits(wl["cache"])
    Pb = synth.to_numpy_bits(wl["P"])
    q_lat = synth.to_numpy_bits(wl["q_lat"])
    q_rope = synth.to_numpy_bits(wl["q_rope"])
    index, *_ = oracle_mod.digest_build(cache, Pb, cfg.r, scalars=False)
    res = oracle_mod.step(cache, q_lat, q_rope, index, Pb, cfg.r, cfg.mode, wl["W"], wl["A"],
                          cfg.scale)
    o, l, _ = _dense_numpy(q_lat[0], q_rope[0], cache[0], cfg.scale)
    assert np.allclose(res["out"][0], o, rtol=1e-10, atol=1e-12)
    assert np.allclose(res["lse"][0], l, rtol=1e-12)


# ------------------------------------------------------- read budget (paper)

def test_read_budget_matches_paper_numbers():
    g = json.load(open(os.path.join(GOLDEN, "read_budget.json")))
    rho, r = g["rho"], g["r"]
    assert budget.ROW_BYTES == g["row_bytes"]
    idx = 2 * (64 + r + 1)
    assert abs(idx - g["index_bytes_per_row_r64_16bit_approx"]) <= 3
    lo, hi = g["admitted_fraction_document_decode"]
    for f in (lo, hi):
        b = budget.reads_bytes(rho, r, f)
        assert abs(b - g["bytes_per_token_rho_1_32_r64_approx"]) <= 6
    f_mid = 0.5 * (lo + hi)
    assert round(1152 / budget.reads_bytes(rho, r, f_mid), 1) == g["ratio_vs_dense_16bit_index_approx"]
    assert round(1152 / budget.reads_bytes(rho, r, f_mid, index_elem_bytes=4), 1) == \
        g["ratio_vs_dense_full_precision_index_approx"]
    assert round(rho * 576) == g["attended_dims_per_token_at_32x"]


# ------------------------------------------------ certificate multiplier (z)

def test_cert_mult_scales_only_the_residual_term(oracle_mod):
    """Eq. (trigger): z / sqrt(d_c - r) multiplies the sketch-residual term
    a_h eta_u; the bf16 rounding terms n_h eps_u + e_h gamma_u stay.  Checked
    against exact rationals on a sample of rows, with a'_h the smallest float
    >= cert_mult * a_h."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, r=32, T=200, W=20, H=4)
    A = wl["A"]
    sh = dec(x[:A]) @ dec(qt[0]).T                     # exact: the sums are exact here
    for cm in (0.0, 0.125, 0.3, 1.0):
        ub = oracle_mod.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A,
                                     cert_mult=cm)
        a2 = []
        for h in range(4):
            want = Fraction(cm) * Fraction(float(a[0, h]))
            f = np.float32(float(want))
            if Fraction(float(f)) < want:
                f = np.nextafter(f, np.float32(np.inf))
            a2.append(Fraction(float(f)))
        for u in range(0, A, 17):
            best = max(Fraction(float(sh[u, h])) + a2[h] * Fraction(float(eta[0, u]))
                       + Fraction(float(nq[0, h])) * Fraction(float(eps[0, u]))
                       + Fraction(float(e[0, h])) * Fraction(float(gam[0, u])) for h in range(4))
            assert abs(Fraction(ub[u]) - best) <= abs(best) * Fraction(1, 2 ** 50)


def test_cert_mult_one_is_the_sound_bound_and_admission_is_monotone(oracle_mod):
    """cert_mult = 1 (z = sqrt(d_c - r)) is the default sound bound; smaller
    multipliers admit nested subsets; cert_mult = 0 keeps only the rounding
    slack, so it admits rows whose index score alone nearly beats theta."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="orthonormal", r=64, T=1024, W=32, H=8, needles=4)
    A = wl["A"]
    key, _ = oracle_mod.index_keys(qt[0], x, A)
    sel, theta = oracle_mod.select(key, A // 32)
    args = (qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A)
    ub1 = oracle_mod.upper_bounds(*args)
    assert np.array_equal(ub1, oracle_mod.upper_bounds(*args, cert_mult=1.0))
    prev = None
    for cm in (0.0, 0.05, 0.2, 0.5, 1.0):
        adm, cnt = oracle_mod.admit(oracle_mod.upper_bounds(*args, cert_mult=cm), sel, theta)
        if prev is not None:
            assert set(prev) <= set(adm)
        prev = adm
    adm0, _ = oracle_mod.admit(oracle_mod.upper_bounds(*args, cert_mult=0.0), sel, theta)
    outside = np.setdiff1d(np.arange(A), sel)
    # every row admitted at cert_mult = 0 has its index score within the rounding slack of theta
    slack = (nq[0].max() * eps[0, :A].max() + e[0].max() * gam[0, :A].max()) * 1.001
    assert np.all(key[adm0] > theta - slack)
    assert len(adm0) < len(outside)


# --------------------------------------------------- calibrated trigger (z)

def test_conformal_chain_from_the_recall_target(oracle_mod):
    """tau = 0.90 gives alpha = 0.05, tau_s = 18/19 and min_hard = 18 (Sec. 5.2);
    z is the ceil((n+1) tau_s)-th smallest required inflation, clamped to Z_max."""
    zq = np.arange(1, 19, dtype=np.float64) * 0.25          # 18 hand-made scores 0.25 .. 4.5
    z, mh, k = oracle_mod.conformal_z(zq)
    assert mh == 18 and k == math.ceil(19 * Fraction(18, 19)) == 18 and z == 4.5
    z, mh, k = oracle_mod.conformal_z(zq[:17])              # one short of min_hard: the clamp
    assert (z, k) == (8.0, 0)
    zq = rng.permutation(np.linspace(0.1, 3.7, 37))
    z, _, k = oracle_mod.conformal_z(zq)
    assert k == math.ceil(38 * Fraction(18, 19)) == 36 and z == np.sort(zq)[35]
    z, _, k = oracle_mod.conformal_z(np.full(100, 9.5))      # above Z_max
    assert k == 96 and z == 8.0
    z, _, _ = oracle_mod.conformal_z(np.full(30, -2.0))      # an inflation, never a deflation
    assert z == 0.0
    # another target: tau = 4/5 -> alpha = 1/10, tau_s = 8/9, min_hard = 8
    z, mh, k = oracle_mod.conformal_z(np.arange(8.0), tau=(4, 5))
    assert mh == 8 and k == 8 and z == 7.0


def test_conformal_z_covers_a_fresh_query_at_tau_s(oracle_mod):
    """Exchangeability alone: for i.i.d. required inflations, a fresh hard
    query's z_q <= z with probability >= tau_s (here 18/19, n = 30)."""
    r = np.random.default_rng(99)
    trials, n, hit = 4000, 30, 0
    for _ in range(trials):
        v = r.standard_normal(n + 1) + 2.0
        z, _, k = oracle_mod.conformal_z(v[:n], zmax=1e9)
        hit += v[n] <= z
    # k = ceil(31 * 18/19) = 30 of 30: coverage (k)/(n+1) = 30/31 >= 18/19
    assert hit / trials >= 18 / 19 - 3 * math.sqrt((18 / 19) * (1 / 19) / trials)


def test_row_max_is_exact_with_ties_to_the_lower_row(oracle_mod):
    H, T = 3, 60
    lat = small_int_bf16((T, 512), -2, 2)
    rope = small_int_bf16((T, 64), -2, 2)
    cache = np.concatenate([lat, rope], 1)
    cache[40] = cache[11]                                   # a tie: rows 11 and 40
    ql = small_int_bf16((H, 512), -2, 2)
    qr = small_int_bf16((H, 64), -2, 2)
    rows = np.array([40, 11, 3, 59, 27], np.int32)
    smax, arg = oracle_mod.row_max(ql, qr, cache, rows)
    S = dec(cache[rows]) @ np.concatenate([dec(ql), dec(qr)], 1).T   # exact (small integers)
    for h in range(H):
        best = S[:, h].max()
        assert smax[h] == best
        assert arg[h] == min(int(u) for u, v in zip(rows, S[:, h]) if v == best)
    smax, arg = oracle_mod.row_max(ql, qr, cache, np.zeros(0, np.int32))
    assert np.all(np.isneginf(smax)) and np.all(arg == -1)


def test_trigger_with_one_threshold_is_the_admission_rule(oracle_mod):
    """With s*_h = theta for every head, margin_u > 0 iff UB_u > theta: the
    fired set (uncapped) equals the certified admission bit for bit, at the
    sound multiplier and at a calibrated one."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="orthonormal", r=64, T=900, W=30, H=8, needles=4)
    A = wl["A"]
    key, _ = oracle_mod.index_keys(qt[0], x, A)
    sel, theta = oracle_mod.select(key, 40)
    for cm in (1.0, 0.1):
        ub = oracle_mod.upper_bounds(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A, cert_mult=cm)
        adm, cnt = oracle_mod.admit(ub, sel, theta)
        m = oracle_mod.trigger_margins(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A,
                                       np.full(8, theta), cm)
        fired, fc = oracle_mod.fire(m, sel)
        assert fc == cnt and np.array_equal(fired, adm)


def test_trigger_margins_per_head_and_topj(oracle_mod):
    """margin_u = max_h (UB_h(u) - s*_h) against per-head UB_h from the
    single-head bound; the top-j cap keeps the j largest margins (ties to
    the lower row), ascending."""
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="orthonormal", r=32, T=500, W=20, H=5, needles=3)
    A = wl["A"]
    smax = np.array([30.0, 25.0, 41.0, 10.0, 33.0])
    cm = 0.2
    m = oracle_mod.trigger_margins(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A, smax, cm)
    per = np.stack([oracle_mod.upper_bounds(qt[0, h:h + 1], a[0, h:h + 1], nq[0, h:h + 1], e[0, h:h + 1],
                                            x, eta[0], eps[0], gam[0], A, cert_mult=cm) - smax[h]
                    for h in range(5)], 1)
    assert np.array_equal(m, per.max(1))
    sel = np.sort(rng.choice(A, 12, replace=False)).astype(np.int32)
    fired, cnt = oracle_mod.fire(m, sel)
    want = [u for u in range(A) if u not in set(sel) and m[u] > 0]
    assert cnt == len(want) and list(fired) == want and cnt > 16
    top, tc = oracle_mod.fire(m, sel, topj=16)
    order = sorted(want, key=lambda u: (-m[u], u))[:16]
    assert tc == 16 and list(top) == sorted(order)


def test_required_inflation_is_where_the_target_starts_to_fire(oracle_mod):
    """For a hard (query, head), the trigger with cert_mult = z_q / sqrt(d_c - r)
    (times 1 + 1e-6) fires the causal argmax row for that head, and times
    1 - 1e-6 it does not: z_q is exactly the required inflation."""
    r = 32
    wl, cache, q_lat, q_rope, index, eta, eps, gam, qt, a, nq, e, x = _tiny_two_tier(
        oracle_mod, basis="orthonormal", r=r, T=700, W=20, H=6, needles=0)
    A, T = wl["A"], wl["T"]
    key, _ = oracle_mod.index_keys(qt[0], x, A)
    sel, _ = oracle_mod.select(key, 20)
    tier1 = np.concatenate([sel, np.arange(A, T, dtype=np.int32)])
    s1, _ = oracle_mod.row_max(q_lat[0], q_rope[0], cache[0], tier1)
    _, am = oracle_mod.row_max(q_lat[0], q_rope[0], cache[0], np.arange(T, dtype=np.int32))
    hard, zq = oracle_mod.required_inflation(qt[0], a[0], nq[0], e[0], x, eta[0], eps[0], gam[0], A, sel, r,
                                             s1, am)
    assert hard.sum() >= 3
    for h in np.nonzero(hard)[0]:
        assert am[h] < A and am[h] not in set(sel)
        assert np.isfinite(zq[h])
        u = int(am[h])
        for f, fires in ((1 + 1e-6, True), (1 - 1e-6, False)):
            cm = zq[h] / math.sqrt(512 - r) * f
            if cm < 0:
                continue
            m = oracle_mod.trigger_margins(qt[0, h:h + 1], a[0, h:h + 1], nq[0, h:h + 1], e[0, h:h + 1], x,
                                           eta[0], eps[0], gam[0], A, s1[h:h + 1], cm)
            assert (m[u] > 0) == fires, (h, f, m[u])


# ---------------------------------------------- data-driven sketch basis V_r

def _lowrank_queries(m, rank, noise, seed=5):
    r_ = np.random.default_rng(seed)
    U, _ = np.linalg.qr(r_.standard_normal((512, rank)))
    g = r_.standard_normal((m, rank)) * 3.0
    q = g @ U.T + noise * r_.standard_normal((m, 512))
    return (q.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16), U


def test_sketch_basis_recovers_a_planted_subspace(oracle_mod):
    """Queries in a planted 48-dim subspace plus small noise: the top-48
    eigenvectors span it (principal angles ~ noise / signal), they are
    orthonormal, satisfy C v = lambda v, and the bf16 basis is contractive."""
    q, U = _lowrank_queries(2000, 48, 0.05)
    P, V, w = oracle_mod.sketch_basis(q, 48)
    assert np.allclose(V.T @ V, np.eye(48), atol=1e-12)
    C = oracle_mod.content_second_moment(q)
    assert np.max(np.abs(C @ V - V * w)) < 1e-9 * w[0]
    s = np.linalg.svd(U.T @ V, compute_uv=False)          # cosines of the principal angles
    assert s.min() > 1 - 1e-4
    assert w[47] > 100 * oracle_mod.sketch_basis(q, 49)[2][48]   # the eigengap after the planted rank
    assert oracle_mod.gershgorin(P) < 1.0
    assert np.all(np.abs(dec(P) - oracle_mod.SKETCH_SCALE * V.T) <= 2.0 ** -8 * np.abs(V.T) + 1e-30)


def test_sketch_basis_is_rotation_equivariant_and_shrinks_the_residual(oracle_mod):
    """The subspace does not depend on the order of the queries; on queries
    of the planted subspace the residual ||(I - V V^T) q|| that the
    certificate multiplies (Lemma (Index certificate)) drops to the noise."""
    q, U = _lowrank_queries(1500, 32, 0.02, seed=8)
    P1, V1, _ = oracle_mod.sketch_basis(q, 32)
    P2, V2, _ = oracle_mod.sketch_basis(q[::-1].copy(), 32)
    assert np.allclose(V1 @ V1.T, V2 @ V2.T, atol=1e-10)
    qq = dec(q)
    res = np.linalg.norm(qq - (qq @ V1) @ V1.T, axis=1) / np.linalg.norm(qq, axis=1)
    # the noise outside the subspace: 0.02 sqrt(512 - 32) against a signal of 3 sqrt(32)
    pred = 0.02 * math.sqrt(512 - 32) / (3.0 * math.sqrt(32))
    assert 0.7 * pred < np.median(res) < 1.3 * pred and res.max() < 2.5 * pred
    full = np.linalg.norm(qq - (qq @ np.linalg.qr(np.random.default_rng(1).standard_normal((512, 32)))[0])
                          @ np.linalg.qr(np.random.default_rng(1).standard_normal((512, 32)))[0].T, axis=1)
    assert np.median(full / np.linalg.norm(qq, axis=1)) > 0.9   # a random basis leaves almost all of it


# ------------------------------------------------------- page-box bound

def _wide_bits(shape, lo, hi, seed):
    """bf16 bits of sign * (1 + m/128) * 2^e, e uniform in [lo, hi), with some
    zeros and negative zeros: fp64 sums of their products round often."""
    r = np.random.default_rng(seed)
    m = r.integers(0, 128, shape)
    e = r.integers(lo, hi, shape)
    sg = r.choice([-1.0, 1.0], shape)
    v = (sg * np.ldexp(1.0 + m / 128.0, e)).astype(np.float32)
    z = r.random(shape) < 0.05
    v[z] = np.where(r.random(int(z.sum())) < 0.5, 0.0, -0.0)
    return (v.view(np.uint32) >> 16).astype(np.uint16)


def test_page_box_brackets_and_attains_every_column(oracle_mod):
    """Box of each page (appendix on prior algorithms, page-bound pruning):
    lo <= x_u <= hi for every row of the page, both ends attained by a row,
    the last page ragged, zeros written as +0."""
    A, n, page = 301, 24, 64
    x = _wide_bits((A, n), -10, 10, 1)
    box = oracle_mod.page_box(x, A, page)
    assert box.shape == (5, 2, n)
    xv = dec(x)
    for j in range(5):
        rows = xv[j * page:min(A, (j + 1) * page)]
        lo, hi = dec(box[j, 0]), dec(box[j, 1])
        assert np.array_equal(lo, rows.min(0)) and np.array_equal(hi, rows.max(0))
    assert not np.any(box == 0x8000)


def test_page_bound_is_the_maximum_over_the_box_corners(oracle_mod):
    """The interval bound is max_h of the largest q.v over v in the box, which
    a linear form attains at a corner: brute force over all 2^n corners in
    exact rationals, on small integers (every fp64 sum exact)."""
    n, H, A, page = 6, 5, 40, 8
    q = small_int_bf16((H, n), -6, 6)
    x = small_int_bf16((A, n), -7, 7)
    box = oracle_mod.page_box(x, A, page)
    bound = oracle_mod.page_bound(q, box)
    import itertools
    for j in range(box.shape[0]):
        lo, hi = box[j, 0], box[j, 1]
        best = None
        for corner in itertools.product((0, 1), repeat=n):
            v = [hi[d] if corner[d] else lo[d] for d in range(n)]
            for h in range(H):
                s = exact_dot(q[h], v)
                best = s if best is None or s > best else best
        assert Fraction(bound[j]) == best


def test_page_bound_dominates_every_key_of_its_page(oracle_mod):
    """bound[j] >= key_u for every row u of page j, bit for bit: each term is
    >= the key's term and fp64 rounding is monotone (inputs spread over 2^40,
    so the sums round at many steps)."""
    n, H, A, page = 64, 16, 700, 32
    q = _wide_bits((H, n), -20, 20, 2)
    x = _wide_bits((A, n), -20, 20, 3)
    key, bad = oracle_mod.index_keys(q, x, A, check_exact=True)
    assert bad > 0   # the sums do round: the inequality is not only exact arithmetic
    bound = oracle_mod.page_bound(q, oracle_mod.page_box(x, A, page))
    for j in range(len(bound)):
        assert np.all(key[j * page:min(A, (j + 1) * page)] <= bound[j])


def test_page_bound_with_pages_of_one_row_is_the_key(oracle_mod):
    """A one-row page's box is the row itself: the bound is that row's index
    key bit for bit (same terms, same order)."""
    n, H, A = 40, 8, 90
    q = _wide_bits((H, n), -15, 15, 4)
    x = _wide_bits((A, n), -15, 15, 5)
    key, _ = oracle_mod.index_keys(q, x, A)
    assert np.array_equal(oracle_mod.page_bound(q, oracle_mod.page_box(x, A, 1)), key)


def test_page_bound_of_a_constant_page_and_of_a_zero_query(oracle_mod):
    """A page whose rows are all equal bounds exactly its key; a zero query
    bounds every page by 0."""
    n, H = 32, 4
    q = rand_bf16((H, n))
    row = rand_bf16((1, n))
    x = np.repeat(row, 16, 0)
    key, _ = oracle_mod.index_keys(q, x, 16)
    assert oracle_mod.page_bound(q, oracle_mod.page_box(x, 16, 16))[0] == key[0]
    z = np.zeros((H, n), np.uint16)
    assert np.all(oracle_mod.page_bound(z, oracle_mod.page_box(rand_bf16((100, n)), 100, 10)) == 0.0)

"""fp64 CPU oracle for the VestigeKV decode-time hot path (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never touches it.  It shares no code with the HIP path:
the C source here is compiled on its own with gcc.

Each function names the passage of the paper (arXiv 2609.03949) it follows;
see ``vkvref.c`` for the arithmetic.  Arrays are numpy; bf16 values travel
as ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vkvref.c")
_LIB = os.path.join(_HERE, "libvkvref.so")

D_LAT, D_ROPE, D_ROW = 512, 64, 576
MODE_ROPE, MODE_DIGEST, MODE_ROPE_DIGEST = 1, 2, 3


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
               "-shared", "-Wall", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        i32 = ctypes.c_int
        lib.vkvref_bf16_to_f64.restype = ctypes.c_double
        lib.vkvref_bf16_to_f64.argtypes = [ctypes.c_uint16]
        lib.vkvref_round_bf16.restype = ctypes.c_uint16
        lib.vkvref_round_bf16.argtypes = [ctypes.c_double]
        lib.vkvref_ru_f32.restype = ctypes.c_float
        lib.vkvref_ru_f32.argtypes = [ctypes.c_double]
        lib.vkvref_ru_sqrt_f32.restype = ctypes.c_float
        lib.vkvref_ru_sqrt_f32.argtypes = [ctypes.c_double]
        lib.vkvref_gershgorin.restype = ctypes.c_double
        lib.vkvref_gershgorin.argtypes = [P, i32]
        lib.vkvref_digest_build.restype = i32
        lib.vkvref_digest_build.argtypes = [P, i64, i64, i64, P, i32, i32, P, i64, P, P, P, i32]
        lib.vkvref_query_prep.restype = i32
        lib.vkvref_query_prep.argtypes = [P, P, i64, i64, P, i32, i32, P, P, P, P]
        lib.vkvref_index_keys.restype = i32
        lib.vkvref_index_keys.argtypes = [P, i64, i32, P, i64, i64, P, P, i32]
        lib.vkvref_select.restype = i32
        lib.vkvref_select.argtypes = [P, i64, i64, P, P]
        lib.vkvref_upper_bounds.restype = i32
        lib.vkvref_upper_bounds.argtypes = [P, i64, i32, P, P, P, P, i64, P, P, P, i64, ctypes.c_double, P,
                                               i32]
        lib.vkvref_admit.restype = i64
        lib.vkvref_admit.argtypes = [P, i64, P, i64, ctypes.c_double, P, i64]
        lib.vkvref_attend.restype = i32
        lib.vkvref_attend.argtypes = [P, P, i64, P, i64, P, i64, ctypes.c_double, P, P, i32]
        lib.vkvref_full_scores.restype = i32
        lib.vkvref_full_scores.argtypes = [P, P, i64, P, i64, i64, P, i32]
        lib.vkvref_conformal_z.restype = i32
        lib.vkvref_conformal_z.argtypes = [P, i64, i64, i64, ctypes.c_double, P, P, P]
        lib.vkvref_row_max.restype = i32
        lib.vkvref_row_max.argtypes = [P, P, i64, P, i64, P, i64, P, P]
        lib.vkvref_trigger_margins.restype = i32
        lib.vkvref_trigger_margins.argtypes = [P, i64, i32, P, P, P, P, i64, P, P, P, i64, ctypes.c_double,
                                               P, P, i32]
        lib.vkvref_fire.restype = i64
        lib.vkvref_fire.argtypes = [P, i64, P, i64, i64, P, i64]
        lib.vkvref_required_inflation.restype = i32
        lib.vkvref_required_inflation.argtypes = [P, i64, i32, P, P, P, P, i64, P, P, P, i64, P, i64, i32, P,
                                                  P, P, P]
        lib.vkvref_page_box.restype = i32
        lib.vkvref_page_box.argtypes = [P, i64, i32, i64, i64, P]
        lib.vkvref_page_bound.restype = i32
        lib.vkvref_page_bound.argtypes = [P, i64, i32, P, i64, P]
        lib.vkvref_max_threads.restype = i32
        lib.vkvref_max_threads.argtypes = []
        _lib = lib
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        a = a.view(np.uint16) if a.dtype.itemsize == 2 else a.astype(np.uint16)
    return a


def max_threads() -> int:
    return int(_load().vkvref_max_threads())


# --------------------------------------------------------------- scalar helpers

def bf16_to_f64(bits: int) -> float:
    return float(_load().vkvref_bf16_to_f64(int(bits)))


def round_bf16(x: float) -> int:
    """fp64 -> bf16 bits, one round-to-nearest-even."""
    return int(_load().vkvref_round_bf16(float(x)))


def ru_f32(x: float) -> float:
    return float(_load().vkvref_ru_f32(float(x)))


def ru_sqrt_f32(x: float) -> float:
    return float(_load().vkvref_ru_sqrt_f32(float(x)))


def decode_bf16(a: np.ndarray) -> np.ndarray:
    """bf16 bits -> fp64 values (exact)."""
    a = _u16(a)
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# --------------------------------------------------------------- basis checks

def gershgorin(P: np.ndarray) -> float:
    """max_j sum_k |(P P^T)_jk| in fp64 -- an upper bound of ||P||_2^2."""
    P = _u16(P)
    return float(_load().vkvref_gershgorin(_ptr(P), int(P.shape[0])))


# --------------------------------------------------------------- the path

def digest_build(cache: np.ndarray, P: np.ndarray | None, r: int, with_rope: bool = True,
                 scalars: bool = True, nthreads: int = 0):
    """Index build over every row of cache [B, T, 576] (Sec. 4.2, index entry).

    Returns (index [B,T,n] uint16, eta, eps, gamma [B,T] float32 or None)."""
    cache = _u16(cache)
    B, T, stride = cache.shape
    if P is None or r == 0:
        P = np.zeros((1, D_LAT), np.uint16)
        r = 0
    P = _u16(P)
    n = (D_ROPE if with_rope else 0) + r
    index = np.zeros((B, T, max(n, 1)), np.uint16)
    eta = eps = gam = None
    if scalars:
        eta = np.zeros((B, T), np.float32)
        eps = np.zeros((B, T), np.float32)
        gam = np.zeros((B, T), np.float32)
    _load().vkvref_digest_build(_ptr(cache), B, T, stride, _ptr(P), int(r), int(with_rope),
                                _ptr(index), index.shape[2], _ptr(eta), _ptr(eps), _ptr(gam),
                                int(nthreads))
    return index[:, :, :n], eta, eps, gam


def query_prep(q_lat: np.ndarray, q_rope: np.ndarray, P: np.ndarray | None, r: int, mode: int):
    """Index-space queries qt [B,H,n] and head scalars (a, n, e) [B,H]."""
    q_lat = _u16(q_lat)
    q_rope = _u16(q_rope)
    B, H, _ = q_lat.shape
    if P is None or r == 0:
        P = np.zeros((1, D_LAT), np.uint16)
        r = 0
    P = _u16(P)
    n = (D_ROPE if mode & 1 else 0) + (r if mode & 2 else 0)
    qt = np.zeros((B, H, max(n, 1)), np.uint16)
    a = np.zeros((B, H), np.float32)
    nq = np.zeros((B, H), np.float32)
    e = np.zeros((B, H), np.float32)
    _load().vkvref_query_prep(_ptr(q_lat), _ptr(q_rope), B, H, _ptr(P), int(r), int(mode),
                              _ptr(qt), _ptr(a), _ptr(nq), _ptr(e))
    return qt[:, :, :n].copy(), a, nq, e


def index_rows(cache_seq: np.ndarray, index_seq: np.ndarray | None, mode: int, r: int,
               index_has_rope: bool = True) -> np.ndarray:
    """The index vectors x_u [T, n] scored for one sequence, per mode."""
    if mode == MODE_ROPE:
        if index_seq is not None and index_has_rope:
            return np.ascontiguousarray(_u16(index_seq)[:, :D_ROPE])
        return np.ascontiguousarray(_u16(cache_seq)[:, D_LAT:D_ROW])
    off = D_ROPE if index_has_rope else 0
    dig = _u16(index_seq)[:, off:off + r]
    if mode == MODE_DIGEST:
        return np.ascontiguousarray(dig)
    rope = _u16(cache_seq)[:, D_LAT:D_ROW] if not index_has_rope else _u16(index_seq)[:, :D_ROPE]
    return np.ascontiguousarray(np.concatenate([rope, dig], axis=1))


def index_keys(qt_seq: np.ndarray, x: np.ndarray, A: int, check_exact: bool = False,
               nthreads: int = 0):
    """key_u = max_h qt_h . x_u for u in [0, A), fp64 (Eq. (trigger), first two terms).

    Returns (key [A] float64, number of inexact (u,h) sums or None)."""
    qt_seq = _u16(qt_seq)
    x = _u16(x)
    H, n = qt_seq.shape
    key = np.zeros(max(A, 1), np.float64)
    bad = ctypes.c_int64(0)
    _load().vkvref_index_keys(_ptr(qt_seq), H, n, _ptr(x), x.shape[1], int(A), _ptr(key),
                              ctypes.addressof(bad) if check_exact else None, int(nthreads))
    return key[:A], (int(bad.value) if check_exact else None)


def page_box(x: np.ndarray, A: int, page: int) -> np.ndarray:
    """Per-page column ranges of the index rows [0, A): [npages, 2, n] bf16 bits
    (lo, hi), pages of `page` rows (appendix on prior algorithms, page-bound
    pruning)."""
    x = _u16(x)
    n = x.shape[1]
    npg = (A + page - 1) // page
    box = np.zeros((max(npg, 1), 2, n), np.uint16)
    _load().vkvref_page_box(_ptr(x), x.shape[1], n, int(A), int(page), _ptr(box))
    return box[:npg]


def page_bound(qt_seq: np.ndarray, box: np.ndarray) -> np.ndarray:
    """bound[j] = max_h sum_d max(qt_hd lo_d, qt_hd hi_d), fp64, d ascending (the
    page-bound equation of the appendix on prior algorithms); >= the index key
    of every row of page j."""
    qt_seq = _u16(qt_seq)
    box = np.ascontiguousarray(_u16(box))
    H, n = qt_seq.shape
    npg = box.shape[0]
    out = np.zeros(max(npg, 1), np.float64)
    _load().vkvref_page_bound(_ptr(qt_seq), H, n, _ptr(box), int(npg), _ptr(out))
    return out[:npg]


def select(key: np.ndarray, k: int):
    """Top-k of [0, A) by (key desc, index asc), ascending; theta = min key in S."""
    key = np.ascontiguousarray(key, np.float64)
    A = key.shape[0]
    sel = np.zeros(max(k, 1), np.int32)
    theta = ctypes.c_double(0.0)
    rc = _load().vkvref_select(_ptr(key) if A else None, A, int(k), _ptr(sel),
                               ctypes.addressof(theta))
    if rc != 0:
        raise ValueError("k out of range")
    return sel[:k].copy(), float(theta.value)


def upper_bounds(qt_seq, a, nq, e, x, eta, eps, gam, A: int, nthreads: int = 0,
                 cert_mult: float = 1.0) -> np.ndarray:
    """UB_u = max_h (s^_h(u) + B_h(u)), fp64 (Lemma (Index certificate)).

    cert_mult = z / sqrt(d_c - r) of Eq. (trigger) scales the sketch-residual
    term a_h eta_u (1 = the sound bound)."""
    qt_seq = _u16(qt_seq)
    x = _u16(x)
    H, n = qt_seq.shape
    f = lambda v: np.ascontiguousarray(v, np.float32)
    a, nq, e, eta, eps, gam = map(f, (a, nq, e, eta, eps, gam))
    ub = np.zeros(max(A, 1), np.float64)
    _load().vkvref_upper_bounds(_ptr(qt_seq), H, n, _ptr(a), _ptr(nq), _ptr(e), _ptr(x),
                                x.shape[1], _ptr(eta), _ptr(eps), _ptr(gam), int(A),
                                float(cert_mult), _ptr(ub), int(nthreads))
    return ub[:A]


def admit(ub: np.ndarray, sel: np.ndarray, theta: float, cap: int | None = None):
    """Rows of [0, A) outside S with UB > theta, ascending; returns (adm, count)."""
    ub = np.ascontiguousarray(ub, np.float64)
    sel = np.ascontiguousarray(sel, np.int32)
    A = ub.shape[0]
    if cap is None:
        cap = A
    adm = np.zeros(max(cap, 1), np.int32)
    cnt = _load().vkvref_admit(_ptr(ub) if A else None, A, _ptr(sel) if sel.size else None,
                               sel.shape[0], float(theta), _ptr(adm), int(cap))
    return adm[:min(cnt, cap)].copy(), int(cnt)


# ------------------------------------------------------- calibrated trigger

def conformal_z(zq, tau=(9, 10), zmax: float = 8.0):
    """z from the required inflations of the hard calibration queries (Sec. 4.2,
    the z paragraph; the closed-form chain of Sec. 5.2).  tau is a rational
    (numerator, denominator).  Returns (z, min_hard, k) with k = 0 when z is
    the Z_max clamp."""
    zq = np.ascontiguousarray(zq, np.float64)
    z = ctypes.c_double(0.0)
    mh = ctypes.c_int64(0)
    k = ctypes.c_int64(0)
    rc = _load().vkvref_conformal_z(_ptr(zq) if zq.size else None, zq.size, int(tau[0]), int(tau[1]),
                                    float(zmax), ctypes.addressof(z), ctypes.addressof(mh),
                                    ctypes.addressof(k))
    if rc != 0:
        raise ValueError("tau must be a rational in (0, 1)")
    return float(z.value), int(mh.value), int(k.value)


def row_max(q_lat_seq, q_rope_seq, cache_seq, rows):
    """Per head: (max exact full score over ``rows``, the row attaining it,
    lower index on ties) -- the tier-1 max logit s*_h of Sec. 4.2."""
    q_lat_seq = _u16(q_lat_seq)
    q_rope_seq = _u16(q_rope_seq)
    cache_seq = _u16(cache_seq)
    rows = np.ascontiguousarray(rows, np.int32)
    H = q_lat_seq.shape[0]
    smax = np.zeros(H, np.float64)
    arg = np.zeros(H, np.int32)
    _load().vkvref_row_max(_ptr(q_lat_seq), _ptr(q_rope_seq), H, _ptr(cache_seq), cache_seq.shape[1],
                           _ptr(rows) if rows.size else None, rows.size, _ptr(smax), _ptr(arg))
    return smax, arg


def trigger_margins(qt_seq, a, nq, e, x, eta, eps, gam, A: int, smax, cert_mult: float,
                    nthreads: int = 0) -> np.ndarray:
    """margin_u = max_h (UB_h(u) - s*_h) over the archived rows (Eq. (trigger)
    against the per-head tier-1 maximum)."""
    qt_seq = _u16(qt_seq)
    x = _u16(x)
    H, n = qt_seq.shape
    f = lambda v: np.ascontiguousarray(v, np.float32)
    a, nq, e, eta, eps, gam = map(f, (a, nq, e, eta, eps, gam))
    smax = np.ascontiguousarray(smax, np.float64)
    m = np.zeros(max(A, 1), np.float64)
    _load().vkvref_trigger_margins(_ptr(qt_seq), H, n, _ptr(a), _ptr(nq), _ptr(e), _ptr(x), x.shape[1],
                                   _ptr(eta), _ptr(eps), _ptr(gam), int(A), float(cert_mult), _ptr(smax),
                                   _ptr(m), int(nthreads))
    return m[:A]


def fire(margin, sel, topj: int = 0, cap: int | None = None):
    """The fired rows (outside S, margin > 0), ascending, capped to the topj
    largest margins when topj > 0.  Returns (rows, count)."""
    margin = np.ascontiguousarray(margin, np.float64)
    sel = np.ascontiguousarray(sel, np.int32)
    A = margin.shape[0]
    if cap is None:
        cap = A
    out = np.zeros(max(cap, 1), np.int32)
    cnt = _load().vkvref_fire(_ptr(margin) if A else None, A, _ptr(sel) if sel.size else None, sel.size,
                              int(topj), _ptr(out), int(cap))
    return out[:min(cnt, cap)].copy(), int(cnt)


def required_inflation(qt_seq, a, nq, e, x, eta, eps, gam, A: int, sel, r: int, tier1_max, argmax):
    """Per head: (hard flag, z_q) of one calibration query (Sec. 4.2)."""
    qt_seq = _u16(qt_seq)
    x = _u16(x)
    H, n = qt_seq.shape
    f = lambda v: np.ascontiguousarray(v, np.float32)
    a, nq, e, eta, eps, gam = map(f, (a, nq, e, eta, eps, gam))
    sel = np.ascontiguousarray(sel, np.int32)
    t1 = np.ascontiguousarray(tier1_max, np.float64)
    am = np.ascontiguousarray(argmax, np.int32)
    hard = np.zeros(H, np.int32)
    zq = np.zeros(H, np.float64)
    _load().vkvref_required_inflation(_ptr(qt_seq), H, n, _ptr(a), _ptr(nq), _ptr(e), _ptr(x), x.shape[1],
                                      _ptr(eta), _ptr(eps), _ptr(gam), int(A),
                                      _ptr(sel) if sel.size else None, sel.size, int(r), _ptr(t1),
                                      _ptr(am), _ptr(hard), _ptr(zq))
    return hard.astype(bool), zq


def attend(q_lat_seq, q_rope_seq, cache_seq, rows, scale: float, nthreads: int = 0):
    """Exact softmax attention of all heads over cache rows ``rows`` (Eq. (setup)).

    Returns (out [H,512] float64, lse [H] float64)."""
    q_lat_seq = _u16(q_lat_seq)
    q_rope_seq = _u16(q_rope_seq)
    cache_seq = _u16(cache_seq)
    rows = np.ascontiguousarray(rows, np.int32)
    H = q_lat_seq.shape[0]
    out = np.zeros((H, D_LAT), np.float64)
    lse = np.zeros(H, np.float64)
    _load().vkvref_attend(_ptr(q_lat_seq), _ptr(q_rope_seq), H, _ptr(cache_seq),
                          cache_seq.shape[1], _ptr(rows) if rows.size else None, rows.shape[0],
                          float(scale), _ptr(out), _ptr(lse), int(nthreads))
    return out, lse


def full_scores(q_lat_seq, q_rope_seq, cache_seq, A: int, nthreads: int = 0) -> np.ndarray:
    """Unscaled full 576-dim scores s_h(u) [A, H] of archived rows (fp64)."""
    q_lat_seq = _u16(q_lat_seq)
    q_rope_seq = _u16(q_rope_seq)
    cache_seq = _u16(cache_seq)
    H = q_lat_seq.shape[0]
    s = np.zeros((max(A, 1), H), np.float64)
    _load().vkvref_full_scores(_ptr(q_lat_seq), _ptr(q_rope_seq), H, _ptr(cache_seq),
                               cache_seq.shape[1], int(A), _ptr(s), int(nthreads))
    return s[:A]


def attend_list(k_sel: np.ndarray, A: int, T: int, adm: np.ndarray | None = None) -> np.ndarray:
    """The attended multiset of one sequence: S, then the recent window [A, T),
    then the admitted rows (Sec. 4.2 figure: kept/recent tier plus fetched rows)."""
    parts = [np.asarray(k_sel, np.int32), np.arange(A, T, dtype=np.int32)]
    if adm is not None:
        parts.append(np.asarray(adm, np.int32))
    return np.concatenate(parts)


def step(cache, q_lat, q_rope, index, P, r: int, mode: int, W: int, k: int, scale: float,
         two_tier: bool = False, eta=None, eps=None, gam=None, cap=None, seqs=None,
         index_has_rope: bool = True, nthreads: int = 0, cert_mult: float = 1.0):
    """One whole decode step on the oracle for the sequences ``seqs``:
    keys -> top-k -> [bound + admission] -> attention.

    Returns a dict of per-sequence results."""
    cache = _u16(cache)
    B, T, _ = cache.shape
    A = T - W
    qt, a, nq, e = query_prep(q_lat, q_rope, P, r, mode)
    res = {"sel": {}, "theta": {}, "adm": {}, "adm_count": {}, "out": {}, "lse": {}, "key": {}}
    for b in (range(B) if seqs is None else seqs):
        x = index_rows(cache[b], None if index is None else index[b], mode, r, index_has_rope)
        key, _ = index_keys(qt[b], x, A, nthreads=nthreads)
        sel, theta = select(key, k)
        adm = None
        if two_tier:
            ub = upper_bounds(qt[b], a[b], nq[b], e[b], x, eta[b], eps[b], gam[b], A, nthreads,
                              cert_mult)
            adm, cnt = admit(ub, sel, theta, cap)
            res["adm"][b] = adm
            res["adm_count"][b] = cnt
        rows = attend_list(sel, A, T, adm)
        out, lse = attend(q_lat[b], q_rope[b], cache[b], rows, scale, nthreads)
        res["sel"][b] = sel
        res["theta"][b] = theta
        res["out"][b] = out
        res["lse"][b] = lse
        res["key"][b] = key
    return res


def step_trigger(cache, q_lat, q_rope, index, P, r: int, mode: int, W: int, k: int, scale: float,
                 eta, eps, gam, cert_mult: float, topj: int = 0, seqs=None, index_has_rope: bool = True,
                 nthreads: int = 0):
    """One decode step with the calibrated trigger (Sec. 4.2): keys -> top-k ->
    s*_h over S and the recent window -> fired rows (some head's bound above
    its threshold; top-j cap) -> attention over S, the window and the fired
    rows.  Returns per-sequence results."""
    cache = _u16(cache)
    B, T, _ = cache.shape
    A = T - W
    qt, a, nq, e = query_prep(q_lat, q_rope, P, r, mode)
    res = {key: {} for key in ("sel", "theta", "smax", "argmax", "fired", "fired_count", "out", "lse",
                               "margin")}
    for b in (range(B) if seqs is None else seqs):
        x = index_rows(cache[b], None if index is None else index[b], mode, r, index_has_rope)
        key, _ = index_keys(qt[b], x, A, nthreads=nthreads)
        sel, theta = select(key, k)
        tier1 = np.concatenate([sel, np.arange(A, T, dtype=np.int32)])
        smax, arg = row_max(q_lat[b], q_rope[b], cache[b], tier1)
        m = trigger_margins(qt[b], a[b], nq[b], e[b], x, eta[b], eps[b], gam[b], A, smax, cert_mult, nthreads)
        fired, cnt = fire(m, sel, topj)
        rows = attend_list(sel, A, T, fired)
        out, lse = attend(q_lat[b], q_rope[b], cache[b], rows, scale, nthreads)
        for name, v in (("sel", sel), ("theta", theta), ("smax", smax), ("argmax", arg), ("fired", fired),
                        ("fired_count", cnt), ("out", out), ("lse", lse), ("margin", m)):
            res[name][b] = v
    return res


# --------------------------------------------------- data-driven sketch basis

SKETCH_SCALE = 1.0 - 2.0 ** -6   # keeps the bf16-rounded basis contractive


def content_second_moment(q: np.ndarray) -> np.ndarray:
    """C = sum_i q_i q_i^T over the prefix content queries q [m, 512] (bf16
    bits; fp64, a library matmul of the exact values)."""
    v = decode_bf16(_u16(q)).reshape(-1, D_LAT)
    return v.T @ v


def sketch_basis(q: np.ndarray, r: int):
    """V_r = the top-r eigenvectors of the prefix content queries' second
    moment (Sec. 4.2, the index entry: V_r from the context's own prefix
    queries), as the digest basis P = RNE_bf16(SKETCH_SCALE * V_r^T) [r, 512].
    Returns (P bits, V_r [512, r] fp64, eigenvalues [r] descending)."""
    C = content_second_moment(q)
    w, V = np.linalg.eigh(C)                 # ascending
    order = np.argsort(-w, kind="stable")[:r]
    V = V[:, order]
    w = w[order]
    # sign: the largest-magnitude component of each eigenvector positive
    idx = np.argmax(np.abs(V), axis=0)
    V = V * np.sign(V[idx, np.arange(r)])
    P = np.vectorize(round_bf16, otypes=[np.uint16])(SKETCH_SCALE * V.T)
    return P, V, w


# ----------------------------------------- query-independent tier-1 selector

SIGMA_BLOCK = 4096    # the close granularity: sigma is computed per fixed block of rows
SIGMA_SINKS = 4       # the first rows of the context, always attended


def lowpass_residual_norm(branch: np.ndarray, kappa: int) -> np.ndarray:
    """sigma_u over one closed block (Sec. 4.1, the sigma equation).

    branch [N, 64]: the 64-dim branch r_u of the block's rows as the cache
    stores it (the trailing 64 dims of each row; bf16 bits).  Along the sequence axis, per channel: the real DFT, bins
    f in [0, kappa) kept and the rest zeroed, the inverse real DFT; sigma_u is
    the norm over the channels of what that low-pass reconstruction misses at
    row u.  Written as the DFT sums (fp64, the twiddle angle reduced mod N):
      X_f = sum_t x_t exp(-2 pi i f t / N),
      L_t = (1/N) [X_0 + 2 sum_{0<f<kappa} Re(X_f exp(2 pi i f t / N))],
    the inverse real transform of the kept half spectrum (each kept bin
    f > 0 stands for its mirror N - f as well).  kappa in [1, N/2]."""
    x = decode_bf16(_u16(branch)).reshape(-1, D_ROPE)
    N = x.shape[0]
    if not 1 <= kappa <= N // 2:
        raise ValueError("kappa must lie in [1, N/2]")
    t = np.arange(N, dtype=np.int64)
    f = np.arange(kappa, dtype=np.int64)
    ang = 2.0 * np.pi * ((f[:, None] * t[None, :]) % N) / N        # [kappa, N]
    c, s = np.cos(ang), np.sin(ang)
    re = c @ x                                                      # Re X_f
    im = -(s @ x)                                                   # Im X_f
    w = np.full(kappa, 2.0)
    w[0] = 1.0
    L = (c.T @ (w[:, None] * re) - s.T @ (w[:, None] * im)) / N     # [N, 64]
    return np.sqrt(np.sum((x - L) ** 2, axis=1))


def sigma_close(cache_seq: np.ndarray, n_closed: int, kappa: int, block: int = SIGMA_BLOCK) -> np.ndarray:
    """sigma for the rows [0, n_closed) of one sequence, block by block (each
    closed block of ``block`` rows is transformed on its own, App. H, block
    close).  n_closed is a multiple of ``block``."""
    cache_seq = _u16(cache_seq)
    if n_closed % block:
        raise ValueError("n_closed must be a multiple of the block")
    out = np.zeros(n_closed)
    for b0 in range(0, n_closed, block):
        out[b0:b0 + block] = lowpass_residual_norm(cache_seq[b0:b0 + block, D_LAT:], kappa)
    return out


def _sigma_order(sigma: np.ndarray, rows: np.ndarray) -> np.ndarray:
    """rows ordered by (sigma desc, row asc) -- the strict total order of the selection."""
    return rows[np.lexsort((rows, -sigma[rows]))]


def sigma_select(sigma: np.ndarray, m: int, nsink: int = SIGMA_SINKS) -> np.ndarray:
    """The sigma tier of the closed rows (Sec. 4.1): the nsink first rows plus
    the sigma-top-m of the other closed rows (sigma desc, lower row first on
    ties), ascending int32.  m larger than the rows on offer keeps them all."""
    n = len(sigma)
    sinks = np.arange(min(nsink, n))
    rest = np.arange(min(nsink, n), n)
    top = _sigma_order(sigma, rest)[:m]
    return np.sort(np.concatenate([sinks, top])).astype(np.int32)


def sigma_select_incremental(sigma: np.ndarray, m: int, nsink: int = SIGMA_SINKS,
                             block: int = SIGMA_BLOCK) -> list[np.ndarray]:
    """The same tier maintained as blocks close (Corollary (Ranking
    stationarity)): after each close the kept set is the top-m of the
    previous kept set together with the new block's rows; decisions are never
    revisited.  Returns the tier after every close."""
    n = len(sigma)
    kept = np.zeros(0, np.int64)
    tiers = []
    for b0 in range(0, n, block):
        new = np.arange(max(b0, nsink), min(b0 + block, n))
        kept = _sigma_order(sigma, np.concatenate([kept, new]))[:m]
        sinks = np.arange(min(nsink, b0 + block, n))
        tiers.append(np.sort(np.concatenate([sinks, kept])).astype(np.int32))
    return tiers


def step_kept(cache, q_lat, q_rope, index, P, r: int, mode: int, W: int, kept, scale: float,
              eta, eps, gam, cert_mult: float, topj: int = 0, seqs=None, index_has_rope: bool = True,
              nthreads: int = 0):
    """One decode step on a given tier-1 set (App. H, per decode step): the
    kept rows ``kept[b]`` of the archive [0, A) (for instance the sigma tier)
    plus the recent window are attended; s*_h is their exact maximum logit;
    archived rows outside the kept set fire when some head's bound exceeds
    it (top-j cap); attention runs over kept, window and fired rows."""
    cache = _u16(cache)
    B, T, _ = cache.shape
    A = T - W
    qt, a, nq, e = query_prep(q_lat, q_rope, P, r, mode)
    res = {key: {} for key in ("smax", "argmax", "fired", "fired_count", "out", "lse", "margin")}
    for b in (range(B) if seqs is None else seqs):
        sel = np.asarray(kept[b], np.int32)
        x = index_rows(cache[b], None if index is None else index[b], mode, r, index_has_rope)
        tier1 = np.concatenate([sel, np.arange(A, T, dtype=np.int32)])
        smax, arg = row_max(q_lat[b], q_rope[b], cache[b], tier1)
        m = trigger_margins(qt[b], a[b], nq[b], e[b], x, eta[b], eps[b], gam[b], A, smax, cert_mult, nthreads)
        fired, cnt = fire(m, sel, topj)
        rows = attend_list(sel, A, T, fired)
        out, lse = attend(q_lat[b], q_rope[b], cache[b], rows, scale, nthreads)
        for name, v in (("smax", smax), ("argmax", arg), ("fired", fired), ("fired_count", cnt), ("out", out),
                        ("lse", lse), ("margin", m)):
            res[name][b] = v
    return res

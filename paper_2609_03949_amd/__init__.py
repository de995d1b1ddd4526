"""Python binding of libvkv (the VestigeKV decode-time hot path on MI355X).

Argument marshalling only: every step of the path runs in the HIP kernels of
``libvkv.so`` behind the C ABI declared in ``include/vkv.h``.  torch provides
device memory and the current stream.  There is no fallback: if the library is
missing or a call fails, an exception is raised.

Names follow the C ABI: ``digest_build``, ``workspace_size``, ``score``,
``select``, ``admit``, ``attend``, ``step_run``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch  # noqa: F401  (loads the HIP runtime the library binds to)

__all__ = [
    "VKV_MODE_ROPE", "VKV_MODE_DIGEST", "VKV_MODE_ROPE_DIGEST", "VkvError", "Context", "Step",
    "lib_path", "load", "digest_build", "workspace_size", "query_prep", "score", "select", "admit", "attend",
    "step_run", "step_run_static", "check_rows", "row_max", "trigger", "required_inflation", "conformal_z",
    "step_run_trigger", "sketch_workspace_size", "sketch_basis", "sigma_workspace_size", "sigma_close",
    "sigma_tier_size", "sigma_select", "step_run_kept", "pack_rows", "page_box", "page_bound", "SIGMA_BLOCK",
    "exported_symbols",
]

VKV_MODE_ROPE, VKV_MODE_DIGEST, VKV_MODE_ROPE_DIGEST = 1, 2, 3
D_LAT, D_ROPE, D_ROW = 512, 64, 576

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libvkv.so")

exported_symbols = (
    "vkv_create", "vkv_destroy", "vkv_status_string", "vkv_last_error", "vkv_version",
    "vkv_digest_build", "vkv_workspace_size", "vkv_query_prep", "vkv_score", "vkv_select", "vkv_admit",
    "vkv_attend", "vkv_step_run", "vkv_step_run_static", "vkv_check_rows", "vkv_set_timing", "vkv_score_timing",
    "vkv_row_max", "vkv_trigger", "vkv_required_inflation", "vkv_conformal_z", "vkv_step_run_trigger",
    "vkv_sketch_workspace_size", "vkv_sketch_basis", "vkv_sigma_workspace_size", "vkv_sigma_close",
    "vkv_sigma_select", "vkv_step_run_kept", "vkv_pack_rows", "vkv_page_box", "vkv_page_bound",
)
SIGMA_BLOCK = 4096


class VkvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libvkv error {code}: {msg}")
        self.code = code


class _Step(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int64), ("H", ctypes.c_int64), ("T", ctypes.c_int64), ("W", ctypes.c_int64),
        ("mode", ctypes.c_int32), ("r", ctypes.c_int32),
        ("q_lat", ctypes.c_void_p), ("q_rope", ctypes.c_void_p),
        ("cache", ctypes.c_void_p), ("cache_row_stride", ctypes.c_int64),
        ("cache_batch_stride", ctypes.c_int64),
        ("index", ctypes.c_void_p), ("index_row_stride", ctypes.c_int64),
        ("index_batch_stride", ctypes.c_int64), ("index_has_rope", ctypes.c_int32),
        ("reserved0", ctypes.c_int32),
        ("P", ctypes.c_void_p), ("eta", ctypes.c_void_p), ("eps", ctypes.c_void_p),
        ("gam", ctypes.c_void_p),
    ]


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def load():
    """Load libvkv.so (built by ``__graft_entry__.build()``); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"libvkv.so not built ({_LIB_PATH}); run __graft_entry__.build()")
    lib = ctypes.CDLL(_LIB_PATH)
    P, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    sp = ctypes.POINTER(_Step)
    lib.vkv_create.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]
    lib.vkv_destroy.argtypes = [P]
    lib.vkv_status_string.restype = ctypes.c_char_p
    lib.vkv_status_string.argtypes = [ctypes.c_int]
    lib.vkv_last_error.restype = ctypes.c_char_p
    lib.vkv_last_error.argtypes = [P]
    lib.vkv_version.argtypes = []
    lib.vkv_digest_build.argtypes = [P, P, i64, i64, i64, i64, P, i32, i32, P, i64, i64, P, P, P, P]
    lib.vkv_workspace_size.argtypes = [sp, i64, i64, ctypes.POINTER(ctypes.c_size_t)]
    lib.vkv_query_prep.argtypes = [P, sp, P, ctypes.c_size_t, P]
    f32 = ctypes.c_float
    lib.vkv_score.argtypes = [P, sp, P, ctypes.c_size_t, P, P, f32, P]
    lib.vkv_select.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P]
    lib.vkv_admit.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P, f32, P, P, i64, P]
    lib.vkv_attend.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P, i64, ctypes.c_float, P, P, P]
    lib.vkv_step_run.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P, P, P, P, i64,
                                 f32, f32, P, P, P]
    lib.vkv_check_rows.argtypes = [P, sp, i64, P, P, P, i64, P]
    lib.vkv_step_run_static.argtypes = [P, sp, i64, P, P, P, P, P, P, i64, f32, f32, P, P, P]
    lib.vkv_row_max.argtypes = [P, sp, P, i64, i32, P, P, P]
    lib.vkv_trigger.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, f32, P, i64, P, P, i64, P]
    lib.vkv_required_inflation.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P, P, P, P]
    lib.vkv_conformal_z.argtypes = [P, i64, i64, i64, ctypes.c_double, P, P, P]
    lib.vkv_step_run_trigger.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P, P, f32, P, P, i64, P, P, i64,
                                         f32, P, P, P]
    lib.vkv_sketch_workspace_size.argtypes = [i32, ctypes.POINTER(ctypes.c_size_t)]
    lib.vkv_sketch_basis.argtypes = [P, P, i64, i32, i32, P, ctypes.c_size_t, P, P, P]
    lib.vkv_sigma_workspace_size.argtypes = [i64, i64, ctypes.POINTER(ctypes.c_size_t)]
    lib.vkv_sigma_close.argtypes = [P, P, i64, i64, i64, i64, i64, i64, i32, P, ctypes.c_size_t, P, i64, P]
    lib.vkv_sigma_select.argtypes = [P, P, i64, i64, i64, i64, i32, P, P]
    lib.vkv_step_run_kept.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P, f32, P, P, i64, P, P, i64,
                                      ctypes.c_float, P, P, P]
    lib.vkv_pack_rows.argtypes = [P, P, P, i64, i64, P, P, P]
    lib.vkv_page_box.argtypes = [P, sp, i64, P, P]
    lib.vkv_page_bound.argtypes = [P, sp, P, ctypes.c_size_t, i64, P, P, P]
    lib.vkv_set_timing.argtypes = [P, ctypes.c_int]
    lib.vkv_score_timing.argtypes = [P, ctypes.POINTER(ctypes.c_float), ctypes.c_int]
    for name in exported_symbols:
        getattr(lib, name).restype = getattr(lib, name).restype or ctypes.c_int
    for name in ("vkv_create", "vkv_destroy", "vkv_digest_build", "vkv_workspace_size",
                 "vkv_query_prep", "vkv_score",
                 "vkv_select", "vkv_admit", "vkv_attend", "vkv_step_run", "vkv_step_run_static",
                 "vkv_check_rows", "vkv_version", "vkv_row_max", "vkv_trigger", "vkv_required_inflation",
                 "vkv_conformal_z", "vkv_step_run_trigger",
                 "vkv_set_timing", "vkv_score_timing"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libvkv must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class Context:
    """A libvkv context bound to one HIP device."""

    def __init__(self, device: int = 0):
        self.lib = load()
        self.handle = ctypes.c_void_p()
        rc = self.lib.vkv_create(ctypes.byref(self.handle), int(device))
        if rc != 0:
            raise VkvError(rc, self.lib.vkv_last_error(None).decode())
        self.device = device

    def check(self, rc: int):
        if rc != 0:
            raise VkvError(rc, self.lib.vkv_last_error(self.handle).decode())

    def set_timing(self, enable: bool):
        """Record the duration of the score scan of each ``step_run``."""
        self.check(self.lib.vkv_set_timing(self.handle, 1 if enable else 0))

    def score_timing(self) -> list:
        """ms of each score scan ``step_run`` timed since the last read."""
        buf = (ctypes.c_float * 512)()
        n = self.lib.vkv_score_timing(self.handle, buf, 512)
        if n < 0:
            self.check(n)
        return [float(buf[i]) for i in range(n)]

    def close(self):
        if self.handle:
            self.lib.vkv_destroy(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Step:
    """The inputs of one decode step (``vkv_step``), from device tensors.

    cache [B,T,576], q_lat [B,H,512], q_rope [B,H,64] (bf16); index [B,T,cols]
    or None; P [r,512] or None; eta/eps/gam [B,T] fp32 or None."""

    def __init__(self, cache, q_lat, q_rope, W: int, mode: int, r: int = 0, index=None,
                 index_has_rope: bool = True, P=None, eta=None, eps=None, gam=None):
        B, T, cw = cache.shape
        H = q_lat.shape[1]
        self.tensors = (cache, q_lat, q_rope, index, P, eta, eps, gam)  # keep alive
        s = _Step()
        s.B, s.H, s.T, s.W = B, H, T, int(W)
        s.mode, s.r = int(mode), int(r)
        s.q_lat, s.q_rope = _ptr(q_lat), _ptr(q_rope)
        s.cache = _ptr(cache)
        s.cache_row_stride, s.cache_batch_stride = cw, T * cw
        if index is not None:
            s.index = _ptr(index)
            s.index_row_stride = index.shape[2]
            s.index_batch_stride = index.shape[1] * index.shape[2]
        s.index_has_rope = 1 if index_has_rope else 0
        s.P = _ptr(P)
        s.eta, s.eps, s.gam = _ptr(eta), _ptr(eps), _ptr(gam)
        self.c = s
        self.B, self.H, self.T, self.W, self.A = B, H, T, int(W), T - int(W)
        self.mode, self.r = int(mode), int(r)
        self.device = cache.device

    @property
    def ref(self):
        return ctypes.byref(self.c)


def digest_build(ctx: Context, cache: torch.Tensor, P: Optional[torch.Tensor], r: int,
                 with_rope: bool = True, index: Optional[torch.Tensor] = None,
                 eta: Optional[torch.Tensor] = None, eps: Optional[torch.Tensor] = None,
                 gam: Optional[torch.Tensor] = None, stream=None):
    """vkv_digest_build: fills ``index`` [B,T,cols] (and the certificate
    scalars when ``eta``/``eps``/``gam`` are given)."""
    B, T, cw = cache.shape
    irs = index.shape[2] if index is not None else 0
    ctx.check(ctx.lib.vkv_digest_build(
        ctx.handle, _ptr(cache), B, T, cw, T * cw, _ptr(P), int(r), 1 if with_rope else 0,
        _ptr(index), irs, T * irs, _ptr(eta), _ptr(eps), _ptr(gam), _stream(stream)))


def workspace_size(step: Step, k: int, cap: int = 0) -> int:
    lib = load()
    n = ctypes.c_size_t(0)
    rc = lib.vkv_workspace_size(step.ref, int(k), int(cap), ctypes.byref(n))
    if rc != 0:
        raise VkvError(rc, lib.vkv_last_error(None).decode())
    return int(n.value)


def alloc_workspace(step: Step, k: int, cap: int = 0) -> torch.Tensor:
    """A device workspace tensor of ``workspace_size`` bytes (256-B aligned)."""
    n = workspace_size(step, k, cap)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=step.device)


def query_prep(ctx: Context, step: Step, ws: torch.Tensor, stream=None):
    ctx.check(ctx.lib.vkv_query_prep(ctx.handle, step.ref, _ptr(ws), ws.numel(), _stream(stream)))


def score(ctx: Context, step: Step, ws: torch.Tensor, key: Optional[torch.Tensor] = None,
          ub: Optional[torch.Tensor] = None, stream=None, cert_mult: float = 1.0):
    ctx.check(ctx.lib.vkv_score(ctx.handle, step.ref, _ptr(ws), ws.numel(), _ptr(key), _ptr(ub),
                                float(cert_mult), _stream(stream)))


def select(ctx: Context, step: Step, ws: torch.Tensor, k: int, sel: torch.Tensor,
           theta: torch.Tensor, stream=None):
    ctx.check(ctx.lib.vkv_select(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(sel),
                                 _ptr(theta), _stream(stream)))


def admit(ctx: Context, step: Step, ws: torch.Tensor, k: int, sel: torch.Tensor,
          theta: torch.Tensor, ub: torch.Tensor, adm: torch.Tensor, adm_count: torch.Tensor,
          cap: int, stream=None, cert_mult: float = 1.0):
    ctx.check(ctx.lib.vkv_admit(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(sel),
                                _ptr(theta), _ptr(ub), float(cert_mult), _ptr(adm), _ptr(adm_count),
                                int(cap), _stream(stream)))


def attend(ctx: Context, step: Step, ws: torch.Tensor, k: int, sel: torch.Tensor,
           adm: Optional[torch.Tensor], adm_count: Optional[torch.Tensor], cap: int, scale: float,
           out: torch.Tensor, lse: torch.Tensor, stream=None):
    ctx.check(ctx.lib.vkv_attend(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(sel),
                                 _ptr(adm), _ptr(adm_count), int(cap), float(scale), _ptr(out),
                                 _ptr(lse), _stream(stream)))


def step_run(ctx: Context, step: Step, ws: torch.Tensor, k: int, key: torch.Tensor,
             ub: Optional[torch.Tensor], sel: torch.Tensor, theta: torch.Tensor,
             adm: Optional[torch.Tensor], adm_count: Optional[torch.Tensor], cap: int,
             scale: float, out: torch.Tensor, lse: torch.Tensor, stream=None,
             cert_mult: float = 1.0):
    ctx.check(ctx.lib.vkv_step_run(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(key),
                                   _ptr(ub), _ptr(sel), _ptr(theta), _ptr(adm), _ptr(adm_count),
                                   int(cap), float(cert_mult), float(scale), _ptr(out), _ptr(lse),
                                   _stream(stream)))


def step_run_static(ctx: Context, step: Step, k: int, key: torch.Tensor, ub: Optional[torch.Tensor],
                    sel: torch.Tensor, theta: torch.Tensor, adm: Optional[torch.Tensor],
                    adm_count: Optional[torch.Tensor], cap: int, scale: float, out: torch.Tensor,
                    lse: torch.Tensor, stream=None, cert_mult: float = 1.0):
    """vkv_step_run_static: the step on the library's static workspace (no allocation)."""
    ctx.check(ctx.lib.vkv_step_run_static(ctx.handle, step.ref, int(k), _ptr(key), _ptr(ub), _ptr(sel),
                                          _ptr(theta), _ptr(adm), _ptr(adm_count), int(cap),
                                          float(cert_mult), float(scale), _ptr(out), _ptr(lse),
                                          _stream(stream)))


def row_max(ctx: Context, step: Step, rows: Optional[torch.Tensor], add_recent: bool,
            smax: torch.Tensor, argmax: torch.Tensor, stream=None):
    """vkv_row_max: per head, the exact max full score over ``rows`` [B,n]
    (None: the whole archive), plus the recent window if ``add_recent``."""
    n = rows.shape[1] if rows is not None else 0
    ctx.check(ctx.lib.vkv_row_max(ctx.handle, step.ref, _ptr(rows), int(n), 1 if add_recent else 0,
                                  _ptr(smax), _ptr(argmax), _stream(stream)))


def trigger(ctx: Context, step: Step, ws: torch.Tensor, k: int, sel: torch.Tensor, ub: torch.Tensor,
            cert_mult: float, smax: torch.Tensor, topj: int, fired: torch.Tensor,
            fired_count: torch.Tensor, cap: int, stream=None):
    ctx.check(ctx.lib.vkv_trigger(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(sel), _ptr(ub),
                                  float(cert_mult), _ptr(smax), int(topj), _ptr(fired), _ptr(fired_count),
                                  int(cap), _stream(stream)))


def required_inflation(ctx: Context, step: Step, ws: torch.Tensor, k: int, sel: torch.Tensor,
                       tier1_max: torch.Tensor, argmax: torch.Tensor, hard: torch.Tensor, zq: torch.Tensor,
                       stream=None):
    ctx.check(ctx.lib.vkv_required_inflation(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(sel),
                                             _ptr(tier1_max), _ptr(argmax), _ptr(hard), _ptr(zq),
                                             _stream(stream)))


def conformal_z(zq, tau=(9, 10), zmax: float = 8.0):
    """vkv_conformal_z on host values; returns (z, min_hard, k)."""
    import numpy as _np
    lib = load()
    v = _np.ascontiguousarray(zq, _np.float64)
    z = ctypes.c_double(0.0)
    mh = ctypes.c_int64(0)
    k = ctypes.c_int64(0)
    rc = lib.vkv_conformal_z(v.ctypes.data if v.size else None, v.size, int(tau[0]), int(tau[1]), float(zmax),
                             ctypes.byref(z), ctypes.byref(mh), ctypes.byref(k))
    if rc != 0:
        raise VkvError(rc, lib.vkv_last_error(None).decode())
    return float(z.value), int(mh.value), int(k.value)


def step_run_trigger(ctx: Context, step: Step, ws: torch.Tensor, k: int, key, ub, sel, theta,
                     cert_mult: float, smax, argmax, topj: int, fired, fired_count, cap: int,
                     scale: float, out, lse, stream=None):
    ctx.check(ctx.lib.vkv_step_run_trigger(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(key),
                                           _ptr(ub), _ptr(sel), _ptr(theta), float(cert_mult), _ptr(smax),
                                           _ptr(argmax), int(topj), _ptr(fired), _ptr(fired_count), int(cap),
                                           float(scale), _ptr(out), _ptr(lse), _stream(stream)))


def sketch_workspace_size(r: int) -> int:
    lib = load()
    n = ctypes.c_size_t(0)
    rc = lib.vkv_sketch_workspace_size(int(r), ctypes.byref(n))
    if rc != 0:
        raise VkvError(rc, lib.vkv_last_error(None).decode())
    return int(n.value)


def sketch_basis(ctx: Context, q: torch.Tensor, r: int, iters: int, ws: torch.Tensor, P: torch.Tensor,
                 energy: Optional[torch.Tensor] = None, stream=None):
    """vkv_sketch_basis: P [r,512] bf16 from the prefix content queries
    q [m,512] bf16; energy [2] fp64 = (captured, total) second moment
    (synchronises the stream)."""
    m = q.numel() // D_LAT
    ctx.check(ctx.lib.vkv_sketch_basis(ctx.handle, _ptr(q), int(m), int(r), int(iters), _ptr(ws), ws.numel(),
                                       _ptr(P), _ptr(energy), _stream(stream)))


def sigma_workspace_size(B: int, nblk: int) -> int:
    lib = load()
    n = ctypes.c_size_t(0)
    rc = lib.vkv_sigma_workspace_size(int(B), int(nblk), ctypes.byref(n))
    if rc != 0:
        raise VkvError(rc, lib.vkv_last_error(None).decode())
    return int(n.value)


def sigma_close(ctx: Context, cache: torch.Tensor, t0: int, nblk: int, kappa: int, ws: torch.Tensor,
                sigma: torch.Tensor, stream=None):
    """vkv_sigma_close over cache [B, T, row_stride>=576] bf16 into sigma [B, S] fp64."""
    B, T = cache.shape[0], cache.shape[1]
    ctx.check(ctx.lib.vkv_sigma_close(ctx.handle, _ptr(cache), B, T, cache.stride(1), cache.stride(0), int(t0),
                                      int(nblk), int(kappa), _ptr(ws), ws.numel(), _ptr(sigma), sigma.stride(0),
                                      _stream(stream)))


def sigma_tier_size(n_closed: int, m: int, nsink: int = 4) -> int:
    lo = min(nsink, n_closed)
    return lo + min(m, n_closed - lo)


def sigma_select(ctx: Context, sigma: torch.Tensor, n_closed: int, m: int, nsink: int, kept: torch.Tensor,
                 stream=None):
    """vkv_sigma_select: kept [B, sigma_tier_size(n_closed, m, nsink)] int32."""
    ctx.check(ctx.lib.vkv_sigma_select(ctx.handle, _ptr(sigma), sigma.shape[0], int(n_closed), sigma.stride(0),
                                       int(m), int(nsink), _ptr(kept), _stream(stream)))


def step_run_kept(ctx: Context, step: Step, ws: torch.Tensor, k: int, kept, key, ub, cert_mult: float, smax,
                  argmax, topj: int, fired, fired_count, cap: int, scale: float, out, lse, stream=None):
    ctx.check(ctx.lib.vkv_step_run_kept(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(k), _ptr(kept), _ptr(key),
                                        _ptr(ub), float(cert_mult), _ptr(smax), _ptr(argmax), int(topj),
                                        _ptr(fired), _ptr(fired_count), int(cap), float(scale), _ptr(out),
                                        _ptr(lse), _stream(stream)))


def pack_rows(ctx: Context, lists: torch.Tensor, counts: torch.Tensor, offsets: torch.Tensor,
              packed: torch.Tensor, stream=None):
    """vkv_pack_rows: lists [n, cap] int32, counts [n] -> offsets [n+1], packed."""
    n, cap = lists.shape[0], lists.shape[-1]
    ctx.check(ctx.lib.vkv_pack_rows(ctx.handle, _ptr(lists), _ptr(counts), int(n), int(cap), _ptr(offsets),
                                    _ptr(packed), _stream(stream)))


def page_box(ctx: Context, step: Step, page: int, box: torch.Tensor, stream=None):
    """vkv_page_box: box [B, ceil(A / page), 2, n] bf16 <- per-page column ranges of the index rows."""
    ctx.check(ctx.lib.vkv_page_box(ctx.handle, step.ref, int(page), _ptr(box), _stream(stream)))


def page_bound(ctx: Context, step: Step, ws: torch.Tensor, page: int, box: torch.Tensor, bound: torch.Tensor,
               stream=None):
    """vkv_page_bound: bound [B, ceil(A / page)] float64 <- the pages' interval bounds (after query_prep)."""
    ctx.check(ctx.lib.vkv_page_bound(ctx.handle, step.ref, _ptr(ws), ws.numel(), int(page), _ptr(box), _ptr(bound),
                                     _stream(stream)))


def check_rows(ctx: Context, step: Step, k: int, sel: Optional[torch.Tensor],
               adm: Optional[torch.Tensor] = None, adm_count: Optional[torch.Tensor] = None,
               cap: int = 0, stream=None):
    """vkv_check_rows: the row-set invariant on caller buffers (synchronises)."""
    ctx.check(ctx.lib.vkv_check_rows(ctx.handle, step.ref, int(k), _ptr(sel), _ptr(adm),
                                     _ptr(adm_count), int(cap), _stream(stream)))


class Buffers:
    """Output and intermediate buffers of one step, on the step's device."""

    def __init__(self, step: Step, k: int, two_tier: bool = False, cap: Optional[int] = None,
                 cert_mult: float = 1.0):
        dev = step.device
        self.cert_mult = float(cert_mult)
        B, H, A = step.B, step.H, step.A
        self.k = int(k)
        self.cap = (A if cap is None else int(cap)) if two_tier else 0
        self.key = torch.empty(B, max(A, 1), dtype=torch.float32, device=dev)
        self.ub = torch.empty(B, max(A, 1), dtype=torch.float32, device=dev) if two_tier else None
        self.sel = torch.empty(B, max(self.k, 1), dtype=torch.int32, device=dev)
        self.theta = torch.empty(B, dtype=torch.float64, device=dev)
        self.adm = torch.empty(B, max(self.cap, 1), dtype=torch.int32, device=dev) if two_tier else None
        self.adm_count = torch.zeros(B, dtype=torch.int32, device=dev) if two_tier else None
        self.out = torch.empty(B, H, D_LAT, dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty(B, H, dtype=torch.float32, device=dev)
        self.ws = alloc_workspace(step, self.k, self.cap)

    def run(self, ctx: Context, step: Step, scale: float, stream=None):
        step_run(ctx, step, self.ws, self.k, self.key, self.ub, self.sel, self.theta, self.adm,
                 self.adm_count, self.cap, scale, self.out, self.lse, stream, self.cert_mult)

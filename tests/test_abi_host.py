"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point include/vkv.h declares, and refuses invalid arguments
before touching the device."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vkv.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(vkv_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    import paper_2609_03949_amd as vkv
    return vkv.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("vkv_digest_build", "vkv_score", "vkv_select", "vkv_admit", "vkv_attend",
              "vkv_step_run", "vkv_workspace_size", "vkv_create", "vkv_destroy"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    import paper_2609_03949_amd as vkv
    nm = subprocess.run(["nm", "-D", "--defined-only", vkv.lib_path()], capture_output=True,
                        text=True, check=True).stdout
    exported = set(re.findall(r"\bT (vkv_\w+)$", nm, flags=re.M))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)
    assert set(vkv.exported_symbols) == set(declared_functions())


def test_status_strings_and_version(lib):
    assert lib.vkv_version() >= 100
    assert lib.vkv_status_string(0) == b"ok"
    for code in range(-8, 0):
        assert lib.vkv_status_string(code) != b"unknown status"


def _step(**kw):
    import paper_2609_03949_amd as vkv
    s = vkv._Step()
    s.B, s.H, s.T, s.W, s.mode, s.r = 2, 16, 4096, 128, 3, 64
    fake = 1 << 20                       # aligned non-null host value; never dereferenced
    s.q_lat = s.q_rope = s.cache = s.index = s.P = fake
    s.cache_row_stride, s.cache_batch_stride = 576, 4096 * 576
    s.index_row_stride, s.index_batch_stride = 128, 4096 * 128
    s.index_has_rope = 1
    for k, v in kw.items():
        setattr(s, k, v)
    return s


def _ws_size(lib, s, k=100, cap=0):
    n = ctypes.c_size_t(0)
    rc = lib.vkv_workspace_size(ctypes.byref(s), k, cap, ctypes.byref(n))
    return rc, n.value


@pytest.mark.parametrize("field,value,code", [
    ("B", 0, -2), ("H", 129, -2), ("H", 0, -2), ("T", 0, -2), ("W", 5000, -2),
    ("mode", 4, -1), ("r", 48, -4), ("r", 1024, -4), ("q_lat", 0, -1),
    ("cache_row_stride", 500, -3), ("index_row_stride", 100, -3), ("cache", (1 << 20) + 2, -3),
])
def test_workspace_size_validation(lib, field, value, code):
    rc, _ = _ws_size(lib, _step(**{field: value}))
    assert rc == code, (field, value, rc, lib.vkv_last_error(None))


def test_workspace_size_ok_and_k_range(lib):
    s = _step()
    rc, n = _ws_size(lib, s)
    assert rc == 0 and n > 0 and n % 256 == 0
    assert _ws_size(lib, s, k=4096 - 128 + 1)[0] == -1
    assert _ws_size(lib, s, k=-1)[0] == -1
    assert _ws_size(lib, s, cap=5000)[0] == -1
    # the admission capacity only grows the attention partials
    assert _ws_size(lib, s, cap=2000)[1] >= n


def test_rope_mode_rules(lib):
    assert _ws_size(lib, _step(mode=1, r=0, index=0))[0] == 0       # in-place branch slice
    assert _ws_size(lib, _step(mode=1, r=64))[0] == -1              # ROPE takes r = 0
    assert _ws_size(lib, _step(mode=3, index_has_rope=0))[0] == -4  # branch must be in the index
    assert _ws_size(lib, _step(mode=2, index=0))[0] == -1           # digest needs the index


def test_null_context_is_refused(lib):
    s = _step()
    P = ctypes.c_void_p
    assert lib.vkv_score(None, ctypes.byref(s), P(1 << 20), 1 << 20, P(1 << 20), None,
                         ctypes.c_float(1.0), None) == -1
    assert lib.vkv_admit(None, ctypes.byref(s), None, 0, 1, None, None, None, ctypes.c_float(1.0),
                         None, None, 0, None) == -1
    assert lib.vkv_check_rows(None, ctypes.byref(s), 1, None, None, None, 0, None) == -1
    assert lib.vkv_select(None, ctypes.byref(s), None, 0, 1, None, None, None) == -1
    assert lib.vkv_attend(None, ctypes.byref(s), None, 0, 1, None, None, None, 0, ctypes.c_float(0.1),
                          None, None, None) == -1
    assert lib.vkv_page_box(None, ctypes.byref(s), 64, P(1 << 20), None) == -1
    assert lib.vkv_page_bound(None, ctypes.byref(s), P(1 << 20), 1 << 20, 64, P(1 << 20), P(1 << 20), None) == -1
    assert b"ctx" in lib.vkv_last_error(None)


def test_conformal_z_host_function_matches_the_oracle(lib, oracle_mod):
    """vkv_conformal_z is host code (no device): the library's quantile equals
    the oracle's for assorted calibration sets, targets and clamps."""
    import numpy as np
    import paper_2609_03949_amd as vkv
    rng = np.random.default_rng(7)
    for n in (0, 5, 17, 18, 19, 37, 64, 500):
        for tau in ((9, 10), (4, 5), (19, 20)):
            for zmax in (8.0, 2.0):
                zq = rng.standard_normal(n) * 3 + 1
                assert vkv.conformal_z(zq, tau, zmax) == oracle_mod.conformal_z(zq, tau, zmax)
    with pytest.raises(vkv.VkvError):
        vkv.conformal_z([1.0], (10, 10))


def test_header_is_plain_c(tmp_path):
    """include/vkv.h is a C header: it compiles as C99 with warnings on, and a
    C translation unit can take the address of every declared entry point."""
    import shutil
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use.c"
    names = declared_functions()
    src.write_text('#include "vkv.h"\nvoid* table[] = {' + ", ".join(f"(void*)&{n}" for n in names) + "};\n")
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-I", os.path.dirname(HEADER),
                        str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr

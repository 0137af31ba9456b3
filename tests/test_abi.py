"""The C ABI library loads and exports every entry point its header declares, and its
host-side argument checks answer without touching a GPU (CPU only)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fovea.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fovea_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    import paper_2608_22883_amd.fovea as f

    return f


def test_header_declares_the_entry_points():
    assert _declared() == sorted([
        "fovea_abi_version", "fovea_status_str", "fovea_create", "fovea_destroy",
        "fovea_build_memory_workspace", "fovea_build_memory", "fovea_retrieve_fuse_workspace",
        "fovea_retrieve_fuse", "fovea_retrieve_fuse_noalloc",
        "fovea_last_error", "fovea_profile", "fovea_profile_read", "fovea_lm_topk_workspace",
        "fovea_lm_topk", "fovea_retrieve_fuse_backward_workspace", "fovea_retrieve_fuse_backward",
        "fovea_build_memory_backward_workspace", "fovea_build_memory_backward"])


def test_library_exports_every_declared_symbol(lib):
    raw = ctypes.CDLL(lib.LIB_PATH)
    for name in _declared():
        assert hasattr(raw, name), name
    assert sorted(lib.EXPORTED) == _declared()


def test_version_and_status_strings(lib):
    assert lib.fovea_abi_version() == 1
    for st in range(6):
        assert lib.fovea_status_str(st) and "unknown" not in lib.fovea_status_str(st)
    assert "unknown" in lib.fovea_status_str(99)


def _dims(lib, **kw):
    d = dict(d=256, d_v=256, d_m=128, d_c=512, n_depth=7, dtype=lib.FOVEA_F32, ln_eps=1e-5,
             rms_eps=1e-6)
    d.update(kw)
    return lib.Dims(**d)


def _params(lib):
    P = lib.Params()
    for n in lib.PARAM_TENSORS:
        setattr(P, n, 4096)   # non-null placeholders: never dereferenced on these paths
    P.b_g2 = -2.0
    return P


def _create(lib, dims, params):
    ctx = ctypes.c_void_p(12345)
    st = lib.lib.fovea_create(ctypes.byref(ctx), ctypes.byref(dims) if dims else None,
                              ctypes.byref(params) if params else None, None)
    return st, ctx.value


def test_create_rejects_bad_arguments_on_the_host(lib):
    P = _params(lib)
    assert lib.lib.fovea_create(None, ctypes.byref(_dims(lib)), ctypes.byref(P), None) == lib.FOVEA_ERR_INVALID_ARG
    st, ctx = _create(lib, None, P)
    assert st == lib.FOVEA_ERR_INVALID_ARG and ctx is None
    for bad in (dict(d=0), dict(d_m=-64), dict(n_depth=0), dict(dtype=7), dict(ln_eps=float("nan")),
                dict(rms_eps=-1.0)):
        assert _create(lib, _dims(lib, **bad), P)[0] == lib.FOVEA_ERR_INVALID_ARG, bad
    P2 = _params(lib)
    P2.W_Q = None
    assert _create(lib, _dims(lib), P2)[0] == lib.FOVEA_ERR_INVALID_ARG
    P3 = _params(lib)
    P3.b_g2 = float("nan")
    assert _create(lib, _dims(lib), P3)[0] == lib.FOVEA_ERR_INVALID_ARG
    for unsup in (dict(d=100), dict(d_m=96), dict(d_c=500), dict(d_v=65)):
        assert _create(lib, _dims(lib, **unsup), P)[0] == lib.FOVEA_ERR_UNSUPPORTED, unsup


def test_null_context_paths(lib):
    assert lib.lib.fovea_retrieve_fuse_workspace(None, 1, 10, 10, 10, 4) == 0
    assert lib.lib.fovea_build_memory_workspace(None, 10) == 0
    st = lib.lib.fovea_retrieve_fuse(None, 1, None, 0, 0, None, None, None, None, 0, 0, None,
                                     None, None, 0, 1, None, None, None, None, None, None, None,
                                     0, None)
    assert st == lib.FOVEA_ERR_INVALID_ARG
    st = lib.lib.fovea_retrieve_fuse_noalloc(None, 1, None, 0, 0, None, None, None, None, 0, 0, None,
                                             None, None, 0, 1, None, None, None, None, None, None, None)
    assert st == lib.FOVEA_ERR_INVALID_ARG
    assert lib.lib.fovea_build_memory(None, 1, None, None, None, None, 0, None) == lib.FOVEA_ERR_INVALID_ARG
    assert lib.lib.fovea_last_error(None, None, None) == lib.FOVEA_ERR_INVALID_ARG
    assert lib.lib.fovea_profile(None, 1) == lib.FOVEA_ERR_INVALID_ARG
    assert lib.lib.fovea_profile_read(None, 4, None, None, None) == -1
    assert lib.lib.fovea_lm_topk_workspace(None, 4, 32000, 6) == 0
    assert lib.lib.fovea_retrieve_fuse_backward_workspace(None, 1, 4, 8, 4) == 0
    assert lib.lib.fovea_build_memory_backward_workspace(None, 4) == 0
    assert lib.lib.fovea_build_memory_backward(None, None, 1, None, None, None, None, None, None,
                                               None, None, None, 0, None) == lib.FOVEA_ERR_INVALID_ARG
    assert lib.lib.fovea_retrieve_fuse_backward(
        None, None, 1, None, 0, 0, None, None, None, 0, 0, None, None, None, None, 1, None, None,
        None, None, None, None, 0, None) == lib.FOVEA_ERR_INVALID_ARG
    assert lib.lib.fovea_lm_topk(None, 4, None, None, 32000, 6, None, None, None, 0,
                                 None) == lib.FOVEA_ERR_INVALID_ARG
    lib.lib.fovea_destroy(None)


def test_header_limits_match_the_binding(lib):
    src = open(HEADER).read()
    for name in ("FOVEA_MAX_M", "FOVEA_MAX_KMAX", "FOVEA_LM_MAX_K", "FOVEA_LM_MAX_VOCAB",
                 "FOVEA_LM_MAX_ROWS", "FOVEA_STATIC_WORKSPACE_BYTES"):
        m = re.search(r"#define\s+" + name + r"\s+\(?([0-9]+)u?(?:\s*<<\s*([0-9]+))?", src)
        assert m, name
        val = int(m.group(1)) << int(m.group(2) or 0)
        assert getattr(lib, name) == val, name

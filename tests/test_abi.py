"""CPU checks of the C ABI: the library loads, exports every symbol the header
declares, and rejects bad arguments on the host before any launch."""

import ctypes
import os
import re

import pytest

from paper_2605_01910_amd import santa as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "santa.h")).read()
    return sorted(set(re.findall(r"\b(santa_[a-z_]+)\s*\(", text)))


def test_header_declarations_match_binding_exports():
    assert declared_symbols() == sorted(S.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = S.load()
    for name in declared_symbols():
        assert hasattr(lib, name), name


def _shape(B=1, Hq=32, Hkv=8, d=128, dtype=0):
    return S.santa_shape_t(B, Hq, Hkv, d, dtype)


def _kv(n=32768, k=16, v=16, ctx=None, bt=None, ps=0, mp=0, sn=8 * 128):
    return S.santa_kv_t(k, v, n * 8 * 128, sn, 128, ctx, bt, ps, mp, n)


def ws_size(shape, kv, Sn, kind):
    return S.load().santa_workspace_size(ctypes.byref(shape), ctypes.byref(kv), Sn, kind)


def test_workspace_size_is_positive_and_grows_with_batch():
    a = ws_size(_shape(B=1), _kv(), 256, S.SANTA_KIND_STRATIFIED)
    b = ws_size(_shape(B=16), _kv(), 256, S.SANTA_KIND_STRATIFIED)
    assert 0 < a < b
    assert ws_size(_shape(), _kv(), 256, S.SANTA_KIND_DENSE) > 0
    assert ws_size(_shape(), _kv(), 256, S.SANTA_KIND_BERNOULLI) >= a


@pytest.mark.parametrize("shape,kv,Sn,kind", [
    (_shape(d=64), _kv(), 256, 1),           # head_dim != 128
    (_shape(Hq=12, Hkv=8), _kv(), 256, 1),   # Hq not a multiple of Hkv
    (_shape(Hq=48, Hkv=3), _kv(), 256, 1),   # G = 16 unsupported
    (_shape(), _kv(n=0), 256, 1),            # empty cache
    (_shape(), _kv(), 0, 1),                 # S = 0
    (_shape(), _kv(), (1 << 24) + 1, 2),     # S too large
    (_shape(), _kv(), 256, 7),               # bad kind
    (_shape(dtype=5), _kv(), 256, 0),        # bad dtype
])
def test_workspace_size_rejects_invalid(shape, kv, Sn, kind):
    assert ws_size(shape, kv, Sn, kind) == 0


def call_sys(shape, kv, Sn=256, u=16, out=16, ws=256, ws_bytes=1 << 40, q=16):
    lib = S.load()
    st = lib.santa_decode_systematic(q, ctypes.byref(kv), ctypes.byref(shape), 0.088, Sn, u, None,
                                     out, ws, ws_bytes, None)
    return st, lib.santa_last_error().decode()


def test_host_validation_errors_before_any_launch():
    # all of these fail in host validation, so no device pointer is touched
    assert call_sys(_shape(), _kv(), q=None)[0] == S.SANTA_ERR_INVALID_ARG
    assert call_sys(_shape(), _kv(), u=None)[0] == S.SANTA_ERR_INVALID_ARG
    assert call_sys(_shape(), _kv(), Sn=0)[0] == S.SANTA_ERR_INVALID_ARG
    assert call_sys(_shape(d=256), _kv())[0] == S.SANTA_ERR_UNSUPPORTED
    assert call_sys(_shape(), _kv(k=None))[0] == S.SANTA_ERR_INVALID_ARG
    assert call_sys(_shape(), _kv(k=24))[0] == S.SANTA_ERR_UNSUPPORTED        # misaligned
    assert call_sys(_shape(), _kv(sn=100))[0] == S.SANTA_ERR_UNSUPPORTED      # stride breaks alignment
    assert call_sys(_shape(), _kv(), ws=None)[0] == S.SANTA_ERR_WORKSPACE
    assert call_sys(_shape(), _kv(), ws=64)[0] == S.SANTA_ERR_WORKSPACE       # misaligned workspace
    st, msg = call_sys(_shape(), _kv(), ws_bytes=100)
    assert st == S.SANTA_ERR_WORKSPACE and "too small" in msg
    # paged: page size must be a power of two, table must cover n_k
    assert call_sys(_shape(), _kv(bt=16, ps=12, mp=4096))[0] == S.SANTA_ERR_UNSUPPORTED
    assert call_sys(_shape(), _kv(bt=16, ps=16, mp=10))[0] == S.SANTA_ERR_INVALID_ARG


def test_bernoulli_validation():
    lib = S.load()
    sh, kv = _shape(), _kv()
    kt = S.santa_kt_t(16, 8 * 128 * 32768, 128 * 32768, 32768)

    def call(kt_=kt, Bd=1, mode=0, uq=16, kvx=kv):
        return lib.santa_decode_bernoulli_qk(16, ctypes.byref(kt_), ctypes.byref(kvx), ctypes.byref(sh),
                                             0.088, Bd, mode, uq, 256, 16, None, None, 16, 256,
                                             1 << 40, None)

    assert call(mode=2) == S.SANTA_ERR_INVALID_ARG
    assert call(Bd=0) == S.SANTA_ERR_INVALID_ARG
    assert call(uq=None) == S.SANTA_ERR_INVALID_ARG
    assert call(kt_=S.santa_kt_t(16, 0, 0, 100)) == S.SANTA_ERR_INVALID_ARG      # stride_d < n_k
    assert call(kvx=_kv(bt=16, ps=16, mp=4096)) == S.SANTA_ERR_UNSUPPORTED       # paged


def test_status_strings():
    lib = S.load()
    assert lib.santa_status_string(0) == b"SANTA_OK"
    assert lib.santa_status_string(3) == b"SANTA_ERR_WORKSPACE"


def test_time_next_call_needs_both_events_or_neither():
    lib = S.load()
    assert lib.santa_time_next_call(None, None) == S.SANTA_OK
    st = lib.santa_time_next_call(ctypes.c_void_p(0x1000), None)
    assert st == S.SANTA_ERR_INVALID_ARG
    assert b"both" in lib.santa_last_error()
    assert lib.santa_time_next_call(None, None) == S.SANTA_OK


def test_stream_read_validation():
    # every rejection happens on the host, before a launch
    lib = S.load()
    P = ctypes.c_void_p
    ok_buf, ok_sink = P(0x100000), P(0x200000)
    assert lib.santa_stream_read(None, 1024, ok_sink, None) == S.SANTA_ERR_INVALID_ARG
    assert lib.santa_stream_read(ok_buf, 1024, None, None) == S.SANTA_ERR_INVALID_ARG
    assert lib.santa_stream_read(ok_buf, 0, ok_sink, None) == S.SANTA_ERR_INVALID_ARG
    assert lib.santa_stream_read(ok_buf, 1000, ok_sink, None) == S.SANTA_ERR_INVALID_ARG
    assert lib.santa_stream_read(P(0x100008), 1024, ok_sink, None) == S.SANTA_ERR_INVALID_ARG
    assert b"aligned" in lib.santa_last_error()


def _plan(shape, kv, Sn, kind, path="auto", splits=0):
    with S.options(path, splits):
        return S.santa_plan_info(shape, kv, Sn, kind)


def test_path_choice_by_size_cache_and_kind():
    """The host picks a path without launching anything: the scheduled path
    for systematic and stratified steps where it measured fastest (S <= 1024;
    paged caches up to 8192 workgroups, FP8 up to 2048) and for i.i.d. steps
    at G <= 4 with S <= 256, or larger S on grids of at most 256 workgroups,
    else the persistent launch within one resident
    round and the two-launch path beyond it; Bernoulli steps never take the
    scheduled path, nor does a row that needs more than 64 splits."""
    sysk, strat, iid = S.SANTA_KIND_SYSTEMATIC, S.SANTA_KIND_STRATIFIED, S.SANTA_KIND_IID
    rows, two, one = "k_row_sampled", "k_stream_cdf + k_value_heads", "k_fused_sampled"
    p1 = _plan(_shape(B=1), _kv(), 256, strat)
    assert (p1["path"], p1["kernels"], p1["splits"]) == (S.SANTA_PATH_SCHEDULED, rows, 32)
    assert _plan(_shape(B=1), _kv(), 512, sysk)["kernels"] == rows
    assert _plan(_shape(B=1), _kv(), 1024, sysk)["kernels"] == rows
    assert _plan(_shape(B=1), _kv(), 1024, strat)["kernels"] == rows
    assert _plan(_shape(B=1), _kv(), 2048, strat)["kernels"] == one
    for B in (2, 16):
        for kind in (sysk, strat):
            p = _plan(_shape(B=B), _kv(), 256, kind)
            assert (p["path"], p["kernels"]) == (S.SANTA_PATH_SCHEDULED, rows), (B, p)
    assert _plan(_shape(B=16), _kv(), 1024, sysk)["kernels"] == rows
    assert _plan(_shape(B=16), _kv(), 2048, sysk)["kernels"] == two
    assert _plan(_shape(B=16), _kv(), 256, iid)["kernels"] == rows
    assert _plan(_shape(B=1), _kv(), 256, iid)["kernels"] == rows
    # i.i.d. thresholds on the scheduled path: in registers up to S = 256, in
    # LDS above that on grids of at most 256 workgroups, G <= 4
    assert _plan(_shape(B=1), _kv(), 384, iid)["kernels"] == rows
    assert _plan(_shape(B=16), _kv(), 384, iid)["kernels"] == two
    assert _plan(_shape(B=1, Hq=16, Hkv=2), _kv(), 256, iid)["kernels"] == one
    paged = _kv(n=65536, bt=16, ps=16, mp=4096)
    assert _plan(_shape(B=16), paged, 256, sysk)["kernels"] == rows
    assert _plan(_shape(B=64), paged, 256, sysk)["kernels"] == two
    fp8 = _kv()
    fp8.kv_dtype, fp8.k_scale, fp8.v_scale = S.SANTA_KV_FP8_E4M3, 16, 16
    assert _plan(_shape(B=8), fp8, 256, sysk)["kernels"] == rows
    assert _plan(_shape(B=16), fp8, 256, sysk)["kernels"] == two
    assert _plan(_shape(B=16), fp8, 256, sysk, "rows")["kernels"] == "k_row_sampled"
    # forced paths, and the scheduled option's limit of 64 splits per row
    assert _plan(_shape(B=1), _kv(), 256, strat, "rows")["kernels"] == "k_row_sampled"
    assert _plan(_shape(B=16), _kv(), 256, sysk, "two")["kernels"] == "k_stream_cdf + k_value_heads"
    assert _plan(_shape(B=16), _kv(), 256, sysk, "one")["kernels"] == "k_fused_sampled"
    p128 = _plan(_shape(B=16), _kv(n=131072), 256, sysk, "rows")
    assert p128["splits"] > 64 and p128["kernels"] == "k_stream_cdf + k_value_heads"
    # the scheduled path keeps the one-launch path's workspace layout
    assert (_plan(_shape(B=16), _kv(), 256, strat, "rows")["workspace"] ==
            _plan(_shape(B=16), _kv(), 256, strat, "one")["workspace"])


def test_flash_path_choice():
    """S2ANTA-flash takes the scheduled kernel (k_row_flash) under the automatic
    and scheduled options for G <= 4 and at most 64 splits per row, with the
    small split budget (32 splits at batch 1, 32k keys); G = 8, more splits or
    the one-launch / two-launch options keep the flash mode of k_fused_dense.
    Its plan never needs more workspace than santa_workspace_size reports for
    the flash kind (the dense layout)."""
    flash = S.SANTA_KIND_FLASH
    p = _plan(_shape(B=1), _kv(), 0, flash)
    assert (p["path"], p["kernels"], p["splits"]) == (S.SANTA_PATH_SCHEDULED, "k_row_flash", 32)
    assert _plan(_shape(B=16), _kv(), 0, flash, "rows")["kernels"] == "k_row_flash"
    for opt in ("one", "two"):
        assert _plan(_shape(B=1), _kv(), 0, flash, opt)["kernels"] == "k_fused_dense (flash mode)"
    assert _plan(_shape(B=1, Hq=16, Hkv=2), _kv(), 0, flash)["kernels"] == "k_fused_dense (flash mode)"
    assert _plan(_shape(B=16), _kv(n=131072), 0, flash)["kernels"] == "k_fused_dense (flash mode)"
    for B in (1, 4, 16):
        need = ws_size(_shape(B=B), _kv(), 0, flash)
        assert _plan(_shape(B=B), _kv(), 0, flash)["workspace"] <= need

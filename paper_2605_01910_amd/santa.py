"""Thin ctypes binding of libsanta (include/santa.h).

The functions below carry the C entry points' names and do argument
marshalling only: they turn torch tensors into device pointers and C structs,
pass the current HIP stream, and raise ``SantaError`` on a non-OK status.
Every step of the decode runs in the library's HIP kernels; there is no
fallback path.  PyTorch provides device memory and streams.
"""

from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsanta.so")

SANTA_OK, SANTA_ERR_INVALID_ARG, SANTA_ERR_UNSUPPORTED, SANTA_ERR_WORKSPACE, SANTA_ERR_HIP = range(5)
SANTA_BF16, SANTA_F32 = 0, 1
SANTA_KV_AS_Q, SANTA_KV_FP8_E4M3 = 0, 1
(SANTA_KIND_DENSE, SANTA_KIND_SYSTEMATIC, SANTA_KIND_STRATIFIED, SANTA_KIND_BERNOULLI,
 SANTA_KIND_FLASH, SANTA_KIND_IID) = range(6)
(SANTA_PATH_AUTO, SANTA_PATH_ONE_LAUNCH, SANTA_PATH_TWO_LAUNCH, SANTA_PATH_MULTI,
 SANTA_PATH_SCHEDULED) = range(5)
PATHS = {"auto": SANTA_PATH_AUTO, "one": SANTA_PATH_ONE_LAUNCH, "two": SANTA_PATH_TWO_LAUNCH,
         "multi": SANTA_PATH_MULTI, "rows": SANTA_PATH_SCHEDULED}

# every symbol include/santa.h declares
EXPORTS = ("santa_workspace_size", "santa_workspace_init", "santa_decode_dense",
           "santa_decode_systematic", "santa_decode_stratified", "santa_decode_bernoulli_qk",
           "santa_decode_iid", "santa_decode_flash", "santa_stream_read", "santa_time_next_call",
           "santa_set_options", "santa_get_options", "santa_plan_info",
           "santa_decode_stratified_noalloc", "santa_status_string", "santa_last_error")

STREAM_READ_GROUPS = 4096  # SANTA_STREAM_READ_GROUPS: uint32 words of the sink
STATIC_SCRATCH_BYTES = 64 << 20  # SANTA_STATIC_SCRATCH_BYTES


class SantaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_status_name(status)}: {message}")
        self.status = status


class santa_shape_t(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32)]


class santa_kv_t(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("stride_b", ctypes.c_int64), ("stride_n", ctypes.c_int64),
                ("stride_h", ctypes.c_int64),
                ("ctx_len", ctypes.c_void_p), ("block_table", ctypes.c_void_p),
                ("page_size", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("n_k", ctypes.c_int32),
                ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p),
                ("kv_dtype", ctypes.c_int32), ("k_scale", ctypes.c_void_p),
                ("v_scale", ctypes.c_void_p)]


class santa_kt_t(ctypes.Structure):
    _fields_ = [("k_t", ctypes.c_void_p), ("stride_b", ctypes.c_int64),
                ("stride_h", ctypes.c_int64), ("stride_d", ctypes.c_int64)]


class santa_options_t(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("splits", ctypes.c_int32)]


class santa_plan_info_t(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("splits", ctypes.c_int32),
                ("split_len", ctypes.c_int32), ("workspace", ctypes.c_size_t),
                ("kernels", ctypes.c_char_p)]


_lib: Optional[ctypes.CDLL] = None


def load() -> ctypes.CDLL:
    """Load the in-tree libsanta.so; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(python -m paper_2605_01910_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    SP, KP, TP = ctypes.POINTER(santa_shape_t), ctypes.POINTER(santa_kv_t), ctypes.POINTER(santa_kt_t)
    L.santa_workspace_size.argtypes = [SP, KP, I32, I32]
    L.santa_workspace_size.restype = SZ
    L.santa_workspace_init.argtypes = [P, SZ, P]
    L.santa_decode_dense.argtypes = [P, KP, SP, ctypes.c_float, P, P, SZ, P]
    L.santa_decode_systematic.argtypes = [P, KP, SP, ctypes.c_float, I32, P, P, P, P, SZ, P]
    L.santa_decode_stratified.argtypes = [P, KP, SP, ctypes.c_float, I32, P, P, P, P, SZ, P]
    L.santa_decode_stratified_noalloc.argtypes = [P, KP, SP, ctypes.c_float, I32, P, P, P, P]
    L.santa_decode_bernoulli_qk.argtypes = [P, TP, KP, SP, ctypes.c_float, I32, I32, P, I32, P,
                                            P, P, P, P, SZ, P]
    L.santa_decode_flash.argtypes = [P, KP, SP, ctypes.c_float, I32, I32, P, P, P, P, SZ, P]
    L.santa_decode_iid.argtypes = [P, KP, SP, ctypes.c_float, I32, P, P, P, P, SZ, P]
    L.santa_stream_read.argtypes = [P, SZ, P, P]
    L.santa_time_next_call.argtypes = [P, P]
    OP = ctypes.POINTER(santa_options_t)
    L.santa_set_options.argtypes = [OP]
    L.santa_get_options.argtypes = [OP]
    L.santa_plan_info.argtypes = [SP, KP, I32, I32, ctypes.POINTER(santa_plan_info_t)]
    L.santa_status_string.argtypes = [ctypes.c_int]
    L.santa_status_string.restype = ctypes.c_char_p
    L.santa_last_error.restype = ctypes.c_char_p
    for name in ("santa_workspace_init", "santa_decode_dense", "santa_decode_systematic",
                 "santa_decode_stratified", "santa_decode_bernoulli_qk", "santa_decode_flash",
                 "santa_decode_iid", "santa_stream_read", "santa_time_next_call",
                 "santa_set_options", "santa_get_options", "santa_plan_info",
                 "santa_decode_stratified_noalloc"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _status_name(s: int) -> str:
    try:
        return load().santa_status_string(int(s)).decode()
    except Exception:
        return f"status {s}"


def _check(status: int) -> None:
    if status != SANTA_OK:
        raise SantaError(status, load().santa_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SANTA_BF16
    if t.dtype == torch.float32:
        return SANTA_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


# ---------------------------------------------------------------------------
# descriptor builders (marshalling)
# ---------------------------------------------------------------------------

def shape_of(q: torch.Tensor, num_kv_heads: int) -> santa_shape_t:
    """q: [batch, num_q_heads, head_dim]."""
    B, Hq, d = q.shape
    return santa_shape_t(B, Hq, num_kv_heads, d, _dtype_code(q))


def kv_contiguous(k: torch.Tensor, v: torch.Tensor, ctx_len: Optional[torch.Tensor] = None,
                  layout: str = "nhd") -> santa_kv_t:
    """k, v: [B, n, Hkv, d] (layout 'nhd', sequence-major) or [B, Hkv, n, d] ('hnd')."""
    assert k.shape == v.shape and k.stride() == v.stride() and k.stride(-1) == 1
    if layout == "nhd":
        n = k.shape[1]
        sb, sn, sh = k.stride(0), k.stride(1), k.stride(2)
    else:
        n = k.shape[2]
        sb, sh, sn = k.stride(0), k.stride(1), k.stride(2)
    return santa_kv_t(k.data_ptr(), v.data_ptr(), sb, sn, sh,
                      None if ctx_len is None else ctx_len.data_ptr(), None, 0, 0, n)


def kv_paged(k_pages: torch.Tensor, v_pages: torch.Tensor, block_table: torch.Tensor,
             ctx_len: torch.Tensor, n_k: int) -> santa_kv_t:
    """Pools [pages, Hkv, page_size, d]; block_table int32 [B, max_pages]."""
    assert k_pages.shape == v_pages.shape and k_pages.stride(-1) == 1
    assert block_table.dtype == torch.int32 and block_table.is_contiguous()
    ps = k_pages.shape[2]
    return santa_kv_t(k_pages.data_ptr(), v_pages.data_ptr(), k_pages.stride(0),
                      k_pages.stride(2), k_pages.stride(1), ctx_len.data_ptr(),
                      block_table.data_ptr(), ps, block_table.shape[1], int(n_k))


def set_fp8_cache(kv: santa_kv_t, k_scale: torch.Tensor, v_scale: torch.Tensor) -> santa_kv_t:
    """Mark the cache of ``kv`` as OCP FP8 E4M3 codes (uint8 tensors) with
    float32 dequantisation scales [batch, num_kv_heads] for K and V."""
    assert k_scale.dtype == torch.float32 and v_scale.dtype == torch.float32
    assert k_scale.is_contiguous() and v_scale.is_contiguous()
    kv.kv_dtype = SANTA_KV_FP8_E4M3
    kv.k_scale = k_scale.data_ptr()
    kv.v_scale = v_scale.data_ptr()
    return kv


def kt_feature_major(k_t: torch.Tensor) -> santa_kt_t:
    """k_t: [B, Hkv, d, n] with keys contiguous."""
    assert k_t.stride(-1) == 1
    return santa_kt_t(k_t.data_ptr(), k_t.stride(0), k_t.stride(1), k_t.stride(2))


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def santa_workspace_size(shape: santa_shape_t, kv: santa_kv_t, S: int, kind: int) -> int:
    n = load().santa_workspace_size(ctypes.byref(shape), ctypes.byref(kv), int(S), int(kind))
    if n == 0:
        raise SantaError(SANTA_ERR_INVALID_ARG, "santa_workspace_size: invalid arguments")
    return int(n)


def santa_workspace_init(ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def workspace_error(ws: torch.Tensor) -> int:
    """The int32 at byte 0 of a workspace: nonzero when a bounded wait of a
    single-launch path gave up, which makes that call's outputs invalid.
    Reading it synchronises with the device."""
    return int(ws[:4].view(torch.int32).item())


def check_workspace(ws: torch.Tensor) -> None:
    """Raise SantaError if a bounded wait gave up in a call on this workspace."""
    flag = workspace_error(ws)
    if flag:
        raise SantaError(SANTA_ERR_HIP, f"a bounded wait gave up (workspace flag {flag}); "
                                        "the outputs of the calls since the last "
                                        "santa_workspace_init are not valid")


def alloc_workspace(shape: santa_shape_t, kv: santa_kv_t, S: int, kind: int,
                    device="cuda") -> torch.Tensor:
    """Allocate (torch caching allocator, 256-byte aligned) and initialise a workspace."""
    n = santa_workspace_size(shape, kv, S, kind)
    ws = torch.empty(n + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    ws = ws[off:off + n]
    santa_workspace_init(ws)
    return ws


def santa_decode_dense(q: torch.Tensor, kv: santa_kv_t, shape: santa_shape_t, scale: float,
                       out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_decode_dense(_ptr(q), ctypes.byref(kv), ctypes.byref(shape),
                                     float(scale), _ptr(out), _ptr(ws),
                                     ws.numel() * ws.element_size(), _stream(stream)))


def santa_decode_systematic(q: torch.Tensor, kv: santa_kv_t, shape: santa_shape_t, scale: float,
                            S: int, u: torch.Tensor, idx_out: Optional[torch.Tensor],
                            out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_decode_systematic(_ptr(q), ctypes.byref(kv), ctypes.byref(shape),
                                          float(scale), int(S), _ptr(u), _ptr(idx_out),
                                          _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                                          _stream(stream)))


def santa_decode_stratified(q: torch.Tensor, kv: santa_kv_t, shape: santa_shape_t, scale: float,
                            S: int, u: torch.Tensor, idx_out: Optional[torch.Tensor],
                            out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_decode_stratified(_ptr(q), ctypes.byref(kv), ctypes.byref(shape),
                                          float(scale), int(S), _ptr(u), _ptr(idx_out),
                                          _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                                          _stream(stream)))


def santa_decode_stratified_noalloc(q: torch.Tensor, kv: santa_kv_t, shape: santa_shape_t,
                                    scale: float, S: int, u: torch.Tensor,
                                    idx_out: Optional[torch.Tensor], out: torch.Tensor,
                                    stream=None) -> None:
    _check(load().santa_decode_stratified_noalloc(_ptr(q), ctypes.byref(kv), ctypes.byref(shape),
                                                  float(scale), int(S), _ptr(u), _ptr(idx_out),
                                                  _ptr(out), _stream(stream)))


def santa_decode_bernoulli_qk(q: torch.Tensor, kt: santa_kt_t, kv: santa_kv_t,
                              shape: santa_shape_t, scale: float, B_draws: int, mode: int,
                              u_q: torch.Tensor, S: int, u: torch.Tensor,
                              idx_out: Optional[torch.Tensor],
                              feat_mask_out: Optional[torch.Tensor], out: torch.Tensor,
                              ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_decode_bernoulli_qk(_ptr(q), ctypes.byref(kt), ctypes.byref(kv),
                                            ctypes.byref(shape), float(scale), int(B_draws),
                                            int(mode), _ptr(u_q), int(S), _ptr(u), _ptr(idx_out),
                                            _ptr(feat_mask_out), _ptr(out), _ptr(ws),
                                            ws.numel() * ws.element_size(), _stream(stream)))


def santa_decode_iid(q: torch.Tensor, kv: santa_kv_t, shape: santa_shape_t, scale: float,
                     S: int, u: torch.Tensor, idx_out: Optional[torch.Tensor], out: torch.Tensor,
                     ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_decode_iid(_ptr(q), ctypes.byref(kv), ctypes.byref(shape), float(scale),
                                   int(S), _ptr(u), _ptr(idx_out), _ptr(out), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)))


def santa_decode_flash(q: torch.Tensor, kv: santa_kv_t, shape: santa_shape_t, scale: float,
                       tile: int, S_tile: int, u: torch.Tensor, idx_out: Optional[torch.Tensor],
                       out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(load().santa_decode_flash(_ptr(q), ctypes.byref(kv), ctypes.byref(shape),
                                     float(scale), int(tile), int(S_tile), _ptr(u), _ptr(idx_out),
                                     _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                                     _stream(stream)))


def santa_set_options(path: int = SANTA_PATH_AUTO, splits: int = 0) -> None:
    """Launch options of the calling thread (see santa_options_t)."""
    _check(load().santa_set_options(ctypes.byref(santa_options_t(int(path), int(splits)))))


def santa_get_options() -> tuple:
    o = santa_options_t()
    _check(load().santa_get_options(ctypes.byref(o)))
    return o.path, o.splits


@contextlib.contextmanager
def options(path="auto", splits: int = 0):
    """Context manager: run the body under launch options (path: a
    SANTA_PATH_* code or one of "auto", "one", "two", "multi"), restoring the
    thread's previous options afterwards."""
    prev = santa_get_options()
    santa_set_options(PATHS[path] if isinstance(path, str) else path, splits)
    try:
        yield
    finally:
        santa_set_options(*prev)


def santa_plan_info(shape: santa_shape_t, kv: santa_kv_t, S: int, kind: int) -> dict:
    info = santa_plan_info_t()
    _check(load().santa_plan_info(ctypes.byref(shape), ctypes.byref(kv), int(S), int(kind),
                                  ctypes.byref(info)))
    return {"path": info.path, "splits": info.splits, "split_len": info.split_len,
            "workspace": int(info.workspace), "kernels": info.kernels.decode()}


def santa_stream_read(buf, sink, stream=None) -> None:
    """Stream all bytes of the CUDA tensor `buf` (16-byte aligned, a multiple of
    16 bytes) through the decode kernels' key load; `sink` is an int32 CUDA
    tensor of STREAM_READ_GROUPS words whose first words receive each
    workgroup's XOR fold of what it read (the rest keep their contents).  A measurement helper: timed with santa_time_next_call, it
    gives the attainable read rate for that many bytes."""
    if not (buf.is_cuda and sink.is_cuda):
        raise ValueError("buf and sink must be CUDA tensors")
    if sink.dtype != torch.int32 or sink.numel() < STREAM_READ_GROUPS or not sink.is_contiguous():
        raise ValueError(f"sink must be a contiguous int32 tensor of >= {STREAM_READ_GROUPS} words")
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    _check(load().santa_stream_read(ctypes.c_void_p(buf.data_ptr()),
                                    ctypes.c_size_t(buf.numel() * buf.element_size()),
                                    ctypes.c_void_p(sink.data_ptr()), _stream(stream)))


def santa_time_next_call(start, stop) -> None:
    """Attach two timing events to the kernels of the next santa_decode_* (or
    santa_stream_read) call on this thread (start: first kernel dispatched, stop: last kernel done).
    `start`/`stop` are torch.cuda.Event objects that have been recorded at least
    once (so their HIP event exists), raw hipEvent_t handles, or both None."""
    def handle(e):
        if e is None:
            return None
        h = e.cuda_event if hasattr(e, "cuda_event") else int(e)
        if not h:
            raise ValueError("event has no HIP handle yet: record it once first")
        return ctypes.c_void_p(h)
    _check(load().santa_time_next_call(handle(start), handle(stop)))

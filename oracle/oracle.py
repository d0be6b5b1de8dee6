"""ctypes wrapper of the double-precision CPU oracle (santa_oracle.c).

TEST INFRASTRUCTURE ONLY: the tests, the package smoke check and the
benchmark's CPU-baseline leg are its only users.  The GPU library never loads
it and it never loads the GPU library.  See santa_oracle.c for the paper
passages each step follows and for the readings of points the paper leaves
open.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "santa_oracle.c")
LIB = os.path.join(HERE, "libsanta_oracle.so")

DENSE, SYSTEMATIC, STRATIFIED, IID, BERNOULLI_SYS, IID_SPACINGS = range(6)
KIND = {"dense": DENSE, "systematic": SYSTEMATIC, "stratified": STRATIFIED, "iid": IID,
        "bernoulli": BERNOULLI_SYS, "iid_spacings": IID_SPACINGS}


def build(verbose: bool = False) -> str:
    """Compile the oracle with gcc (portable -O2, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-o", LIB + ".tmp", SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


class _Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("d", ctypes.c_int32), ("n_max", ctypes.c_int32), ("is_f32", ctypes.c_int32),
                ("q", ctypes.c_void_p), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("sb", ctypes.c_int64), ("sn", ctypes.c_int64), ("sh", ctypes.c_int64),
                ("ctx_len", ctypes.c_void_p), ("scale", ctypes.c_double),
                ("kv_fp8", ctypes.c_int32), ("k_scale", ctypes.c_void_p),
                ("v_scale", ctypes.c_void_p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
            build()
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        L.orc_scores.argtypes = [P, ctypes.c_int, P, ctypes.c_int, ctypes.c_int64, ctypes.c_int,
                                 ctypes.c_double, P]
        L.orc_softmax.argtypes = [P, ctypes.c_int, P]
        L.orc_weighted_sum.argtypes = [P, P, ctypes.c_int, ctypes.c_int64, ctypes.c_int,
                                       ctypes.c_int, P]
        L.orc_cdf.argtypes = [P, ctypes.c_int, P]
        L.orc_thresholds.argtypes = [ctypes.c_int, P, ctypes.c_int, P]
        L.orc_inverse_cdf.argtypes = [P, ctypes.c_int, P, ctypes.c_int, P]
        L.orc_gather_mean.argtypes = [P, ctypes.c_int, ctypes.c_int64, ctypes.c_int, P,
                                      ctypes.c_int, P]
        L.orc_bernoulli_weights.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int, P,
                                            ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P]
        L.orc_decode.argtypes = [ctypes.POINTER(_Problem), ctypes.c_int, ctypes.c_int, P, P,
                                 ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, P, P, P,
                                 P, P, P]
        L.orc_decode.restype = ctypes.c_int
        L.orc_flash.argtypes = [P, P, ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, ctypes.c_int, P, P, P, P, P, P]
        L.orc_decode_flash.argtypes = [ctypes.POINTER(_Problem), ctypes.c_int, ctypes.c_int, P,
                                       ctypes.c_int, P, P, P, P, P]
        L.orc_decode_flash.restype = ctypes.c_int
        L.orc_fp8_e4m3_decode.argtypes = [P, ctypes.c_int64, P]
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _elem(a: np.ndarray):
    """(contiguous array, element kind) for bfloat16 bits (uint16, 0), float32
    (1) or float64 (2) input."""
    if a.dtype == np.uint16:
        return np.ascontiguousarray(a), 0
    if a.dtype == np.float64:
        return np.ascontiguousarray(a), 2
    return np.ascontiguousarray(a, dtype=np.float32), 1


def fp8_e4m3_decode(codes: np.ndarray) -> np.ndarray:
    """OCP FP8 E4M3 codes (uint8) -> float64 values, elementwise."""
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    out = np.empty(c.shape, dtype=np.float64)
    lib().orc_fp8_e4m3_decode(_p(c), c.size, _p(out))
    return out


# --------------------------------------------------------------------------
# single steps (one query row)
# --------------------------------------------------------------------------

def scores(w: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """s_j = scale * <w, k_j> for a query ``w`` (float64 [d]) and keys ``k`` [L, d]."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    k, f = _elem(k)
    L, d = k.shape
    s = np.empty(L, dtype=np.float64)
    lib().orc_scores(_p(w), d, _p(k), f, d, L, float(scale), _p(s))
    return s


def softmax(s: np.ndarray) -> np.ndarray:
    s = np.ascontiguousarray(s, dtype=np.float64)
    p = np.empty_like(s)
    lib().orc_softmax(_p(s), s.size, _p(p))
    return p


def weighted_sum(p: np.ndarray, v: np.ndarray) -> np.ndarray:
    p = np.ascontiguousarray(p, dtype=np.float64)
    v, f = _elem(v)
    L, d = v.shape
    out = np.empty(d, dtype=np.float64)
    lib().orc_weighted_sum(_p(p), _p(v), f, d, L, d, _p(out))
    return out


def cdf(p: np.ndarray) -> np.ndarray:
    p = np.ascontiguousarray(p, dtype=np.float64)
    C = np.empty_like(p)
    lib().orc_cdf(_p(p), p.size, _p(C))
    return C


def thresholds(scheme: str, u: np.ndarray, S: int) -> np.ndarray:
    """scheme in {'systematic', 'stratified', 'iid', 'iid_spacings'}; u float32
    ([1], [S], or [S+1] for 'iid_spacings')."""
    code = {"systematic": 0, "stratified": 1, "iid": 2, "iid_spacings": 3}[scheme]
    u = np.ascontiguousarray(u, dtype=np.float32).reshape(-1)
    T = np.empty(S, dtype=np.float64)
    lib().orc_thresholds(code, _p(u), S, _p(T))
    return T


def inverse_cdf(C: np.ndarray, T: np.ndarray) -> np.ndarray:
    C = np.ascontiguousarray(C, dtype=np.float64)
    T = np.ascontiguousarray(T, dtype=np.float64)
    idx = np.empty(T.size, dtype=np.int32)
    lib().orc_inverse_cdf(_p(C), C.size, _p(T), T.size, _p(idx))
    return idx


def gather_mean(v: np.ndarray, idx: np.ndarray) -> np.ndarray:
    v, f = _elem(v)
    L, d = v.shape
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    out = np.empty(d, dtype=np.float64)
    lib().orc_gather_mean(_p(v), f, d, d, _p(idx), idx.size, _p(out))
    return out


def bernoulli_weights(q: np.ndarray, u: np.ndarray, B: int, mode: int, iid: bool = False):
    """q: [G, d] (bf16 bits or float32); u: per-head [G, d*(B if iid else 1)] for
    mode 0, [d*(B if iid else 1)] for mode 1.  Returns (w [G, d] float64, mask [d] uint8)."""
    q, f = _elem(q)
    G, d = q.shape
    u = np.ascontiguousarray(u, dtype=np.float32)
    w = np.empty((G, d), dtype=np.float64)
    mask = np.empty(d, dtype=np.uint8)
    lib().orc_bernoulli_weights(_p(q), f, G, d, _p(u), int(B), int(iid), int(mode), _p(w),
                                _p(mask))
    return w, mask


def flash(s: np.ndarray, v: np.ndarray, tile: int, S_tile: int, a: np.ndarray):
    """S2ANTA-flash on one row: scores ``s`` [L], values ``v`` [L, d], per-tile
    uniforms ``a`` [ceil(L/tile)].  Returns (out [d], idx [T, S_tile],
    tile weights W_t/Z [T], tile estimates O_t [T, d], tile-local CDF [L])."""
    s = np.ascontiguousarray(s, dtype=np.float64)
    v, f = _elem(v)
    L, d = v.shape
    T = (L + tile - 1) // tile
    a = np.ascontiguousarray(a, dtype=np.float32).reshape(-1)
    assert a.size >= T
    out = np.empty(d, dtype=np.float64)
    idx = np.empty((T, S_tile), dtype=np.int32)
    wt = np.empty(T, dtype=np.float64)
    to = np.empty((T, d), dtype=np.float64)
    C = np.empty(L, dtype=np.float64)
    lib().orc_flash(_p(s), _p(v), f, d, L, d, int(tile), int(S_tile), _p(a), _p(idx), _p(out),
                    _p(wt), _p(to), _p(C))
    return out, idx, wt, to, C


# --------------------------------------------------------------------------
# batch driver
# --------------------------------------------------------------------------

class Result:
    def __init__(self, out, idx, cdf, w, mask, rows, threads):
        self.out, self.idx, self.cdf, self.w, self.mask = out, idx, cdf, w, mask
        self.rows, self.threads = rows, threads


def _problem(q, k, v, ctx_len, scale, k_scale, v_scale):
    """The C problem struct (and the arrays it points to, kept alive by the
    caller).  k and v hold q's element type, or FP8 E4M3 codes (uint8) with
    k_scale / v_scale float32 [B, Hkv]."""
    q, f = _elem(q)
    B, Hq, d = q.shape
    if k.dtype == np.uint8:
        assert v.dtype == np.uint8 and k_scale is not None and v_scale is not None
        k, v = np.ascontiguousarray(k), np.ascontiguousarray(v)
        ks = np.ascontiguousarray(k_scale, dtype=np.float32).reshape(-1)
        vs = np.ascontiguousarray(v_scale, dtype=np.float32).reshape(-1)
        fp8 = 1
    else:
        k, fk = _elem(k)
        v, fv = _elem(v)
        assert f == fk == fv, "q, k and v must share one element type"
        ks = vs = None
        fp8 = 0
    _, n, Hkv, _ = k.shape
    assert ks is None or ks.size == B * Hkv
    ctx = np.ascontiguousarray(ctx_len, dtype=np.int32)
    P = _Problem(B, Hq, Hkv, d, n, f, q.ctypes.data, k.ctypes.data, v.ctypes.data,
                 n * Hkv * d, Hkv * d, d, ctx.ctypes.data, float(scale), fp8,
                 None if ks is None else ks.ctypes.data, None if vs is None else vs.ctypes.data)
    return P, (q, k, v, ctx, ks, vs)


def decode(kind: str, q: np.ndarray, k: np.ndarray, v: np.ndarray, ctx_len: np.ndarray,
           scale: float, S: int = 0, u: Optional[np.ndarray] = None,
           u_q: Optional[np.ndarray] = None, B_draws: int = 1, mode: int = 0,
           iid_draws: bool = False, rows: Optional[Sequence[int]] = None,
           want_cdf: bool = False, want_weights: bool = False,
           k_scale: Optional[np.ndarray] = None, v_scale: Optional[np.ndarray] = None) -> Result:
    """One decode step over logical caches ``k``/``v`` of shape [B, n, Hkv, d]
    for the rows ``b*Hq + h`` listed in ``rows`` (all rows if None).  An FP8
    cache holds uint8 E4M3 codes with scales ``k_scale``/``v_scale`` [B, Hkv]."""
    P, keep = _problem(q, k, v, ctx_len, scale, k_scale, v_scale)
    q = keep[0]
    B, Hq, d = q.shape
    n = keep[1].shape[1]
    rows_a = None if rows is None else np.ascontiguousarray(rows, dtype=np.int32)
    nr = B * Hq if rows_a is None else rows_a.size
    out = np.empty((nr, d), dtype=np.float64)
    code = KIND[kind]
    idx = np.empty((nr, max(S, 1)), dtype=np.int32) if code != DENSE else None
    C = np.full((nr, n), np.nan, dtype=np.float64) if want_cdf and code != DENSE else None
    w = np.empty((nr, d), dtype=np.float64) if want_weights and code == BERNOULLI_SYS else None
    mk = np.empty((nr, d), dtype=np.uint8) if want_weights and code == BERNOULLI_SYS else None
    uu = None if u is None else np.ascontiguousarray(u, dtype=np.float32)
    uq = None if u_q is None else np.ascontiguousarray(u_q, dtype=np.float32)
    threads = lib().orc_decode(ctypes.byref(P), code, int(S), _p(uu), _p(uq), int(B_draws),
                               int(mode), int(iid_draws), 0 if rows_a is None else nr,
                               _p(rows_a), _p(out), _p(idx), _p(C), _p(w), _p(mk))
    return Result(out, idx, C, w, mk, rows_a, threads)


def decode_workload(wl, kind: Optional[str] = None, rows: Optional[Sequence[int]] = None,
                    want_cdf: bool = False, want_weights: bool = False) -> Result:
    """Run the oracle on a ``workload.Workload``.  Paged workloads are read
    through their logical per-sequence arrays (never through the page pool), so
    the GPU's page-table indirection is checked independently."""
    kind = kind or wl.kind
    if kind == "flash":
        return _decode_workload_flash(wl, rows, want_cdf)
    if kind == "iid":  # the workload's i.i.d. uniforms are S + 1 per row (spacings)
        kind = "iid_spacings"
    S = wl.S if kind != "dense" else 0
    ks, vs = getattr(wl, "k_scale", None), getattr(wl, "v_scale", None)
    if not wl.paged:
        return decode(kind, wl.q, wl.k, wl.v, wl.ctx_len, wl.scale, S, wl.u, wl.u_q, wl.B_draws,
                      wl.mode, False, rows, want_cdf, want_weights, ks, vs)
    # paged: one sequence at a time through its logical arrays, all of its
    # listed rows in one call
    all_rows = list(range(wl.B * wl.Hq)) if rows is None else list(rows)
    by_b = {}
    for i, r in enumerate(all_rows):
        by_b.setdefault(r // wl.Hq, []).append(i)
    nr = len(all_rows)
    out = np.empty((nr, wl.d))
    idx = np.empty((nr, max(S, 1)), np.int32) if kind != "dense" else None
    cdf = np.full((nr, wl.n_max), np.nan) if want_cdf and kind != "dense" else None
    threads = 1
    for b, pos in by_b.items():
        kb, vb = wl.logical_kv(b)
        L = int(wl.ctx_len[b])
        kk = kb.reshape(1, L, wl.Hkv, wl.d)
        vv = vb.reshape(1, L, wl.Hkv, wl.d)
        ub = None if wl.u is None else wl.u[b:b + 1]
        heads = [all_rows[i] % wl.Hq for i in pos]
        res = decode(kind, wl.q[b:b + 1], kk, vv, np.array([L], np.int32), wl.scale, S, ub, None,
                     wl.B_draws, wl.mode, False, heads, want_cdf, False,
                     None if ks is None else ks[b:b + 1], None if vs is None else vs[b:b + 1])
        threads = max(threads, res.threads)
        out[pos] = res.out
        if idx is not None:
            idx[pos] = res.idx
        if cdf is not None:
            cdf[pos, :L] = res.cdf
    return Result(out, idx, cdf, None, None, np.asarray(all_rows, np.int32), threads)


def decode_flash(q: np.ndarray, k: np.ndarray, v: np.ndarray, ctx_len: np.ndarray, scale: float,
                 tile: int, S_tile: int, u: np.ndarray, rows: Optional[Sequence[int]] = None,
                 want_cdf: bool = False, k_scale: Optional[np.ndarray] = None,
                 v_scale: Optional[np.ndarray] = None) -> Result:
    """S2ANTA-flash over logical caches [B, n, Hkv, d]; ``u`` is [B, Hq,
    ceil(n/tile)].  Result.idx is [rows, T_max*S_tile] (-1 past a row's tiles),
    Result.w the tile weights [rows, T_max]."""
    P, keep = _problem(q, k, v, ctx_len, scale, k_scale, v_scale)
    q = keep[0]
    B, Hq, d = q.shape
    n = keep[1].shape[1]
    Tm = (n + tile - 1) // tile
    rows_a = None if rows is None else np.ascontiguousarray(rows, dtype=np.int32)
    nr = B * Hq if rows_a is None else rows_a.size
    uu = np.ascontiguousarray(u, dtype=np.float32).reshape(-1)
    assert uu.size >= B * Hq * Tm
    out = np.empty((nr, d), dtype=np.float64)
    idx = np.empty((nr, Tm * S_tile), dtype=np.int32)
    wt = np.empty((nr, Tm), dtype=np.float64)
    C = np.full((nr, n), np.nan, dtype=np.float64) if want_cdf else None
    threads = lib().orc_decode_flash(ctypes.byref(P), int(tile), int(S_tile), _p(uu),
                                     0 if rows_a is None else nr, _p(rows_a), _p(out), _p(idx),
                                     _p(wt), _p(C))
    return Result(out, idx, C, wt, None, rows_a, threads)


def _decode_workload_flash(wl, rows, want_cdf) -> Result:
    """decode_workload for kind="flash": contiguous workloads in one batch
    call, paged ones one sequence at a time through their logical arrays."""
    ks, vs = getattr(wl, "k_scale", None), getattr(wl, "v_scale", None)
    if not wl.paged:
        return decode_flash(wl.q, wl.k, wl.v, wl.ctx_len, wl.scale, wl.tile, wl.S_tile, wl.u,
                            rows, want_cdf, ks, vs)
    all_rows = list(range(wl.B * wl.Hq)) if rows is None else list(rows)
    Tm = (wl.n_max + wl.tile - 1) // wl.tile
    outs, idxs, threads = [], [], 1
    for r in all_rows:
        b, h = divmod(r, wl.Hq)
        kb, vb = wl.logical_kv(b)
        L = int(wl.ctx_len[b])
        T = (L + wl.tile - 1) // wl.tile
        res = decode_flash(wl.q[b:b + 1], kb.reshape(1, L, wl.Hkv, wl.d),
                           vb.reshape(1, L, wl.Hkv, wl.d), np.array([L], np.int32), wl.scale,
                           wl.tile, wl.S_tile, np.ascontiguousarray(wl.u[b:b + 1, :, :T]), [h],
                           False, None if ks is None else ks[b:b + 1],
                           None if vs is None else vs[b:b + 1])
        threads = max(threads, res.threads)
        ix = np.full(Tm * wl.S_tile, -1, np.int32)
        ix[:T * wl.S_tile] = res.idx[0][:T * wl.S_tile]
        outs.append(res.out[0])
        idxs.append(ix)
    return Result(np.array(outs), np.array(idxs), None, None, None,
                  np.asarray(all_rows, np.int32), threads)

"""Helpers for the GPU parity tests: move a seeded workload to the device, run
one entry point through the C ABI, and compare with the CPU oracle under the
acceptance rules:

  indices  bit-exact, except that index g is also accepted for threshold T
           when F(g-1) - 1e-5 <= T < F(g) + 1e-5 (F: the oracle's float64 CDF)
  dense    max |out - oracle| <= 2e-2 and relative L2 <= 5e-3
  sampled  max |out - oracle_gather(GPU indices)| <= 2e-2
"""

from __future__ import annotations

import sys
from typing import Optional, Sequence

import numpy as np
import torch

from oracle import oracle as O
from paper_2605_01910_amd import santa as S
from workload.device import DeviceWorkload, current_rows, dev_elems  # noqa: F401

BAND = 1e-5
DENSE_MAX_ABS, DENSE_REL_L2, SAMPLED_MAX_ABS = 2e-2, 5e-3, 2e-2
KIND_CODE = {"dense": S.SANTA_KIND_DENSE, "systematic": S.SANTA_KIND_SYSTEMATIC,
             "stratified": S.SANTA_KIND_STRATIFIED, "bernoulli": S.SANTA_KIND_BERNOULLI,
             "flash": S.SANTA_KIND_FLASH, "iid": S.SANTA_KIND_IID}


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def run(w, kind: Optional[str] = None, layout: str = "nhd", want_idx: bool = True,
        dw: Optional[DeviceWorkload] = None, ws: Optional[torch.Tensor] = None,
        want_mask: bool = False):
    """Run one decode step on the GPU; returns (out float64 [rows, d], idx or None, mask)."""
    kind = kind or w.kind
    dw = dw or DeviceWorkload(w, layout)
    out = torch.empty_like(dw.q)
    Sn = w.S if kind != "dense" else 0
    if ws is None:
        ws = S.alloc_workspace(dw.shape, dw.kv, max(Sn, 1), KIND_CODE[kind])
    idx = None
    if kind == "flash":
        Sn = ((w.n_max + w.tile - 1) // w.tile) * w.S_tile  # draws per row, tile by tile
    if want_idx and kind != "dense":
        idx = torch.full((w.B, w.Hq, Sn), -7, dtype=torch.int32, device="cuda")
    mask = None
    if kind == "dense":
        S.santa_decode_dense(dw.q, dw.kv, dw.shape, w.scale, out, ws)
    elif kind == "systematic":
        S.santa_decode_systematic(dw.q, dw.kv, dw.shape, w.scale, Sn, dw.u, idx, out, ws)
    elif kind == "stratified":
        S.santa_decode_stratified(dw.q, dw.kv, dw.shape, w.scale, Sn, dw.u, idx, out, ws)
    elif kind == "flash":
        S.santa_decode_flash(dw.q, dw.kv, dw.shape, w.scale, w.tile, w.S_tile, dw.u, idx, out, ws)
    elif kind == "iid":
        S.santa_decode_iid(dw.q, dw.kv, dw.shape, w.scale, Sn, dw.u, idx, out, ws)
    elif kind == "bernoulli":
        if want_mask:
            mask = torch.full((w.B, w.Hkv, w.d), 7, dtype=torch.uint8, device="cuda")
        S.santa_decode_bernoulli_qk(dw.q, dw.kt, dw.kv, dw.shape, w.scale, w.B_draws, w.mode,
                                    dw.u_q, Sn, dw.u, idx, mask, out, ws)
    torch.cuda.synchronize()
    S.check_workspace(ws)  # no bounded wait of the call gave up
    o = out.float().cpu().numpy().astype(np.float64).reshape(w.B * w.Hq, w.d)
    ix = None if idx is None else idx.cpu().numpy().reshape(w.B * w.Hq, Sn)
    mk = None if mask is None else mask.cpu().numpy()
    return o, ix, mk


def value_rows(w, b: int, kvh: int) -> np.ndarray:
    """V rows of sequence b, KV head kvh as the oracle reads them: the stored
    elements, or for an FP8 cache their decoded values times the head's scale
    (float64)."""
    _, vb = w.logical_kv(b)
    v = np.ascontiguousarray(vb[:, kvh, :])
    if getattr(w, "kv_dtype", "") == "fp8":
        return O.fp8_e4m3_decode(v) * np.float64(w.v_scale[b, kvh])
    return v


def check_dense(w, out: np.ndarray, rows: Optional[Sequence[int]] = None) -> dict:
    res = O.decode_workload(w, "dense", rows=rows)
    sel = out if rows is None else out[np.asarray(rows)]
    err = np.abs(sel - res.out)
    rel = float(np.linalg.norm(sel - res.out) / max(np.linalg.norm(res.out), 1e-300))
    assert np.all(np.isfinite(sel)), "non-finite GPU output"
    assert err.max() <= DENSE_MAX_ABS, f"dense max abs error {err.max():.3e}"
    assert rel <= DENSE_REL_L2, f"dense relative L2 error {rel:.3e}"
    return {"max_abs": float(err.max()), "rel_l2": rel}


def _thresholds(w, kind: str, row: int) -> np.ndarray:
    if kind == "stratified":
        return O.thresholds("stratified", w.u.reshape(-1, w.S)[row], w.S)
    if kind == "iid":
        return O.thresholds("iid_spacings", w.u.reshape(-1, w.S + 1)[row], w.S)
    return O.thresholds("systematic", w.u.reshape(-1)[row:row + 1], w.S)


def check_sampled(w, out: np.ndarray, idx: np.ndarray, kind: Optional[str] = None,
                  rows: Optional[Sequence[int]] = None, exact: bool = False) -> dict:
    """Band-rule check of every index (exact: every index equal to the
    oracle's, no band) and gather check of every output row."""
    kind = kind or w.kind
    rows = list(range(w.B * w.Hq)) if rows is None else list(rows)
    res = O.decode_workload(w, kind, rows=rows, want_cdf=True)
    band, worst = 0, 0.0
    for i, r in enumerate(rows):
        b, h = divmod(r, w.Hq)
        L = int(w.ctx_len[b])
        g = idx[r]
        if L == 0:
            assert np.all(g == -1) and np.all(out[r] == 0), f"row {r}: empty row convention"
            continue
        assert np.all((g >= 0) & (g < L)), f"row {r}: index out of range {g.min()}..{g.max()}"
        o_idx = res.idx[i]
        C = res.cdf[i, :L]
        T = _thresholds(w, kind if kind in ("stratified", "iid") else "systematic", r)
        diff = np.nonzero(g != o_idx)[0]
        if exact:
            assert diff.size == 0, (f"row {r}: {diff.size} indices differ from the oracle, first "
                                    f"sample {diff[0] if diff.size else -1}")
        for m in diff:
            gm = int(g[m])
            lo = C[gm - 1] if gm > 0 else 0.0
            ok = lo - BAND <= T[m] < C[gm] + BAND
            assert ok, (f"row {r} sample {m}: GPU index {gm}, oracle {o_idx[m]}, T={T[m]!r}, "
                        f"F(g-1)={lo!r}, F(g)={C[gm]!r}")
        band += len(diff)
        ref = O.gather_mean(value_rows(w, b, h // w.G), g)
        e = float(np.abs(out[r] - ref).max())
        worst = max(worst, e)
        assert e <= SAMPLED_MAX_ABS, f"row {r}: sampled max abs error {e:.3e}"
    return {"band_accepted": band, "max_abs": worst, "rows": len(rows)}


def check_flash(w, out: np.ndarray, idx: np.ndarray, rows: Optional[Sequence[int]] = None) -> dict:
    """S2ANTA-flash acceptance: every drawn index equals the oracle's or lies
    within 1e-5 of its threshold on the tile-local CDF (band rule); tiles past
    a row's length hold -1; each output row matches the oracle's merge
    sum_t (W_t/Z) (1/S_tile) sum_i V[g_{t,i}] of the GPU's own draws within
    2e-2."""
    rows = list(range(w.B * w.Hq)) if rows is None else list(rows)
    tile, St = w.tile, w.S_tile
    Tm = (w.n_max + tile - 1) // tile
    band, worst = 0, 0.0
    for r in rows:
        b, h = divmod(r, w.Hq)
        L = int(w.ctx_len[b])
        g = idx[r].reshape(Tm, St)
        if L == 0:
            assert np.all(g == -1) and np.all(out[r] == 0), f"row {r}: empty row convention"
            continue
        kb, vb = w.logical_kv(b)
        T = (L + tile - 1) // tile
        assert np.all(g[T:] == -1), f"row {r}: draws past the row's tiles"
        fp8 = getattr(w, "kv_dtype", "") == "fp8"
        res = O.decode_flash(w.q[b:b + 1], kb.reshape(1, L, w.Hkv, w.d), vb.reshape(1, L, w.Hkv, w.d),
                             np.array([L], np.int32), w.scale, tile, St,
                             w.u[b:b + 1, :, :T].copy() if w.u.shape[2] != T else w.u[b:b + 1],
                             rows=[h], want_cdf=True,
                             k_scale=w.k_scale[b:b + 1] if fp8 else None,
                             v_scale=w.v_scale[b:b + 1] if fp8 else None)
        o_idx = res.idx[0].reshape(-1, St)[:T]
        C = res.cdf[0]
        wt = res.w[0][:T]
        for t in range(T):
            t0 = t * tile
            n = min(tile, L - t0)
            gt = g[t]
            assert np.all((gt >= t0) & (gt < t0 + n)), f"row {r} tile {t}: index outside the tile"
            for i in np.nonzero(gt != o_idx[t])[0]:
                j = int(gt[i]) - t0
                x = (i + float(w.u[b, h, t])) / St
                lo = C[t0 + j - 1] if j > 0 else 0.0
                ok = lo - BAND <= x < C[t0 + j] + BAND
                assert ok, f"row {r} tile {t} draw {i}: GPU {gt[i]}, oracle {o_idx[t][i]}, x={x!r}"
                band += 1
        ref = np.zeros(w.d)
        vk = value_rows(w, b, h // w.G)
        for t in range(T):
            ref += wt[t] * O.gather_mean(np.ascontiguousarray(vk), g[t])
        e = float(np.abs(out[r] - ref).max())
        worst = max(worst, e)
        assert e <= SAMPLED_MAX_ABS, f"row {r}: flash max abs error {e:.3e}"
    return {"band_accepted": band, "max_abs": worst, "rows": len(rows)}

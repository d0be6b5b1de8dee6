"""Seeded synthetic workloads for one decode step of SANTA / S2ANTA attention.

Every array is drawn from ``numpy.random.default_rng(SeedSequence([cfg, stream,
seed, ...]))`` with one stream per kind of input, so a workload is a pure
function of ``(cfg, seed, overrides)``:

    stream 0  query vectors                   stream 4  value-stage uniforms
    stream 1  keys (one child per sequence)   stream 5  context lengths
    stream 2  values (one child per sequence) stream 6  page permutation
    stream 3  planted key positions           stream 7  Bernoulli-query uniforms

Gaussians are drawn in float32, planted in float32 and then rounded to
bfloat16 (round to nearest even).  An FP8 cache (``kv_dtype="fp8"``) instead
holds OCP FP8 E4M3 codes of the keys and values divided by a per-(batch, KV
head) scale, max |x| / 448 over that slab, rounded to nearest even (torch's
float8_e4m3fn cast); queries stay bfloat16.  Uniforms are ``rng.random(dtype=float32)``,
which lies on the 2^-24 grid of [0, 1).

The paper's decode microbenchmark feeds i.i.d. Gaussian q/K/V (Appendix
"Decode-Step Kernel Microbenchmark Details"); the configurations below keep
that and add the structure a trained model's attention has at 32k context: an
attention sink at position 0 and a few heavy keys aligned with the group's
queries.  Planting is input construction only: a key k_j receives
``delta * w`` where ``w`` is the unit vector of the group's summed queries and
``delta`` is chosen so that the mean logit boost over the group's heads equals
the requested value.

This module never computes a softmax, a CDF, a sample or an attention output.
"""

from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import numpy as np

# ---------------------------------------------------------------------------
# bfloat16 <-> float32 bit conversions (numpy has no bfloat16 dtype)
# ---------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return the
    16-bit patterns as uint16.  Inputs must be finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------------------
# The five decode-step workloads
# ---------------------------------------------------------------------------

CONFIGS = {
    # tiny fp32 correctness case: one head, sink at 0, systematic S=64
    1: dict(B=1, Hq=1, Hkv=1, d=128, n=1024, dtype="f32", kind="systematic", S=64,
            q_std=2.0, sink=8.0, heavy=0, heavy_boost=0.0),
    # Llama-3.1-8B layer at 32k context, batch 1, stratified S=256
    2: dict(B=1, Hq=32, Hkv=8, d=128, n=32768, dtype="bf16", kind="stratified", S=256,
            q_std=1.0, sink=8.0, heavy=32, heavy_boost=6.0),
    # same layer, batch 16, systematic S in {128, 256, 512}
    3: dict(B=16, Hq=32, Hkv=8, d=128, n=32768, dtype="bf16", kind="systematic", S=256,
            q_std=1.0, sink=8.0, heavy=32, heavy_boost=6.0),
    # paged cache (16-token pages, shuffled table), batch 64, ragged lengths
    4: dict(B=64, Hq=32, Hkv=8, d=128, n=65536, dtype="bf16", kind="systematic", S=256,
            q_std=1.0, sink=8.0, heavy=32, heavy_boost=6.0,
            paged=True, page_size=16, len_lo=4096, len_hi=65536),
    # Bernoulli ternary query on a feature-major key cache, systematic S=256
    5: dict(B=8, Hq=32, Hkv=8, d=128, n=32768, dtype="bf16", kind="bernoulli", S=256,
            q_std=1.0, sink=8.0, heavy=32, heavy_boost=6.0,
            B_draws=1, mode=0),
}

STREAM_Q, STREAM_K, STREAM_V, STREAM_PLANT, STREAM_U, STREAM_LEN, STREAM_PAGE, STREAM_UQ = range(8)


def _rng(cfg: int, stream: int, seed: int, *extra: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cfg, stream, seed, *extra]))


@dataclasses.dataclass
class Workload:
    """One decode step's inputs.

    Logical caches are sequence-major ``[B, n_max, Hkv, d]`` (the paper's
    ``[n_k, H_kv, d_k]`` per sequence); rows at or beyond ``ctx_len[b]`` are
    zero.  For paged workloads the logical per-sequence arrays are kept in
    ``k_seq``/``v_seq`` (``[L_b, Hkv, d]`` each) and ``k``/``v`` are None.
    Element arrays hold bfloat16 bit patterns (uint16) or float32."""

    cfg: int
    seed: int
    B: int
    Hq: int
    Hkv: int
    d: int
    n_max: int
    dtype: str
    kind: str
    S: int
    scale: float
    q: np.ndarray
    ctx_len: np.ndarray
    u: Optional[np.ndarray]
    k: Optional[np.ndarray] = None
    v: Optional[np.ndarray] = None
    k_seq: Optional[List[np.ndarray]] = None
    v_seq: Optional[List[np.ndarray]] = None
    # paged cache: pools [num_pages, Hkv, page_size, d] and table [B, max_pages]
    page_size: int = 0
    k_pages: Optional[np.ndarray] = None
    v_pages: Optional[np.ndarray] = None
    block_table: Optional[np.ndarray] = None
    # S2ANTA-flash value stage: tile length and draws per tile; u is [B, Hq, ceil(n_max/tile)]
    tile: int = 0
    S_tile: int = 0
    # Bernoulli score stage
    k_t: Optional[np.ndarray] = None          # feature-major keys [B, Hkv, d, n_pad >= n_max]
    u_q: Optional[np.ndarray] = None          # [B, Hq, d] (mode 0) or [B, Hkv, d] (mode 1)
    B_draws: int = 0
    mode: int = 0
    heavy_pos: Optional[np.ndarray] = None    # [B, Hkv, heavy] planted positions
    # FP8 E4M3 cache: k, v (or the pools) hold uint8 codes; element value =
    # scale[b, kv head] * e4m3(code)
    kv_dtype: str = ""
    k_scale: Optional[np.ndarray] = None      # float32 [B, Hkv]
    v_scale: Optional[np.ndarray] = None

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def paged(self) -> bool:
        return self.block_table is not None

    def logical_kv(self, b: int):
        """Sequence ``b``'s keys and values as ``[L_b, Hkv, d]`` arrays."""
        L = int(self.ctx_len[b])
        if self.k_seq is not None:
            return self.k_seq[b], self.v_seq[b]
        return self.k[b, :L], self.v[b, :L]

    def q_f32(self) -> np.ndarray:
        return bf16_bits_to_f32(self.q) if self.dtype == "bf16" else self.q


def _cast(x32: np.ndarray, dtype: str) -> np.ndarray:
    return f32_to_bf16_bits(x32) if dtype == "bf16" else np.ascontiguousarray(x32, dtype=np.float32)


FP8_E4M3_MAX = 448.0


def _quant_fp8(x32: np.ndarray):
    """Per-KV-head FP8 E4M3 quantisation of one sequence's keys or values
    [L, Hkv, d]: scale = max |x| / 448 over the head's slab (1 if it is all
    zero), codes = the E4M3 rounding of x / scale.  Returns (codes uint8,
    scales float32 [Hkv])."""
    import torch
    amax = np.abs(x32).max(axis=(0, 2)) if x32.shape[0] else np.zeros(x32.shape[1], np.float32)
    sc = np.where(amax > 0, amax / np.float32(FP8_E4M3_MAX), np.float32(1.0)).astype(np.float32)
    y = np.ascontiguousarray(x32 / sc[None, :, None], dtype=np.float32)
    codes = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes, sc


def _plant(keys32: np.ndarray, qf: np.ndarray, G: int, scale: float, sink: float,
           heavy_pos: Optional[np.ndarray], heavy_boost: float) -> None:
    """Add ``delta * w`` to the sink (position 0) and heavy keys, in place.

    keys32: [L, Hkv, d] float32 for one sequence; qf: [Hq, d] float32."""
    Hkv = keys32.shape[1]
    for kv in range(Hkv):
        group = qf[kv * G:(kv + 1) * G].astype(np.float64)
        w = group.sum(axis=0)
        w /= np.linalg.norm(w)
        proj = float(np.mean(group @ w))        # > 0 because w is along sum(q)
        if sink and keys32.shape[0] > 0:
            keys32[0, kv] += np.float32(sink / (scale * proj)) * w.astype(np.float32)
        if heavy_pos is not None and heavy_boost:
            delta = np.float32(heavy_boost / (scale * proj))
            for p in heavy_pos[kv]:
                if 1 <= p < keys32.shape[0]:
                    keys32[p, kv] += delta * w.astype(np.float32)


def make_workload(cfg: int, seed: int = 0, **over) -> Workload:
    """Build configuration ``cfg`` (1..5), optionally with overrides of its
    parameters (``B, Hq, Hkv, n, S, kind, dtype, sink, heavy, len_lo, len_hi,
    B_draws, mode, paged, page_size, ctx_len, kv_dtype``, and ``tile, S_tile``
    for kind="flash") for smaller test cases."""
    p = dict(CONFIGS[cfg])
    p.update(over)
    B, Hq, Hkv, d, n = p["B"], p["Hq"], p["Hkv"], p["d"], p["n"]
    dtype, kind, S = p["dtype"], p["kind"], p["S"]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    scale = float(p.get("scale", 1.0 / math.sqrt(d)))
    paged = bool(p.get("paged", False))
    kv_fp8 = p.get("kv_dtype", "") == "fp8"
    if kv_fp8 and (dtype != "bf16" or kind == "bernoulli"):
        raise ValueError("an FP8 cache goes with bfloat16 queries and no Bernoulli scores")

    # query
    qf = _rng(cfg, STREAM_Q, seed).standard_normal((B, Hq, d), dtype=np.float32)
    qf *= np.float32(p["q_std"])
    q = _cast(qf, dtype)
    qf = bf16_bits_to_f32(q) if dtype == "bf16" else q

    # context lengths
    if "ctx_len" in p and p["ctx_len"] is not None:
        ctx = np.asarray(p["ctx_len"], dtype=np.int32).reshape(B)
    elif paged:
        ctx = _rng(cfg, STREAM_LEN, seed).integers(p["len_lo"], p["len_hi"], size=B,
                                                   endpoint=True).astype(np.int32)
    else:
        ctx = np.full(B, n, dtype=np.int32)
    # paged caches are sized by their longest sequence; contiguous ones by n
    n_max = int(ctx.max()) if paged else int(max(n, int(ctx.max()) if B else 0))

    # planted positions: `heavy` distinct positions in [1, L) per (b, kv head)
    nh = int(p.get("heavy", 0))
    heavy_pos = np.full((B, Hkv, nh), -1, dtype=np.int64)   # -1: unused slot
    if nh:
        for b in range(B):
            r = _rng(cfg, STREAM_PLANT, seed, b)
            L = int(ctx[b])
            for kv in range(Hkv):
                m = min(nh, max(L - 1, 0))
                pos = np.sort(r.choice(np.arange(1, max(L, 2)), size=m, replace=False)) if m else []
                heavy_pos[b, kv, :m] = pos

    edt = np.uint8 if kv_fp8 else np.uint16 if dtype == "bf16" else np.float32
    k_seq, v_seq = [], []
    k_sc = np.ones((B, Hkv), np.float32)
    v_sc = np.ones((B, Hkv), np.float32)
    for b in range(B):
        L = int(ctx[b])
        kb = _rng(cfg, STREAM_K, seed, b).standard_normal((L, Hkv, d), dtype=np.float32)
        _plant(kb, qf[b], G, scale, float(p.get("sink", 0.0)), heavy_pos[b] if nh else None,
               float(p.get("heavy_boost", 0.0)))
        vb = _rng(cfg, STREAM_V, seed, b).standard_normal((L, Hkv, d), dtype=np.float32)
        if kv_fp8:
            kc, k_sc[b] = _quant_fp8(kb)
            vc, v_sc[b] = _quant_fp8(vb)
            k_seq.append(kc)
            v_seq.append(vc)
        else:
            k_seq.append(_cast(kb, dtype))
            v_seq.append(_cast(vb, dtype))
        del kb, vb

    w = Workload(cfg=cfg, seed=seed, B=B, Hq=Hq, Hkv=Hkv, d=d, n_max=n_max, dtype=dtype,
                 kind=kind, S=S, scale=scale, q=q, ctx_len=ctx, u=None, heavy_pos=heavy_pos)
    if kv_fp8:
        w.kv_dtype, w.k_scale, w.v_scale = "fp8", k_sc, v_sc

    if paged:
        ps = int(p["page_size"])
        npg = [(int(L) + ps - 1) // ps for L in ctx]
        total = int(sum(npg))
        perm = _rng(cfg, STREAM_PAGE, seed).permutation(total).astype(np.int32)
        max_pages = max(npg) if npg else 1
        table = np.zeros((B, max_pages), dtype=np.int32)
        kp = np.zeros((total, Hkv, ps, d), dtype=edt)
        vp = np.zeros((total, Hkv, ps, d), dtype=edt)
        off = 0
        for b in range(B):
            L = int(ctx[b])
            ids = perm[off:off + npg[b]]
            off += npg[b]
            table[b, :npg[b]] = ids
            for j, pid in enumerate(ids):
                lo, hi = j * ps, min(L, (j + 1) * ps)
                kp[pid, :, :hi - lo] = k_seq[b][lo:hi].transpose(1, 0, 2)
                vp[pid, :, :hi - lo] = v_seq[b][lo:hi].transpose(1, 0, 2)
        w.k_seq, w.v_seq = k_seq, v_seq
        w.page_size, w.k_pages, w.v_pages, w.block_table = ps, kp, vp, table
    else:
        k = np.zeros((B, n_max, Hkv, d), dtype=edt)
        v = np.zeros((B, n_max, Hkv, d), dtype=edt)
        for b in range(B):
            L = int(ctx[b])
            k[b, :L] = k_seq[b]
            v[b, :L] = v_seq[b]
        w.k, w.v = k, v
        del k_seq, v_seq

    # value-stage uniforms: one per row (systematic), S per row (stratified),
    # S + 1 per row (i.i.d. by exponential spacings) or one per row and tile (flash)
    ru = _rng(cfg, STREAM_U, seed)
    if kind in ("systematic", "bernoulli"):
        w.u = ru.random((B, Hq), dtype=np.float32)
    elif kind == "stratified":
        w.u = ru.random((B, Hq, S), dtype=np.float32)
    elif kind == "iid":
        w.u = ru.random((B, Hq, S + 1), dtype=np.float32)
    elif kind == "flash":
        w.tile = int(p.get("tile", 256))
        w.S_tile = int(p.get("S_tile", 16))
        w.u = ru.random((B, Hq, (n_max + w.tile - 1) // w.tile), dtype=np.float32)

    if kind == "bernoulli":
        w.B_draws = int(p.get("B_draws", 1))
        w.mode = int(p.get("mode", 0))
        # feature-major keys [B, Hkv, d, n_pad]; rows padded to 64 keys (128 B bf16)
        n_pad = (n_max + 63) // 64 * 64
        w.k_t = np.zeros((B, Hkv, d, n_pad), dtype=w.k.dtype)
        w.k_t[..., :n_max] = w.k.transpose(0, 2, 3, 1)
        rq = _rng(cfg, STREAM_UQ, seed)
        w.u_q = rq.random((B, Hq if w.mode == 0 else Hkv, d), dtype=np.float32)
    return w

"""Device copies of a seeded synthetic workload (workload.gen) and the C
descriptors that point at them, for the GPU tests and the benchmark.  Input
plumbing only: nothing here computes any part of the attention step."""

from __future__ import annotations

import numpy as np
import torch

from paper_2605_01910_amd import santa as S


def dev_elems(a: np.ndarray) -> torch.Tensor:
    """numpy bf16 bits (uint16), FP8 codes (uint8) or float32 -> device tensor
    of bfloat16 / uint8 / float32."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


class DeviceWorkload:
    """Device copies of a workload plus the C descriptors that point at them."""

    def __init__(self, w, layout: str = "nhd", pass_ctx: bool = True):
        self.w = w
        self.layout = layout
        self.q = dev_elems(w.q)
        self.ctx = torch.from_numpy(w.ctx_len.astype(np.int32)).cuda()
        self.u = None if w.u is None else torch.from_numpy(w.u).cuda()
        if w.paged:
            self.kp, self.vp = dev_elems(w.k_pages), dev_elems(w.v_pages)
            self.bt = torch.from_numpy(w.block_table).cuda()
            self.kv = S.kv_paged(self.kp, self.vp, self.bt, self.ctx, w.n_max)
        else:
            k, v = dev_elems(w.k), dev_elems(w.v)
            if layout == "hnd":
                k, v = k.transpose(1, 2).contiguous(), v.transpose(1, 2).contiguous()
            self.k, self.v = k, v
            self.kv = S.kv_contiguous(k, v, self.ctx if pass_ctx else None, layout)
        if w.kv_dtype == "fp8":
            self.k_scale = torch.from_numpy(w.k_scale).cuda()
            self.v_scale = torch.from_numpy(w.v_scale).cuda()
            S.set_fp8_cache(self.kv, self.k_scale, self.v_scale)
        if w.kind == "bernoulli":
            self.kt_t = dev_elems(w.k_t)
            self.kt = S.kt_feature_major(self.kt_t)
            self.u_q = torch.from_numpy(w.u_q).cuda()
        self.shape = S.shape_of(self.q, w.Hkv)


def current_rows(dw: DeviceWorkload, w):
    """Views of the cache rows at position ctx_len[b] - 1 (the current token),
    per batch: (K [Hkv, d], V [Hkv, d])."""
    out = []
    for b in range(w.B):
        L = int(w.ctx_len[b])
        if w.paged:
            page = int(w.block_table[b, (L - 1) // w.page_size])
            s = (L - 1) % w.page_size
            out.append((dw.kp[page, :, s, :], dw.vp[page, :, s, :]))
        elif dw.layout == "hnd":
            out.append((dw.k[b, :, L - 1], dw.v[b, :, L - 1]))
        else:
            out.append((dw.k[b, L - 1], dw.v[b, L - 1]))
    return out

"""Fused current-token append (App. Decode-Step Kernel Microbenchmark Details,
note on KV-cache appends): the step's key and value rows arrive in k_new /
v_new, the cache rows at ctx_len[b] - 1 hold something else, and the call must
write the rows there inside its launch and attend over them.  The output is
checked against the oracle on the true rows, and the cache rows against
k_new / v_new bit for bit."""

import numpy as np
import pytest
import torch

from paper_2605_01910_amd import santa as S
from tests.gpu_util import (KIND_CODE, DeviceWorkload, check_dense, check_flash, check_sampled,
                            current_rows, log, run)
from workload import make_workload

pytestmark = pytest.mark.gpu

CASES = {
    "sys_one_launch": (2, "systematic", dict(B=2, n=3000, S=128, ctx_len=[3000, 1777]), "one"),
    "strat_two_launch": (2, "stratified", dict(B=3, n=2500, S=64, ctx_len=[2500, 1, 999]), "two"),
    "iid_one_launch": (2, "iid", dict(B=2, n=2000, S=96, ctx_len=[2000, 640]), "one"),
    "sys_paged": (4, "systematic", dict(B=3, len_lo=700, len_hi=3000), "one"),
    "sys_paged_two_launch": (4, "systematic", dict(B=3, len_lo=700, len_hi=3000), "two"),
    "strat_scheduled": (2, "stratified", dict(B=3, n=2500, S=64, ctx_len=[2500, 1, 999]), "rows"),
    "sys_paged_scheduled": (4, "systematic", dict(B=3, len_lo=700, len_hi=3000), "rows"),
    "dense": (2, "dense", dict(B=2, n=3000, ctx_len=[3000, 1234]), "one"),
    "dense_paged": (4, "dense", dict(B=3, len_lo=900, len_hi=2600), "one"),
    "flash": (2, "flash", dict(B=2, n=3000, ctx_len=[3000, 1500]), "rows"),
    "flash_dense_kernel": (2, "flash", dict(B=2, n=3000, ctx_len=[3000, 1500]), "one"),
    "iid_scheduled": (2, "iid", dict(B=2, n=2000, S=96, ctx_len=[2000, 640]), "rows"),
    "sys_f32_no_ctx": (1, "systematic", {}, "one"),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_fused_append(case):
    cfg, kind, over, path = CASES[case]
    gen_kind = "systematic" if kind == "dense" else kind
    w = make_workload(cfg, seed=81, kind=gen_kind, **over)
    log(f"[append/{kind}/{path}] {case} cfg={cfg} {over}")
    dw = DeviceWorkload(w, pass_ctx=case != "sys_f32_no_ctx")
    rows = current_rows(dw, w)
    k_new = torch.stack([k.clone() for k, _ in rows]).contiguous()
    v_new = torch.stack([v.clone() for _, v in rows]).contiguous()
    # poison: a key aligned with the group's queries (a logit of about +36,
    # which would take nearly all the attention) and a constant value row, so
    # that reading the row before the append shows in the output as well
    qg = dw.q.float().view(w.B, w.Hkv, w.Hq // w.Hkv, -1).sum(2)
    for b, (k, v) in enumerate(rows):
        k.copy_(4.0 * torch.sign(qg[b]))
        v.fill_(-2.0)
    dw.kv.k_new, dw.kv.v_new = k_new.data_ptr(), v_new.data_ptr()
    with S.options(path if kind != "dense" else "auto"):
        out, idx, _ = run(w, kind, dw=dw)
    torch.cuda.synchronize()
    for b, (k, v) in enumerate(rows):
        assert torch.equal(k, k_new[b]) and torch.equal(v, v_new[b]), f"cache row of batch {b}"
    if kind == "dense":
        check_dense(w, out)
    elif kind == "flash":
        log(f"  {check_flash(w, out, idx)}")
    else:
        log(f"  {check_sampled(w, out, idx, kind)}")


def test_append_rejected_where_unsupported():
    """The multi-kernel path refuses the append, and k_new without v_new is
    an invalid argument; neither launches anything."""
    w = make_workload(2, B=1, n=700, kind="systematic", S=32, seed=82)
    dw = DeviceWorkload(w)
    z = torch.zeros(w.B, w.Hkv, 128, dtype=dw.k.dtype, device="cuda")
    dw.kv.k_new, dw.kv.v_new = z.data_ptr(), z.data_ptr()
    out = torch.empty_like(dw.q)
    with S.options("multi"):
        ws = S.alloc_workspace(dw.shape, dw.kv, w.S, KIND_CODE["systematic"])
        with pytest.raises(S.SantaError) as e:
            S.santa_decode_systematic(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, None, out, ws)
    assert e.value.status == S.SANTA_ERR_UNSUPPORTED
    dw.kv.v_new = None
    with pytest.raises(S.SantaError) as e:
        S.santa_decode_systematic(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, None, out, ws)
    assert e.value.status == S.SANTA_ERR_INVALID_ARG

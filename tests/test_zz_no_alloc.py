"""santa_decode_stratified_noalloc (the no-allocation form of
santa_decode_stratified, for callers that cannot allocate device memory)
against santa_decode_stratified with a caller workspace, through the C ABI:
outputs and indices bit for bit, on two calls in a row, the second with a
smaller input (fewer rows and keys, so the static array holds the first
call's data past what the second call uses), then the first shape again; a
call whose workspace would exceed the array is rejected before any launch."""

import numpy as np
import pytest
import torch

from paper_2605_01910_amd import santa as S
from tests.gpu_util import DeviceWorkload, check_sampled, log
from workload import make_workload

pytestmark = pytest.mark.gpu


def _both(w):
    dw = DeviceWorkload(w)
    ws = S.alloc_workspace(dw.shape, dw.kv, w.S, S.SANTA_KIND_STRATIFIED)
    res = []
    for noalloc in (False, True):
        out = torch.full_like(dw.q, float("nan"))
        idx = torch.full((w.B, w.Hq, w.S), -7, dtype=torch.int32, device="cuda")
        if noalloc:
            S.santa_decode_stratified_noalloc(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, idx, out)
        else:
            S.santa_decode_stratified(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, idx, out, ws)
        torch.cuda.synchronize()
        res.append((out.float().cpu().numpy().astype(np.float64).reshape(w.B * w.Hq, w.d),
                    idx.cpu().numpy().reshape(w.B * w.Hq, w.S)))
    S.check_workspace(ws)
    (o_ws, i_ws), (o_na, i_na) = res
    assert np.array_equal(i_na, i_ws), "indices differ from the workspace call"
    assert np.array_equal(o_na, o_ws), "outputs differ from the workspace call"
    return o_na, i_na


CALLS = [
    ("batch 4, 8192 keys", dict(B=4, n=8192, ctx_len=[8192, 5000, 1, 777], S=256)),
    ("batch 1, 3000 keys", dict(B=1, n=3000, S=64)),
    ("batch 4, 8192 keys again", dict(B=4, n=8192, ctx_len=[8192, 5000, 1, 777], S=256)),
]


@pytest.mark.parametrize("path", ["auto", "two", "rows"])
def test_noalloc_matches_workspace_call(path):
    with S.options(path):
        for i, (name, over) in enumerate(CALLS):
            w = make_workload(2, seed=120 + i, kind="stratified", **over)
            log(f"[noalloc/{path}] call {i}: {name}")
            out, idx = _both(w)
            check_sampled(w, out, idx)


def test_noalloc_full_batch1_shape():
    w = make_workload(2, seed=0)
    log("[noalloc] Llama-3.1-8B 32k, batch 1, stratified S=256")
    out, idx = _both(w)
    check_sampled(w, out, idx)


def test_noalloc_rejects_calls_beyond_the_array():
    """Batch 16 with 32k keys on the two-launch path needs about 37 MB; batch
    64 needs more than the 64 MiB array and is refused on the host."""
    w = make_workload(2, B=2, n=64, kind="stratified", S=8, seed=130)
    dw = DeviceWorkload(w)
    kv = S.santa_kv_t.from_buffer_copy(dw.kv)
    kv.n_k = 1 << 20          # a cache of 2^20 keys per sequence (no kernel runs)
    kv.ctx_len = None
    shape = S.santa_shape_t(64, w.Hq, w.Hkv, w.d, dw.shape.dtype)
    need = S.santa_workspace_size(shape, kv, w.S, S.SANTA_KIND_STRATIFIED)
    assert need > S.STATIC_SCRATCH_BYTES
    out = torch.empty(64, w.Hq, w.d, dtype=dw.q.dtype, device="cuda")
    q = torch.zeros_like(out)
    u = torch.zeros(64, w.Hq, w.S, device="cuda")
    with pytest.raises(S.SantaError) as e:
        S.santa_decode_stratified_noalloc(q, kv, shape, w.scale, w.S, u, None, out)
    assert e.value.status == S.SANTA_ERR_WORKSPACE

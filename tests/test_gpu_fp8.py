"""GPU parity of the FP8 E4M3 cache (one byte per key and value element,
per-(batch, KV head) dequantisation scales; q and out bfloat16) against the
CPU oracle through the C ABI.  A quantised cache is complementary to SANTA
(Sec. 1; Related Work): the kernels read half the key bytes and the
sampled value rows at one byte per element.

- Every E4M3 code decodes exactly: one-key rows whose value row repeats one
  code give that code's value as the output, bit for bit.
- Dense, systematic, stratified, i.i.d. and flash steps match the oracle
  (which decodes the codes from the format's definition) under the usual
  acceptance rules, on ragged, paged, G = 8 and both sampled paths, and at
  the full Llama-3.1-8B 32k shapes of batch 1 and batch 16.
"""

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_01910_amd import santa as S
from tests.gpu_util import check_dense, check_flash, check_sampled, log, run
from workload import make_workload

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind", ["dense", "systematic"])
def test_every_e4m3_code_decodes_exactly(kind):
    w = make_workload(2, B=256, Hq=1, Hkv=1, n=16, ctx_len=[1] * 256, kind="systematic", S=8,
                      kv_dtype="fp8", seed=101)
    w.v[:, 0, 0, :] = np.arange(256, dtype=np.uint8)[:, None]
    w.v_scale[:] = 1.0
    out, _, _ = run(w, kind)
    ref = O.fp8_e4m3_decode(np.arange(256, dtype=np.uint8))
    nan = np.isnan(ref)
    got = out[:, 0]
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan]), np.nonzero(got[~nan] != ref[~nan])
    assert np.all(out[~nan] == out[~nan][:, :1])


CASES = {
    "dense_ragged": (2, "dense", dict(B=2, n=3000, ctx_len=[3000, 1234])),
    "dense_paged": (4, "dense", dict(B=3, len_lo=900, len_hi=2600)),
    "dense_g8": (2, "dense", dict(B=1, Hq=16, Hkv=2, n=2100)),
    "sys_ragged": (2, "systematic", dict(B=2, n=3000, S=128, ctx_len=[3000, 777])),
    "strat_ragged": (2, "stratified", dict(B=2, n=2500, S=256, ctx_len=[2500, 1])),
    "sys_paged": (4, "systematic", dict(B=3, len_lo=700, len_hi=3000)),
    "strat_g8": (2, "stratified", dict(B=1, Hq=16, Hkv=2, n=2100, S=64)),
    "iid": (2, "iid", dict(B=2, n=2000, S=96, ctx_len=[2000, 640])),
    "sys_empty_row": (2, "systematic", dict(B=3, n=600, S=32, ctx_len=[600, 0, 5])),
    "flash": (2, "flash", dict(B=2, n=3000, ctx_len=[3000, 1500], tile=128, S_tile=4)),
}


@pytest.mark.parametrize("path", ["one", "two", "rows"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_fp8_parity(case, path):
    cfg, kind, over = CASES[case]
    if path == "two" and kind in ("dense", "flash"):
        pytest.skip("one launch path for dense and flash")
    gen_kind = "systematic" if kind == "dense" else kind
    w = make_workload(cfg, seed=102, kind=gen_kind, kv_dtype="fp8", **over)
    log(f"[fp8/{kind}/{path}] {case} cfg={cfg} {over}")
    with S.options(path):
        out, idx, _ = run(w, kind)
    if kind == "dense":
        log(f"  {check_dense(w, out)}")
    elif kind == "flash":
        log(f"  {check_flash(w, out, idx)}")
    else:
        log(f"  {check_sampled(w, out, idx, kind)}")


@pytest.mark.timeout(300)
def test_fp8_cfg2_full_every_row():
    w = make_workload(2, seed=0, kv_dtype="fp8")
    log(f"[fp8 full cfg2] {w.kind} S={w.S}")
    o_null, _, _ = run(w, want_idx=False)
    out, idx, _ = run(w)
    assert np.array_equal(o_null, out)
    log(f"  sampled {check_sampled(w, out, idx)}")
    d, _, _ = run(w, "dense")
    log(f"  dense {check_dense(w, d)}")


@pytest.mark.timeout(600)
def test_fp8_cfg3_full_every_row():
    w = make_workload(3, seed=0, kv_dtype="fp8")
    log(f"[fp8 full cfg3] {w.kind} S={w.S}")
    out, idx, _ = run(w)
    log(f"  sampled {check_sampled(w, out, idx)}")
    d, _, _ = run(w, "dense")
    log(f"  dense {check_dense(w, d)}")


def test_fp8_rejected_where_unsupported():
    w = make_workload(2, B=1, n=700, kind="systematic", S=32, kv_dtype="fp8", seed=103)
    from workload.device import DeviceWorkload
    dw = DeviceWorkload(w)
    out = torch.empty_like(dw.q)
    with S.options("multi"):
        with pytest.raises(S.SantaError) as e:
            ws = S.alloc_workspace(dw.shape, dw.kv, w.S, S.SANTA_KIND_SYSTEMATIC)
            S.santa_decode_systematic(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, None, out, ws)
        assert e.value.status == S.SANTA_ERR_UNSUPPORTED
    dw.kv.k_scale = None
    ws = S.alloc_workspace(dw.shape, dw.kv, w.S, S.SANTA_KIND_SYSTEMATIC)
    with pytest.raises(S.SantaError) as e:
        S.santa_decode_systematic(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, None, out, ws)
    assert e.value.status == S.SANTA_ERR_INVALID_ARG

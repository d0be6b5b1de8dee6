"""GPU edge cases of the sampled steps, against the CPU oracle through the C ABI.

- idx_out = NULL: the configuration the benchmark times writes no indices;
  its output must equal, bit for bit, the output of the same call with
  idx_out, and match the oracle's gather of those indices.
- Extreme uniforms (Sec. 2.1, "Construction": U on [0, 1/S)): u = 0 and
  u = 1 - 2^-24, systematic and every stratum of the stratified step.
- Uniform scores with S = L: systematic sampling returns every index once.
- A dominant sink (+60 and +120 logits): the other keys' mass is below
  float32 resolution (at +120 every other split's weight underflows to 0),
  so every threshold, up to the one just below 1, must take the sink; the
  indices are compared with the oracle's exactly, with no band.
- Co-residency: a decode issued while a kernel on another stream holds the
  device keeps parity and never sets the workspace's wait flag.
"""

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_01910_amd import santa as S
from tests.gpu_util import KIND_CODE, DeviceWorkload, check_sampled, log, run
from workload import make_workload

pytestmark = pytest.mark.gpu

ONE_MINUS = np.float32(1.0) - np.float32(2.0 ** -24)


def _null_vs_idx(w, kind, path="auto"):
    dw = DeviceWorkload(w)
    with S.options(path):
        ws = S.alloc_workspace(dw.shape, dw.kv, w.S, KIND_CODE[kind])
        o_null, none, _ = run(w, kind, dw=dw, ws=ws, want_idx=False)
        o_idx, idx, _ = run(w, kind, dw=dw, ws=ws)
    assert none is None
    assert np.array_equal(o_null, o_idx), "idx_out = NULL changes the output"
    return o_null, idx


@pytest.mark.timeout(300)
@pytest.mark.parametrize("kind,S_", [("stratified", 256), ("systematic", 256), ("iid", 256),
                                     ("systematic", 1024)])
def test_cfg2_full_idx_null_bitwise(kind, S_):
    w = make_workload(2, seed=0, kind=kind, S=S_)
    log(f"[idx NULL] cfg2 full {kind} S={S_}")
    out, idx = _null_vs_idx(w, kind)
    log(f"  {check_sampled(w, out, idx, kind)}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("kind", ["systematic", "iid"])
def test_cfg3_full_idx_null_bitwise(kind):
    w = make_workload(3, seed=0, kind=kind, S=256)
    log(f"[idx NULL] cfg3 full {kind} S=256")
    out, idx = _null_vs_idx(w, kind)
    log(f"  {check_sampled(w, out, idx, kind)}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("kind", ["systematic", "stratified"])
def test_cfg3_full_scheduled_idx_null_bitwise(kind):
    w = make_workload(3, seed=0, kind=kind, S=256)
    log(f"[idx NULL] cfg3 full {kind} S=256, scheduled path")
    out, idx = _null_vs_idx(w, kind, "rows")
    log(f"  {check_sampled(w, out, idx, kind)}")


@pytest.mark.parametrize("path", ["one", "two", "rows"])
@pytest.mark.parametrize("kind", ["systematic", "stratified"])
@pytest.mark.parametrize("uval", [0.0, float(ONE_MINUS)])
def test_extreme_uniforms(uval, kind, path):
    w = make_workload(2, B=2, n=6000, kind=kind, S=256, ctx_len=[6000, 2345], seed=91)
    w.u = np.full_like(w.u, np.float32(uval))
    log(f"[u={uval!r}] {kind} path={path}")
    dw = DeviceWorkload(w)
    with S.options(path):
        out, idx, _ = run(w, kind, dw=dw)
    log(f"  {check_sampled(w, out, idx, kind)}")
    # the last threshold of every row stays inside the row
    assert np.all(idx[:, -1] < np.repeat(w.ctx_len, w.Hq))


@pytest.mark.parametrize("path", ["one", "two", "rows"])
@pytest.mark.parametrize("L", [4096, 1000])
def test_uniform_scores_S_equals_L_every_index_once(L, path):
    """q = 0 makes every score 0: p is uniform, and systematic sampling with
    S = L puts exactly one threshold in every key's interval."""
    w = make_workload(2, B=1, Hq=4, Hkv=1, n=L, kind="systematic", S=L, seed=92)
    w.q = np.zeros_like(w.q)
    w.u = np.full_like(w.u, np.float32(0.5))
    with S.options(path):
        out, idx, _ = run(w, "systematic")
    for r in range(w.Hq):
        assert np.array_equal(idx[r], np.arange(L)), f"row {r}"
    check_sampled(w, out, idx, exact=True)


@pytest.mark.parametrize("path", ["one", "two", "rows"])
@pytest.mark.parametrize("kind", ["systematic", "stratified"])
@pytest.mark.parametrize("sink", [60.0, 120.0])
def test_dominant_sink_takes_every_threshold(sink, kind, path):
    w = make_workload(2, B=1, n=32768, kind=kind, S=256, sink=sink, heavy=0, seed=93)
    w.u = np.full_like(w.u, ONE_MINUS)
    ref = O.decode_workload(w, kind)
    log(f"[sink +{sink}] {kind} path={path}: oracle indices in {ref.idx.min()}..{ref.idx.max()}")
    with S.options(path):
        out, idx, _ = run(w, kind)
    if sink >= 120.0:
        assert np.all(ref.idx == 0)
        assert np.all(idx == 0)
    # the fp32 path must pick exactly the oracle's keys wherever the oracle's
    # thresholds are clear of the tail's sub-resolution mass
    log(f"  {check_sampled(w, out, idx, kind, exact=sink >= 120.0)}")


@pytest.mark.timeout(300)
def test_decode_beside_a_kernel_on_another_stream():
    """A large matrix product on a second stream occupies the device while
    the one-launch sampled and dense steps run; their workgroups may start
    late, and the bounded row waits must still complete."""
    w = make_workload(2, B=4, n=8192, kind="stratified", S=256, seed=94)
    dw = DeviceWorkload(w)
    ws = S.alloc_workspace(dw.shape, dw.kv, w.S, KIND_CODE["stratified"])
    a = torch.randn(6144, 6144, device="cuda")
    b = torch.randn(6144, 6144, device="cuda")
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    outs = []
    for rep in range(3):
        with torch.cuda.stream(side):
            for _ in range(2):
                c = a @ b
        out = torch.empty_like(dw.q)
        idx = torch.empty((w.B, w.Hq, w.S), dtype=torch.int32, device="cuda")
        S.santa_decode_stratified(dw.q, dw.kv, dw.shape, w.scale, w.S, dw.u, idx, out, ws)
        torch.cuda.synchronize()
        assert S.workspace_error(ws) == 0, f"a row wait gave up (rep {rep})"
        o = out.float().cpu().numpy().astype(np.float64).reshape(w.B * w.Hq, w.d)
        outs.append(o)
        check_sampled(w, o, idx.cpu().numpy().reshape(w.B * w.Hq, w.S))
    del c
    assert all(np.array_equal(outs[0], o) for o in outs[1:])

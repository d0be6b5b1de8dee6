"""GPU parity at the full benchmark shapes, in the launch configuration the
benchmark times (default split counts and path choice, seed 0 as in bench.py).

Every configuration is checked on every row, configuration 4 (paged, 64
sequences of 4k..64k keys) included."""

import numpy as np
import pytest

from paper_2605_01910_amd import santa as S
from tests.gpu_util import check_dense, check_sampled, log, run
from workload import make_workload

pytestmark = pytest.mark.gpu


def test_cfg2_full_every_row():
    w = make_workload(2, seed=0)
    log(f"[full cfg2] B={w.B} n={w.n_max} {w.kind} S={w.S}")
    out, idx, _ = run(w)
    log(f"  sampled {check_sampled(w, out, idx)}")
    d, _, _ = run(w, "dense")
    log(f"  dense {check_dense(w, d)}")


@pytest.mark.parametrize("kind,S", [("systematic", 128), ("systematic", 512), ("systematic", 1024),
                                    ("stratified", 1024), ("systematic", 2048)])
def test_cfg2_shape_paper_budgets_every_row(kind, S):
    """The batch-1 32k shape at the paper's two operating budgets."""
    w = make_workload(2, seed=0, kind=kind, S=S)
    log(f"[full cfg2 shape] {kind} S={S}")
    out, idx, _ = run(w)
    log(f"  sampled {check_sampled(w, out, idx)}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("S", [128, 256, 512])
def test_cfg3_full_every_row(S):
    w = make_workload(3, seed=0, S=S)
    log(f"[full cfg3] B={w.B} n={w.n_max} {w.kind} S={w.S}")
    out, idx, _ = run(w)
    log(f"  sampled {check_sampled(w, out, idx)}")
    if S == 256:
        d, _, _ = run(w, "dense")
        log(f"  dense {check_dense(w, d)}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("kind", ["systematic", "stratified"])
def test_cfg3_full_scheduled_every_row(kind):
    w = make_workload(3, seed=0, kind=kind, S=256)
    log(f"[full cfg3, scheduled] B={w.B} n={w.n_max} {w.kind} S={w.S}")
    with S.options("rows"):
        out, idx, _ = run(w)
    log(f"  sampled {check_sampled(w, out, idx)}")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("path", ["auto", "rows"])
def test_cfg4_paged_full_every_row(path):
    w = make_workload(4, seed=0)
    log(f"[full cfg4] B={w.B} n_max={w.n_max} ctx {w.ctx_len.min()}..{w.ctx_len.max()} "
        f"rows={w.B * w.Hq}")
    with S.options(path):
        out, idx, _ = run(w)
    log(f"  sampled ({path}) {check_sampled(w, out, idx)}")
    if path == "auto":
        d, _, _ = run(w, "dense")
        log(f"  dense {check_dense(w, d)}")


@pytest.mark.timeout(300)
def test_cfg5_bernoulli_full_every_row():
    from oracle import oracle as O
    w = make_workload(5, seed=0)
    log(f"[full cfg5] B={w.B} n={w.n_max} bernoulli mode={w.mode} S={w.S}")
    out, idx, mask = run(w, want_mask=True)
    log(f"  sampled {check_sampled(w, out, idx, 'bernoulli')}")
    res = O.decode_workload(w, "bernoulli", rows=[b * w.Hq + kv * w.G for b in range(w.B)
                                                  for kv in range(w.Hkv)], want_weights=True)
    assert np.array_equal(mask, res.mask.reshape(w.B, w.Hkv, w.d)), "feature mask differs"

"""GPU parity of every entry point against the CPU oracle, through the C ABI.

Sizes span several splits and a ragged tail; edge cases cover single-key
rows, S > L, S = 1, empty rows, fp32 and bf16, G in {1, 2, 4, 8}, both
contiguous layouts and the paged cache."""

import numpy as np
import pytest
import torch

from paper_2605_01910_amd import santa as S
from tests.gpu_util import (KIND_CODE, DeviceWorkload, check_dense, check_sampled, log, run)
from workload import make_workload

pytestmark = pytest.mark.gpu

DENSE_CASES = {
    "cfg1_f32": (1, {}),
    "cfg2_ragged_b2": (2, dict(B=2, n=3000, ctx_len=[3000, 1234])),
    "cfg2_g8": (2, dict(B=1, Hq=16, Hkv=2, n=2100)),
    "cfg2_g2": (2, dict(B=2, Hq=8, Hkv=4, n=700)),
    "cfg2_single_key": (2, dict(B=2, n=17, ctx_len=[1, 17])),
    "cfg4_paged": (4, dict(B=3, len_lo=900, len_hi=2600)),
}


@pytest.mark.parametrize("case", sorted(DENSE_CASES))
def test_dense_parity(case):
    cfg, over = DENSE_CASES[case]
    log(f"[dense] {case} cfg={cfg} {over}")
    w = make_workload(cfg, seed=11, **over)
    out, _, _ = run(w, "dense")
    log(f"  {check_dense(w, out)}")


def test_dense_head_major_layout():
    w = make_workload(2, B=2, n=1500, seed=12)
    log("[dense] head-major layout")
    out_h, _, _ = run(w, "dense", layout="hnd")
    check_dense(w, out_h)


SAMPLED_CASES = {
    "cfg1_sys": (1, "systematic", {}),
    "cfg2_strat_small": (2, "stratified", dict(B=2, n=2500, ctx_len=[2500, 777])),
    "cfg3_sys_s128": (3, "systematic", dict(B=3, n=3000, S=128)),
    "cfg3_sys_s512": (3, "systematic", dict(B=2, n=5000, S=512)),
    "sys_S_gt_L": (2, "systematic", dict(B=2, n=40, S=256, ctx_len=[40, 3])),
    "strat_S1": (2, "stratified", dict(B=2, n=900, S=1)),
    "sys_single_key": (2, "systematic", dict(B=2, n=33, S=16, ctx_len=[1, 33])),
    "sys_g8": (2, "systematic", dict(B=1, Hq=16, Hkv=2, n=2100, S=64)),
    "strat_g1_bf16": (2, "stratified", dict(B=2, Hq=4, Hkv=4, n=1100, S=32)),
    "sys_empty_row": (2, "systematic", dict(B=3, n=600, S=32, ctx_len=[600, 0, 5])),
    "cfg4_paged_sys": (4, "systematic", dict(B=4, len_lo=700, len_hi=3000)),
    # large budgets in the one-launch kernel: closed-form claim ranges with
    # hundreds of claims per split and long union lists (the shared gather)
    "sys_s2048_long_union": (2, "systematic", dict(B=1, n=20000, S=2048)),
    "strat_s1024_staged_limit": (2, "stratified", dict(B=1, n=12000, S=1024)),
    "strat_s1100_unstaged": (2, "stratified", dict(B=1, n=6000, S=1100)),
}


@pytest.mark.parametrize("case", sorted(SAMPLED_CASES))
def test_sampled_parity(case):
    cfg, kind, over = SAMPLED_CASES[case]
    log(f"[{kind}] {case} cfg={cfg} {over}")
    w = make_workload(cfg, seed=21, kind=kind, **over)
    out, idx, _ = run(w, kind)
    log(f"  {check_sampled(w, out, idx, kind)}")


def test_sampled_head_major_layout():
    w = make_workload(2, B=2, n=1800, kind="systematic", S=64, seed=22)
    log("[systematic] head-major layout")
    out, idx, _ = run(w, layout="hnd")
    check_sampled(w, out, idx)


BERN_CASES = {
    "mode0_B1": dict(B=2, n=1500, mode=0, B_draws=1),
    "mode1_B1": dict(B=2, n=1500, mode=1, B_draws=1),
    "mode0_B4": dict(B=1, n=2100, mode=0, B_draws=4, ctx_len=[2001]),
    "mode1_B8_ragged": dict(B=2, n=999, mode=1, B_draws=8, ctx_len=[999, 123]),
}


@pytest.mark.parametrize("case", sorted(BERN_CASES))
def test_bernoulli_parity(case):
    over = BERN_CASES[case]
    log(f"[bernoulli] {case} {over}")
    w = make_workload(5, seed=31, **over)
    out, idx, mask = run(w, "bernoulli", want_mask=True)
    log(f"  {check_sampled(w, out, idx, 'bernoulli')}")
    from oracle import oracle as O
    res = O.decode_workload(w, "bernoulli", rows=[b * w.Hq + kv * w.G for b in range(w.B)
                                                  for kv in range(w.Hkv)], want_weights=True)
    ref_mask = res.mask.reshape(w.B, w.Hkv, w.d)
    assert np.array_equal(mask, ref_mask), "feature mask differs from the oracle"


def test_repeat_calls_are_bitwise_identical():
    w = make_workload(2, B=2, n=4000, kind="stratified", S=256, seed=41)
    dw = DeviceWorkload(w)
    log("[determinism] stratified x2, dense x2")
    o1, i1, _ = run(w, dw=dw)
    o2, i2, _ = run(w, dw=dw)
    assert np.array_equal(o1, o2) and np.array_equal(i1, i2)
    d1, _, _ = run(w, "dense", dw=dw)
    d2, _, _ = run(w, "dense", dw=dw)
    assert np.array_equal(d1, d2)


def test_ctx_len_null_means_full_length():
    w = make_workload(2, B=2, n=1300, kind="systematic", S=64, seed=42)
    dw = DeviceWorkload(w, pass_ctx=False)
    log("[systematic] ctx_len = NULL")
    out, idx, _ = run(w, dw=dw)
    check_sampled(w, out, idx)


def test_workspace_reuse_across_shapes():
    """One workspace sized for the larger call serves a smaller call next."""
    from paper_2605_01910_amd import santa as S
    big = make_workload(2, B=2, n=3000, kind="systematic", S=128, seed=43)
    small = make_workload(2, B=1, n=700, kind="systematic", S=128, seed=44)
    dwb, dws = DeviceWorkload(big), DeviceWorkload(small)
    ws = S.alloc_workspace(dwb.shape, dwb.kv, 128, S.SANTA_KIND_SYSTEMATIC)
    log("[workspace] big then small")
    ob, ib, _ = run(big, dw=dwb, ws=ws)
    os_, is_, _ = run(small, dw=dws, ws=ws)
    check_sampled(big, ob, ib)
    check_sampled(small, os_, is_)


MULTI_CASES = {
    "dense_cfg2": (2, "dense", dict(B=2, n=3000, ctx_len=[3000, 1234])),
    "strat_cfg2": (2, "stratified", dict(B=2, n=2500, ctx_len=[2500, 777])),
    "sys_paged": (4, "systematic", dict(B=3, len_lo=700, len_hi=3000)),
    "sys_f32": (1, "systematic", {}),
}


@pytest.mark.parametrize("case", sorted(MULTI_CASES))
def test_multi_kernel_variant_parity(case):
    """The multi-kernel path (score/CDF stash, offsets, sample, merge launches)."""
    cfg, kind, over = MULTI_CASES[case]
    log(f"[multi/{kind}] {case} cfg={cfg} {over}")
    w = make_workload(cfg, seed=51, kind=kind if kind != "dense" else "systematic", **over)
    with S.options("multi"):
        out, idx, _ = run(w, kind)
    if kind == "dense":
        check_dense(w, out)
    else:
        log(f"  {check_sampled(w, out, idx, kind)}")


@pytest.mark.parametrize("splits", [16, 64, 200])
def test_fused_split_counts(splits):
    """Fused path at other split counts."""
    w = make_workload(2, B=3, n=5000, kind="stratified", S=128, ctx_len=[5000, 2222, 17], seed=52)
    log(f"[fused splits={splits}]")
    with S.options("auto", splits):
        out, idx, _ = run(w)
        check_sampled(w, out, idx)
        d, _, _ = run(w, "dense")
        check_dense(w, d)


def test_fused_barrier_flag_stays_clear():
    """The fused path's bounded barrier wait never gives up on these inputs."""
    w = make_workload(2, B=16, n=1024, kind="systematic", S=64, seed=53)
    dw = DeviceWorkload(w)
    ws = S.alloc_workspace(dw.shape, dw.kv, w.S, S.SANTA_KIND_SYSTEMATIC)
    for _ in range(3):
        out, idx, _ = run(w, dw=dw, ws=ws)
    check_sampled(w, out, idx)
    assert S.workspace_error(ws) == 0


@pytest.mark.parametrize("case", sorted(SAMPLED_CASES))
def test_two_launch_sampled_parity(case):
    """The large-batch sampled path (key stream with CDF stash, then one
    workgroup per query head) forced on every sampled case."""
    cfg, kind, over = SAMPLED_CASES[case]
    log(f"[two-launch/{kind}] {case} cfg={cfg} {over}")
    w = make_workload(cfg, seed=23, kind=kind, **over)
    with S.options("two"):
        out, idx, _ = run(w, kind)
    log(f"  {check_sampled(w, out, idx, kind)}")


@pytest.mark.parametrize("case", sorted(SAMPLED_CASES))
def test_scheduled_sampled_parity(case):
    """The scheduled path (one hardware-scheduled launch, a workgroup per
    split keeping its CDF in LDS across the row barrier) forced on every
    sampled case; cases with more than 64 splits per row take the two-launch
    path under the same option."""
    cfg, kind, over = SAMPLED_CASES[case]
    log(f"[scheduled/{kind}] {case} cfg={cfg} {over}")
    w = make_workload(cfg, seed=25, kind=kind, **over)
    with S.options("rows"):
        out, idx, _ = run(w, kind)
    log(f"  {check_sampled(w, out, idx, kind)}")


def test_scheduled_many_rows_reuses_counters():
    """The scheduled path over far more workgroups than are resident at once
    (its counter barrier): ragged rows (one empty), G in {4, 8}, and three
    calls in a row on one workspace (the row counters move on by two
    arrivals per split)."""
    lens = [(37 * i * i + 11 * i) % 9000 for i in range(24)]
    lens[3] = 0
    lens[7] = 9000
    for over in (dict(), dict(Hq=32, Hkv=4)):
        w = make_workload(3, B=24, n=9000, kind="stratified", S=128, ctx_len=lens, seed=56,
                          **over)
        dw = DeviceWorkload(w)
        with S.options("rows"):
            plan = S.santa_plan_info(dw.shape, dw.kv, w.S, S.SANTA_KIND_STRATIFIED)
            assert plan["kernels"] == "k_row_sampled", plan
            ws = S.alloc_workspace(dw.shape, dw.kv, w.S, S.SANTA_KIND_STRATIFIED)
            log(f"[scheduled rows] B={w.B} G={w.G} n={w.n_max} T={plan['splits']}")
            for _ in range(3):
                out, idx, _ = run(w, dw=dw, ws=ws)
                check_sampled(w, out, idx)
        assert S.workspace_error(ws) == 0


def test_scheduled_direct_barrier_many_splits_and_mode_changes():
    """The scheduled path's direct row barrier (grids of at most 256
    workgroups: statistics mailbox, LDS merge) at 64 splits per row with G in
    {4, 8}, ragged rows, three calls in a row on one workspace, and calls of
    the counter barrier (a larger grid) interleaved on the same workspace: the
    mailbox must be empty again after every call and the counters consistent
    across the two arrival counts."""
    cases = [dict(B=1, Hq=16, Hkv=4, n=65536, S=256),
             dict(B=1, Hq=32, Hkv=4, n=65536, S=256),
             dict(B=2, Hq=8, Hkv=2, n=65536, S=128, ctx_len=[65536, 23001])]
    big = make_workload(3, B=24, n=9000, kind="systematic", S=128, seed=58)
    with S.options("rows"):
        dwb = DeviceWorkload(big)
        calls = [(big, dwb, S.SANTA_KIND_SYSTEMATIC)]
        for over in cases:
            w = make_workload(3, kind="stratified", seed=57, **over)
            calls.append((w, DeviceWorkload(w), S.SANTA_KIND_STRATIFIED))
        # one workspace, sized for the call that needs the most
        sizes = [S.santa_workspace_size(d.shape, d.kv, w.S, k) for w, d, k in calls]
        w0, d0, k0 = calls[sizes.index(max(sizes))]
        ws = S.alloc_workspace(d0.shape, d0.kv, w0.S, k0)
        for w, dw, kind in calls[1:]:
            plan = S.santa_plan_info(dw.shape, dw.kv, w.S, kind)
            assert plan["kernels"] == "k_row_sampled" and plan["splits"] == 64, plan
            log(f"[scheduled direct] B={w.B} G={w.G} n={w.n_max} T={plan['splits']}")
            for _ in range(3):
                out, idx, _ = run(w, dw=dw, ws=ws)
                check_sampled(w, out, idx)
            log(f"[scheduled counter] B={big.B} G={big.G} n={big.n_max}")
            out, idx, _ = run(big, dw=dwb, ws=ws)
            check_sampled(big, out, idx)
        assert S.workspace_error(ws) == 0


@pytest.mark.parametrize("case", sorted(SAMPLED_CASES))
def test_one_launch_sampled_parity(case):
    """The small-batch sampled path forced on every sampled case."""
    cfg, kind, over = SAMPLED_CASES[case]
    log(f"[one-launch/{kind}] {case} cfg={cfg} {over}")
    w = make_workload(cfg, seed=24, kind=kind, **over)
    with S.options("one"):
        out, idx, _ = run(w, kind)
    log(f"  {check_sampled(w, out, idx, kind)}")


def test_one_launch_many_rounds():
    """One launch over far more rows than one resident round holds: every
    workgroup handles a split of several rows, rows have ragged lengths (one
    empty), and three calls in a row reuse the row counters."""
    lens = [(37 * i * i + 11 * i) % 9000 for i in range(24)]
    lens[3] = 0
    lens[7] = 9000
    w = make_workload(3, B=24, n=9000, kind="systematic", S=64, ctx_len=lens, seed=54)
    dw = DeviceWorkload(w)
    with S.options("one"):
        ws = max((S.alloc_workspace(dw.shape, dw.kv, w.S, k)
                  for k in (S.SANTA_KIND_SYSTEMATIC, S.SANTA_KIND_DENSE)), key=lambda x: x.numel())
        log(f"[rounds] B={w.B} n={w.n_max} rows={w.B * w.Hkv}")
        for _ in range(3):
            out, idx, _ = run(w, dw=dw, ws=ws)
            check_sampled(w, out, idx)
            d, _, _ = run(w, "dense", dw=dw, ws=ws)
            check_dense(w, d)
    assert S.workspace_error(ws) == 0


def test_workspace_shared_by_both_sampled_paths():
    """The counters keep their place in every fused layout: one workspace
    serves the one-launch path, the two-launch path and the dense step in any
    order."""
    w = make_workload(2, B=4, n=3000, kind="stratified", S=128, seed=55)
    dw = DeviceWorkload(w)
    spaces = [S.alloc_workspace(dw.shape, dw.kv, 1, S.SANTA_KIND_DENSE)]
    for path in ("one", "two", "rows"):
        with S.options(path):
            spaces.append(S.alloc_workspace(dw.shape, dw.kv, w.S, S.SANTA_KIND_STRATIFIED))
    ws = max(spaces, key=lambda x: x.numel())
    log("[workspace] one, two, rows, dense, one, rows")
    for path in ("one", "two", "rows", "dense", "one", "rows"):
        if path == "dense":
            d, _, _ = run(w, "dense", dw=dw, ws=ws)
            check_dense(w, d)
            continue
        with S.options(path):
            out, idx, _ = run(w, dw=dw, ws=ws)
        check_sampled(w, out, idx)


def test_workspace_shared_by_every_kind():
    """Every layout keeps the error flag and the counter area at the front, so
    one workspace serves Bernoulli, multi-kernel, one-launch, two-launch and
    dense calls interleaved in any order."""
    ws_ = make_workload(2, B=2, n=3000, kind="systematic", S=128, seed=71)
    wb = make_workload(5, B=2, n=1500, mode=1, B_draws=1, seed=72)
    ds, db = DeviceWorkload(ws_), DeviceWorkload(wb)
    spaces = [S.alloc_workspace(db.shape, db.kv, wb.S, S.SANTA_KIND_BERNOULLI),
              S.alloc_workspace(ds.shape, ds.kv, 1, S.SANTA_KIND_DENSE)]
    for path in ("one", "two", "multi", "rows"):
        with S.options(path):
            spaces.append(S.alloc_workspace(ds.shape, ds.kv, ws_.S, S.SANTA_KIND_SYSTEMATIC))
    ws = max(spaces, key=lambda x: x.numel())
    order = ["one", "bernoulli", "rows", "one", "multi", "one", "two", "bernoulli", "two",
             "rows", "dense", "multi", "rows", "one"]
    log(f"[workspace] {' '.join(order)}")
    for step in order:
        with S.options(step if step in ("one", "two", "multi", "rows") else "auto"):
            if step == "bernoulli":
                out, idx, _ = run(wb, "bernoulli", dw=db, ws=ws)
                check_sampled(wb, out, idx, "bernoulli")
            elif step == "dense":
                d, _, _ = run(ws_, "dense", dw=ds, ws=ws)
                check_dense(ws_, d)
            else:
                out, idx, _ = run(ws_, dw=ds, ws=ws)
                check_sampled(ws_, out, idx)
        assert S.workspace_error(ws) == 0, step

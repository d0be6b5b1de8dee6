"""Pins of the oracle's Bernoulli batch driver (the composition of the
Bernoulli query weights with the score, softmax and systematic value stages;
Sec. 5, Eq. "qk_estimator" and Eq. "mean_group_query"; App. C).

Each case chooses the query and the Bernoulli uniforms so that the weights
w are known in closed form and exactly representable, then requires the
driver's Bernoulli result (indices and outputs) to equal, bit for bit, the
systematic driver run on a query equal to those weights.  A mistake in the
composition -- another head's weight row, the query used in place of its
weights, a wrong or doubled scale, a wrong uniform row -- changes the scores
and fails the comparison.  The feature mask is checked against the union over
the GQA group of the features with a nonzero weight.
"""

import numpy as np
import pytest

from oracle import oracle as O
from workload import bf16_bits_to_f32, f32_to_bf16_bits, make_workload

ONE_MINUS = np.float32(1.0) - np.float32(2.0 ** -24)   # largest float32 below 1


def _workload(mode, B_draws, dtype="bf16", seed=11):
    w = make_workload(5, B=2, Hq=8, Hkv=2, n=300, ctx_len=[300, 177], dtype=dtype,
                      mode=mode, B_draws=B_draws, seed=seed)
    assert w.kind == "bernoulli" and w.u.shape == (w.B, w.Hq)
    return w


def _set_q(w, qf):
    """Replace the workload's query by the float32 values qf (exact in its dtype)."""
    qf = np.ascontiguousarray(qf, dtype=np.float32)
    w.q = f32_to_bf16_bits(qf) if w.dtype == "bf16" else qf
    assert np.array_equal(w.q_f32(), qf), "query must be exact in the workload's dtype"


def _same_as_systematic(w, q_equiv):
    """Bernoulli driver on w == systematic driver on w with query q_equiv."""
    rb = O.decode_workload(w, "bernoulli", want_cdf=True, want_weights=True)
    saved = w.q
    _set_q(w, q_equiv)
    rs = O.decode_workload(w, "systematic", want_cdf=True)
    w.q = saved
    assert np.array_equal(rb.idx, rs.idx)
    assert np.array_equal(rb.out, rs.out)
    assert np.array_equal(rb.cdf, rs.cdf, equal_nan=True)
    # the weights the driver used are the equivalent query, row by row
    assert np.array_equal(rb.w, np.asarray(q_equiv, np.float64).reshape(w.B * w.Hq, w.d))
    return rb


def _check_mask_is_group_union(w, res):
    G = w.G
    nz = (res.w != 0).reshape(w.B, w.Hkv, G, w.d)
    union = nz.any(axis=2)
    mk = res.mask.reshape(w.B, w.Hkv, G, w.d)
    for g in range(G):
        assert np.array_equal(mk[:, :, g, :].astype(bool), union)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("B_draws", [1, 4])
def test_equal_magnitudes_give_the_query_itself(mode, B_draws):
    """|q_i| equal everywhere: pi_i = 1, every draw keeps the feature, and
    w = q exactly (mode 0: (norm/B) sign(q) B; mode 1: m_i = norm and
    w = norm q / m).  Signs differ across heads and features, so a weight row
    taken from the wrong head changes the scores."""
    w = _workload(mode, B_draws)
    rng = np.random.default_rng(3)
    qf = np.where(rng.random((w.B, w.Hq, w.d)) < 0.5, -0.75, 0.75).astype(np.float32)
    _set_q(w, qf)
    res = _same_as_systematic(w, qf)
    assert res.mask.all()
    _check_mask_is_group_union(w, res)


def test_mode0_zero_uniforms_give_full_norm_ternary_query():
    """u = 0 and B = 1: b_i = [0 < pi_i] keeps every nonzero feature, so w is
    the per-head ternary query norm_h * sign(q) (not q itself)."""
    w = _workload(0, 1)
    w.u_q = np.zeros_like(w.u_q)
    qf = w.q_f32().copy()
    qf[0, 1, 5] = 0.0                                   # a zero feature stays zero
    _set_q(w, qf)
    norm = np.abs(qf).max(axis=2, keepdims=True)
    res = _same_as_systematic(w, norm * np.sign(qf))
    _check_mask_is_group_union(w, res)


def test_mode0_uniforms_near_one_keep_only_the_largest_features():
    """u = 1 - 2^-24 and B = 1: b_i = [u < |q_i|/norm] holds only where
    |q_i| = norm, so w is +-norm at each head's largest features, 0 elsewhere,
    and the mask is the union of those features over the group."""
    w = _workload(0, 1)
    w.u_q = np.full_like(w.u_q, ONE_MINUS)
    qf = w.q_f32()
    norm = np.abs(qf).max(axis=2, keepdims=True)
    q_eq = np.where(np.abs(qf) == norm, np.sign(qf) * norm, 0.0).astype(np.float32)
    res = _same_as_systematic(w, q_eq)
    _check_mask_is_group_union(w, res)
    assert res.mask.reshape(w.B * w.Hq, w.d).sum(axis=1).max() <= w.G


def test_mode0_stratified_counts_over_four_draws():
    """B = 4, u = 0: the stratified count is #{n < 4 : n/4 < pi_i} =
    ceil(4 pi_i), so w = (norm/4) sign(q) ceil(4 pi), decided in float32.
    The query has bfloat16 values held as float32 so that w is exact."""
    w = _workload(0, 4, dtype="f32")
    qf = bf16_bits_to_f32(f32_to_bf16_bits(w.q_f32()))
    _set_q(w, qf)
    w.u_q = np.zeros_like(w.u_q)
    norm = np.abs(qf).max(axis=2, keepdims=True)
    pi = (np.abs(qf) / norm).astype(np.float32)
    cnt = sum((np.float32(n) / np.float32(4) < pi).astype(np.float32) for n in range(4))
    q_eq = (norm / np.float32(4)) * np.sign(qf) * cnt
    _same_as_systematic(w, q_eq.astype(np.float32))


def test_mode1_zero_uniforms_give_group_norm_signs():
    """Mode 1, u = 0, B = 1, with |q_{g,i}| = a_i shared by the group's heads:
    m_i = a_i, pi_i > 0 keeps every feature, m_hat_i = norm and
    w_{g,i} = norm q_{g,i} / a_i = norm sign(q_{g,i})."""
    w = _workload(1, 1)
    assert w.u_q.shape == (w.B, w.Hkv, w.d)
    w.u_q = np.zeros_like(w.u_q)
    rng = np.random.default_rng(4)
    a = bf16_bits_to_f32(f32_to_bf16_bits(rng.uniform(0.25, 2.0, (w.B, w.Hkv, 1, w.d)).astype(np.float32)))
    sgn = np.where(rng.random((w.B, w.Hkv, w.G, w.d)) < 0.5, -1.0, 1.0).astype(np.float32)
    qf = (sgn * a).reshape(w.B, w.Hq, w.d)
    _set_q(w, qf)
    norm = a.max(axis=3, keepdims=True)
    res = _same_as_systematic(w, (sgn * norm).reshape(w.B, w.Hq, w.d))
    assert res.mask.all()


@pytest.mark.parametrize("mode", [0, 1])
def test_mask_is_union_of_nonzero_weights_random_draws(mode):
    w = _workload(mode, 1, seed=12)
    res = O.decode_workload(w, "bernoulli", want_weights=True)
    _check_mask_is_group_union(w, res)
    assert 0 < res.mask.mean() < 1


def test_mode0_uniform_rows_follow_the_heads():
    """Per-head uniforms that differ by row: u = 0 keeps every nonzero
    feature (w = norm sign(q)), u = 1 - 2^-24 only the largest ones.  A driver
    that reads another head's uniforms gives another query."""
    w = _workload(0, 1, seed=13)
    qf = w.q_f32()
    keep_all = (np.arange(w.B)[:, None] + np.arange(w.Hq)[None, :]) % 3 == 0   # [B, Hq]
    w.u_q = np.where(keep_all[:, :, None], np.float32(0.0), ONE_MINUS).astype(np.float32)
    w.u_q = np.broadcast_to(w.u_q, (w.B, w.Hq, w.d)).copy()
    norm = np.abs(qf).max(axis=2, keepdims=True)
    q_eq = np.where(keep_all[:, :, None] | (np.abs(qf) == norm), np.sign(qf) * norm, 0.0)
    res = _same_as_systematic(w, q_eq.astype(np.float32))
    _check_mask_is_group_union(w, res)


def test_mode1_uniform_rows_follow_the_kv_heads():
    """Mode 1 reads one uniform row per (batch, KV head): with |q_{g,i}| = a_i
    shared by the group, u = 0 keeps every feature and u = 1 - 2^-24 only the
    features with a_i = norm, group by group."""
    w = _workload(1, 1, seed=14)
    rng = np.random.default_rng(5)
    a = bf16_bits_to_f32(f32_to_bf16_bits(rng.uniform(0.25, 2.0, (w.B, w.Hkv, 1, w.d)).astype(np.float32)))
    sgn = np.where(rng.random((w.B, w.Hkv, w.G, w.d)) < 0.5, -1.0, 1.0).astype(np.float32)
    _set_q(w, (sgn * a).reshape(w.B, w.Hq, w.d))
    keep_all = np.array([[True, False], [False, True]])                      # [B, Hkv]
    w.u_q = np.broadcast_to(np.where(keep_all[:, :, None], np.float32(0.0), ONE_MINUS),
                            (w.B, w.Hkv, w.d)).astype(np.float32).copy()
    norm = a.max(axis=3, keepdims=True)
    kept = keep_all[:, :, None, None] | (a == norm)
    q_eq = np.where(kept, sgn * norm, 0.0).reshape(w.B, w.Hq, w.d)
    res = _same_as_systematic(w, q_eq.astype(np.float32))
    _check_mask_is_group_union(w, res)

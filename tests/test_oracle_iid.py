"""Pins of the oracle's i.i.d. SANTA thresholds built by exponential spacings
(S + 1 uniforms, normalised partial sums of unit exponentials; the GPU's
i.i.d. path uses the same construction because it needs no sort).  They are
checked against facts of the order statistics of S independent uniforms and
of the i.i.d. estimator of Sec. 2 (Eq. "stochastic-add-only-attn"; App. A,
the variance tr(Sigma)/S of the multinomial estimator), not against the
oracle itself.  CPU only."""

import math

import numpy as np
import pytest
from scipy import stats

from oracle import oracle as O


def test_spacings_thresholds_strictly_increasing_in_unit_interval():
    rng = np.random.default_rng(1)
    for S in (1, 2, 7, 256, 1024):
        u = rng.random(S + 1, dtype=np.float32)
        T = O.thresholds("iid_spacings", u, S)
        assert np.all(T > 0) and np.all(T < 1) and np.all(np.diff(T) > 0)


def test_spacings_single_threshold_is_uniform():
    """S = 1: T = E_0 / (E_0 + E_1) is uniform on [0, 1) (KS test)."""
    rng = np.random.default_rng(2)
    T = np.array([O.thresholds("iid_spacings", rng.random(2, dtype=np.float32), 1)[0]
                  for _ in range(4000)])
    assert stats.kstest(T, "uniform").pvalue > 1e-3


def test_spacings_match_order_statistic_means_and_law():
    """E[T_(m)] = (m+1)/(S+1) for the m-th of S sorted uniforms, and T_(m) is
    Beta(m+1, S-m) distributed (KS test on two order statistics)."""
    rng = np.random.default_rng(3)
    S, N = 8, 6000
    T = np.array([O.thresholds("iid_spacings", rng.random(S + 1, dtype=np.float32), S)
                  for _ in range(N)])
    mean = T.mean(0)
    sd = T.std(0, ddof=1) / math.sqrt(N)
    assert np.all(np.abs(mean - (np.arange(S) + 1) / (S + 1)) <= 5 * sd)
    for m in (0, 5):
        assert stats.kstest(T[:, m], stats.beta(m + 1, S - m).cdf).pvalue > 1e-3


def _row(seed, L, d):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal(d).astype(np.float32) * 2
    k = rng.standard_normal((L, d)).astype(np.float32)
    v = rng.standard_normal((L, d)).astype(np.float32)
    return q, k, v


def test_spacings_estimator_unbiased_with_multinomial_variance():
    """Monte Carlo over 10^4 draws: the mean is within 5 SE of dense AV and
    the total variance matches tr(Sigma)/S of S i.i.d. categorical draws
    (chi-square band), which a dependent (e.g. stratified) sampler fails."""
    N, L, d, S = 10000, 24, 6, 4
    q, k, v = _row(11, L, d)
    Q = np.broadcast_to(q, (N, 1, d)).copy()
    K = np.broadcast_to(k[None, :, None, :], (N, L, 1, d)).copy()
    V = np.broadcast_to(v[None, :, None, :], (N, L, 1, d)).copy()
    u = np.random.default_rng(12).random((N, 1, S + 1), dtype=np.float32)
    res = O.decode("iid_spacings", Q, K, V, np.full(N, L, np.int32), 0.3, S, u)
    p = O.softmax(O.scores(q.astype(np.float64), k, 0.3))
    av = O.weighted_sum(p, v)
    mean = res.out.mean(0)
    se = res.out.std(0, ddof=1) / math.sqrt(N)
    assert np.all(np.abs(mean - av) <= 5 * se + 1e-12)
    vv = v.astype(np.float64)
    trace = float((p[:, None] * (vv - av) ** 2).sum()) / S
    emp = float(((res.out - av) ** 2).sum(1).mean())
    assert 0.9 * trace <= emp <= 1.1 * trace


def test_spacings_batch_driver_indices():
    """The batch driver's i.i.d.-by-spacings indices are the inverse CDF of the
    spacings thresholds; S per row, non-decreasing."""
    rng = np.random.default_rng(5)
    B, Hq, n, d, S = 2, 2, 40, 4, 16
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    k = rng.standard_normal((B, n, 1, d)).astype(np.float32)
    v = rng.standard_normal((B, n, 1, d)).astype(np.float32)
    u = rng.random((B, Hq, S + 1), dtype=np.float32)
    ctx = np.array([40, 17], np.int32)
    res = O.decode("iid_spacings", q, k, v, ctx, 0.5, S, u)
    for r in range(B * Hq):
        b, h = divmod(r, Hq)
        L = int(ctx[b])
        C = O.cdf(O.softmax(O.scores(q[b, h].astype(np.float64), k[b, :L, 0], 0.5)))
        T = O.thresholds("iid_spacings", u[b, h], S)
        assert np.array_equal(res.idx[r], np.searchsorted(C, T, side="right").clip(max=L - 1))
        assert np.all(np.diff(res.idx[r]) >= 0)

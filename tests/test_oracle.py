"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each check is a library
routine that has the same definition (torch SDPA, numpy searchsorted), a value
the paper prints (tests/golden), a closed form, an exact integral, brute force
on a tiny input, or a statistical law with its standard error.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import oracle as O
from workload import bf16_bits_to_f32, make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def sdpa_ref(q, k, v, scale):
    """torch SDPA (float64, CPU) for one query row: q [d], k/v [L, d]."""
    qt = torch.tensor(np.asarray(q, np.float64))[None, None, None, :]
    kt = torch.tensor(np.asarray(k, np.float64))[None, None]
    vt = torch.tensor(np.asarray(v, np.float64))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)[0, 0, 0].numpy()


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# ----------------------------------------------------------------------------
# P1: dense attention
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("L", [1, 2, 3, 7, 64])
def test_dense_matches_torch_sdpa(L):
    rng = np.random.default_rng(L)
    d = 16
    q, k, v = (_f32(rng.standard_normal(s)) for s in ((d,), (L, d), (L, d)))
    scale = 1 / math.sqrt(d)
    s = O.scores(q.astype(np.float64), k, scale)
    out = O.weighted_sum(O.softmax(s), v)
    np.testing.assert_allclose(out, sdpa_ref(q, k, v, scale), rtol=0, atol=1e-13)


def test_dense_single_key_returns_that_value():
    rng = np.random.default_rng(1)
    q, k, v = _f32(rng.standard_normal(8)), _f32(rng.standard_normal((1, 8))), _f32(rng.standard_normal((1, 8)))
    out = O.weighted_sum(O.softmax(O.scores(q.astype(np.float64), k, 0.3)), v)
    assert np.array_equal(out, v[0].astype(np.float64))


def test_dense_equal_scores_give_mean_of_values():
    rng = np.random.default_rng(2)
    L, d = 37, 8
    k, v = _f32(rng.standard_normal((L, d))), _f32(rng.standard_normal((L, d)))
    out = O.weighted_sum(O.softmax(O.scores(np.zeros(d), k, 1.0)), v)
    np.testing.assert_allclose(out, v.astype(np.float64).mean(0), atol=1e-14)


def test_dense_invariant_to_constant_score_shift():
    rng = np.random.default_rng(3)
    L, d = 50, 8
    q, k, v = _f32(rng.standard_normal(d)), _f32(rng.standard_normal((L, d))), _f32(rng.standard_normal((L, d)))
    # adding delta to every key shifts every score by scale * <q, delta>
    delta = _f32(3.0 * q / np.dot(q, q))
    o1 = O.weighted_sum(O.softmax(O.scores(q.astype(np.float64), k, 0.5)), v)
    o2 = O.weighted_sum(O.softmax(O.scores(q.astype(np.float64), _f32(k + delta), 0.5)), v)
    np.testing.assert_allclose(o1, o2, atol=1e-5)   # k + delta is rounded to float32


def test_batch_driver_gqa_ragged_matches_sdpa():
    """The batch driver's row -> (b, h, kv head) mapping and ragged lengths."""
    w = make_workload(2, B=3, Hq=8, Hkv=2, n=97, ctx_len=[97, 40, 1], seed=5)
    res = O.decode_workload(w, "dense")
    qf = w.q_f32()
    k, v = bf16_bits_to_f32(w.k), bf16_bits_to_f32(w.v)
    for b in range(w.B):
        L = int(w.ctx_len[b])
        for h in range(w.Hq):
            kv = h // w.G
            ref = sdpa_ref(qf[b, h], k[b, :L, kv], v[b, :L, kv], w.scale)
            np.testing.assert_allclose(res.out[b * w.Hq + h], ref, atol=1e-12)


# ----------------------------------------------------------------------------
# P2: inverse CDF and the worked example
# ----------------------------------------------------------------------------

def test_inverse_cdf_matches_searchsorted_right():
    rng = np.random.default_rng(7)
    for L in (1, 2, 5, 300):
        p = rng.random(L) ** 3
        p /= p.sum()
        C = O.cdf(p)
        T = np.concatenate([rng.random(64), C[:-1], [0.0, C[-1], np.nextafter(C[-1], 2)]])
        T.sort()
        ref = np.minimum(np.searchsorted(C, T, side="right"), L - 1)
        assert np.array_equal(O.inverse_cdf(C, T), ref)


def test_inverse_cdf_brute_force_interval_membership():
    """Every returned J satisfies F(J-1) <= T < F(J) (App. A, unbiasedness proof)."""
    rng = np.random.default_rng(8)
    p = np.array([0.1, 0.0, 0.25, 0.0, 0.0, 0.4, 0.25])
    C = O.cdf(p)
    T = np.sort(rng.random(500))
    for t, j in zip(T, O.inverse_cdf(C, T)):
        lo = 0.0 if j == 0 else C[j - 1]
        assert lo <= t < C[j] or (j == len(p) - 1 and t >= C[j])
        assert p[j] > 0        # zero-mass keys are never chosen


def test_cdf_is_running_sum():
    p = np.array([0.5, 0.25, 0.125, 0.125])
    assert np.array_equal(O.cdf(p), np.array([0.5, 0.75, 0.875, 1.0]))


def test_worked_example_from_paper():
    g = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    S, p = g["S"], np.array(g["p"])
    T = O.thresholds("systematic", np.array([g["u"]], np.float32), S)
    idx = O.inverse_cdf(O.cdf(p), T)
    assert idx.tolist() == g["expected_idx_0based"]
    assert [i + 1 for i in idx] == g["paper_samples_1based"]
    rng = np.random.default_rng(9)
    V = _f32(rng.standard_normal((g["n_k"], 6)))
    est = O.gather_mean(V, idx)
    np.testing.assert_allclose(est, (V[0] + V[0] + V[2]).astype(np.float64) / 3, atol=1e-15)
    np.testing.assert_allclose(est, np.array(g["expected_weights"]) @ V.astype(np.float64), atol=1e-15)


# ----------------------------------------------------------------------------
# P3 / P4: systematic special cases
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 2, 8, 64, 1024])
def test_systematic_S_equals_n_uniform_returns_each_index_once(n):
    rng = np.random.default_rng(n)
    d = 4
    k = np.zeros((n, d), np.float32)                    # equal scores -> uniform p
    p = O.softmax(O.scores(np.ones(d), k, 1.0))
    C = O.cdf(p)
    for u in list(rng.random(20, dtype=np.float32)) + [0.0, np.float32(1 - 2 ** -24)]:
        T = O.thresholds("systematic", np.array([u], np.float32), n)
        assert np.array_equal(O.inverse_cdf(C, T), np.arange(n))


@pytest.mark.parametrize("n", [3, 7, 100])
def test_systematic_S_equals_n_non_power_of_two(n):
    k = np.zeros((n, 4), np.float32)
    C = O.cdf(O.softmax(O.scores(np.ones(4), k, 1.0)))
    for u in np.linspace(1e-6, 1 - 1e-6, 17).astype(np.float32):
        T = O.thresholds("systematic", np.array([u], np.float32), n)
        assert np.array_equal(O.inverse_cdf(C, T), np.arange(n))


def test_systematic_u_zero_gives_exact_quantiles():
    for S in (1, 3, 64, 256):
        T = O.thresholds("systematic", np.array([0.0], np.float32), S)
        assert np.array_equal(T, np.arange(S) / S)


def test_stratified_thresholds_lie_in_their_strata():
    rng = np.random.default_rng(11)
    S = 128
    u = rng.random(S, dtype=np.float32)
    T = O.thresholds("stratified", u, S)
    m = np.arange(S)
    assert np.all(T >= m / S) and np.all(T < (m + 1) / S)


def test_iid_thresholds_are_sorted_uniforms():
    rng = np.random.default_rng(12)
    u = rng.random(50, dtype=np.float32)
    assert np.array_equal(O.thresholds("iid", u, 50), np.sort(u.astype(np.float64)))


# ----------------------------------------------------------------------------
# P5: exact integral over the systematic offset equals dense AV
# ----------------------------------------------------------------------------

def _random_row(rng, L, d, sharp=1.0):
    q = _f32(rng.standard_normal(d) * sharp)
    k = _f32(rng.standard_normal((L, d)))
    v = _f32(rng.standard_normal((L, d)))
    return q, k, v


@pytest.mark.parametrize("L,S", [(5, 1), (13, 4), (40, 8), (64, 64), (200, 16)])
def test_systematic_integral_over_u_equals_dense(L, S):
    """est(u) is piecewise constant in u with breakpoints frac(S F(j)); the
    exact integral over u in [0,1) is AV (App. A, Prop. 'Unbiasedness of S2ANTA')."""
    rng = np.random.default_rng(100 + L + S)
    d = 8
    q, k, v = _random_row(rng, L, d, sharp=2.0)
    scale = 1 / math.sqrt(d)
    p = O.softmax(O.scores(q.astype(np.float64), k, scale))
    C = O.cdf(p)
    brk = np.unique(np.concatenate([[0.0, 1.0], np.mod(S * C, 1.0)]))
    total, unresolved = np.zeros(d), 0.0
    for a, b in zip(brk[:-1], brk[1:]):
        u32 = np.float32((a + b) / 2)
        if not (a < float(u32) < b):
            unresolved += b - a                         # narrower than float32 spacing
            continue
        T = O.thresholds("systematic", np.array([u32]), S)
        total += (b - a) * O.gather_mean(v, O.inverse_cdf(C, T))
    ref = sdpa_ref(q, k, v, scale)
    bound = 1e-12 + unresolved * 2 * np.abs(v).max()
    assert np.abs(total - ref).max() <= bound


def test_systematic_grid_average_within_bound():
    """Grid version: N float32 midpoints; error <= L * max|V_j - V_j'| / (N S)."""
    rng = np.random.default_rng(21)
    L, d, S, N = 300, 8, 16, 4096
    q, k, v = _random_row(rng, L, d, sharp=2.0)
    p = O.softmax(O.scores(q.astype(np.float64), k, 0.35))
    C = O.cdf(p)
    acc = np.zeros(d)
    for i in range(N):
        T = O.thresholds("systematic", np.array([(i + 0.5) / N], np.float32), S)
        acc += O.gather_mean(v, O.inverse_cdf(C, T))
    acc /= N
    ref = O.weighted_sum(p, v)
    spread = (v.max(0) - v.min(0)).max()
    assert np.abs(acc - ref).max() <= L * spread / (N * S)


def test_stratified_integral_per_stratum_equals_dense():
    """Stratified: each stratum's T_m is uniform on I_m, so the estimate's mean
    is (1/S) sum_m S * integral over I_m of V_{F^-1(t)} dt = AV."""
    rng = np.random.default_rng(22)
    L, d, S = 60, 6, 8
    q, k, v = _random_row(rng, L, d, sharp=2.0)
    p = O.softmax(O.scores(q.astype(np.float64), k, 0.4))
    C = O.cdf(p)
    mean, unresolved = np.zeros(d), 0.0
    for m in range(S):
        inside = (S * C - m)
        brk = np.unique(np.concatenate([[0.0, 1.0], inside[(inside > 0) & (inside < 1)]]))
        for a, b in zip(brk[:-1], brk[1:]):
            u = np.full(S, 0.0, np.float32)
            u[m] = np.float32((a + b) / 2)
            if not (a < float(u[m]) < b):
                unresolved += (b - a) / S                 # narrower than float32 spacing
                continue
            idx = O.inverse_cdf(C, O.thresholds("stratified", u, S))
            mean += (b - a) * v[idx[m]].astype(np.float64) / S
    bound = 1e-12 + unresolved * 2 * np.abs(v).max()
    assert np.abs(mean - O.weighted_sum(p, v)).max() <= bound


# ----------------------------------------------------------------------------
# P6 / P7 / P8: Monte Carlo mean, variance laws and the Bernstein tail
# ----------------------------------------------------------------------------

def _replicated(kind, N, L, d, S, seed, sharp=2.0):
    """N copies of one query row with independent uniforms, through the batch driver."""
    rng = np.random.default_rng(seed)
    q, k, v = _random_row(rng, L, d, sharp)
    Q = np.broadcast_to(q, (N, 1, d)).copy()
    K = np.broadcast_to(k[None, :, None, :], (N, L, 1, d)).copy()
    V = np.broadcast_to(v[None, :, None, :], (N, L, 1, d)).copy()
    ur = np.random.default_rng(seed + 1)
    u = ur.random((N, 1), dtype=np.float32) if kind == "systematic" else ur.random((N, 1, S), dtype=np.float32)
    res = O.decode(kind, Q, K, V, np.full(N, L, np.int32), 0.3, S, u)
    p = O.softmax(O.scores(q.astype(np.float64), k, 0.3))
    return res, q, k, v, p


@pytest.mark.parametrize("kind", ["iid", "stratified", "systematic"])
def test_monte_carlo_mean_converges_to_dense(kind):
    N, L, d, S = 10000, 32, 8, 4
    res, q, k, v, _ = _replicated(kind, N, L, d, S, seed=31)
    mean = res.out.mean(0)
    se = res.out.std(0, ddof=1) / math.sqrt(N)
    ref = sdpa_ref(q, k, v, 0.3)
    assert np.all(np.abs(mean - ref) <= 5 * se + 1e-12)


def _var_traces(p, v, S):
    """Closed forms (App. 'Implementation & Measurement Protocol', VarTrace):
    multinomial tr(Sigma)/S and independent equal-mass stratified (1/S^2) sum_m tr(Sigma_m)."""
    v = v.astype(np.float64)
    mu = p @ v
    tr = float(p @ (v * v).sum(1) - mu @ mu)
    C = np.concatenate([[0.0], np.cumsum(p)])
    strat = 0.0
    for m in range(S):
        lo, hi = m / S, (m + 1) / S
        w = np.clip(np.minimum(C[1:], hi) - np.maximum(C[:-1], lo), 0, None) * S   # within-stratum pmf
        mum = w @ v
        strat += float(w @ (v * v).sum(1) - mum @ mum)
    return tr / S, strat / S ** 2


def test_iid_variance_matches_closed_form():
    N, L, d, S = 20000, 24, 6, 4
    res, q, k, v, p = _replicated("iid", N, L, d, S, seed=41)
    mc = float(((res.out - p @ v.astype(np.float64)) ** 2).sum(1).mean())
    iid, _ = _var_traces(p, v, S)
    assert abs(mc / iid - 1) < 0.05


def test_stratified_variance_matches_closed_form_and_dominance():
    N, L, d, S = 20000, 24, 6, 4
    res, q, k, v, p = _replicated("stratified", N, L, d, S, seed=42)
    mc = float(((res.out - p @ v.astype(np.float64)) ** 2).sum(1).mean())
    iid, strat = _var_traces(p, v, S)
    assert abs(mc / strat - 1) < 0.05
    assert strat <= iid


def test_stratified_closed_form_never_exceeds_iid():
    """Variance-dominance theorem (App. A, 'Variance Reduction for S2ANTA-Strat')."""
    rng = np.random.default_rng(43)
    for _ in range(200):
        L, S = int(rng.integers(1, 40)), int(rng.integers(1, 33))
        p = rng.random(L) ** 4
        p /= p.sum()
        v = rng.standard_normal((L, 5))
        iid, strat = _var_traces(p, v, S)
        assert strat <= iid * (1 + 1e-12) + 1e-15


def test_bernstein_tail_bound_holds():
    """App. B: P(||err|| >= t) <= 2 exp(-S t^2 / (2 (v + Vmax t / 3)))."""
    N, L, d, S = 20000, 20, 4, 8
    res, q, k, v, p = _replicated("iid", N, L, d, S, seed=44)
    mu = p @ v.astype(np.float64)
    err = np.linalg.norm(res.out - mu, axis=1)
    vq = float(p @ ((v.astype(np.float64) - mu) ** 2).sum(1))
    vmax = float(np.linalg.norm(v.astype(np.float64) - mu, axis=1).max())
    for t in np.linspace(0.2, 2.0, 10) * math.sqrt(vq):
        emp = float((err >= t).mean())
        bound = 2 * math.exp(-S * t * t / (2 * (vq + vmax * t / 3)))
        assert emp <= min(1.0, bound) + 3 * math.sqrt(max(emp, 1 / N) / N)


# ----------------------------------------------------------------------------
# P9: Bernoulli query estimator
# ----------------------------------------------------------------------------

def test_bernoulli_expected_weights_equal_query_mode0():
    """E[q_hat] = q (Sec. 5): the stratified count's mean over u in [0,1) is B*pi."""
    rng = np.random.default_rng(51)
    G, d, B, N = 2, 10, 4, 4096
    q = _f32(rng.standard_normal((G, d)))
    acc = np.zeros((G, d))
    for i in range(N):
        u = np.full((G, d), (i + 0.5) / N, np.float32)
        w, _ = O.bernoulli_weights(q, u, B, mode=0)
        acc += w
    acc /= N
    # each count is a step function of u with B breakpoints -> error <= B/N per feature
    norm = np.abs(q).max(1, keepdims=True)
    assert np.all(np.abs(acc - q) <= norm * (B / N) / B + 1e-12)


def test_bernoulli_expected_weights_equal_query_mode0_iid_enumeration():
    """Exact enumeration of all 2^d Bernoulli masks (B = 1, small d): E[q_hat] = q."""
    rng = np.random.default_rng(52)
    d = 8
    q = _f32(rng.standard_normal((1, d)))
    norm = float(np.abs(q).max())
    pi = np.abs(q[0]).astype(np.float64) / norm
    mean = np.zeros(d)
    for mask in range(2 ** d):
        bits = np.array([(mask >> i) & 1 for i in range(d)], np.float64)
        prob = np.prod(np.where(bits == 1, pi, 1 - pi))
        # realise this mask with uniforms: u < pi where bit set, u >= pi otherwise
        u = np.where(bits == 1, 0.0, np.nextafter(pi.astype(np.float32), 2)).astype(np.float32)
        u = np.where((bits == 0) & (pi >= 1), np.float32(0.0), u)
        if np.any((bits == 0) & (pi >= 1)):
            continue                                       # impossible mask (prob 0)
        w, _ = O.bernoulli_weights(q, u.reshape(1, d), 1, mode=0, iid=True)
        mean += prob * w[0]
    np.testing.assert_allclose(mean, q[0].astype(np.float64), atol=1e-12)


def test_bernoulli_deterministic_when_all_magnitudes_equal():
    rng = np.random.default_rng(53)
    d = 16
    q = _f32(np.sign(rng.standard_normal((1, d))) * 0.75)
    for B in (1, 2, 4):
        w, mask = O.bernoulli_weights(q, rng.random((1, d), dtype=np.float32), B, mode=0)
        assert np.array_equal(w[0], q[0].astype(np.float64)) and mask.all()


def test_bernoulli_iid_score_variance_and_access_fraction():
    """Var(p_hat_j) = (1/B) sum_i K_ji^2 (norm |q_i| - q_i^2); P(feature kept) = 1-(1-pi)^B."""
    rng = np.random.default_rng(54)
    d, L, B, N = 32, 6, 2, 20000
    q = _f32(rng.standard_normal((1, d)))
    k = rng.standard_normal((L, d))
    norm = float(np.abs(q).max())
    pi = np.abs(q[0]).astype(np.float64) / norm
    U = rng.random((N, 1, B * d), dtype=np.float32)
    ps, kept = [], []
    for n in range(N):
        w, mask = O.bernoulli_weights(q, U[n], B, mode=0, iid=True)
        ps.append(k @ w[0])
        kept.append(mask.mean())
    ps = np.array(ps)
    var_cf = (k ** 2 @ (norm * np.abs(q[0]) - q[0].astype(np.float64) ** 2)) / B
    assert np.all(np.abs(ps.var(0) / var_cf - 1) < 0.06)
    np.testing.assert_allclose(ps.mean(0), k @ q[0], atol=5 * np.sqrt(var_cf / N).max())
    assert abs(np.mean(kept) - np.mean(1 - (1 - pi) ** B)) < 0.01


def test_bernoulli_mean_group_mode1_unbiased_and_zero_features():
    rng = np.random.default_rng(55)
    G, d, B, N = 4, 12, 2, 4096
    q = _f32(rng.standard_normal((G, d)))
    q[:, 3] = 0.0                                        # m_3 = 0 -> weight 0, not fetched
    acc = np.zeros((G, d))
    for i in range(N):
        w, mask = O.bernoulli_weights(q, np.full(d, (i + 0.5) / N, np.float32), B, mode=1)
        assert mask[3] == 0 and np.all(w[:, 3] == 0)
        acc += w
    acc /= N
    m = np.abs(q).mean(0)
    assert np.all(np.abs(acc - q) <= np.abs(q) / m.clip(1e-30) * m.max() / N + 1e-12)


def test_bernoulli_error_matches_paper_figure():
    """App. C figure: at B=4, rel-L2 score error ~60% (standard) vs ~30% (stratified)."""
    g = json.load(open(os.path.join(GOLDEN, "bernoulli_error.json")))
    d, n, B, inst = g["d"], g["n_k"], g["B"], g["instances"]
    rng = np.random.default_rng(56)
    e_iid, e_str = [], []
    for _ in range(inst):
        q = _f32(rng.standard_normal((1, d)))
        K = rng.standard_normal((n, d)) / math.sqrt(d)
        p = K @ q[0]
        w, _ = O.bernoulli_weights(q, rng.random((1, B * d), dtype=np.float32), B, mode=0, iid=True)
        e_iid.append(np.linalg.norm(K @ w[0] - p) / np.linalg.norm(p))
        w, _ = O.bernoulli_weights(q, rng.random((1, d), dtype=np.float32), B, mode=0)
        e_str.append(np.linalg.norm(K @ w[0] - p) / np.linalg.norm(p))
    assert abs(np.mean(e_iid) - g["paper_rel_l2_iid"]) <= g["tolerance_abs"]
    assert abs(np.mean(e_str) - g["paper_rel_l2_stratified"]) <= g["tolerance_abs"]
    assert np.mean(e_str) < np.mean(e_iid)


# ----------------------------------------------------------------------------
# P10 / P11: gather and structural invariants on workload-shaped inputs
# ----------------------------------------------------------------------------

def test_gather_mean_definition():
    rng = np.random.default_rng(61)
    V = _f32(rng.standard_normal((9, 5)))
    idx = np.array([8, 0, 0, 3], np.int32)
    np.testing.assert_allclose(O.gather_mean(V, idx), V[idx].astype(np.float64).mean(0), atol=1e-15)


@pytest.mark.parametrize("kind", ["systematic", "stratified"])
def test_sampled_indices_structural_invariants(kind):
    w = make_workload(2, B=2, n=700, kind=kind, S=64, ctx_len=[700, 333], seed=3)
    res = O.decode_workload(w, want_cdf=True)
    for r in range(w.B * w.Hq):
        b = r // w.Hq
        L = int(w.ctx_len[b])
        ix = res.idx[r]
        assert ix.size == w.S
        assert np.all(np.diff(ix) >= 0) and ix.min() >= 0 and ix.max() < L
        p = np.diff(np.concatenate([[0.0], res.cdf[r, :L]]))
        assert np.all(p[ix] > 0)


def test_zero_length_row_convention():
    w = make_workload(2, B=2, Hq=4, Hkv=1, n=50, ctx_len=[50, 0], S=8, seed=4)
    res = O.decode_workload(w)
    assert np.all(res.out[4:] == 0) and np.all(res.idx[4:] == -1)

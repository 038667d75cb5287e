"""Pins of the oracle's coverage objective and batched responsibility solver:
normalised/monotone/submodular F (Eq. cond-submodular), brute-force checks of
the deployed certificate (Eq. deployed-approximation, cond-batched-bound) and
final certificate (Eq. cond-final-cert), the sequential-greedy special case
with its (1 - (1-1/K)^K) bound (Eq. cond-greedy-residual), the bank mixture
(Eq. cond-bank-mixture), the grounded-mode identity (Eq. cond-grounded-mode)
and the zero-gain stable fill (App. H totality rule)."""
import itertools
import math

import numpy as np
import pytest

from oracle import gmc_oracle as O

P = O.GmcParams()


def _rand_cbar(rng, m, n, sparsity=0.5):
    c = rng.exponential(size=(m, n)) * (rng.random((m, n)) > sparsity)
    return c / c.sum()


def _brute_opt(cbar, k):
    n = cbar.shape[1]
    best = -1.0
    for s in itertools.combinations(range(n), k):
        best = max(best, O.coverage(cbar, s))
    return best


def test_coverage_normalised_monotone_submodular():
    rng = np.random.default_rng(0)
    cbar = _rand_cbar(rng, 15, 10)
    assert O.coverage(cbar, []) == 0.0
    for _ in range(200):
        a = set(rng.choice(10, size=rng.integers(0, 5), replace=False).tolist())
        b = a | set(rng.choice(10, size=rng.integers(0, 4), replace=False).tolist())
        i = int(rng.integers(10))
        if i in b:
            continue
        fa, fb = O.coverage(cbar, a), O.coverage(cbar, b)
        assert fb >= fa - 1e-15
        ga = O.coverage(cbar, a | {i}) - fa
        gb = O.coverage(cbar, b | {i}) - fb
        assert ga >= gb - 1e-15


def test_marginal_gains_equal_set_differences():
    # Delta(i | S) = F(S u {i}) - F(S) = sum_m [Cbar_mi - b_m(S)]_+
    rng = np.random.default_rng(1)
    cbar = _rand_cbar(rng, 12, 9)
    s = [2, 5]
    cov = cbar[:, s].max(axis=1)
    u = O.marginal_gains(cbar, cov)
    for i in range(9):
        assert u[i] == pytest.approx(O.coverage(cbar, s + [i]) - O.coverage(cbar, s), abs=1e-15)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("k,b", [(3, 1), (4, 2), (5, 2), (6, 3)])
def test_batched_certificate_against_brute_force(seed, k, b):
    # F(S_T) >= c_B F(S*) + (1 - c_B) F(S_0) with S_0 empty, and
    # F(S)/F(V) <= F(S)/F(S*) <= 1
    rng = np.random.default_rng(100 + seed)
    n = 11
    cbar = _rand_cbar(rng, 14, n)
    p = O.GmcParams(pool_mult=2)
    sel = O.select_support(cbar, k, b, p)
    assert len(set(sel["order"].tolist())) == k
    opt = _brute_opt(cbar, k)
    fs = O.coverage(cbar, sel["order"])
    assert fs == pytest.approx(sel["f_s"], rel=1e-12)
    assert fs >= sel["c_b"] * opt - 1e-14
    assert all(0.0 <= r["q"] <= 1.0 + 1e-12 for r in sel["rounds"])
    fv = O.coverage(cbar, range(n))
    assert fs / fv <= fs / opt + 1e-14 <= 1.0 + 1e-12
    assert len(sel["rounds"]) == math.ceil(k / b)


def _textbook_greedy(cbar, k):
    n = cbar.shape[1]
    s = []
    for _ in range(k):
        base = O.coverage(cbar, s)
        gains = [(O.coverage(cbar, s + [i]) - base, -i) for i in range(n) if i not in s]
        g, neg_i = max(gains)
        s.append(-neg_i)
    return s


@pytest.mark.parametrize("seed", range(8))
def test_single_token_batches_reduce_to_sequential_greedy(seed):
    # b = 1 with a pool of one is exact sequential greedy; it meets
    # F(S_K) >= [1 - (1 - 1/K)^K] F(S*)
    rng = np.random.default_rng(200 + seed)
    n, k = 10, 4
    cbar = _rand_cbar(rng, 13, n, sparsity=0.3)
    p = O.GmcParams(pool_mult=1)
    sel = O.select_support(cbar, k, 1, p)
    greedy = _textbook_greedy(cbar, k)
    assert sel["order"].tolist() == greedy
    opt = _brute_opt(cbar, k)
    assert O.coverage(cbar, greedy) >= (1 - (1 - 1 / k) ** k) * opt - 1e-14


def test_zero_gain_tokens_fill_in_source_order():
    # App. H: when all remaining gains are zero, stable source order fills the
    # exact budget without changing F
    m, n = 6, 10
    cbar = np.zeros((m, n))
    cbar[0:2, 7] = [0.3, 0.1]
    cbar[2:4, 3] = [0.2, 0.25]
    cbar[4:6, 5] = [0.05, 0.1]
    sel = O.select_support(cbar, 6, 2, P)
    assert sel["order"].tolist() == [3, 7, 5, 0, 1, 2]
    assert sel["f_s"] == pytest.approx(cbar.max(axis=1).sum())


def test_responsibility_prefers_complementary_tokens():
    # Eq. responsibility: two duplicates covering one client group and one
    # token covering another.  Singleton gains rank the duplicates first, but
    # responsibility splits the group's residual between the duplicates, so a
    # batch of two takes one duplicate and the complementary token.
    cbar = np.array([[0.50, 0.50, 0.00],
                     [0.50, 0.50, 0.00],
                     [0.00, 0.00, 0.60]])
    p = O.GmcParams(pool_mult=2)
    sel = O.select_support(cbar, 2, 2, p)
    assert sorted(sel["order"].tolist()) == [0, 2]


def test_pool_and_batch_sizes_in_last_round():
    # reading R11: pool = min(4b, N - |S|), last batch = K - |S|
    rng = np.random.default_rng(3)
    cbar = _rand_cbar(rng, 20, 30, sparsity=0.1)
    sel = O.select_support(cbar, 21, 8, P)
    sizes = [len(r["batch"]) for r in sel["rounds"]]
    assert sizes == [8, 8, 5]
    pools = [len(r["pool"]) for r in sel["rounds"]]
    assert pools == [30, 22, 14]


def test_bank_mixture_and_final_certificate():
    # Eq. cond-bank-mixture: F(S)/F(V) = sum_b omega_b c_b, sum omega_b = 1
    rng = np.random.default_rng(4)
    n, t, hq = 30, 3, 2
    h = rng.standard_normal((n, 16))
    q = rng.standard_normal((t, hq, 8))
    k = rng.standard_normal((n, 1, 8))
    g = rng.standard_normal((hq, 4, 16)) / 4
    yy, xx = np.divmod(np.arange(n), 6)
    pos = np.stack([np.zeros(n, int), yy, xx], axis=1)
    r = O.gmc_single(h, q, k, pos, g, 9, P)
    sat = r["saturation"]
    assert sum(v["omega"] for v in sat.values()) == pytest.approx(1.0)
    mix = sum(v["omega"] * v["c"] for v in sat.values())
    assert mix == pytest.approx(r["selection"]["f_s"] / r["f_v"], rel=1e-12)


def test_grounded_mode_identity():
    # Eq. cond-grounded-mode: max_(j in S) e_gj = max_i e_gi - (Z_g / alpha_g) D_g
    rng = np.random.default_rng(5)
    n, t, hq = 20, 4, 2
    h = rng.standard_normal((n, 12))
    q = rng.standard_normal((t, hq, 6))
    k = rng.standard_normal((n, 1, 6))
    g = rng.standard_normal((hq, 4, 12)) / 3
    yy, xx = np.divmod(np.arange(n), 5)
    pos = np.stack([np.zeros(n, int), yy, xx], axis=1)
    cl = O.build_clients(h, q, k, pos, g, P)
    s = np.array([1, 4, 9, 13])
    for hh in range(hq):
        for tt in range(t):
            e = cl["e"][hh, tt]
            zg = e.sum()
            alpha = P.beta_msg * cl["omega"][hh] * cl["nu"][tt]
            row = cl["cbar"][hh * t + tt]
            np.testing.assert_allclose(row, alpha * e / zg, rtol=1e-12)
            dg = alpha * (row.max() / alpha - row[s].max() / alpha)
            assert e[s].max() == pytest.approx(e.max() - zg / alpha * dg, rel=1e-10)


def test_bank_matrix_mass_equals_nominal_mass():
    # Eq. cond-effective-bank-mass: the deployed matrix mass of bank b is
    # beta_b M_b^-1 sum_m a_m; rows are normalised, so with every row active
    # the appearance rows total 0.5, the spatial rows 0.25 and the grounded
    # rows beta_msg sum_h omega_h sum_t nu_t = 1
    rng = np.random.default_rng(6)
    n, t, hq = 25, 3, 4
    h = rng.standard_normal((n, 10))
    q = rng.standard_normal((t, hq, 6))
    k = rng.standard_normal((n, 2, 6))
    g = rng.standard_normal((hq, 4, 10)) / 3
    yy, xx = np.divmod(np.arange(n), 5)
    pos = np.stack([np.zeros(n, int), yy, xx], axis=1)
    cl = O.build_clients(h, q, k, pos, g, P)
    tot = {b: cl["cbar"][cl["banks"] == b].sum() for b in (0, 1, 2)}
    assert tot[0] == pytest.approx(P.beta_msg, rel=1e-12)
    assert tot[1] == pytest.approx(P.beta_app, rel=1e-12)
    assert tot[2] == pytest.approx(P.beta_spa, rel=1e-12)
    assert cl["cbar"].shape[0] == hq * t + n + P.landmarks ** 2

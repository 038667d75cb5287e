"""Pins of the oracle's appearance and spatial banks: the Gibbs modal
identity and coverage-quantization bound (App. I Eq. cond-gibbs,
cond-coverage-quantization), the bounded bank reducing to the exact bank
under an orthogonal +-1 projection, and the landmark modes on a 16x16 grid."""
import math

import numpy as np
import pytest
import scipy.linalg

from oracle import gmc_oracle as O

P = O.GmcParams()


def _unit(rng, n, d):
    x = rng.standard_normal((n, d))
    return x / np.linalg.norm(x, axis=1, keepdims=True)


def test_appearance_rows_are_distributions():
    x = _unit(np.random.default_rng(0), 30, 8)
    pv = O.appearance_bank(x, P)
    np.testing.assert_allclose(pv.sum(axis=1), 1.0, rtol=1e-12)
    assert np.all(pv > 0)


@pytest.mark.parametrize("seed", range(4))
def test_gibbs_modal_identity(seed):
    # Eq. cond-gibbs: max_(j in S) P^V_m(j) / P^V_m(m) = exp(-d_m(S)^2 / (2 tau_v))
    rng = np.random.default_rng(seed)
    x = _unit(rng, 40, 6)
    pv = O.appearance_bank(x, P)
    s = rng.choice(40, size=7, replace=False)
    d = np.min(np.linalg.norm(x[:, None, :] - x[None, s, :], axis=2), axis=1)
    ratio = pv[:, s].max(axis=1) / np.diag(pv)
    np.testing.assert_allclose(ratio, np.exp(-d ** 2 / (2 * P.tau_v)), rtol=1e-10)


@pytest.mark.parametrize("seed", range(4))
def test_coverage_quantization_bound(seed):
    # Eq. cond-coverage-quantization: (1/N) sum d_m^2 <= 2 tau_v D_V / (beta_V p0 r0)
    rng = np.random.default_rng(10 + seed)
    n = 50
    x = _unit(rng, n, 5)
    pv = O.appearance_bank(x, P)
    s = rng.choice(n, size=12, replace=False)
    d = np.min(np.linalg.norm(x[:, None, :] - x[None, s, :], axis=2), axis=1)
    self_mass = np.diag(pv)
    r = pv[:, s].max(axis=1) / self_mass
    p0, r0 = self_mass.min(), r.min()
    deficit = P.beta_app / n * np.sum(self_mass * (1 - r))
    assert np.mean(d ** 2) <= 2 * P.tau_v / (P.beta_app * p0 * r0) * deficit * (1 + 1e-12)


def test_bounded_bank_with_hadamard_projection_equals_exact_bank():
    # a Hadamard +-1 projection is sqrt(d) times an orthogonal map, so the
    # normalised projected states keep every cosine: with M_V = N the bounded
    # bank equals the exact one, and with M_V < N it keeps rows floor(kN/M_V)
    d, n = 64, 20
    rng = np.random.default_rng(3)
    h = rng.standard_normal((n, d)) * rng.uniform(0.5, 3, size=(n, 1))
    had = scipy.linalg.hadamard(d).astype(float)
    p_all = O.GmcParams(app_max_clients=n)
    pv_b, clients = O.appearance_bank_bounded(h, had, p_all)
    _, x, _, _ = O.row_features(h, P)
    pv = O.appearance_bank(x, P)
    np.testing.assert_allclose(pv_b, pv, rtol=1e-10)
    assert np.array_equal(clients, np.arange(n))
    p_sub = O.GmcParams(app_max_clients=6)
    pv_s, cl_s = O.appearance_bank_bounded(h, had, p_sub)
    assert np.array_equal(cl_s, [0, 3, 6, 10, 13, 16])
    np.testing.assert_allclose(pv_s, pv[cl_s], rtol=1e-10)


def test_spatial_landmark_modes_on_16x16_grid():
    # 16x16 landmarks on a 16x16 grid: landmark (a,b) sits exactly on the
    # cell centre of token (a,b), which is its unique mode
    yy, xx = np.divmod(np.arange(256), 16)
    pos = np.stack([np.zeros(256, int), yy, xx], axis=1)
    ps = O.spatial_bank(pos, P)
    assert ps.shape == (256, 256)
    np.testing.assert_allclose(ps.sum(axis=1), 1.0, rtol=1e-12)
    assert np.array_equal(np.argmax(ps, axis=1), np.arange(256))
    srt = np.sort(ps, axis=1)
    assert np.all(srt[:, -1] > srt[:, -2])


def test_spatial_coordinates_ignore_time_and_offsets():
    # reading R6: (h, w) cell centres in [0,1]^2; the temporal id is not used
    yy, xx = np.divmod(np.arange(12), 4)
    pos = np.stack([np.arange(12) % 3, yy + 5, xx + 2], axis=1)
    pc = O.spatial_coordinates(pos)
    np.testing.assert_allclose(pc[:, 0], (yy + 0.5) / 3)
    np.testing.assert_allclose(pc[:, 1], (xx + 0.5) / 4)


def test_spatial_bank_is_gaussian_in_distance():
    # P^S_m(i) / P^S_m(j) = exp(-(|p_i - l|^2 - |p_j - l|^2)/tau_s) for one row
    yy, xx = np.divmod(np.arange(36), 6)
    pos = np.stack([np.zeros(36, int), yy, xx], axis=1)
    ps = O.spatial_bank(pos, P)
    pc = O.spatial_coordinates(pos)
    a, b = 3, 11
    land = np.array([(a + 0.5) / 16, (b + 0.5) / 16])
    d2 = np.sum((pc - land) ** 2, axis=1)
    row = ps[a * 16 + b]
    np.testing.assert_allclose(row / row[0], np.exp(-(d2 - d2[0]) / P.tau_s), rtol=1e-9)

"""Pins of the oracle's historical message views (App. H "Native message
clients": separate client rows per completed view, head patterns concatenated
over views with sqrt(beta_v) after scaling each view's atoms to unit average
norm, Eq. cond-head-pattern; energy from the current view, Eq.
cond-grounded-energy; masses of Table cond-config, reading R14).  CPU only."""
import math

import numpy as np
import pytest

from oracle import gmc_oracle as O

P = O.GmcParams()


def _view(seed, n=30, t=4, d=32, hq=4, hkv=2, dh=8):
    rng = np.random.default_rng(seed)
    return dict(hidden=rng.standard_normal((n, d)), q=rng.standard_normal((t, hq, dh)),
                k=rng.standard_normal((n, hkv, dh)), probe=rng.standard_normal((hq, 4, d)) / math.sqrt(d))


def _pos(n, w=6):
    yy, xx = np.divmod(np.arange(n), w)
    return np.stack([np.zeros(n, int), yy, xx], axis=1).astype(np.int32)


def _run(cur, hist, k_req=9, p=P):
    return O.gmc_single(cur["hidden"], cur["q"], cur["k"], _pos(cur["hidden"].shape[0]), cur["probe"], k_req, p,
                        keep_intermediates=True, hist=hist)


def test_view_masses_of_the_configuration_table():
    # current/history mass 0.5/0.5 with two historical views; one view alone
    # carries the whole message mass
    assert O.view_mass(2, P) == [0.5, 0.25, 0.25]
    assert O.view_mass(1, P) == [0.5, 0.5]
    assert O.view_mass(0, P) == [1.0]


def test_zero_history_mass_reduces_to_the_single_view_operator():
    cur = _view(1)
    hist = [_view(2), _view(3)]
    p0 = O.GmcParams(hist_mass=0.0)
    single = _run(cur, [])
    views = _run(cur, hist, p=p0)
    assert np.array_equal(views["out_idx"], single["out_idx"])
    np.testing.assert_allclose(views["out_hidden"], single["out_hidden"], rtol=1e-12, atol=0)
    np.testing.assert_allclose(views["clients"]["omega"], single["clients"]["omega"], rtol=1e-12)
    mg = cur["q"].shape[0] * cur["probe"].shape[0]
    cb = views["clients"]["cbar"]
    assert cb.shape[0] == single["clients"]["cbar"].shape[0] + 2 * mg
    assert np.all(cb[mg:3 * mg] == 0.0)          # the historical rows carry no mass


def test_head_pattern_is_the_gram_of_concatenated_normalised_atoms():
    # Eq. cond-head-pattern written out: per head, concatenate over views the
    # flattened atoms A[t,i] [Z_h[i]; sigma_h] divided by the view's mean atom
    # norm and scaled by sqrt(beta_v); the pattern Gram is their Gram matrix
    views = [O.message_view(v["hidden"], v["q"], v["k"], v["probe"], P) for v in (_view(4), _view(5), _view(6))]
    mass = [0.5, 0.25, 0.25]
    hq = views[0]["a"].shape[0]
    flat = []
    for hh in range(hq):
        parts = []
        for v, beta in zip(views, mass):
            atoms = []
            for t in range(v["a"].shape[1]):
                for i in range(v["a"].shape[2]):
                    atoms.append(v["a"][hh, t, i] * np.append(v["z"][hh, i], v["sigma"][hh]))
            atoms = np.array(atoms)
            abar = np.mean(np.linalg.norm(atoms, axis=1))
            parts.append(math.sqrt(beta) * atoms.ravel() / abar)
        flat.append(np.concatenate(parts))
    flat = np.array(flat)
    got = O.head_pattern([v["gram"] for v in views], [v["abar"] for v in views], mass)
    np.testing.assert_allclose(got, flat @ flat.T, rtol=1e-10)


def test_duplicated_current_view_is_the_single_view_operator():
    # two historical views equal to the current one: the three copies of each
    # grounded row (masses 0.5, 0.25, 0.25) cover like one row of mass 1, the
    # pattern Gram is the single view's, so omega, F on any support and the
    # selected support are the single-view operator's
    cur = _view(7, hq=8)
    single = _run(cur, [])
    dup = _run(cur, [dict(cur), dict(cur)])
    np.testing.assert_allclose(dup["clients"]["omega"], single["clients"]["omega"], rtol=1e-12)
    mg = cur["q"].shape[0] * cur["probe"].shape[0]
    cb, cs = dup["clients"]["cbar"], single["clients"]["cbar"]
    np.testing.assert_allclose(cb[:mg] + cb[mg:2 * mg] + cb[2 * mg:3 * mg], cs[:mg], rtol=1e-13, atol=1e-18)
    rng = np.random.default_rng(0)
    for _ in range(5):
        sup = rng.choice(cur["hidden"].shape[0], size=6, replace=False)
        assert O.coverage(cb, sup) == pytest.approx(O.coverage(cs, sup), rel=1e-12)
    assert np.array_equal(dup["out_idx"], single["out_idx"])


def test_history_scale_invariance_and_current_view_energy():
    # each view's atoms are scaled to unit average norm, so multiplying a
    # historical view's probe by 4 (exact in binary) changes its raw atoms but
    # not the head pattern, its client rows or anything downstream; the
    # population weights use the current view's energy only, so they do not
    # move either
    cur, h1, h2 = _view(8, hq=8), _view(9, hq=8), _view(10, hq=8)
    base = _run(cur, [h1, h2])
    h1s = dict(h1)
    h1s["probe"] = 4.0 * h1["probe"]
    scaled = _run(cur, [h1s, h2])
    v0 = base["clients"]["hist_views"][0]
    v1 = scaled["clients"]["hist_views"][0]
    assert not np.allclose(v0["e"], v1["e"])
    np.testing.assert_allclose(v1["e"], 4.0 * v0["e"], rtol=1e-12)
    np.testing.assert_allclose(scaled["clients"]["pattern"], base["clients"]["pattern"], rtol=1e-12)
    np.testing.assert_allclose(scaled["clients"]["cbar"], base["clients"]["cbar"], rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(scaled["clients"]["ebar"], base["clients"]["ebar"], rtol=1e-12)
    assert np.array_equal(scaled["out_idx"], base["out_idx"])
    # swapping which of two views is current (equal masses 0.5 / 0.5) keeps
    # the head pattern and omega and swaps the two views' grounded row
    # blocks, but the energy follows the current view's atoms
    a, b = _view(14, hq=8), _view(15, hq=8)
    ab = _run(a, [b])["clients"]
    ba = _run(b, [a])["clients"]
    np.testing.assert_allclose(ab["pattern"], ba["pattern"], rtol=1e-12)
    np.testing.assert_allclose(ab["omega"], ba["omega"], rtol=1e-12)
    assert np.unique(np.round(ab["omega"], 12)).size > 1        # not the trivial uniform split
    mg = a["q"].shape[0] * a["probe"].shape[0]
    np.testing.assert_allclose(ab["cbar"][:mg], ba["cbar"][mg:2 * mg], rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(ab["cbar"][mg:2 * mg], ba["cbar"][:mg], rtol=1e-12, atol=1e-18)
    en_a = O.grounded_energy(ab["e"], ab["omega"], ab["nu"])[0]
    en_b = O.grounded_energy(ba["e"], ab["omega"], ab["nu"])[0]
    np.testing.assert_allclose(ab["ebar"], en_a, rtol=1e-12)
    np.testing.assert_allclose(ba["ebar"], en_b, rtol=1e-12)
    assert not np.allclose(en_a, en_b)


def test_grounded_bank_mass_with_views():
    # every active grounded row is a distribution and the view masses sum to
    # beta_msg, so the grounded rows of all views carry beta_msg in total
    # (head weights and query weights each sum to one)
    cur = _view(11)
    r = _run(cur, [_view(12), _view(13)])
    c = r["clients"]
    assert np.all(c["active"]) and all(np.all(v["active"]) for v in c["hist_views"])
    grounded = c["cbar"][c["banks"] == 0]
    assert grounded.sum() == pytest.approx(P.beta_msg, rel=1e-12)

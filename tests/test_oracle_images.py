"""Pins of the oracle's multi-image prompts (Sec. 3.1 totality rule
K = min{N, max{K_r, I}}; App. H "Batched complementary support": one
max-gain seed per image; Eq. cond-aux-clients: appearance and spatial rows
restricted to their image, landmarks on each image's own grid; Eq.
cond-assignment: image-compatible carriers only; reading R15).  CPU only."""
import math

import numpy as np
import pytest

from oracle import gmc_oracle as O

P = O.GmcParams()


def _prompt(seed=0, grids=((5, 6), (4, 4), (3, 5)), t=4, d=32, hq=4, hkv=2, dh=8):
    """Images laid out one after another; positions (0, row, col) on each
    image's own grid, offset in h so that raw grids do not coincide."""
    rng = np.random.default_rng(seed)
    pos, img = [], []
    for g, (gh, gw) in enumerate(grids):
        yy, xx = np.divmod(np.arange(gh * gw), gw)
        pos.append(np.stack([np.zeros(gh * gw, int), yy + 7 * g, xx + 3 * g], axis=1))
        img.append(np.full(gh * gw, g))
    pos = np.concatenate(pos).astype(np.int32)
    img = np.concatenate(img)
    n = pos.shape[0]
    h = rng.standard_normal((n, d))
    q = rng.standard_normal((t, hq, dh))
    k = rng.standard_normal((n, hkv, dh))
    probe = rng.standard_normal((hq, 4, d)) / math.sqrt(d)
    return h, q, k, pos, probe, img


def _run(k_req, seed=0, **kw):
    h, q, k, pos, probe, img = _prompt(seed, **kw)
    r = O.gmc_single(h, q, k, pos, probe, k_req, P, keep_intermediates=True, img=img)
    return r, img


def test_budget_expands_to_one_carrier_per_image():
    # K_r = 1 < I = 3: the budget becomes 3, one carrier in each image
    r, img = _run(1)
    assert r["k"] == 3
    assert sorted(img[r["out_idx"]].tolist()) == [0, 1, 2]
    assert r["selection"]["rounds"] == []            # the seeds fill the budget


def test_seeds_are_each_images_largest_singleton_gain():
    r, img = _run(12)
    cb = r["clients"]["cbar"]
    u = cb.sum(axis=0)                                # F({i}) from the empty set
    order = r["selection"]["order"]
    for g in range(3):
        members = np.flatnonzero(img == g)
        best = members[u[members] == u[members].max()].min()
        assert order[g] == best
    # the certificate's anchor F(S_0) is the seeds' coverage
    assert r["selection"]["f0"] == pytest.approx(O.coverage(cb, order[:3]), rel=1e-14)


def test_assignment_never_crosses_an_image_and_every_image_keeps_a_carrier():
    for k_req in (3, 5, 12, 30):
        r, img = _run(k_req, seed=1)
        pi = r["assignment"]["pi"]
        assert np.all(img[pi] == img), k_req
        assert set(img[r["out_idx"]].tolist()) == {0, 1, 2}
        # each carrier's population stays inside its image
        assert np.all(r["transport"]["mass"] > 0)


def test_single_carrier_images_have_zero_gap():
    # K = I: every image has exactly one carrier, so every gap is 0 and the
    # separability gate closes (s_x = 0): uniform population weights
    r, img = _run(1, seed=2)
    a = r["assignment"]
    assert np.all(a["delta"] == 0.0)
    assert a["sx"] == 0.0
    assert np.all(r["m"] == 1.0)


def test_appearance_and_spatial_rows_stay_in_their_image():
    r, img = _run(12, seed=3)
    c = r["clients"]
    pv, ps = c["pv"], c["ps"]
    same = img[:, None] == img[None, :]
    assert np.all(pv[~same] == 0.0)
    np.testing.assert_allclose(pv.sum(axis=1), 1.0, rtol=1e-13)
    L2 = P.landmarks ** 2
    assert ps.shape[0] == 3 * L2
    h, q, k, pos, probe, _ = _prompt(3)
    for g in range(3):
        members = np.flatnonzero(img == g)
        rows = ps[g * L2:(g + 1) * L2]
        assert np.all(np.delete(rows, members, axis=1) == 0.0)
        # each image's landmark rows are the single-image spatial bank of its
        # own tokens on its own grid
        np.testing.assert_allclose(rows[:, members], O.spatial_bank(pos[members], P), rtol=1e-12, atol=1e-300)
    # masses: beta / M_b per row, every row a distribution
    cb, banks = c["cbar"], c["banks"]
    assert cb[banks == 1].sum() == pytest.approx(P.beta_app, rel=1e-12)
    assert cb[banks == 2].sum() == pytest.approx(P.beta_spa, rel=1e-12)


def test_one_image_is_the_single_image_operator():
    h, q, k, pos, probe, img = _prompt(4)
    zero = np.zeros(h.shape[0], dtype=np.int64)
    a = O.gmc_single(h, q, k, pos, probe, 9, P, img=zero)
    b = O.gmc_single(h, q, k, pos, probe, 9, P)
    assert np.array_equal(a["out_idx"], b["out_idx"])
    np.testing.assert_array_equal(a["out_hidden"], b["out_hidden"])


def test_images_with_unrelated_content_split_the_budget_by_coverage():
    # a tiny brute-force check of the objective the seeds start: with T = 0
    # the client matrix is block diagonal over the images, so F is the sum of
    # the images' own facility objectives on their carriers
    h, q, k, pos, probe, img = _prompt(5, t=0)
    r = O.gmc_single(h, q[:0], k, pos, probe, 7, P, keep_intermediates=True, img=img)
    cb = r["clients"]["cbar"]
    sup = r["selection"]["order"]
    total = 0.0
    for g in range(3):
        rows = np.flatnonzero(np.any(cb[:, img == g] > 0, axis=1))
        assert np.all(cb[np.ix_(rows, np.flatnonzero(img != g))] == 0.0)
        total += O.coverage(cb[rows], sup[img[sup] == g]) if np.any(img[sup] == g) else 0.0
    assert O.coverage(cb, sup) == pytest.approx(total, rel=1e-13)

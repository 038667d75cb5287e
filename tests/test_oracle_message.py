"""Pins of the oracle's budget rule and message side against what the paper
fixes: the totality rule, closed forms of the native softmax slice, the mass
coordinate, the head-weight formula on constructed patterns, and the energy
fallback.  CPU only."""
import json
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import gmc_oracle as O

P = O.GmcParams()
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_frozen_constants_match_config_table():
    # App. H Table cond-config: every deployed constant, read from a fixture
    with open(os.path.join(GOLDEN, "config_table.json")) as f:
        table = json.load(f)
    for key, val in table.items():
        if key.startswith("_"):
            continue
        assert getattr(P, key) == pytest.approx(val, rel=0, abs=0), key


@pytest.mark.parametrize("n,kr,imgs,want", [(10, 20, 1, 10), (10, 0, 1, 1), (10, -3, 1, 1),
                                            (10, 4, 1, 4), (10, 1, 3, 3), (5, 5, 1, 5)])
def test_budget_totality_rule(n, kr, imgs, want):
    # Sec. 3.1: K = min{N, max{K_r, I}}
    assert O.realized_budget(n, kr, imgs) == want


def _small(seed=0, n=24, t=5, d=32, hq=4, hkv=2, dh=8):
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((n, d))
    q = rng.standard_normal((t, hq, dh))
    k = rng.standard_normal((n, hkv, dh))
    g = rng.standard_normal((hq, 4, d)) / math.sqrt(d)
    yy, xx = np.divmod(np.arange(n), 6)
    pos = np.stack([np.zeros(n, int), yy, xx], axis=1).astype(np.int32)
    return h, q, k, g, pos


def test_identity_when_k_equals_n():
    # App. H totality rule: K = N returns the unmodified execution
    h, q, k, g, pos = _small()
    for kr in (24, 100):
        r = O.gmc_single(h, q, k, pos, g, kr, P)
        assert r["identity"]
        assert np.array_equal(r["out_hidden"], h)
        assert np.array_equal(r["out_pos"], pos)
        assert np.array_equal(r["out_idx"], np.arange(24))


def test_native_attention_is_library_softmax_over_all_keys():
    # Eq. cond-native-message: the visual columns of one softmax over the
    # visual and nonvisual keys; here the nonvisual keys are summarised by a
    # log-sum-exp column, so scipy's softmax over [visual, nonvisual] must agree
    h, q, k, g, pos = _small(1)
    t, hq, dh = q.shape
    nonvis = np.random.default_rng(3).standard_normal((hq, t)) * 2.0
    a = O.native_attention(q, k, nonvis)
    for hh in range(hq):
        kv = hh // (hq // k.shape[1])
        logits = q[:, hh, :] @ k[:, kv, :].T / math.sqrt(dh)
        full = scipy.special.softmax(np.concatenate([logits, nonvis[hh][:, None]], axis=1), axis=1)
        np.testing.assert_allclose(a[hh], full[:, :-1], rtol=1e-12, atol=0)
    a0 = O.native_attention(q, k, None)
    for hh in range(hq):
        kv = hh // (hq // k.shape[1])
        ref = scipy.special.softmax(q[:, hh, :] @ k[:, kv, :].T / math.sqrt(dh), axis=1)
        np.testing.assert_allclose(a0[hh], ref, rtol=1e-12, atol=0)


def test_gqa_head_mapping():
    # query head h reads kv head floor(h Hkv / Hq): zero keys on kv head 1 make
    # heads 2,3 (of 4, 2 kv heads) uniform and leave heads 0,1 peaked
    h, q, k, g, pos = _small(2)
    k = k.copy()
    k[:, 1, :] = 0.0
    a = O.native_attention(q, k)
    n = k.shape[0]
    assert np.allclose(a[2], 1.0 / n) and np.allclose(a[3], 1.0 / n)
    assert not np.allclose(a[0], 1.0 / n) and not np.allclose(a[1], 1.0 / n)


def _clients(h, q, k, pos, g, nonvis=None, p=P):
    return O.build_clients(h, q, k, pos, g, p, None, nonvis)


def test_grounded_rows_are_distributions_and_ignore_nonvisual_denominator():
    # Eq. grounded-client: P^G = ||u_i|| / sum_j ||u_j||; the native row
    # denominator scales every atom of a row equally and cancels
    h, q, k, g, pos = _small(4)
    c0 = _clients(h, q, k, pos, g)
    nonvis = np.random.default_rng(5).standard_normal((q.shape[1], q.shape[0])) * 3.0
    c1 = _clients(h, q, k, pos, g, nonvis)
    np.testing.assert_allclose(c0["pg"].sum(axis=2), 1.0, rtol=1e-12)
    assert np.all(c0["pg"] >= 0)
    np.testing.assert_allclose(c1["pg"], c0["pg"], rtol=1e-10, atol=1e-15)
    assert not np.allclose(c1["a"], c0["a"])       # the attention mass did change


def test_grounded_rows_with_zero_probe_equal_attention():
    # G = 0 => Z = 0 => sigma = eps_mass (Eq. mass-coordinate) for every head,
    # every atom is A[t,i] * [0; eps] and P^G equals the attention row itself
    h, q, k, g, pos = _small(6)
    c = _clients(h, q, k, pos, np.zeros_like(g))
    assert np.all(c["sigma"] == P.eps_mass)
    np.testing.assert_allclose(c["pg"], c["a"], rtol=1e-12)


def test_uniform_attention_gives_norm_proportional_client():
    # q = 0 => A = 1/N exactly, so P^G(i) = ||w_h[i]|| / sum_j ||w_h[j]||
    h, q, k, g, pos = _small(7)
    c = _clients(h, np.zeros_like(q), k, pos, g)
    n = h.shape[0]
    assert np.allclose(c["a"], 1.0 / n, rtol=1e-14)
    for hh in range(g.shape[0]):
        w = np.concatenate([c["z"][hh], np.full((n, 1), c["sigma"][hh])], axis=1)
        l2 = np.linalg.norm(w, axis=1)
        np.testing.assert_allclose(c["pg"][hh, 0], l2 / l2.sum(), rtol=1e-12)


def test_mass_coordinate_of_identical_tokens():
    # all tokens equal => every Z_h[i] = z0 and ||Z_h||_F / sqrt(N r) = ||z0|| / sqrt(r)
    rng = np.random.default_rng(8)
    d, n = 16, 9
    v = rng.standard_normal(d)
    h = np.tile(v, (n, 1))
    g = rng.standard_normal((3, 4, d))
    _, _, _, xt = O.row_features(h, P)
    z = O.value_probe(xt, g)
    sig = O.mass_coordinate(z, P)
    xv = v / math.sqrt(np.mean(v * v) + P.rms_eps)
    for hh in range(3):
        z0 = g[hh] @ xv
        assert sig[hh] == pytest.approx(np.linalg.norm(z0) / 2.0, rel=1e-12)


def test_folded_value_probe_with_bias():
    # Z_h = (V_h O_h) P with V = x~ W^V + b^V, computed step by step, equals
    # the folded map x~ G_h + b_h with G_h = (W^V O_h P)^T and b_h = b^V O_h P
    rng = np.random.default_rng(21)
    n, d, dh, r, hq = 7, 24, 8, 4, 3
    h = rng.standard_normal((n, d))
    wv = rng.standard_normal((hq, d, dh))
    bv = rng.standard_normal((hq, dh))
    o = rng.standard_normal((hq, dh, d))
    pr, _ = np.linalg.qr(rng.standard_normal((d, r)))
    _, _, _, xt = O.row_features(h, P)
    g = np.zeros((hq, r, d))
    bias = np.zeros((hq, r))
    ref = np.zeros((hq, n, r))
    for hh in range(hq):
        v = xt @ wv[hh] + bv[hh]
        ref[hh] = (v @ o[hh]) @ pr
        g[hh] = (wv[hh] @ o[hh] @ pr).T
        bias[hh] = bv[hh] @ o[hh] @ pr
    np.testing.assert_allclose(O.value_probe(xt, g, bias), ref, rtol=1e-10, atol=1e-10)
    # without the bias term the folded map misses exactly b_h on every token
    np.testing.assert_allclose(O.value_probe(xt, g), ref - bias[:, None, :], rtol=1e-10, atol=1e-10)


def test_rmsnorm_features():
    # x~ = h / sqrt(mean h^2 + eps): mean square ms/(ms+eps); x is unit
    h, *_ = _small(9)
    norm, x, rms, xt = O.row_features(h, P)
    ms = np.mean(h * h, axis=1)
    np.testing.assert_allclose(np.mean(xt * xt, axis=1), ms / (ms + P.rms_eps), rtol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(x, axis=1), 1.0, rtol=1e-12)
    np.testing.assert_allclose(rms, np.sqrt(ms), rtol=1e-12)


def test_query_weights_terminal_double():
    # the terminal prompt query weighs twice the others; weights sum to one
    nu = O.query_weights(5, P)
    np.testing.assert_allclose(nu, [1 / 6] * 4 + [2 / 6])
    assert O.query_weights(1, P)[0] == 1.0
    assert O.query_weights(0, P).size == 0


def _gram_from_patterns(u):
    return u @ u.T


def test_head_weights_orthogonal_identical_groups():
    # Eq. cond-head-weight: 4 mutually orthogonal groups of identical patterns
    # have zero dispersion, so every member gets (1/4)/n_c exactly
    rng = np.random.default_rng(10)
    basis = np.linalg.qr(rng.standard_normal((12, 4)))[0].T     # 4 orthonormal rows
    groups = [0, 0, 1, 2, 2, 2, 3, 1, 0, 3]
    scale = rng.uniform(0.5, 2.0, size=len(groups))
    u = np.stack([scale[i] * basis[gid] for i, gid in enumerate(groups)])
    abar = rng.uniform(0.1, 1.0, size=len(groups))
    omega, centres, assign = O.head_weights(_gram_from_patterns(u), abar, P)
    counts = np.bincount(groups)
    np.testing.assert_allclose(omega, [0.25 / counts[gid] for gid in groups], rtol=1e-12)
    assert omega.sum() == pytest.approx(1.0)


def test_head_weights_hand_computed_dispersion():
    # three heads around e1 (cosines 0.8 to the first) and one head on e3,
    # at most 2 clusters.  Farthest-first: centre 0 (largest pattern), then
    # head 3 (cosine 0).  Cluster {0,1,2} has mean direction e1, so
    # d = (0, 0.2, 0.2); weights inside it are proportional to
    # (1/0.05, 1/0.25, 1/0.25) = (20, 4, 4); each cluster gets 1/2.
    c, s = 0.8, 0.6
    u = np.array([[1, 0, 0], [c, s, 0], [c, -s, 0], [0, 0, 1]], dtype=float)
    u[0] *= 3.0                               # largest pre-normalisation pattern
    abar = np.ones(4)
    p2 = O.GmcParams(max_head_clusters=2)
    omega, centres, assign = O.head_weights(_gram_from_patterns(u), abar, p2)
    assert centres == [0, 3]
    np.testing.assert_allclose(omega, [10 / 28, 2 / 28, 2 / 28, 0.5], rtol=1e-12)


def test_head_weights_inactive_head_and_ties():
    # a zero-energy head gets omega = 0; a duplicate of a centre joins the
    # earliest centre; an emptied cluster is dropped from C
    u = np.array([[2, 0], [1, 0], [0, 0], [0, 1]], dtype=float)
    omega, centres, assign = O.head_weights(_gram_from_patterns(u), np.ones(4), P)
    assert omega[2] == 0.0 and assign[2] == -1
    assert omega.sum() == pytest.approx(1.0)
    np.testing.assert_allclose(omega, [0.25, 0.25, 0.0, 0.5], rtol=1e-12)


def test_head_pattern_gram_matches_flattened_atoms():
    # Gamma_hg is the inner product of the flattened atoms A_h[t,i] [Z_h[i]; sigma_h]
    h, q, k, g, pos = _small(11, n=10, t=3)
    c = _clients(h, q, k, pos, g)
    hq = g.shape[0]
    flat = []
    for hh in range(hq):
        atoms = []
        for t in range(q.shape[0]):
            for i in range(h.shape[0]):
                atoms.extend(c["a"][hh, t, i] * np.append(c["z"][hh, i], c["sigma"][hh]))
        flat.append(atoms)
    flat = np.array(flat)
    np.testing.assert_allclose(c["gram"], flat @ flat.T, rtol=1e-12)


def test_energy_fallback_and_normalisation():
    # Eq. cond-grounded-energy: ebar has mean one; T = 0 falls back to 1
    h, q, k, g, pos = _small(12)
    c = _clients(h, q, k, pos, g)
    assert c["ebar"].mean() == pytest.approx(1.0)
    c0 = _clients(h, q[:0], k, pos, g)
    assert np.all(c0["ebar"] == 1.0)
    assert c0["cbar"].shape[0] == h.shape[0] + P.landmarks ** 2


def test_energy_single_head_single_query_closed_form():
    # one head, one query: omega = nu = 1, so e_i = A[0,i] ||w[i]||
    h, q, k, g, pos = _small(13, hq=1, hkv=1, t=1)
    c = _clients(h, q, k, pos, g)
    assert c["omega"][0] == pytest.approx(1.0)
    e = c["a"][0, 0] * c["ell"][0]
    np.testing.assert_allclose(c["ebar"], e / e.mean(), rtol=1e-12)


def test_energy_two_heads_two_queries_hand_computed():
    # Eq. cond-grounded-energy with unequal head weights and T = 2 queries
    # (nu = (1/3, 2/3): the terminal query counts twice).  Atom norms:
    # head 0 has 1 at (t=0, i=0), head 1 has 2 at (t=1, i=1), all else 0.
    #   e_0^2 = omega_0 nu_0 1^2 = 1/4 * 1/3 * 1 = 1/12
    #   e_1^2 = omega_1 nu_1 2^2 = 3/4 * 2/3 * 4 = 2
    # so ebar = 2 (sqrt(1/12), sqrt(2)) / (sqrt(1/12) + sqrt(2))
    #         = (2, 2 sqrt(24)) / (1 + sqrt(24)).
    e = np.zeros((2, 2, 2))
    e[0, 0, 0] = 1.0
    e[1, 1, 1] = 2.0
    omega = np.array([0.25, 0.75])
    nu = O.query_weights(2, P)
    np.testing.assert_allclose(nu, [1 / 3, 2 / 3], rtol=1e-15)
    ebar, en = O.grounded_energy(e, omega, nu)
    np.testing.assert_allclose(en, [math.sqrt(1 / 12), math.sqrt(2)], rtol=1e-14)
    r = math.sqrt(24)
    np.testing.assert_allclose(ebar, [2 / (1 + r), 2 * r / (1 + r)], rtol=1e-14)


def test_energy_weights_heads_not_uniformly():
    # the same token energy from two heads: a head with weight 3/4 counts
    # three times a head with weight 1/4 (e^2 is linear in omega):
    # token 0 draws 1 from head 0, token 1 draws 1 from head 1, one query,
    # so e = (sqrt(1/4), sqrt(3/4)) and ebar = 2 (1, sqrt 3) / (1 + sqrt 3).
    e = np.zeros((2, 1, 2))
    e[0, 0, 0] = 1.0
    e[1, 0, 1] = 1.0
    ebar, en = O.grounded_energy(e, np.array([0.25, 0.75]), O.query_weights(1, P))
    np.testing.assert_allclose(en, [0.5, math.sqrt(0.75)], rtol=1e-14)
    s3 = math.sqrt(3)
    np.testing.assert_allclose(ebar, [2 / (1 + s3), 2 * s3 / (1 + s3)], rtol=1e-14)


def test_head_weights_first_centre_is_largest_pre_normalisation_pattern():
    # Eq. cond-head-pattern: the first farthest-first centre is the head with
    # the largest sqrt(beta Gamma_hh) / abar_h (the pattern after scaling the
    # atoms to unit average norm), not the largest raw Gram diagonal.
    # Four unit directions in a plane at 0, 50, 95 and 150 degrees; raw norms
    # (2, 1.5, 1, 1), mean atom norms (2, 1, 1, 1): the largest raw pattern is
    # head 0, the largest normalised one is head 1 (1.5 vs 1).
    #   first centre head 1 -> farthest is head 3 (100 deg); head 0 (50 deg
    #   from 1, 150 from 3) and head 2 (45 from 1, 55 from 3) join head 1:
    #   clusters {0, 1, 2} and {3}, so omega_3 = 1/2.
    #   (first centre head 0 would give centres 0, 3 and clusters {0, 1},
    #   {2, 3}, omega_3 < 1/2.)
    ang = np.radians([0.0, 50.0, 95.0, 150.0])
    norms = np.array([2.0, 1.5, 1.0, 1.0])
    u = norms[:, None] * np.stack([np.cos(ang), np.sin(ang)], axis=1)
    abar = np.array([2.0, 1.0, 1.0, 1.0])
    p2 = O.GmcParams(max_head_clusters=2)
    omega, centres, assign = O.head_weights(_gram_from_patterns(u), abar, p2)
    assert centres == [1, 3]
    assert assign.tolist() == [0, 0, 0, 1]
    assert omega[3] == pytest.approx(0.5, rel=1e-14)
    assert omega[:3].sum() == pytest.approx(0.5, rel=1e-14)
    # head 1 sits nearest the cluster mean, so it gets the largest share
    assert np.argmax(omega[:3]) == 1

"""Pins of the oracle's realisation audit (Prop. 2 Eq. message-bound; App. I
Eq. cond-message-decomposition, Eq. cond-softmax-bound, Eq.
cond-message-polar; App. G Eq. cond-message-error).  CPU only."""
import math

import numpy as np
import pytest

from oracle import gmc_oracle as O


def _case(seed, n=40, kc=9, t=5, hq=4, hkv=2, dh=8, nonvis=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((t, hq, dh)) * 1.5
    k = rng.standard_normal((n, hkv, dh))
    v = rng.standard_normal((n, hkv, dh))
    k_c = rng.standard_normal((kc, hkv, dh))
    v_c = rng.standard_normal((kc, hkv, dh))
    carrier_of = np.concatenate([np.arange(kc), rng.integers(0, kc, size=n - kc)])
    rng.shuffle(carrier_of)
    w = rng.uniform(0.1, 1.0, size=(hq, t))
    nv = rng.standard_normal((hq, t)) * 2 if nonvis else None
    return q, k, v, k_c, v_c, carrier_of, w, nv


@pytest.mark.parametrize("seed", range(6))
def test_exact_message_decomposition(seed):
    # y - y~ = sum_i a_gi (v_i - v~_pi(i)) + sum_j (M_gj - abar_gj) v~_j
    r = O.message_audit(*_case(seed))["rows"]
    np.testing.assert_allclose(r["y"] - r["yc"], r["term1"] + r["term2"], rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("seed", range(12))
def test_grouped_mass_within_the_softmax_contraction_bound(seed):
    # ||M_g - abar_g||_1 <= ||u^F_g - u^S_g||_inf (Eq. cond-softmax-bound),
    # with and without the nonvisual keys as singleton categories
    for nonvis in (True, False):
        r = O.message_audit(*_case(seed, nonvis=nonvis))["rows"]
        assert np.all(r["l1"] <= r["bound"] + 1e-12)
        assert np.all(r["l1"] > 0)


def test_bound_and_mass_vanish_when_compact_equals_grouped_full():
    # a compact logit equal to the grouped Full logit log sum_(i in C_j)
    # exp(s_i) of its cluster gives the same category softmax: zero l1 gap
    # and a zero bound (here one token per cluster, compact keys = keys)
    q, k, v, _, _, _, w, nv = _case(3)
    n = k.shape[0]
    r = O.message_audit(q, k, v, k, v, np.arange(n), w, nv)["rows"]
    assert np.allclose(r["bound"], 0.0, atol=1e-12)
    assert np.allclose(r["l1"], 0.0, atol=1e-13)


def test_polar_identity_and_weight_scale_invariance():
    q, k, v, k_c, v_c, carrier_of, w, nv = _case(7)
    a = O.message_audit(q, k, v, k_c, v_c, carrier_of, w, nv)
    e2 = (a["norm_diff"] / a["norm_y"]) ** 2
    assert e2 == pytest.approx(1 + a["alpha"] ** 2 - 2 * a["alpha"] * a["kappa"], rel=1e-12)
    assert e2 == pytest.approx((1 - a["alpha"]) ** 2 + 2 * a["alpha"] * (1 - a["kappa"]), rel=1e-12)
    b = O.message_audit(q, k, v, k_c, v_c, carrier_of, 7.0 * w, nv)
    for key in ("alpha", "kappa"):
        assert b[key] == pytest.approx(a[key], rel=1e-12)
    # e_M only up to its 1e-8 regulariser in the denominator
    assert b["e_m"] == pytest.approx(a["e_m"], rel=1e-7)
    # all weight on one client: e_M is that client's relative message error
    w1 = np.zeros_like(w)
    w1[2, 3] = 1.0
    c = O.message_audit(q, k, v, k_c, v_c, carrier_of, w1, nv)
    y, yc = a["rows"]["y"][2, 3], a["rows"]["yc"][2, 3]
    assert c["e_m"] == pytest.approx(np.linalg.norm(y - yc) / (np.linalg.norm(y) + 1e-8), rel=1e-12)


def test_identity_compaction_has_no_message_error():
    # K = N with every token its own carrier and unchanged keys and values
    q, k, v, _, _, _, w, nv = _case(11)
    n = k.shape[0]
    a = O.message_audit(q, k, v, k, v, np.arange(n), w, nv)
    assert a["e_m"] == pytest.approx(0.0, abs=1e-14)
    assert a["alpha"] == pytest.approx(1.0, rel=1e-14) and a["kappa"] == pytest.approx(1.0, rel=1e-14)
    assert np.allclose(a["rows"]["term1"], 0.0) and np.allclose(a["rows"]["term2"], 0.0)


def test_messages_against_explicit_sums():
    # brute force on one client: y = sum_i a_i v_i with a the visual slice of
    # the softmax over visual logits and the nonvisual log-sum-exp
    q, k, v, k_c, v_c, carrier_of, w, nv = _case(13, n=7, kc=3, t=2, hq=2, hkv=1, dh=4)
    r = O.message_audit(q, k, v, k_c, v_c, carrier_of, w, nv)["rows"]
    h, t = 1, 0
    s = [float(np.dot(q[t, h], k[i, 0])) / 2.0 for i in range(7)]
    den = sum(math.exp(x) for x in s) + math.exp(nv[h, t])
    y = sum(math.exp(s[i]) / den * v[i, 0] for i in range(7))
    np.testing.assert_allclose(r["y"][h, t], y, rtol=1e-12)
    m = [sum(math.exp(s[i]) / den for i in range(7) if carrier_of[i] == j) for j in range(3)]
    sc = [float(np.dot(q[t, h], k_c[j, 0])) / 2.0 for j in range(3)]
    den_c = sum(math.exp(x) for x in sc) + math.exp(nv[h, t])
    ac = [math.exp(x) / den_c for x in sc]
    assert r["l1"][h, t] == pytest.approx(sum(abs(m[j] - ac[j]) for j in range(3)), rel=1e-12)
    uf = [math.log(sum(math.exp(s[i]) for i in range(7) if carrier_of[i] == j)) for j in range(3)]
    assert r["bound"][h, t] == pytest.approx(max(abs(uf[j] - sc[j]) for j in range(3)), rel=1e-12)


def test_client_weights_enter_the_stack_as_square_roots():
    # splitting a client into two identical ones that share its weight leaves
    # the stacked norms unchanged, which holds only when the stacked rows are
    # sqrt(w_g) y_g (so ||Y||^2 = sum_g w_g ||y_g||^2)
    q, k, v, k_c, v_c, carrier_of, w, nv = _case(17)
    a = O.message_audit(q, k, v, k_c, v_c, carrier_of, w, nv)
    q2 = np.concatenate([q, q[:1]], axis=0)
    w2 = np.concatenate([w, w[:, :1] / 2], axis=1)
    w2[:, 0] /= 2
    nv2 = np.concatenate([nv, nv[:, :1]], axis=1)
    b = O.message_audit(q2, k, v, k_c, v_c, carrier_of, w2, nv2)
    for key in ("norm_y", "norm_yc", "norm_diff", "alpha", "kappa"):
        assert b[key] == pytest.approx(a[key], rel=1e-12), key


def test_query_heads_read_their_kv_group():
    # head h reads kv head floor(h Hkv / Hq): with kv head 1's values zeroed,
    # heads 2 and 3 (of 4, 2 kv heads) carry no message, heads 0 and 1 do
    q, k, v, k_c, v_c, carrier_of, w, nv = _case(19)
    v = v.copy()
    v[:, 1, :] = 0.0
    r = O.message_audit(q, k, v, k_c, v_c, carrier_of, w, nv)["rows"]
    assert np.all(r["y"][2:] == 0.0)
    assert np.all(np.linalg.norm(r["y"][:2], axis=2) > 0)

"""Follow-mode parity checker: HIP outputs and traces vs the fp64 oracle.

The batched responsibility solver is a sequential heuristic; one near-tie
decided differently by fp32 rounding changes every later round.  So the
checker walks the oracle along the GPU's recorded decisions:

  * each round, the GPU pool must be a valid top-p set of the oracle's gains
    over the unselected tokens: no excluded token beats an included one by
    more than REL_TIE x the largest gain, and among exactly equal gains the
    lower source index wins.  Where the oracle's own cut has a margin above
    the tolerance this forces the identical pool.  The same rule applies to
    the batch chosen from the pool by the oracle's responsibility scores on
    that pool.  The oracle then continues from the GPU's choice.
  * every discarded token's representative must be a valid argmax of the
    oracle's kappa for the followed support (absolute tolerance KAPPA_TOL);
    selected tokens represent themselves.
  * out_idx must equal the followed support exactly; out_pos = pos3d[out_idx]
    exactly; out_hidden within the relative L2 bound of the dtype of the
    oracle's transport on the GPU's assignment.

Test infrastructure only.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from oracle import gmc_oracle as O

REL_TIE = 1e-3       # candidate-margin tolerance (relative to the top score)
KAPPA_TOL = 1e-3     # assignment tolerance (kappa is on the cosine scale)
REL_L2 = {"f32": 1e-4, "bf16": 2e-2}
CLIENT_TOL = 1e-4    # relative L2 of the pre-weighted client matrix per bank
# Element bounds.  Client entries: fp32 logits and cosines from bf16 products
# over d = 3584 carry absolute errors of a few 1e-6 (random-walk sum of
# 2^-24-sized roundings), which exp(. / tau) with tau = 0.2 turns into relative
# errors near 1e-5 of an entry; bounded by CLIENT_ELEM x the row's largest
# entry.  Gains: sums of such entries over M rows, bounded by GAIN_ELEM x the
# round's largest gain.  Output rows: the fp32 transport is exact to ~1e-6,
# so each row is within ROW_REL_L2 of the oracle (one bf16 rounding,
# 2^-9 / sqrt 3 RMS, under 4e-3) and every bf16 element within one ulp of the
# correctly rounded oracle value, up to ELEM_ABS x the row's largest entry
# for entries that a centroid's cancellation leaves small.
CLIENT_ELEM = 1e-4
GAIN_ELEM = 1e-4
ROW_REL_L2 = {"f32": 1e-4, "bf16": 4e-3}
ELEM_ABS = 1e-5
# Certificate: U_t relative, the round's coverage gain relative to F(S)
CERT_U_REL = 1e-4
CERT_GAIN_ABS = 1e-5


@dataclasses.dataclass
class FollowReport:
    rounds: int = 0
    pool_near_ties: int = 0
    batch_near_ties: int = 0
    assign_near_ties: int = 0
    min_pool_margin: float = np.inf
    min_batch_margin: float = np.inf
    client_rel_l2: Optional[dict] = None
    client_elem_max: float = 0.0     # max |delta| / row max over the client matrix
    gain_elem_max: float = 0.0       # max |delta| / round max over the per-round gains
    out_rel_l2: float = 0.0
    row_rel_l2_max: float = 0.0
    bf16_ulp_frac: float = 1.0
    cert_u_rel_max: float = 0.0
    cert_gain_abs_max: float = 0.0   # relative to F(S)
    cert_c_b: Optional[tuple] = None  # (gpu, oracle)
    identical_to_free_oracle: bool = True
    rounds_log: Optional[list] = None


def _valid_top(score: np.ndarray, cand: np.ndarray, chosen: np.ndarray, count: int, what: str):
    """Assert `chosen` is a valid top-`count` subset of `cand` under `score`
    (indexed by source token).  Returns the number of swaps versus the
    oracle's own (score desc, index asc) choice."""
    chosen = np.asarray(chosen, dtype=np.int64)
    assert chosen.size == count, f"{what}: size {chosen.size} != {count}"
    assert np.unique(chosen).size == count, f"{what}: duplicate entries"
    cset = set(cand.tolist())
    assert all(int(c) in cset for c in chosen), f"{what}: entry outside the candidates"
    inside = np.zeros(score.shape[0], dtype=bool)
    inside[chosen] = True
    out = cand[~inside[cand]]
    top = float(score[cand].max()) if cand.size else 0.0
    tol = REL_TIE * top
    if out.size:
        worst_in = float(score[chosen].min())
        best_out = float(score[out].max())
        assert worst_in >= best_out - tol, (
            f"{what}: excluded score {best_out:.9g} beats included {worst_in:.9g} by more than {tol:.3g}")
        # exact ties (exact zeros included) resolve to the lower source index
        for v in np.intersect1d(score[chosen], score[out]):
            ins = chosen[score[chosen] == v]
            outs = out[score[out] == v]
            assert ins.max() < outs.min(), f"{what}: equal scores {v} not resolved by lower index"
    own = O.top_by_score(score[cand], cand, count)
    return int(count - np.intersect1d(own, chosen).size)


def follow_selection(cbar: np.ndarray, k: int, b: int, pools, batches, p: O.GmcParams,
                     rep: FollowReport, gains=None, scores=None, seeds=()):
    """Walk the oracle along the GPU's per-round pools and batches.  With the
    GPU's per-round gains and pool scores, compare them element by element.
    Records the oracle's certificate terms of every followed round."""
    m, n = cbar.shape
    cov = np.zeros(m)
    chosen = np.zeros(n, dtype=bool)
    for j in seeds:                      # S_0 of a multi-image prompt
        chosen[j] = True
        cov = np.maximum(cov, cbar[:, j])
    n_sel = len(seeds)
    rounds = -(-(k - n_sel) // b)
    rep.rounds_log = []
    for r in range(rounds):
        cand = np.flatnonzero(~chosen)
        u = O.marginal_gains(cbar, cov)
        psize = min(p.pool_mult * b, cand.size)
        gp = np.asarray([x for x in pools[r] if x >= 0], dtype=np.int64)
        srt = np.sort(u[cand])[::-1]
        if gains is not None:
            g = np.asarray(gains[r], np.float64)
            top = float(u[cand].max()) if cand.size else 0.0
            err = float(np.max(np.abs(g[cand] - u[cand]))) if cand.size else 0.0
            rel = err / top if top > 0 else err
            rep.gain_elem_max = max(rep.gain_elem_max, rel)
            assert rel <= GAIN_ELEM, f"round {r} gains: max |delta| {err:.3e} vs top gain {top:.3e}"
            assert np.all(g[chosen] == 0.0), f"round {r}: selected tokens must carry gain 0"
        rep.min_pool_margin = min(rep.min_pool_margin, O._cut_margin(srt, psize))
        rep.pool_near_ties += _valid_top(u, cand, gp, psize, f"round {r} pool")
        gp = np.sort(gp)
        s = O.responsibility_scores(cbar, cov, gp, p)
        s_full = np.zeros(n)
        s_full[gp] = s
        bsize = min(b, k - n_sel)
        gb = np.asarray([x for x in batches[r] if x >= 0], dtype=np.int64)
        if scores is not None:
            sg = np.asarray(scores[r], np.float64)[:gp.size]
            top = float(s.max()) if s.size else 0.0
            err = float(np.max(np.abs(sg - s))) if s.size else 0.0
            assert err <= GAIN_ELEM * max(top, 1e-30), f"round {r} scores: max |delta| {err:.3e} vs top {top:.3e}"
        bmargin = O._cut_margin(np.sort(s)[::-1], bsize)
        rep.min_batch_margin = min(rep.min_batch_margin, bmargin)
        rep.batch_near_ties += _valid_top(s_full, gp, gb, bsize, f"round {r} batch")
        new_cov = np.maximum(cov, cbar[:, gb].max(axis=1))
        u_top = float(srt[:k].sum())
        gain = float(new_cov.sum() - cov.sum())
        rep.rounds_log.append(dict(u_top=u_top, gain=gain, q=gain / u_top if u_top > 0 else 0.0,
                                   pool_margin=O._cut_margin(srt, psize), batch_margin=bmargin))
        chosen[gb] = True
        n_sel += bsize
        cov = new_cov
    rep.rounds = rounds
    return np.flatnonzero(chosen), cov


def check_certificate(diag: dict, rep: FollowReport, f_s: float):
    """The GPU's in-call certificate (gmc_get_diag) against the oracle's terms
    of the followed rounds: U_t, the coverage gain, q_t, c_B and the margins."""
    log = rep.rounds_log
    assert diag["has_certificate"] == 1, "no certificate computed"
    assert len(diag["q"]) == len(log)
    for r, o in enumerate(log):
        u_rel = abs(diag["u_top"][r] - o["u_top"]) / max(o["u_top"], 1e-30)
        g_abs = abs(diag["gain"][r] - o["gain"]) / max(f_s, 1e-30)
        rep.cert_u_rel_max = max(rep.cert_u_rel_max, u_rel)
        rep.cert_gain_abs_max = max(rep.cert_gain_abs_max, g_abs)
        assert u_rel <= CERT_U_REL, f"round {r}: U_t {diag['u_top'][r]} vs {o['u_top']}"
        assert g_abs <= CERT_GAIN_ABS, f"round {r}: gain {diag['gain'][r]} vs {o['gain']}"
        qtol = o["q"] * CERT_U_REL + CERT_GAIN_ABS * f_s / max(o["u_top"], 1e-30) + 1e-7
        assert abs(diag["q"][r] - o["q"]) <= qtol, f"round {r}: q {diag['q'][r]} vs {o['q']}"
        for key in ("pool_margin", "batch_margin"):
            g, w = diag[key][r], o[key]
            if np.isinf(w):
                assert np.isinf(g), f"round {r} {key}: {g} vs inf"
            else:
                assert abs(g - w) <= 3 * GAIN_ELEM, f"round {r} {key}: {g} vs {w}"
    c_b = 1.0 - float(np.prod([1.0 - o["q"] for o in log]))
    rep.cert_c_b = (diag["c_b"], c_b)
    assert abs(diag["c_b"] - c_b) <= 1e-4 * max(c_b, 1e-6) + 1e-6, f"c_B {diag['c_b']} vs {c_b}"


def follow_assignment(x, pc, support, gpu_pi, p: O.GmcParams, rep: FollowReport, img=None):
    a = O.assign_population(x, pc, support, p, img)
    kappa = a["kappa"]                       # [N][K], columns in ascending support order
    sup = a["support"]
    slot = {int(j): jj for jj, j in enumerate(sup)}
    n = x.shape[0]
    gpu_pi = np.asarray(gpu_pi, dtype=np.int64)
    assert np.all(gpu_pi[sup] == sup), "selected tokens must represent themselves"
    disc = np.setdiff1d(np.arange(n), sup)
    for i in disc:
        j = int(gpu_pi[i])
        assert j in slot, f"token {i} assigned to non-support token {j}"
        best = kappa[i].max()
        got = kappa[i, slot[j]]
        assert got >= best - KAPPA_TOL, f"token {i}: kappa {got:.6f} vs best {best:.6f}"
        if j != int(a["pi"][i]):
            rep.assign_near_ties += 1
    return a


def bf16_round(a: np.ndarray) -> np.ndarray:
    from paper_2608_02134_amd.synth import round_bf16
    return round_bf16(np.asarray(a, dtype=np.float32))


def check_seeds(cbar: np.ndarray, img: np.ndarray, gpu_seeds: np.ndarray) -> np.ndarray:
    """The GPU's image seeds must be valid per-image argmaxes of the oracle's
    singleton gains F({i}) (near ties within REL_TIE of the largest gain, exact
    ties to the lower index).  Returns them in image order."""
    u = cbar.sum(axis=0)
    tol = REL_TIE * float(u.max())
    out = []
    for g in range(int(img.max()) + 1):
        members = np.flatnonzero(img == g)
        mine = [int(j) for j in gpu_seeds if img[j] == g]
        assert len(mine) == 1, f"image {g}: {len(mine)} seeds"
        j = mine[0]
        best = float(u[members].max())
        assert u[j] >= best - tol, f"image {g}: seed {j} gain {u[j]} vs best {best}"
        ties = members[u[members] == u[j]]
        assert j == ties.min(), f"image {g}: equal gains not resolved by lower index"
        out.append(j)
    return np.asarray(out, dtype=np.int64)


def check_problem(h, q, k, pos, probe, k_req, gpu: dict, dtype: str, p: O.GmcParams = O.GmcParams(),
                  app_proj=None, nonvis=None, probe_bias=None, hist=(), img=None) -> FollowReport:
    """Full follow-mode check of one problem.  `gpu` holds numpy arrays:
    out_hidden, out_pos, out_idx and, from the trace, round_pool, round_batch,
    assign, and optionally client, omega, ebar, stats."""
    rep = FollowReport()
    h = np.asarray(h, np.float64)
    n = h.shape[0]
    n_img = 1 if img is None else int(np.max(img)) + 1
    if n_img == 1:
        img = None
    kk = O.realized_budget(n, k_req, n_img)
    assert gpu["out_idx"].shape == (kk,)
    if kk == n:
        assert np.array_equal(gpu["out_idx"], np.arange(n))
        assert np.array_equal(gpu["out_pos"], pos)
        assert np.array_equal(np.asarray(gpu["out_hidden"], np.float64), h)
        return rep
    cl = O.build_clients(h, q, k, pos, probe, p, app_proj, nonvis, probe_bias, hist, img)
    cbar = cl["cbar"]
    if gpu.get("client") is not None:
        rel = {}
        for bank in (0, 1, 2):
            rows = cl["banks"] == bank
            if not rows.any():
                continue
            ref = cbar[rows]
            got = np.asarray(gpu["client"], np.float64)[rows]
            rel[bank] = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
            assert rel[bank] < CLIENT_TOL, f"client bank {bank} rel L2 {rel[bank]:.3e}"
            rmax = np.max(np.abs(ref), axis=1, keepdims=True)
            act = rmax[:, 0] > 0
            elem = np.abs(got - ref)[act] / rmax[act]
            worst = float(elem.max()) if elem.size else 0.0
            rep.client_elem_max = max(rep.client_elem_max, worst)
            assert worst <= CLIENT_ELEM, f"client bank {bank}: an entry off by {worst:.3e} of its row max"
            assert np.all(got[~act] == 0.0), f"client bank {bank}: an inactive row is not zero"
        rep.client_rel_l2 = rel
    if gpu.get("omega") is not None and q.shape[0] > 0:
        np.testing.assert_allclose(gpu["omega"], cl["omega"], atol=1e-4, err_msg="head weights")
    if gpu.get("ebar") is not None:
        eb = cl["ebar"]
        assert np.linalg.norm(gpu["ebar"] - eb) / np.linalg.norm(eb) < 1e-4, "normalised energy"
    b = p.batch_b_bounded if cl["bounded"] else p.batch_b
    seeds = ()
    if img is not None:
        in_rounds = set(int(x) for x in np.asarray(gpu["round_batch"]).ravel() if x >= 0)
        gpu_seeds = np.asarray([j for j in gpu["out_idx"] if int(j) not in in_rounds], dtype=np.int64)
        seeds = check_seeds(cbar, img, gpu_seeds)
    support, cov = follow_selection(cbar, kk, b, gpu["round_pool"], gpu["round_batch"], p, rep,
                                    gpu.get("round_gains"), gpu.get("round_scores"), seeds)
    assert np.array_equal(np.asarray(gpu["out_idx"], np.int64), support), "out_idx != followed support"
    assert np.array_equal(gpu["out_pos"], pos[support]), "out_pos != pos3d[out_idx]"
    a = follow_assignment(cl["x"], cl["pc"], support, gpu["assign"], p, rep, img)
    m = O.population_weights(cl["ebar"], a["sx"], p)
    tr = O.transport(h, np.asarray(gpu["assign"], np.int64), support, m, p)
    ref = tr["out"]
    got = np.asarray(gpu["out_hidden"], np.float64)
    rep.out_rel_l2 = float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
    assert rep.out_rel_l2 < REL_L2[dtype], f"out_hidden rel L2 {rep.out_rel_l2:.3e}"
    # every carrier row on its own
    row_rel = np.linalg.norm(got - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
    rep.row_rel_l2_max = float(row_rel.max())
    assert rep.row_rel_l2_max < ROW_REL_L2[dtype], (
        f"carrier row {int(np.argmax(row_rel))} rel L2 {rep.row_rel_l2_max:.3e}")
    if dtype == "bf16":
        # every element within one bf16 ulp of the correctly rounded oracle value
        want = bf16_round(ref).astype(np.float64)
        mag = np.maximum(np.abs(want), 1e-38)
        ulp = 2.0 ** (np.floor(np.log2(mag)) - 7)
        slack = ELEM_ABS * np.max(np.abs(ref), axis=1, keepdims=True)
        ok = np.abs(got - want) <= ulp + slack
        rep.bf16_ulp_frac = float(np.mean(np.abs(got - want) <= ulp))
        bad = np.argwhere(~ok)
        assert bad.size == 0, (f"{bad.shape[0]} bf16 outputs beyond one ulp, first at {tuple(bad[0])}: "
                               f"{got[tuple(bad[0])]} vs {want[tuple(bad[0])]}")
    if gpu.get("stats") is not None:
        st = gpu["stats"]
        assert st[8] == 0, f"device status word {st[8]} (grid barrier timeout)"
        assert abs(st[0] - a["sx"]) < 1e-4 + 1e-3 * a["sx"], f"s_x {st[0]} vs {a['sx']}"
        fs = float(cov.sum())
        assert abs(st[2] - fs) <= 1e-4 * fs, f"F(S) {st[2]} vs {fs}"
        fv = float(cbar.max(axis=1).sum())
        assert abs(st[3] - fv) <= 1e-4 * fv, f"F(V) {st[3]} vs {fv}"
        # per-bank objectives (grounded, appearance, spatial): omega_b and
        # the saturation c_b of the bank mixture follow from them
        for bank in (0, 1, 2):
            rows = cl["banks"] == bank
            fsb = float(cov[rows].sum()) if rows.any() else 0.0
            fvb = float(cbar[rows].max(axis=1).sum()) if rows.any() else 0.0
            assert abs(st[9 + bank] - fsb) <= 1e-4 * fs, f"F_{bank}(S) {st[9 + bank]} vs {fsb}"
            assert abs(st[12 + bank] - fvb) <= 1e-4 * fv, f"F_{bank}(V) {st[12 + bank]} vs {fvb}"
    if gpu.get("diag") is not None:
        check_certificate(gpu["diag"], rep, float(cov.sum()))
    free = O.select_support(cbar, kk, b, p, O.image_seeds(cbar, img) if img is not None else ())
    rep.identical_to_free_oracle = bool(np.array_equal(np.sort(free["order"]), support))
    if rep.pool_near_ties == 0 and rep.batch_near_ties == 0:
        assert rep.identical_to_free_oracle
    return rep

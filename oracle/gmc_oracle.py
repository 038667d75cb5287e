"""Plain fp64 CPU oracle of the GMC boundary operator.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the
HIP library and its Python binding) never calls it, and it shares no code,
table or helper with that path.

It follows the paper ("Messages, Not Tokens: Grounded Coresets for Faithful
VLM Compression") step by step, in its notation, in float64:

  budget          Sec. 3.1 problem formulation; App. H "Batched complementary
                  support" (totality rule)
  message         Sec. 3.2; App. H Eq. cond-native-message,
                  Eq. cond-mass-coordinate, Eq. cond-grounded-client
  head weights    App. H Eq. cond-head-pattern, Eq. cond-head-weight
  banks           Sec. 3.2; App. H Eq. cond-aux-clients, Eq. cond-coverage,
                  Eq. cond-effective-bank-mass
  selection       Sec. 3.3 Eq. coverage, Eq. responsibility;
                  App. H Eq. cond-responsibility
  certificates    Prop. 1 Eq. deployed-approximation; App. I
                  Eq. cond-final-cert, Eq. cond-bank-mixture
  assignment      Sec. 3.4; App. H Eq. cond-assignment,
                  Eq. cond-population-gate
  transport       Sec. 3.4 Eq. transport; App. H Eq. cond-transport,
                  Eq. cond-grounded-energy
  compaction      App. H "Index map and physical token accounting"
  audit           Prop. 2 Eq. message-bound; App. I Eq. cond-message-
                  decomposition, Eq. cond-softmax-bound, Eq. cond-message-
                  polar; App. G Eq. cond-message-error

Readings where the paper is silent are listed in ``READINGS`` and in the
design notes; each is a named constant below.  Pins against the paper's
identities, bounds, special cases and brute force live in tests/.

Parity status: every function here is pinned by at least one test except the
exact index choices of the batched responsibility heuristic on generic data,
which the paper fixes only through its rules (no printed toy instance):
for those, "parity unpinned" beyond the brute-force bounds, the b=1 greedy
special case and the zero-gain fill order.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

__all__ = [
    "GmcParams", "READINGS", "realized_budget", "row_features", "value_probe",
    "mass_coordinate", "native_attention", "grounded_energy_rows",
    "query_weights", "head_pattern_gram", "head_weights", "grounded_energy",
    "appearance_bank", "appearance_bank_bounded", "spatial_coordinates",
    "spatial_bank", "client_matrix", "coverage", "marginal_gains",
    "responsibility_scores", "top_by_score", "select_support",
    "assignment_gaps", "separability_gate", "ambiguity_gate",
    "assign_population", "population_weights", "transport", "compact",
    "gmc_single", "gmc", "prune_rounds", "index_map", "compact_sequence",
    "gather_cache", "head_pattern", "head_weights_from_pattern", "view_mass",
    "message_view", "image_seeds", "message_audit",
]


@dataclasses.dataclass(frozen=True)
class GmcParams:
    """Frozen settings (App. H, Table cond-config) plus the readings below."""
    probe_rank: int = 4
    lambda_mass: float = 1.0
    eps_mass: float = 1e-8
    beta_msg: float = 1.0          # reading R1
    beta_app: float = 0.5
    beta_spa: float = 0.25
    tau_v: float = 0.2
    tau_s: float = 0.02
    landmarks: int = 16
    batch_b: int = 16
    pool_mult: int = 4
    tau_r: float = 0.1
    resp_eps: float = 1e-30        # reading R9
    spatial_w: float = 0.5
    gate_t: float = 0.08
    gate_p: float = 8.0
    amb_margin: float = 0.05       # reading R5
    amb_p: float = 8.0             # reading R5
    g_form: str = "smooth"         # reading R5 ("smooth" | "hard")
    pop_strength: float = 0.5
    tau_j: float = 1.0             # reading R10
    max_head_clusters: int = 4
    disp_eps: float = 0.05
    terminal_q_weight: float = 2.0
    rms_eps: float = 1e-6          # reading R4
    norm_eps: float = 1e-12        # reading R9
    restore_eps: float = 1e-6      # reading R9
    bounded_threshold_n: int = 4096  # reading R8
    app_rank: int = 128
    app_max_clients: int = 4096
    batch_b_bounded: int = 512
    hist_mass: float = 0.5         # reading R14


READINGS = {
    "R1": "grounded (message) bank mass beta_msg = 1: current+history masses "
          "0.5+0.5; with no history view supplied the current view carries both",
    "R2": "grounded row (h,t) weight = beta_msg * omega_h * nu_t * a_(h,t); "
          "reduces to beta/M * a_m for uniform omega and nu; nu_t is not used in "
          "head patterns",
    "R3": "native nonvisual softmax denominator enters as an optional per-(h,t) "
          "log-sum-exp; P^G is invariant to it",
    "R4": "value path folded into a per-head probe G_h [r][d]; x~ = RMSNorm(h) "
          "with eps 1e-6 and unit gain; an optional value bias folds into "
          "b_h = b^V O_h P added to Z_h[i]",
    "R5": "local ambiguity g_i = exp(-(delta_i/0.05)^8) (hard variant: "
          "1[delta_i < 0.05])",
    "R6": "spatial coordinates are grid-cell centres in [0,1]^2 from (h,w); "
          "the temporal id is not a spatial coordinate but is kept in out_pos",
    "R7": "one image per problem (I = 1); frames of one clip are one image",
    "R8": "bounded appearance bank iff N > 4096, with b = 512",
    "R9": "epsilons: responsibility 1e-30, normalisation 1e-12, RMS restore 1e-6",
    "R10": "transport blend tau_j = 1 (appendix form R_j(c_j))",
    "R11": "pool = top-min(4b, N-|S|) unselected tokens; last batch K-|S|",
    "R12": "farthest-first picks min(4, active heads) centres; ties to the "
           "earliest centre; empty clusters are dropped",
    "R13": "ties in every ranking go to the lower source index",
    "R15": "multi-image prompts: image ids per token; K = min(N, max(K_r, I)); "
           "S_0 = one largest-singleton-gain token per image (ties to the lower "
           "index); every image has its own 16 x 16 landmarks on its own grid "
           "(M_S = 256 I) and its appearance clients cover its own tokens; "
           "assignment and the gap delta use the image's carriers; the exact "
           "appearance bank only (N <= 4096)",
    "R14": "historical views: the message mass beta_msg splits into the current "
           "view's (1 - hist_mass) beta_msg and hist_mass beta_msg shared equally "
           "by the historical views (0.5 / 0.5 with two views: 0.5, 0.25, 0.25); "
           "each view has its own states, queries, keys and folded value probe; "
           "with no historical view the current view carries beta_msg",
}


# ----------------------------------------------------------------------------
# Budget (Sec. 3.1 problem formulation; App. H totality rule)
# ----------------------------------------------------------------------------
def realized_budget(n: int, k_req: int, n_images: int = 1) -> int:
    """K = min{N, max{K_r, I}}."""
    return int(min(n, max(k_req, n_images)))


# ----------------------------------------------------------------------------
# Boundary features
# ----------------------------------------------------------------------------
def row_features(h: np.ndarray, p: GmcParams):
    """Norms, unit directions x_i = h_i/max(||h_i||, eps) (App. H assignment),
    RMS values, and the next block's RMSNorm x~_i (unit gain, reading R4)."""
    h = np.asarray(h, dtype=np.float64)
    norm = np.sqrt(np.sum(h * h, axis=1))
    x = h / np.maximum(norm, p.norm_eps)[:, None]
    ms = np.mean(h * h, axis=1)
    rms = np.sqrt(ms)
    xt = h / np.sqrt(ms + p.rms_eps)[:, None]
    return norm, x, rms, xt


def value_probe(xt: np.ndarray, probe: np.ndarray, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Z_h = (V_h O_h) P as one folded per-head map: Z[h][i][c] = x~_i . G[h][c]
    (+ b[h][c] = (b^V O_h P)[c] when the value projection has a bias b^V)."""
    z = np.einsum("nd,hrd->hnr", xt, np.asarray(probe, np.float64))
    if bias is not None:
        z = z + np.asarray(bias, np.float64)[:, None, :]
    return z


def mass_coordinate(z: np.ndarray, p: GmcParams) -> np.ndarray:
    """sigma_h = sqrt(lambda_mass) max{||Z_h||_F / sqrt(N r), eps_mass}
    (Eq. mass-coordinate / cond-mass-coordinate)."""
    hq, n, r = z.shape
    fro = np.sqrt(np.sum(z * z, axis=(1, 2)))
    return math.sqrt(p.lambda_mass) * np.maximum(fro / math.sqrt(n * r), p.eps_mass)


def native_attention(q: np.ndarray, k: np.ndarray, nonvis_lse: Optional[np.ndarray] = None):
    """Visual-column slice of the native softmax (Eq. cond-native-message).

    q [T][Hq][dh], k [N][Hkv][dh]; head h reads kv head floor(h*Hkv/Hq).
    The denominator combines the visual logits with an optional nonvisual
    log-sum-exp per (h,t) (reading R3).  Returns A [Hq][T][N].
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    t, hq, dh = q.shape
    n, hkv, _ = k.shape
    a = np.empty((hq, t, n))
    for h in range(hq):
        g = (h * hkv) // hq
        s = q[:, h, :] @ k[:, g, :].T / math.sqrt(dh)          # [T][N]
        mx = s.max(axis=1, keepdims=True)
        lse = mx[:, 0] + np.log(np.sum(np.exp(s - mx), axis=1))
        if nonvis_lse is not None:
            lse = np.logaddexp(lse, np.asarray(nonvis_lse, np.float64)[h])
        a[h] = np.exp(s - lse[:, None])
    return a


def grounded_energy_rows(a: np.ndarray, z: np.ndarray, sigma: np.ndarray):
    """Atom norms e_(h,t,i) = ||u_i^(h,t)|| with u = A[t,i][Z_h[i]; sigma_h]
    (Eq. grounded-client).  Returns e [Hq][T][N] and l [Hq][N] = ||w_h[i]||."""
    ell = np.sqrt(np.sum(z * z, axis=2) + sigma[:, None] ** 2)   # [Hq][N]
    e = a * ell[:, None, :]
    return e, ell


def query_weights(t: int, p: GmcParams) -> np.ndarray:
    """nu_t: the terminal prompt query counts terminal_q_weight times the
    others; normalised to sum one (App. H native message clients)."""
    if t == 0:
        return np.zeros(0)
    w = np.ones(t)
    w[-1] = p.terminal_q_weight
    return w / w.sum()


def head_pattern_gram(a: np.ndarray, z: np.ndarray, sigma: np.ndarray) -> np.ndarray:
    """Gamma_hg = <vec U_h, vec U_g> = sum_(t,i) A_h A_g <w_h[i], w_g[i]>,
    the Gram of the flattened per-head atoms (Eq. cond-head-pattern)."""
    hq, t, n = a.shape
    w = np.concatenate([z, np.broadcast_to(sigma[:, None, None], (hq, n, 1))], axis=2)
    # the (t, i, c) sum grouped as sum_i <w_h[i], w_g[i]> * sum_t A_h[t,i] A_g[t,i]
    aa = np.einsum("hti,gti->hgi", a, a)                          # [Hq][Hq][N]
    ww = np.einsum("hic,gic->hgi", w, w)                          # [Hq][Hq][N]
    return np.sum(aa * ww, axis=2)


def head_pattern(grams, mean_atom_norms, view_mass) -> np.ndarray:
    """Gram of the pre-normalisation head patterns concat_v[sqrt(beta_v)
    vec(U_h^v)] with U_h^v the view's atoms scaled to unit average atom norm
    (Eq. cond-head-pattern): sum_v beta_v Gamma^v_hg / (abar^v_h abar^v_g); a
    view in which a head has no energy (abar = 0) adds nothing for it."""
    hq = grams[0].shape[0]
    out = np.zeros((hq, hq))
    for gram, abar, beta in zip(grams, mean_atom_norms, view_mass):
        inv = np.where(abar > 0, 1.0 / np.where(abar > 0, abar, 1.0), 0.0)
        out += beta * gram * inv[:, None] * inv[None, :]
    return out


def head_weights(gram: np.ndarray, mean_atom_norm: np.ndarray, p: GmcParams):
    """Farthest-first cosine head clustering and inverse-dispersion weights
    (Eq. cond-head-pattern, Eq. cond-head-weight; reading R12) for one
    message view of mass beta_msg.

    gram: Gamma [Hq][Hq]; mean_atom_norm: average atom norm per head, which
    sets the pre-normalisation pattern norm sqrt(beta Gamma_hh)/abar_h.
    Returns (omega [Hq], centres list, cluster id per head (-1 inactive)).
    """
    return head_weights_from_pattern(head_pattern([gram], [mean_atom_norm], [p.beta_msg]), p)


def head_weights_from_pattern(pattern: np.ndarray, p: GmcParams):
    """Farthest-first clustering on the Gram of the pre-normalisation head
    patterns (head_pattern): the first centre has the largest pattern norm,
    each next one the smallest maximum cosine to the centres chosen; heads
    join their nearest centre (ties to the earlier one); omega by Eq.
    cond-head-weight over the non-empty clusters."""
    hq = pattern.shape[0]
    diag = np.diag(pattern).copy()
    active = diag > 0
    omega = np.zeros(hq)
    assign = -np.ones(hq, dtype=np.int64)
    n_active = int(active.sum())
    if n_active == 0:
        return omega, [], assign
    nrm = np.sqrt(np.where(active, diag, 1.0))
    cos = pattern / nrm[:, None] / nrm[None, :]
    pre = np.where(active, np.sqrt(np.where(active, diag, 0.0)), -np.inf)
    centres = [int(np.argmax(pre))]
    n_c = min(p.max_head_clusters, n_active)
    while len(centres) < n_c:
        best, best_val = -1, np.inf
        for hh in range(hq):
            if not active[hh] or hh in centres:
                continue
            v = max(cos[hh, c] for c in centres)
            if v < best_val:
                best, best_val = hh, v
        centres.append(best)
    for hh in range(hq):
        if not active[hh]:
            continue
        sims = [cos[hh, c] for c in centres]
        assign[hh] = int(np.argmax(sims))          # first maximum: earliest centre
    clusters = [np.flatnonzero(assign == c) for c in range(len(centres))]
    clusters = [m for m in clusters if m.size > 0]
    n_clusters = len(clusters)
    for members in clusters:
        sub = cos[np.ix_(members, members)]
        mean_norm = math.sqrt(max(sub.sum(), 0.0))
        disp = 1.0 - sub.sum(axis=1) / mean_norm        # d_h = 1 - u_h . mu_c
        inv = 1.0 / (disp + p.disp_eps)
        omega[members] = inv / inv.sum() / n_clusters
    return omega, centres, assign


def grounded_energy(e: np.ndarray, omega: np.ndarray, nu: np.ndarray):
    """e_i = (sum_h omega_h ||r_i^(h,.)||^2)^(1/2), r = sqrt(nu_t) u, and
    ebar_i = e_i / mean_j e_j with the uniform fallback ebar = 1
    (Eq. cond-grounded-energy)."""
    hq, t, n = e.shape
    if t == 0:
        return np.ones(n), np.zeros(n)
    per_head = np.einsum("t,htn->hn", nu, e * e)
    en = np.sqrt(np.einsum("h,hn->n", omega, per_head))
    mean = en.mean()
    if not mean > 0:
        return np.ones(n), en
    return en / mean, en


# ----------------------------------------------------------------------------
# Auxiliary banks (Eq. cond-aux-clients)
# ----------------------------------------------------------------------------
def _row_softmax(logits: np.ndarray) -> np.ndarray:
    mx = logits.max(axis=1, keepdims=True)
    ex = np.exp(logits - mx)
    return ex / ex.sum(axis=1, keepdims=True)


def appearance_bank(x: np.ndarray, p: GmcParams, img: Optional[np.ndarray] = None) -> np.ndarray:
    """P^V_m(i) = softmax_i(x_m . x_i / tau_v), one client per token; with
    image ids, each client's distribution covers its own image's tokens
    (App. H: appearance and spatial rows are restricted to their image)."""
    logits = (x @ x.T) / p.tau_v
    if img is not None:
        logits = np.where(img[:, None] == img[None, :], logits, -np.inf)
    return _row_softmax(logits)


def appearance_bank_bounded(h: np.ndarray, proj: np.ndarray, p: GmcParams):
    """Long-prefix bank: states projected by the fixed +-1 matrix, normalised,
    and at most M_V uniformly spaced clients m_k = floor(k N / M_V)."""
    n = h.shape[0]
    y = np.asarray(h, np.float64) @ np.asarray(proj, np.float64).T
    y = y / np.maximum(np.sqrt(np.sum(y * y, axis=1)), p.norm_eps)[:, None]
    mv = min(p.app_max_clients, n)
    clients = (np.arange(mv) * n) // mv
    return _row_softmax((y[clients] @ y.T) / p.tau_v), clients


def spatial_coordinates(pos: np.ndarray, img: Optional[np.ndarray] = None) -> np.ndarray:
    """Original-grid (h, w) mapped to cell centres in [0,1]^2 (reading R6),
    over each image's own grid when image ids are given."""
    hh = pos[:, 1].astype(np.float64)
    ww = pos[:, 2].astype(np.float64)
    if img is None:
        img = np.zeros(pos.shape[0], dtype=np.int64)
    out = np.empty((pos.shape[0], 2))
    for g in np.unique(img):
        sel = img == g
        h0, w0 = hh[sel].min(), ww[sel].min()
        gh, gw = hh[sel].max() - h0 + 1.0, ww[sel].max() - w0 + 1.0
        out[sel, 0] = (hh[sel] - h0 + 0.5) / gh
        out[sel, 1] = (ww[sel] - w0 + 0.5) / gw
    return out


def spatial_bank(pos: np.ndarray, p: GmcParams, img: Optional[np.ndarray] = None) -> np.ndarray:
    """P^S_ab(i) = softmax_i(-||p_i - l_ab||^2 / tau_s) around the L x L
    landmarks l_ab = ((a+.5)/L, (b+.5)/L); row index a*L + b.  With image ids
    every image has its own L x L landmarks on its own grid, and each such
    row covers that image's tokens (Eq. cond-aux-clients: 1[I_i = I_m]);
    row index g L^2 + a L + b for image g."""
    pc = spatial_coordinates(pos, img)
    grid = (np.arange(p.landmarks) + 0.5) / p.landmarks
    la, lb = np.meshgrid(grid, grid, indexing="ij")
    land = np.stack([la.ravel(), lb.ravel()], axis=1)
    d2 = np.sum((land[:, None, :] - pc[None, :, :]) ** 2, axis=2)
    if img is None:
        return _row_softmax(-d2 / p.tau_s)
    rows = []
    for g in range(int(img.max()) + 1):
        rows.append(_row_softmax(np.where((img == g)[None, :], -d2 / p.tau_s, -np.inf)))
    return np.concatenate(rows, axis=0)


# ----------------------------------------------------------------------------
# Client matrix (Eq. cond-coverage) and coverage objective (Eq. coverage)
# ----------------------------------------------------------------------------
def client_matrix(pg: np.ndarray, active: np.ndarray, omega: np.ndarray, nu: np.ndarray,
                  pv: np.ndarray, ps: np.ndarray, p: GmcParams, hist_pg=(), hist_active=(), view_mass=None):
    """Stack the three banks into Cbar [M][N] with preweights.

    Grounded row (h,t) of message view v: beta_v omega_h nu_t a_(h,t) P^G
    (reading R2; beta_v = beta_msg with one view, reading R14 with historical
    views, whose rows follow the current view's, view by view);
    appearance row: beta_app / M_V P^V; spatial row: beta_spa / M_S P^S.
    Returns Cbar and the bank id of every row (0 grounded, 1 appearance,
    2 spatial).
    """
    hq, t, n = pg.shape
    rows, banks = [], []
    if t > 0:
        views = [(pg, active)] + list(zip(hist_pg, hist_active))
        mass = [p.beta_msg] if view_mass is None else view_mass
        for (pgv, actv), beta in zip(views, mass):
            wg = beta * omega[:, None] * nu[None, :] * actv
            rows.append((wg[:, :, None] * pgv).reshape(hq * t, n))
            banks.append(np.zeros(hq * t, dtype=np.int64))
    rows.append(p.beta_app / pv.shape[0] * pv)
    banks.append(np.ones(pv.shape[0], dtype=np.int64))
    rows.append(p.beta_spa / ps.shape[0] * ps)
    banks.append(np.full(ps.shape[0], 2, dtype=np.int64))
    return np.concatenate(rows, axis=0), np.concatenate(banks)


def coverage(cbar: np.ndarray, support) -> float:
    """F(S) = sum_m max_(i in S) Cbar_mi, F(empty) = 0."""
    s = np.asarray(list(support), dtype=np.int64)
    if s.size == 0:
        return 0.0
    return float(cbar[:, s].max(axis=1).sum())


def marginal_gains(cbar: np.ndarray, cov: np.ndarray) -> np.ndarray:
    """u_i = sum_m [Cbar_mi - b_m]_+ with b_m the current coverage maxima."""
    return np.maximum(cbar - cov[:, None], 0.0).sum(axis=0)


def responsibility_scores(cbar: np.ndarray, cov: np.ndarray, pool: np.ndarray,
                          p: GmcParams) -> np.ndarray:
    """s_i = sum_m rho_mi R_mi over the pool, with rho the pool softmax of
    R_mi / (tau_r max_(j in pool) R_mj + eps) (Eq. cond-responsibility)."""
    r = np.maximum(cbar[:, pool] - cov[:, None], 0.0)          # [M][|pool|]
    mu = r.max(axis=1, keepdims=True)
    rho = _row_softmax(r / (p.tau_r * mu + p.resp_eps))
    return np.sum(rho * r, axis=0)


def top_by_score(score: np.ndarray, cand: np.ndarray, count: int) -> np.ndarray:
    """The `count` candidates with the largest score; equal scores go to the
    lower source index (reading R13).  Returned in rank order."""
    cand = np.asarray(cand, dtype=np.int64)
    order = np.lexsort((cand, -score))
    return cand[order[:count]]


def _cut_margin(sorted_vals: np.ndarray, count: int) -> float:
    """Relative gap at a cut, (v_(count) - v_(count+1)) / v_(1); an exact
    zero-zero cut is resolved by index and counts as infinite."""
    if count >= sorted_vals.size or count == 0:
        return math.inf
    a, b = sorted_vals[count - 1], sorted_vals[count]
    if a == 0.0 and b == 0.0:
        return math.inf
    top = sorted_vals[0]
    return (a - b) / top if top > 0 else math.inf


def select_support(cbar: np.ndarray, k: int, b: int, p: GmcParams, seed_set=()):
    """Batched responsibility selection (Sec. 3.3; Eq. cond-responsibility).

    Rounds until |S| = K: residual gains over unselected tokens, a pool of the
    min(pool_mult*b, N-|S|) best gains, responsibility scores over the pool,
    the min(b, K-|S|) best scores enter together, then the coverage maxima are
    refreshed.  Zero-gain tokens then fill in source order automatically.

    Returns dict with the support in selection order, per-round pools and
    batches, the certificate factors q_t (Prop. 1) and the decision margins.
    """
    m, n = cbar.shape
    cov = np.zeros(m)
    chosen = np.zeros(n, dtype=bool)
    order = []
    for j in seed_set:
        chosen[j] = True
        order.append(int(j))
        cov = np.maximum(cov, cbar[:, j])
    f0 = float(cov.sum())
    rounds = []
    while len(order) < k:
        cand = np.flatnonzero(~chosen)
        u_all = marginal_gains(cbar, cov)
        u = u_all[cand]
        psize = min(p.pool_mult * b, cand.size)
        pool = top_by_score(u, cand, psize)
        u_sorted = np.sort(u)[::-1]
        s = responsibility_scores(cbar, cov, pool, p)
        bsize = min(b, k - len(order))
        batch = top_by_score(s, pool, bsize)
        s_sorted = np.sort(s)[::-1]
        # certificate factor q_t = [F(S u B) - F(S)] / U_t, U_t = K largest u
        u_top = float(u_sorted[:k].sum())
        new_cov = np.maximum(cov, cbar[:, batch].max(axis=1))
        gain = float(new_cov.sum() - cov.sum())
        q = gain / u_top if u_top > 0 else 0.0
        rounds.append(dict(pool=np.sort(pool), batch=batch, u=u_all.copy(),
                           s=dict(zip(pool.tolist(), s.tolist())), q=q, gain=gain,
                           u_top=u_top,
                           pool_margin=_cut_margin(u_sorted, psize),
                           batch_margin=_cut_margin(s_sorted, bsize)))
        chosen[batch] = True
        order.extend(int(j) for j in batch)
        cov = new_cov
    c_b = 1.0 - float(np.prod([1.0 - r["q"] for r in rounds])) if rounds else 0.0
    return dict(order=np.array(order, dtype=np.int64), rounds=rounds, cov=cov,
                f_s=float(cov.sum()), f0=f0, c_b=c_b)


# ----------------------------------------------------------------------------
# Population assignment (Sec. 3.4; Eq. cond-assignment, cond-population-gate)
# ----------------------------------------------------------------------------
def assignment_gaps(x: np.ndarray, support: np.ndarray, img: Optional[np.ndarray] = None):
    """cos_ij = x_i . x_j for j in S (-inf for j in another image: S_i holds
    the image-compatible carriers) and delta_i = best - second best
    compatible cosine (delta = 0 when S_i has one member)."""
    cos = x @ x[support].T                                      # [N][K]
    if img is not None:
        cos = np.where(img[:, None] == img[support][None, :], cos, -np.inf)
    if support.size < 2:
        return cos, np.zeros(x.shape[0])
    top2 = -np.sort(-cos, axis=1)[:, :2]
    delta = np.where(np.isfinite(top2[:, 1]), top2[:, 0] - top2[:, 1], 0.0)
    return cos, delta


def separability_gate(delta: np.ndarray, discarded: np.ndarray, p: GmcParams) -> float:
    """s_x = 1 - exp[-(mean_(i discarded) delta_i / t)^p]; mean 0 when none."""
    dbar = float(delta[discarded].mean()) if discarded.any() else 0.0
    return 1.0 - math.exp(-((dbar / p.gate_t) ** p.gate_p)), dbar


def ambiguity_gate(delta: np.ndarray, p: GmcParams) -> np.ndarray:
    """Local ambiguity g_i from the selected-cosine gap (reading R5)."""
    if p.g_form == "hard":
        return (delta < p.amb_margin).astype(np.float64)
    return np.exp(-((delta / p.amb_margin) ** p.amb_p))


def assign_population(x: np.ndarray, pc: np.ndarray, support: np.ndarray, p: GmcParams,
                      img: Optional[np.ndarray] = None):
    """pi(i) = argmax_(j in S_i) cos_ij + 0.5 s_x g_i exp(-||p_i - p_j||^2/tau_s)
    over the image-compatible carriers S_i; ties to the lower source index;
    selected tokens represent themselves."""
    n = x.shape[0]
    sup = np.sort(np.asarray(support, dtype=np.int64))
    cos, delta = assignment_gaps(x, sup, img)
    discarded = np.ones(n, dtype=bool)
    discarded[sup] = False
    sx, dbar = separability_gate(delta, discarded, p)
    g = ambiguity_gate(delta, p)
    d2 = np.sum((pc[:, None, :] - pc[sup][None, :, :]) ** 2, axis=2)
    kappa = cos + p.spatial_w * sx * g[:, None] * np.exp(-d2 / p.tau_s)
    pi = sup[np.argmax(kappa, axis=1)]                          # first max = lowest index
    pi[sup] = sup
    srt = -np.sort(-kappa, axis=1)
    with np.errstate(invalid="ignore"):
        kmargin = srt[:, 0] - srt[:, 1] if sup.size > 1 else np.full(n, np.inf)
    kmargin = np.where(np.isnan(kmargin), np.inf, kmargin)
    kmargin[sup] = np.inf
    return dict(pi=pi, sx=sx, dbar=dbar, delta=delta, g=g, kappa_margin=kmargin,
                cos=cos, kappa=kappa, support=sup)


# ----------------------------------------------------------------------------
# Transport (Sec. 3.4 Eq. transport; App. H Eq. cond-transport)
# ----------------------------------------------------------------------------
def population_weights(ebar: np.ndarray, sx: float, p: GmcParams) -> np.ndarray:
    """m_i = (1 - alpha s_x) + alpha s_x ebar_i (Eq. cond-population-gate)."""
    return (1.0 - p.pop_strength * sx) + p.pop_strength * sx * ebar


def transport(h: np.ndarray, pi: np.ndarray, support: np.ndarray, m: np.ndarray, p: GmcParams):
    """M_j, weighted centroid c_j, blend, and RMS restoration
    R_j(u) = u rms(h_j) / (rms(u) + eps).  Returns per-support-member arrays
    in ascending source order, plus the pre-restoration centroids."""
    h = np.asarray(h, np.float64)
    sup = np.sort(np.asarray(support, dtype=np.int64))
    slot = -np.ones(h.shape[0], dtype=np.int64)
    slot[sup] = np.arange(sup.size)
    mass = np.zeros(sup.size)
    acc = np.zeros((sup.size, h.shape[1]))
    np.add.at(mass, slot[pi], m)
    np.add.at(acc, slot[pi], m[:, None] * h)
    cen = acc / mass[:, None]
    v = (1.0 - p.tau_j) * h[sup] + p.tau_j * cen
    rms_h = np.sqrt(np.mean(h[sup] ** 2, axis=1))
    rms_v = np.sqrt(np.mean(v ** 2, axis=1))
    out = v * (rms_h / (rms_v + p.restore_eps))[:, None]
    return dict(support=sup, mass=mass, centroid=cen, out=out)


def compact(support: np.ndarray, htilde: np.ndarray, pos: np.ndarray):
    """Stable, order-preserving gather: ascending source indices, their
    transported states, and their original (t,h,w) ids."""
    sup = np.asarray(support, dtype=np.int64)
    order = np.argsort(sup, kind="stable")
    idx = sup[order]
    return idx, htilde[order], pos[idx]


# ----------------------------------------------------------------------------
# Sequence compaction after pruning (App. H "Index map and physical token
# accounting"; the cached deployment gathers prefix K/V by the same indices)
# ----------------------------------------------------------------------------
def index_map(seq_len: int, vis_start: int, n: int, kept_visual):
    """iota over the original positions of a sequence whose visual tokens sit
    at [vis_start, vis_start + n): the visual positions not kept are deleted
    and every retained position keeps its order.  Returns iota (new position,
    -1 for a deleted one) and keep (the retained original positions, i.e. the
    inverse map), walking the sequence once."""
    kept = {vis_start + int(j) for j in kept_visual}
    iota = np.full(seq_len, -1, dtype=np.int64)
    keep = []
    for i in range(seq_len):
        if vis_start <= i < vis_start + n and i not in kept:
            continue
        iota[i] = len(keep)
        keep.append(i)
    return iota, np.asarray(keep, dtype=np.int64)


def compact_sequence(seq_rows, vis_rows, seq_pos, vis_start: int, n: int, kept_visual):
    """The boundary sequence after compaction: text positions keep their
    states, the retained visual token j receives its transported state (row k
    of vis_rows for the k-th kept token, ascending), and every retained
    position keeps its original position ids.  Returns iota, keep, the rows
    and the position ids."""
    seq_rows = np.asarray(seq_rows)
    iota, keep = index_map(seq_rows.shape[0], vis_start, n, kept_visual)
    out = seq_rows[keep].copy()
    for k, j in enumerate(np.asarray(kept_visual, dtype=np.int64)):
        out[iota[vis_start + j]] = np.asarray(vis_rows)[k]
    return iota, keep, out, np.asarray(seq_pos)[keep]


def gather_cache(cache, keep):
    """Prefix-layer cache rows gathered at the retained original positions
    (axis -2 is the sequence axis)."""
    return np.take(np.asarray(cache), np.asarray(keep, dtype=np.int64), axis=-2)


# ----------------------------------------------------------------------------
# Realisation audit (Prop. 2 Eq. message-bound; App. I Eq.
# cond-message-decomposition, Eq. cond-softmax-bound, Eq. cond-message-polar;
# App. G Eq. cond-message-error)
# ----------------------------------------------------------------------------
def message_audit(q, k, v, k_c, v_c, carrier_of, weights=None, nonvis_lse=None):
    """Signed-message realisation audit of one problem.

    q [T][Hq][dh] queries, k / v [N][Hkv][dh] the full visual keys and values,
    k_c / v_c [K][Hkv][dh] the compact sequence's keys and values at the K
    carriers, carrier_of [N] the carrier slot (0..K-1) each source token was
    transported to, weights [Hq][T] the client weights (uniform 1/(Hq T) when
    None), nonvis_lse [Hq][T] the nonvisual keys' log-sum-exp shared by both
    softmaxes.  Per client g = (h, t):
      y_g = sum_i a_gi v_i (Full), y~_g = sum_j abar_gj v~_j (compact),
      M_gj = sum_(i in C_j) a_gi, term1_g = sum_i a_gi (v_i - v~_pi(i)),
      term2_g = sum_j (M_gj - abar_gj) v~_j  (y - y~ = term1 + term2),
      l1_g = ||M_g - abar_g||_1 and its bound ||u^F_g - u^S_g||_inf with
      u^F_gj = log sum_(i in C_j) exp(s_gi) and u^S_gj the compact logit.
    Stacked with sqrt(weights): e_M = ||Y - Y~|| / (||Y|| + 1e-8), the
    amplitude ratio alpha and the cosine kappa of the polar identity."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    k_c = np.asarray(k_c, np.float64)
    v_c = np.asarray(v_c, np.float64)
    carrier_of = np.asarray(carrier_of, dtype=np.int64)
    t, hq, dh = q.shape
    n, hkv, _ = k.shape
    kc = k_c.shape[0]
    w = np.full((hq, t), 1.0 / (hq * t)) if weights is None else np.asarray(weights, np.float64)
    onehot = np.zeros((n, kc))
    onehot[np.arange(n), carrier_of] = 1.0
    rows = dict(y=np.zeros((hq, t, dh)), yc=np.zeros((hq, t, dh)), term1=np.zeros((hq, t, dh)),
                term2=np.zeros((hq, t, dh)), l1=np.zeros((hq, t)), bound=np.zeros((hq, t)),
                lse_full=np.zeros((hq, t)), lse_comp=np.zeros((hq, t)))
    for h in range(hq):
        g = (h * hkv) // hq
        s_f = q[:, h, :] @ k[:, g, :].T / math.sqrt(dh)          # [T][N]
        s_c = q[:, h, :] @ k_c[:, g, :].T / math.sqrt(dh)        # [T][K]
        lse_f = np.log(np.sum(np.exp(s_f - s_f.max(axis=1, keepdims=True)), axis=1)) + s_f.max(axis=1)
        lse_c = np.log(np.sum(np.exp(s_c - s_c.max(axis=1, keepdims=True)), axis=1)) + s_c.max(axis=1)
        if nonvis_lse is not None:
            lse_f = np.logaddexp(lse_f, np.asarray(nonvis_lse, np.float64)[h])
            lse_c = np.logaddexp(lse_c, np.asarray(nonvis_lse, np.float64)[h])
        a = np.exp(s_f - lse_f[:, None])                         # Full visual attention
        ac = np.exp(s_c - lse_c[:, None])                        # compact attention
        m = a @ onehot                                           # grouped Full mass M_gj
        rows["y"][h] = a @ v[:, g, :]
        rows["yc"][h] = ac @ v_c[:, g, :]
        rows["term1"][h] = a @ (v[:, g, :] - v_c[carrier_of, g, :])
        rows["term2"][h] = (m - ac) @ v_c[:, g, :]
        rows["l1"][h] = np.abs(m - ac).sum(axis=1)
        with np.errstate(divide="ignore"):
            u_f = np.log(m) + lse_f[:, None]                    # grouped Full logits
        rows["bound"][h] = np.max(np.abs(u_f - s_c), axis=1)
        rows["lse_full"][h] = lse_f
        rows["lse_comp"][h] = lse_c
    sw = np.sqrt(w)[:, :, None]
    Y, Yc = sw * rows["y"], sw * rows["yc"]
    ny, nyc = float(np.linalg.norm(Y)), float(np.linalg.norm(Yc))
    diff = float(np.linalg.norm(Y - Yc))
    return dict(rows=rows, e_m=diff / (ny + 1e-8), alpha=nyc / ny if ny > 0 else 0.0,
                kappa=float(np.sum(Y * Yc)) / (ny * nyc) if ny > 0 and nyc > 0 else 0.0,
                norm_y=ny, norm_yc=nyc, norm_diff=diff)


# ----------------------------------------------------------------------------
# The whole operator for one image (Algorithm 1, steps 2-6)
# ----------------------------------------------------------------------------
def view_mass(n_hist: int, p: GmcParams):
    """Masses of the current and the historical message views (reading R14)."""
    if n_hist == 0:
        return [p.beta_msg]
    return [p.beta_msg * (1.0 - p.hist_mass)] + [p.beta_msg * p.hist_mass / n_hist] * n_hist


def message_view(h, q, k, probe, p: GmcParams, nonvis_lse=None, probe_bias=None):
    """One message view (Eq. cond-native-message, Eq. cond-mass-coordinate,
    Eq. cond-grounded-client): value coordinates Z from the view's own states
    and folded probe, the mass coordinate, the native attention slice, atom
    norms, row sums, P^G rows, the view's head-pattern Gram and mean atom
    norms."""
    h = np.asarray(h, np.float64)
    n = h.shape[0]
    t = q.shape[0]
    hq = probe.shape[0]
    _, _, _, xt = row_features(h, p)
    z = value_probe(xt, probe, probe_bias)
    sigma = mass_coordinate(z, p)
    if t == 0:
        return dict(z=z, sigma=sigma, a=np.zeros((hq, 0, n)), e=np.zeros((hq, 0, n)), ell=None,
                    pg=np.zeros((hq, 0, n)), active=np.zeros((hq, 0), dtype=bool), gram=np.zeros((hq, hq)),
                    abar=np.zeros(hq))
    a = native_attention(q, k, nonvis_lse)
    e, ell = grounded_energy_rows(a, z, sigma)
    zrow = e.sum(axis=2)                                     # [Hq][T]
    active = zrow > 0
    pg = np.where(active[:, :, None], e / np.where(active, zrow, 1.0)[:, :, None], 0.0)
    return dict(z=z, sigma=sigma, a=a, e=e, ell=ell, pg=pg, active=active,
                gram=head_pattern_gram(a, z, sigma), abar=e.reshape(hq, -1).mean(axis=1))


def image_seeds(cbar: np.ndarray, img: np.ndarray) -> np.ndarray:
    """S_0 of a multi-image prompt: in every image the token of largest
    singleton gain u_i = F({i}) = sum_m Cbar_mi, ties to the lower index
    (App. H "Batched complementary support")."""
    u = cbar.sum(axis=0)
    seeds = []
    for g in range(int(img.max()) + 1):
        members = np.flatnonzero(img == g)
        seeds.append(int(members[np.argmax(u[members])]))
    return np.asarray(seeds, dtype=np.int64)


def build_clients(h, q, k, pos, probe, p: GmcParams, app_proj=None, nonvis_lse=None, probe_bias=None,
                  hist=(), img=None):
    """Steps 2 of Algorithm 1: the three client banks and all message-side
    quantities.  `hist` lists completed historical message views, each a dict
    of its own hidden, q, k, probe and optionally nonvis_lse, probe_bias
    (App. H native message clients).  `img` gives each token's image (ids
    0..I-1, every id present) for a multi-image prompt: appearance and
    spatial rows then stay within their image (reading R15).  Returns a dict
    of intermediates."""
    h = np.asarray(h, np.float64)
    n = h.shape[0]
    t = q.shape[0]
    norm, x, rms, xt = row_features(h, p)
    hq = probe.shape[0]
    nu = query_weights(t, p)
    cur = message_view(h, q, k, probe, p, nonvis_lse, probe_bias)
    views = [message_view(v["hidden"], v["q"], v["k"], v["probe"], p, v.get("nonvis_lse"), v.get("probe_bias"))
             for v in hist] if t > 0 else []
    mass = view_mass(len(views), p)
    if t > 0:
        pattern = head_pattern([cur["gram"]] + [v["gram"] for v in views],
                               [cur["abar"]] + [v["abar"] for v in views], mass)
        omega, centres, clus = head_weights_from_pattern(pattern, p)
        # population weights use the current view's energy only
        ebar, en = grounded_energy(cur["e"], omega, nu)
    else:
        pattern = np.zeros((hq, hq))
        omega, centres, clus = np.zeros(hq), [], -np.ones(hq, dtype=np.int64)
        ebar, en = np.ones(n), np.zeros(n)
    bounded = n > p.bounded_threshold_n
    if img is not None and (int(img.max()) + 1 > 1) and bounded:
        raise ValueError("multi-image prompts use the exact appearance bank (reading R15)")
    if bounded:
        if app_proj is None:
            raise ValueError("bounded appearance bank needs the projection matrix")
        pv, app_clients = appearance_bank_bounded(h, app_proj, p)
    else:
        pv, app_clients = appearance_bank(x, p, img), np.arange(n)
    ps = spatial_bank(pos, p, img)
    cbar, banks = client_matrix(cur["pg"], cur["active"], omega, nu, pv, ps, p,
                                [v["pg"] for v in views], [v["active"] for v in views], mass)
    return dict(norm=norm, x=x, rms=rms, xt=xt, z=cur["z"], sigma=cur["sigma"], a=cur["a"], e=cur["e"],
                ell=cur["ell"], pg=cur["pg"], active=cur["active"], gram=cur["gram"], abar=cur["abar"],
                pattern=pattern, view_mass=mass, hist_views=views, omega=omega, centres=centres,
                clusters=clus, nu=nu, ebar=ebar, energy=en, pv=pv, ps=ps,
                app_clients=app_clients, cbar=cbar, banks=banks, bounded=bounded,
                pc=spatial_coordinates(pos, img), img=img)


def bank_saturation(cbar: np.ndarray, banks: np.ndarray, support) -> dict:
    """Z_b = F_b(V), omega_b = Z_b / sum Z, c_b = F_b(S)/Z_b and the final
    certificate F(S)/F(V) = sum_b omega_b c_b (Eq. cond-effective-bank-mass,
    Eq. cond-bank-mixture)."""
    sup = np.asarray(list(support), dtype=np.int64)
    out = {}
    zs = {}
    for bnk in np.unique(banks):
        rows = cbar[banks == bnk]
        zb = float(rows.max(axis=1).sum())
        fb = float(rows[:, sup].max(axis=1).sum()) if sup.size else 0.0
        zs[int(bnk)] = (zb, fb)
    tot = sum(v[0] for v in zs.values())
    for bnk, (zb, fb) in zs.items():
        out[bnk] = dict(z=zb, f=fb, omega=zb / tot if tot > 0 else 0.0,
                        c=fb / zb if zb > 0 else 0.0)
    return out


def gmc_single(h, q, k, pos, probe, k_req: int, p: GmcParams = GmcParams(),
               app_proj=None, nonvis_lse=None, keep_intermediates: bool = False, probe_bias=None, hist=(),
               img=None):
    """One problem end to end: budget, clients, selection, assignment,
    transport and compaction.  Returns out_hidden (fp64, before the cast to
    the residual dtype), out_pos, out_idx and diagnostics."""
    h = np.asarray(h, np.float64)
    n = h.shape[0]
    if img is not None:
        img = np.asarray(img, dtype=np.int64)
        n_img = int(img.max()) + 1
        if n_img == 1:
            img = None
    else:
        n_img = 1
    kk = realized_budget(n, k_req, n_img)
    if kk == n:
        return dict(out_hidden=h.copy(), out_pos=np.asarray(pos).copy(),
                    out_idx=np.arange(n, dtype=np.int64), identity=True, k=kk)
    cl = build_clients(h, q, k, pos, probe, p, app_proj, nonvis_lse, probe_bias, hist, img)
    b = p.batch_b_bounded if cl["bounded"] else p.batch_b
    seeds = image_seeds(cl["cbar"], img) if img is not None else ()
    sel = select_support(cl["cbar"], kk, b, p, seeds)
    asg = assign_population(cl["x"], cl["pc"], sel["order"], p, img)
    m = population_weights(cl["ebar"], asg["sx"], p)
    tr = transport(h, asg["pi"], sel["order"], m, p)
    idx, out_h, out_pos = compact(tr["support"], tr["out"], np.asarray(pos))
    res = dict(out_hidden=out_h, out_pos=out_pos, out_idx=idx, identity=False, k=kk,
               selection=sel, assignment=asg, m=m, transport=tr, b=b,
               saturation=bank_saturation(cl["cbar"], cl["banks"], sel["order"]),
               f_v=float(cl["cbar"].max(axis=1).sum()))
    if keep_intermediates:
        res["clients"] = cl
    return res


def gmc(hidden, text_q, vis_k, pos3d, probe, k_req: int, p: GmcParams = GmcParams(),
        app_proj=None, nonvis_lse=None, probe_bias=None):
    """Batched entry: independent problems, same shapes."""
    return [gmc_single(hidden[i], text_q[i], vis_k[i], pos3d[i], probe, k_req, p, app_proj,
                       None if nonvis_lse is None else nonvis_lse[i], probe_bias=probe_bias)
            for i in range(hidden.shape[0])]


def prune_rounds(k: int, n: int, p: GmcParams = GmcParams()) -> int:
    """Number of selection rounds ceil(K / b) for the path N selects."""
    b = p.batch_b_bounded if n > p.bounded_threshold_n else p.batch_b
    kk = realized_budget(n, k)
    return 0 if kk == n else -(-kk // b)

"""GPU parity of the signed-message realisation audit (App. G Eq.
cond-message-error; App. I Eq. cond-message-decomposition, Eq.
cond-softmax-bound, Eq. cond-message-polar) against the fp64 oracle, on
seeded synthetic Full and compact keys, values and carrier maps."""
import numpy as np
import pytest

from oracle import gmc_oracle as O
from paper_2608_02134_amd import synth
from paper_2608_02134_amd.binding import Pruner, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

# Tolerances: fp32 logits of bf16 inputs over dh <= 128 carry absolute errors
# near 1e-6, so attention weights and the messages they sum (over N <= 1296
# terms) are within ~1e-5 relative; bounded by 1e-4 of each client's largest
# message entry (vectors) and 1e-4 relative (norms, e_M, alpha, kappa).
VEC_TOL = 1e-4
REL_TOL = 1e-4

CASES = {
    # the Qwen2.5-VL-7B boundary: 1296 visual tokens, 256 carriers, 64 queries
    "qwen": dict(dtype="bf16", n=1296, k=256, t=64, hq=28, hkv=4, dh=128, nonvis=True, weights=True),
    # ragged: N, K and T off every tile multiple, no nonvisual part, uniform weights
    "ragged_fp32": dict(dtype="f32", n=203, k=37, t=7, hq=8, hkv=2, dh=64, nonvis=False, weights=False),
    "small_heads": dict(dtype="bf16", n=150, k=20, t=20, hq=4, hkv=1, dh=32, nonvis=True, weights=False),
}


def _inputs(seed, dtype, n, k, t, hq, hkv, dh, nonvis, weights):
    rng = np.random.default_rng(seed)
    def draw(shape, scale=1.0):
        a = (rng.standard_normal(shape) * scale).astype(np.float32)
        return synth.round_bf16(a) if dtype == "bf16" else a
    q = draw((1, t, hq, dh), 1.2)
    kf, vf = draw((1, n, hkv, dh)), draw((1, n, hkv, dh))
    kc, vc = draw((1, k, hkv, dh)), draw((1, k, hkv, dh))
    carrier = np.concatenate([np.arange(k), rng.integers(0, k, size=n - k)]).astype(np.int32)
    rng.shuffle(carrier)
    w = rng.uniform(0.2, 1.0, size=(1, hq, t)).astype(np.float32) if weights else None
    nv = (rng.standard_normal((1, hq, t)) * 2).astype(np.float32) if nonvis else None
    return q, kf, vf, kc, vc, carrier[None, :], w, nv


@pytest.mark.parametrize("case", list(CASES))
def test_audit_parity(case):
    c = CASES[case]
    print(f"\n[case] audit {case}: {c}", flush=True)
    q, kf, vf, kc, vc, carrier, w, nv = _inputs(7, **c)
    # a context of the audit's head layout (the probe only sizes the config)
    tdt = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
    probe = torch.zeros((c["hq"], 4, 64), dtype=tdt, device="cuda")
    pr = Pruner(d=64, n_q_heads=c["hq"], n_kv_heads=c["hkv"], head_dim=c["dh"], probe=probe, dtype=tdt,
                max_batch=1, max_n=c["n"], max_t=c["t"])
    try:
        dt = c["dtype"]
        dev = lambda a: to_device(a, dt, torch)
        out, rows, vec = pr.audit(dev(q), dev(kf), dev(vf), dev(kc), dev(vc), torch.from_numpy(carrier).cuda(),
                                  None if w is None else torch.from_numpy(w).cuda(),
                                  None if nv is None else torch.from_numpy(nv).cuda(), rows=True, vectors=True)
        torch.cuda.synchronize()
        out, rows, vec = out.cpu().numpy()[0], rows.cpu().numpy()[0], vec.cpu().numpy()[0]
    finally:
        pr.close()
    ref = O.message_audit(q[0], kf[0], vf[0], kc[0], vc[0], carrier[0], None if w is None else w[0],
                          None if nv is None else nv[0])
    r = ref["rows"]
    for i, key in enumerate(("y", "yc", "term1", "term2")):
        want = r[key]
        scale = np.max(np.abs(r["y"]), axis=2, keepdims=True)
        err = np.max(np.abs(vec[:, :, i, :] - want) / scale)
        print(f"  {key}: max |delta| / max|y_g| = {err:.2e}", flush=True)
        assert err <= VEC_TOL, key
    np.testing.assert_allclose(rows[:, :, 6], r["l1"], rtol=REL_TOL, atol=1e-7)
    np.testing.assert_allclose(rows[:, :, 7], r["bound"], rtol=REL_TOL, atol=1e-5)
    assert np.all(rows[:, :, 6] <= rows[:, :, 7] + 1e-5)        # the contraction bound on the GPU values
    np.testing.assert_allclose(rows[:, :, 3], np.sum((r["y"] - r["yc"]) ** 2, axis=2), rtol=1e-3, atol=1e-9)
    for i, key in enumerate(("e_m", "alpha", "kappa", "norm_y", "norm_yc", "norm_diff")):
        assert out[i] == pytest.approx(ref[key], rel=REL_TOL), key
    assert out[6] <= 1e-5
    # the polar identity on the GPU's own outputs
    e2 = (out[5] / out[3]) ** 2
    assert e2 == pytest.approx(1 + out[1] ** 2 - 2 * out[1] * out[2], rel=1e-3)


def test_audit_after_a_prune():
    """Chained use: prune a Qwen-shape problem, build the compact keys and
    values of the transported states with seeded key / value maps, audit;
    checks what holds at any size: the decomposition, the contraction bound
    and the polar identity on the GPU's outputs."""
    from .gpu_run import run
    prob = synth.make_problem("qwen", grid=(1, 24, 24), t=16, k=96)
    w = prob.workload
    outs, pr = run(prob, torch)
    try:
        g = outs[0]
        rng = np.random.default_rng(3)
        wk = (rng.standard_normal((w.d, w.hkv * w.dh)) / np.sqrt(w.d)).astype(np.float32)
        wv = (rng.standard_normal((w.d, w.hkv * w.dh)) / np.sqrt(w.d)).astype(np.float32)
        proj = lambda hs, m: synth.round_bf16((hs @ m).reshape(1, -1, w.hkv, w.dh).astype(np.float32))
        kf, vf = proj(prob.hidden[0], wk), proj(prob.hidden[0], wv)
        kc, vc = proj(g["out_hidden"], wk), proj(g["out_hidden"], wv)
        slot = {int(j): s for s, j in enumerate(g["out_idx"])}
        carrier = np.array([[slot[int(j)] for j in g["assign"]]], dtype=np.int32)
        dev = lambda a: to_device(a, w.dtype, torch)
        out, rows, vec = pr.audit(dev(prob.text_q), dev(kf), dev(vf), dev(kc), dev(vc),
                                  torch.from_numpy(carrier).cuda(), rows=True, vectors=True)
        torch.cuda.synchronize()
        out, rows, vec = out.cpu().numpy()[0], rows.cpu().numpy()[0], vec.cpu().numpy()[0]
    finally:
        pr.close()
    print(f"\n  e_M {out[0]:.4f} alpha {out[1]:.4f} kappa {out[2]:.4f}", flush=True)
    np.testing.assert_allclose(vec[:, :, 0] - vec[:, :, 1], vec[:, :, 2] + vec[:, :, 3], atol=1e-5)
    assert np.all(rows[:, :, 6] <= rows[:, :, 7] + 1e-5)
    e2 = (out[5] / out[3]) ** 2
    assert e2 == pytest.approx(1 + out[1] ** 2 - 2 * out[1] * out[2], rel=1e-3)
    assert 0.0 < out[0] < 1.0


def test_audit_between_prunes_on_other_streams():
    """The audit's scratch is the client-matrix buffer: an audit on a second
    stream waits for the pruning call before it, and the next pruning call
    on the first stream waits for the audit, so both prunes equal a prune
    run alone (the operator is deterministic)."""
    from .gpu_run import run
    prob = synth.make_problem("qwen", grid=(1, 24, 24), t=16, k=96)
    w = prob.workload
    ref, pr = run(prob, torch, trace=False)
    try:
        dev = lambda a: to_device(a, w.dtype, torch)
        hid, q, kk = dev(prob.hidden), dev(prob.text_q), dev(prob.vis_k)
        pos = torch.from_numpy(prob.pos3d).cuda()
        rng = np.random.default_rng(5)
        vv = dev(synth.round_bf16(rng.standard_normal(prob.vis_k.shape).astype(np.float32)))
        carrier = torch.from_numpy((np.arange(w.n) % prob.k).astype(np.int32)[None, :]).cuda()
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            a = pr.prune(hid, q, kk, pos, prob.k)
        with torch.cuda.stream(s2):
            out, _, _ = pr.audit(q, kk, vv, kk[:, :prob.k].contiguous(), vv[:, :prob.k].contiguous(), carrier)
        with torch.cuda.stream(s1):
            b = pr.prune(hid, q, kk, pos, prob.k)
        torch.cuda.synchronize()
        for res in (a, b):
            assert np.array_equal(res[2][0].cpu().numpy(), ref[0]["out_idx"])
            assert np.array_equal(res[0][0].float().cpu().numpy(), ref[0]["out_hidden"])
        assert np.all(np.isfinite(out.cpu().numpy()))
    finally:
        pr.close()

"""gmc_prune_static (no device allocation; workspace in a static device
array) against gmc_prune_ex (the context's workspace) on the same inputs,
through the C-ABI: two calls in a row, the second smaller, then a call too
large for the array (rejected on the host)."""
import numpy as np
import pytest

from paper_2608_02134_amd import binding, synth
from paper_2608_02134_amd.binding import from_device, make_pruner, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _inputs(prob):
    w = prob.workload
    return (to_device(prob.hidden, w.dtype, torch), to_device(prob.text_q, w.dtype, torch),
            to_device(prob.vis_k, w.dtype, torch), torch.from_numpy(prob.pos3d).cuda())


def _static(cfg, prob, hid, q, kk, pos):
    w = prob.workload
    kr = binding.gmc_realized_k(w.n, prob.k)
    oh = torch.empty((w.batch, kr, w.d), dtype=hid.dtype, device=hid.device)
    op = torch.empty((w.batch, kr, 3), dtype=torch.int32, device=hid.device)
    oi = torch.empty((w.batch, kr), dtype=torch.int32, device=hid.device)
    code = binding.gmc_prune_static(cfg, w.batch, hid.data_ptr(), q.data_ptr(), kk.data_ptr(), pos.data_ptr(),
                                    w.n, w.t, prob.k, oh.data_ptr(), op.data_ptr(), oi.data_ptr(), None,
                                    torch.cuda.current_stream().cuda_stream)
    assert code == binding.GMC_OK, binding.gmc_last_error()
    return oh, op, oi


def test_static_scratch_matches_context_workspace():
    big = synth.make_problem("qwen", grid=(1, 30, 30), t=32, k=150)
    small = synth.make_problem("qwen", grid=(1, 20, 21), t=24, k=83)
    print(f"\n[case] no-alloc: N={big.workload.n} then N={small.workload.n}", flush=True)
    pr = make_pruner(big, torch)
    try:
        results = []
        for prob in (big, small):
            hid, q, kk, pos = _inputs(prob)
            ref = pr.prune(hid, q, kk, pos, prob.k)
            got = _static(pr.cfg, prob, hid, q, kk, pos)
            torch.cuda.synchronize()
            results.append((ref, got))
        for ref, got in results:
            assert torch.equal(got[2], ref[2]), "out_idx"
            assert torch.equal(got[1], ref[1]), "out_pos"
            assert np.array_equal(from_device(got[0], torch), from_device(ref[0], torch)), "out_hidden"
    finally:
        pr.close()


def test_static_scratch_rejects_a_call_beyond_its_size():
    doc = synth.make_problem("doc", grid=(1, 64, 64), t=128, k=820)
    w = doc.workload
    pr = make_pruner(synth.make_problem("qwen", grid=(1, 8, 8), t=4, k=10), torch)   # for a config
    try:
        cfg = binding.GmcConfig.from_buffer_copy(pr.cfg)
        probe = to_device(doc.probe, w.dtype, torch)
        cfg.d, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim = w.d, w.hq, w.hkv, w.dh
        cfg.value_probe = probe.data_ptr()
        hid = torch.zeros((1, w.n, w.d), dtype=torch.bfloat16, device="cuda")
        q = torch.zeros((1, w.t, w.hq, w.dh), dtype=torch.bfloat16, device="cuda")
        kk = torch.zeros((1, w.n, w.hkv, w.dh), dtype=torch.bfloat16, device="cuda")
        pos = torch.zeros((1, w.n, 3), dtype=torch.int32, device="cuda")
        oh = torch.empty((1, doc.k, w.d), dtype=torch.bfloat16, device="cuda")
        op = torch.empty((1, doc.k, 3), dtype=torch.int32, device="cuda")
        oi = torch.empty((1, doc.k), dtype=torch.int32, device="cuda")
        code = binding.gmc_prune_static(cfg, 1, hid.data_ptr(), q.data_ptr(), kk.data_ptr(), pos.data_ptr(),
                                        w.n, w.t, doc.k, oh.data_ptr(), op.data_ptr(), oi.data_ptr())
        assert code == binding.GMC_ERR_CAPACITY
        assert "static scratch" in binding.gmc_last_error()
    finally:
        pr.close()

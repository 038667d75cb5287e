"""Run the HIP operator through the C-ABI binding on seeded inputs and
return numpy results (test infrastructure)."""
from __future__ import annotations

import numpy as np

from paper_2608_02134_amd import binding, synth


def to_device(a: np.ndarray, dtype: str, torch):
    if dtype == "bf16":
        bits = synth.bf16_bits(a).view(np.int16)
        return torch.from_numpy(np.ascontiguousarray(bits)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def from_device(t, torch) -> np.ndarray:
    return t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


def make_pruner(prob: synth.Problem, torch, max_k=0, probe_bias=None, **overrides):
    w = prob.workload
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    probe = to_device(prob.probe, w.dtype, torch)
    proj = None if prob.app_proj is None else to_device(prob.app_proj, w.dtype, torch)
    bias = None if probe_bias is None else torch.from_numpy(np.ascontiguousarray(probe_bias, np.float32)).cuda()
    return binding.Pruner(d=w.d, n_q_heads=w.hq, n_kv_heads=w.hkv, head_dim=w.dh, probe=probe,
                          dtype=tdt, max_batch=w.batch, max_n=w.n, max_t=max(w.t, 1),
                          max_k=max_k, app_projection=proj, probe_bias=bias, **overrides)


def run(prob: synth.Problem, torch, k=None, trace=True, nonvis=None, pruner=None, **overrides):
    """One gmc_prune_ex call; returns (list of per-problem dicts, pruner)."""
    w = prob.workload
    pr = pruner or make_pruner(prob, torch, **overrides)
    hid = to_device(prob.hidden, w.dtype, torch)
    q = to_device(prob.text_q, w.dtype, torch)
    kk = to_device(prob.vis_k, w.dtype, torch)
    pos = torch.from_numpy(prob.pos3d).cuda()
    nv = None if nonvis is None else torch.from_numpy(np.ascontiguousarray(nonvis, np.float32)).cuda()
    kreq = prob.k if k is None else k
    res = pr.prune(hid, q, kk, pos, kreq, nonvis_lse=nv, trace=trace)
    torch.cuda.synchronize()
    outs = []
    for b in range(w.batch):
        d = dict(out_hidden=from_device(res[0][b], torch), out_pos=res[1][b].cpu().numpy(),
                 out_idx=res[2][b].cpu().numpy().astype(np.int64))
        if trace:
            for key, v in res[3].items():
                d[key] = v[b].cpu().numpy()
        outs.append(d)
    return outs, pr

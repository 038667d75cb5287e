"""Run the HIP operator through the C-ABI binding on seeded inputs and
return numpy results (test infrastructure)."""
from __future__ import annotations

import numpy as np

from paper_2608_02134_amd import binding, synth
from paper_2608_02134_amd.binding import from_device, make_pruner, to_device  # noqa: F401


def run(prob: synth.Problem, torch, k=None, trace=True, nonvis=None, pruner=None, hist=None, **overrides):
    """One gmc_prune_ex call (gmc_prune_views with historical views, a list of
    synth.HistView); returns (list of per-problem dicts, pruner)."""
    w = prob.workload
    if prob.n_images > 1 and "max_images" not in overrides:
        overrides["max_images"] = prob.n_images
    pr = pruner or make_pruner(prob, torch, hist=hist, **overrides)
    hid = to_device(prob.hidden, w.dtype, torch)
    q = to_device(prob.text_q, w.dtype, torch)
    kk = to_device(prob.vis_k, w.dtype, torch)
    pos = torch.from_numpy(prob.pos3d).cuda()
    nv = None if nonvis is None else torch.from_numpy(np.ascontiguousarray(nonvis, np.float32)).cuda()
    kreq = prob.k if k is None else k
    hv = None if not hist else [(to_device(v.hidden, w.dtype, torch), to_device(v.text_q, w.dtype, torch),
                                 to_device(v.vis_k, w.dtype, torch)) for v in hist]
    img = None if prob.image_id is None else torch.from_numpy(prob.image_id).cuda()
    res = pr.prune(hid, q, kk, pos, kreq, nonvis_lse=nv, trace=trace, hist=hv, image_id=img,
                   n_images=prob.n_images)
    torch.cuda.synchronize()
    outs = []
    for b in range(w.batch):
        d = dict(out_hidden=from_device(res[0][b], torch), out_pos=res[1][b].cpu().numpy(),
                 out_idx=res[2][b].cpu().numpy().astype(np.int64))
        if trace:
            for key, v in res[3].items():
                d[key] = v[b].cpu().numpy()
            # the call's in-pass certificate and the device status (checked)
            code, dg = binding.gmc_get_diag(b)
            assert code == binding.GMC_OK, f"gmc_get_diag({b}): {binding.gmc_last_error()}"
            d["diag"] = dg if dg["has_certificate"] else None
        outs.append(d)
    return outs, pr
